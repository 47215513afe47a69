// Launchers whose kernels are not in this build yet: they report
// hipErrorNotSupported, which the ABI turns into FW_E_HIP.
#include "fw_internal.hpp"

namespace fw {
size_t best_subset_ws_bytes(int64_t, int) { return 256; }
hipError_t launch_best_subset(const fw_rows &, int, int32_t *, float *, float *, float *, float *,
                              int32_t *, void *, hipStream_t) { return hipErrorNotSupported; }
size_t swap_ws_bytes(const fw_rows &, int, int) { return 256; }
hipError_t launch_swap(const fw_rows &, int, int, int32_t *, float *, int32_t *, float *, void *,
                       hipStream_t) { return hipErrorNotSupported; }
size_t curve_ws_bytes(const fw_rows &) { return 256; }
hipError_t launch_curve(const fw_rows &, float *, float *, int32_t *, void *, hipStream_t) {
    return hipErrorNotSupported;
}
size_t compact_ws_bytes(int64_t, int64_t) { return 256; }
hipError_t launch_compact(int, const void *, const void *, int64_t, int64_t, int64_t, int64_t,
                          const float *, int64_t, int, int64_t *, int32_t *, void *, void *, float *,
                          float *, int64_t *, void *, hipStream_t) { return hipErrorNotSupported; }
}  // namespace fw
