// Exact per-row selection helpers shared by the top-k kernels.
#pragma once

#include "fw_common.hpp"

namespace fw {

// Radix select over order-preserving keys: the key of the k-th largest
// element and the number `rem` of elements equal to it that the top-k takes
// (they are the first `rem` ties in index order).
__device__ inline void radix_select_desc(const float *zr, int64_t n, int k, int *hist, int *sh,
                                  uint32_t *key_out, int *rem_out) {
    const int tid = threadIdx.x, nt = blockDim.x;
    uint32_t prefix = 0, pmask = 0;
    int rem = k;
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = tid; i < 256; i += nt) hist[i] = 0;
        __syncthreads();
        for (int64_t j = tid; j < n; j += nt) {
            uint32_t u = ord_key(zr[j]);
            if ((u & pmask) == prefix) atomicAdd(&hist[(u >> shift) & 255u], 1);
        }
        __syncthreads();
        if (tid == 0) {
            int cum = 0, bsel = 0;
            for (int bb = 255; bb >= 0; --bb) {
                if (cum + hist[bb] >= rem) { bsel = bb; break; }
                cum += hist[bb];
            }
            sh[0] = bsel;
            sh[1] = rem - cum;
        }
        __syncthreads();
        prefix |= (uint32_t)sh[0] << shift;
        pmask |= 255u << shift;
        rem = sh[1];
        __syncthreads();
    }
    *key_out = prefix;
    *rem_out = rem;
}

// Index of the rem-th (1-based) element equal to `key`, scanning j ascending.
__device__ inline int64_t nth_tie(const float *zr, int64_t n, uint32_t key, int rem, int *scan, int *sh) {
    const int tid = threadIdx.x, nt = blockDim.x;
    const int64_t chunk = (n + nt - 1) / nt;
    const int64_t lo = tid * chunk, hi = (lo + chunk < n) ? lo + chunk : n;
    int c = 0;
    for (int64_t j = lo; j < hi; ++j) c += (ord_key(zr[j]) == key);
    int total;
    int ex = block_exclusive_scan(c, scan, &total);
    if (ex < rem && rem <= ex + c) {
        int need = rem - ex;
        for (int64_t j = lo; j < hi; ++j) {
            if (ord_key(zr[j]) == key && --need == 0) { sh[2] = (int)j; break; }
        }
    }
    __syncthreads();
    int64_t r = sh[2];
    __syncthreads();
    return r;
}

}  // namespace fw
