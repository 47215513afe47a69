"""Python binding of libfw (ctypes).  Argument marshalling only: every step of
the computation runs in the HIP library.  PyTorch supplies device memory and
the current stream.  If libfw.so is missing the calls raise FwError; there is
no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libfw.so")

FW_F32, FW_BF16 = 0, 1
STATUS = {0: "FW_OK", 1: "FW_E_NULL", 2: "FW_E_SHAPE", 3: "FW_E_DTYPE", 4: "FW_E_UNSUPPORTED",
          5: "FW_E_WORKSPACE", 6: "FW_E_HIP"}
ENTRY_POINTS = ("fw_dense_topk", "fw_best_subset", "fw_swap", "fw_dropped_mass_curve",
                "fw_ragged_compact", "fw_pool_subset", "fw_group_vote", "fw_maxpool_scores")
# entry points that take no workspace: their scratch is a static device array
NOALLOC_ENTRY_POINTS = ("fw_dense_topk_noalloc",)
# columns of fw_pool_subset's stats (FW_POOL_* in include/fw.h)
POOL_STATS = ("es_top", "es_pool", "es_bal", "kappa_hat", "c_hat", "kappa_bal", "dropped", "phi",
              "diam", "sigma", "bound_diam", "bound_var", "ef_fw", "es_geo", "pi_hat", "fw_steps")


class FwError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class Rows(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int32), ("q", ctypes.c_void_p), ("k", ctypes.c_void_p),
                ("v", ctypes.c_void_p), ("H", ctypes.c_int64), ("G", ctypes.c_int64),
                ("n", ctypes.c_int64), ("d", ctypes.c_int64), ("scale", ctypes.c_void_p),
                ("bias", ctypes.c_void_p)]


_lib = None
P = ctypes.c_void_p
I32, I64, SZ = ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
RP = ctypes.POINTER(Rows)

_SIGS = {
    "fw_dense_topk_workspace_size": (SZ, [RP, P, I32]),
    "fw_dense_topk": (I32, [RP, P, I32, P, P, P, P, P, P, SZ, P]),
    "fw_dense_topk_noalloc": (I32, [RP, P, I32, P, P, P, P, P, P]),
    "fw_best_subset_workspace_size": (SZ, [RP, I32]),
    "fw_best_subset": (I32, [RP, I32, P, P, P, P, P, P, P, SZ, P]),
    "fw_swap_workspace_size": (SZ, [RP, I32, I32]),
    "fw_swap": (I32, [RP, I32, I32, P, P, P, P, P, SZ, P]),
    "fw_dropped_mass_curve_workspace_size": (SZ, [RP]),
    "fw_dropped_mass_curve": (I32, [RP, P, P, P, P, SZ, P]),
    "fw_ragged_compact_workspace_size": (SZ, [I64, I64, I64, I64]),
    "fw_maxpool_scores": (I32, [P, I64, I64, I32, P, P]),
    "fw_ragged_compact": (I32, [I32, P, P, I64, I64, I64, I64, P, I64, I32, I64, P, P, P, P, P, P, P,
                                P, SZ, P]),
    "fw_pool_subset_workspace_size": (SZ, [RP, I32, P, P]),
    "fw_pool_subset": (I32, [RP, I32, P, P, I32, I32, P, P, P, P, P, P, ctypes.c_float, P, P, P, SZ, P]),
    "fw_group_vote_workspace_size": (SZ, [RP, I32, I32]),
    "fw_group_vote": (I32, [RP, I32, I32, P, P, P, P, P, SZ, P]),
    "fw_last_error": (ctypes.c_char_p, []),
    "fw_version": (ctypes.c_char_p, []),
}


def lib() -> ctypes.CDLL:
    """Load libfw.so (built in-tree by __graft_entry__.build())."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise FwError(-1, f"{LIB_PATH} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != 0:
        raise FwError(status, lib().fw_last_error().decode())


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _torch():
    import torch
    return torch


def _stream() -> int:
    return _torch().cuda.current_stream().cuda_stream


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.float32:
        return FW_F32
    if t.dtype == torch.bfloat16:
        return FW_BF16
    raise FwError(3, f"unsupported tensor dtype {t.dtype}")


def _rows(q, k, v=None, scale=None, bias=None) -> Rows:
    for name, t in (("q", q), ("k", k), ("v", v), ("scale", scale), ("bias", bias)):
        if t is not None and not (t.is_cuda and t.is_contiguous()):
            raise FwError(2, f"{name} must be a contiguous device tensor")
    if q.dim() != 3 or k.dim() != 3:
        raise FwError(2, "q must be [H][G][d] and k [H][n][d]")
    H, G, d = q.shape
    n = k.shape[1]
    return Rows(_dtype_code(q), q.data_ptr(), k.data_ptr(), _ptr(v), H, G, n, d, _ptr(scale),
                _ptr(bias))


def _workspace(nbytes: int, device):
    torch = _torch()
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


def version() -> str:
    return lib().fw_version().decode()


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------

def dense_topk(q, k, v, ks: Sequence[int], scale=None, bias=None, *, want_o=True, want_os=True,
               want_idx=True, ws=None) -> Dict[str, object]:
    torch = _torch()
    rows = _rows(q, k, v, scale, bias)
    ks_arr = (ctypes.c_int32 * len(ks))(*[int(x) for x in ks])
    H, G, n, d = rows.H, rows.G, rows.n, rows.d
    dev = q.device
    nk = len(ks)
    out = {
        "o": torch.empty((H, G, d), dtype=torch.float32, device=dev) if want_o else None,
        "o_s": torch.empty((nk, H, G, d), dtype=torch.float32, device=dev) if want_os else None,
        "gap": torch.empty((nk, H, G), dtype=torch.float32, device=dev),
        "dropped": torch.empty((nk, H, G), dtype=torch.float32, device=dev),
        "topk_idx": torch.empty((H, G, max(ks)), dtype=torch.int32, device=dev) if want_idx else None,
    }
    L = lib()
    need = L.fw_dense_topk_workspace_size(ctypes.byref(rows), ks_arr, nk)
    if ws is None or ws.numel() < need:
        ws = _workspace(need, dev)
    _check(L.fw_dense_topk(ctypes.byref(rows), ks_arr, nk, _ptr(out["o"]), _ptr(out["o_s"]),
                           _ptr(out["gap"]), _ptr(out["dropped"]), _ptr(out["topk_idx"]),
                           ws.data_ptr(), ws.numel(), _stream()))
    out["_ws"] = ws
    return out


def dense_topk_noalloc(q, k, v, ks: Sequence[int], scale=None, bias=None, *, want_o=True, want_os=True,
                       want_idx=True) -> Dict[str, object]:
    """``dense_topk`` through fw_dense_topk_noalloc: the library's static
    per-device scratch array in place of a workspace."""
    torch = _torch()
    rows = _rows(q, k, v, scale, bias)
    ks_arr = (ctypes.c_int32 * len(ks))(*[int(x) for x in ks])
    H, G, n, d = rows.H, rows.G, rows.n, rows.d
    dev = q.device
    nk = len(ks)
    out = {
        "o": torch.empty((H, G, d), dtype=torch.float32, device=dev) if want_o else None,
        "o_s": torch.empty((nk, H, G, d), dtype=torch.float32, device=dev) if want_os else None,
        "gap": torch.empty((nk, H, G), dtype=torch.float32, device=dev),
        "dropped": torch.empty((nk, H, G), dtype=torch.float32, device=dev),
        "topk_idx": torch.empty((H, G, max(ks)), dtype=torch.int32, device=dev) if want_idx else None,
    }
    _check(lib().fw_dense_topk_noalloc(ctypes.byref(rows), ks_arr, nk, _ptr(out["o"]), _ptr(out["o_s"]),
                                       _ptr(out["gap"]), _ptr(out["dropped"]), _ptr(out["topk_idx"]),
                                       _stream()))
    return out


def best_subset(q, k, v, kb: int, scale=None, bias=None, *, ws=None) -> Dict[str, object]:
    torch = _torch()
    rows = _rows(q, k, v, scale, bias)
    H, G = rows.H, rows.G
    dev = q.device
    f = lambda: torch.empty((H, G), dtype=torch.float32, device=dev)
    out = {"best_idx": torch.empty((H, G, kb), dtype=torch.int32, device=dev), "best_gap": f(),
           "topk_gap": f(), "closed": f(), "dropped_topk": f(),
           "topk_idx": torch.empty((H, G, kb), dtype=torch.int32, device=dev)}
    L = lib()
    need = L.fw_best_subset_workspace_size(ctypes.byref(rows), kb)
    if ws is None or ws.numel() < need:
        ws = _workspace(need, dev)
    _check(L.fw_best_subset(ctypes.byref(rows), kb, _ptr(out["best_idx"]), _ptr(out["best_gap"]),
                            _ptr(out["topk_gap"]), _ptr(out["closed"]), _ptr(out["dropped_topk"]),
                            _ptr(out["topk_idx"]), ws.data_ptr(), ws.numel(), _stream()))
    out["_ws"] = ws
    return out


def swap(q, k, v, kb: int, max_iters: int, scale=None, bias=None, *, ws=None) -> Dict[str, object]:
    torch = _torch()
    rows = _rows(q, k, v, scale, bias)
    H, G = rows.H, rows.G
    dev = q.device
    out = {"s_idx": torch.empty((H, G, kb), dtype=torch.int32, device=dev),
           "gap_traj": torch.empty((H, G, max_iters + 1), dtype=torch.float32, device=dev),
           "n_swaps": torch.empty((H, G), dtype=torch.int32, device=dev),
           "dropped": torch.empty((H, G), dtype=torch.float32, device=dev)}
    L = lib()
    need = L.fw_swap_workspace_size(ctypes.byref(rows), kb, max_iters)
    if ws is None or ws.numel() < need:
        ws = _workspace(need, dev)
    _check(L.fw_swap(ctypes.byref(rows), kb, max_iters, _ptr(out["s_idx"]), _ptr(out["gap_traj"]),
                     _ptr(out["n_swaps"]), _ptr(out["dropped"]), ws.data_ptr(), ws.numel(),
                     _stream()))
    out["_ws"] = ws
    return out


def pool_subset(q, k, v, budgets: Sequence, max_swaps: int, scale=None, bias=None, *,
                fw_iters: int = 64, flat_threshold: float = 0.25, want_cells=True, ws=None) -> Dict[str, object]:
    """budgets: a sequence of (s, extra).  Returns, per budget b (lists in the
    same order): pool_idx[b] [H][G][s+extra], best_idx[b], bal_idx[b] and
    geo_idx[b] [H][G][s] (views of the concatenated per-row lists the library
    writes), and stacked n_swaps [nb][H][G], stats [nb][H][G][16] (columns
    POOL_STATS), cell_median and cell_flat [nb][H]."""
    torch = _torch()
    rows = _rows(q, k, v, scale, bias)
    H, G = rows.H, rows.G
    dev = q.device
    nb = len(budgets)
    sv = (ctypes.c_int32 * nb)(*[int(b[0]) for b in budgets])
    ev = (ctypes.c_int32 * nb)(*[int(b[1]) for b in budgets])
    Ptot = sum(int(b[0]) + int(b[1]) for b in budgets)
    Stot = sum(int(b[0]) for b in budgets)
    pool = torch.empty((H, G, Ptot), dtype=torch.int32, device=dev)
    best = torch.empty((H, G, Stot), dtype=torch.int32, device=dev)
    bal = torch.empty((H, G, Stot), dtype=torch.int32, device=dev)
    geo = torch.empty((H, G, Stot), dtype=torch.int32, device=dev)
    out = {"n_swaps": torch.empty((nb, H, G), dtype=torch.int32, device=dev),
           "stats": torch.empty((nb, H, G, len(POOL_STATS)), dtype=torch.float32, device=dev),
           "cell_median": torch.empty((nb, H), dtype=torch.float32, device=dev) if want_cells else None,
           "cell_flat": torch.empty((nb, H), dtype=torch.uint8, device=dev) if want_cells else None}
    L = lib()
    need = L.fw_pool_subset_workspace_size(ctypes.byref(rows), nb, sv, ev)
    if ws is None or ws.numel() < need:
        ws = _workspace(need, dev)
    _check(L.fw_pool_subset(ctypes.byref(rows), nb, sv, ev, max_swaps, fw_iters, pool.data_ptr(), best.data_ptr(),
                            bal.data_ptr(), geo.data_ptr(), _ptr(out["n_swaps"]), _ptr(out["stats"]),
                            float(flat_threshold),
                            _ptr(out["cell_median"]), _ptr(out["cell_flat"]), ws.data_ptr(), ws.numel(),
                            _stream()))
    po = so = 0
    out["pool_idx"], out["best_idx"], out["bal_idx"], out["geo_idx"] = [], [], [], []
    for s_, e_ in budgets:
        out["pool_idx"].append(pool[..., po:po + s_ + e_])
        out["best_idx"].append(best[..., so:so + s_])
        out["bal_idx"].append(bal[..., so:so + s_])
        out["geo_idx"].append(geo[..., so:so + s_])
        po += s_ + e_
        so += s_
    out["_ws"] = ws
    return out


def group_vote(q, k, v, s: int, group_size: int, scale=None, bias=None) -> Dict[str, object]:
    """Rows of a unit ordered (query head) x (position); returns vote_idx
    [H][T][s] (T = G / group_size) and per row es_vote, es_top, dropped."""
    torch = _torch()
    rows = _rows(q, k, v, scale, bias)
    H, G = rows.H, rows.G
    dev = q.device
    f = lambda: torch.empty((H, G), dtype=torch.float32, device=dev)
    out = {"vote_idx": torch.empty((H, max(G // max(group_size, 1), 1), s), dtype=torch.int32, device=dev),
           "es_vote": f(), "es_top": f(), "dropped": f()}
    _check(lib().fw_group_vote(ctypes.byref(rows), s, group_size, _ptr(out["vote_idx"]), _ptr(out["es_vote"]),
                               _ptr(out["es_top"]), _ptr(out["dropped"]), None, 0, _stream()))
    return out


def dropped_mass_curve(q, k, scale=None, bias=None, *, want_order=True, ws=None) -> Dict[str, object]:
    torch = _torch()
    rows = _rows(q, k, None, scale, bias)
    H, n = rows.H, rows.n
    dev = q.device
    out = {"importance": torch.empty((H, n), dtype=torch.float32, device=dev),
           "curve": torch.empty((H, n + 1), dtype=torch.float32, device=dev),
           "order": torch.empty((H, n), dtype=torch.int32, device=dev) if want_order else None}
    L = lib()
    need = L.fw_dropped_mass_curve_workspace_size(ctypes.byref(rows))
    if ws is None or ws.numel() < need:
        ws = _workspace(need, dev)
    _check(L.fw_dropped_mass_curve(ctypes.byref(rows), _ptr(out["importance"]), _ptr(out["curve"]),
                                   _ptr(out["order"]), ws.data_ptr(), ws.numel(), _stream()))
    out["_ws"] = ws
    return out


def maxpool_scores(scores, kernel: int):
    """SnapKV's max pooling of [H][n] scores over kernel // 2 positions on
    either side."""
    torch = _torch()
    if not (scores.is_cuda and scores.is_contiguous() and scores.dtype == torch.float32 and scores.dim() == 2):
        raise FwError(2, "scores must be a contiguous [H][n] float32 device tensor")
    out = torch.empty_like(scores)
    _check(lib().fw_maxpool_scores(scores.data_ptr(), scores.shape[0], scores.shape[1], kernel, out.data_ptr(),
                                   _stream()))
    return out


def ragged_compact(k, v, importance, budget: int, floor: int, heads_per_layer: int, *, cap: int = 0,
                   ws=None) -> Dict[str, object]:
    torch = _torch()
    for name, t in (("k", k), ("v", v), ("importance", importance)):
        if not (t.is_cuda and t.is_contiguous()):
            raise FwError(2, f"{name} must be a contiguous device tensor")
    H, n, d = k.shape
    dev = k.device
    out = {"offsets": torch.empty(H + 1, dtype=torch.int64, device=dev),
           "kept_pos": torch.empty(max(budget, 1), dtype=torch.int32, device=dev),
           "k_out": torch.empty((max(budget, 1), d), dtype=k.dtype, device=dev),
           "v_out": torch.empty((max(budget, 1), d), dtype=v.dtype, device=dev),
           "tau": torch.empty(1, dtype=torch.float32, device=dev),
           "dropped": torch.empty(H, dtype=torch.float32, device=dev),
           "bytes_held": torch.empty(3, dtype=torch.int64, device=dev)}
    L = lib()
    need = L.fw_ragged_compact_workspace_size(H, n, d, budget)
    if ws is None or ws.numel() < need:
        ws = _workspace(need, dev)
    _check(L.fw_ragged_compact(_dtype_code(k), k.data_ptr(), v.data_ptr(), H, heads_per_layer, n, d,
                               importance.data_ptr(), budget, floor, cap, out["offsets"].data_ptr(),
                               out["kept_pos"].data_ptr(), out["k_out"].data_ptr(),
                               out["v_out"].data_ptr(), out["tau"].data_ptr(),
                               out["dropped"].data_ptr(), out["bytes_held"].data_ptr(),
                               ws.data_ptr(), ws.numel(), _stream()))
    out["_ws"] = ws
    return out


# ---------------------------------------------------------------------------
# moving generated workloads onto the device
# ---------------------------------------------------------------------------

def upload(rows, device="cuda") -> Dict[str, object]:
    """Copy a workloads.Rows batch to the device as torch tensors (bf16 bits
    are reinterpreted as torch.bfloat16)."""
    torch = _torch()

    def dev(a):
        if a is None:
            return None
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).to(device).view(torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a)).to(device)

    return dict(q=dev(rows.q), k=dev(rows.k), v=dev(rows.v), scale=dev(rows.scale),
                bias=dev(rows.bias))
