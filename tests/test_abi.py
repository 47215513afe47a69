"""C ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects invalid arguments with the documented status
before anything is launched."""
import ctypes
import os
import re

import pytest

from paper_2608_25230_amd import fw

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fw.h")


def _declared():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(fw_[a-z_]+)\s*\(", txt)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(fw.LIB_PATH):
        pytest.skip("libfw.so not built")
    return fw.lib()


def test_header_declares_every_entry_point():
    names = _declared()
    for ep in fw.ENTRY_POINTS:
        assert ep in names
        if ep != "fw_maxpool_scores":  # the one entry point without a workspace
            assert ep + "_workspace_size" in names


def test_header_declares_the_noalloc_entry_point():
    names = _declared()
    for ep in fw.NOALLOC_ENTRY_POINTS:
        assert ep in names and ep + "_workspace_size" not in names


def test_dense_topk_noalloc_validation(L):
    """Argument errors and a request beyond the static scratch size are
    rejected on the host, before any device is queried."""
    ks = _ks(4, 8)
    call = lambda rows, ks, nk, gap=1, dropped=1: L.fw_dense_topk_noalloc(
        rows, ks, nk, None, None, gap, dropped, None, None)
    assert call(None, ks, 2) == 1
    assert call(_rows(), ks, 2, gap=None) == 1
    assert call(_rows(), _ks(4, 4), 2) == 2
    assert call(_rows(dtype=9), ks, 2) == 3
    # fp32 rows take the general path, whose workspace holds every logit:
    # 4096 rows x 8192 keys x 4 bytes = 128 MiB > the 64 MiB scratch array
    big = _rows(H=1, G=4096, n=8192, d=8)
    need = L.fw_dense_topk_workspace_size(big, ks, 2)
    assert need > 64 << 20
    assert call(big, ks, 2) == 4
    assert b"scratch" in L.fw_last_error()


def test_every_declared_symbol_is_exported(L):
    for name in _declared():
        assert hasattr(L, name), name


def test_version_and_error_string(L):
    assert "libfw" in fw.version()
    assert isinstance(L.fw_last_error(), bytes)


def _rows(dtype=0, H=2, G=3, n=16, d=8, q=1, k=1, v=1):
    # dummy non-NULL addresses: validation fails before any dereference
    return fw.Rows(dtype, q, k, v, H, G, n, d, None, None)


def _ks(*v):
    return (ctypes.c_int32 * len(v))(*v)


def test_dense_topk_validation(L):
    r = _rows()
    ks = _ks(4, 8)
    call = lambda rows, ks, nk, gap=1, dropped=1, ws=1, wsb=1 << 40: L.fw_dense_topk(
        rows, ks, nk, None, None, gap, dropped, None, ws, wsb, None)
    assert call(None, ks, 2) == 1
    assert call(ctypes.byref(_rows(dtype=7)), ks, 2) == 3
    assert call(ctypes.byref(_rows(q=None)), ks, 2) == 1
    assert call(ctypes.byref(_rows(v=None)), ks, 2) == 1
    assert call(ctypes.byref(_rows(d=0)), ks, 2) == 2
    assert call(ctypes.byref(_rows(d=257)), ks, 2) == 2
    assert call(ctypes.byref(_rows(n=0)), ks, 2) == 2
    assert call(ctypes.byref(r), None, 2) == 1
    assert call(ctypes.byref(r), ks, 0) == 2
    assert call(ctypes.byref(r), ks, 9) == 2
    assert call(ctypes.byref(r), _ks(4, 17), 2) == 2
    assert call(ctypes.byref(r), _ks(0), 1) == 2
    assert call(ctypes.byref(r), _ks(4, 4), 2) == 2
    assert call(ctypes.byref(r), ks, 2, gap=None) == 1
    assert call(ctypes.byref(r), ks, 2, ws=None) == 5
    need = L.fw_dense_topk_workspace_size(ctypes.byref(r), ks, 2)
    assert need > 0
    assert call(ctypes.byref(r), ks, 2, wsb=need - 1) == 5
    assert L.fw_dense_topk_workspace_size(ctypes.byref(_rows(d=0)), ks, 2) == 0
    assert b"workspace" in L.fw_last_error() or b"d must" in L.fw_last_error()
    big = _rows(n=20000)
    assert L.fw_dense_topk(ctypes.byref(big), _ks(16385), 1, None, None, 1, 1, 1, 1, 1 << 50,
                           None) == 4


def test_best_subset_validation(L):
    call = lambda rows, k, bi=1, bg=1: L.fw_best_subset(rows, k, bi, bg, None, None, None, None, 1,
                                                        1 << 40, None)
    assert call(ctypes.byref(_rows()), 0) == 2
    assert call(ctypes.byref(_rows()), 17) == 2
    assert call(ctypes.byref(_rows(n=65)), 4) == 4
    assert call(ctypes.byref(_rows(n=64)), 32) == 4  # C(64,32) >= 2^31
    assert call(ctypes.byref(_rows()), 4, bi=None) == 1
    assert call(ctypes.byref(_rows(v=None)), 4) == 1
    r = _rows(n=24)
    assert L.fw_best_subset_workspace_size(ctypes.byref(r), 6) > 0
    assert L.fw_best_subset(ctypes.byref(r), 6, 1, 1, None, None, None, None, None, 0, None) == 5


def test_swap_validation(L):
    call = lambda rows, k, it, si=1, gt=1, ns=1: L.fw_swap(rows, k, it, si, gt, ns, None, 1, 1 << 40,
                                                           None)
    assert call(ctypes.byref(_rows()), 0, 4) == 2
    assert call(ctypes.byref(_rows()), 4, -1) == 2
    assert call(ctypes.byref(_rows()), 4, 5000) == 2
    assert call(ctypes.byref(_rows()), 4, 4, gt=None) == 1
    assert call(ctypes.byref(_rows(dtype=3)), 4, 4) == 3


def test_curve_validation(L):
    call = lambda rows, imp=1, cur=1: L.fw_dropped_mass_curve(rows, imp, cur, None, 1, 1 << 40, None)
    assert call(ctypes.byref(_rows(v=None)), imp=None) == 1
    assert call(ctypes.byref(_rows(v=None)), cur=None) == 1
    assert call(ctypes.byref(_rows(v=None, H=0))) == 2
    assert call(None) == 1


def test_compact_validation(L):
    def call(dtype=1, H=4, hpl=2, n=64, d=8, budget=100, floor=8, cap=0, outs=1):
        return L.fw_ragged_compact(dtype, 1, 1, H, hpl, n, d, 1, budget, floor, cap, outs, outs, outs,
                                   outs, None, None, None, 1, 1 << 40, None)
    assert call(dtype=5) == 3
    assert call(hpl=3) == 2
    assert call(budget=31) == 2  # below H*floor
    assert call(budget=257) == 2  # above H*n
    assert call(floor=-1) == 2
    assert call(cap=4) == 2       # cap below the floor
    assert call(cap=-1) == 2
    assert call(cap=20) == 2      # budget 100 above H*cap = 80
    assert call(outs=None) == 1
    assert L.fw_ragged_compact_workspace_size(4, 64, 8, 100) > 0


def test_maxpool_validation(L):
    assert L.fw_maxpool_scores(None, 2, 8, 7, 1, None) == 1
    assert L.fw_maxpool_scores(1, 2, 8, 7, None, None) == 1
    assert L.fw_maxpool_scores(1, 0, 8, 7, 2, None) == 2
    assert L.fw_maxpool_scores(1, 2, 8, 6, 2, None) == 2     # even kernel
    assert L.fw_maxpool_scores(1, 2, 8, 7, 1, None) == 2     # aliasing
    assert L.fw_maxpool_scores(1, 2, 8, 0, 2, None) == 2


def test_pool_subset_validation(L):
    r = _rows(n=64, d=8)
    def call(rows, s=(4,), e=(8,), ms=4, best=1, stats=1, ws=1, wsb=1 << 40, nb=None, fwi=16):
        sv, ev = _ks(*s), _ks(*e)
        return L.fw_pool_subset(rows, len(s) if nb is None else nb, sv, ev, ms, fwi, None, best, None, None, None,
                                stats, 0.25, None, None, ws, wsb, None)
    assert call(None) == 1
    assert call(ctypes.byref(_rows(dtype=7))) == 3
    assert call(ctypes.byref(_rows(v=None))) == 1
    assert call(ctypes.byref(r), s=(0,)) == 2                 # s < 1
    assert call(ctypes.byref(r), e=(-1,)) == 2                # extra < 0
    assert call(ctypes.byref(_rows(n=6))) == 2                # s + extra > n
    assert call(ctypes.byref(r), ms=-1) == 2
    assert call(ctypes.byref(r), ms=5000) == 2
    assert call(ctypes.byref(r), fwi=-1) == 2
    assert call(ctypes.byref(r), fwi=5000) == 2
    assert call(ctypes.byref(r), s=(4, 8), e=(8, 4), nb=0) == 2
    assert call(ctypes.byref(r), s=(1,) * 5, e=(1,) * 5) == 2   # more than FW_POOL_MAX_BUDGETS
    assert call(ctypes.byref(_rows(n=200)), s=(40,), e=(30,)) == 4   # more than 64 pool keys
    assert call(ctypes.byref(_rows(n=9000))) == 4             # row longer than 8192
    assert call(ctypes.byref(r), best=None) == 1
    assert call(ctypes.byref(r), stats=None) == 1
    assert call(ctypes.byref(r), ws=None) == 5
    assert call(ctypes.byref(r), wsb=0) == 5
    ws = lambda rows, s, e: L.fw_pool_subset_workspace_size(rows, len(s), _ks(*s), _ks(*e))
    assert ws(ctypes.byref(r), (4,), (8,)) > 0
    assert ws(ctypes.byref(r), (4,), (2,)) > 0                # dropped-set enumeration: a token size
    assert ws(ctypes.byref(_rows(n=200)), (40,), (30,)) == 0
    # the paper's four (s, extra) settings in one call
    big = _rows(n=4096, d=128)
    assert ws(ctypes.byref(big), (4, 8, 16, 32), (24, 12, 6, 4)) > 0


def test_group_vote_validation(L):
    call = lambda rows, s=4, gs=2, vote=1, ev=1, et=1: L.fw_group_vote(rows, s, gs, vote, ev, et, None, None, 0, None)
    r = _rows(G=4, n=64, d=8)
    assert call(None) == 1
    assert call(ctypes.byref(_rows(dtype=7))) == 3
    assert call(ctypes.byref(_rows(v=None))) == 1
    assert call(ctypes.byref(r), gs=3) == 2          # does not divide G
    assert call(ctypes.byref(r), gs=0) == 2
    assert call(ctypes.byref(r), s=0) == 2
    assert call(ctypes.byref(r), s=65) == 2          # s > n
    assert call(ctypes.byref(_rows(G=4, n=1000)), s=300) == 4
    assert call(ctypes.byref(_rows(G=4, n=20000)), s=4) == 4   # more LDS than a workgroup has
    assert call(ctypes.byref(r), vote=None) == 1
    assert call(ctypes.byref(r), ev=None) == 1
    assert L.fw_group_vote_workspace_size(ctypes.byref(r), 4, 2) == 0
