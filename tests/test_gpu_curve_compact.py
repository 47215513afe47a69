"""GPU parity of fw_dropped_mass_curve and fw_ragged_compact against the
oracle: window importance, the curve, the global allocation and the ragged
gather (bitwise)."""
import math

import numpy as np
import pytest

from oracle import fw_oracle as O
from paper_2608_25230_amd import workloads as W
from tests import parity_workers as PW
from tests.parity import TOL, record, rel_vec, same_bits, t2np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_fw():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_25230_amd import fw
    fw.lib()
    return torch, fw


def _curve(torch, fw, rows, dev=None):
    dev = dev or fw.upload(rows)
    out = fw.dropped_mass_curve(dev["q"], dev["k"], dev["scale"], dev["bias"])
    torch.cuda.synchronize()
    return dev, {key: t2np(val) for key, val in out.items() if not key.startswith("_")}


def _check_curve(rows, out, hs):
    tol = TOL[rows.dtype]
    q, K = rows.as_f64("q"), rows.as_f64("k")
    bias = None if rows.bias is None else rows.bias.astype(np.float64)
    for h in hs:
        r = O.importance(q[h], K[h], float(rows.scale[h]), bias)
        assert rel_vec(out["importance"][h], r) <= tol, h
        c = O.dropped_mass_curve(r)
        cg = out["curve"][h].astype(np.float64)
        assert np.all(np.abs(cg - c) <= tol * np.maximum(c, 1e-7)), h
        # stage 1: the oracle's curve of the GPU's own scores, and the order
        imp = out["importance"][h].astype(np.float64)
        c1 = O.dropped_mass_curve(imp)
        assert np.all(np.abs(cg - c1) <= 1e-6 * np.maximum(c1, 1e-12) + 1e-12), h
        order = np.lexsort((np.arange(imp.size), -imp))
        assert np.array_equal(out["order"][h], order), h


def test_curve_small_shapes(torch_fw):
    torch, fw = torch_fw
    for (H, G, n, d, dt) in [(4, 8, 1500, 64, "bf16"), (3, 5, 777, 32, "f32"), (2, 20, 513, 128, "bf16"),
                             (1, 1, 1, 8, "f32"), (2, 3, 64, 256, "bf16")]:
        rows = W.window_rows(55, n, H, G, n, d, dt)
        dev, out = _curve(torch, fw, rows)
        _check_curve(rows, out, range(H))
        assert np.allclose(out["curve"][:, 0], 1.0, atol=1e-5)
        assert np.all(out["curve"][:, n] == 0.0)
        assert np.all(np.diff(out["curve"], axis=1) <= 0)


@pytest.mark.parametrize("shape", [
    dict(H=3, G=64, n=5000, bias=False),   # ragged last chunk
    dict(H=2, G=16, n=4096, bias=True),
    dict(H=2, G=32, n=777, bias=True),
    dict(H=1, G=48, n=9000, bias=False),
])
def test_curve_window_mfma_shapes(torch_fw, shape):
    """bf16, d = 128, 16..64 window rows: the MFMA importance path."""
    torch, fw = torch_fw
    H, G, n = shape["H"], shape["G"], shape["n"]
    rows = W.window_rows(56, n + G, H, G, n, 128, "bf16")
    if shape["bias"]:
        rng = np.random.default_rng(n)
        bias = (rng.standard_normal(n) * 2.0).astype(np.float32)
        bias[0] = 4.0
        rows = W.Rows(rows.dtype, rows.q, rows.k, rows.v, rows.scale, bias)
    dev, out = _curve(torch, fw, rows)
    _check_curve(rows, out, range(H))
    assert np.allclose(out["curve"][:, 0], 1.0, atol=1e-4)
    assert np.all(out["curve"][:, n] == 0.0)


def test_curve_tied_scores_across_sort_tiles(torch_fw):
    """Unit 0 has zero window queries and an integer bias, so its scores take
    five values over 20000 keys (bitwise ties spread over three tiles of the
    sort); the order must keep equal scores by index.  Unit 1 is ordinary."""
    torch, fw = torch_fw
    H, G, n = 2, 16, 20000
    rows = W.window_rows(57, 7, H, G, n, 128, "bf16")
    q = rows.q.copy()
    q[0] = W.bf16_bits(np.zeros((G, 128), np.float32))
    rng = np.random.default_rng(3)
    bias = np.clip(np.round(rng.standard_normal(n)), -2, 2).astype(np.float32)
    rows = W.Rows(rows.dtype, q, rows.k, rows.v, rows.scale, bias)
    dev, out = _curve(torch, fw, rows)
    _check_curve(rows, out, range(H))
    assert len(np.unique(out["importance"][0])) <= 5


def _compact(torch, fw, k, v, imp, budget, floor, hpl, cap=0):
    out = fw.ragged_compact(k, v, imp, budget, floor, hpl, cap=cap)
    torch.cuda.synchronize()
    res = {}
    for key, val in out.items():
        if key.startswith("_"):
            continue
        if val.dtype == torch.bfloat16:
            res[key] = t2np(val.view(torch.int16)).view(np.uint16)
        else:
            res[key] = t2np(val)
    return res


def _check_compact(Knp, Vnp, imp, out, budget, floor, hpl, elem, cap=0):
    a = O.allocate(imp.astype(np.float64), budget, floor, cap if cap else None)
    c = O.compact(Knp, Vnp, a["keep"], hpl, elem)
    assert np.array_equal(out["offsets"], c["offsets"])
    assert np.array_equal(out["kept_pos"][:budget], c["kept_pos"])
    assert np.array_equal(out["k_out"][:budget].view(np.uint8), c["k_out"].view(np.uint8))
    assert np.array_equal(out["v_out"][:budget].view(np.uint8), c["v_out"].view(np.uint8))
    assert np.array_equal(out["bytes_held"], c["bytes_held"])
    assert out["tau"][0] == np.float32(a["tau"]) or (math.isinf(a["tau"]) and math.isinf(out["tau"][0]))
    assert np.allclose(out["dropped"], a["dropped"], rtol=1e-5, atol=1e-7)
    return a


@pytest.mark.parametrize("case", [
    dict(H=8, hpl=4, n=300, d=64, floor=32, frac=0.1, dt="bf16", ties=True),
    dict(H=6, hpl=2, n=100, d=8, floor=5, frac=0.5, dt="f32", ties=False),
    dict(H=4, hpl=4, n=50, d=3, floor=60, frac=1.0, dt="f32", ties=True),  # floor > n, keep all
    dict(H=5, hpl=1, n=70, d=16, floor=10, frac=0.0, dt="bf16", ties=True),  # floor only
    dict(H=16, hpl=8, n=1000, d=128, floor=0, frac=0.02, dt="bf16", ties=True),
    # budget enforcement: a per-unit cap
    dict(H=8, hpl=4, n=300, d=64, floor=32, frac=0.2, dt="bf16", ties=True, cap=60),
    dict(H=6, hpl=2, n=100, d=8, floor=5, frac=0.5, dt="f32", ties=False, cap=40),
    dict(H=5, hpl=5, n=200, d=16, floor=8, frac=1.0, dt="f32", ties=True, cap=30),   # every unit at its cap
    dict(H=4, hpl=2, n=64, d=8, floor=8, frac=0.5, dt="f32", ties=True, cap=8),      # cap = floor
    dict(H=4, hpl=2, n=64, d=8, floor=4, frac=0.3, dt="f32", ties=True, cap=100),    # cap above n
])
def test_compact_exact(torch_fw, case):
    torch, fw = torch_fw
    rng = np.random.default_rng(7)
    H, n, d = case["H"], case["n"], case["d"]
    imp = rng.random((H, n)).astype(np.float32)
    if case["ties"]:
        imp = np.round(imp * 20) / 20  # many equal scores, ties at tau
        imp = imp.astype(np.float32)
    f = min(case["floor"], n)
    budget = H * f + int(case["frac"] * H * (n - f))
    if case["dt"] == "bf16":
        Knp = rng.integers(0, 1 << 16, (H, n, d)).astype(np.uint16)
        Vnp = rng.integers(0, 1 << 16, (H, n, d)).astype(np.uint16)
        k = torch.from_numpy(Knp.view(np.int16)).cuda().view(torch.bfloat16)
        v = torch.from_numpy(Vnp.view(np.int16)).cuda().view(torch.bfloat16)
        elem = 2
    else:
        Knp = rng.standard_normal((H, n, d)).astype(np.float32)
        Vnp = rng.standard_normal((H, n, d)).astype(np.float32)
        k, v = torch.from_numpy(Knp).cuda(), torch.from_numpy(Vnp).cuda()
        elem = 4
    cap = case.get("cap", 0)
    if cap:
        budget = min(budget, H * min(cap, n))
    out = _compact(torch, fw, k, v, torch.from_numpy(imp).cuda(), budget, case["floor"], case["hpl"], cap)
    a = _check_compact(Knp, Vnp, imp, out, budget, case["floor"], case["hpl"], elem, cap)
    if cap:
        assert a["counts"].max() <= cap


def test_full_size_curve_and_compact(torch_fw):
    """32 x 8 cells, n = 131072, window 64, global 10 % budget with a 32-entry
    floor: sampled cells against the oracle's importance and curve; the
    allocation and gather checked exactly against the oracle's allocation of
    the GPU's own scores."""
    torch, fw = torch_fw
    wl = W.curve_ragged(seed=0)
    rows = wl.rows
    dev, out = _curve(torch, fw, rows)
    _, out2 = _curve(torch, fw, rows, dev)
    for key in out:  # a second call gives the same bits
        assert same_bits(out[key], out2[key]), key
    _check_curve(rows, out, [0, 137])
    assert np.allclose(out["curve"][:, 0], 1.0, atol=1e-4)
    imp_t = torch.from_numpy(out["importance"]).cuda()
    co = fw.ragged_compact(dev["k"], dev["v"], imp_t, wl.budget, wl.floor, wl.heads_per_layer)
    co2 = fw.ragged_compact(dev["k"], dev["v"], imp_t, wl.budget, wl.floor, wl.heads_per_layer)
    torch.cuda.synchronize()
    for key in ("offsets", "kept_pos", "k_out", "v_out", "tau", "dropped", "bytes_held"):
        x, y = co[key], co2[key]
        if x.dtype == torch.bfloat16:
            x, y = x.view(torch.int16), y.view(torch.int16)
        assert same_bits(t2np(x), t2np(y)), key
    del co2
    offsets = t2np(co["offsets"])
    a = O.allocate(out["importance"].astype(np.float64), wl.budget, wl.floor)
    want = np.concatenate([[0], np.cumsum(a["counts"])])
    assert np.array_equal(offsets, want)
    kept = t2np(co["kept_pos"])
    rng = np.random.default_rng(3)
    for h in rng.choice(rows.H, 6, replace=False):
        pos = np.nonzero(a["keep"][h])[0]
        assert np.array_equal(kept[offsets[h]:offsets[h + 1]], pos)
        ko = t2np(co["k_out"][offsets[h]:offsets[h + 1]].view(torch.int16)).view(np.uint16)
        assert np.array_equal(ko, rows.k[h][pos])
        vo = t2np(co["v_out"][offsets[h]:offsets[h + 1]].view(torch.int16)).view(np.uint16)
        assert np.array_equal(vo, rows.v[h][pos])
    bh = t2np(co["bytes_held"])
    assert bh[0] == wl.budget * 2 * 128 * 2 and bh[2] == rows.H * rows.n * 2 * 128 * 2
    assert bh[0] <= bh[1] <= bh[2]
    print("bytes held ragged/padded/full:", bh.tolist(), "tau", t2np(co["tau"])[0])
    # stage 2: against the allocation of the oracle's own float64 scores, the
    # kept sets may differ only at entries whose score is within tolerance of
    # the threshold
    jobs = [(5, 0, h, rows.G, rows.n, rows.d) for h in range(rows.H)]
    r_or = np.stack(PW.pool_map(PW.importance_cell, jobs))
    a2 = O.allocate(r_or, wl.budget, wl.floor)
    keep = np.zeros((rows.H, rows.n), bool)
    for h in range(rows.H):
        keep[h, kept[offsets[h]:offsets[h + 1]]] = True
    diff = keep ^ a2["keep"]
    tau = a2["tau"]
    near = np.abs(r_or - tau) <= TOL[rows.dtype] * tau
    far = int(np.count_nonzero(diff & ~near))
    worst_imp = float(max(rel_vec(out["importance"][h], r_or[h]) for h in range(rows.H)))
    record("allocation_full_size_stage2", differing_entries=int(diff.sum()), beyond_tolerance=far,
           tau=float(tau), worst_importance_rel=worst_imp)
    print("stage 2: entries kept differently", int(diff.sum()), "beyond tolerance of tau", far)
    assert far == 0
    assert worst_imp <= TOL[rows.dtype]


@pytest.mark.parametrize("kernel", [1, 3, 7])
def test_maxpool_scores(torch_fw, kernel):
    """SnapKV's pooling against the oracle, bit for bit (a max of float32
    values), including windows cut by both ends of a unit."""
    torch, fw = torch_fw
    rng = np.random.default_rng(kernel)
    r = rng.random((5, 333)).astype(np.float32)
    out = t2np(fw.maxpool_scores(torch.from_numpy(r).cuda(), kernel))
    assert np.array_equal(out, O.maxpool_scores(r.astype(np.float64), kernel).astype(np.float32))


def test_full_size_enforced_allocation(torch_fw):
    """The full-size cells with SnapKV's pooled score and the uniform per-head
    budget as the cap (enforcement caps every head at SnapKV's count): the
    allocation checked exactly against the oracle on the GPU's own scores."""
    torch, fw = torch_fw
    wl = W.curve_ragged(seed=0)
    rows = wl.rows
    dev, out = _curve(torch, fw, rows)
    pooled = fw.maxpool_scores(torch.from_numpy(out["importance"]).cuda(), 7)
    cap = int(math.ceil(wl.budget / rows.H))
    co = fw.ragged_compact(dev["k"], dev["v"], pooled, wl.budget, wl.floor, wl.heads_per_layer, cap=cap)
    torch.cuda.synchronize()
    a = O.allocate(t2np(pooled).astype(np.float64), wl.budget, wl.floor, cap)
    assert np.array_equal(t2np(co["offsets"]), np.concatenate([[0], np.cumsum(a["counts"])]))
    assert a["counts"].max() <= cap
    kept = t2np(co["kept_pos"])
    offsets = t2np(co["offsets"])
    for h in (0, 77, 255):
        assert np.array_equal(kept[offsets[h]:offsets[h + 1]], np.nonzero(a["keep"][h])[0])
