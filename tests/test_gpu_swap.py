"""GPU parity of fw_swap (the balancing selector) against the oracle."""
import numpy as np
import pytest

from oracle import fw_oracle as O
from paper_2608_25230_amd import workloads as W
from tests import parity_workers as PW
from tests.parity import TOL, Tally, record, same_bits, t2np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_fw():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_25230_amd import fw
    fw.lib()
    return torch, fw


def _run(torch, fw, rows, k, iters):
    dev = fw.upload(rows)
    out = fw.swap(dev["q"], dev["k"], dev["v"], k, iters, dev["scale"], dev["bias"])
    torch.cuda.synchronize()
    return {key: t2np(val) for key, val in out.items() if not key.startswith("_")}


def _check(rows, k, iters, out, cells, method="auto", min_exact=0.75, name=None):
    """Each row of `cells` against the oracle's balancing selector, classified
    at the first step where the two trajectories could part (see
    tests.parity_workers.classify_swap); properties of the GPU's outputs on
    every listed row.  At least `min_exact` of the rows must follow the
    oracle exactly, and none may fail."""
    tol = TOL[rows.dtype]
    q, K = rows.as_f64("q"), rows.as_f64("k")
    bias = None if rows.bias is None else rows.bias.astype(np.float64)
    if method == "auto":
        method = "direct" if rows.n <= 32 else "gform"
    jobs = []
    for h, g in cells:
        z = O.logits(q[h, g], K[h], float(rows.scale[h]), bias)
        gs = out["s_idx"][h, g]
        gt = out["gap_traj"][h, g].astype(np.float64)
        gn = int(out["n_swaps"][h, g])
        assert np.all(np.diff(gs) > 0)
        assert np.all(np.diff(gt[: gn + 1]) < 0)
        assert np.all(np.isnan(gt[gn + 1:]))
        p = O.weights(z)
        dref = O.dropped_mass(p, gs)
        assert abs(out["dropped"][h, g] - dref) <= tol * max(dref, 1e-6)
        jobs.append((z, rows.v[h], k, iters, gs, gt, gn, method, PW.SWAP_REL[rows.dtype]))
    res = [PW.classify_swap(j) for j in jobs] if len(jobs) <= 4 else PW.pool_map(PW.classify_swap, jobs)
    tally = Tally()
    for (h, g), (st, note) in zip(cells, res):
        tally.add(st == "exact", st == "tie", f"{(h, g)}: {note}")
    assert tally.fail == 0, tally
    assert tally.exact >= min_exact * len(cells), tally
    if name:
        record(name, rows=len(cells), tally=tally)
    return tally


def test_example_2_3_swap_on_gpu(torch_fw):
    torch, fw = torch_fw
    rows = W.Rows("f32", np.zeros((1, 1, 1), np.float32), np.zeros((1, 3, 1), np.float32),
                  np.array([-1, 1, 5], np.float32).reshape(1, 3, 1), np.ones(1, np.float32),
                  np.log(np.array([0.45, 0.45, 0.10])).astype(np.float32))
    out = _run(torch, fw, rows, 2, 8)
    assert out["s_idx"][0, 0].tolist() == [0, 2]
    assert out["n_swaps"][0, 0] == 1
    assert out["gap_traj"][0, 0, 0] == pytest.approx(0.5, rel=1e-6)
    assert out["gap_traj"][0, 0, 1] == pytest.approx(9 / 22, rel=1e-6)
    assert np.all(np.isnan(out["gap_traj"][0, 0, 2:]))


def test_tiny_rows_all(torch_fw):
    torch, fw = torch_fw
    wl = W.tiny_exhaustive(seed=0)
    out = _run(torch, fw, wl.rows, wl.k, 64)
    t = _check(wl.rows, wl.k, 64, out, [(h, 0) for h in range(wl.rows.H)], method="direct",
               name="swap_tiny_all_rows")
    print("tiny swap:", t)


@pytest.mark.parametrize("shape", [
    dict(kv_heads=2, q_per_kv=2, rows_per_q=4, n=1000, d=128, k=48, max_iters=12),
    dict(kv_heads=1, q_per_kv=3, rows_per_q=3, n=333, d=64, k=100, max_iters=30),
    dict(kv_heads=1, q_per_kv=1, rows_per_q=5, n=130, d=16, k=1, max_iters=5),
    # bf16, d = 128, n a multiple of 16: the MFMA pair sweep
    dict(kv_heads=2, q_per_kv=2, rows_per_q=4, n=1024, d=128, k=100, max_iters=12),
    dict(kv_heads=1, q_per_kv=2, rows_per_q=3, n=2064, d=128, k=600, max_iters=8),
    dict(kv_heads=1, q_per_kv=1, rows_per_q=4, n=4096, d=128, k=1030, max_iters=6),
    # d not a multiple of 8: the element-wise loads beside the 16-byte chunks
    dict(kv_heads=1, q_per_kv=2, rows_per_q=2, n=300, d=20, k=30, max_iters=6),
])
def test_long_rows_bf16(torch_fw, shape):
    torch, fw = torch_fw
    wl = W.swap_long_rows(seed=5, heavy=4, **shape)
    k, it = shape["k"], shape["max_iters"]
    out = _run(torch, fw, wl.rows, k, it)
    cells = [(h, g) for h in range(wl.rows.H) for g in range(wl.rows.G)]
    t = _check(wl.rows, k, it, out, cells, method="gform",
               name="swap_long_rows_n%d_d%d_k%d" % (shape["n"], shape["d"], shape["k"]))
    print(shape, t)


def test_long_rows_fp32_and_zero_iters(torch_fw):
    torch, fw = torch_fw
    rows = W.sink_rows(41, 0, 2, 3, 200, 32, "f32", sink=4.0)
    out = _run(torch, fw, rows, 20, 10)
    _check(rows, 20, 10, out, [(h, g) for h in range(2) for g in range(3)], method="gform")
    out0 = _run(torch, fw, rows, 20, 0)
    assert np.all(out0["n_swaps"] == 0)
    outn = _run(torch, fw, rows, 200, 5)
    assert np.all(outn["n_swaps"] == 0) and np.all(outn["gap_traj"][..., 0] < 1e-6)


def test_full_size_swap_sampled(torch_fw):
    """8 kv units x 128 rows, n = 32768, k = 1024, up to 64 swaps, in the
    benchmark's launch configuration; two rows of every unit (16 rows, one of
    each of the first and the last query head) against the oracle step by
    step, properties on all rows."""
    torch, fw = torch_fw
    wl = W.swap_long_rows(seed=0)
    out = _run(torch, fw, wl.rows, wl.k, wl.max_iters)
    out2 = _run(torch, fw, wl.rows, wl.k, wl.max_iters)
    for key in out:  # a second call gives the same bits
        assert same_bits(out[key], out2[key]), key
    cells = [(h, g) for h in range(wl.rows.H) for g in (3 + 5 * h, wl.rows.G - 1 - 7 * h)]
    t = _check(wl.rows, wl.k, wl.max_iters, out, cells, method="gform", name="swap_full_size_16_rows")
    print("full-size swap sampled:", t, "swaps: median", np.median(out["n_swaps"]),
          "max", out["n_swaps"].max())
    gt = out["gap_traj"]
    ns = out["n_swaps"]
    for h in range(gt.shape[0]):
        for g in range(gt.shape[1]):
            seg = gt[h, g, : ns[h, g] + 1]
            assert np.all(np.diff(seg) < 0) and np.all(np.isnan(gt[h, g, ns[h, g] + 1:]))
    assert np.all((out["dropped"] >= 0) & (out["dropped"] <= 1))


def test_long_rows_tied_pairs_fall_back_to_full_sweep(torch_fw):
    """Uniform weights over keys whose values repeat 8 distinct rows: every
    pair of the same two value kinds ties, so thousands of pairs survive the
    pruned search's lower bound and the row falls back to the full sweep.
    Rows whose oracle path meets a float64 tie may take another tied pair;
    every step must still take a best swap."""
    torch, fw = torch_fw
    rng = np.random.default_rng(11)
    n, d, k = 2048, 128, 512
    base = rng.standard_normal((8, d)).astype(np.float32)
    V = base[rng.integers(0, 8, n)][None]
    K = rng.standard_normal((1, n, d)).astype(np.float32)
    q = np.zeros((1, 2, d), np.float32)
    rows = W.Rows("bf16", W.bf16_bits(q), W.bf16_bits(K), W.bf16_bits(V),
                  np.full(1, 1.0 / np.sqrt(d), np.float32))
    out = _run(torch, fw, rows, k, 4)
    t = _check(rows, k, 4, out, [(0, 0), (0, 1)], method="gform", min_exact=0.0, name="swap_tied_pairs")
    assert np.all(out["n_swaps"] >= 1)
    print("tied pairs:", t)


def test_full_size_rows_converge_to_local_optima(torch_fw):
    """Rows of the full-size workload (n = 32,768, k = 1,024) with room for
    enough swaps: most stop on their own, within about 100 to 700 swaps, and
    the set a row stops at is a local optimum (no (kept, dropped) swap lowers
    its float64 error beyond the float32 search's precision), checked by the
    oracle's full neighbourhood."""
    torch, fw = torch_fw
    wl = W.swap_long_rows(seed=0)
    r = wl.rows
    rows = W.Rows(r.dtype, r.q[:1, :8], r.k[:1], r.v[:1], r.scale[:1], r.bias)
    iters = 2048
    out = _run(torch, fw, rows, wl.k, iters)
    ns = out["n_swaps"][0]
    stopped = [g for g in range(rows.G) if ns[g] < iters]
    print("swaps until the rule stops:", ns.tolist())
    assert len(stopped) >= 6
    q, K = rows.as_f64("q"), rows.as_f64("k")
    bias = rows.bias.astype(np.float64)
    jobs = []
    for g in stopped[:4]:
        z = O.logits(q[0, g], K[0], float(rows.scale[0]), bias)
        jobs.append((z, rows.v[0], out["s_idx"][0, g], float(out["gap_traj"][0, g, ns[g]])))
    res = PW.pool_map(PW.local_optimum_margin, jobs)
    for (es_g, best, gap_gpu), g in zip(res, stopped[:4]):
        assert abs(gap_gpu - es_g) <= PW.SWAP_REL["bf16"] * es_g, (g, gap_gpu, es_g)
        assert best >= es_g * (1 - PW.SWAP_REL["bf16"]), (g, best, es_g)
    record("swap_full_size_converged_local_optima", rows=len(jobs), swaps=[int(ns[g]) for g in stopped[:4]],
           worst_margin=float(min(b / e - 1 for e, b, _ in res)))
