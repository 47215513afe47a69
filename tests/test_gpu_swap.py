"""GPU parity of fw_swap (the balancing selector) against the oracle."""
import numpy as np
import pytest

from oracle import fw_oracle as O
from paper_2608_25230_amd import workloads as W
from tests.parity import TOL, Tally, rel_scalar, t2np

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


def _check(rows, k, iters, out, cells, method="auto"):
    tol = TOL[rows.dtype]
    q, K, V = rows.as_f64("q"), rows.as_f64("k"), rows.as_f64("v")
    bias = None if rows.bias is None else rows.bias.astype(np.float64)
    tally = Tally()
    for h, g in cells:
        z = O.logits(q[h, g], K[h], float(rows.scale[h]), bias)
        p = O.weights(z)
        S, traj, ns = O.swap_rule(p, V[h], k, iters, start=O.top_mass_set(z, k), method=method)
        gs = out["s_idx"][h, g]
        gt = out["gap_traj"][h, g]
        gn = int(out["n_swaps"][h, g])
        assert np.all(np.diff(gs) > 0)
        # the trajectory is the float64 es of each accepted set
        es_final_gpu = O.forced_error(p, V[h], gs)
        assert rel_scalar(gt[gn], es_final_gpu, 1e-9) <= tol
        assert rel_scalar(gt[0], traj[0], 1e-9) <= tol
        assert np.all(np.diff(gt[: gn + 1]) < 0)
        assert np.all(np.isnan(gt[gn + 1:]))
        exact = np.array_equal(gs, S) and gn == ns
        if exact:
            assert np.allclose(gt[: gn + 1], traj[: ns + 1], rtol=tol)
        tie = abs(es_final_gpu - traj[ns]) <= tol * traj[ns] + 1e-12
        tally.add(exact, tie, f"{(h, g)} gpu {gn} swaps es {es_final_gpu:.6g}, oracle {ns} es {traj[ns]:.6g}")
        assert abs(out["dropped"][h, g] - O.dropped_mass(p, gs)) <= tol * max(O.dropped_mass(p, gs), 1e-6)
    assert tally.fail == 0, tally
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
    t = _check(wl.rows, wl.k, 64, out, [(h, 0) for h in range(wl.rows.H)], method="direct")
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
    t = _check(wl.rows, k, it, out, cells, method="gform")
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
    benchmark's launch configuration; two rows against the oracle, properties
    on all rows."""
    torch, fw = torch_fw
    wl = W.swap_long_rows(seed=0)
    out = _run(torch, fw, wl.rows, wl.k, wl.max_iters)
    t = _check(wl.rows, wl.k, wl.max_iters, out, [(0, 0), (5, 77)], method="gform")
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
    The sets must still match the oracle (ties to the smaller (i, j))."""
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
    t = _check(rows, k, 4, out, [(0, 0), (0, 1)], method="gform")
    assert np.all(out["n_swaps"] >= 1)
    print("tied pairs:", t)
