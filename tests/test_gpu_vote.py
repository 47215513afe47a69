"""GPU parity of fw_group_vote (Section 2.1's group vote) against the oracle:
groups of one row, small fp32 groups (vector and scalar row loads), model-
shaped bf16 groups and the full-size candidate-set workload on sampled
groups."""
import math

import numpy as np
import pytest

from oracle import fw_oracle as O
from paper_2608_25230_amd import workloads as W
from tests.parity import Tally, rel_scalar, same_bits, t2np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_fw():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_25230_amd import fw
    fw.lib()
    return torch, fw


def _run(torch, fw, rows, s, gs):
    dev = fw.upload(rows)
    out = fw.group_vote(dev["q"], dev["k"], dev["v"], s, gs, dev["scale"], dev["bias"])
    torch.cuda.synchronize()
    return {key: t2np(val) for key, val in out.items()}


def _check(rows, s, gs, out, groups, tol):
    q, K, V = rows.as_f64("q"), rows.as_f64("k"), rows.as_f64("v")
    bias = None if rows.bias is None else rows.bias.astype(np.float64)
    T = rows.G // gs
    tally = Tally()
    for h, t in groups:
        members = [m * T + t for m in range(gs)]
        Z = np.stack([O.logits(q[h, g], K[h], float(rows.scale[h]), bias) for g in members])
        ref = O.group_vote(Z, V[h], s)
        gv = out["vote_idx"][h, t]
        exact = np.array_equal(gv, ref["vote"])
        sc = ref["score"]
        kth = np.sort(sc)[::-1][s - 1]
        tie = set(gv.tolist()) ^ set(ref["vote"].tolist()) <= set(np.nonzero(np.abs(sc - kth) <= tol * kth)[0].tolist())
        tally.add(exact, tie, f"group {(h, t)} gpu {gv} ref {ref['vote']}")
        P = O.weights(Z)
        for i, g in enumerate(members):
            floor = 1e-6 * np.linalg.norm(O.dense_output(P[i], V[h]))
            es_v = ref["es_vote"][i] if exact else O.forced_error(P[i], V[h], np.sort(gv))
            assert rel_scalar(out["es_vote"][h, g], es_v, floor) <= tol, (h, g, "es_vote")
            assert rel_scalar(out["es_top"][h, g], ref["es_top"][i], floor) <= tol, (h, g, "es_top")
            if exact:
                assert rel_scalar(out["dropped"][h, g], ref["dropped"][i], 1e-7) <= tol, (h, g, "dropped")
    assert tally.fail == 0, tally
    return tally


def _fp32_rows(seed, H, G, n, d, temp, sink):
    rng = np.random.default_rng(seed)
    q = (rng.standard_normal((H, G, d)) * temp).astype(np.float32)
    K = rng.standard_normal((H, n, d)).astype(np.float32)
    V = rng.standard_normal((H, n, d)).astype(np.float32)
    bias = None
    if sink:
        bias = np.zeros(n, np.float32)
        bias[0] = sink
    return W.Rows(W.F32, q, K, V, np.full(H, 1.0 / math.sqrt(d), np.float32), bias)


def test_group_of_one_votes_its_own_top_mass_set(torch_fw):
    torch, fw = torch_fw
    rows = _fp32_rows(3, 2, 5, 50, 16, 2.0, 4.0)
    out = _run(torch, fw, rows, 6, 1)
    _check(rows, 6, 1, out, [(h, t) for h in range(2) for t in range(5)], tol=1e-5)
    np.testing.assert_allclose(out["es_vote"], out["es_top"], rtol=1e-6)


@pytest.mark.parametrize("cfg", [
    # (H, G, n, d, s, group_size, temp, sink)
    (2, 6, 40, 16, 4, 3, 2.0, 0.0),    # vector loads
    (2, 8, 37, 12, 6, 4, 3.0, 4.0),    # ragged n, one element per lane
    (3, 4, 64, 64, 8, 2, 1.5, 4.0),
    (2, 4, 300, 16, 80, 2, 1.0, 0.0),  # s > 64: one workgroup argmax per pick
])
def test_small_groups_fp32(torch_fw, cfg):
    torch, fw = torch_fw
    H, G, n, d, s, gs, temp, sink = cfg
    rows = _fp32_rows(30 + n + d, H, G, n, d, temp, sink)
    out = _run(torch, fw, rows, s, gs)
    t = _check(rows, s, gs, out, [(h, t) for h in range(H) for t in range(G // gs)], tol=1e-5)
    print(cfg, t)


def test_model_groups_bf16(torch_fw):
    torch, fw = torch_fw
    wl = W.pool_rows(seed=4, layers=1, kv_heads=2, q_per_kv=4, rows_per_q=6, n=1024)
    out = _run(torch, fw, wl.rows, 8, 4)
    t = _check(wl.rows, 8, 4, out, [(h, t) for h in range(wl.rows.H) for t in range(6)], tol=2e-2)
    print(t)


def test_full_size_groups_sampled(torch_fw):
    """The candidate-set workload (256 units, 4 query heads x 6 positions,
    n = 4096) at s = 8 with groups of the 4 query heads of a position."""
    torch, fw = torch_fw
    wl = W.pool_rows(seed=0)
    out = _run(torch, fw, wl.rows, 8, 4)
    out2 = _run(torch, fw, wl.rows, 8, 4)
    for key in out:  # a second call gives the same bits
        assert same_bits(out[key], out2[key]), key
    rng = np.random.default_rng(11)
    groups = [(int(h), int(t)) for h, t in zip(rng.choice(wl.rows.H, 6, replace=False), rng.integers(0, 6, 6))]
    t = _check(wl.rows, 8, 4, out, groups, tol=2e-2)
    print(t)
    v = out["vote_idx"].reshape(-1, 8)
    assert v.min() >= 0 and v.max() < wl.rows.n
    assert all(np.unique(r).size == 8 for r in v[:256])
    assert np.all(out["es_vote"] >= 0) and np.all(out["es_top"] >= 0)
    assert np.all((out["dropped"] >= 0) & (out["dropped"] <= 1))
