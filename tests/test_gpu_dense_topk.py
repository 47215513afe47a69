"""GPU parity of fw_dense_topk against the float64 oracle."""
import math

import numpy as np
import pytest

from oracle import fw_oracle as O
from paper_2608_25230_amd import workloads as W
from tests import parity_workers as PW
from tests.parity import TOL, Tally, record, rel_scalar, rel_vec, t2np

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_fw():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_25230_amd import fw
    fw.lib()
    return torch, fw


def _oracle_rows(rows, ks, units=None, gsel=None):
    q, k, v = rows.as_f64("q"), rows.as_f64("k"), rows.as_f64("v")
    bias = None if rows.bias is None else rows.bias.astype(np.float64)
    units = range(rows.H) if units is None else units
    res = {}
    for h in units:
        Z = O.logits(q[h], k[h], float(rows.scale[h]), bias)
        for g in (range(rows.G) if gsel is None else gsel):
            res[(h, g)] = (Z[g], O.row_dense_topk(Z[g], v[h], ks))
    return res


def _compare(rows, ks, out, ref, torch, z_gpu=None):
    tol = TOL[rows.dtype]
    o, o_s, gap, drop, idx = (t2np(out[x]) for x in ("o", "o_s", "gap", "dropped", "topk_idx"))
    tally = Tally()
    worst = dict(o=0.0, o_s=0.0, gap=0.0, dropped=0.0)
    for (h, g), (z, r) in ref.items():
        onorm = np.linalg.norm(r["o"])
        worst["o"] = max(worst["o"], rel_vec(o[h, g], r["o"]))
        for t, k in enumerate(ks):
            worst["o_s"] = max(worst["o_s"], rel_vec(o_s[t, h, g], r["o_s"][t]))
            worst["gap"] = max(worst["gap"], float(rel_scalar(gap[t, h, g], r["gap"][t], 1e-6 * onorm)))
            worst["dropped"] = max(worst["dropped"], float(rel_scalar(drop[t, h, g], r["dropped"][t], 1e-6)))
        kmax = max(ks)
        gset, oset = idx[h, g, :kmax], r["topk_idx"][:kmax]
        exact = np.array_equal(gset, oset)
        tie = False
        if not exact:
            # tie case: every key where the rank orders differ has an oracle
            # logit within tolerance of the logit at that rank
            diff = np.nonzero(gset != oset)[0]
            zk = z[oset[diff]]
            tie = np.all(np.abs(z[gset[diff]] - zk) <= 1e-4 * np.maximum(1.0, np.abs(zk)))
        tally.add(exact, tie, f"row {(h, g)}")
        if z_gpu is not None:  # stage 1: the oracle's rule on the GPU's own logits
            zg = z_gpu[h * rows.G + g].astype(np.float64)
            assert np.array_equal(O.top_mass_set(zg, kmax), gset), f"select logic differs at {(h, g)}"
    assert tally.fail == 0, tally
    for key, val in worst.items():
        assert val <= tol, f"{key}: worst relative error {val:.3g} > {tol}"
    return tally


def _run(torch, fw, rows, ks):
    dev = fw.upload(rows)
    out = fw.dense_topk(dev["q"], dev["k"], dev["v"], ks, dev["scale"], dev["bias"])
    torch.cuda.synchronize()
    R, n = rows.H * rows.G, rows.n
    z_gpu = out["_ws"][: R * n * 4].view(torch.float32).cpu().numpy().reshape(R, n)
    return out, z_gpu


def test_tiny_exhaustive_rows_fp32(torch_fw):
    torch, fw = torch_fw
    wl = W.tiny_exhaustive(seed=0)
    ks = (4, 1, 16, 8)
    out, zg = _run(torch, fw, wl.rows, ks)
    ref = _oracle_rows(wl.rows, ks)
    t = _compare(wl.rows, ks, out, ref, torch, zg)
    print("tiny fp32:", t)
    gap = t2np(out["gap"])
    assert np.all(gap[2] == 0.0)  # k = n keeps everything


@pytest.mark.parametrize("shape", [
    dict(layers=2, kv_heads=2, q_per_kv=2, rows_per_q=16, n=549, d=128, ks=(16, 64, 128)),
    dict(layers=1, kv_heads=3, q_per_kv=1, rows_per_q=7, n=300, d=64, ks=(300, 5, 299)),
    dict(layers=1, kv_heads=1, q_per_kv=3, rows_per_q=11, n=1000, d=100, ks=(1, 999, 64, 2, 500)),
])
def test_streaming_rows_bf16(torch_fw, shape):
    torch, fw = torch_fw
    ks = shape.pop("ks")
    wl = W.streaming_topk(seed=1, ks=ks, **shape)
    out, zg = _run(torch, fw, wl.rows, ks)
    ref = _oracle_rows(wl.rows, ks)
    t = _compare(wl.rows, ks, out, ref, torch, zg)
    print(shape, t)


def test_fp32_ragged_and_equal_logits(torch_fw):
    """Exact ties: q = 0 makes every logit equal the bias; the top-k set must
    then be the lowest indices (ties to the lower index)."""
    torch, fw = torch_fw
    rng = np.random.default_rng(3)
    H, G, n, d = 3, 5, 77, 16
    rows = W.Rows("f32", np.zeros((H, G, d), np.float32), rng.standard_normal((H, n, d)).astype(np.float32),
                  rng.standard_normal((H, n, d)).astype(np.float32), np.ones(H, np.float32),
                  np.round(rng.standard_normal(n), 0).astype(np.float32))
    ks = (1, 10, 40, 77)
    out, zg = _run(torch, fw, rows, ks)
    ref = _oracle_rows(rows, ks)
    _compare(rows, ks, out, ref, torch, zg)
    idx = t2np(out["topk_idx"])
    for (h, g), (z, r) in ref.items():
        assert np.array_equal(idx[h, g], r["topk_idx"])  # exact ties resolved identically


def test_full_size_streaming_all_rows(torch_fw):
    """The 32 x 8 x 256-row workload at n = 4096: every one of the 65,536 rows
    against the oracle (a process pool), in the benchmark's launch
    configuration (no index output) and with the rank-ordered indices; the
    two launches give the same bits for o, o_S, gap and dropped mass."""
    torch, fw = torch_fw
    wl = W.streaming_topk(seed=0)
    r = wl.rows
    ks = wl.ks
    dev = fw.upload(r)
    full = fw.dense_topk(dev["q"], dev["k"], dev["v"], ks, dev["scale"], dev["bias"])
    lean = fw.dense_topk(dev["q"], dev["k"], dev["v"], ks, dev["scale"], dev["bias"], want_idx=False)
    torch.cuda.synchronize()
    o, o_s, gap, drop, idx = (t2np(full[x]) for x in ("o", "o_s", "gap", "dropped", "topk_idx"))
    for key in ("o", "o_s", "gap", "dropped"):
        assert np.array_equal(t2np(lean[key]).view(np.uint32), t2np(full[key]).view(np.uint32)), key
    del dev, full, lean
    jobs = [(h, r.q[h], r.k[h], r.v[h], float(r.scale[h]), r.bias, tuple(ks), o[h], o_s[:, h], gap[:, h],
             drop[:, h], idx[h]) for h in range(r.H)]
    res = PW.pool_map(PW.dense_topk_unit, jobs)
    worst = {key: max(x[0][key] for x in res) for key in res[0][0]}
    exact, tie, fail = (sum(x[1][i] for x in res) for i in range(3))
    where = max(res, key=lambda x: x[0]["o_s"])[2]
    print("full-size all rows:", worst, "exact", exact, "ties", tie, "fail", fail, "worst o_s at", where)
    record("dense_topk_full_size_all_rows", rows=r.H * r.G, worst=worst, exact=exact, ties=tie, fail=fail,
           worst_o_s_at=list(where))
    assert fail == 0 and exact + tie == r.H * r.G
    for key, val in worst.items():
        assert val <= TOL[r.dtype], f"{key}: worst relative error {val:.3g}"
    assert np.all((drop >= 0) & (drop <= 1))
    assert np.all(np.diff(drop, axis=0) <= 1e-7)  # more keys kept, less dropped
    assert np.all(np.isfinite(gap)) and np.all(gap >= 0)
