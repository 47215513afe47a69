"""GPU parity of fw_pool_subset (candidate set, ES_pool, pool-restricted
balancing, certificate statistics; Definition 2.5, Lemma 2.2, Section 2.3)
against the oracle: the paper's Example 2.3, small rows on every row, model-
shaped bf16 rows, degenerate pools and the benchmark's full size on sampled
rows with properties on all rows."""
import math

import numpy as np
import pytest

from oracle import fw_oracle as O
from paper_2608_25230_amd import workloads as W
from tests import parity_workers as PW
from tests.parity import Tally, record, rel_scalar, same_bits, t2np

pytestmark = pytest.mark.gpu

STATS = ("es_top", "es_pool", "es_bal", "kappa_hat", "c_hat", "kappa_bal", "dropped", "phi",
         "diam", "sigma", "bound_diam", "bound_var", "ef_fw", "es_geo", "pi_hat", "fw_steps")
FW_ITERS = 64


@pytest.fixture(scope="module")
def torch_fw():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_25230_amd import fw
    fw.lib()
    assert tuple(fw.POOL_STATS) == STATS
    return torch, fw


def _run(torch, fw, rows, budgets, max_swaps, threshold=0.25):
    """One call for every budget; a numpy dict per budget."""
    dev = fw.upload(rows)
    o = fw.pool_subset(dev["q"], dev["k"], dev["v"], budgets, max_swaps, dev["scale"], dev["bias"],
                       fw_iters=FW_ITERS, flat_threshold=threshold)
    torch.cuda.synchronize()
    return [{"pool_idx": t2np(o["pool_idx"][b]), "best_idx": t2np(o["best_idx"][b]),
             "bal_idx": t2np(o["bal_idx"][b]), "geo_idx": t2np(o["geo_idx"][b]),
             "n_swaps": t2np(o["n_swaps"][b]), "stats": t2np(o["stats"][b]),
             "cell_median": t2np(o["cell_median"][b]), "cell_flat": t2np(o["cell_flat"][b])}
            for b in range(len(budgets))]


def _check_rows(rows, s, extra, max_swaps, out, hs, tol, gs=None, refs=None):
    """Every row of units hs against the oracle.  Index sets must match or be
    tie cases: top-mass keys whose logits are within tol of the s-th logit,
    extra keys whose single-key errors are within tol of the last one taken,
    and chosen sets whose float64 error is within tol of the oracle's.  The
    Frank-Wolfe estimate: EF_FW within tol (floor 1e-7 D), the geometric set
    equal to the oracle's or, where the two Frank-Wolfe paths parted, a set
    whose float64 error is within tol of the oracle's, with es_geo checked
    against the oracle's error of the GPU's own geometric set."""
    q, K, V = rows.as_f64("q"), rows.as_f64("k"), rows.as_f64("v")
    bias = None if rows.bias is None else rows.bias.astype(np.float64)
    tally = Tally()
    for h in hs:
        for g in (range(rows.G) if gs is None else gs):
            z = O.logits(q[h, g], K[h], float(rows.scale[h]), bias)
            ref = refs[(h, g)] if refs is not None else O.row_pool(z, V[h], s, extra, max_swaps, FW_ITERS)
            p = O.weights(z)
            pid = out["pool_idx"][h, g]
            top_ok = np.array_equal(pid[:s], ref["top"])
            zs = np.sort(z)[::-1]
            top_tie = set(pid[:s].tolist()) ^ set(ref["top"].tolist()) <= set(
                np.nonzero(np.abs(z - zs[s - 1]) <= tol * max(1.0, abs(zs[s - 1])))[0].tolist())
            ex_ok = np.array_equal(pid[s:], ref["extras"])
            e = O.single_key_errors(p, V[h])
            last = e[ref["extras"][-1]] if extra else 0.0
            ex_tie = (not top_ok) or set(pid[s:].tolist()) ^ set(ref["extras"].tolist()) <= set(
                np.nonzero(np.abs(e - last) <= tol * max(last, 1e-300))[0].tolist())
            tally.add(top_ok and ex_ok, top_tie and ex_tie, f"pool row {(h, g)}")
            same_pool = top_ok and ex_ok
            gb, gbal = out["best_idx"][h, g], out["bal_idx"][h, g]
            if same_pool:
                exact = np.array_equal(gb, ref["best_idx"])
                tie = O.forced_error(p, V[h], gb) <= ref["es_pool"] * (1 + tol) + 1e-15
                tally.add(exact, tie, f"best row {(h, g)} gpu {gb} ref {ref['best_idx']}")
                exact = np.array_equal(gbal, ref["bal_idx"]) and out["n_swaps"][h, g] == ref["n_swaps"]
                tie = abs(O.forced_error(p, V[h], gbal) - ref["es_bal"]) <= tol * ref["es_bal"] + 1e-15
                tally.add(exact, tie, f"bal row {(h, g)} gpu {gbal} ref {ref['bal_idx']}")
                ggeo = out["geo_idx"][h, g]
                es_g = O.forced_error(p, V[h], ggeo)
                exact = np.array_equal(ggeo, ref["geo_idx"])
                tie = abs(es_g - ref["es_geo"]) <= tol * ref["es_geo"] + 1e-15
                tally.add(exact, tie, f"geo row {(h, g)} gpu {ggeo} ref {ref['geo_idx']}")
                st = out["stats"][h, g]
                assert rel_scalar(st[STATS.index("es_geo")], es_g, 1e-6 * ref["diam"]) <= tol, (h, g, "es_geo")
                ef_floor = 1e-7 * ref["diam"]
                assert rel_scalar(st[STATS.index("ef_fw")], ref["ef_fw"], ef_floor) <= tol, \
                    (h, g, "ef_fw", st[STATS.index("ef_fw")], ref["ef_fw"])
                if ref["ef_fw"] > ef_floor:
                    assert rel_scalar(st[STATS.index("pi_hat")], ref["pi_hat"], 1e-12) <= 2 * tol, (h, g, "pi_hat")
                assert 0 <= st[STATS.index("fw_steps")] <= FW_ITERS
            floor = 1e-6 * np.linalg.norm(O.dense_output(p, V[h]))
            st = out["stats"][h, g]
            for c, name in enumerate(STATS):
                if name in ("ef_fw", "es_geo", "pi_hat", "fw_steps"):
                    continue  # checked above, against the GPU's own Frank-Wolfe path
                if not same_pool and name in ("es_pool", "es_bal", "kappa_hat", "c_hat", "kappa_bal"):
                    continue
                refv = ref[name]
                if name == "c_hat":
                    assert abs(st[c] - refv) <= tol, (h, g, name, st[c], refv)
                elif math.isinf(refv):
                    assert math.isinf(st[c]), (h, g, name)
                else:
                    fl = floor if name.startswith(("es", "phi", "bound")) else 1e-12
                    assert rel_scalar(st[c], refv, fl) <= tol, (h, g, name, st[c], refv)
    assert tally.fail == 0, tally
    return tally


def _cells(out, G, threshold=0.25):
    drop = out["stats"][..., STATS.index("dropped")].astype(np.float64)
    med = np.array([np.median(drop[h]) for h in range(drop.shape[0])])
    np.testing.assert_allclose(out["cell_median"], med, rtol=1e-6, atol=1e-9)
    assert np.array_equal(out["cell_flat"].astype(bool), out["cell_median"] > threshold)


def _fp32_rows(seed, H, G, n, d, temp=1.0, sink=0.0):
    rng = np.random.default_rng(seed)
    q = (rng.standard_normal((H, G, d)) * temp).astype(np.float32)
    K = rng.standard_normal((H, n, d)).astype(np.float32)
    V = rng.standard_normal((H, n, d)).astype(np.float32)
    bias = None
    if sink:
        bias = np.zeros(n, np.float32)
        bias[0] = sink
    return W.Rows(W.F32, q, K, V, np.full(H, 1.0 / math.sqrt(d), np.float32), bias)


def test_example_2_3_pool_on_gpu(torch_fw):
    """Example 2.3 as an instance (q = 0, bias = log p): the candidate set with
    one extra key is every key, ES_pool = 9/22 at {0, 2}, kappa_hat = 11/9,
    c_hat = 2/11, Phi = 9/20, D = 9/2, sigma^2 = 63/20, one balancing swap."""
    torch, fw = torch_fw
    p = np.array([0.45, 0.45, 0.10])
    rows = W.Rows(W.F32, np.zeros((1, 1, 1), np.float32), np.zeros((1, 3, 1), np.float32),
                  np.array([[[-1.0], [1.0], [5.0]]], np.float32), np.ones(1, np.float32),
                  np.log(p).astype(np.float32))
    out = _run(torch, fw, rows, [(2, 1)], 8)[0]
    st = out["stats"][0, 0]
    assert out["pool_idx"][0, 0].tolist() == [0, 1, 2]
    assert out["best_idx"][0, 0].tolist() == [0, 2] and out["bal_idx"][0, 0].tolist() == [0, 2]
    assert out["n_swaps"][0, 0] == 1
    want = dict(es_top=0.5, es_pool=9 / 22, es_bal=9 / 22, kappa_hat=11 / 9, c_hat=2 / 11, kappa_bal=1.0,
                dropped=0.1, phi=0.45, diam=4.5, sigma=math.sqrt(3.15), bound_diam=0.9,
                bound_var=math.sqrt(0.35), es_geo=0.5, fw_steps=1)
    for c, name in enumerate(STATS):
        if name in want:
            assert st[c] == pytest.approx(want[name], rel=1e-5), name
    # EF(2) = 0: one Frank-Wolfe step from v = 1 toward v = -1 lands on mu = 1/2
    assert st[STATS.index("ef_fw")] <= 1e-6
    assert st[STATS.index("pi_hat")] > 1e5
    assert out["geo_idx"][0, 0].tolist() == [0, 1]


@pytest.mark.parametrize("cfg", [
    # (H, G, n, d, s, extra, temp, sink)
    (3, 7, 48, 16, 4, 8, 2.0, 0.0),     # vectorised rows, odd G (median of one value)
    (2, 8, 61, 12, 3, 9, 3.0, 4.0),     # ragged n, d not a multiple of 8: one element per lane
    (2, 6, 40, 64, 8, 12, 1.5, 4.0),    # the s = 8 setting
    (2, 5, 33, 8, 6, 0, 2.0, 0.0),      # no extra keys: the pool is A*_s
    (2, 6, 50, 16, 30, 3, 2.5, 4.0),    # few dropped keys: enumeration through the dropped set
    (2, 6, 20, 16, 2, 4, 3.0, 0.0),     # dropped set larger than the kept set, still direct
    (1, 3, 4500, 16, 6, 10, 2.0, 4.0),  # over 16 keys per thread: the top-key picks rescan LDS
    (1, 3, 100, 16, 62, 2, 2.0, 0.0),   # a pool of 64 keys: the full mask, one balancing lane per key
    (2, 3, 200, 16, 4, 24, 2.0, 4.0),   # 28 keys, walks of 14: a walk width not a multiple of four
    (1, 2, 120, 16, 32, 5, 2.0, 0.0),   # dropped sets of 37 keys over three ranges, walks of up to 15
])
def test_small_rows_fp32_all(torch_fw, cfg):
    torch, fw = torch_fw
    H, G, n, d, s, extra, temp, sink = cfg
    rows = _fp32_rows(100 + H * n + d, H, G, n, d, temp, sink)
    out = _run(torch, fw, rows, [(s, extra)], 16)[0]
    t = _check_rows(rows, s, extra, 16, out, range(H), tol=1e-5)
    _cells(out, G)
    print(cfg, t)
    if extra == 0:
        assert np.all(out["n_swaps"] == 0)
        assert np.array_equal(np.sort(out["pool_idx"], axis=-1), out["best_idx"])


def test_several_budgets_in_one_call(torch_fw):
    """Walk and dropped-set enumerations, an empty extra set and a repeated
    budget in one call: each budget's lists and statistics match the oracle
    and a call with that budget alone."""
    torch, fw = torch_fw
    H, G, n, d = 2, 6, 40, 32
    rows = _fp32_rows(77, H, G, n, d, 2.0, 4.0)
    budgets = [(4, 8), (10, 3), (2, 0), (4, 8)]
    outs = _run(torch, fw, rows, budgets, 16)
    for (s, extra), out in zip(budgets, outs):
        t = _check_rows(rows, s, extra, 16, out, range(H), tol=1e-5)
        _cells(out, G)
        alone = _run(torch, fw, rows, [(s, extra)], 16)[0]
        for key in ("pool_idx", "best_idx", "bal_idx", "n_swaps", "stats"):
            assert np.array_equal(out[key], alone[key]), (s, extra, key)
        print((s, extra), t)


def test_pool_of_every_key_matches_exhaustive(torch_fw):
    """s + extra = n: the candidate set is every key, so ES_pool is the full
    ES that fw_best_subset computes on the same rows."""
    torch, fw = torch_fw
    H, G, n, d, s = 2, 8, 16, 32, 4
    rows = _fp32_rows(9, H, G, n, d, 2.0, 4.0)
    out = _run(torch, fw, rows, [(s, n - s)], 32)[0]
    dev = fw.upload(rows)
    ex = fw.best_subset(dev["q"], dev["k"], dev["v"], s, dev["scale"], dev["bias"])
    torch.cuda.synchronize()
    assert np.array_equal(out["best_idx"], t2np(ex["best_idx"]))
    np.testing.assert_allclose(out["stats"][..., STATS.index("es_pool")], t2np(ex["best_gap"]), rtol=1e-6)
    _check_rows(rows, s, n - s, 32, out, range(H), tol=1e-5)


def test_model_rows_bf16(torch_fw):
    """Model-shaped bf16 rows (outlier channels, sink) at n = 1024, every row,
    the paper's four budgets in one call."""
    torch, fw = torch_fw
    wl = W.pool_rows(seed=3, layers=1, kv_heads=2, q_per_kv=2, rows_per_q=3, n=1024)
    budgets = wl.meta["budgets"]
    outs = _run(torch, fw, wl.rows, budgets, 64)
    for (s, extra), out in zip(budgets, outs):
        t = _check_rows(wl.rows, s, extra, 64, out, range(wl.rows.H), tol=2e-2)
        _cells(out, wl.rows.G)
        print((s, extra), t)


def test_full_size_pool_sampled(torch_fw):
    """The benchmark's workload (256 units x 24 rows, n = 4096, the paper's
    four budgets in one call): 16 sampled rows per budget (4 rows of 4 units)
    against the oracle, properties of the statistics on all rows."""
    torch, fw = torch_fw
    wl = W.pool_rows(seed=0)
    budgets = wl.meta["budgets"]
    outs = _run(torch, fw, wl.rows, budgets, wl.max_iters)
    outs2 = _run(torch, fw, wl.rows, budgets, wl.max_iters)
    for o1, o2 in zip(outs, outs2):  # a second call gives the same bits
        for key in o1:
            assert (o1[key] is None and o2[key] is None) or same_bits(o1[key], o2[key]), key
    rng = np.random.default_rng(5)
    r = wl.rows
    bias = None if r.bias is None else r.bias.astype(np.float64)
    for (s, extra), out in zip(budgets, outs):
        hs = sorted(rng.choice(r.H, 4, replace=False).tolist())
        gs = sorted(rng.choice(r.G, 4, replace=False).tolist())
        cells = [(h, g) for h in hs for g in gs]
        jobs = []
        for h, g in cells:
            z = O.logits(PW._bf16(r.q[h, g]), PW._bf16(r.k[h]), float(r.scale[h]), bias)
            jobs.append((z, r.v[h], s, extra, wl.max_iters, FW_ITERS))
        refs = dict(zip(cells, PW.pool_map(PW.pool_row_ref, jobs)))
        tally = Tally()
        for u, h in enumerate(hs):
            sub = {k2: v2[[h]] for k2, v2 in out.items() if v2 is not None and v2.shape[0] == r.H}
            t = _check_rows(r.unit(h), s, extra, wl.max_iters, sub, [0], tol=2e-2, gs=gs,
                            refs={(0, g): refs[(h, g)] for g in gs})
            tally.exact += t.exact
            tally.ties += t.ties
        record(f"pool_full_size_s{s}_extra{extra}", rows=len(cells), tally=tally)
        print((s, extra), tally)
        st = out["stats"].reshape(-1, len(STATS))
        col = {name: st[:, c].astype(np.float64) for c, name in enumerate(STATS)}
        eps = 1e-5
        assert np.all(col["kappa_hat"] >= 1 - eps) and np.all((col["c_hat"] >= 0) & (col["c_hat"] <= 1))
        assert np.all(col["es_pool"] <= col["es_bal"] * (1 + eps) + 1e-12)
        assert np.all(col["es_bal"] <= col["es_top"] * (1 + eps) + 1e-12)
        assert np.all(col["es_top"] <= col["bound_diam"] * (1 + eps))
        assert np.all(col["es_top"] <= col["bound_var"] * (1 + eps))
        np.testing.assert_allclose(col["phi"], col["es_top"] * (1 - col["dropped"]), rtol=1e-4)
        # the geometric set is one of the pool's s-subsets, and Frank-Wolfe
        # starts at a pool value no farther than D from mu
        assert np.all(col["es_geo"] >= col["es_pool"] * (1 - eps) - 1e-12)
        assert np.all(col["ef_fw"] <= col["diam"] * (1 + eps))
        assert np.all((col["fw_steps"] >= 0) & (col["fw_steps"] <= FW_ITERS))
        assert np.all((out["n_swaps"] >= 0) & (out["n_swaps"] <= wl.max_iters))
        pid = out["pool_idx"].reshape(-1, s + extra)
        assert all(np.unique(r).size == s + extra for r in pid[:64]) and pid.min() >= 0 and pid.max() < 4096
        bi = out["best_idx"].reshape(-1, s)
        assert np.all(np.diff(bi, axis=1) > 0)
        _cells(out, wl.rows.G)


@pytest.mark.parametrize("budget", [(32, 5), (32, 6)])
def test_cap_widening_full_length_rows(torch_fw, budget):
    """The widened enumeration cap of Section 2.2 (Enumeration: five and six
    keys beyond A*_32, C(37, 5) = 435,897 and C(38, 6) = 2,760,681 subsets per
    row) on full-length bf16 rows (n = 4096): 8 rows against the oracle, which
    enumerates every s-subset of the pool."""
    torch, fw = torch_fw
    s, extra = budget
    wl = W.pool_rows(seed=7, layers=1, kv_heads=1, q_per_kv=4, rows_per_q=2, n=4096)
    r = wl.rows
    out = _run(torch, fw, r, [budget], 64)[0]
    bias = None if r.bias is None else r.bias.astype(np.float64)
    cells = [(0, g) for g in range(r.G)]
    jobs = [(O.logits(PW._bf16(r.q[h, g]), PW._bf16(r.k[h]), float(r.scale[h]), bias), r.v[h], s, extra, 64,
             FW_ITERS) for h, g in cells]
    refs = dict(zip(cells, PW.pool_map(PW.pool_row_ref, jobs, workers=min(8, len(jobs)))))
    t = _check_rows(r, s, extra, 64, out, [0], tol=2e-2, refs=refs)
    record(f"pool_cap_widening_s{s}_extra{extra}", rows=len(cells), subsets_per_row=math.comb(s + extra, s),
           tally=t)
    print(budget, t)
    st = out["stats"].reshape(-1, len(STATS))
    assert np.all(st[:, STATS.index("es_pool")] <= st[:, STATS.index("es_top")] * (1 + 1e-5))
