"""GPU parity of fw_dense_topk on the fused single-kernel path (bf16, d = 128,
n in {1024, 2048, 4096}, rows per unit a multiple of 16, up to three budgets)
against the float64 oracle, including the rows that the fused kernel hands to
its exact fallback (equal logits, long runs of tied logits at the threshold)."""
import numpy as np
import pytest

from paper_2608_25230_amd import workloads as W
from tests.parity import t2np
from tests.test_gpu_dense_topk import _compare, _oracle_rows

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_fw():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_25230_amd import fw
    fw.lib()
    return torch, fw


def _run(torch, fw, rows, ks, **kw):
    dev = fw.upload(rows)
    out = fw.dense_topk(dev["q"], dev["k"], dev["v"], ks, dev["scale"], dev["bias"], **kw)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("cfg", [
    dict(n=1024, ks=(128,), kv_heads=2, rows_per_q=8),
    dict(n=1024, ks=(1, 1024), kv_heads=1, rows_per_q=8),
    dict(n=2048, ks=(64, 512, 1000), kv_heads=2, rows_per_q=4),
    dict(n=4096, ks=(128, 512, 1024), kv_heads=2, rows_per_q=4),
    dict(n=4096, ks=(4096, 7), kv_heads=1, rows_per_q=4),
])
def test_fused_shapes_all_rows(torch_fw, cfg):
    torch, fw = torch_fw
    ks = cfg.pop("ks")
    wl = W.streaming_topk(seed=11, layers=1, q_per_kv=4, d=128, ks=ks, **cfg)
    out = _run(torch, fw, wl.rows, ks)
    ref = _oracle_rows(wl.rows, ks)
    t = _compare(wl.rows, ks, out, ref, torch)
    print(cfg, t)
    if max(ks) == cfg["n"]:
        gap = t2np(out["gap"])
        assert np.all(gap[list(ks).index(cfg["n"])] == 0.0)


def test_fused_without_bias_and_outputs_optional(torch_fw):
    torch, fw = torch_fw
    wl = W.streaming_topk(seed=12, layers=1, kv_heads=2, q_per_kv=2, rows_per_q=8, n=2048, d=128,
                          ks=(256, 32))
    rows = W.Rows(wl.rows.dtype, wl.rows.q, wl.rows.k, wl.rows.v, wl.rows.scale, None)
    ks = (256, 32)
    full = _run(torch, fw, rows, ks)
    ref = _oracle_rows(rows, ks)
    _compare(rows, ks, full, ref, torch)
    lean = _run(torch, fw, rows, ks, want_o=False, want_os=False, want_idx=False)
    assert np.array_equal(t2np(lean["gap"]), t2np(full["gap"]))
    assert np.array_equal(t2np(lean["dropped"]), t2np(full["dropped"]))


def test_fused_fallback_rows(torch_fw):
    """Rows whose logits are all equal (q = 0, no bias) or take few distinct
    values (q = 0, integer bias: hundreds of keys share the threshold logit)
    leave the fused kernel's histogram selection and are recomputed exactly;
    ordinary rows of the same units stay on the fused path."""
    torch, fw = torch_fw
    wl = W.streaming_topk(seed=13, layers=1, kv_heads=2, q_per_kv=2, rows_per_q=8, n=1024, d=128,
                          ks=(100, 300, 700))
    r = wl.rows
    q = r.q.copy()
    zero = W.bf16_bits(np.zeros(r.d, np.float32))
    q[0, 0] = zero
    q[1, 5] = zero
    q[1, 15] = zero
    rng = np.random.default_rng(5)
    for bias in (None, np.round(rng.standard_normal(r.n) * 1.5).astype(np.float32)):
        rows = W.Rows(r.dtype, q, r.k, r.v, r.scale, bias)
        ks = (100, 300, 700)
        out = _run(torch, fw, rows, ks)
        ref = _oracle_rows(rows, ks)
        _compare(rows, ks, out, ref, torch)
        idx = t2np(out["topk_idx"])
        for (h, g) in ((0, 0), (1, 5), (1, 15)):
            assert np.array_equal(idx[h, g], ref[(h, g)][1]["topk_idx"])  # exact ties: lower index first


def test_fused_matches_general_path(torch_fw):
    """The same rows through the fused kernel (three budgets) and through the
    general three-launch path (four budgets force it) agree to float32
    rounding of the logits."""
    torch, fw = torch_fw
    wl = W.streaming_topk(seed=14, layers=1, kv_heads=2, q_per_kv=2, rows_per_q=8, n=4096, d=128,
                          ks=(128, 512, 1024))
    dev = fw.upload(wl.rows)
    a = fw.dense_topk(dev["q"], dev["k"], dev["v"], (128, 512, 1024), dev["scale"], dev["bias"])
    b = fw.dense_topk(dev["q"], dev["k"], dev["v"], (128, 512, 1024, 2048), dev["scale"], dev["bias"])
    torch.cuda.synchronize()
    ga, gb = t2np(a["gap"]), t2np(b["gap"])[:3]
    assert np.allclose(ga, gb, rtol=2e-2, atol=1e-6)
    oa, ob = t2np(a["o"]), t2np(b["o"])
    assert np.max(np.abs(oa - ob)) <= 2e-2 * np.max(np.abs(ob))
    ia, ib = t2np(a["topk_idx"]), t2np(b["topk_idx"])[..., :1024]
    same = np.mean([len(np.intersect1d(x, y)) / 1024 for x, y in zip(ia.reshape(-1, 1024), ib.reshape(-1, 1024))])
    assert same > 0.995


def test_fused_tied_threshold_logits(torch_fw):
    """Unit 0 stores every key twice (keys 2j and 2j + 1 equal), so with odd
    budgets the threshold logit's equal twin is left out by index alone (the
    exact tier rule); unit 1 keeps distinct logits (one compare per budget).
    Both stay on the fused path (a threshold bin holds a few dozen logits).
    Channel 0 of V is +64 on even keys and -64 on odd ones, so a twin wrongly
    kept or dropped moves o_S far beyond tolerance; and a selected key 2j + 1
    implies that its twin 2j, equal in logit and lower in index, is selected."""
    torch, fw = torch_fw
    ks = (127, 511, 999)
    wl = W.streaming_topk(seed=15, layers=1, kv_heads=2, q_per_kv=2, rows_per_q=8, n=2048, d=128, ks=ks)
    r = wl.rows
    k, v = r.k.copy(), r.v.copy()
    k[0, 1::2] = k[0, 0::2]
    v[0, 0::2, 0] = W.bf16_bits(np.float32(64.0))
    v[0, 1::2, 0] = W.bf16_bits(np.float32(-64.0))
    rows = W.Rows(r.dtype, r.q, k, v, r.scale, r.bias)
    out = _run(torch, fw, rows, ks)
    ref = _oracle_rows(rows, ks)
    t = _compare(rows, ks, out, ref, torch)
    print("tied thresholds:", t)
    # the fused workspace starts with one fallback flag per row: none is set
    R = rows.H * rows.G
    flags = out["_ws"][: R * 4].view(torch.int32).cpu().numpy()
    assert not flags.any(), np.nonzero(flags)
    idx = t2np(out["topk_idx"])
    for g in range(rows.G):
        for kv in ks:
            sel = set(idx[0, g, :kv].tolist())
            odd = [j for j in sel if j % 2 == 1 and j > 1]
            assert all(j - 1 in sel for j in odd), (g, kv)
