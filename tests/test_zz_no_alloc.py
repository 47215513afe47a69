"""fw_dense_topk_noalloc (the library's static per-device scratch array in
place of a workspace) against fw_dense_topk, the entry point whose kernels it
shares: outputs must be bitwise equal, on two calls in a row, the second with a
smaller input, on both the fused bf16 path and the general path."""
import numpy as np
import pytest

from paper_2608_25230_amd import fw

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _device():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    return "cuda:0"


def _inputs(dtype, H, G, n, d, seed, bias):
    g = torch.Generator().manual_seed(seed)
    q = torch.randn(H, G, d, generator=g).to(dtype)
    k = torch.randn(H, n, d, generator=g).to(dtype)
    v = torch.randn(H, n, d, generator=g).to(dtype)
    b = None
    if bias:
        b = torch.zeros(n)
        b[0] = 4.0
    dev = _device()
    to = lambda t: None if t is None else t.to(dev).contiguous()
    return to(q), to(k), to(v), to(b)


def _compare(a, b, what):
    for key in ("o", "o_s", "gap", "dropped", "topk_idx"):
        x, y = a[key], b[key]
        assert (x is None) == (y is None), (what, key)
        if x is None:
            continue
        xn, yn = x.cpu().numpy(), y.cpu().numpy()
        assert np.array_equal(xn.view(np.uint32) if xn.dtype == np.float32 else xn,
                              yn.view(np.uint32) if yn.dtype == np.float32 else yn), (what, key)


# (dtype, H, G, n, d, ks, bias): the first two take the fused bf16 kernel,
# the last two the general path; each pair runs the larger input first
CASES = [
    (torch.bfloat16, 4, 32, 2048, 128, (64, 256, 512), True),
    (torch.bfloat16, 2, 16, 1024, 128, (32, 128), False),
    (torch.float32, 3, 5, 300, 64, (7, 40, 299), True),
    (torch.float32, 2, 3, 77, 16, (5, 77), False),
]


@pytest.mark.parametrize("pair", [(0, 1), (2, 3)], ids=["fused", "general"])
def test_noalloc_matches_the_workspace_entry_point(pair):
    for rep, ci in enumerate(pair):
        dtype, H, G, n, d, ks, bias = CASES[ci]
        print(f"noalloc case {ci}: dtype={dtype} H={H} G={G} n={n} d={d} ks={ks}", flush=True)
        q, k, v, b = _inputs(dtype, H, G, n, d, seed=100 + ci, bias=bias)
        ref = fw.dense_topk(q, k, v, ks, None, b)
        got = fw.dense_topk_noalloc(q, k, v, ks, None, b)
        torch.cuda.synchronize()
        _compare(got, ref, f"case {ci} call {rep}")
        # outputs the caller leaves out stay out
        part = fw.dense_topk_noalloc(q, k, v, ks, None, b, want_o=False, want_os=False, want_idx=False)
        torch.cuda.synchronize()
        assert np.array_equal(part["gap"].cpu().numpy().view(np.uint32), ref["gap"].cpu().numpy().view(np.uint32))
        assert np.array_equal(part["dropped"].cpu().numpy().view(np.uint32),
                              ref["dropped"].cpu().numpy().view(np.uint32))


def test_noalloc_rejects_a_request_beyond_the_scratch():
    dev = _device()
    q = torch.zeros(1, 4096, 8, device=dev)
    k = torch.zeros(1, 8192, 8, device=dev)
    v = torch.zeros(1, 8192, 8, device=dev)
    with pytest.raises(fw.FwError) as e:
        fw.dense_topk_noalloc(q, k, v, (4, 8))
    assert e.value.status == 4 and "scratch" in str(e.value)
