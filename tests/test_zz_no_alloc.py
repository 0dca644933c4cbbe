"""gbla_forward_noalloc against gbla_forward (GPU, through the C ABI).

The no-allocation entry point runs the same kernels as gbla_forward with its
scratch in the library's fixed device array, so on the same inputs it gives
the same bits.  Two calls in a row, the second on a smaller input, each
compared with gbla_forward on its own workspace; then a shape whose scratch
exceeds the array is refused.
"""
import pytest
import torch

from paper_2606_07317_amd import inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


@pytest.fixture(scope="module")
def G():
    from paper_2606_07317_amd import gbla
    gbla.load_library()
    return gbla


def _both(G, w, dev):
    inp = inputs.make_inputs(w)
    t = inputs.device_tensors(inp, dev)
    args = (t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"])
    kw = dict(eps=inp.eps, cu_seqlens=t["cu_seqlens"], max_seqlen=t["max_seqlen"])
    out = torch.empty(t["q"].shape, dtype=torch.float32, device=dev)
    y0 = G.forward_noalloc(*args, out=out, **kw)
    ref = G.forward(*args, **kw)
    torch.cuda.synchronize()
    return y0, ref


def test_noalloc_matches_forward_twice_second_smaller(G, dev):
    print("no-alloc forward: the bench workload, then a smaller one", flush=True)
    big = inputs.WORKLOADS["b1_n32768_d64"]
    small = inputs.WORKLOADS["b8_n2048_d64"].with_(batch=2, heads=3, seqlen=1000, seed=61)
    for w in (big, small):
        y, ref = _both(G, w, dev)
        assert torch.equal(y, ref), w.name


def test_noalloc_ragged_and_refusal(G, dev):
    print("no-alloc forward: ragged d=64, then an oversized shape", flush=True)
    w = inputs.WORKLOADS["ragged64_d128"].with_(heads=2, head_dim=64, seed=62)
    inp = inputs.make_inputs(w, lengths=[300, 0, 77, 1024])
    t = inputs.device_tensors(inp, dev)
    args = (t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"])
    kw = dict(eps=inp.eps, cu_seqlens=t["cu_seqlens"], max_seqlen=t["max_seqlen"])
    y = G.forward_noalloc(*args, **kw)
    ref = G.forward(*args, **kw)
    torch.cuda.synchronize()
    assert torch.equal(y, ref)
    big = inputs.WORKLOADS["b1_n32768_d64"].with_(batch=8)
    binp = inputs.make_inputs(big.with_(seqlen=16))  # tensors of a small batch, the shape of a big one
    bt = inputs.device_tensors(binp, dev)
    shape = G.make_shape(bt["q"], bt["conv_w"], binp.eps, None, None)
    shape.seqlen = 1 << 20
    assert G.load_library().gbla_workspace_bytes(shape) > G.NOALLOC_SCRATCH_BYTES
    st = G.load_library().gbla_forward_noalloc(shape, *[G._ptr(x) for x in (
        bt["q"], bt["k"], bt["v"], bt["a"], bt["r"], bt["conv_w"], bt["gamma"])], None,
        G._ptr(bt["q"]), G._stream(None))
    assert st == 4  # GBLA_ERR_WORKSPACE, nothing launched
