"""Parity of the HIP path (through the C ABI) with the fp64 oracle.

Tolerance (elementwise, allclose form): |x - x_ref| <= tol + tol * |x_ref| with
tol = 1e-5 for fp32 inputs and 2e-2 for bf16 inputs (fp32 accumulation).
The state S, z of the bf16 path is additionally held to an error bound
derived from its arithmetic: each product g_j phi(kt_j)[c] vt_j[e] carries at
most two bf16 roundings (relative 2^-8 together), so
|S - S_ref| <= 2^-7 * sum_j g_j phi(kt_j)[c] |vt_j[e]| + 1e-6 (2x margin).
"""
import numpy as np
import pytest
import torch

from paper_2606_07317_amd import inputs

pytestmark = pytest.mark.gpu

TOL = {inputs.F32: 1e-5, inputs.BF16: 2e-2}


def say(*a):
    print(*a, flush=True)


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


def close(got, ref, tol, what):
    got = np.asarray(got, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.isfinite(got).all(), what + ": non-finite output"
    err = np.abs(got - ref)
    bad = err > tol + tol * np.abs(ref)
    rel = err / np.maximum(np.abs(ref), 1e-6)
    say("  %-28s max abs %.3e  max rel %.3e  worst err/tol %.3f" %
        (what, err.max(), rel.max(), (err / (tol + tol * np.abs(ref))).max()))
    assert not bad.any(), "%s: %d of %d outside tol %g (max abs err %.3e)" % (
        what, int(bad.sum()), bad.size, tol, err.max())


def run_forward(G, inp, dev, **kw):
    t = inputs.device_tensors(inp, dev)
    y = G.forward(t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"], eps=inp.eps,
                  cu_seqlens=t["cu_seqlens"], max_seqlen=t["max_seqlen"], **kw)
    torch.cuda.synchronize()
    return y.cpu().numpy()


def small(name, **kw):
    return inputs.WORKLOADS[name].with_(**kw)


# Cases the oracle finishes in well under a second that still span several
# chunks and readout tiles and end in ragged tails.
SMALL_CASES = {
    "tiny_f32": inputs.WORKLOADS["tiny_f32"],
    "f32_d64_n1000": small("tiny_f32", batch=2, heads=3, seqlen=1000, head_dim=64, seed=21),
    "f32_d128_n700_W3": small("tiny_f32", batch=1, heads=2, seqlen=700, head_dim=128, conv_width=3, seed=22),
    "bf16_d64_n1000": small("b8_n2048_d64", batch=2, heads=3, seqlen=1000, seed=23),
    "bf16_d32_n3001_W2": small("b8_n2048_d64", batch=1, heads=2, seqlen=3001, head_dim=32, conv_width=2, seed=24),
    "bf16_d128_n777_W1": small("b8_n2048_d64", batch=2, heads=2, seqlen=777, head_dim=128, conv_width=1, seed=25),
    "bf16_d128_n3000_W4": small("b8_n2048_d64", batch=1, heads=2, seqlen=3000, head_dim=128, seed=28),
    "bf16_d64_n1": small("b8_n2048_d64", batch=3, heads=2, seqlen=1, seed=26),
    "bf16_d64_n5": small("b8_n2048_d64", batch=2, heads=2, seqlen=5, seed=27),
}
RAGGED_CASES = {
    "ragged_d128_mixed": (small("ragged64_d128", heads=2, seed=31), [5, 0, 300, 1, 77, 2049, 3]),
    "ragged_d64_long": (small("ragged64_d128", heads=3, head_dim=64, seed=32), [4100, 17, 0, 0, 999]),
    # 256-token chunks at this size: whole-chunk sequences (no partial unit),
    # partial units that tie on their number of 32-token steps, an empty and a
    # one-token sequence (the d = 128 state pass takes units longest first)
    "ragged_d128_units": (small("ragged64_d128", heads=2, seed=34),
                          [512, 256, 1, 768, 300, 0, 256, 33, 32, 1024, 255]),
    "ragged_f32_d32": (inputs.Workload("rf32", batch=3, heads=2, seqlen=0, head_dim=32, conv_width=4,
                                       dtype=inputs.F32, seed=33, ragged=True), [31, 2, 600]),
}


def all_small():
    cases = [(k, w, None) for k, w in SMALL_CASES.items()]
    cases += [(k, w, l) for k, (w, l) in RAGGED_CASES.items()]
    return cases


IDS = [c[0] for c in all_small()]


@pytest.mark.parametrize("name,w,lens", all_small(), ids=IDS)
def test_conv1d_parity(G, dev, orc, name, w, lens):
    say("conv1d", name)
    inp = inputs.make_inputs(w, lengths=lens)
    t = inputs.device_tensors(inp, dev)
    qt, kt, vt = G.conv1d(t["q"], t["k"], t["v"], t["conv_w"], cu_seqlens=t["cu_seqlens"],
                          max_seqlen=t["max_seqlen"])
    torch.cuda.synchronize()
    ref = orc.forward_inputs(inp, want=("qt", "kt", "vt"))
    for got, nm in ((qt, "qt"), (kt, "kt"), (vt, "vt")):
        close(got.cpu().numpy(), ref[nm], 1e-5, nm)


@pytest.mark.parametrize("name,w,lens", all_small(), ids=IDS)
def test_state_parity(G, dev, orc, name, w, lens):
    say("state", name)
    inp = inputs.make_inputs(w, lengths=lens)
    t = inputs.device_tensors(inp, dev)
    S, z = G.state(t["k"], t["v"], t["a"], t["conv_w"], cu_seqlens=t["cu_seqlens"],
                   max_seqlen=t["max_seqlen"])
    torch.cuda.synchronize()
    ref = orc.forward_inputs(inp, want=("S", "z", "kt", "vt", "g"))
    tol = TOL[w.dtype]
    S_got, z_got = S.cpu().numpy(), z.cpu().numpy()
    close(S_got, ref["S"], tol, "S")
    close(z_got, ref["z"], tol, "z")
    if w.dtype == inputs.BF16:
        # arithmetic bound per element (see module docstring)
        kt, vt, g = ref["kt"], ref["vt"], ref["g"]
        ph = np.where(kt > 0, kt + 1, np.exp(np.minimum(kt, 0)))
        if inp.cu_seqlens is None:
            B = np.einsum("shj,shjc,shje->shce", g, ph, np.abs(vt))
        else:
            cu = inp.cu_seqlens
            B = np.stack([np.einsum("hj,hjc,hje->hce", g[:, a:b], ph[:, a:b], np.abs(vt[:, a:b]))
                          for a, b in zip(cu[:-1], cu[1:])])
        err = np.abs(S_got - ref["S"])
        say("  S err / bound: %.3f" % (err / (2 ** -7 * B + 1e-6)).max())
        assert (err <= 2 ** -7 * B + 1e-6).all()
        np.testing.assert_allclose(z_got, ref["z"], rtol=1e-4, atol=1e-7)


@pytest.mark.parametrize("name,w,lens", all_small(), ids=IDS)
def test_forward_parity(G, dev, orc, name, w, lens):
    say("forward", name)
    inp = inputs.make_inputs(w, lengths=lens)
    y = run_forward(G, inp, dev)
    ref = orc.forward_inputs(inp)["y"]
    close(y, ref, TOL[w.dtype], "y")


@pytest.mark.parametrize("name", ["b8_n2048_d64", "b2_n8192_d64", "b1_n32768_d64"])
def test_forward_parity_full_workloads(G, dev, orc, name):
    say("forward full", name)
    inp = inputs.make_inputs(name)
    y = run_forward(G, inp, dev)
    ref = orc.forward_inputs(inp)["y"]
    close(y, ref, TOL[inp.workload.dtype], "y " + name)


def test_forward_parity_ragged64_d128(G, dev, orc):
    say("forward full ragged64_d128")
    inp = inputs.make_inputs("ragged64_d128")
    say("  T =", inp.tokens)
    y = run_forward(G, inp, dev)
    ref = orc.forward_inputs(inp)["y"]
    close(y, ref, TOL[inp.workload.dtype], "y ragged64_d128")


# Ablation switches (the paper's ablation table): each alone and all three
# (BLA, Eq. (1)), on the bf16 and fp32 paths, d = 32 / 64 / 128, dense and ragged.
SWITCH_CASES = ["bf16_d64_n1000", "f32_d64_n1000", "ragged_d128_mixed", "bf16_d32_n3001_W2"]


def _case(name):
    if name in SMALL_CASES:
        return SMALL_CASES[name], None
    return RAGGED_CASES[name]


def _switch_flags(G, sw):
    return {"no_gate": G.NO_GATE, "no_conv": G.NO_CONV, "no_norm": G.NO_NORM, "bla": G.BLA}[sw]


@pytest.mark.parametrize("sw", ["no_gate", "no_conv", "no_norm", "bla"])
@pytest.mark.parametrize("name", SWITCH_CASES)
def test_forward_switch_parity(G, dev, orc, name, sw):
    say("forward switch", sw, name)
    w, lens = _case(name)
    flags = _switch_flags(G, sw)
    inp = inputs.make_inputs(w, lengths=lens)
    t = inputs.device_tensors(inp, dev)
    # inputs a switch removes are passed as None: the library must not read them
    a = None if flags & G.NO_GATE else t["a"]
    cw = None if flags & G.NO_CONV else t["conv_w"]
    r = None if flags & G.NO_NORM else t["r"]
    gm = None if flags & G.NO_NORM else t["gamma"]
    y = G.forward(t["q"], t["k"], t["v"], a, r, cw, gm, eps=inp.eps, cu_seqlens=t["cu_seqlens"],
                  max_seqlen=t["max_seqlen"], flags=flags)
    torch.cuda.synchronize()
    ref = orc.forward_inputs(inp, want=("y",), gate=not flags & G.NO_GATE,
                             conv=not flags & G.NO_CONV, norm=not flags & G.NO_NORM)["y"]
    close(y.cpu().numpy(), ref, TOL[w.dtype], "y " + sw)


@pytest.mark.parametrize("name", ["bf16_d64_n1000", "ragged_d128_mixed"])
def test_state_and_conv_switches(G, dev, orc, name):
    say("state/conv switches", name)
    w, lens = _case(name)
    inp = inputs.make_inputs(w, lengths=lens)
    t = inputs.device_tensors(inp, dev)
    # uniform gates: S and z carry g_j = 1/n
    S, z = G.state(t["k"], t["v"], None, t["conv_w"], cu_seqlens=t["cu_seqlens"],
                   max_seqlen=t["max_seqlen"], flags=G.NO_GATE)
    torch.cuda.synchronize()
    ref = orc.forward_inputs(inp, want=("S", "z"), gate=False)
    close(S.cpu().numpy(), ref["S"], TOL[w.dtype], "S no_gate")
    close(z.cpu().numpy(), ref["z"], TOL[w.dtype], "z no_gate")
    # identity conv returns the inputs exactly
    qt, kt, vt = G.conv1d(t["q"], t["k"], t["v"], None, cu_seqlens=t["cu_seqlens"],
                          max_seqlen=t["max_seqlen"], flags=G.NO_CONV)
    torch.cuda.synchronize()
    for got, x in ((qt, t["q"]), (kt, t["k"]), (vt, t["v"])):
        assert torch.equal(got, x.float()), "identity conv must return its input"


def test_state_then_readout_equals_forward(G, dev):
    say("state+readout == forward")
    inp = inputs.make_inputs(SMALL_CASES["bf16_d64_n1000"])
    t = inputs.device_tensors(inp, dev)
    y = G.forward(t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"], eps=inp.eps)
    shape = G.make_shape(t["q"], t["conv_w"], inp.eps, None, None)
    ws = G.alloc_workspace(shape, dev)
    G.state(t["k"], t["v"], t["a"], t["conv_w"], workspace=ws)
    y2 = G.readout(t["q"], t["r"], t["conv_w"], t["gamma"], ws, eps=inp.eps)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)


@pytest.mark.parametrize("name", ["bf16_d64_n1000", "f32_d64_n1000"])
def test_timed_readout_equals_readout(G, dev, name):
    """gbla_readout_timed gives gbla_readout's bits, and the events the launch
    records bracket the kernel alone: a positive time within that of events
    recorded around the call."""
    say("timed readout, " + name)
    inp = inputs.make_inputs(SMALL_CASES[name])
    t = inputs.device_tensors(inp, dev)
    shape = G.make_shape(t["q"], t["conv_w"], inp.eps, None, None)
    ws = G.alloc_workspace(shape, dev)
    G.state(t["k"], t["v"], t["a"], t["conv_w"], workspace=ws)
    y = G.readout(t["q"], t["r"], t["conv_w"], t["gamma"], ws, eps=inp.eps)
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    for e in ev[:2]:
        e.record(stream)
    ev[2].record(stream)
    y2 = G.readout(t["q"], t["r"], t["conv_w"], t["gamma"], ws, eps=inp.eps,
                   kernel_events=(ev[0], ev[1]))
    ev[3].record(stream)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    kernel_ms, call_ms = ev[0].elapsed_time(ev[1]), ev[2].elapsed_time(ev[3])
    say("  kernel %.2f us, call %.2f us" % (1e3 * kernel_ms, 1e3 * call_ms))
    assert 0.0 < kernel_ms <= call_ms


def test_deterministic(G, dev):
    say("determinism")
    inp = inputs.make_inputs(small("b8_n2048_d64", batch=2, heads=4, seqlen=5000, seed=40))
    t = inputs.device_tensors(inp, dev)
    args = (t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"])
    y1 = G.forward(*args, eps=inp.eps)
    y2 = G.forward(*args, eps=inp.eps)
    torch.cuda.synchronize()
    assert torch.equal(y1, y2)


def test_forward_under_graph_capture(G, dev):
    """A captured forward replays correctly (its launches record no memset
    and need no cleared workspace): every replay, with eager work and
    synchronisations between them, equals the eager result."""
    say("graph capture")
    inp = inputs.make_inputs(SMALL_CASES["bf16_d64_n1000"])
    t = inputs.device_tensors(inp, dev)
    args = (t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"])
    shape = G.make_shape(t["q"], t["conv_w"], inp.eps, None, None)
    ws = G.alloc_workspace(shape, dev)
    eager = G.forward(*args, eps=inp.eps, workspace=ws).clone()
    out = torch.empty_like(eager)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        G.forward(*args, eps=inp.eps, workspace=ws, out=out)  # warm up on the side stream
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        G.forward(*args, eps=inp.eps, workspace=ws, out=out)
    for i in range(3):
        out.fill_(float("nan"))
        other = G.forward(*args, eps=inp.eps, workspace=ws)  # eager work in between
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(out, eager), "replay %d" % i
        assert torch.equal(other, eager)


def test_output_guard_canaries(G, dev):
    say("guard canaries")
    inp = inputs.make_inputs(small("b8_n2048_d64", batch=2, heads=2, seqlen=333, seed=41))
    t = inputs.device_tensors(inp, dev)
    n = inp.q.size
    pad = 4096
    buf = torch.full((n + 2 * pad,), 12345.0, dtype=torch.float32, device=dev)
    out = buf[pad:pad + n].view(inp.q.shape)
    assert out.data_ptr() % 16 == 0
    G.forward(t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"], eps=inp.eps, out=out)
    torch.cuda.synchronize()
    b = buf.cpu()
    assert torch.all(b[:pad] == 12345.0) and torch.all(b[pad + n:] == 12345.0)
    assert torch.isfinite(out).all()


def test_workspace_reuse_across_shapes(G, dev, orc):
    say("workspace reuse")
    big = inputs.make_inputs(small("b8_n2048_d64", batch=2, heads=2, seqlen=3000, seed=42))
    little = inputs.make_inputs(small("b8_n2048_d64", batch=1, heads=2, seqlen=100, seed=43))
    tb = inputs.device_tensors(big, dev)
    shape = G.make_shape(tb["q"], tb["conv_w"], big.eps, None, None)
    ws = G.alloc_workspace(shape, dev)
    for inp in (big, little, big):
        t = inputs.device_tensors(inp, dev)
        y = G.forward(t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"], eps=inp.eps,
                      workspace=ws)
        torch.cuda.synchronize()
        close(y.cpu().numpy(), orc.forward_inputs(inp)["y"], 2e-2, "y reuse")


def test_gate_shift_invariance_fp32(G, dev):
    say("gate shift invariance")
    inp = inputs.make_inputs(small("tiny_f32", seqlen=700, seed=44))
    t = inputs.device_tensors(inp, dev)
    y1 = G.forward(t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"], eps=inp.eps)
    y2 = G.forward(t["q"], t["k"], t["v"], t["a"] + 3.0, t["r"], t["conv_w"], t["gamma"], eps=inp.eps)
    torch.cuda.synchronize()
    np.testing.assert_allclose(y2.cpu().numpy(), y1.cpu().numpy(), rtol=1e-5, atol=1e-5)


def test_timed_forward_equals_forward(G, dev):
    """gbla_forward_timed gives gbla_forward's bits, and its events bracket
    the pass's kernels (a positive time no longer than events around the
    call)."""
    say("timed forward")
    inp = inputs.make_inputs(SMALL_CASES["bf16_d64_n1000"])
    t = inputs.device_tensors(inp, dev)
    args = (t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"])
    ref = G.forward(*args, eps=inp.eps)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    st = torch.cuda.current_stream()
    for e in ev:
        e.record(st)  # the HIP events exist from here on
    ev[2].record(st)
    y = G.forward(*args, eps=inp.eps, kernel_events=(ev[0], ev[1]))
    ev[3].record(st)
    torch.cuda.synchronize()
    assert torch.equal(y, ref)
    kernel_ms, call_ms = ev[0].elapsed_time(ev[1]), ev[2].elapsed_time(ev[3])
    say("  kernels %.2f us, call %.2f us" % (1e3 * kernel_ms, 1e3 * call_ms))
    assert 0.0 < kernel_ms <= call_ms


def test_binding_rejects_bad_buffers(G, dev):
    """The binding checks caller buffers before any pointer reaches the
    library: an output of the wrong shape, dtype or device, a workspace of
    the wrong dtype, on the host, or too small."""
    say("binding buffer checks")
    inp = inputs.make_inputs(SMALL_CASES["bf16_d64_n5"])
    t = inputs.device_tensors(inp, dev)
    args = (t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"])
    shape = G.make_shape(t["q"], t["conv_w"], inp.eps, None, None)
    need = G.workspace_bytes(shape)
    bad_out = [torch.empty(t["q"].shape[:-1] + (t["q"].shape[-1] - 1,), device=dev),
               torch.empty(t["q"].shape, dtype=torch.bfloat16, device=dev),
               torch.empty(t["q"].shape)]
    for out in bad_out:
        with pytest.raises((ValueError, TypeError)):
            G.forward(*args, eps=inp.eps, out=out)
    bad_ws = [torch.empty(need, dtype=torch.float32, device=dev),
              torch.empty(need, dtype=torch.uint8),
              torch.empty(need - 1, dtype=torch.uint8, device=dev)]
    for ws in bad_ws:
        with pytest.raises((ValueError, TypeError)):
            G.forward(*args, eps=inp.eps, workspace=ws)
        with pytest.raises((ValueError, TypeError)):
            G.state(t["k"], t["v"], t["a"], t["conv_w"], workspace=ws)
    good = G.forward(*args, eps=inp.eps)
    torch.cuda.synchronize()
    assert torch.isfinite(good).all()


@pytest.mark.parametrize("d", [32, 64, 128])
def test_stream_ceiling_moves_every_byte(G, dev, d):
    """gbla_stream_ceiling reads every 16-byte piece of q, k, v, r and each
    token's logit once and writes y: its output is the XOR of the four
    inputs' bits per 16-byte piece, plus the logit's bits on the token's
    first 32-bit word, written twice per piece."""
    say("stream ceiling d=%d" % d)
    gen = torch.Generator().manual_seed(50 + d)
    shp = (2, 3, 37, d)
    ts = [torch.randint(-2**15, 2**15, shp, generator=gen, dtype=torch.int16) for _ in range(4)]
    a = torch.randint(0, 2**15, shp[:-1], generator=gen, dtype=torch.int16)
    dev_t = [t.view(torch.bfloat16).to(dev) for t in ts]
    y = G.stream_ceiling(dev_t[0], dev_t[1], dev_t[2], a.view(torch.bfloat16).to(dev), dev_t[3])
    torch.cuda.synchronize()
    words = [t.numpy().view(np.uint32).reshape(-1, 4) for t in ts]  # 16-byte pieces
    x = words[0] ^ words[1] ^ words[2] ^ words[3]
    per_token = d // 8
    first = np.arange(x.shape[0]) % per_token == 0
    x = x.copy()
    x[first, 0] += a.numpy().view(np.uint16).reshape(-1).astype(np.uint32)
    want = np.repeat(x, 2, axis=0).reshape(-1)
    got = y.cpu().numpy().view(np.uint32).reshape(-1)
    assert np.array_equal(got, want)
