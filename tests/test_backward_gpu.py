"""Parity of the HIP backward pass (gbla_backward, through the C ABI) with the
fp64 backward oracle, which is itself pinned by finite differences of the
forward oracle.

Tolerance (allclose form, per gradient tensor): |x - x_ref| <= tol * (|x_ref| +
rms(x_ref)) with tol = 1e-4 for both input dtypes.  The backward computes in
fp32 from the exact values of the inputs (bf16 activations widen exactly;
the state is recomputed with fp32 products), so both dtypes carry only fp32
rounding: sums over up to a few thousand tokens, n * 2^-24 ~ 2e-4 in the
worst case, observed near 1e-6.  The rms term is the scale of the tensor:
every gradient is a sum of signed terms (over tokens for dS, dz, dgamma and
the taps; over channels for dQh, t and dg), so an element that cancels to
near zero carries the rounding of its terms, not of its value.

One-token sequences are degenerate: o = vt exactly (S = g phi(kt) vt^T and
z = g phi(kt) with g = 1), so L does not depend on q, k or a, and dq, dk, da
and the q, k taps vanish; the kernel leaves the rounding of the cancelled
terms there.  Those terms are products of the same factors (Qh, P, dnum, vt)
as dv = g dS^T P, so the residue is held to 2^-16 * rms(dv): a few hundred
fp32 ulps of that scale (observed below 2e-6 of it).
"""
import numpy as np
import pytest
import torch

from paper_2606_07317_amd import inputs
from tests.test_parity_gpu import RAGGED_CASES, SMALL_CASES, say

pytestmark = pytest.mark.gpu

TOL = {inputs.F32: 1e-4, inputs.BF16: 1e-4}
NAMES = ("dq", "dk", "dv", "da", "dr", "dconv_w", "dgamma")


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


def close_scaled(got, ref, tol, what):
    got = np.asarray(got, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.isfinite(got).all(), what + ": non-finite output"
    scale = np.sqrt(np.mean(ref * ref)) if ref.size else 0.0
    err = np.abs(got - ref)
    lim = tol * (np.abs(ref) + scale) + 1e-30
    say("  %-10s max abs %.3e  rms(ref) %.3e  worst err/tol %.3f" %
        (what, err.max() if err.size else 0.0, scale, (err / lim).max() if err.size else 0.0))
    bad = err > lim
    assert not bad.any(), "%s: %d of %d outside tol %g (max abs err %.3e)" % (
        what, int(bad.sum()), bad.size, tol, err.max())


def run_backward(G, inp, dy, dev):
    t = inputs.device_tensors(inp, dev)
    g = G.backward(t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"],
                   torch.from_numpy(dy).to(dev), eps=inp.eps, cu_seqlens=t["cu_seqlens"],
                   max_seqlen=t["max_seqlen"])
    torch.cuda.synchronize()
    return {n: g[n].cpu().numpy() for n in NAMES}


CASES = [(k, w, None) for k, w in SMALL_CASES.items()]
CASES += [(k, w, l) for k, (w, l) in RAGGED_CASES.items()]


@pytest.mark.parametrize("name,w,lens", CASES, ids=[c[0] for c in CASES])
def test_backward_parity(G, dev, name, w, lens):
    from oracle import gbla_backward
    say("backward", name)
    inp = inputs.make_inputs(w, lengths=lens)
    dy = inputs.make_cotangent(inp)
    got = run_backward(G, inp, dy, dev)
    ref = gbla_backward.backward_inputs(inp, dy)
    if lens is None and w.seqlen == 1:
        # L depends on v, r, gamma and the v taps only
        for n, val in (("dq", got["dq"]), ("dk", got["dk"]), ("da", got["da"]),
                       ("dconv_w[q,k]", got["dconv_w"][:2])):
            bound = 2.0 ** -16 * float(np.sqrt(np.mean(ref["dv"] ** 2)))
            say("  %-10s max abs %.3e  (zero; bound %.3e)" % (n, np.abs(val).max(), bound))
            assert np.abs(val).max() <= bound, n
        for n in ("dv", "dr", "dgamma"):
            close_scaled(got[n], ref[n], TOL[w.dtype], n)
        close_scaled(got["dconv_w"][2], ref["dconv_w"][2], TOL[w.dtype], "dconv_w[v]")
        return
    for n in NAMES:
        close_scaled(got[n], ref[n], TOL[w.dtype], n)


def test_backward_is_deterministic(G, dev):
    """Every reduction runs in an order fixed by the shape: two calls give
    the same bits."""
    w, lens = RAGGED_CASES["ragged_d64_long"]
    inp = inputs.make_inputs(w, lengths=lens)
    dy = inputs.make_cotangent(inp)
    a = run_backward(G, inp, dy, dev)
    b = run_backward(G, inp, dy, dev)
    for n in NAMES:
        assert np.array_equal(a[n], b[n]), n


@pytest.mark.parametrize("name", ["b8_n2048_d64", "b1_n32768_d64"])
def test_backward_parity_full_size(G, dev, name):
    """The benchmark workloads at full size, every element, in the launch
    configuration bench.py --pass backward times."""
    from oracle import gbla_backward
    say("backward full size", name)
    inp = inputs.make_inputs(name)
    dy = inputs.make_cotangent(inp)
    got = run_backward(G, inp, dy, dev)
    ref = gbla_backward.backward_inputs(inp, dy)
    for n in NAMES:
        close_scaled(got[n], ref[n], TOL[inp.workload.dtype], n)


# Ablation switches (the paper's ablation table): each alone and all three
# (BLA, Eq. (1)), through both matrix-core arrangements (d = 32 / 64 with dS
# summed in the query pass, d = 128 with its separate dS pass), dense and
# ragged.
SWITCH_CASES = ["bf16_d64_n1000", "f32_d64_n1000", "ragged_d128_mixed", "bf16_d32_n3001_W2"]


@pytest.mark.parametrize("sw", ["no_gate", "no_conv", "no_norm", "bla"])
@pytest.mark.parametrize("name", SWITCH_CASES)
def test_backward_switch_parity(G, dev, name, sw):
    from oracle import gbla_backward
    say("backward switch", sw, name)
    w, lens = (SMALL_CASES[name], None) if name in SMALL_CASES else RAGGED_CASES[name]
    flags = {"no_gate": G.NO_GATE, "no_conv": G.NO_CONV, "no_norm": G.NO_NORM, "bla": G.BLA}[sw]
    gate, conv, norm = not flags & G.NO_GATE, not flags & G.NO_CONV, not flags & G.NO_NORM
    inp = inputs.make_inputs(w, lengths=lens)
    dy = inputs.make_cotangent(inp)
    t = inputs.device_tensors(inp, dev)
    # inputs a switch removes are passed as None: the library must not read
    # them, nor write their gradients
    g = G.backward(t["q"], t["k"], t["v"], t["a"] if gate else None, t["r"] if norm else None,
                   t["conv_w"] if conv else None, t["gamma"] if norm else None,
                   torch.from_numpy(dy).to(dev), eps=inp.eps, cu_seqlens=t["cu_seqlens"],
                   max_seqlen=t["max_seqlen"], flags=flags)
    torch.cuda.synchronize()
    ref = gbla_backward.backward_inputs(inp, dy, gate=gate, conv=conv, norm=norm)
    kept = ["dq", "dk", "dv"] + (["da"] if gate else []) + (["dconv_w"] if conv else [])
    kept += ["dr", "dgamma"] if norm else []
    assert sorted(g) == sorted(kept)
    for n in kept:
        close_scaled(g[n].cpu().numpy(), ref[n], TOL[w.dtype], n)


def test_backward_parity_ragged_full_size_sampled(G, dev):
    """The ragged d = 128 workload at full size (64 sequences, T = 177,929)
    through the launch configuration bench.py uses: per-token gradients of
    eight sampled sequences (the longest, the shortest and six seeded others)
    against the oracle run on those sequences alone.  Every per-token
    gradient of a sequence depends on that sequence only; dgamma and the tap
    gradients, summed over the batch, are covered by the smaller cases."""
    import dataclasses
    from oracle import gbla_backward
    say("backward full size, ragged64_d128 (sampled sequences)")
    inp = inputs.make_inputs("ragged64_d128")
    dy = inputs.make_cotangent(inp)
    got = run_backward(G, inp, dy, dev)
    lens = inp.lengths()
    cu = inp.cu_seqlens.astype(np.int64)
    rng = np.random.default_rng(7)
    pick = sorted(set([int(np.argmax(lens)), int(np.argmin(lens))] +
                      [int(x) for x in rng.choice(len(lens), 6, replace=False)]))
    rows = np.concatenate([np.arange(cu[s], cu[s + 1]) for s in pick])
    sub_cu = np.concatenate([[0], np.cumsum(lens[pick])]).astype(np.int32)
    sub = dataclasses.replace(inp, workload=inp.workload.with_(batch=len(pick)), q=inp.q[:, rows],
                              k=inp.k[:, rows], v=inp.v[:, rows], a=inp.a[:, rows], r=inp.r[:, rows],
                              cu_seqlens=sub_cu)
    ref = gbla_backward.backward_inputs(sub, dy[:, rows])
    say("  sequences %s, %d tokens" % (pick, len(rows)))
    for n in ("dq", "dk", "dv", "da", "dr"):
        close_scaled(got[n][:, rows], ref[n], TOL[inp.workload.dtype], n)
