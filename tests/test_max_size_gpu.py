"""Parity at the longest head slices each kernel family handles, and just past
them, through inputs that repeat along the sequence.

The streaming kernels (and the matrix-core backward) address one (sequence,
head) slice with 32-bit byte offsets, so they take slices whose fp32 rows
stay below 2^31 bytes; longer slices go to kernels with 64-bit indexing.  At
d = 64 the switch is at n = 2^23 tokens: m = 8191 periods of P = 1024 tokens
is the longest slice of the first family, m = 8192 the shortest of the
second.  No oracle run covers 2^23 tokens, so the test uses a property that
holds at any length (Section 2.1):

Periodic inputs.  q, k, v, a, r repeat with period P, and the last W - 1 rows
of q, k, v in every period are zero.  The conv window of a period's first
rows then sees zeros, as at the sequence start, so the convolved rows repeat
too.  The softmax gates of a periodic a are the period's gates divided by m,
so S and z over m periods equal those of one period, and y over m periods is
y of one period, repeated.

Backward, with a periodic dy.  dS and dz over m periods are m times a
period's sums while g is divided by m, so every per-token gradient equals
that of a two-period sequence (the conv backward, which looks ahead, couples
a period's last rows with the next period's first ones: rows of the first
m - 1 periods match the first period of the two-period run, rows of the last
period its second), and dgamma and the taps' gradients are m / 2 times the
two-period ones.

Tolerances are those of the other parity tests: 2e-2 (allclose form) for the
bf16 forward, 1e-4 * (|ref| + rms(ref)) per gradient tensor.
"""
import dataclasses

import numpy as np
import pytest
import torch

from paper_2606_07317_amd import inputs
from tests.test_parity_gpu import say

pytestmark = pytest.mark.gpu

P = 1024          # period, tokens
D = 64
LIMITS = [8191, 8192]  # periods: the longest streaming slice, the first past it
IDS = ["longest_32bit_slice", "first_64bit_slice"]


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


def period_inputs(seed: int, W: int = 4) -> inputs.Inputs:
    w = inputs.Workload("period", batch=1, heads=1, seqlen=P, head_dim=D, conv_width=W,
                        dtype=inputs.BF16, seed=seed)
    inp = inputs.make_inputs(w)
    q, k, v = (x.copy() for x in (inp.q, inp.k, inp.v))
    for x in (q, k, v):
        x[:, :, P - (W - 1):, :] = 0  # +0.0 in bf16
    return dataclasses.replace(inp, q=q, k=k, v=v)


def repeated(inp: inputs.Inputs, reps: int) -> inputs.Inputs:
    """The same period `reps` times, on the host (for the oracle)."""
    cat = lambda x: np.concatenate([x] * reps, axis=2)
    return dataclasses.replace(inp, workload=inp.workload.with_(seqlen=P * reps), q=cat(inp.q),
                               k=cat(inp.k), v=cat(inp.v), a=cat(inp.a), r=cat(inp.r))


def long_tensors(inp: inputs.Inputs, m: int, dev) -> dict:
    """The period `m` times, built on the device."""
    t = inputs.device_tensors(inp, dev)
    for n in ("q", "k", "v", "r"):
        t[n] = t[n].repeat(1, 1, m, 1)
    t["a"] = t["a"].repeat(1, 1, m)
    return t


def worst_ratio(got: torch.Tensor, ref: torch.Tensor, lim: torch.Tensor) -> float:
    """max |got - ref| / lim over the broadcast shapes, in chunks on the device."""
    worst = 0.0
    for c in range(0, got.shape[0], 512):
        g = got[c:c + 512].double()
        if not torch.isfinite(g).all():
            return float("inf")
        worst = max(worst, float(((g - ref).abs() / lim).max()))
    return worst


def slice_is_streamed(m: int) -> bool:
    return m * P * D * 4 < 2 ** 31


@pytest.mark.parametrize("m", LIMITS, ids=IDS)
def test_forward_at_the_slice_limit(G, dev, orc, m):
    say("forward, %d periods of %d (%s path)" % (m, P, "32-bit" if slice_is_streamed(m) else "64-bit"))
    inp = period_inputs(seed=50)
    ref = torch.from_numpy(orc.forward_inputs(inp)["y"].reshape(P, D)).to(dev)
    t = long_tensors(inp, m, dev)
    y = G.forward(t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"], eps=inp.eps)
    torch.cuda.synchronize()
    tol = 2e-2
    r = worst_ratio(y.view(m, P, D), ref, tol + tol * ref.abs())
    say("  y  worst err/tol %.3f" % r)
    assert r <= 1.0


@pytest.mark.parametrize("m", LIMITS, ids=IDS)
def test_backward_at_the_slice_limit(G, dev, m):
    from oracle import gbla_backward
    say("backward, %d periods of %d (%s path)" % (m, P, "32-bit" if slice_is_streamed(m) else "64-bit"))
    inp = period_inputs(seed=51)
    dy = inputs.make_cotangent(inp)
    two = repeated(inp, 2)
    ref = gbla_backward.backward_inputs(two, np.concatenate([dy, dy], axis=2))
    t = long_tensors(inp, m, dev)
    dyl = torch.from_numpy(dy).to(dev).repeat(1, 1, m, 1)
    g = G.backward(t["q"], t["k"], t["v"], t["a"], t["r"], t["conv_w"], t["gamma"], dyl, eps=inp.eps)
    torch.cuda.synchronize()
    tol = 1e-4
    for name in ("dq", "dk", "dv", "dr", "da"):
        rr = torch.from_numpy(ref[name].reshape(2, P, -1)).to(dev)
        lim = tol * (rr.abs() + rr.pow(2).mean().sqrt())
        got = g[name].view(m, P, -1)
        r_in = worst_ratio(got[:m - 1], rr[0], lim[0])
        r_last = worst_ratio(got[m - 1:], rr[1], lim[1])
        say("  %-7s worst err/tol %.3f (periods 0..m-2), %.3f (last)" % (name, r_in, r_last))
        assert r_in <= 1.0 and r_last <= 1.0, name
    for name in ("dgamma", "dconv_w"):
        rr = ref[name] * (m / 2.0)
        got = g[name].cpu().numpy().astype(np.float64)
        lim = tol * (np.abs(rr) + np.sqrt(np.mean(rr ** 2)))
        r = float((np.abs(got - rr) / lim).max())
        say("  %-7s worst err/tol %.3f" % (name, r))
        assert np.isfinite(got).all() and r <= 1.0, name
