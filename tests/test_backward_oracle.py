"""Pins of the fp64 backward oracle (oracle/gbla_backward.py).

Every gradient is checked against central finite differences of the C forward
oracle (a separate implementation of the forward pass) on the scalar
L = sum(y * dy): a dropped term, a wrong sign or a transposed operand in any
step of the chain rule fails here.  No GPU is needed.
"""
import numpy as np
import pytest

from oracle import gbla_backward


def problem(seed, nseq=2, H=2, n=9, d=5, W=4, ragged=None):
    rng = np.random.default_rng(seed)
    if ragged is None:
        shp = (nseq, H, n, d)
        cu = None
        rows = n
    else:
        cu = np.concatenate([[0], np.cumsum(ragged)]).astype(np.int32)
        nseq, rows = len(ragged), int(cu[-1])
        shp = (H, rows, d)
    p = {x: rng.standard_normal(shp) for x in ("q", "k", "v", "r")}
    p["a"] = rng.standard_normal(shp[:-1])
    p["conv_w"] = 0.5 * rng.standard_normal((3, H, d, W))
    p["gamma"] = 1.0 + 0.1 * rng.standard_normal((H, d))
    dy = rng.standard_normal(shp)
    meta = dict(nseq=nseq, heads=H, rows=rows, d=d, W=W, dtype="f64", eps=1e-3, cu_seqlens=cu)
    return p, dy, meta


def loss(orc, p, dy, meta):
    y = orc.forward(p["q"], p["k"], p["v"], p["a"], p["r"], p["conv_w"], p["gamma"],
                    want=("y",), **meta)["y"]
    return float(np.sum(y * dy))


GRAD_OF = {"q": "dq", "k": "dk", "v": "dv", "a": "da", "r": "dr", "conv_w": "dconv_w",
           "gamma": "dgamma"}


def check_fd(orc, p, dy, meta, samples=6, seed=0, h=1e-5):
    g = gbla_backward.backward(p["q"], p["k"], p["v"], p["a"], p["r"], p["conv_w"], p["gamma"],
                               dy, **meta)
    rng = np.random.default_rng(seed)
    for name, gname in GRAD_OF.items():
        x = p[name]
        assert g[gname].shape == x.shape, (gname, g[gname].shape, x.shape)
        for flat in rng.choice(x.size, size=min(samples, x.size), replace=False):
            idx = np.unravel_index(flat, x.shape)
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            fd = (loss(orc, dict(p, **{name: xp}), dy, meta) -
                  loss(orc, dict(p, **{name: xm}), dy, meta)) / (2 * h)
            got = g[gname][idx]
            assert abs(got - fd) <= 1e-6 + 1e-5 * abs(fd), (gname, idx, got, fd)


@pytest.mark.parametrize("W", [1, 2, 4])
def test_backward_matches_finite_differences_dense(orc, W):
    p, dy, meta = problem(10 + W, W=W)
    check_fd(orc, p, dy, meta, seed=W)


def test_backward_matches_finite_differences_ragged(orc):
    # an empty sequence, a one-token sequence and sequences shorter than W
    p, dy, meta = problem(21, H=2, d=4, W=4, ragged=[5, 0, 1, 3, 8])
    check_fd(orc, p, dy, meta, samples=8, seed=3)


def test_backward_of_linear_pieces(orc):
    """Closed forms: L is linear in gamma, so dgamma is exactly
    sum_i dy oh silu(r) from the forward oracle's oh; and the softmax gradient
    sums to zero over each sequence (logits are shift invariant)."""
    p, dy, meta = problem(31)
    g = gbla_backward.backward(p["q"], p["k"], p["v"], p["a"], p["r"], p["conv_w"], p["gamma"],
                               dy, **meta)
    oh = orc.forward(p["q"], p["k"], p["v"], p["a"], p["r"], p["conv_w"], p["gamma"],
                     want=("oh",), **meta)["oh"]
    silu = p["r"] / (1.0 + np.exp(-p["r"]))
    np.testing.assert_allclose(g["dgamma"], np.einsum("shie->he", dy * oh * silu), rtol=1e-12)
    np.testing.assert_allclose(g["da"].sum(axis=-1), 0.0, atol=1e-12)


def test_gate_gradient_has_no_centering_term(orc):
    """o is invariant to scaling all gates of a sequence (the normaliser cancels
    between numerator and denominator), so by Euler's theorem
    sum_j g_j dL/dg_j = 0 and the softmax Jacobian's centering term vanishes:
    da_j = g_j dL/dg_j.  The oracle with that term removed must agree with the
    full one to rounding on random data."""
    import types
    src = open(gbla_backward.__file__).read()
    old = "da = g * (dg - np.sum(g * dg))"
    assert src.count(old) == 1
    mod = types.ModuleType("gbla_backward_no_center")
    exec(compile(src.replace(old, "da = g * dg"), gbla_backward.__file__, "exec"), mod.__dict__)
    for seed in (51, 52):
        p, dy, meta = problem(seed, nseq=3)
        args = (p["q"], p["k"], p["v"], p["a"], p["r"], p["conv_w"], p["gamma"], dy)
        full = gbla_backward.backward(*args, **meta)["da"]
        nocenter = mod.backward(*args, **meta)["da"]
        np.testing.assert_allclose(nocenter, full, rtol=1e-9, atol=1e-14)


def test_rmsnorm_gradient_along_o_is_eps_sized():
    """do = rs doh - rs^3/d (doh . o) o satisfies do . o = eps rs^3 (doh . o)
    exactly (rs^-2 = mean(o^2) + eps): the kernels use this closed form for
    dden = -(do . o) / den instead of summing do . o."""
    rng = np.random.default_rng(5)
    for eps in (0.0, 1e-6, 1e-3, 0.5):
        o = rng.standard_normal((50, 16)) * rng.uniform(0.01, 10, (50, 1))
        doh = rng.standard_normal((50, 16))
        d = o.shape[1]
        rs = 1.0 / np.sqrt(np.mean(o * o, axis=1) + eps)
        s1 = np.sum(doh * o, axis=1)
        do = rs[:, None] * doh - (rs ** 3 / d * s1)[:, None] * o
        np.testing.assert_allclose(np.sum(do * o, axis=1), eps * rs ** 3 * s1,
                                   rtol=1e-9, atol=1e-12 * np.abs(rs * s1).max())


def test_backward_without_the_gated_norm_matches_finite_differences(orc):
    """norm=False is the layer with y = o (the ablation without gated RMSNorm):
    its gradients against finite differences of the forward oracle's o."""
    p, dy, meta = problem(61, W=3)
    g = gbla_backward.backward(p["q"], p["k"], p["v"], p["a"], p["r"], p["conv_w"], p["gamma"],
                               dy, norm=False, **meta)

    def loss_o(pp):
        o = orc.forward(pp["q"], pp["k"], pp["v"], pp["a"], pp["r"], pp["conv_w"], pp["gamma"],
                        want=("o",), **meta)["o"]
        return float(np.sum(o * dy))

    rng = np.random.default_rng(2)
    h = 1e-5
    for name, gname in (("q", "dq"), ("k", "dk"), ("v", "dv"), ("a", "da"), ("conv_w", "dconv_w")):
        x = p[name]
        for flat in rng.choice(x.size, size=5, replace=False):
            idx = np.unravel_index(flat, x.shape)
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            fd = (loss_o(dict(p, **{name: xp})) - loss_o(dict(p, **{name: xm}))) / (2 * h)
            assert abs(g[gname][idx] - fd) <= 1e-6 + 1e-5 * abs(fd), (gname, idx)
    assert not g["dr"].any() and not g["dgamma"].any()


def test_periodic_inputs_repeat_the_period(orc):
    """The property the slice-limit GPU tests rest on, pinned on the oracles:
    with q, k, v, a, r repeating with period P and the last W - 1 rows of
    q, k, v zero in every period, y over m periods is y of one period
    repeated; with dy repeating too, every per-token gradient over m periods
    equals the two-period one (rows of periods 0..m-2 the first period, rows
    of the last period the second), and dgamma and the taps' gradients scale
    by m / 2."""
    import dataclasses
    from paper_2606_07317_amd import inputs
    P, W, m = 48, 4, 5
    w = inputs.Workload("period", batch=1, heads=2, seqlen=P, head_dim=8, conv_width=W,
                        dtype=inputs.BF16, seed=52)
    inp = inputs.make_inputs(w)
    q, k, v = (x.copy() for x in (inp.q, inp.k, inp.v))
    for x in (q, k, v):
        x[:, :, P - (W - 1):, :] = 0
    inp = dataclasses.replace(inp, q=q, k=k, v=v)

    def rep(x, r):
        return np.concatenate([x] * r, axis=2)

    def repeated(r):
        return dataclasses.replace(inp, workload=w.with_(seqlen=P * r), q=rep(inp.q, r),
                                   k=rep(inp.k, r), v=rep(inp.v, r), a=rep(inp.a, r), r=rep(inp.r, r))

    y1 = orc.forward_inputs(inp)["y"]
    ym = orc.forward_inputs(repeated(m))["y"]
    np.testing.assert_allclose(ym, rep(y1, m), rtol=1e-11, atol=1e-12)
    dy = inputs.make_cotangent(inp)
    g2 = gbla_backward.backward_inputs(repeated(2), rep(dy, 2))
    gm = gbla_backward.backward_inputs(repeated(m), rep(dy, m))
    for name in ("dq", "dk", "dv", "dr", "da"):
        a2, am = g2[name], gm[name]
        first, last = a2[:, :, :P], a2[:, :, P:]
        for p in range(m):
            want = last if p == m - 1 else first
            np.testing.assert_allclose(am[:, :, p * P:(p + 1) * P], want, rtol=1e-9,
                                       atol=1e-12 * np.abs(a2).max(), err_msg=name)
    for name in ("dgamma", "dconv_w"):
        np.testing.assert_allclose(gm[name], g2[name] * (m / 2.0), rtol=1e-9,
                                   atol=1e-12 * np.abs(g2[name]).max(), err_msg=name)
