"""Pins of the full-layer oracle (oracle/gbla_layer.py), on the CPU.

The layer applies the Conv1D to X before the projections (Section 2.1); the
boundary oracle applies it to the projected q, k, v.  The two agree exactly
when the conv taps are shared across channels, which ties the layer oracle to
the independently pinned forward oracle."""
import numpy as np
import pytest

from oracle import gbla_layer


def layer_problem(seed, nseq=2, L=11, dm=12, H=2, d=4, W=4, ragged=None, shared=False):
    rng = np.random.default_rng(seed)
    if ragged is not None:
        cu = np.concatenate([[0], np.cumsum(ragged)]).astype(np.int32)
        nseq, T = len(ragged), int(cu[-1])
        x = rng.standard_normal((T, dm))
    else:
        cu = None
        x = rng.standard_normal((nseq, L, dm))
    if shared:
        cx = np.broadcast_to(rng.standard_normal(W), (dm, W)).copy()
    else:
        cx = rng.standard_normal((dm, W))
    N = 4 * H * d + H
    wp = rng.standard_normal((N, dm)) / np.sqrt(dm)
    gamma = 1.0 + 0.1 * rng.standard_normal((H, d))
    meta = dict(nseq=nseq, rows=L if cu is None else int(cu[-1]), heads=H, d=d, dtype="f64",
                eps=1e-6, cu_seqlens=cu)
    return x, cx, wp, gamma, meta


def test_round_bf16_ties_and_values():
    one = 1.0
    ulp = 2.0 ** -7                                          # bf16 spacing in [1, 2)
    assert gbla_layer.round_bf16(one + ulp / 2) == one       # tie -> even
    assert gbla_layer.round_bf16(one + 3 * ulp / 2) == one + 2 * ulp
    assert gbla_layer.round_bf16(one + ulp / 2 + 1e-12) == one + ulp
    assert gbla_layer.round_bf16(-3.0) == -3.0
    # agrees with rounding the fp32 bit pattern (for fp32-representable values)
    from paper_2606_07317_amd import inputs
    x = np.random.default_rng(1).standard_normal(10000).astype(np.float32)
    want = inputs.bf16_bits_to_f32(inputs.f32_to_bf16_bits(x)).astype(np.float64)
    np.testing.assert_array_equal(gbla_layer.round_bf16(x.astype(np.float64)), want)


def test_conv_x_against_numpy_convolve():
    rng = np.random.default_rng(2)
    X = rng.standard_normal((9, 5))
    for W in (1, 2, 3, 4):
        cx = rng.standard_normal((5, W))
        got = gbla_layer.conv_x(X, cx)
        for m in range(5):
            np.testing.assert_allclose(got[:, m], np.convolve(X[:, m], cx[m, ::-1])[:9], rtol=1e-14,
                                       atol=1e-14)


@pytest.mark.parametrize("W", [1, 2, 4])
def test_shared_taps_equal_the_boundary_form(orc, W):
    """conv(X) W = conv(X W) for channel-shared taps: the layer equals the
    boundary oracle fed unconvolved q, k, v with the core conv on, and a, r
    taken from the convolved embeddings."""
    x, cx, wp, gamma, meta = layer_problem(10 + W, W=W, shared=True)
    H, d = meta["heads"], meta["d"]
    y = gbla_layer.layer_forward(orc, x, cx, wp, gamma, **meta)["y"]
    flat = gbla_layer.project(x, np.eye(1, W, W - 1).repeat(cx.shape[0], 0), wp,
                              **{k: meta[k] for k in ("nseq", "rows", "heads", "d", "dtype")})
    conv_ar = gbla_layer.project(x, cx, wp, **{k: meta[k] for k in ("nseq", "rows", "heads", "d", "dtype")})
    taps = np.broadcast_to(cx[0], (3, H, d, W)).copy()
    ref = orc.forward(flat["q"], flat["k"], flat["v"], conv_ar["a"], conv_ar["r"], taps, gamma,
                      nseq=meta["nseq"], heads=H, rows=meta["rows"], d=d, W=W, dtype="f64",
                      eps=meta["eps"])["y"]
    np.testing.assert_allclose(y, ref, rtol=1e-10, atol=1e-12)


def test_ragged_equals_per_sequence(orc):
    lens = [5, 0, 1, 9]
    x, cx, wp, gamma, meta = layer_problem(20, ragged=lens)
    y = gbla_layer.layer_forward(orc, x, cx, wp, gamma, want=("y", "q", "a"), **meta)
    cu = meta["cu_seqlens"]
    for s, L in enumerate(lens):
        if L == 0:
            continue
        m1 = dict(meta, nseq=1, rows=L, cu_seqlens=None)
        one = gbla_layer.layer_forward(orc, x[cu[s]:cu[s + 1]][None], cx, wp, gamma,
                                       want=("y", "q", "a"), **m1)
        np.testing.assert_allclose(y["y"][:, cu[s]:cu[s + 1]], one["y"][0], rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(y["q"][:, cu[s]:cu[s + 1]], one["q"][0], rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(y["a"][:, cu[s]:cu[s + 1]], one["a"][0], rtol=1e-12, atol=1e-14)


def test_projection_layout_and_causality():
    """Row h*d + e of each block is head h, channel e; a token's projections
    depend only on its conv window (tokens i-W+1 .. i of its sequence)."""
    x, cx, wp, gamma, meta = layer_problem(30, nseq=1, L=10, dm=6, H=3, d=2, W=3)
    pm = {k: meta[k] for k in ("nseq", "rows", "heads", "d", "dtype")}
    p = gbla_layer.project(x, cx, wp, **pm)
    Xt = gbla_layer.conv_x(x[0], cx)
    H, d = 3, 2
    for blk, name in enumerate(("q", "k", "v", "r")):
        for h in range(H):
            for e in range(d):
                np.testing.assert_allclose(p[name][0, h, :, e], Xt @ wp[blk * H * d + h * d + e],
                                           rtol=1e-13, atol=1e-13)
    for h in range(H):
        np.testing.assert_allclose(p["a"][0, h], Xt @ wp[4 * H * d + h], rtol=1e-13, atol=1e-13)
    x2 = x.copy()
    x2[0, 6] += 1.0
    p2 = gbla_layer.project(x2, cx, wp, **pm)
    changed = np.abs(p2["q"] - p["q"]).max(axis=(0, 1, 3)) > 0
    assert list(np.nonzero(changed)[0]) == [6, 7, 8]


def test_rounding_is_applied_to_both_stages():
    x, cx, wp, gamma, meta = layer_problem(40, nseq=1, L=6, dm=8, H=1, d=4)
    pm = {k: meta[k] for k in ("nseq", "rows", "heads", "d", "dtype")}
    p = gbla_layer.project(x, cx, wp, rounding=True, **pm)
    for name in ("q", "k", "v", "r", "a"):
        np.testing.assert_array_equal(gbla_layer.round_bf16(p[name]), p[name])
    Xt = gbla_layer.round_bf16(gbla_layer.conv_x(x[0], cx))
    np.testing.assert_array_equal(p["q"][0, 0], gbla_layer.round_bf16(Xt @ wp[:4].T))
