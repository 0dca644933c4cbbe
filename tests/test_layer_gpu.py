"""Parity of the full layer (gbla_layer_project, gbla_layer_forward, through
the C ABI) with the fp64 layer oracle run with the same bf16 rounding points
(Xt and the projections rounded to bf16).

Projections: the kernel sums K = d_model products in fp32 before its bf16
rounding, the oracle in fp64, and the kernel's Xt comes from an fp32 conv;
so an element may sit one bf16 step away from the oracle's, plus the fp32
sum's error.  Bound: |x - x_ref| <= 2^-7 |x_ref| + 2^-10 sum_k |Xt_k| |W_k|
(one step of 2^-7 relative at most, and 1 ulp of the largest terms for the
sums and the Xt roundings, with margin).
Layer output: the attention core's bf16 tolerance, |y - y_ref| <= 2e-2 (1 +
|y_ref|).
"""
import numpy as np
import pytest
import torch

from paper_2606_07317_amd import inputs
from tests.test_parity_gpu import say

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


LW = inputs.LayerWorkload
CASES = {
    "dm128_h2_d64_n300": (LW("l1", batch=2, seqlen=300, d_model=128, heads=2, head_dim=64,
                              conv_width=4, seed=81), None),
    "dm192_h3_d32_n77_W2": (LW("l2", batch=1, seqlen=77, d_model=192, heads=3, head_dim=32,
                                conv_width=2, seed=82), None),
    "dm256_h1_d128_n129_W1": (LW("l3", batch=2, seqlen=129, d_model=256, heads=1, head_dim=128,
                                  conv_width=1, seed=83), None),
    "ragged_dm128_h2_d64": (LW("l4", batch=4, seqlen=0, d_model=128, heads=2, head_dim=64,
                               conv_width=4, seed=84, ragged=True), [5, 0, 130, 1, 200]),
    # more tiles than the GEMM's 256 persistent workgroups: 275 x 3 tiles in the
    # plain order, the last token tile partial, sequences crossing tile edges
    "ragged_dm128_h2_d64_T70351": (LW("l5", batch=5, seqlen=0, d_model=128, heads=2, head_dim=64,
                                      conv_width=4, seed=85, ragged=True),
                                   [30001, 17, 0, 40000, 333]),
    # 64 x 5 tiles in the XCD-grouped order, with 128-token sequences (a tile
    # holds two, so the scatter computes each token's sequence)
    "dm128_h4_d64_b128_n128": (LW("l6", batch=128, seqlen=128, d_model=128, heads=4, head_dim=64,
                                  conv_width=3, seed=86), None),
}


# Projection-only cases at model widths that are multiples of 1024 with H d a
# multiple of 256: the kernel stages each tile's output and writes it under
# the next tile's products.  Every workgroup owns several tiles here, the
# last feature tile (the gate logits) is written at once, and the ragged
# batch ends in a partial token tile.
DEFER_CASES = {
    "dm1024_h16_d64_b4_n2048": (LW("d1", batch=4, seqlen=2048, d_model=1024, heads=16, head_dim=64,
                                    conv_width=4, seed=91), None),
    "ragged_dm1024_h16_d64_T5000": (LW("d2", batch=4, seqlen=0, d_model=1024, heads=16, head_dim=64,
                                        conv_width=4, seed=92, ragged=True), [1800, 1, 3000, 199]),
    # 64 K steps per tile: the staged pieces run out after the first 32
    "dm2048_h8_d128_b2_n512": (LW("d3", batch=2, seqlen=512, d_model=2048, heads=8, head_dim=128,
                                   conv_width=3, seed=93), None),
}


def oracle_meta(inp):
    w = inp.workload
    rows = w.seqlen if inp.cu_seqlens is None else int(inp.cu_seqlens[-1])
    return dict(nseq=w.batch if inp.cu_seqlens is None else len(inp.cu_seqlens) - 1, rows=rows,
                heads=w.heads, d=w.head_dim, dtype="bf16", cu_seqlens=inp.cu_seqlens)


@pytest.mark.parametrize("name", sorted(CASES) + sorted(DEFER_CASES))
def test_layer_project_parity(G, dev, name):
    from oracle import gbla_layer
    w, lens = CASES[name] if name in CASES else DEFER_CASES[name]
    say("layer project", name)
    inp = inputs.make_layer_inputs(w, lens)
    t = inputs.layer_device_tensors(inp, dev)
    got = G.layer_project(t["x"], t["conv_x"], t["w_proj"], w.heads, w.head_dim,
                          cu_seqlens=t["cu_seqlens"], max_seqlen=t["max_seqlen"])
    torch.cuda.synchronize()
    meta = oracle_meta(inp)
    ref = gbla_layer.project(inp.x, inp.conv_x, inp.w_proj, rounding=True, **meta)
    # sum_k |Xt_k| |W_k|: the same projection of the absolute values
    absx = gbla_layer.project(np.abs(inputs.bf16_bits_to_f32(inp.x)).astype(np.float32),
                              np.abs(inp.conv_x), np.abs(inputs.bf16_bits_to_f32(inp.w_proj)),
                              **dict(meta, dtype="f32"))
    for n in ("q", "k", "v", "r", "a"):
        g = got[n].float().cpu().numpy().astype(np.float64)
        err = np.abs(g - ref[n])
        lim = 2.0 ** -7 * np.abs(ref[n]) + 2.0 ** -10 * absx[n]
        say("  %s max abs %.3e, worst err/bound %.3f, exact %.4f" %
            (n, err.max() if err.size else 0, (err / np.maximum(lim, 1e-30)).max() if err.size else 0,
             np.mean(err == 0) if err.size else 1))
        assert (err <= lim).all(), n


@pytest.mark.parametrize("name", sorted(CASES))
def test_layer_forward_parity(G, dev, orc, name):
    from oracle import gbla_layer
    w, lens = CASES[name]
    say("layer forward", name)
    inp = inputs.make_layer_inputs(w, lens)
    t = inputs.layer_device_tensors(inp, dev)
    y = G.layer_forward(t["x"], t["conv_x"], t["w_proj"], t["gamma"], eps=w.eps,
                        cu_seqlens=t["cu_seqlens"], max_seqlen=t["max_seqlen"])
    torch.cuda.synchronize()
    ref = gbla_layer.layer_forward(orc, inp.x, inp.conv_x, inp.w_proj, inp.gamma, eps=w.eps,
                                   rounding=True, **oracle_meta(inp))["y"]
    got = y.cpu().numpy().astype(np.float64)
    err = np.abs(got - ref)
    say("  y max abs %.3e, worst err/tol %.3f" % (err.max() if err.size else 0,
                                                 (err / (2e-2 * (1 + np.abs(ref)))).max() if err.size else 0))
    assert np.isfinite(got).all()
    assert (err <= 2e-2 * (1 + np.abs(ref))).all()


def test_layer_forward_full_size_table5(G, dev, orc):
    """The paper's Table 5 layer (batch 8, d_model 1024, 16 heads of 64) at
    L = 2048, every output, in the launch configuration bench.py times."""
    from oracle import gbla_layer
    w = inputs.LAYER_WORKLOADS["layer_b8_n2048"]
    say("layer forward full size", w.name)
    inp = inputs.make_layer_inputs(w)
    t = inputs.layer_device_tensors(inp, dev)
    y = G.layer_forward(t["x"], t["conv_x"], t["w_proj"], t["gamma"], eps=w.eps)
    torch.cuda.synchronize()
    ref = gbla_layer.layer_forward(orc, inp.x, inp.conv_x, inp.w_proj, inp.gamma, eps=w.eps,
                                   rounding=True, **oracle_meta(inp))["y"]
    got = y.cpu().numpy().astype(np.float64)
    err = np.abs(got - ref)
    say("  y max abs %.3e, worst err/tol %.3f" % (err.max(), (err / (2e-2 * (1 + np.abs(ref)))).max()))
    assert np.isfinite(got).all()
    assert (err <= 2e-2 * (1 + np.abs(ref))).all()


def test_layer_forward_full_size_long_sampled(G, dev, orc):
    """The bench's layer workload (Table 5's layer at L = 32768, batch 8) in
    its launch configuration: sequences 0 and 7 of the full batch against the
    oracle run on those two sequences alone (every output of a sequence
    depends on that sequence only)."""
    import dataclasses
    from oracle import gbla_layer
    w = inputs.LAYER_WORKLOADS["layer_b8_n32768"]
    say("layer forward full size, sampled", w.name)
    inp = inputs.make_layer_inputs(w)
    t = inputs.layer_device_tensors(inp, dev)
    y = G.layer_forward(t["x"], t["conv_x"], t["w_proj"], t["gamma"], eps=w.eps)
    torch.cuda.synchronize()
    pick = [0, 7]
    got = y[pick].cpu().numpy().astype(np.float64)
    del y, t
    sub = dataclasses.replace(inp, workload=w.with_(batch=len(pick)), x=inp.x[pick])
    ref = gbla_layer.layer_forward(orc, sub.x, sub.conv_x, sub.w_proj, sub.gamma, eps=w.eps,
                                   rounding=True, **oracle_meta(sub))["y"]
    err = np.abs(got - ref)
    say("  y max abs %.3e, worst err/tol %.3f" % (err.max(), (err / (2e-2 * (1 + np.abs(ref)))).max()))
    assert np.isfinite(got).all()
    assert (err <= 2e-2 * (1 + np.abs(ref))).all()
