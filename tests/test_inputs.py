"""The seeded input recipe: reproducible, shaped like the workloads, bf16
rounded to nearest even exactly as torch rounds."""
import numpy as np
import torch

from paper_2606_07317_amd import inputs


def test_reproducible_and_shaped():
    a = inputs.make_inputs("tiny_f32")
    b = inputs.make_inputs("tiny_f32")
    for n in ("q", "k", "v", "a", "r", "conv_w", "gamma"):
        assert np.array_equal(getattr(a, n), getattr(b, n))
    assert a.q.shape == (1, 2, 256, 32) and a.q.dtype == np.float32
    assert a.a.shape == (1, 2, 256)
    assert a.conv_w.shape == (3, 2, 32, 4)
    # identity-centred taps: the current-token tap is near 1, the others near 0
    assert abs(a.conv_w[..., 3].mean() - 1.0) < 0.05 and abs(a.conv_w[..., :3].mean()) < 0.05


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 7
    x[:4] = [1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8, 0.0]  # ties to even
    ours = inputs.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    assert np.array_equal(inputs.bf16_bits_to_f32(ours), torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_ragged_lengths_recipe():
    w = inputs.WORKLOADS["ragged64_d128"]
    rng = np.random.Generator(np.random.PCG64(w.seed))
    lens = inputs.draw_lengths(rng, w)
    assert len(lens) == 64 and lens.min() >= 16 and lens.max() <= 32768
    # lognormal(7.5, 1): median about e^7.5 = 1808
    assert 800 < np.median(lens) < 4000


def test_small_ragged_override_and_empty_sequences():
    w = inputs.WORKLOADS["ragged64_d128"].with_(heads=2, head_dim=32)
    inp = inputs.make_inputs(w, lengths=[3, 0, 17, 1])
    assert inp.cu_seqlens.tolist() == [0, 3, 3, 20, 21]
    assert inp.q.shape == (2, 21, 32) and inp.a.shape == (2, 21)
    assert inp.nseq == 4 and inp.tokens == 21
