"""Plant plausible mistakes in a copy of the oracle (on the CPU) and check
that the pin suite catches every one of them.

Each mutant is the oracle's C source with one textual change (a dropped term,
a wrong sign or index, a transposed operand, a swapped weight), compiled with
gcc into a temporary library.  The unmodified source must pass every pin.
"""
import os
import shutil
import tempfile

import pytest

import oracle
from tests import test_oracle_pins as pins

SRC = os.path.join(os.path.dirname(oracle.__file__), "gbla_oracle.c")

# (name, original text, replacement); the original must occur exactly once.
MUTANTS = [
    ("tap_order_flipped", "int64_t src = i - (W - 1) + t;", "int64_t src = i - t;"),
    ("conv_drops_first_token", "if (src < 0) continue;", "if (src <= 0) continue;"),
    ("phi_without_plus_one", "return u > 0.0 ? u + 1.0 : exp(u);", "return u > 0.0 ? u : exp(u) - 1.0;"),
    ("phi_branch_shifted", "return u > 0.0 ? u + 1.0 : exp(u);", "return u > 1.0 ? u + 1.0 : exp(u);"),
    ("gates_unnormalised", "for (int64_t j = 0; j < L; ++j) g[j] /= denom;", ""),
    ("gate_not_applied", "double kh = g[j] * gbla_oracle_phi(kt[(size_t)j * d + c]);",
     "double kh = gbla_oracle_phi(kt[(size_t)j * d + c]);"),
    ("state_transposed", "S[(size_t)c * d + e] += kh * vt[(size_t)j * d + e];",
     "S[(size_t)e * d + c] += kh * vt[(size_t)j * d + e];"),
    ("readout_transposed", "o[e] += qh * S[(size_t)c * d + e];", "o[e] += qh * S[(size_t)e * d + c];"),
    ("query_phi_missing", "double qh = gbla_oracle_phi(qt[(size_t)i * d + c]);",
     "double qh = qt[(size_t)i * d + c];"),
    ("denominator_dropped", "for (int e = 0; e < d; ++e) o[e] /= den;", ""),
    ("z_ungated", "z[c] += kh;", "z[c] += gbla_oracle_phi(kt[(size_t)j * d + c]);"),
    ("rms_wrong_count", "ms /= (double)d;", "ms /= (double)(d + 1);"),
    ("rms_eps_dropped", "const double inv = 1.0 / sqrt(ms + P->eps);", "const double inv = 1.0 / sqrt(ms);"),
    ("silu_is_sigmoid", "static double silu(double x) { return x / (1.0 + exp(-x)); }",
     "static double silu(double x) { return 1.0 / (1.0 + exp(-x)); }"),
    ("silu_sign", "static double silu(double x) { return x / (1.0 + exp(-x)); }",
     "static double silu(double x) { return x / (1.0 + exp(x)); }"),
    ("gamma_head_ignored", "const double* gam = gamma + (size_t)h * d;", "const double* gam = gamma;"),
    ("k_uses_q_taps", "conv_slice(P, k, conv_w + ((size_t)1 * H + h) * d * W, s, h, L, kt);",
     "conv_slice(P, k, conv_w + ((size_t)0 * H + h) * d * W, s, h, L, kt);"),
    ("v_uses_k_taps", "conv_slice(P, v, conv_w + ((size_t)2 * H + h) * d * W, s, h, L, vt);",
     "conv_slice(P, v, conv_w + ((size_t)1 * H + h) * d * W, s, h, L, vt);"),
    ("taps_head_ignored", "conv_slice(P, q, conv_w + ((size_t)0 * H + h) * d * W, s, h, L, qt);",
     "conv_slice(P, q, conv_w + ((size_t)0 * H + 0) * d * W, s, h, L, qt);"),
    ("packed_head_offset_dropped", "return (size_t)h * (size_t)P->rows + (size_t)P->offsets[s] + (size_t)i;",
     "return (size_t)P->offsets[s] + (size_t)i;"),
    ("softmax_max_sign", "if (aj > amax) amax = aj;", "if (aj < amax || amax == -INFINITY) amax = aj;"),
]


def pin_suite(orc):
    """Run the pins against ``orc``; return the names of the failing ones."""
    checks = [
        ("golden", lambda: pins.test_golden_handworked(orc)),
        ("phi", lambda: pins.test_phi_closed_form(orc)),
        ("convolve", lambda: pins.test_conv_matches_numpy_convolve(orc, 4)),
        ("causality", lambda: pins.test_conv_causality(orc)),
        ("identity_shift", lambda: pins.test_conv_identity_and_shift(orc)),
        ("ragged", lambda: pins.test_conv_does_not_cross_sequences(orc)),
        ("softmax", lambda: pins.test_gates_are_sequence_softmax(orc)),
        ("permutation", lambda: pins.test_state_permutation_invariance(orc)),
        ("bruteforce", lambda: pins.test_readout_matches_quadratic_bruteforce(orc, 7)),
        ("unit_rms", lambda: pins.test_unit_rms(orc)),
        ("gamma", lambda: pins.test_gate_and_gamma(orc)),
        ("eq1", lambda: pins.test_reduces_to_bla_eq1(orc)),
        ("paper_form", lambda: pins.test_paper_form_conv_on_embeddings(orc)),
        ("heads", lambda: pins.test_heads_use_their_own_weights(orc)),
    ]
    failed = []
    for name, fn in checks:
        try:
            fn()
        except (AssertionError, ValueError, FloatingPointError):
            failed.append(name)
    return failed


@pytest.fixture(scope="module")
def workdir():
    d = tempfile.mkdtemp(prefix="gbla_mutants_")
    yield d
    shutil.rmtree(d, ignore_errors=True)


def _compile(workdir, name, text):
    src = os.path.join(workdir, name + ".c")
    with open(src, "w") as f:
        f.write(text)
    return oracle.load(oracle.build(force=True, out=os.path.join(workdir, name + ".so"), src=src))


def test_unmodified_oracle_passes_every_pin(workdir):
    orc = _compile(workdir, "original", open(SRC).read())
    assert pin_suite(orc) == []


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_pins_catch_mutant(workdir, name, old, new):
    text = open(SRC).read()
    assert text.count(old) == 1, "mutation anchor must occur exactly once: " + old
    orc = _compile(workdir, name, text.replace(old, new))
    failed = pin_suite(orc)
    assert failed, "no pin caught mutant " + name
