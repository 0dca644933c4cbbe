"""Each plausible mistake in the backward oracle must fail its finite-difference
pins: the test rebuilds the oracle module from its source with one textual
change and checks that the pins reject it."""
import importlib.util
import os
import types

import numpy as np
import pytest

import oracle
from tests.test_backward_oracle import check_fd, problem

SRC = os.path.join(os.path.dirname(oracle.__file__), "gbla_backward.py")

MUTANTS = {
    "dden_sign": ("dden = -np.sum(do * o, axis=1) / den", "dden = np.sum(do * o, axis=1) / den"),
    "rms_power": ("rs ** 3 / d", "rs ** 2 / d"),
    "state_transpose": ("t = vt @ dS.T + dz[None, :]", "t = vt @ dS + dz[None, :]"),
    "dvt_transpose": ("dvt = g[:, None] * (P @ dS)", "dvt = g[:, None] * (P @ dS.T)"),
    # (dropping the centering term sum_l g_l dg_l is NOT a mistake: the output is
    # invariant to scaling all gates, so that sum is zero; see the pin below)
    "softmax_factor": ("da = g * (dg - np.sum(g * dg))", "da = dg - np.sum(g * dg)"),
    "conv_shift": ("dx[:L - sh] += w[:, t] * dxt[sh:]", "dx[sh:] += w[:, t] * dxt[:L - sh]"),
    "silu_derivative": ("(1.0 + r * (1.0 - sig))", "(1.0 + r * sig)"),
    "dz_term": ("dQh = dnum @ S.T + dden[:, None] * z[None, :]", "dQh = dnum @ S.T"),
}


def mutated_module(old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, old
    mod = types.ModuleType("gbla_backward_mutant")
    exec(compile(src.replace(old, new), SRC, "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_mutant_fails_pins(orc, name, monkeypatch):
    import tests.test_backward_oracle as t
    monkeypatch.setattr(t, "gbla_backward", mutated_module(*MUTANTS[name]))
    p, dy, meta = problem(41)
    with pytest.raises(AssertionError):
        t.check_fd(orc, p, dy, meta, samples=6, seed=1)
