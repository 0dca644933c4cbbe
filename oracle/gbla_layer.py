"""Plain fp64 oracle of the full GBLA layer from the input embeddings X
(Section 2.1: the Conv1D on X, the per-head projections, then the GBLA
attention with the gated RMSNorm).

TEST INFRASTRUCTURE ONLY: the tests use it; the product path never imports
it, and it shares no code with the HIP library.

For each sequence (tokens i, model channels m, heads h, head channels e):

    Xt[i][m] = sum_{t<W} cx[m][t] X[i-W+1+t][m]      (Section 2.1, "Conv1D":
                                                   causal, depthwise, zero
                                                   before the sequence start)
    Q = Xt W_Q,  K = Xt W_K,  V = Xt W_V           (the same item)
    a = Xt w_g                                      ("Key gating")
    R = Xt W_R                                      ("RMSNorm with gating")
    y = the GBLA attention and gated RMSNorm of (Q, K, V, a, R) per head
        (the forward oracle, with its own conv switched off: identity taps)

The projection weights come stacked as one matrix Wp [N, d_model] (the rows
are output features): rows h*d + e are W_Q's column (h, e), then W_K, W_V,
W_R in the same order, then the H rows of w_g.  So P = Xt Wp^T holds every
projection of a token in one row.

With ``round_bf16=True`` the oracle also rounds Xt and P to bf16 (round to
nearest, ties to even), the precision at which a bf16 layer stores them;
everything else stays fp64.
"""
from __future__ import annotations

from typing import Optional

import numpy as np


def round_bf16(x) -> np.ndarray:
    """Round to the nearest value with an 8-bit significand (bf16), ties to
    even.  Finite inputs in the normal range only."""
    x = np.asarray(x, dtype=np.float64)
    m, e = np.frexp(x)                      # x = m 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(np.ldexp(m, 8)), e - 8)


def conv_x(X, cx) -> np.ndarray:
    """Causal depthwise conv of one sequence X [L, d_model] with taps
    cx [d_model, W] (tap W-1 on the current token)."""
    L = X.shape[0]
    W = cx.shape[1]
    out = np.zeros_like(X)
    for t in range(W):
        sh = W - 1 - t                      # X[i - sh]
        if sh < L:
            out[sh:] += cx[:, t] * X[:L - sh]
    return out


def _widen(x, dtype: str) -> np.ndarray:
    x = np.asarray(x)
    if dtype == "bf16":
        return (x.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return x.astype(np.float64)


def project(x, cx, w_proj, *, nseq: int, rows: int, heads: int, d: int, dtype: str,
            cu_seqlens: Optional[np.ndarray] = None, rounding: bool = False) -> dict:
    """The conv and the projections: q, k, v, r [nseq, H, rows, d] (dense) or
    [H, T, d] (ragged) and a without the trailing d, in fp64."""
    X = _widen(x, dtype)
    cx = np.asarray(cx, dtype=np.float64)
    Wp = np.asarray(w_proj, dtype=np.float64) if dtype != "bf16" else _widen(w_proj, dtype)
    dm = cx.shape[0]
    if cu_seqlens is None:
        X = X.reshape(nseq, rows, dm)
        seqs = [X[s] for s in range(nseq)]
    else:
        X = X.reshape(-1, dm)
        seqs = [X[int(cu_seqlens[s]):int(cu_seqlens[s + 1])] for s in range(nseq)]
    Hd = heads * d
    outs = []
    for Xs in seqs:
        Xt = conv_x(Xs, cx)
        if rounding:
            Xt = round_bf16(Xt)
        P = Xt @ Wp.T
        if rounding:
            P = round_bf16(P)
        outs.append(P)
    res = {}
    for name, blk in (("q", 0), ("k", 1), ("v", 2), ("r", 3)):
        parts = [P[:, blk * Hd:(blk + 1) * Hd].reshape(-1, heads, d).transpose(1, 0, 2)
                 for P in outs]                                   # [H, L_s, d]
        res[name] = (np.stack(parts) if cu_seqlens is None
                     else np.concatenate(parts, axis=1) if parts else np.zeros((heads, 0, d)))
    gparts = [P[:, 4 * Hd:4 * Hd + heads].T for P in outs]          # [H, L_s]
    res["a"] = (np.stack(gparts) if cu_seqlens is None
                else np.concatenate(gparts, axis=1) if gparts else np.zeros((heads, 0)))
    return res


def layer_forward(orc, x, cx, w_proj, gamma, *, nseq: int, rows: int, heads: int, d: int,
                  dtype: str, eps: float, cu_seqlens: Optional[np.ndarray] = None,
                  rounding: bool = False, want=("y",)) -> dict:
    """y of the whole layer (in the core's layout), and the projections when
    ``want`` names them.  ``orc`` is the forward oracle."""
    p = project(x, cx, w_proj, nseq=nseq, rows=rows, heads=heads, d=d, dtype=dtype,
                cu_seqlens=cu_seqlens, rounding=rounding)
    ident = np.ones((3, heads, d, 1))
    T = p["q"].shape[1] if cu_seqlens is not None else rows
    core = orc.forward(p["q"], p["k"], p["v"], p["a"], p["r"], ident, gamma, nseq=nseq,
                       heads=heads, rows=T, d=d, W=1, dtype="f64", eps=eps,
                       cu_seqlens=cu_seqlens, want=tuple(w for w in want if w not in p))
    core.update({k: v for k, v in p.items() if k in want})
    return core
