"""Seeded synthetic inputs for the GBLA forward pass, and the workload table.

This module only draws random numbers and packs them into arrays.  It holds
none of the method's arithmetic, so both the fp64 oracle and the HIP path can
take their inputs from it without sharing any computation.

What the arrays mean (GBLA, Section 2.1 of the paper):

* ``q, k, v``   projected queries / keys / values of every head, before the
  Conv1D (the boundary applies the conv to the projected tensors),
* ``a``         key-gate logits, one scalar per token and head (the argument of
  the sequence softmax in the key-gating item),
* ``r``         output-gate input, the argument of SiLU in the gated RMSNorm item,
* ``conv_w``    causal depthwise Conv1D taps ``[3, H, d, W]`` ordered q, k, v;
  tap ``W-1`` multiplies the current token,
* ``gamma``     RMSNorm weight ``[H, d]``.

Layouts: dense ``[B, H, n, d]`` (``a``: ``[B, H, n]``); ragged ``[H, T, d]``
(``a``: ``[H, T]``) with ``cu_seqlens`` int32 ``[N_s + 1]`` marking where each
sequence starts inside the packed token axis.

Recipe (fixed draw order from ``numpy.random.Generator(PCG64(seed))``):
sequence lengths (ragged workloads only), q, k, v, a, r, conv noise, gamma noise.
Activations are standard normal, drawn in fp32 and, for bf16 workloads, rounded
once to bf16 with round-to-nearest-even.  Taps are ``0.1*N(0,1)`` plus 1 on the
current-token tap; gamma is ``1 + 0.1*N(0,1)``.  Ragged lengths are
``clip(rint(lognormal(7.5, 1.0)), 16, 32768)``.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

F32 = "f32"
BF16 = "bf16"


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    batch: int            # B (dense) or number of sequences N_s (ragged)
    heads: int            # H
    seqlen: int           # n (dense); ignored for ragged (drawn)
    head_dim: int         # d
    conv_width: int       # W
    dtype: str            # F32 or BF16, the dtype of q, k, v, a, r
    seed: int
    ragged: bool = False
    eps: float = 1e-6
    len_mu: float = 7.5
    len_sigma: float = 1.0
    len_min: int = 16
    len_max: int = 32768

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads, named by what they are.  The n=32768, H=8, d=64 bf16
# one is the throughput workload; the others are parity cases.
WORKLOADS = {
    "tiny_f32": Workload("tiny_f32", batch=1, heads=2, seqlen=256, head_dim=32,
                         conv_width=4, dtype=F32, seed=0),
    "b8_n2048_d64": Workload("b8_n2048_d64", batch=8, heads=8, seqlen=2048,
                             head_dim=64, conv_width=4, dtype=BF16, seed=1),
    "b2_n8192_d64": Workload("b2_n8192_d64", batch=2, heads=8, seqlen=8192,
                             head_dim=64, conv_width=4, dtype=BF16, seed=2),
    "b1_n32768_d64": Workload("b1_n32768_d64", batch=1, heads=8, seqlen=32768,
                              head_dim=64, conv_width=4, dtype=BF16, seed=3),
    "ragged64_d128": Workload("ragged64_d128", batch=64, heads=8, seqlen=0,
                              head_dim=128, conv_width=4, dtype=BF16, seed=4,
                              ragged=True),
}
WORKLOAD_ORDER = ["tiny_f32", "b8_n2048_d64", "b2_n8192_d64", "b1_n32768_d64",
                  "ragged64_d128"]
THROUGHPUT_WORKLOAD = "b1_n32768_d64"


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round-to-nearest-even) and return the raw
    16-bit patterns as uint16.  Inputs here are finite normals; NaN is kept NaN."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    # 32-bit arithmetic does not wrap for finite or infinite patterns (at most
    # 0xFF800000 + 0x8000); NaN patterns, which could, are replaced below.
    u = x.view(np.uint32)
    rounded = ((u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
               >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        rounded[nan] = 0x7FC0
    return rounded


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen raw bf16 patterns (uint16) to fp32 exactly."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


@dataclasses.dataclass
class Inputs:
    workload: Workload
    q: np.ndarray          # uint16 (bf16 bits) or float32
    k: np.ndarray
    v: np.ndarray
    a: np.ndarray
    r: np.ndarray
    conv_w: np.ndarray     # float32 [3, H, d, W]
    gamma: np.ndarray      # float32 [H, d]
    cu_seqlens: Optional[np.ndarray]  # int32 [N_s + 1] or None (dense)
    eps: float

    @property
    def nseq(self) -> int:
        return self.workload.batch

    @property
    def rows(self) -> int:
        """Tokens per head: n (dense) or T (ragged)."""
        return int(self.cu_seqlens[-1]) if self.cu_seqlens is not None else self.workload.seqlen

    @property
    def tokens(self) -> int:
        """Total tokens of the batch (sum of sequence lengths)."""
        return self.rows if self.cu_seqlens is not None else self.workload.batch * self.workload.seqlen

    def lengths(self) -> np.ndarray:
        if self.cu_seqlens is None:
            return np.full(self.workload.batch, self.workload.seqlen, dtype=np.int64)
        return np.diff(self.cu_seqlens.astype(np.int64))


def draw_lengths(rng: np.random.Generator, w: Workload) -> np.ndarray:
    raw = rng.lognormal(mean=w.len_mu, sigma=w.len_sigma, size=w.batch)
    return np.clip(np.rint(raw), w.len_min, w.len_max).astype(np.int64)


def make_inputs(w: Workload | str, lengths: Optional[np.ndarray] = None) -> Inputs:
    """Draw one seeded batch for workload ``w``.

    ``lengths`` overrides the drawn ragged lengths (small ragged test cases);
    the override is consumed instead of the length draw, so the rest of the
    draw order is unchanged."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    rng = np.random.Generator(np.random.PCG64(w.seed))
    H, d, W = w.heads, w.head_dim, w.conv_width
    if w.ragged:
        if lengths is None:
            lengths = draw_lengths(rng, w)
        lengths = np.asarray(lengths, dtype=np.int64)
        if len(lengths) != w.batch:
            w = w.with_(batch=len(lengths))
        cu = np.zeros(len(lengths) + 1, dtype=np.int64)
        np.cumsum(lengths, out=cu[1:])
        if cu[-1] >= 2**31:
            raise ValueError("ragged batch too large for int32 offsets")
        cu_seqlens = cu.astype(np.int32)
        T = int(cu[-1])
        act_shape = (H, T, d)
        gate_shape = (H, T)
    else:
        cu_seqlens = None
        act_shape = (w.batch, H, w.seqlen, d)
        gate_shape = (w.batch, H, w.seqlen)

    def act(shape):
        x = rng.standard_normal(size=shape, dtype=np.float32)
        return f32_to_bf16_bits(x) if w.dtype == BF16 else x

    q = act(act_shape)
    k = act(act_shape)
    v = act(act_shape)
    a = act(gate_shape)
    r = act(act_shape)
    conv_w = (0.1 * rng.standard_normal(size=(3, H, d, W), dtype=np.float32)).astype(np.float32)
    conv_w[..., W - 1] += np.float32(1.0)
    gamma = (np.float32(1.0) + np.float32(0.1) * rng.standard_normal(size=(H, d), dtype=np.float32)).astype(np.float32)
    return Inputs(w, q, k, v, a, r, conv_w, gamma, cu_seqlens, w.eps)


def make_cotangent(inp: Inputs, seed_offset: int = 1000) -> np.ndarray:
    """Seeded dL/dy for a backward test: fp32 standard normal in the layout of
    ``q``, from its own generator (seed = workload seed + ``seed_offset``)."""
    rng = np.random.Generator(np.random.PCG64(inp.workload.seed + seed_offset))
    return rng.standard_normal(size=inp.q.shape, dtype=np.float32)


@dataclasses.dataclass(frozen=True)
class LayerWorkload:
    """A full-layer batch: embeddings X [B, L, d_model] (or packed [T, d_model])."""
    name: str
    batch: int
    seqlen: int           # L (dense); ignored for ragged
    d_model: int
    heads: int
    head_dim: int
    conv_width: int
    seed: int
    ragged: bool = False
    eps: float = 1e-6

    def with_(self, **kw) -> "LayerWorkload":
        return dataclasses.replace(self, **kw)


# Table 5's layer (batch 8, model width 1024, 16 heads of 64) at two lengths.
LAYER_WORKLOADS = {
    "layer_b8_n2048": LayerWorkload("layer_b8_n2048", batch=8, seqlen=2048, d_model=1024, heads=16,
                                    head_dim=64, conv_width=4, seed=5),
    "layer_b8_n32768": LayerWorkload("layer_b8_n32768", batch=8, seqlen=32768, d_model=1024,
                                     heads=16, head_dim=64, conv_width=4, seed=6),
}


@dataclasses.dataclass
class LayerInputs:
    workload: LayerWorkload
    x: np.ndarray          # uint16 bf16 bits, [B, L, d_model] or [T, d_model]
    conv_x: np.ndarray     # float32 [d_model, W]
    w_proj: np.ndarray     # uint16 bf16 bits, [4*H*d + H, d_model]
    gamma: np.ndarray      # float32 [H, d]
    cu_seqlens: Optional[np.ndarray]


def make_layer_inputs(w: LayerWorkload, lengths=None) -> LayerInputs:
    """Draw order from PCG64(seed): lengths (ragged only), x, conv noise,
    weights, gamma noise.  x ~ N(0, 1) and the weights ~ N(0, 1/d_model), both
    rounded once to bf16, so every projection is about N(0, 1); taps are
    0.1 N(0, 1) plus 1 on the current token; gamma is 1 + 0.1 N(0, 1)."""
    rng = np.random.Generator(np.random.PCG64(w.seed))
    if w.ragged:
        lengths = np.asarray(lengths, dtype=np.int64)
        cu = np.zeros(len(lengths) + 1, dtype=np.int64)
        np.cumsum(lengths, out=cu[1:])
        cu_seqlens = cu.astype(np.int32)
        xs = (int(cu[-1]), w.d_model)
        if len(lengths) != w.batch:
            w = w.with_(batch=len(lengths))
    else:
        cu_seqlens = None
        xs = (w.batch, w.seqlen, w.d_model)
    x = f32_to_bf16_bits(rng.standard_normal(size=xs, dtype=np.float32))
    conv_x = (0.1 * rng.standard_normal(size=(w.d_model, w.conv_width), dtype=np.float32)).astype(np.float32)
    conv_x[:, -1] += np.float32(1.0)
    N = w.heads * (4 * w.head_dim + 1)
    wp = rng.standard_normal(size=(N, w.d_model), dtype=np.float32) / np.float32(np.sqrt(w.d_model))
    w_proj = f32_to_bf16_bits(wp.astype(np.float32))
    gamma = (np.float32(1.0) + np.float32(0.1) * rng.standard_normal(size=(w.heads, w.head_dim),
                                                                      dtype=np.float32)).astype(np.float32)
    return LayerInputs(w, x, conv_x, w_proj, gamma, cu_seqlens)


def layer_device_tensors(inp: LayerInputs, device) -> dict:
    import torch
    out = {"x": to_torch(inp.x, BF16, device), "w_proj": to_torch(inp.w_proj, BF16, device),
           "conv_x": torch.from_numpy(np.ascontiguousarray(inp.conv_x)).to(device),
           "gamma": torch.from_numpy(np.ascontiguousarray(inp.gamma)).to(device)}
    out["cu_seqlens"] = (torch.from_numpy(inp.cu_seqlens).to(device)
                         if inp.cu_seqlens is not None else None)
    out["max_seqlen"] = (int(np.diff(inp.cu_seqlens).max()) if inp.cu_seqlens is not None
                         and len(inp.cu_seqlens) > 1 else None)
    return out


def to_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact fp64 view of an activation array stored as ``dtype``."""
    if dtype == BF16:
        return bf16_bits_to_f32(x).astype(np.float64)
    return np.asarray(x, dtype=np.float32).astype(np.float64)


def to_torch(x: np.ndarray, dtype: str, device):
    """Copy one activation array to a torch tensor (bf16 patterns become
    torch.bfloat16 with the same bits)."""
    import torch
    if dtype == BF16:
        t = torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(device)


def device_tensors(inp: Inputs, device) -> dict:
    """All arrays of ``inp`` as torch tensors on ``device``."""
    import torch
    dt = inp.workload.dtype
    out = {n: to_torch(getattr(inp, n), dt, device) for n in ("q", "k", "v", "a", "r")}
    out["conv_w"] = torch.from_numpy(np.ascontiguousarray(inp.conv_w)).to(device)
    out["gamma"] = torch.from_numpy(np.ascontiguousarray(inp.gamma)).to(device)
    out["cu_seqlens"] = (torch.from_numpy(inp.cu_seqlens).to(device)
                         if inp.cu_seqlens is not None else None)
    out["max_seqlen"] = int(inp.lengths().max()) if inp.cu_seqlens is not None and inp.nseq else None
    return out
