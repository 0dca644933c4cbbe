"""Python binding of libgbla.so (argument marshalling only).

Every step of the GBLA forward pass runs in the HIP kernels behind the C ABI
declared in ``include/gbla.h``; this module checks tensor metadata, passes
device pointers and the current HIP stream, and turns status codes into
exceptions.  PyTorch provides device memory and streams, nothing else.  If
the library is not built this module raises; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional, Tuple

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libgbla.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "gbla.h")

GBLA_F32 = 0
GBLA_BF16 = 1
# Ablation switches (shape.flags); all three together is plain BLA, Eq. (1).
NO_GATE = 1   # uniform key gates; gate_logits may be None
NO_CONV = 2   # identity Conv1D; conv_w may be None
NO_NORM = 4   # out = o; out_gate and norm_w may be None
BLA = NO_GATE | NO_CONV | NO_NORM
STATUS_NAMES = {0: "GBLA_OK", 1: "GBLA_ERR_INVALID_ARGUMENT", 2: "GBLA_ERR_UNSUPPORTED",
                3: "GBLA_ERR_MISALIGNED", 4: "GBLA_ERR_WORKSPACE", 5: "GBLA_ERR_HIP"}


class GblaError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__("%s failed: %s" % (where, STATUS_NAMES.get(status, status)))


class Shape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("heads", ctypes.c_int32), ("seqlen", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("conv_width", ctypes.c_int32),
                ("max_seqlen", ctypes.c_int32), ("dtype", ctypes.c_int32), ("eps", ctypes.c_float),
                ("flags", ctypes.c_uint32)]


class LayerShape(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("seqlen", ctypes.c_int32), ("d_model", ctypes.c_int32),
                ("heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("conv_width", ctypes.c_int32), ("max_seqlen", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("eps", ctypes.c_float)]


_lib = None


def load_library(path: str = LIB_PATH):
    """Load libgbla.so and declare its signatures.  Raises if it is missing."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise GblaError(-1, "loading %s (not built: run __graft_entry__.build())" % path)
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    SP = ctypes.POINTER(Shape)
    sz = ctypes.c_size_t
    lib.gbla_workspace_bytes.argtypes = [SP]
    lib.gbla_workspace_bytes.restype = sz
    lib.gbla_forward.argtypes = [SP, P, P, P, P, P, P, P, P, P, sz, P, P]
    lib.gbla_forward.restype = ctypes.c_int
    lib.gbla_forward_timed.argtypes = [SP, P, P, P, P, P, P, P, P, P, sz, P, P, P, P]
    lib.gbla_forward_timed.restype = ctypes.c_int
    lib.gbla_conv1d.argtypes = [SP, P, P, P, P, P, P, P, P, P]
    lib.gbla_conv1d.restype = ctypes.c_int
    lib.gbla_state.argtypes = [SP, P, P, P, P, P, P, sz, P, P, P]
    lib.gbla_state.restype = ctypes.c_int
    lib.gbla_readout.argtypes = [SP, P, P, P, P, P, P, sz, P, P]
    lib.gbla_readout.restype = ctypes.c_int
    lib.gbla_readout_timed.argtypes = [SP, P, P, P, P, P, P, sz, P, P, P, P]
    lib.gbla_readout_timed.restype = ctypes.c_int
    lib.gbla_forward_noalloc.argtypes = [SP, P, P, P, P, P, P, P, P, P, P]
    lib.gbla_forward_noalloc.restype = ctypes.c_int
    lib.gbla_stream_ceiling.argtypes = [P, P, P, P, P, ctypes.c_int64, ctypes.c_int32, P, P]
    lib.gbla_stream_ceiling.restype = ctypes.c_int
    lib.gbla_backward_workspace_bytes.argtypes = [SP]
    lib.gbla_backward_workspace_bytes.restype = sz
    lib.gbla_backward.argtypes = [SP, P, P, P, P, P, P, P, P, P, P, sz, P, P, P, P, P, P, P, P]
    lib.gbla_backward.restype = ctypes.c_int
    LP = ctypes.POINTER(LayerShape)
    lib.gbla_layer_workspace_bytes.argtypes = [LP]
    lib.gbla_layer_workspace_bytes.restype = sz
    lib.gbla_layer_project.argtypes = [LP, P, P, P, P, P, sz, P, P, P, P, P, P]
    lib.gbla_layer_project.restype = ctypes.c_int
    lib.gbla_layer_forward.argtypes = [LP, P, P, P, P, P, P, sz, P, P]
    lib.gbla_layer_forward.restype = ctypes.c_int
    lib.gbla_status_string.argtypes = [ctypes.c_int]
    lib.gbla_status_string.restype = ctypes.c_char_p
    if path == LIB_PATH:
        _lib = lib
    return lib


def declared_functions(header: str = HEADER_PATH):
    """Names of the functions that include/gbla.h declares."""
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gbla_[a-z0-9_]+)\s*\(", text)))


# ---------------------------------------------------------------------------
# Tensor marshalling.
# ---------------------------------------------------------------------------
def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return GBLA_BF16
    if t.dtype == torch.float32:
        return GBLA_F32
    raise TypeError("activations must be bfloat16 or float32, got %s" % t.dtype)


def _check(t: torch.Tensor, name: str, dtype=None, device=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if not t.is_cuda:
        raise ValueError("%s must live on the GPU" % name)
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if device is not None and t.device != device:
        raise ValueError("%s is on %s, expected %s" % (name, t.device, device))


def _check_out(out: torch.Tensor, shape, dev, name: str = "out"):
    """An output buffer the kernels write in full: fp32, contiguous, on the
    device of the inputs, with exactly the expected shape."""
    _check(out, name, torch.float32, dev)
    if tuple(out.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(out.shape), tuple(shape)))


def _check_ws(ws: torch.Tensor, dev, need: int, name: str = "workspace"):
    """Caller-supplied scratch: a contiguous uint8 tensor on the inputs'
    device, at least ``need`` bytes (the library checks the size and the
    256-byte alignment again)."""
    _check(ws, name, torch.uint8, dev)
    if ws.numel() < need:
        raise ValueError("%s holds %d bytes, %d needed" % (name, ws.numel(), need))


def make_shape(q: torch.Tensor, conv_w: Optional[torch.Tensor], eps: float,
               cu_seqlens: Optional[torch.Tensor], max_seqlen: Optional[int],
               flags: int = 0) -> Shape:
    if cu_seqlens is None:
        if q.dim() != 4:
            raise ValueError("dense q must be [B, H, n, d]")
        B, H, n, d = q.shape
        batch, rows, msl = B, n, 0
    else:
        if q.dim() != 3:
            raise ValueError("ragged q must be [H, T, d]")
        H, rows, d = q.shape
        batch = cu_seqlens.numel() - 1
        msl = int(max_seqlen) if max_seqlen is not None else rows
    if conv_w is None:
        if not flags & NO_CONV:
            raise ValueError("conv_w is required unless flags has NO_CONV")
        W = 1  # identity conv
    else:
        if conv_w.dim() != 4 or tuple(conv_w.shape[:3]) != (3, H, d):
            raise ValueError("conv_w must be [3, H, d, W]")
        W = conv_w.shape[3]
    return Shape(batch, H, rows, d, W, msl, _dtype_code(q), float(eps), int(flags))


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _raise(st: int, where: str):
    if st != 0:
        raise GblaError(st, where)


def workspace_bytes(shape: Shape) -> int:
    n = load_library().gbla_workspace_bytes(ctypes.byref(shape))
    if n == 0:
        raise GblaError(1, "gbla_workspace_bytes")
    return int(n)


def alloc_workspace(shape: Shape, device) -> torch.Tensor:
    """Caller-owned scratch for gbla_forward / gbla_state (256-byte aligned)."""
    return torch.empty(workspace_bytes(shape), dtype=torch.uint8, device=device)


def _check_inputs(q, k, v, a, r, conv_w, norm_w, cu_seqlens):
    dev = q.device
    for t, nm in ((q, "q"), (k, "k"), (v, "v"), (r, "out_gate")):
        if t is not None:
            _check(t, nm, q.dtype, dev)
            if t.shape != q.shape:
                raise ValueError("%s has shape %s, expected %s" % (nm, tuple(t.shape), tuple(q.shape)))
    if a is not None:
        _check(a, "gate_logits", q.dtype, dev)
        if a.shape != q.shape[:-1]:
            raise ValueError("gate_logits must have shape %s" % (tuple(q.shape[:-1]),))
    if conv_w is not None:
        _check(conv_w, "conv_w", torch.float32, dev)
    if norm_w is not None:
        _check(norm_w, "norm_w", torch.float32, dev)
        if norm_w.shape != (q.shape[-3], q.shape[-1]):
            raise ValueError("norm_w must be [H, d]")
    if cu_seqlens is not None:
        _check(cu_seqlens, "cu_seqlens", torch.int32, dev)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def forward(q, k, v, gate_logits, out_gate, conv_w, norm_w, eps: float = 1e-6,
            cu_seqlens=None, max_seqlen=None, workspace=None, out=None, stream=None,
            flags: int = 0, kernel_events=None) -> torch.Tensor:
    """y = GBLA(q, k, v, a, r) on the GPU (o under NO_NORM); see include/gbla.h
    for the layouts and the ablation switches in ``flags``.
    ``kernel_events`` = (start, stop) torch.cuda.Events recorded just before
    the pass's first kernel and as its last kernel ends (gbla_forward_timed);
    each must have been recorded once before, so that its HIP event exists."""
    _check_inputs(q, k, v, gate_logits, out_gate, conv_w, norm_w, cu_seqlens)
    shape = make_shape(q, conv_w, eps, cu_seqlens, max_seqlen, flags)
    if workspace is None:
        workspace = alloc_workspace(shape, q.device)
    _check_ws(workspace, q.device, workspace_bytes(shape))
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    _check_out(out, q.shape, q.device)
    args = (ctypes.byref(shape), _ptr(q), _ptr(k), _ptr(v), _ptr(gate_logits), _ptr(out_gate),
            _ptr(conv_w), _ptr(norm_w), _ptr(cu_seqlens), _ptr(workspace), workspace.numel(),
            _ptr(out), _stream(stream))
    if kernel_events is None:
        _raise(load_library().gbla_forward(*args), "gbla_forward")
    else:
        handles = [e.cuda_event for e in kernel_events]
        if not all(handles):
            raise ValueError("kernel_events must have been recorded once before")
        _raise(load_library().gbla_forward_timed(*args, *handles), "gbla_forward_timed")
    return out


NOALLOC_SCRATCH_BYTES = 16 << 20  # GBLA_NOALLOC_SCRATCH_BYTES


def forward_noalloc(q, k, v, gate_logits, out_gate, conv_w, norm_w, eps: float = 1e-6,
                    cu_seqlens=None, max_seqlen=None, out=None, stream=None,
                    flags: int = 0) -> torch.Tensor:
    """gbla_forward_noalloc: the forward with the library's fixed device
    scratch instead of a workspace (for callers that cannot allocate; give
    ``out`` to allocate nothing here either)."""
    _check_inputs(q, k, v, gate_logits, out_gate, conv_w, norm_w, cu_seqlens)
    shape = make_shape(q, conv_w, eps, cu_seqlens, max_seqlen, flags)
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    _check_out(out, q.shape, q.device)
    st = load_library().gbla_forward_noalloc(
        ctypes.byref(shape), _ptr(q), _ptr(k), _ptr(v), _ptr(gate_logits), _ptr(out_gate),
        _ptr(conv_w), _ptr(norm_w), _ptr(cu_seqlens), _ptr(out), _stream(stream))
    _raise(st, "gbla_forward_noalloc")
    return out


def conv1d(q, k, v, conv_w, cu_seqlens=None, max_seqlen=None, stream=None, flags: int = 0
           ) -> Tuple[torch.Tensor, torch.Tensor, torch.Tensor]:
    """The Conv1D alone: fp32 q_t, k_t, v_t in the layout of q."""
    _check_inputs(q, k, v, None, None, conv_w, None, cu_seqlens)
    shape = make_shape(q, conv_w, 0.0, cu_seqlens, max_seqlen, flags)
    outs = [torch.empty(q.shape, dtype=torch.float32, device=q.device) for _ in range(3)]
    st = load_library().gbla_conv1d(ctypes.byref(shape), _ptr(q), _ptr(k), _ptr(v), _ptr(conv_w),
                                    _ptr(cu_seqlens), *[_ptr(o) for o in outs], _stream(stream))
    _raise(st, "gbla_conv1d")
    return tuple(outs)


def state(k, v, gate_logits, conv_w, cu_seqlens=None, max_seqlen=None, workspace=None,
          stream=None, flags: int = 0) -> Tuple[torch.Tensor, torch.Tensor]:
    """The normalised global state S [N,H,d,d] and z [N,H,d] (fp32)."""
    _check_inputs(k, k, v, gate_logits, None, conv_w, None, cu_seqlens)
    shape = make_shape(k, conv_w, 0.0, cu_seqlens, max_seqlen, flags)
    if workspace is None:
        workspace = alloc_workspace(shape, k.device)
    _check_ws(workspace, k.device, workspace_bytes(shape))
    N, H, d = shape.batch, shape.heads, shape.head_dim
    S = torch.empty((N, H, d, d), dtype=torch.float32, device=k.device)
    z = torch.empty((N, H, d), dtype=torch.float32, device=k.device)
    st = load_library().gbla_state(ctypes.byref(shape), _ptr(k), _ptr(v), _ptr(gate_logits),
                                   _ptr(conv_w), _ptr(cu_seqlens), _ptr(workspace),
                                   workspace.numel(), _ptr(S), _ptr(z), _stream(stream))
    _raise(st, "gbla_state")
    return S, z


def readout(q, out_gate, conv_w, norm_w, workspace, eps: float = 1e-6, cu_seqlens=None,
            max_seqlen=None, out=None, stream=None, flags: int = 0,
            kernel_events=None) -> torch.Tensor:
    """Readout + gated RMSNorm from the state a preceding state() call left in
    ``workspace``.  ``kernel_events`` = (start, stop) torch.cuda.Events that
    are recorded when the readout kernel begins and ends (gbla_readout_timed);
    each must have been recorded once before, so that its HIP event exists."""
    _check_inputs(q, None, None, None, out_gate, conv_w, norm_w, cu_seqlens)
    shape = make_shape(q, conv_w, eps, cu_seqlens, max_seqlen, flags)
    _check_ws(workspace, q.device, workspace_bytes(shape))
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=q.device)
    _check_out(out, q.shape, q.device)
    args = (ctypes.byref(shape), _ptr(q), _ptr(out_gate), _ptr(conv_w), _ptr(norm_w),
            _ptr(cu_seqlens), _ptr(workspace), workspace.numel(), _ptr(out), _stream(stream))
    if kernel_events is None:
        _raise(load_library().gbla_readout(*args), "gbla_readout")
    else:
        handles = [e.cuda_event for e in kernel_events]
        if not all(handles):
            raise ValueError("kernel_events must have been recorded once before")
        _raise(load_library().gbla_readout_timed(*args, *handles), "gbla_readout_timed")
    return out


def stream_ceiling(q, k, v, gate_logits, out_gate, out=None, stream=None) -> torch.Tensor:
    """Measurement aid (gbla_stream_ceiling): one launch that moves the
    forward's bytes for these bf16 tensors (q, k, v, out_gate read, one logit
    per token read, fp32 out written) with none of its arithmetic."""
    dev = q.device
    for t, nm in ((q, "q"), (k, "k"), (v, "v"), (out_gate, "out_gate")):
        _check(t, nm, torch.bfloat16, dev)
        if t.shape != q.shape:
            raise ValueError("%s must have the shape of q" % nm)
    _check(gate_logits, "gate_logits", torch.bfloat16, dev)
    if gate_logits.shape != q.shape[:-1]:
        raise ValueError("gate_logits must have shape %s" % (tuple(q.shape[:-1]),))
    if out is None:
        out = torch.empty(q.shape, dtype=torch.float32, device=dev)
    _check_out(out, q.shape, dev)
    d = q.shape[-1]
    st = load_library().gbla_stream_ceiling(_ptr(q), _ptr(k), _ptr(v), _ptr(gate_logits),
                                            _ptr(out_gate), q.numel() // d, d, _ptr(out),
                                            _stream(stream))
    _raise(st, "gbla_stream_ceiling")
    return out


def backward_workspace_bytes(shape: Shape) -> int:
    n = load_library().gbla_backward_workspace_bytes(ctypes.byref(shape))
    if n == 0:
        raise GblaError(1, "gbla_backward_workspace_bytes")
    return int(n)


def backward(q, k, v, gate_logits, out_gate, conv_w, norm_w, dy, eps: float = 1e-6,
             cu_seqlens=None, max_seqlen=None, workspace=None, stream=None,
             grads: Optional[dict] = None, flags: int = 0) -> dict:
    """Gradients of sum(forward(...) * dy) with respect to every input (fp32):
    a dict with dq, dk, dv, da (gate logits), dr (out gate), dconv_w, dgamma
    (norm weight), shaped like the inputs.  ``grads`` may hold preallocated
    fp32 outputs under those names; they are overwritten.  Under the ablation
    switches in ``flags`` the removed inputs may be None and their gradients
    are left out of the dict."""
    _check_inputs(q, k, v, gate_logits, out_gate, conv_w, norm_w, cu_seqlens)
    dev = q.device
    _check(dy, "dy", torch.float32, dev)
    if dy.shape != q.shape:
        raise ValueError("dy must have the shape of q")
    shape = make_shape(q, conv_w, eps, cu_seqlens, max_seqlen, flags)
    if workspace is None:
        workspace = torch.empty(backward_workspace_bytes(shape), dtype=torch.uint8, device=dev)
    _check_ws(workspace, dev, backward_workspace_bytes(shape))
    f32 = dict(dtype=torch.float32, device=dev)
    want = {n: q.shape for n in ("dq", "dk", "dv")}
    if not flags & NO_NORM:
        want.update(dr=q.shape, dgamma=norm_w.shape)
    if not flags & NO_GATE:
        want.update(da=q.shape[:-1])
    if not flags & NO_CONV:
        want.update(dconv_w=conv_w.shape)
    g = dict(grads or {})
    for n, shp in want.items():
        if n not in g:
            g[n] = torch.empty(shp, **f32)
        _check(g[n], n, torch.float32, dev)
        if g[n].shape != shp:
            raise ValueError("%s must have shape %s" % (n, tuple(shp)))
    st = load_library().gbla_backward(
        ctypes.byref(shape), _ptr(q), _ptr(k), _ptr(v), _ptr(gate_logits), _ptr(out_gate),
        _ptr(conv_w), _ptr(norm_w), _ptr(cu_seqlens), _ptr(dy), _ptr(workspace), workspace.numel(),
        _ptr(g["dq"]), _ptr(g["dk"]), _ptr(g["dv"]), _ptr(g.get("da")), _ptr(g.get("dr")),
        _ptr(g.get("dconv_w")), _ptr(g.get("dgamma")), _stream(stream))
    _raise(st, "gbla_backward")
    return g


# ---------------------------------------------------------------------------
# The full layer from the embeddings X.
# ---------------------------------------------------------------------------
def layer_shape(x, conv_x, heads: int, head_dim: int, eps: float, cu_seqlens=None,
                max_seqlen=None) -> LayerShape:
    if cu_seqlens is None:
        if x.dim() != 3:
            raise ValueError("dense x must be [B, L, d_model]")
        B, L, dm = x.shape
        batch, rows, msl = B, L, 0
    else:
        if x.dim() != 2:
            raise ValueError("ragged x must be [T, d_model]")
        rows, dm = x.shape
        batch = cu_seqlens.numel() - 1
        msl = int(max_seqlen) if max_seqlen is not None else rows
    if conv_x.dim() != 2 or conv_x.shape[0] != dm:
        raise ValueError("conv_x must be [d_model, W]")
    return LayerShape(batch, rows, dm, heads, head_dim, conv_x.shape[1], msl, _dtype_code(x),
                      float(eps))


def _check_layer(x, conv_x, w_proj, heads, head_dim, cu_seqlens):
    dev = x.device
    _check(x, "x", torch.bfloat16, dev)
    _check(conv_x, "conv_x", torch.float32, dev)
    _check(w_proj, "w_proj", torch.bfloat16, dev)
    if w_proj.shape != (heads * (4 * head_dim + 1), x.shape[-1]):
        raise ValueError("w_proj must be [H*(4*d+1), d_model]")
    if cu_seqlens is not None:
        _check(cu_seqlens, "cu_seqlens", torch.int32, dev)


def layer_project(x, conv_x, w_proj, heads: int, head_dim: int, cu_seqlens=None,
                  max_seqlen=None, workspace=None, stream=None) -> dict:
    """Conv1D on x and the stacked projections: bf16 q, k, v, r in the
    attention layout ([B,H,L,d] or [H,T,d]) and the gate logits a."""
    _check_layer(x, conv_x, w_proj, heads, head_dim, cu_seqlens)
    shape = layer_shape(x, conv_x, heads, head_dim, 0.0, cu_seqlens, max_seqlen)
    if workspace is None:
        workspace = torch.empty(layer_workspace_bytes(shape), dtype=torch.uint8, device=x.device)
    _check_ws(workspace, x.device, layer_workspace_bytes(shape))
    if cu_seqlens is None:
        act = (shape.batch, heads, shape.seqlen, head_dim)
    else:
        act = (heads, shape.seqlen, head_dim)
    out = {n: torch.empty(act, dtype=torch.bfloat16, device=x.device) for n in ("q", "k", "v", "r")}
    out["a"] = torch.empty(act[:-1], dtype=torch.bfloat16, device=x.device)
    st = load_library().gbla_layer_project(
        ctypes.byref(shape), _ptr(x), _ptr(conv_x), _ptr(w_proj), _ptr(cu_seqlens), _ptr(workspace),
        workspace.numel(), _ptr(out["q"]), _ptr(out["k"]), _ptr(out["v"]), _ptr(out["r"]),
        _ptr(out["a"]), _stream(stream))
    _raise(st, "gbla_layer_project")
    return out


def layer_workspace_bytes(shape: LayerShape) -> int:
    n = load_library().gbla_layer_workspace_bytes(ctypes.byref(shape))
    if n == 0:
        raise GblaError(1, "gbla_layer_workspace_bytes")
    return int(n)


def layer_forward(x, conv_x, w_proj, norm_w, eps: float = 1e-6, cu_seqlens=None,
                  max_seqlen=None, workspace=None, out=None, stream=None) -> torch.Tensor:
    """The whole layer from the embeddings x; y in the attention layout."""
    if norm_w.dim() != 2:
        raise ValueError("norm_w must be [H, d]")
    heads, head_dim = norm_w.shape
    _check_layer(x, conv_x, w_proj, heads, head_dim, cu_seqlens)
    _check(norm_w, "norm_w", torch.float32, x.device)
    shape = layer_shape(x, conv_x, heads, head_dim, eps, cu_seqlens, max_seqlen)
    if workspace is None:
        workspace = torch.empty(layer_workspace_bytes(shape), dtype=torch.uint8, device=x.device)
    _check_ws(workspace, x.device, layer_workspace_bytes(shape))
    act = ((shape.batch, heads, shape.seqlen, head_dim) if cu_seqlens is None
           else (heads, shape.seqlen, head_dim))
    if out is None:
        out = torch.empty(act, dtype=torch.float32, device=x.device)
    _check_out(out, act, x.device)
    st = load_library().gbla_layer_forward(
        ctypes.byref(shape), _ptr(x), _ptr(conv_x), _ptr(w_proj), _ptr(norm_w), _ptr(cu_seqlens),
        _ptr(workspace), workspace.numel(), _ptr(out), _stream(stream))
    _raise(st, "gbla_layer_forward")
    return out
