"""ctypes wrapper of the fp64 CPU oracle (``oracle/gbla_oracle.c``).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg
of the benchmark use it; the product path never imports it.

The oracle computes the GBLA forward pass of the paper (Section 2 and
Section 2.1) in fp64 with plain loops; see the header of ``gbla_oracle.c``
for the definition it follows, step by step.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gbla_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

DTYPE_CODES = {"f32": 0, "bf16": 1, "f64": 2}


def build(force: bool = True, out: Optional[str] = None, src: Optional[str] = None,
          extra_flags=()) -> str:
    """Compile the oracle with gcc (-O2, OpenMP, no fast-math)."""
    out = out or _LIB
    src = src or _SRC
    if force or not os.path.exists(out) or os.path.getmtime(out) < os.path.getmtime(src):
        tmp = out + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-Wall",
               *extra_flags, src, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, out)
    return out


class Oracle:
    def __init__(self, path: str):
        self.path = path
        lib = ctypes.CDLL(path)
        p = ctypes.c_void_p
        i32 = ctypes.c_int32
        lib.gbla_oracle_forward.argtypes = [i32, i32, i32, i32, i32, i32, p, ctypes.c_double,
                                            p, p, p, p, p, p, p,
                                            p, p, p, p, p, p, p, p, p, i32]
        lib.gbla_oracle_forward.restype = ctypes.c_int
        lib.gbla_oracle_phi.argtypes = [ctypes.c_double]
        lib.gbla_oracle_phi.restype = ctypes.c_double
        lib.gbla_oracle_max_threads.argtypes = []
        lib.gbla_oracle_max_threads.restype = i32
        self.lib = lib

    def phi(self, u: float) -> float:
        return self.lib.gbla_oracle_phi(float(u))

    def max_threads(self) -> int:
        return int(self.lib.gbla_oracle_max_threads())

    def forward(self, q, k, v, a, r, conv_w, gamma, *, nseq: int, heads: int, rows: int,
                d: int, W: int, dtype: str, eps: float, cu_seqlens=None,
                want=("y",), nthreads: int = 0) -> dict:
        """Run the oracle.

        ``q, k, v, r`` are ``[nseq, H, rows, d]`` (dense) or ``[H, T, d]``
        (ragged, ``cu_seqlens`` given); ``a`` the same without ``d``.  They may
        be float32, float64 or uint16 bf16 bit patterns (``dtype`` says which).
        ``want`` selects outputs among y, qt, kt, vt, g, S, z, o, oh."""
        code = DTYPE_CODES[dtype]
        np_dt = {"f32": np.float32, "bf16": np.uint16, "f64": np.float64}[dtype]
        acts = [np.ascontiguousarray(x, dtype=np_dt) for x in (q, k, v, a, r)]
        act_elems = heads * rows * d if cu_seqlens is not None else nseq * heads * rows * d
        gate_elems = act_elems // d
        for x, n_el in zip(acts, (act_elems,) * 3 + (gate_elems, act_elems)):
            if x.size != n_el:
                raise ValueError("activation size %d, expected %d" % (x.size, n_el))
        cw = np.ascontiguousarray(conv_w, dtype=np.float64)
        gm = np.ascontiguousarray(gamma, dtype=np.float64)
        if cw.size != 3 * heads * d * W or gm.size != heads * d:
            raise ValueError("conv_w / gamma size mismatch")
        offs = None
        if cu_seqlens is not None:
            offs = np.ascontiguousarray(cu_seqlens, dtype=np.int32)
            if offs.size != nseq + 1:
                raise ValueError("cu_seqlens must have nseq + 1 entries")
        act_shape = (heads, rows, d) if cu_seqlens is not None else (nseq, heads, rows, d)
        gate_shape = act_shape[:-1]
        shapes = {"y": act_shape, "qt": act_shape, "kt": act_shape, "vt": act_shape,
                  "g": gate_shape, "S": (nseq, heads, d, d), "z": (nseq, heads, d),
                  "o": act_shape, "oh": act_shape}
        outs = {}
        for name in want:
            outs[name] = np.zeros(shapes[name], dtype=np.float64)

        def ptr(x):
            return None if x is None else x.ctypes.data_as(ctypes.c_void_p)

        rc = self.lib.gbla_oracle_forward(
            nseq, heads, rows, d, W, code, ptr(offs), float(eps),
            *[ptr(x) for x in acts], ptr(cw), ptr(gm),
            *[ptr(outs.get(n)) for n in ("y", "qt", "kt", "vt", "g", "S", "z", "o", "oh")],
            int(nthreads))
        if rc != 0:
            raise ValueError("oracle rejected its arguments (code %d)" % rc)
        return outs

    def forward_inputs(self, inp, want=("y",), nthreads: int = 0, gate: bool = True,
                       conv: bool = True, norm: bool = True) -> dict:
        """Run the oracle on a ``paper_2606_07317_amd.inputs.Inputs`` batch.

        ``gate``, ``conv`` and ``norm`` are the ablations of the paper's
        ablation table (Section 3, "Ablation", Table 4), expressed through the inputs
        so that the arithmetic above is unchanged:
          gate=False  constant logits, hence uniform gates g_j = 1/n
                      (Section 2.1, key gating; the softmax of a constant);
          conv=False  identity taps (tap W-1 = 1, the others 0), so qt = q;
          norm=False  the un-normalised readout o is returned as "y".
        All three off is bidirectional linear attention, Eq. (1)."""
        w = inp.workload
        a, conv_w = inp.a, inp.conv_w
        if not gate:
            a = np.zeros_like(inp.a)
        if not conv:
            conv_w = np.zeros_like(inp.conv_w)
            conv_w[..., w.conv_width - 1] = 1.0
        req = tuple(("o" if (x == "y" and not norm) else x) for x in want)
        res = self.forward(inp.q, inp.k, inp.v, a, inp.r, conv_w, inp.gamma,
                           nseq=inp.nseq, heads=w.heads, rows=inp.rows if inp.cu_seqlens is not None else w.seqlen,
                           d=w.head_dim, W=w.conv_width, dtype=w.dtype, eps=inp.eps,
                           cu_seqlens=inp.cu_seqlens, want=tuple(dict.fromkeys(req)), nthreads=nthreads)
        if not norm and "y" in want:
            res["y"] = res["o"]
        return res


_default: Optional[Oracle] = None


def load(path: Optional[str] = None) -> Oracle:
    """Load the oracle library, compiling it first if it is missing or stale.

    ``GBLA_ORACLE_LIB`` in the environment names another build of the same
    source to load instead (the sanitizer test runs the pins on one built
    with AddressSanitizer and UBSan)."""
    global _default
    if path is not None:
        return Oracle(path)
    if _default is None:
        alt = os.environ.get("GBLA_ORACLE_LIB")
        if alt:
            _default = Oracle(alt)
        else:
            build(force=False)
            _default = Oracle(_LIB)
    return _default
