"""Host-side checks of the C ABI: the library loads, exports every function
include/gbla.h declares, sizes its workspace from the shape alone, and
rejects bad arguments before anything reaches the GPU.  No kernel runs here:
every call below fails validation on the host."""
import ctypes

import pytest

from paper_2606_07317_amd import gbla

ALIGNED = 0x10000          # fake, 256-byte aligned device addresses; never dereferenced
MIS = 0x10008


@pytest.fixture(scope="module")
def lib():
    return gbla.load_library()


def shape(**kw):
    base = dict(batch=1, heads=8, seqlen=32768, head_dim=64, conv_width=4, max_seqlen=0,
                dtype=gbla.GBLA_BF16, eps=1e-6)
    base.update(kw)
    return gbla.Shape(**base)


def test_exports_every_declared_function(lib):
    names = gbla.declared_functions()
    assert {"gbla_forward", "gbla_workspace_bytes", "gbla_conv1d", "gbla_state",
            "gbla_readout", "gbla_readout_timed", "gbla_forward_timed", "gbla_status_string",
            "gbla_backward",
            "gbla_backward_workspace_bytes", "gbla_layer_workspace_bytes", "gbla_layer_project",
            "gbla_layer_forward"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    for code, name in gbla.STATUS_NAMES.items():
        assert lib.gbla_status_string(code).decode() == name
    assert lib.gbla_status_string(99).decode() == "GBLA_ERR_UNKNOWN"


def test_workspace_bytes(lib):
    ws = lib.gbla_workspace_bytes(ctypes.byref(shape()))
    assert ws > 0 and ws % 256 == 0
    # partial records: at least one (d*d + d + 2)-float record per chunk of every head
    assert ws >= 8 * 32 * (64 * 64 + 66) * 4
    # stays modest: under 32 MiB for the n=32768, H=8, d=64 workload
    assert ws < 32 << 20
    ragged = lib.gbla_workspace_bytes(ctypes.byref(shape(batch=64, seqlen=190000, head_dim=128,
                                                         max_seqlen=32768)))
    assert ragged > 0
    for bad in (shape(head_dim=48), shape(conv_width=5), shape(conv_width=0), shape(dtype=7),
                shape(heads=0), shape(batch=0), shape(seqlen=-1), shape(eps=-1.0),
                shape(eps=float("inf"))):
        assert lib.gbla_workspace_bytes(ctypes.byref(bad)) == 0
    assert lib.gbla_workspace_bytes(None) == 0


def _forward(lib, s, ws_bytes=None, **ptrs):
    p = dict(q=ALIGNED, k=ALIGNED, v=ALIGNED, a=ALIGNED, r=ALIGNED, w=ALIGNED, g=ALIGNED,
             cu=None, ws=ALIGNED, out=ALIGNED)
    p.update(ptrs)
    if ws_bytes is None:
        ws_bytes = lib.gbla_workspace_bytes(ctypes.byref(s))
    return lib.gbla_forward(ctypes.byref(s), p["q"], p["k"], p["v"], p["a"], p["r"], p["w"], p["g"],
                            p["cu"], p["ws"], ws_bytes, p["out"], None)


def test_forward_rejects_before_launch(lib):
    s = shape()
    assert _forward(lib, s, q=None) == 1
    assert _forward(lib, s, out=None) == 1
    assert _forward(lib, s, a=None) == 1
    assert _forward(lib, s, q=MIS) == 3
    assert _forward(lib, s, out=ALIGNED + 4) == 3
    assert _forward(lib, s, w=ALIGNED + 4) == 3
    assert _forward(lib, s, a=ALIGNED + 1) == 3        # bf16 logits need 2-byte alignment
    assert _forward(lib, s, ws=ALIGNED + 16) == 3      # workspace needs 256 bytes
    assert _forward(lib, s, ws=None) == 4
    assert _forward(lib, s, ws_bytes=1024) == 4
    assert _forward(lib, shape(head_dim=96)) == 2
    assert _forward(lib, shape(conv_width=8)) == 2
    assert _forward(lib, shape(dtype=3)) == 2
    assert _forward(lib, shape(eps=float("nan"))) == 1
    assert _forward(lib, shape(heads=-2)) == 1
    assert lib.gbla_forward(None, ALIGNED, ALIGNED, ALIGNED, ALIGNED, ALIGNED, ALIGNED, ALIGNED,
                            None, ALIGNED, 1 << 30, ALIGNED, None) == 1


def test_ragged_requires_nonnegative_bound(lib):
    s = shape(batch=4, seqlen=100, max_seqlen=-1)
    assert _forward(lib, s, cu=ALIGNED) == 1


def test_other_entry_points_reject_before_launch(lib):
    s = shape()
    P = ALIGNED
    assert lib.gbla_conv1d(ctypes.byref(s), P, P, None, P, None, P, P, P, None) == 1
    assert lib.gbla_conv1d(ctypes.byref(shape(head_dim=16)), P, P, P, P, None, P, P, P, None) == 2
    assert lib.gbla_state(ctypes.byref(s), P, P, P, P, None, P, 16, P, P, None) == 4
    assert lib.gbla_state(ctypes.byref(s), P, P, P, P, None, P + 8, 1 << 40, P, P, None) == 3
    assert lib.gbla_readout(ctypes.byref(s), None, P, P, P, None, P, 1 << 40, P, None) == 1
    assert lib.gbla_readout(ctypes.byref(s), P, P, P, P, None, None, 1 << 40, P, None) == 4
    assert lib.gbla_readout(ctypes.byref(s), P, P, P, P, None, P, 0, P, None) == 4
    # the timed variant checks its arguments as gbla_readout does, events aside
    assert lib.gbla_readout_timed(ctypes.byref(s), None, P, P, P, None, P, 1 << 40, P, None, P, P) == 1
    assert lib.gbla_readout_timed(ctypes.byref(s), P, P, P, P, None, P, 0, P, None, None, None) == 4


def test_ablation_switches_validation(lib):
    """Inputs removed by a switch may be NULL (or anything) and are not
    checked; unknown flag bits are rejected.  Each call still fails on the
    missing workspace, which is checked after the inputs, so nothing launches."""
    assert lib.gbla_workspace_bytes(ctypes.byref(shape(flags=8))) == 0
    assert _forward(lib, shape(flags=8)) == 1
    assert _forward(lib, shape(), a=None, ws=None) == 1
    assert _forward(lib, shape(flags=gbla.NO_GATE), a=None, ws=None) == 4
    assert _forward(lib, shape(), w=None, ws=None) == 1
    assert _forward(lib, shape(flags=gbla.NO_CONV), w=None, ws=None) == 4
    assert _forward(lib, shape(flags=gbla.NO_CONV), w=ALIGNED + 4, ws=None) == 4
    assert _forward(lib, shape(), r=None, g=None, ws=None) == 1
    assert _forward(lib, shape(flags=gbla.NO_NORM), r=None, g=None, ws=None) == 4
    assert _forward(lib, shape(flags=gbla.BLA), a=None, r=None, w=None, g=None, ws=None) == 4
    # the switches do not relax the inputs they leave in use
    assert _forward(lib, shape(flags=gbla.BLA), q=None, ws=None) == 1
    P = ALIGNED
    assert lib.gbla_state(ctypes.byref(shape(flags=gbla.NO_GATE)), P, P, None, P, None,
                          None, 0, P, P, None) == 4
    assert lib.gbla_readout(ctypes.byref(shape(flags=gbla.NO_NORM)), P, None, P, None, None,
                            None, 0, P, None) == 4
    assert lib.gbla_conv1d(ctypes.byref(shape(flags=gbla.NO_CONV, head_dim=16)), P, P, P, None,
                           None, P, P, P, None) == 2


def _backward(lib, s, ws_bytes=None, **ptrs):
    P = ALIGNED
    p = dict(q=P, k=P, v=P, a=P, r=P, w=P, g=P, cu=None, dy=P, ws=P, dq=P, dk=P, dv=P, da=P,
             dr=P, dw=P, dg=P)
    p.update(ptrs)
    if ws_bytes is None:
        ws_bytes = lib.gbla_backward_workspace_bytes(ctypes.byref(s))
    return lib.gbla_backward(ctypes.byref(s), p["q"], p["k"], p["v"], p["a"], p["r"], p["w"],
                             p["g"], p["cu"], p["dy"], p["ws"], ws_bytes, p["dq"], p["dk"],
                             p["dv"], p["da"], p["dr"], p["dw"], p["dg"], None)


def test_backward_workspace_and_validation(lib):
    s = shape()
    bwd = lib.gbla_backward_workspace_bytes(ctypes.byref(s))
    # three fp32 activation-sized buffers at least
    assert bwd % 256 == 0 and bwd >= 3 * 8 * 32768 * 64 * 4
    assert lib.gbla_backward_workspace_bytes(ctypes.byref(shape(head_dim=48))) == 0
    assert lib.gbla_backward_workspace_bytes(None) == 0
    for name in ("q", "k", "v", "a", "r", "w", "g", "dy", "dq", "dk", "dv", "da", "dr", "dw",
                 "dg"):
        assert _backward(lib, s, **{name: None}) == 1, name
    for name in ("q", "dy", "dq", "dr", "w", "g", "dw", "dg"):
        assert _backward(lib, s, **{name: MIS}) == 3, name
    assert _backward(lib, s, da=ALIGNED + 2) == 3      # fp32 gradient of the logits
    assert _backward(lib, s, ws=None) == 4
    assert _backward(lib, s, ws=ALIGNED + 64) == 3
    assert _backward(lib, s, ws_bytes=3 * 8 * 32768 * 64 * 4) == 4   # the dq~, dk~, dv~ buffers alone
    assert _backward(lib, shape(head_dim=16)) == 2
    assert _backward(lib, shape(flags=8)) == 1
    # switches: removed inputs and their gradients may be NULL (each call still
    # stops at the missing workspace, which is checked last)
    assert _backward(lib, shape(flags=gbla.NO_GATE), a=None, da=None, ws=None) == 4
    assert _backward(lib, shape(flags=gbla.NO_CONV), w=None, dw=None, ws=None) == 4
    assert _backward(lib, shape(flags=gbla.NO_NORM), r=None, g=None, dr=None, dg=None, ws=None) == 4
    assert _backward(lib, shape(flags=gbla.BLA), a=None, da=None, w=None, dw=None, r=None, g=None,
                     dr=None, dg=None, ws=None) == 4
    assert _backward(lib, shape(flags=gbla.BLA), q=None, ws=None) == 1
    assert _backward(lib, shape(flags=gbla.NO_NORM), dw=None, ws=None) == 1


def lshape(**kw):
    base = dict(batch=8, seqlen=2048, d_model=1024, heads=16, head_dim=64, conv_width=4,
                max_seqlen=0, dtype=gbla.GBLA_BF16, eps=1e-6)
    base.update(kw)
    return gbla.LayerShape(**base)


def test_layer_validation(lib):
    s = lshape()
    ws = lib.gbla_layer_workspace_bytes(ctypes.byref(s))
    # Xt, four bf16 projections of every token and head, the gate logits and the core
    assert ws >= 8 * 2048 * 1024 * 2 + 4 * 8 * 2048 * 16 * 64 * 2 + 8 * 2048 * 16 * 2
    for bad in (lshape(dtype=gbla.GBLA_F32), lshape(d_model=100), lshape(d_model=0),
                lshape(head_dim=48), lshape(conv_width=5), lshape(heads=0), lshape(seqlen=-1)):
        assert lib.gbla_layer_workspace_bytes(ctypes.byref(bad)) == 0
    P = ALIGNED
    fwd = lambda s, **kw: lib.gbla_layer_forward(
        ctypes.byref(s), kw.get("x", P), kw.get("c", P), kw.get("w", P), kw.get("g", P), None,
        kw.get("ws", P), kw.get("wsb", ws), kw.get("out", P), None)
    assert fwd(s, x=None) == 1
    assert fwd(s, w=MIS) == 3
    assert fwd(s, out=None) == 1
    assert fwd(s, ws=None) == 4
    assert fwd(s, ws=P + 64) == 3
    assert fwd(s, wsb=1024) == 4
    assert fwd(lshape(dtype=gbla.GBLA_F32)) == 2
    assert fwd(lshape(d_model=96)) == 2
    proj = lambda s, **kw: lib.gbla_layer_project(
        ctypes.byref(s), kw.get("x", P), kw.get("c", P), kw.get("w", P), None, kw.get("ws", P),
        kw.get("wsb", ws), kw.get("q", P), P, P, P, kw.get("a", P), None)
    assert proj(s, q=None) == 1
    assert proj(s, a=None) == 1
    assert proj(s, a=P + 1) == 3
    assert proj(s, x=MIS) == 3
    assert proj(s, ws=None) == 4
    assert proj(s, wsb=1024) == 4
    assert proj(lshape(head_dim=16)) == 2


def test_stream_ceiling_rejects_before_launch(lib):
    """The measurement aid checks its arguments on the host like the entry
    points of the method (codes of include/gbla.h); a zero count launches
    nothing."""
    def call(q=ALIGNED, k=ALIGNED, v=ALIGNED, a=ALIGNED, r=ALIGNED, n=1024, d=64, out=ALIGNED):
        return lib.gbla_stream_ceiling(q, k, v, a, r, n, d, out, None)
    assert call(q=None) == 1
    assert call(out=None) == 1
    assert call(n=-1) == 1
    assert call(d=48) == 2
    assert call(k=MIS) == 3
    assert call(out=ALIGNED + 8) == 3
    assert call(a=ALIGNED + 1) == 3
    assert call(n=0) == 0


def test_noalloc_refuses_shapes_beyond_its_scratch(lib):
    """gbla_forward_noalloc checks the shape, then refuses any whose scratch
    exceeds GBLA_NOALLOC_SCRATCH_BYTES, before any HIP call (so these run
    without a GPU)."""
    big = shape(batch=16, heads=16, seqlen=32768)  # far above 16 MiB of partials
    assert lib.gbla_workspace_bytes(ctypes.byref(big)) > gbla.NOALLOC_SCRATCH_BYTES
    args = [ALIGNED] * 7 + [None, ALIGNED, None]  # q..norm_w, cu_seqlens, out, stream
    assert lib.gbla_forward_noalloc(ctypes.byref(big), *args) == 4
    assert lib.gbla_forward_noalloc(ctypes.byref(shape(head_dim=96)), *args) == 2
    assert lib.gbla_forward_noalloc(ctypes.byref(shape(eps=-1.0)), *args) == 1
    assert lib.gbla_forward_noalloc(None, *args) == 1
