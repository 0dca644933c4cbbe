// gbla_api.cpp -- the C ABI of libgbla.so: argument validation and the
// entry points declared in include/gbla.h (the plans live in gbla_plan.cpp
// and gbla_ext_plan.cpp).
//
// Every check runs on the host before anything is enqueued, and none of them
// touches the HIP runtime, so a rejected call has no side effect.
#include <math.h>
#include <stdint.h>

#include "gbla.h"
#include "gbla_ext.h"
#include "gbla_plan.h"

using gbla::Plan;

namespace {

gbla_status check_ws(const Plan& p, const void* ws, size_t ws_bytes) {
  if (!ws) return GBLA_ERR_WORKSPACE;
  if (!gbla::aligned(ws, 256)) return GBLA_ERR_MISALIGNED;
  if (ws_bytes < p.total_bytes) return GBLA_ERR_WORKSPACE;
  return GBLA_OK;
}

size_t elem_bytes(const Plan& p) { return p.dtype == GBLA_BF16 ? 2 : 4; }

gbla_status check_acts(const Plan& p, std::initializer_list<const void*> acts) {
  for (const void* a : acts) {
    if (!a) return GBLA_ERR_INVALID_ARGUMENT;
    if (!gbla::aligned(a, 16)) return GBLA_ERR_MISALIGNED;
  }
  (void)p;
  return GBLA_OK;
}

gbla_status check_logits(const Plan& p, const void* a) {
  if (!a) return GBLA_ERR_INVALID_ARGUMENT;
  if (!gbla::aligned(a, elem_bytes(p))) return GBLA_ERR_MISALIGNED;
  return GBLA_OK;
}

// An input that the switch `flag` removes: NULL inside the library when the
// switch is on (whatever the caller passed), otherwise the caller's pointer.
template <typename Ptr>
Ptr unless(const Plan& p, uint32_t flag, Ptr ptr) {
  return (p.flags & flag) ? nullptr : ptr;
}

// Checks of the inputs that are in use: present and aligned.
gbla_status check_used(std::initializer_list<const void*> used) {
  for (const void* a : used) {
    if (!a) return GBLA_ERR_INVALID_ARGUMENT;
    if (!gbla::aligned(a, 16)) return GBLA_ERR_MISALIGNED;
  }
  return GBLA_OK;
}

#define GBLA_TRY(expr)                  \
  do {                                  \
    gbla_status _st = (expr);           \
    if (_st != GBLA_OK) return _st;     \
  } while (0)

}  // namespace


namespace gbla {

gbla_status forward_entry(const gbla_shape* shape, const void* q, const void* k, const void* v,
                          const void* gate_logits, const void* out_gate, const float* conv_w,
                          const float* norm_w, const int32_t* cu_seqlens, void* workspace,
                          size_t workspace_bytes, float* out, void* stream, KernelEvents ev) {
  Plan p;
  GBLA_TRY(gbla::make_plan(shape, cu_seqlens != nullptr, &p));
  gate_logits = unless(p, GBLA_NO_GATE, gate_logits);
  conv_w = unless(p, GBLA_NO_CONV, conv_w);
  out_gate = unless(p, GBLA_NO_NORM, out_gate);
  norm_w = unless(p, GBLA_NO_NORM, norm_w);
  GBLA_TRY(check_acts(p, {q, k, v, out}));
  if (!(p.flags & GBLA_NO_CONV)) GBLA_TRY(check_used({conv_w}));
  if (!(p.flags & GBLA_NO_NORM)) GBLA_TRY(check_used({out_gate, norm_w}));
  if (!(p.flags & GBLA_NO_GATE)) GBLA_TRY(check_logits(p, gate_logits));
  GBLA_TRY(check_ws(p, workspace, workspace_bytes));
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (ev.start && hipEventRecord(ev.start, st) != hipSuccess) return GBLA_ERR_HIP;
  GBLA_TRY(gbla::launch_state(p, k, v, gate_logits, conv_w, cu_seqlens, workspace, nullptr,
                              nullptr, nullptr, st));
  gbla::KernelEvents last;
  last.stop = ev.stop;
  return gbla::launch_readout(p, q, out_gate, conv_w, norm_w, cu_seqlens, workspace, out, st,
                              last);
}

}  // namespace gbla

extern "C" {

size_t gbla_workspace_bytes(const gbla_shape* shape) {
  // The shape alone does not say whether cu_seqlens will be given, so the
  // size covers both readings (dense: B*n tokens, ragged: T = seqlen tokens)
  // -- each one the library accepts; 0 only when it accepts neither.
  size_t most = 0;
  for (int ragged = 0; ragged < 2; ++ragged) {
    Plan p;
    if (gbla::make_plan(shape, ragged != 0, &p) == GBLA_OK && p.total_bytes > most)
      most = p.total_bytes;
  }
  return most;
}


gbla_status gbla_forward(const gbla_shape* shape, const void* q, const void* k, const void* v,
                         const void* gate_logits, const void* out_gate, const float* conv_w,
                         const float* norm_w, const int32_t* cu_seqlens, void* workspace,
                         size_t workspace_bytes, float* out, void* stream) {
  return gbla::forward_entry(shape, q, k, v, gate_logits, out_gate, conv_w, norm_w, cu_seqlens,
                             workspace, workspace_bytes, out, stream, {});
}

gbla_status gbla_forward_timed(const gbla_shape* shape, const void* q, const void* k,
                               const void* v, const void* gate_logits, const void* out_gate,
                               const float* conv_w, const float* norm_w,
                               const int32_t* cu_seqlens, void* workspace,
                               size_t workspace_bytes, float* out, void* stream,
                               void* start_event, void* stop_event) {
  gbla::KernelEvents ev;
  ev.start = static_cast<hipEvent_t>(start_event);
  ev.stop = static_cast<hipEvent_t>(stop_event);
  return gbla::forward_entry(shape, q, k, v, gate_logits, out_gate, conv_w, norm_w, cu_seqlens,
                             workspace, workspace_bytes, out, stream, ev);
}

gbla_status gbla_conv1d(const gbla_shape* shape, const void* q, const void* k, const void* v,
                        const float* conv_w, const int32_t* cu_seqlens, float* q_t, float* k_t,
                        float* v_t, void* stream) {
  Plan p;
  GBLA_TRY(gbla::make_plan(shape, cu_seqlens != nullptr, &p));
  conv_w = unless(p, GBLA_NO_CONV, conv_w);
  GBLA_TRY(check_acts(p, {q, k, v, q_t, k_t, v_t}));
  if (!(p.flags & GBLA_NO_CONV)) GBLA_TRY(check_used({conv_w}));
  return gbla::launch_conv(p, q, k, v, conv_w, cu_seqlens, q_t, k_t, v_t,
                           static_cast<hipStream_t>(stream));
}

gbla_status gbla_state(const gbla_shape* shape, const void* k, const void* v,
                       const void* gate_logits, const float* conv_w, const int32_t* cu_seqlens,
                       void* workspace, size_t workspace_bytes, float* S, float* z,
                       void* stream) {
  Plan p;
  GBLA_TRY(gbla::make_plan(shape, cu_seqlens != nullptr, &p));
  gate_logits = unless(p, GBLA_NO_GATE, gate_logits);
  conv_w = unless(p, GBLA_NO_CONV, conv_w);
  GBLA_TRY(check_acts(p, {k, v, S, z}));
  if (!(p.flags & GBLA_NO_CONV)) GBLA_TRY(check_used({conv_w}));
  if (!(p.flags & GBLA_NO_GATE)) GBLA_TRY(check_logits(p, gate_logits));
  GBLA_TRY(check_ws(p, workspace, workspace_bytes));
  return gbla::launch_state(p, k, v, gate_logits, conv_w, cu_seqlens, workspace, S, z, nullptr,
                            static_cast<hipStream_t>(stream));
}

static gbla_status readout_entry(const gbla_shape* shape, const void* q, const void* out_gate,
                                 const float* conv_w, const float* norm_w,
                                 const int32_t* cu_seqlens, void* workspace,
                                 size_t workspace_bytes, float* out, void* stream,
                                 gbla::KernelEvents ev) {
  Plan p;
  GBLA_TRY(gbla::make_plan(shape, cu_seqlens != nullptr, &p));
  conv_w = unless(p, GBLA_NO_CONV, conv_w);
  out_gate = unless(p, GBLA_NO_NORM, out_gate);
  norm_w = unless(p, GBLA_NO_NORM, norm_w);
  GBLA_TRY(check_acts(p, {q, out}));
  if (!(p.flags & GBLA_NO_CONV)) GBLA_TRY(check_used({conv_w}));
  if (!(p.flags & GBLA_NO_NORM)) GBLA_TRY(check_used({out_gate, norm_w}));
  GBLA_TRY(check_ws(p, workspace, workspace_bytes));
  return gbla::launch_readout(p, q, out_gate, conv_w, norm_w, cu_seqlens, workspace, out,
                              static_cast<hipStream_t>(stream), ev);
}

gbla_status gbla_readout(const gbla_shape* shape, const void* q, const void* out_gate,
                         const float* conv_w, const float* norm_w, const int32_t* cu_seqlens,
                         void* workspace, size_t workspace_bytes, float* out, void* stream) {
  return readout_entry(shape, q, out_gate, conv_w, norm_w, cu_seqlens, workspace,
                       workspace_bytes, out, stream, {});
}

gbla_status gbla_readout_timed(const gbla_shape* shape, const void* q, const void* out_gate,
                               const float* conv_w, const float* norm_w,
                               const int32_t* cu_seqlens, void* workspace,
                               size_t workspace_bytes, float* out, void* stream,
                               void* start_event, void* stop_event) {
  gbla::KernelEvents ev;
  ev.start = static_cast<hipEvent_t>(start_event);
  ev.stop = static_cast<hipEvent_t>(stop_event);
  return readout_entry(shape, q, out_gate, conv_w, norm_w, cu_seqlens, workspace,
                       workspace_bytes, out, stream, ev);
}

size_t gbla_backward_workspace_bytes(const gbla_shape* shape) {
  // as gbla_workspace_bytes: the larger of the accepted readings
  size_t most = 0;
  for (int ragged = 0; ragged < 2; ++ragged) {
    Plan p0, p;
    if (gbla::make_plan(shape, ragged != 0, &p0) != GBLA_OK) continue;
    if (gbla::backward_plan(p0, &p) != GBLA_OK) continue;
    const size_t bytes = gbla::make_bwd_layout(p).total_bytes;
    if (bytes > most) most = bytes;
  }
  return most;
}

gbla_status gbla_backward(const gbla_shape* shape, const void* q, const void* k, const void* v,
                          const void* gate_logits, const void* out_gate, const float* conv_w,
                          const float* norm_w, const int32_t* cu_seqlens, const float* dy,
                          void* workspace, size_t workspace_bytes, float* dq, float* dk,
                          float* dv, float* d_gate_logits, float* d_out_gate, float* d_conv_w,
                          float* d_norm_w, void* stream) {
  Plan p0, p;
  GBLA_TRY(gbla::make_plan(shape, cu_seqlens != nullptr, &p0));
  GBLA_TRY(gbla::backward_plan(p0, &p));
  // inputs a switch removes, and their gradients, are NULL inside the library
  gate_logits = unless(p, GBLA_NO_GATE, gate_logits);
  d_gate_logits = unless(p, GBLA_NO_GATE, d_gate_logits);
  conv_w = unless(p, GBLA_NO_CONV, conv_w);
  d_conv_w = unless(p, GBLA_NO_CONV, d_conv_w);
  out_gate = unless(p, GBLA_NO_NORM, out_gate);
  norm_w = unless(p, GBLA_NO_NORM, norm_w);
  d_out_gate = unless(p, GBLA_NO_NORM, d_out_gate);
  d_norm_w = unless(p, GBLA_NO_NORM, d_norm_w);
  GBLA_TRY(check_acts(p, {q, k, v, dy, dq, dk, dv}));
  if (!(p.flags & GBLA_NO_CONV)) GBLA_TRY(check_used({conv_w, d_conv_w}));
  if (!(p.flags & GBLA_NO_NORM)) GBLA_TRY(check_used({out_gate, norm_w, d_out_gate, d_norm_w}));
  if (!(p.flags & GBLA_NO_GATE)) {
    GBLA_TRY(check_logits(p, gate_logits));
    if (!d_gate_logits) return GBLA_ERR_INVALID_ARGUMENT;
    if (!gbla::aligned(d_gate_logits, sizeof(float))) return GBLA_ERR_MISALIGNED;
  }
  const gbla::BwdLayout L = gbla::make_bwd_layout(p);
  if (!workspace) return GBLA_ERR_WORKSPACE;
  if (!gbla::aligned(workspace, 256)) return GBLA_ERR_MISALIGNED;
  if (workspace_bytes < L.total_bytes) return GBLA_ERR_WORKSPACE;
  return gbla::launch_backward(p, L, q, k, v, gate_logits, out_gate, conv_w, norm_w, cu_seqlens,
                               dy, workspace, dq, dk, dv, d_gate_logits, d_out_gate, d_conv_w,
                               d_norm_w, static_cast<hipStream_t>(stream));
}

size_t gbla_layer_workspace_bytes(const gbla_layer_shape* shape) {
  // as gbla_workspace_bytes: the larger of the accepted readings
  size_t most = 0;
  for (int ragged = 0; ragged < 2; ++ragged) {
    gbla::LayerPlan L;
    if (gbla::make_layer_plan(shape, ragged != 0, &L) == GBLA_OK && L.total_bytes > most)
      most = L.total_bytes;
  }
  return most;
}

gbla_status gbla_layer_project(const gbla_layer_shape* shape, const void* x, const float* conv_x,
                               const void* w_proj, const int32_t* cu_seqlens, void* workspace,
                               size_t workspace_bytes, void* q, void* k, void* v, void* r,
                               void* a, void* stream) {
  gbla::LayerPlan L;
  GBLA_TRY(gbla::make_layer_plan(shape, cu_seqlens != nullptr, &L));
  GBLA_TRY(check_used({x, conv_x, w_proj, q, k, v, r}));
  if (!a) return GBLA_ERR_INVALID_ARGUMENT;
  if (!gbla::aligned(a, 2)) return GBLA_ERR_MISALIGNED;
  if (!workspace) return GBLA_ERR_WORKSPACE;
  if (!gbla::aligned(workspace, 256)) return GBLA_ERR_MISALIGNED;
  if (workspace_bytes < L.total_bytes) return GBLA_ERR_WORKSPACE;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  return gbla::launch_project(L, x, conv_x, w_proj, cu_seqlens, ws + L.off_xt, q, k, v, r, a,
                              static_cast<hipStream_t>(stream));
}

gbla_status gbla_layer_forward(const gbla_layer_shape* shape, const void* x, const float* conv_x,
                               const void* w_proj, const float* norm_w,
                               const int32_t* cu_seqlens, void* workspace, size_t workspace_bytes,
                               float* out, void* stream) {
  gbla::LayerPlan L;
  GBLA_TRY(gbla::make_layer_plan(shape, cu_seqlens != nullptr, &L));
  GBLA_TRY(check_used({x, conv_x, w_proj, norm_w, out}));
  if (!workspace) return GBLA_ERR_WORKSPACE;
  if (!gbla::aligned(workspace, 256)) return GBLA_ERR_MISALIGNED;
  if (workspace_bytes < L.total_bytes) return GBLA_ERR_WORKSPACE;
  unsigned char* ws = static_cast<unsigned char*>(workspace);
  hipStream_t st = static_cast<hipStream_t>(stream);
  void *q = ws + L.off_q, *k = ws + L.off_k, *v = ws + L.off_v, *r = ws + L.off_r, *a = ws + L.off_a;
  GBLA_TRY(gbla::launch_project(L, x, conv_x, w_proj, cu_seqlens, ws + L.off_xt, q, k, v, r, a, st));
  void* cws = ws + L.off_core;
  GBLA_TRY(gbla::launch_state(L.core, k, v, a, nullptr, cu_seqlens, cws, nullptr, nullptr,
                              nullptr, st));
  return gbla::launch_readout(L.core, q, r, nullptr, norm_w, cu_seqlens, cws, out, st);
}

const char* gbla_status_string(gbla_status status) {
  switch (status) {
    case GBLA_OK: return "GBLA_OK";
    case GBLA_ERR_INVALID_ARGUMENT: return "GBLA_ERR_INVALID_ARGUMENT";
    case GBLA_ERR_UNSUPPORTED: return "GBLA_ERR_UNSUPPORTED";
    case GBLA_ERR_MISALIGNED: return "GBLA_ERR_MISALIGNED";
    case GBLA_ERR_WORKSPACE: return "GBLA_ERR_WORKSPACE";
    case GBLA_ERR_HIP: return "GBLA_ERR_HIP";
  }
  return "GBLA_ERR_UNKNOWN";
}

}  // extern "C"
