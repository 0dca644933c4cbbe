// gbla_api.cpp -- the C ABI of libgbla.so: argument validation, the launch
// plan and the entry points declared in include/gbla.h.
//
// Every check runs on the host before anything is enqueued, and none of them
// touches the HIP runtime, so a rejected call has no side effect.
#include <math.h>
#include <stdint.h>

#include "gbla.h"
#include "gbla_plan.h"

namespace gbla {
namespace {

constexpr int kMaxGridY = 65535;
constexpr int64_t kMaxGridX = 2147483647LL;
constexpr int kReadoutTile = 512;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int64_t next_pow2(int64_t x) {
  int64_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

}  // namespace

gbla_status make_plan(const gbla_shape* s, bool ragged, Plan* p) {
  if (!s || !p) return GBLA_ERR_INVALID_ARGUMENT;
  if (s->batch < 1 || s->heads < 1 || s->seqlen < 0) return GBLA_ERR_INVALID_ARGUMENT;
  if (s->head_dim != 32 && s->head_dim != 64 && s->head_dim != 128) return GBLA_ERR_UNSUPPORTED;
  if (s->conv_width < 1 || s->conv_width > 4) return GBLA_ERR_UNSUPPORTED;
  if (s->dtype != GBLA_F32 && s->dtype != GBLA_BF16) return GBLA_ERR_UNSUPPORTED;
  if (!(s->eps >= 0.0f) || !isfinite(s->eps)) return GBLA_ERR_INVALID_ARGUMENT;
  if (ragged && s->max_seqlen < 0) return GBLA_ERR_INVALID_ARGUMENT;
  if (s->heads > kMaxGridY) return GBLA_ERR_UNSUPPORTED;
  if (s->flags & ~(uint32_t)GBLA_BLA) return GBLA_ERR_INVALID_ARGUMENT;

  Plan q{};
  q.nseq = s->batch;
  q.heads = s->heads;
  q.rows = s->seqlen;
  q.d = s->head_dim;
  q.W = s->conv_width;
  q.dtype = s->dtype;
  q.ragged = ragged ? 1 : 0;
  q.eps = s->eps;
  q.flags = s->flags;
  q.tokens = ragged ? (int64_t)s->seqlen : (int64_t)s->batch * s->seqlen;

  // Chunk of the state reduction: about one workgroup per CU over all heads,
  // a power of two between 256 and 2048 tokens.  Depends on the shape only.
  const int64_t work = q.tokens * q.heads;
  int64_t chunk = next_pow2((work + 255) / 256);
  if (chunk < 256) chunk = 256;
  if (chunk > 2048) chunk = 2048;
  q.chunk = (int32_t)chunk;
  q.rtile = kReadoutTile;

  // Upper bounds valid for both layouts: sum_s max(1, ceil(len_s / u)) <=
  // tokens / u + N.  The partial records are sized with this bound so the
  // workspace layout is the same for the dense and the ragged call.
  const int64_t units_cap = q.tokens / q.chunk + q.nseq;
  const int64_t runits_cap = q.tokens / q.rtile + q.nseq;
  if (units_cap > kMaxGridX || runits_cap > kMaxGridX) return GBLA_ERR_UNSUPPORTED;
  if (ragged) {
    q.chunks_per_seq = 0;
    q.rtiles_per_seq = 0;
    q.units = (int32_t)units_cap;
    q.runits = (int32_t)runits_cap;
  } else {
    int64_t cps = ((int64_t)q.rows + q.chunk - 1) / q.chunk;
    int64_t rps = ((int64_t)q.rows + q.rtile - 1) / q.rtile;
    if (cps < 1) cps = 1;
    if (rps < 1) rps = 1;
    q.chunks_per_seq = (int32_t)cps;
    q.rtiles_per_seq = (int32_t)rps;
    q.units = (int32_t)(cps * q.nseq);
    q.runits = (int32_t)(rps * q.nseq);
  }

  q.rec_floats = (int32_t)align_up((size_t)q.d * q.d + q.d + 2, 64);
  const size_t nmb = q.d / 16 + 1, nkb = q.d / 32;
  const size_t lane_bytes = q.dtype == GBLA_BF16 ? 16 : 32;
  q.frag_bytes = align_up(nmb * nkb * 64 * lane_bytes, 256);
  q.off_partials = 0;
  const size_t part_bytes = (size_t)units_cap * q.heads * q.rec_floats * sizeof(float);
  q.off_frags = align_up(q.off_partials + part_bytes, 256);
  q.total_bytes = align_up(q.off_frags + (size_t)q.nseq * q.heads * q.frag_bytes, 256);
  *p = q;
  return GBLA_OK;
}

Plan backward_plan(const Plan& p) {
  // Units of 512 tokens, whatever the forward's: long enough to amortise each
  // workgroup's set-up (A operands, the ordered wave sums), short enough for
  // two workgroups per CU at n = 32768, H = 8 (measured against 256 and 1024).
  Plan b = p;
  b.chunk = 512;
  if (p.ragged) {
    b.units = (int32_t)(b.tokens / b.chunk + b.nseq);
  } else {
    int64_t cps = ((int64_t)b.rows + b.chunk - 1) / b.chunk;
    if (cps < 1) cps = 1;
    b.chunks_per_seq = (int32_t)cps;
    b.units = (int32_t)(cps * b.nseq);
  }
  return b;
}

gbla_status make_layer_plan(const gbla_layer_shape* s, bool ragged, LayerPlan* p) {
  if (!s || !p) return GBLA_ERR_INVALID_ARGUMENT;
  if (s->batch < 1 || s->heads < 1 || s->seqlen < 0) return GBLA_ERR_INVALID_ARGUMENT;
  if (s->dtype != GBLA_BF16) return GBLA_ERR_UNSUPPORTED;
  if (s->d_model < 64 || s->d_model > 16384 || s->d_model % 64 != 0) return GBLA_ERR_UNSUPPORTED;
  if (s->conv_width < 1 || s->conv_width > 4) return GBLA_ERR_UNSUPPORTED;
  LayerPlan L{};
  L.nseq = s->batch;
  L.rows = s->seqlen;
  L.d_model = s->d_model;
  L.heads = s->heads;
  L.d = s->head_dim;
  L.W = s->conv_width;
  L.ragged = ragged ? 1 : 0;
  const int64_t tokens = ragged ? (int64_t)s->seqlen : (int64_t)s->batch * s->seqlen;
  const int64_t features = (int64_t)s->heads * (4 * (int64_t)s->head_dim + 1);
  // 32-bit buffer offsets over X and the weights
  if (tokens * s->d_model * 2 >= (int64_t(1) << 31)) return GBLA_ERR_UNSUPPORTED;
  if (features * s->d_model * 2 >= (int64_t(1) << 31)) return GBLA_ERR_UNSUPPORTED;
  L.tokens = (int32_t)tokens;
  L.features = (int32_t)features;
  gbla_shape cs{};
  cs.batch = s->batch;
  cs.heads = s->heads;
  cs.seqlen = s->seqlen;
  cs.head_dim = s->head_dim;
  cs.conv_width = 1;
  cs.max_seqlen = ragged ? s->max_seqlen : 0;
  cs.dtype = GBLA_BF16;
  cs.eps = s->eps;
  cs.flags = GBLA_NO_CONV;
  gbla_status st = make_plan(&cs, ragged, &L.core);
  if (st != GBLA_OK) return st;
  const size_t act = (size_t)tokens * s->heads * s->head_dim * 2;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, 256);
    return at;
  };
  L.off_xt = take((size_t)tokens * s->d_model * 2);
  L.off_q = take(act);
  L.off_k = take(act);
  L.off_v = take(act);
  L.off_r = take(act);
  L.off_a = take((size_t)tokens * s->heads * 2);
  L.off_core = take(L.core.total_bytes);
  L.total_bytes = off;
  *p = L;
  return GBLA_OK;
}

BwdLayout make_bwd_layout(const Plan& p) {
  BwdLayout L{};
  const size_t pairs = (size_t)p.nseq * p.heads, d = p.d, f = sizeof(float);
  const size_t unit_recs = (size_t)p.units * p.heads;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t at = off;
    off = align_up(off + bytes, 256);
    return at;
  };
  L.off_S = take(pairs * d * d * f);
  L.off_z = take(pairs * d * f);
  L.off_mz = take(pairs * 2 * f);
  L.off_dsp = take(unit_recs * p.rec_floats * f);
  L.off_dS = take(pairs * (d * d + d) * f);
  L.off_dgp = take(unit_recs * d * f);
  L.off_dxt = take(3 * (size_t)p.tokens * p.heads * d * f);
  L.off_dcp = take(unit_recs * 3 * d * 4 * f);
  L.total_bytes = off;
  return L;
}

}  // namespace gbla

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

extern "C" {

size_t gbla_workspace_bytes(const gbla_shape* shape) {
  // The shape alone does not say whether cu_seqlens will be given, so the
  // size covers both readings (dense: B*n tokens, ragged: T = seqlen tokens).
  Plan dense, ragged;
  if (gbla::make_plan(shape, false, &dense) != GBLA_OK) return 0;
  if (gbla::make_plan(shape, true, &ragged) != GBLA_OK) return 0;
  return dense.total_bytes > ragged.total_bytes ? dense.total_bytes : ragged.total_bytes;
}

gbla_status gbla_forward(const gbla_shape* shape, const void* q, const void* k, const void* v,
                         const void* gate_logits, const void* out_gate, const float* conv_w,
                         const float* norm_w, const int32_t* cu_seqlens, void* workspace,
                         size_t workspace_bytes, float* out, void* stream) {
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
  GBLA_TRY(gbla::launch_state(p, k, v, gate_logits, conv_w, cu_seqlens, workspace, nullptr,
                              nullptr, nullptr, st));
  return gbla::launch_readout(p, q, out_gate, conv_w, norm_w, cu_seqlens, workspace, out, st);
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

gbla_status gbla_readout(const gbla_shape* shape, const void* q, const void* out_gate,
                         const float* conv_w, const float* norm_w, const int32_t* cu_seqlens,
                         void* workspace, size_t workspace_bytes, float* out, void* stream) {
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
                              static_cast<hipStream_t>(stream));
}

size_t gbla_backward_workspace_bytes(const gbla_shape* shape) {
  Plan dense, ragged;
  if (gbla::make_plan(shape, false, &dense) != GBLA_OK) return 0;
  if (gbla::make_plan(shape, true, &ragged) != GBLA_OK) return 0;
  const size_t a = gbla::make_bwd_layout(gbla::backward_plan(dense)).total_bytes;
  const size_t b = gbla::make_bwd_layout(gbla::backward_plan(ragged)).total_bytes;
  return a > b ? a : b;
}

gbla_status gbla_backward(const gbla_shape* shape, const void* q, const void* k, const void* v,
                          const void* gate_logits, const void* out_gate, const float* conv_w,
                          const float* norm_w, const int32_t* cu_seqlens, const float* dy,
                          void* workspace, size_t workspace_bytes, float* dq, float* dk,
                          float* dv, float* d_gate_logits, float* d_out_gate, float* d_conv_w,
                          float* d_norm_w, void* stream) {
  Plan p0;
  GBLA_TRY(gbla::make_plan(shape, cu_seqlens != nullptr, &p0));
  if (p0.flags != 0) return GBLA_ERR_UNSUPPORTED;
  const Plan p = gbla::backward_plan(p0);
  GBLA_TRY(check_acts(p, {q, k, v, out_gate, dy, dq, dk, dv, d_out_gate}));
  GBLA_TRY(check_used({conv_w, norm_w, d_conv_w, d_norm_w}));
  GBLA_TRY(check_logits(p, gate_logits));
  if (!d_gate_logits) return GBLA_ERR_INVALID_ARGUMENT;
  if (!gbla::aligned(d_gate_logits, sizeof(float))) return GBLA_ERR_MISALIGNED;
  const gbla::BwdLayout L = gbla::make_bwd_layout(p);
  if (!workspace) return GBLA_ERR_WORKSPACE;
  if (!gbla::aligned(workspace, 256)) return GBLA_ERR_MISALIGNED;
  if (workspace_bytes < L.total_bytes) return GBLA_ERR_WORKSPACE;
  return gbla::launch_backward(p, L, q, k, v, gate_logits, out_gate, conv_w, norm_w, cu_seqlens,
                               dy, workspace, dq, dk, dv, d_gate_logits, d_out_gate, d_conv_w,
                               d_norm_w, static_cast<hipStream_t>(stream));
}

size_t gbla_layer_workspace_bytes(const gbla_layer_shape* shape) {
  gbla::LayerPlan dense, ragged;
  if (gbla::make_layer_plan(shape, false, &dense) != GBLA_OK) return 0;
  if (gbla::make_layer_plan(shape, true, &ragged) != GBLA_OK) return 0;
  return dense.total_bytes > ragged.total_bytes ? dense.total_bytes : ragged.total_bytes;
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
