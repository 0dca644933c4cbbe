// gbla_ext_plan.cpp -- plans of the backward pass and of the full layer.
#include <stdint.h>

#include "gbla.h"
#include "gbla_ext.h"

namespace gbla {

gbla_status backward_plan(const Plan& p, Plan* out) {
  // Units of 512 tokens, whatever the forward's: long enough to amortise each
  // workgroup's set-up (A operands, the ordered wave sums), short enough for
  // two workgroups per CU at n = 32768, H = 8 (measured against 256 and 1024).
  Plan b = p;
  b.chunk = 512;
  int64_t units;
  if (p.ragged) {
    units = b.tokens / b.chunk + b.nseq;
  } else {
    int64_t cps = ((int64_t)b.rows + b.chunk - 1) / b.chunk;
    if (cps < 1) cps = 1;
    b.chunks_per_seq = (int32_t)cps;
    units = cps * b.nseq;
  }
  if (units > 2147483647LL) return GBLA_ERR_UNSUPPORTED;  // the grid's x extent
  b.units = (int32_t)units;
  *out = b;
  return GBLA_OK;
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
