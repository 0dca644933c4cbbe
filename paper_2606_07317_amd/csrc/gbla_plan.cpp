// gbla_plan.cpp -- the launch plan of the attention pass: split sizes and the
// workspace layout, a function of the shape alone.
#include <math.h>
#include <stdint.h>

#include "gbla.h"
#include "gbla_plan.h"

namespace gbla {
namespace {

constexpr int kMaxGridY = 65535;
constexpr int64_t kMaxGridX = 2147483647LL;
constexpr int kReadoutTile = 512;

int64_t next_pow2(int64_t x) {
  int64_t p = 1;
  while (p < x) p <<= 1;
  return p;
}

}  // namespace

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

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

}  // namespace gbla
