// gbla_state128.hip -- the state reduction of the bf16 forward pass at head
// dim 128 (gfx950).
//
// One workgroup (8 waves) reduces one chunk of tokens of one (sequence, head)
// to a partial record [S_p | z_p | m_p | l_p] (Section 2.1, key-gating item:
// the matrix form K^T V and K^T 1 with K = g (.) phi(K)):
//     S_p = sum_j w_j phi(kt_j) vt_j^T,  z_p = sum_j w_j phi(kt_j),
//     w_j = exp(a_j - m_p),  m_p = max_j a_j,  l_p = sum_j w_j.
//
// At d = 128 the bound is the vector ALU, not memory: phi(kt) costs about
// fifteen vector instructions per (token, key channel) and the 514 bytes of a
// token-head leave about 40 CU cycles for it at full HBM rate.  So every
// (token, key channel) is formed exactly once per workgroup: wave w owns key
// channels 16w .. 16w + 15 and all 128 value channels, and the waves share
// the token rows through one LDS ring instead of each loading its own.
//
//   * Staging: each step of 32 tokens (8 KB of keys, 8 KB of values) is
//     loaded once by the whole workgroup, one 16-byte vector per thread and
//     tensor, three steps ahead in registers, and written to a ring of four
//     slots one step ahead; one barrier per step.  In a slot the channels
//     are grouped by 16 (one MFMA tile), 32 rows per group, groups padded by
//     64 bytes, and row bit 2 is flipped when row bit 3 is set: the sixteen
//     rows of a transposed read then fall on distinct bank groups, and every
//     address of the loop is a per-lane base plus an immediate.
//   * Keys: ds_read_b64_tr_b16 hands each lane four consecutive tokens of one
//     channel; three reads give the twelve-row window of its eight tokens, so
//     the key conv, phi and the gate weight are applied in registers and the
//     result is the A operand of v_mfma_f32_16x16x32_bf16 (16 key channels x
//     32 tokens).
//   * Values: the conv is linear and per channel, so it is moved past the
//     token sum (taps u_tau, tap 3 on the current token):
//         S_p[c][e] = sum_tau u_tau[e] M_tau[c][e],
//         M_tau     = sum_j w_j phi(kt_j) v_{j-3+tau}^T,
//     each M_tau an MFMA accumulator fed with raw bf16 value rows at a shift
//     of tau - 3 tokens (odd shifts take one alignbit per dword).  v enters
//     the products exactly and the taps are applied once, in fp32, at the
//     end.  z_p is summed in fp32 from the unrounded gated keys.
//   * Overlap: waves w and w + 4 share a SIMD.  Waves 0-3 form A(i) and then
//     multiply it; waves 4-7 first multiply A(i - 1) (its value rows are
//     still in the ring) and then form A(i).  After each barrier one wave of
//     every SIMD is in its vector phase while the other is in its MFMA phase.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "gbla_device.h"
#include "gbla_plan.h"

namespace gbla {
namespace {

struct S128 {
  static constexpr int D = 128;
  static constexpr int kWaves = 8;
  static constexpr int kNT = 64 * kWaves;
  static constexpr int kStep = 32;                          // tokens per step (MFMA K)
  static constexpr int kStepBytes = kStep * 2 * D;          // one step of rows in memory
  static constexpr int kGroups = D / 16;                    // 16-channel groups
  static constexpr int kGroupBytes = kStep * 32 + 64;       // 32 rows of 32 bytes + pad
  static constexpr int kHalf = kGroups * kGroupBytes;       // keys (or values) of a slot
  static constexpr int kSlots = 4;
  static constexpr int kKeys = 0;
  static constexpr int kVals = kSlots * kHalf;
  static constexpr int kRing = 2 * kSlots * kHalf;
  static constexpr int kMaxChunk = 2048;
  static constexpr int kLds = kRing + kMaxChunk * 4;        // + gate weights of the chunk
};
static_assert(S128::kWaves == S128::kGroups, "one wave per 16 key channels");
static_assert((S128::kSlots - 1) * S128::kHalf + S128::kHalf < 65536,
              "offsets from a per-lane base must fit the 16-bit LDS immediate");

// Byte offset of (row r, channel c) in a key or value half-slot.
__device__ __forceinline__ int hoff(int r, int c) {
  const int rp = r ^ (((r >> 3) & 1) << 2);
  return (c >> 4) * S128::kGroupBytes + rp * 32 + (c & 15) * 2;
}

__device__ __forceinline__ u32x2_t tr_read2(const unsigned char* p) {
  return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                         (__attribute__((address_space(3))) i16x4_t*)(p)));
}

__device__ __forceinline__ void ring_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

__global__ void __launch_bounds__(S128::kNT, 1)
state128_kernel(Plan P, const uint16_t* __restrict__ kin, const uint16_t* __restrict__ vin,
                const uint16_t* __restrict__ ain, const float* __restrict__ conv_w,
                const int32_t* __restrict__ cu, float* __restrict__ partials) {
  using C = S128;
  constexpr int D = C::D;
  __shared__ __attribute__((aligned(16))) unsigned char lds[C::kLds];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool late = wave >= 4;  // multiplies one step behind
  const int h = blockIdx.y, g = blockIdx.x;
  int s, chunk;
  if (!unit_of<C::kNT>(P, cu, P.chunk, P.chunks_per_seq, g, &s, &chunk)) return;
  s = __builtin_amdgcn_readfirstlane(s);
  chunk = __builtin_amdgcn_readfirstlane(chunk);
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int64_t t0 = (int64_t)chunk * P.chunk;
  const int64_t t1 = min(len, t0 + (int64_t)P.chunk);
  const int w0 = (int)t0;  // slice-relative first token
  const int ntok = t1 > t0 ? (int)(t1 - t0) : 0;
  const int nsteps = (ntok + C::kStep - 1) / C::kStep;
  float* rec = partials + ((size_t)h * P.units + g) * P.rec_floats;

  const __amdgpu_buffer_rsrc_t rk = make_rsrc(kin + base_row * D, (uint32_t)(len * 2 * D));
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vin + base_row * D, (uint32_t)(len * 2 * D));
  // no logits (uniform gates): an empty range, so every logit reads as 0
  const __amdgpu_buffer_rsrc_t ra =
      ain ? make_rsrc(ain + base_row, (uint32_t)(len * 2)) : make_rsrc(kin, 0u);

  // Lane roles: token group gq (tokens 8 gq .. 8 gq + 7 of a step) and
  // column j (key channel 16 wave + j of A, value channel 16 nb + j of B).
  const int gq = lane >> 4, j = lane & 15;
  constexpr float kLog2e = 1.4426950408889634f, kLn2 = 0.6931471805599453f;
  float wk[4];
  load_taps4(conv_w, P.heads, h, 1, D, P.W, 16 * wave + j, wk);

  // Gate logits of the chunk (every wave reads all of them; tokens outside
  // the chunk read as zero and get -inf added).
  uint32_t abits[C::kMaxChunk / 64];
  float amask[C::kMaxChunk / 64];
#pragma unroll
  for (int i = 0; i < C::kMaxChunk / 64; ++i) {
    const int tok = lane + 64 * i;
    const bool valid = tok < ntok;
    abits[i] = __builtin_amdgcn_raw_buffer_load_b16(ra, valid ? (uint32_t)(w0 + tok) * 2u : kOutOfRange,
                                                    0, 0);
    amask[i] = valid ? 0.0f : -INFINITY;
  }

  // Staging: thread -> (row, 16-byte chunk) of a step.
  const int srow = tid >> 4, sch = tid & 15;
  const uint32_t goff = (uint32_t)(((w0 + srow) * D + sch * 8) * 2);
  const int soff = hoff(srow, sch * 8);
  u32x4_t bk[2], bv[2];
  auto issue = [&](int step, int buf) {
    const uint32_t o = step < nsteps ? goff + (uint32_t)step * C::kStepBytes : kOutOfRange;
    bk[buf] = __builtin_amdgcn_raw_buffer_load_b128(rk, o, 0, 0);
    bv[buf] = __builtin_amdgcn_raw_buffer_load_b128(rv, o, 0, 0);
  };
  auto commit = [&](auto slot_c, int buf) {
    constexpr int sl = decltype(slot_c)::value;
    *reinterpret_cast<u32x4_t*>(lds + C::kKeys + sl * C::kHalf + soff) = bk[buf];
    *reinterpret_cast<u32x4_t*>(lds + C::kVals + sl * C::kHalf + soff) = bv[buf];
  };
  // Rows 28..31 of the step before the chunk: the conv window of its first
  // tokens (zero before the sequence start, where the offset wraps out of range).
  const uint32_t poff = srow >= C::kStep - 4 && nsteps > 0 ? goff - (uint32_t)C::kStepBytes : kOutOfRange;
  const u32x4_t pk = __builtin_amdgcn_raw_buffer_load_b128(rk, poff, 0, 0);
  const u32x4_t pv = __builtin_amdgcn_raw_buffer_load_b128(rv, poff, 0, 0);
  issue(0, 0);
  issue(1, 1);
  __builtin_amdgcn_sched_barrier(0);

  // ---- gate weights: m, w_j = exp(a_j - m), l; wave w stores entries
  // 256 w .. 256 w + 255 (every wave computes all of them) ----
  float av[C::kMaxChunk / 64];
  float mloc = -INFINITY;
#pragma unroll
  for (int i = 0; i < C::kMaxChunk / 64; ++i) {
    av[i] = __uint_as_float(abits[i] << 16) + amask[i];
    mloc = fmaxf(mloc, av[i]);
  }
  const float mw = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                                              __builtin_bit_cast(int, wave_max(mloc))));
  float* wts = reinterpret_cast<float*>(lds + C::kRing);
  float lsum = 0.0f;
#pragma unroll
  for (int i = 0; i < C::kMaxChunk / 64; ++i) {
    const float w = av[i] == -INFINITY ? 0.0f : __expf(av[i] - mw);
    if (i / 4 == wave) wts[lane + 64 * i] = w;
    lsum += w;
  }
  const float lw = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                                              __builtin_bit_cast(int, wave_sum(lsum))));
#pragma unroll
  for (int tap = 0; tap < 4; ++tap) wk[tap] *= kLog2e;

  // ---- per-lane read bases.  Read r of a window hands the lane rows
  // 8 gq - 4 + 4 r + [0, 4) of its channel; rows before 0 are rows 28..31 of
  // the previous slot.  Base [0] serves windows in slots 1..3 (offset by
  // (slot - 1) halves), base [1] the window in slot 0. ----
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
  const int row0 = 8 * gq - 4 + (j >> 2);
  const int kcol = 16 * wave + 4 * (j & 3), vcol = 4 * (j & 3);
  const int o0 = hoff(row0 & (C::kStep - 1), 0);
  const unsigned char* kb0 = lds + C::kKeys + o0 + kcol / 16 * C::kGroupBytes + (kcol & 15) * 2 +
                             (gq == 0 ? 0 : C::kHalf);
  const unsigned char* kb1 = kb0 + (gq == 0 ? (C::kSlots - 1) * C::kHalf : -C::kHalf);
  const unsigned char* kr1 = lds + C::kKeys + hoff(row0 + 4, kcol);
  const unsigned char* kr2 = lds + C::kKeys + hoff(row0 + 8, kcol);
  const unsigned char* vb0 = lds + C::kVals + o0 + vcol * 2 + (gq == 0 ? 0 : C::kHalf);
  const unsigned char* vb1 = vb0 + (gq == 0 ? (C::kSlots - 1) * C::kHalf : -C::kHalf);
  const unsigned char* vr1 = lds + C::kVals + hoff(row0 + 4, vcol);
  const unsigned char* vr2 = lds + C::kVals + hoff(row0 + 8, vcol);
  const float* wl = wts + 8 * gq;

  f32x4_t acc[4][C::kGroups];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int b = 0; b < C::kGroups; ++b) acc[u][b] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  float zacc = 0.0f;
  u32x4_t A = {0u, 0u, 0u, 0u};

  // Reads of a step's key window (slot sl) and gate weights; issued ahead of
  // the work that uses them, so that LDS latency hides behind other work.
  struct KeyIn {
    u32x2_t t[3];
    f32x4_t wa, wb;
  };
  auto kread = [&](auto slot_c, int i) {
    constexpr int sl = decltype(slot_c)::value;
    KeyIn r;
    r.t[0] = tr_read2(sl == 0 ? kb1 : kb0 + (sl - 1) * C::kHalf);
    r.t[1] = tr_read2(kr1 + sl * C::kHalf);
    r.t[2] = tr_read2(kr2 + sl * C::kHalf);
    r.wa = *reinterpret_cast<const f32x4_t*>(wl + C::kStep * i);
    r.wb = *reinterpret_cast<const f32x4_t*>(wl + C::kStep * i + 4);
    return r;
  };
  // A = w phi(kt) of key channel 16 wave + j over the lane's eight tokens.
  auto kcompute = [&](const KeyIn& r) {
    const float wj[8] = {r.wa[0], r.wa[1], r.wa[2], r.wa[3], r.wb[0], r.wb[1], r.wb[2], r.wb[3]};
    float xk[12];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      xk[4 * q + 0] = bf16_lo(r.t[q][0]); xk[4 * q + 1] = bf16_hi(r.t[q][0]);
      xk[4 * q + 2] = bf16_lo(r.t[q][1]); xk[4 * q + 3] = bf16_hi(r.t[q][1]);
    }
    float kw[8];
#pragma unroll
    for (int o = 0; o < 8; ++o) {
      float kc = wk[0] * xk[o + 1];  // kt * log2(e)
#pragma unroll
      for (int tap = 1; tap < 4; ++tap) kc = fmaf(wk[tap], xk[o + 1 + tap], kc);
      // phi(x) = max(x, 0) + exp(min(x, 0)) = ln2 max(x', 0) + 2^min(x', 0)
      const float ph = fmaf(kLn2, fmaxf(kc, 0.0f), __builtin_amdgcn_exp2f(fminf(kc, 0.0f)));
      kw[o] = wj[o] * ph;
      zacc += kw[o];
    }
#pragma unroll
    for (int p = 0; p < 4; ++p) A[p] = pack_bf16x2(kw[2 * p], kw[2 * p + 1]);
  };

  // The twelve-row value window of channel group nb of the step in slot sl.
  struct ValIn {
    u32x2_t t[3];
  };
  auto vread = [&](auto slot_c, int nb) {
    constexpr int sl = decltype(slot_c)::value;
    const int go = nb * C::kGroupBytes;
    ValIn r;
    r.t[0] = tr_read2((sl == 0 ? vb1 : vb0 + (sl - 1) * C::kHalf) + go);
    r.t[1] = tr_read2(vr1 + sl * C::kHalf + go);
    r.t[2] = tr_read2(vr2 + sl * C::kHalf + go);
    return r;
  };
  // The products of A with the value rows of the step in slot sl:
  // B[tau] = rows of the lane's eight tokens shifted by tau - 3.  The window
  // of group nb + 1 is read while group nb is multiplied; `first` holds
  // group 0's, read by the caller.
  auto values = [&](auto slot_c, const ValIn& first) {
    const bf16x8_t a = __builtin_bit_cast(bf16x8_t, A);
    ValIn cur = first;
#pragma unroll
    for (int nb = 0; nb < C::kGroups; ++nb) {
      ValIn nxt;
      if (nb + 1 < C::kGroups) nxt = vread(slot_c, nb + 1);
      const uint32_t pw[6] = {cur.t[0][0], cur.t[0][1], cur.t[1][0],
                              cur.t[1][1], cur.t[2][0], cur.t[2][1]};
      u32x4_t B[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        B[0][m] = __builtin_amdgcn_alignbit(pw[m + 1], pw[m], 16);
        B[1][m] = pw[m + 1];
        B[2][m] = __builtin_amdgcn_alignbit(pw[m + 2], pw[m + 1], 16);
        B[3][m] = pw[m + 2];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        acc[u][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, __builtin_bit_cast(bf16x8_t, B[u]),
                                                             acc[u][nb], 0, 0, 0);
      if (nb + 1 < C::kGroups) cur = nxt;
    }
  };

  // One step i (slot sl = i mod 4): barrier, stage step i + 1 into its slot
  // (the slot of step i - 3) and refill its registers with step i + 3, then
  // compute.  The loop runs whole turns of four steps; steps past the chunk
  // see only zero rows and zero gate weights and add nothing, so there is no
  // branch in it.
  auto step = [&](auto late_c, auto slot_c, int i) {
    constexpr int sl = decltype(slot_c)::value;
    constexpr int nx = (sl + 1) & 3, buf = (sl + 1) & 1;
    ring_barrier();
    commit(std::integral_constant<int, nx>{}, buf);
    issue(i + 3, buf);
    if constexpr (!decltype(late_c)::value) {
      const KeyIn kr = kread(slot_c, i);
      const ValIn v0 = vread(slot_c, 0);
      kcompute(kr);
      values(slot_c, v0);
    } else {
      constexpr auto prev = std::integral_constant<int, (sl + 3) & 3>{};
      const ValIn v0 = vread(prev, 0);
      const KeyIn kr = kread(slot_c, i);
      values(prev, v0);
      kcompute(kr);
    }
  };
  auto run = [&](auto late_c) {
    const int nturns = (nsteps + 3) / 4;
    for (int it = 0; it < nturns; ++it) {
      const int i = 4 * it;
      step(late_c, I0{}, i);
      step(late_c, I1{}, i + 1);
      step(late_c, I2{}, i + 2);
      step(late_c, I3{}, i + 3);
    }
    // the late waves' last product: A of step 4 nturns - 1, rows in slot 3
    if constexpr (decltype(late_c)::value) values(I3{}, vread(I3{}, 0));
  };

  if (nsteps > 0) {
    // Before the first step: the window rows before the chunk (slot 3, rows
    // 28..31; the other rows of slot 3 get zeros) and step 0 (slot 0).  Slot 2
    // is cleared: the late waves' first product reads it (with A = 0).
    *reinterpret_cast<u32x4_t*>(lds + C::kKeys + 3 * C::kHalf + soff) = pk;
    *reinterpret_cast<u32x4_t*>(lds + C::kVals + 3 * C::kHalf + soff) = pv;
    const u32x4_t zero4 = {0u, 0u, 0u, 0u};
    *reinterpret_cast<u32x4_t*>(lds + C::kKeys + 2 * C::kHalf + soff) = zero4;
    *reinterpret_cast<u32x4_t*>(lds + C::kVals + 2 * C::kHalf + soff) = zero4;
    commit(I0{}, 0);
    issue(2, 0);
    if (late)
      run(std::true_type{});
    else
      run(std::false_type{});
  }

  // ---- the record: S[c][e] = sum_tau u_tau[e] M_tau[c][e] for key channels
  // c = 16 wave + 4 gq + q and value channels e = 16 nb + j ----
#pragma unroll
  for (int nb = 0; nb < C::kGroups; ++nb) {
    float u[4];
    load_taps4(conv_w, P.heads, h, 2, D, P.W, 16 * nb + j, u);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      float sv = u[0] * acc[0][nb][q];
#pragma unroll
      for (int t = 1; t < 4; ++t) sv = fmaf(u[t], acc[t][nb][q], sv);
      rec[(16 * wave + 4 * gq + q) * D + 16 * nb + j] = sv;
    }
  }
  zacc += __shfl_xor(zacc, 16);
  zacc += __shfl_xor(zacc, 32);
  if (gq == 0) rec[D * D + 16 * wave + j] = zacc;
  if (wave == 0 && lane == 0) {
    rec[D * D + D] = mw;
    rec[D * D + D + 1] = lw;
  }
}

}  // namespace

gbla_status launch_state128(const Plan& p, const void* k, const void* v, const void* a,
                            const float* conv_w, const int32_t* cu, float* partials, hipStream_t st) {
  if (p.d != S128::D || p.chunk > S128::kMaxChunk || p.chunk % S128::kStep != 0)
    return GBLA_ERR_UNSUPPORTED;  // the plan never asks for this
  const dim3 grid(p.units, p.heads);
  hipLaunchKernelGGL(state128_kernel, grid, dim3(S128::kNT), 0, st, p, (const uint16_t*)k,
                     (const uint16_t*)v, (const uint16_t*)a, conv_w, cu, partials);
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}

}  // namespace gbla
