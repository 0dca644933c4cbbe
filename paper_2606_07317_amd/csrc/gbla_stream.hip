// gbla_stream.hip -- streaming kernels of the bf16 GBLA forward pass for
// head dims 32 and 64 (gfx950).
//
// state_stream_kernel: one workgroup reduces one chunk of tokens of one
// (sequence, head) to a partial state (Section 2.1, key-gating item, matrix
// form K^T V and K^T 1 with K = g (.) phi(K)):
//     S_p = sum_j w_j phi(kt_j) vt_j^T,  z_p = sum_j w_j phi(kt_j),
//     w_j = exp(a_j - m_p),  m_p = max_j a_j,  l_p = sum_j w_j.
// Each of the four waves owns a quarter of the chunk and never waits for the
// others until the final merge.  A wave streams its tokens 16 at a time:
// raw bf16 k and v rows are loaded two steps ahead into registers, written
// row-major into a per-wave LDS ring (16-byte chunks XOR-swizzled by row),
// and read back with ds_read_b64_tr_b16, which hands each lane four
// consecutive tokens of one channel.  Twelve tokens (three reads) give the
// lane the causal conv window of its eight tokens, so the conv, phi and the
// gate weight are applied in registers and the results are already the
// operands of v_mfma_f32_32x32x16_bf16: A = w phi(kt) (channel c, 8 tokens),
// B = vt as bf16 hi + bf16 lo (channel e, 8 tokens).
//
// readout_stream_kernel: see its own comment below.
//
// All global traffic of the hot loops goes through raw buffer descriptors
// that span one (sequence, head) slice: rows before the sequence start or
// past its end read as zero, stores past the tile end are dropped.  There
// are no branches around memory instructions, so the compiler's wait counts
// stay exact and the prefetched loads remain in flight.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "gbla_device.h"
#include "gbla_plan.h"

namespace gbla {
namespace {

__device__ __forceinline__ u32x4_t bload16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

__device__ __forceinline__ i16x4_t tr_read(const unsigned char* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) i16x4_t*)(p));
}

template <int D>
struct SS {
  static constexpr int kStep = 16;                     // tokens per MFMA K block
  static constexpr int kRowBytes = 2 * D;               // one bf16 row
  static constexpr int kChunks = kRowBytes / 16;        // 16-byte chunks per row
  static constexpr int kSlotBytes = kStep * kRowBytes;  // one step of one tensor
  static constexpr int kVec = kSlotBytes / (64 * 16);   // 16-byte vectors per lane per step
  static constexpr int kSlots = 4;                      // ring depth
  static constexpr int kRing = 2 * kSlots * kSlotBytes; // k and v rings of one wave
  static constexpr int kT = D / 32;                     // 32-wide MFMA tiles per side
  static constexpr int kWaves = 4;                      // waves per workgroup
  static constexpr int kNT = 64 * kWaves;
  static constexpr int kMaxQ = 512;                     // tokens per wave (chunk <= 2048)
  static constexpr int kWaveBytes = kRing > D * D * 4 ? kRing : D * D * 4;
  static constexpr int kLds = kWaves * kWaveBytes + kWaves * kMaxQ * 4;
};

// Byte offset of element e (a multiple of 4) of row r inside a slot, with the
// 16-byte chunks of each row XOR-swizzled by the row index.
template <int D>
__device__ __forceinline__ int swz(int r, int e) {
  using C = SS<D>;
  const int c = e >> 3, half = (e >> 2) & 1;
  return r * C::kRowBytes + ((c ^ (r & (C::kChunks - 1))) << 4) + (half << 3);
}

template <int D>
__global__ void __launch_bounds__(SS<D>::kNT, 1)
state_stream_kernel(Plan P, const uint16_t* __restrict__ kin, const uint16_t* __restrict__ vin,
                    const uint16_t* __restrict__ ain, const float* __restrict__ conv_w,
                    const int32_t* __restrict__ cu, float* __restrict__ partials) {
  using C = SS<D>;
  constexpr int kT = C::kT;
  __shared__ __attribute__((aligned(16))) unsigned char lds[C::kLds];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.y, g = blockIdx.x;
  int s, chunk;
  if (!unit_of<C::kNT>(P, cu, P.chunk, P.chunks_per_seq, g, &s, &chunk)) return;
  s = __builtin_amdgcn_readfirstlane(s);
  chunk = __builtin_amdgcn_readfirstlane(chunk);
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int64_t t0 = (int64_t)chunk * P.chunk;
  const int64_t t1 = min(len, t0 + (int64_t)P.chunk);
  float* rec = partials + ((size_t)h * P.units + g) * P.rec_floats;

  const int Q = P.chunk / C::kWaves;               // tokens per wave
  const int w0 = (int)(t0 + (int64_t)wave * Q);    // slice-relative token range
  const int w1 = (int)min(t1, (int64_t)w0 + Q);
  const int nsteps = w1 > w0 ? (w1 - w0 + C::kStep - 1) / C::kStep : 0;
  unsigned char* ring = lds + wave * C::kWaveBytes;  // [2 tensors][kSlots][slot]
  float* wbuf = reinterpret_cast<float*>(lds + C::kWaves * C::kWaveBytes) + wave * C::kMaxQ;

  const __amdgpu_buffer_rsrc_t rk = make_rsrc(kin + base_row * D, (uint32_t)(len * C::kRowBytes));
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vin + base_row * D, (uint32_t)(len * C::kRowBytes));
  const __amdgpu_buffer_rsrc_t ra = make_rsrc(ain + base_row, (uint32_t)(len * 2));

  // Loop-invariant global values first (taps, gate logits), so that the
  // waits for them precede every prefetch.
  float wk[kT][4], wvt[kT][4];
#pragma unroll
  for (int t = 0; t < kT; ++t) {
    load_taps4(conv_w, P.heads, h, 1, D, P.W, 32 * t + (lane & 31), wk[t]);
    load_taps4(conv_w, P.heads, h, 2, D, P.W, 32 * t + (lane & 31), wvt[t]);
  }
  uint32_t abits[C::kMaxQ / 64];
#pragma unroll
  for (int i = 0; i < C::kMaxQ / 64; ++i) {
    const int tok = w0 + lane + 64 * i;
    abits[i] = __builtin_amdgcn_raw_buffer_load_b16(ra, (uint32_t)tok * 2u, 0, 0);
  }

  // ---- register-staged loads of one step (rows w0 + 16*step + [0, 16)) ----
  u32x4_t stage[2][2][C::kVec];  // [in-flight buffer][tensor][vector]
  auto issue = [&](int step, int buf, int first_row) {
#pragma unroll
    for (int x = 0; x < C::kVec; ++x) {
      const int u = x * 64 + lane;
      const int row = u / C::kChunks, ch = u % C::kChunks;
      const int tok = w0 + step * C::kStep + row;
      const uint32_t off = row >= first_row ? (uint32_t)(tok * D + ch * 8) * 2u : kOutOfRange;
      stage[buf][0][x] = bload16(rk, off);
      stage[buf][1][x] = bload16(rv, off);
    }
  };
  auto commit = [&](int step, int buf) {
    const int slot = (step + C::kSlots) % C::kSlots;
#pragma unroll
    for (int x = 0; x < C::kVec; ++x) {
      const int u = x * 64 + lane;
      const int row = u / C::kChunks, ch = u % C::kChunks;
      const int off = row * C::kRowBytes + ((ch ^ (row & (C::kChunks - 1))) << 4);
#pragma unroll
      for (int tn = 0; tn < 2; ++tn)
        *reinterpret_cast<u32x4_t*>(ring + (tn * C::kSlots + slot) * C::kSlotBytes + off) =
            stage[buf][tn][x];
    }
  };

  // Only rows 12..15 of the step before the wave's first token are needed
  // (the conv window); the others are masked off.
  issue(-1, 1, nsteps > 0 ? C::kStep - 4 : C::kStep);
  issue(0, 0, nsteps > 0 ? 0 : C::kStep);

  // ---- gate weights of the wave's tokens: m_w, w_j = exp(a_j - m_w), l_w ----
  float av[C::kMaxQ / 64];
  float mloc = -INFINITY;
#pragma unroll
  for (int i = 0; i < C::kMaxQ / 64; ++i) {
    const int tok = w0 + lane + 64 * i;
    av[i] = (64 * i < Q && tok < w1) ? __uint_as_float(abits[i] << 16) : -INFINITY;
    mloc = fmaxf(mloc, av[i]);
  }
  const float mw = wave_max(mloc);
  float lsum = 0.0f;
#pragma unroll
  for (int i = 0; i < C::kMaxQ / 64; ++i) {
    if (64 * i < Q) {
      const float wv = av[i] == -INFINITY ? 0.0f : __expf(av[i] - mw);
      wbuf[lane + 64 * i] = wv;
      lsum += wv;
    }
  }
  const float lw = wave_sum(lsum);

  f32x16_t acc[kT][kT];
#pragma unroll
  for (int a = 0; a < kT; ++a)
#pragma unroll
    for (int b = 0; b < kT; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[a][b][i] = 0.0f;
  float zacc[kT];
#pragma unroll
  for (int t = 0; t < kT; ++t) zacc[t] = 0.0f;

  commit(-1, 1);
  issue(1, 1, nsteps > 1 ? 0 : C::kStep);
  commit(0, 0);
  issue(2, 0, nsteps > 2 ? 0 : C::kStep);

  // Lane roles for the transposed reads and the MFMA operands.
  const int half = lane >> 5;             // token half of the 16-token step
  const int grp_ch = 16 * ((lane >> 4) & 1);
  const int j = lane & 15;
  const int src_row = j >> 2, src_ch = 4 * (j & 3);

  auto step_body = [&](int i, auto nb) {
    constexpr int kNext = decltype(nb)::value;  // staging buffer of step i+1
    const unsigned char* kcur = ring + (0 * C::kSlots + i % C::kSlots) * C::kSlotBytes;
    const unsigned char* kprv = ring + (0 * C::kSlots + (i + C::kSlots - 1) % C::kSlots) * C::kSlotBytes;
    const unsigned char* vcur = ring + (1 * C::kSlots + i % C::kSlots) * C::kSlotBytes;
    const unsigned char* vprv = ring + (1 * C::kSlots + (i + C::kSlots - 1) % C::kSlots) * C::kSlotBytes;
    // gate weights of the lane's eight tokens
    const f32x4_t wa = *reinterpret_cast<const f32x4_t*>(wbuf + 16 * i + 8 * half);
    const f32x4_t wb = *reinterpret_cast<const f32x4_t*>(wbuf + 16 * i + 8 * half + 4);
    const float wj[8] = {wa[0], wa[1], wa[2], wa[3], wb[0], wb[1], wb[2], wb[3]};

    u32x4_t A[kT], Bh[kT], Bl[kT];
#pragma unroll
    for (int t = 0; t < kT; ++t) {
      const int e0 = 32 * t + grp_ch + src_ch;
      float xk[12], xv[12];
#pragma unroll
      for (int r = 0; r < 3; ++r) {
        const int row = 8 * half + 4 * r - 4 + src_row;  // -4 .. 15
        const unsigned char* kb = row < 0 ? kprv : kcur;
        const unsigned char* vb = row < 0 ? vprv : vcur;
        const int rr = row < 0 ? row + 16 : row;
        const i16x4_t qk = tr_read(kb + swz<D>(rr, e0));
        const i16x4_t qv = tr_read(vb + swz<D>(rr, e0));
        const u32x2_t uk = __builtin_bit_cast(u32x2_t, qk);
        const u32x2_t uv = __builtin_bit_cast(u32x2_t, qv);
        xk[4 * r + 0] = bf16_lo(uk[0]); xk[4 * r + 1] = bf16_hi(uk[0]);
        xk[4 * r + 2] = bf16_lo(uk[1]); xk[4 * r + 3] = bf16_hi(uk[1]);
        xv[4 * r + 0] = bf16_lo(uv[0]); xv[4 * r + 1] = bf16_hi(uv[0]);
        xv[4 * r + 2] = bf16_lo(uv[1]); xv[4 * r + 3] = bf16_hi(uv[1]);
      }
      float kw[8], vt[8];
#pragma unroll
      for (int o = 0; o < 8; ++o) {
        float kc = wk[t][0] * xk[o + 1];
        float vc = wvt[t][0] * xv[o + 1];
#pragma unroll
        for (int tap = 1; tap < 4; ++tap) {
          kc = fmaf(wk[t][tap], xk[o + 1 + tap], kc);
          vc = fmaf(wvt[t][tap], xv[o + 1 + tap], vc);
        }
        const float ph = fmaxf(kc, 0.0f) + __expf(fminf(kc, 0.0f));
        kw[o] = wj[o] * ph;
        zacc[t] += kw[o];
        vt[o] = vc;
      }
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        A[t][p] = pack_bf16x2(kw[2 * p], kw[2 * p + 1]);
        const uint32_t hi = pack_bf16x2(vt[2 * p], vt[2 * p + 1]);
        Bh[t][p] = hi;
        Bl[t][p] = pack_bf16x2(vt[2 * p] - bf16_lo(hi), vt[2 * p + 1] - bf16_hi(hi));
      }
    }
#pragma unroll
    for (int a = 0; a < kT; ++a)
#pragma unroll
      for (int b = 0; b < kT; ++b) {
        acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, A[a]), __builtin_bit_cast(bf16x8_t, Bh[b]), acc[a][b], 0, 0, 0);
        acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, A[a]), __builtin_bit_cast(bf16x8_t, Bl[b]), acc[a][b], 0, 0, 0);
      }
    // Stage step i+1 into the ring (its slot held step i-3) and refill the
    // freed registers with step i+3.  Both run unconditionally so the wait
    // counts are the same on every path; steps past the end are loaded with
    // every row out of range (no memory traffic, zeros).
    commit(i + 1, kNext);
    issue(i + 3, kNext, i + 3 < nsteps ? 0 : C::kStep);
  };
  int i = 0;
  for (; i + 1 < nsteps; i += 2) {
    step_body(i, std::integral_constant<int, 1>{});
    step_body(i + 1, std::integral_constant<int, 0>{});
  }
  if (i < nsteps) step_body(i, std::integral_constant<int, 1>{});

  // ---- merge the four waves' partial states into the chunk's record ----
#pragma unroll
  for (int t = 0; t < kT; ++t) zacc[t] += __shfl_xor(zacc[t], 32);
  __syncthreads();  // every wave is done with its ring
  float* Sw = reinterpret_cast<float*>(ring);
#pragma unroll
  for (int a = 0; a < kT; ++a)
#pragma unroll
    for (int b = 0; b < kT; ++b)
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int c = 32 * a + 8 * (q / 4) + 4 * half + (q % 4);
        const int e = 32 * b + (lane & 31);
        Sw[c * D + e] = acc[a][b][q];
      }
  float* zw = wbuf;  // reuse: z_w[D], m_w, l_w
  if (lane < 32) {
#pragma unroll
    for (int t = 0; t < kT; ++t) zw[32 * t + lane] = zacc[t];
  }
  if (lane == 0) {
    zw[D] = mw;
    zw[D + 1] = lw;
  }
  __syncthreads();
  const float* wb0 = reinterpret_cast<const float*>(lds + C::kWaves * C::kWaveBytes);
  float mws[C::kWaves], f[C::kWaves];
  float M = -INFINITY;
#pragma unroll
  for (int w = 0; w < C::kWaves; ++w) {
    mws[w] = wb0[w * C::kMaxQ + D];
    M = fmaxf(M, mws[w]);
  }
#pragma unroll
  for (int w = 0; w < C::kWaves; ++w) f[w] = mws[w] == -INFINITY ? 0.0f : __expf(mws[w] - M);
#pragma unroll
  for (int k = 0; k < D * D / C::kNT; ++k) {
    const int x = k * C::kNT + tid;
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < C::kWaves; ++w)
      v = fmaf(f[w], reinterpret_cast<const float*>(lds + w * C::kWaveBytes)[x], v);
    rec[x] = v;
  }
  if (tid < D) {
    float v = 0.0f;
#pragma unroll
    for (int w = 0; w < C::kWaves; ++w) v = fmaf(f[w], wb0[w * C::kMaxQ + tid], v);
    rec[D * D + tid] = v;
  }
  if (tid == 0) {
    float l = 0.0f;
#pragma unroll
    for (int w = 0; w < C::kWaves; ++w) l = fmaf(f[w], wb0[w * C::kMaxQ + D + 1], l);
    rec[D * D + D] = M;
    rec[D * D + D + 1] = l;
  }
}

// ---------------------------------------------------------------------------
// readout_stream_kernel: one workgroup handles a tile of P.rtile tokens of one
// (sequence, head); each wave a quarter of it, 32 tokens per iteration.
//   o_i = phi(qt_i)^T S / phi(qt_i)^T z,
//   y_i = o_i / sqrt(mean_e o_i^2 + eps) * gamma * SiLU(r_i)
// q rows are staged through a per-wave LDS ring (register-staged loads one
// group ahead, 16-byte chunks XOR-swizzled by row; r one group ahead); each
// lane reads the four rows of its token's conv window, so lane (n, gq) gets
// phi(qt) of token n for channels 32*kb + 8*gq + [0, 8): the B operand of
// v_mfma_f32_16x16x32_bf16.  The A operands [S^T; z^T] stay in registers
// for the whole tile.  The gated-RMSNorm epilogue reduces each token's
// squares over the four lanes that hold its 64 (or 32) channels.
template <int D>
struct RS {
  static constexpr int kGroup = 32;                     // tokens per wave iteration
  static constexpr int kRowBytes = 2 * D;
  static constexpr int kChunks = kRowBytes / 16;
  static constexpr int kSlotBytes = kGroup * kRowBytes;
  static constexpr int kVec = kSlotBytes / 1024;        // 16-byte vectors per lane per group
  static constexpr int kSlots = 3;
  static constexpr int kNMB = D / 16 + 1, kNKB = D / 32;
  static constexpr int kLds = 4 * kSlots * kSlotBytes;
};

template <int D>
__global__ void __launch_bounds__(kThreads, 2)
readout_stream_kernel(Plan P, const uint16_t* __restrict__ qin, const uint16_t* __restrict__ rin,
                      const float* __restrict__ conv_w, const float* __restrict__ gamma,
                      const int32_t* __restrict__ cu, const unsigned char* __restrict__ frags,
                      float* __restrict__ out) {
  using C = RS<D>;
  constexpr int NMB = C::kNMB, NKB = C::kNKB;
  __shared__ __attribute__((aligned(16))) unsigned char lds[C::kLds];
  __shared__ __attribute__((aligned(16))) float taps_q[D][4];  // right-aligned, tap 3 = current
  __shared__ __attribute__((aligned(16))) float gam[D];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.y, g = blockIdx.x;
  int s, tile;
  if (!unit_of(P, cu, P.rtile, P.rtiles_per_seq, g, &s, &tile)) return;
  s = __builtin_amdgcn_readfirstlane(s);
  tile = __builtin_amdgcn_readfirstlane(tile);
  if (tid < D) {
    load_taps4(conv_w, P.heads, h, 0, D, P.W, tid, taps_q[tid]);
    gam[tid] = gamma[(size_t)h * D + tid];
  }
  __syncthreads();
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int64_t tt0 = (int64_t)tile * P.rtile;
  const int64_t tt1 = min(len, tt0 + (int64_t)P.rtile);
  const int per_wave = P.rtile >> 2;
  const int r0 = (int)(tt0 + (int64_t)wave * per_wave);  // slice-relative
  const int r1 = (int)min(tt1, (int64_t)r0 + per_wave);
  if (r1 <= r0) return;  // no block-wide synchronisation follows
  const int ngroups = (r1 - r0 + C::kGroup - 1) / C::kGroup;
  unsigned char* ring = lds + wave * C::kSlots * C::kSlotBytes;

  const int n = lane & 15, gq = lane >> 4;
  const size_t sh = (size_t)s * P.heads + h;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(qin + base_row * D, (uint32_t)(len * C::kRowBytes));
  const __amdgpu_buffer_rsrc_t rr = make_rsrc(rin + base_row * D, (uint32_t)(len * C::kRowBytes));
  // stores of tokens at or past r1 fall outside this range and are dropped
  const __amdgpu_buffer_rsrc_t ro = make_rsrc(out + base_row * D, (uint32_t)r1 * (uint32_t)(4 * D));

  // Readout operands [S^T; z^T]: loaded before any prefetch so that their
  // wait precedes the pipeline.
  const unsigned char* fr = frags + sh * P.frag_bytes;
  u32x4_t A[NMB][NKB];
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) A[mb][kb] = load16(fr + (((size_t)mb * NKB + kb) * 64 + lane) * 16);

  // ---- staged loads: q rows of a group, r chunks of the lane's two tokens ----
  u32x4_t qst[C::kVec];
  u32x4_t rst[2][NKB];
  auto issue_q = [&](int grp, int first_row) {
#pragma unroll
    for (int x = 0; x < C::kVec; ++x) {
      const int u = x * 64 + lane;
      const int row = u / C::kChunks, ch = u % C::kChunks;
      const int tok = r0 + grp * C::kGroup + row;
      qst[x] = bload16(rq, row >= first_row ? (uint32_t)(tok * D + ch * 8) * 2u : kOutOfRange);
    }
  };
  auto issue_r = [&](int grp, bool live) {
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) {
      const int tok = r0 + grp * C::kGroup + 16 * jb + n;
#pragma unroll
      for (int qq = 0; qq < NKB; ++qq)
        rst[jb][qq] = bload16(rr, live ? (uint32_t)(tok * D + 32 * qq + 8 * gq) * 2u : kOutOfRange);
    }
  };
  auto commit_q = [&](int grp) {
    const int slot = (grp + C::kSlots) % C::kSlots;
#pragma unroll
    for (int x = 0; x < C::kVec; ++x) {
      const int u = x * 64 + lane;
      const int row = u / C::kChunks, ch = u % C::kChunks;
      *reinterpret_cast<u32x4_t*>(ring + slot * C::kSlotBytes + row * C::kRowBytes +
                                  ((ch ^ (row & (C::kChunks - 1))) << 4)) = qst[x];
    }
  };

  // Rows 29..31 of the group before the wave's first token (the conv window).
  issue_q(-1, C::kGroup - 3);
  commit_q(-1);
  issue_q(0, 0);
  issue_r(0, true);
  commit_q(0);
  issue_q(1, ngroups > 1 ? 0 : C::kGroup);

  for (int grp = 0; grp < ngroups; ++grp) {
    const unsigned char* cur = ring + (grp % C::kSlots) * C::kSlotBytes;
    const unsigned char* prv = ring + ((grp + C::kSlots - 1) % C::kSlots) * C::kSlotBytes;
    // B operands phi(qt) of both 16-token blocks, channel chunk by chunk.
    u32x4_t B[2][NKB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
      f32x4_t wq[8];
#pragma unroll
      for (int c = 0; c < 8; ++c) wq[c] = *reinterpret_cast<const f32x4_t*>(taps_q[32 * kb + 8 * gq + c]);
#pragma unroll
      for (int jb = 0; jb < 2; ++jb) {
        const int row = 16 * jb + n;
        float x[4][8];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int rw = row - 3 + t;
          const unsigned char* base = rw < 0 ? prv : cur;
          const int rrow = rw < 0 ? rw + C::kGroup : rw;
          const int ch = 4 * kb + gq;
          const u32x4_t u = *reinterpret_cast<const u32x4_t*>(
              base + rrow * C::kRowBytes + ((ch ^ (rrow & (C::kChunks - 1))) << 4));
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            x[t][2 * w] = bf16_lo(u[w]);
            x[t][2 * w + 1] = bf16_hi(u[w]);
          }
        }
        float f[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          float acc = wq[c][0] * x[0][c];
#pragma unroll
          for (int t = 1; t < 4; ++t) acc = fmaf(wq[c][t], x[t][c], acc);
          f[c] = fmaxf(acc, 0.0f) + __expf(fminf(acc, 0.0f));
        }
#pragma unroll
        for (int w = 0; w < 4; ++w) B[jb][kb][w] = pack_bf16x2(f[2 * w], f[2 * w + 1]);
      }
    }
#pragma unroll
    for (int jb = 0; jb < 2; ++jb) {
      const int row = 16 * jb + n;
      f32x4_t acc[NMB];
#pragma unroll
      for (int mb = 0; mb < NMB; ++mb) acc[mb] = (f32x4_t){0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb)
          acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, A[mb][kb]),
                                                            __builtin_bit_cast(bf16x8_t, B[jb][kb]),
                                                            acc[mb], 0, 0, 0);
      const float inv_den = __builtin_amdgcn_rcpf(acc[NMB - 1][0]);
      float ss = 0.0f;
#pragma unroll
      for (int mb = 0; mb < NMB - 1; ++mb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          acc[mb][i] *= inv_den;
          ss = fmaf(acc[mb][i], acc[mb][i], ss);
        }
      ss += __shfl_xor(ss, 16);
      ss += __shfl_xor(ss, 32);
      const float scale = __builtin_amdgcn_rsqf(ss * (1.0f / D) + P.eps);
      const int tok = r0 + grp * C::kGroup + row;
#pragma unroll
      for (int qq = 0; qq < NKB; ++qq) {
        const u32x4_t rw = rst[jb][qq];
        const f32x4_t g0 = *reinterpret_cast<const f32x4_t*>(&gam[32 * qq + 8 * gq]);
        const f32x4_t g1 = *reinterpret_cast<const f32x4_t*>(&gam[32 * qq + 8 * gq + 4]);
        f32x4_t y0, y1;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float ra = i & 1 ? bf16_hi(rw[i >> 1]) : bf16_lo(rw[i >> 1]);
          const float rb = i & 1 ? bf16_hi(rw[2 + (i >> 1)]) : bf16_lo(rw[2 + (i >> 1)]);
          const float sa = ra * __builtin_amdgcn_rcpf(1.0f + __expf(-ra));
          const float sb = rb * __builtin_amdgcn_rcpf(1.0f + __expf(-rb));
          y0[i] = acc[2 * qq][i] * scale * g0[i] * sa;
          y1[i] = acc[2 * qq + 1][i] * scale * g1[i] * sb;
        }
        const uint32_t off = (uint32_t)(tok * D + 32 * qq + 8 * gq) * 4u;
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, y0), ro, off, 0, 0);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, y1), ro, off + 16, 0, 0);
      }
    }
    // Stage group grp+1 into the ring (its slot held group grp-2), then
    // refill the registers: r of group grp+1 first, q rows of group grp+2
    // (fully out of range past the end, so the wait counts never change).
    commit_q(grp + 1);
    issue_r(grp + 1, grp + 1 < ngroups);
    issue_q(grp + 2, grp + 2 < ngroups ? 0 : C::kGroup);
  }
}

}  // namespace

bool stream_supported(const Plan& p) {
  // Every (sequence, head) slice must stay below 2^31 bytes for the 32-bit
  // buffer offsets; the fp32 output rows are the widest.
  return p.dtype == GBLA_BF16 && (p.d == 32 || p.d == 64) &&
         p.chunk <= SS<64>::kWaves * SS<64>::kMaxQ && p.chunk % (16 * SS<64>::kWaves) == 0 &&
         p.rtile % 128 == 0 && (int64_t)p.rows * p.d * 4 < (int64_t(1) << 31);
}

gbla_status launch_state_stream(const Plan& p, const void* k, const void* v, const void* a,
                                const float* conv_w, const int32_t* cu, float* partials,
                                hipStream_t st) {
  const dim3 grid(p.units, p.heads);
  if (p.d == 64)
    hipLaunchKernelGGL((state_stream_kernel<64>), grid, dim3(SS<64>::kNT), 0, st, p,
                       (const uint16_t*)k, (const uint16_t*)v, (const uint16_t*)a, conv_w, cu, partials);
  else
    hipLaunchKernelGGL((state_stream_kernel<32>), grid, dim3(SS<32>::kNT), 0, st, p,
                       (const uint16_t*)k, (const uint16_t*)v, (const uint16_t*)a, conv_w, cu, partials);
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}

gbla_status launch_readout_stream(const Plan& p, const void* q, const void* r, const float* conv_w,
                                  const float* gamma, const int32_t* cu, const unsigned char* frags,
                                  float* out, hipStream_t st) {
  const dim3 grid(p.runits, p.heads);
  if (p.d == 64)
    hipLaunchKernelGGL((readout_stream_kernel<64>), grid, dim3(kThreads), 0, st, p,
                       (const uint16_t*)q, (const uint16_t*)r, conv_w, gamma, cu, frags, out);
  else
    hipLaunchKernelGGL((readout_stream_kernel<32>), grid, dim3(kThreads), 0, st, p,
                       (const uint16_t*)q, (const uint16_t*)r, conv_w, gamma, cu, frags, out);
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}

}  // namespace gbla
