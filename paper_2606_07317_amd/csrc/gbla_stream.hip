// gbla_stream.hip -- streaming kernels of the bf16 GBLA forward pass for
// head dims 32 and 64 (gfx950).
//
// state_stream_kernel: one workgroup reduces one chunk of tokens of one
// (sequence, head) to a partial state (Section 2.1, key-gating item, matrix
// form K^T V and K^T 1 with K = g (.) phi(K)):
//     S_p = sum_j w_j phi(kt_j) vt_j^T,  z_p = sum_j w_j phi(kt_j),
//     w_j = exp(a_j - m_p),  m_p = max_j a_j,  l_p = sum_j w_j.
// The chunk is split into token parts; the waves of a part share its tokens
// and split the key channels (one 32-channel MFMA tile each) and, at
// d = 128, the value channels into halves.  Every wave then holds at most
// 128 accumulators, so two waves run on every SIMD and each one's vector
// work overlaps the other's MFMAs.  A wave streams its tokens 16 at a time:
// raw bf16 key (its 32 channels) and value (its channels) rows are loaded
// two steps ahead into registers, written row-major into the wave's LDS
// rings (16-byte chunks XOR-swizzled by row), and read back with
// ds_read_b64_tr_b16, which hands each lane four
// consecutive tokens of one channel.  Twelve key tokens (three reads) give
// the lane the causal conv window of its eight tokens, so the key conv, phi
// and the gate weight are applied in registers and the results are already
// the A operand of v_mfma_f32_32x32x16_bf16 (channel c, 8 tokens).
// The value conv is linear and acts channel by channel, so it is moved past
// the token sum: with taps u_tau (tap 3 on the current token),
//     S_p[c][e] = sum_tau u_tau[e] M_tau[c][e],
//     M_tau     = sum_j w_j phi(kt_j) v_{j-3+tau}^T,
// and each M_tau is one MFMA accumulator fed with raw bf16 v rows read at a
// shift of tau - 3 tokens.  The value path costs no vector ALU work in the
// loop and v enters the products exactly; the taps are applied once, in fp32,
// when the accumulators are merged.
//
// readout_stream_kernel: see its own comment below.
//
// All global traffic of the hot loops goes through raw buffer descriptors
// that span one (sequence, head) slice: rows before the sequence start or
// past its end read as zero, stores past the tile end are dropped.  There
// are no branches around memory instructions, so the compiler's wait counts
// stay exact and the prefetched loads remain in flight.
#include <hip/hip_ext.h>
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
  static constexpr int kStep = 16;                       // tokens per MFMA K block
  // The waves of a token part split the key channels into 32-channel tiles
  // and, at d = 128, the value channels into halves, so that every wave holds
  // at most 128 accumulators and two waves run on each SIMD.
  static constexpr int kKH = D / 32;                      // key tiles
  static constexpr int kVH = D == 128 ? 2 : 1;            // value slices
  static constexpr int kVD = D / kVH;                     // value channels per wave
  static constexpr int kWaves = 8;
  static constexpr int kNT = 64 * kWaves;
  static constexpr int kParts = kWaves / (kKH * kVH);     // token parts of a chunk
  static constexpr int kTB = kVD / 32;                    // 32-wide value tiles per wave
  static constexpr int kStepBytes = kStep * 2 * D;        // one step of rows in memory
  static constexpr int kKRow = 64;                        // a wave's 32 key channels of a row
  static constexpr int kVRow = 2 * kVD;                   // a wave's value channels of a row
  static constexpr int kKChunks = kKRow / 16, kVChunks = kVRow / 16;
  static constexpr int kKSlot = kStep * kKRow, kVSlot = kStep * kVRow;
  static constexpr int kKVec = kKSlot / 1024, kVVec = kVSlot / 1024;  // 16-byte vectors per lane
  static constexpr int kSlots = 4;                        // ring depth
  static constexpr int kKRing = kSlots * kKSlot;
  static constexpr int kRing = kKRing + kSlots * kVSlot;  // one wave's rings
  static constexpr int kMaxChunk = 2048;
  static constexpr int kMaxQ = kMaxChunk / kParts;        // tokens per part
  static constexpr int kPartFloats = D * D + D + 2;       // S, z, m, l of a part
  static constexpr int kMerge = kParts * kPartFloats * 4;
  static constexpr int kRings = kWaves * kRing > kMerge ? kWaves * kRing : kMerge;
  static constexpr int kLds = kRings + kParts * kMaxQ * 4;  // + gate weights per part
};

// Byte offset of element e (a multiple of 4) of row r of a slot whose rows
// hold `Chunks` 16-byte chunks, XOR-swizzled by the row index.
template <int Chunks>
__device__ __forceinline__ int swz(int r, int e) {
  const int c = e >> 3, half = (e >> 2) & 1;
  return r * Chunks * 16 + ((c ^ (r & (Chunks - 1))) << 4) + (half << 3);
}

template <int D>
__global__ void __launch_bounds__(SS<D>::kNT, 1)
state_stream_kernel(Plan P, const uint16_t* __restrict__ kin, const uint16_t* __restrict__ vin,
                    const uint16_t* __restrict__ ain, const float* __restrict__ conv_w,
                    const int32_t* __restrict__ cu, float* __restrict__ partials) {
  using C = SS<D>;
  constexpr int kTB = C::kTB;
  __shared__ __attribute__((aligned(16))) unsigned char lds[C::kLds];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int part = wave / (C::kKH * C::kVH);
  const int kh = (wave / C::kVH) % C::kKH, vh = wave % C::kVH;
  const int vc0 = vh * C::kVD;  // first value channel of the wave
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

  const int Q = P.chunk / C::kParts;               // tokens per part
  const int w0 = (int)(t0 + (int64_t)part * Q);    // slice-relative token range
  const int w1 = (int)min(t1, (int64_t)w0 + Q);
  const int nsteps = w1 > w0 ? (w1 - w0 + C::kStep - 1) / C::kStep : 0;
  // The loop turns the ring once per iteration (kSlots steps), so that every
  // LDS address is a per-lane base plus an immediate.  Steps past nsteps see
  // only out-of-range rows and zero gate weights and add nothing.
  const int nturns = (nsteps + C::kSlots - 1) / C::kSlots;
  unsigned char* ring = lds + wave * C::kRing;  // [key slots][value slots]
  // gate weights of the part: every wave of the part writes the same values
  // before it reads them, so no barrier is needed
  float* wbuf = reinterpret_cast<float*>(lds + C::kRings) + part * C::kMaxQ;

  const __amdgpu_buffer_rsrc_t rk = make_rsrc(kin + base_row * D, (uint32_t)(len * 2 * D));
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vin + base_row * D, (uint32_t)(len * 2 * D));
  // no logits (uniform gates): an empty range, so every logit reads as 0
  const __amdgpu_buffer_rsrc_t ra =
      ain ? make_rsrc(ain + base_row, (uint32_t)(len * 2)) : make_rsrc(kin, 0u);

  // Loop-invariant global values first (taps, gate logits), so that the
  // waits for them precede every prefetch.  The key taps carry a factor
  // log2(e): the loop then forms kt * log2(e) and phi needs only exp2.  The
  // value taps are needed only by the final merge.
  constexpr float kLog2e = 1.4426950408889634f, kLn2 = 0.6931471805599453f;
  const int kch = 32 * kh + (lane & 31);  // the lane's key channel
  float wk[4], wv[kTB][4];
  load_taps4(conv_w, P.heads, h, 1, D, P.W, kch, wk);
#pragma unroll
  for (int b = 0; b < kTB; ++b) load_taps4(conv_w, P.heads, h, 2, D, P.W, vc0 + 32 * b + (lane & 31), wv[b]);
  // Gate logits of the part's tokens; tokens outside it read as zero and get
  // -inf added below (an add, not a select on the loaded value, so that the
  // loads stay ahead of the prefetches instead of being sunk into branches).
  uint32_t abits[C::kMaxQ / 64];
  float amask[C::kMaxQ / 64];
#pragma unroll
  for (int i = 0; i < C::kMaxQ / 64; ++i) {
    const int tok = w0 + lane + 64 * i;
    const bool valid = 64 * i < Q && tok < w1;
    abits[i] = __builtin_amdgcn_raw_buffer_load_b16(ra, valid ? (uint32_t)tok * 2u : kOutOfRange, 0, 0);
    amask[i] = valid ? 0.0f : -INFINITY;
  }

  // ---- per-lane constants: the row / 16-byte chunk of a step that each
  // vector of the staged loads holds, and where it goes in the rings ----
  int kgoff[C::kKVec], kgrow[C::kKVec], vgoff[C::kVVec], vgrow[C::kVVec];
  unsigned char *kwp[C::kKVec], *vwp[C::kVVec];
#pragma unroll
  for (int x = 0; x < C::kKVec; ++x) {
    const int u = x * 64 + lane;
    const int row = u / C::kKChunks, ch = u % C::kKChunks;
    kgrow[x] = row;
    kgoff[x] = ((w0 + row) * D + 32 * kh + ch * 8) * 2;
    kwp[x] = ring + row * C::kKRow + ((ch ^ (row & (C::kKChunks - 1))) << 4);
  }
#pragma unroll
  for (int x = 0; x < C::kVVec; ++x) {
    const int u = x * 64 + lane;
    const int row = u / C::kVChunks, ch = u % C::kVChunks;
    vgrow[x] = row;
    vgoff[x] = ((w0 + row) * D + vc0 + ch * 8) * 2;
    vwp[x] = ring + C::kKRing + row * C::kVRow + ((ch ^ (row & (C::kVChunks - 1))) << 4);
  }

  u32x4_t sk[2][C::kKVec], sv[2][C::kVVec];  // [in-flight buffer = step % 2][vector]
  auto issue = [&](int step, int buf, bool live) {
#pragma unroll
    for (int x = 0; x < C::kKVec; ++x)
      sk[buf][x] = bload16(rk, live ? (uint32_t)(kgoff[x] + step * C::kStepBytes) : kOutOfRange);
#pragma unroll
    for (int x = 0; x < C::kVVec; ++x)
      sv[buf][x] = bload16(rv, live ? (uint32_t)(vgoff[x] + step * C::kStepBytes) : kOutOfRange);
  };
  auto commit = [&](int slot, int buf) {
#pragma unroll
    for (int x = 0; x < C::kKVec; ++x)
      *reinterpret_cast<u32x4_t*>(kwp[x] + slot * C::kKSlot) = sk[buf][x];
#pragma unroll
    for (int x = 0; x < C::kVVec; ++x)
      *reinterpret_cast<u32x4_t*>(vwp[x] + slot * C::kVSlot) = sv[buf][x];
  };
  // Of the step before the part's first token only rows 12..15 (the conv
  // window) are needed; they sit in the vectors from kXk / kXv on.
  constexpr int kXk = 12 * C::kKChunks / 64, kXv = 12 * C::kVChunks / 64;
  u32x4_t mk[C::kKVec - kXk], mv[C::kVVec - kXv];
#pragma unroll
  for (int x = kXk; x < C::kKVec; ++x)
    mk[x - kXk] = bload16(rk, kgrow[x] >= C::kStep - 4 && nsteps > 0
                                  ? (uint32_t)(kgoff[x] - C::kStepBytes) : kOutOfRange);
#pragma unroll
  for (int x = kXv; x < C::kVVec; ++x)
    mv[x - kXv] = bload16(rv, vgrow[x] >= C::kStep - 4 && nsteps > 0
                                  ? (uint32_t)(vgoff[x] - C::kStepBytes) : kOutOfRange);
  issue(0, 0, nsteps > 0);
  issue(1, 1, nsteps > 1);
  // Keep every load above in flight before any of the work below: the
  // scheduler would otherwise hoist the gate pass (and its wait for the
  // logits) ahead of the prefetches.
  __builtin_amdgcn_sched_barrier(0);

  // ---- gate weights of the part's tokens: m_w, w_j = exp(a_j - m_w), l_w ----
  float av[C::kMaxQ / 64];
  float mloc = -INFINITY;
#pragma unroll
  for (int i = 0; i < C::kMaxQ / 64; ++i) {
    av[i] = __uint_as_float(abits[i] << 16) + amask[i];
    mloc = fmaxf(mloc, av[i]);
  }
  const float mw = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                                              __builtin_bit_cast(int, wave_max(mloc))));
  float lsum = 0.0f;
#pragma unroll
  for (int i = 0; i < C::kMaxQ / 64; ++i) {
    // every entry is written: the padded steps of the last turn read zeros
    const float wv = av[i] == -INFINITY ? 0.0f : __expf(av[i] - mw);
    wbuf[lane + 64 * i] = wv;
    lsum += wv;
  }
  const float lw = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                                              __builtin_bit_cast(int, wave_sum(lsum))));

  f32x16_t acc[4][kTB];  // M_tau restricted to the wave's 32 key channels
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int b = 0; b < kTB; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[u][b][i] = 0.0f;
  float zacc = 0.0f;
#pragma unroll
  for (int tap = 0; tap < 4; ++tap) wk[tap] *= kLog2e;

  // Lane roles for the transposed reads and the MFMA operands.  Read r hands
  // the lane rows 8*half - 4 + 4r + [0, 4) of one channel (key channel kch,
  // value channel vc0 + 32b + (lane & 31)); rows before 0 are rows 12..15 of the
  // previous slot.
  const int half = lane >> 5;  // token half of the 16-token step
  const int grp_ch = 16 * ((lane >> 4) & 1);
  const int j = lane & 15;
  const int src_row = j >> 2, src_ch = 4 * (j & 3);
  const int row0 = 8 * half - 4 + src_row;
  const bool prv = row0 < 0;
  const int rr0 = prv ? row0 + C::kStep : row0;
  // [read 0 for slots >= 1, read 0 for slot 0, read 1, read 2]
  const unsigned char* kp[4];
  const unsigned char* vp[kTB][4];
  {
    const int e0 = grp_ch + src_ch;
    const int o0 = swz<C::kKChunks>(rr0, e0);
    kp[0] = ring + o0 - (prv ? C::kKSlot : 0);
    kp[1] = ring + o0 + (prv ? (C::kSlots - 1) * C::kKSlot : 0);
    kp[2] = ring + swz<C::kKChunks>(row0 + 4, e0);
    kp[3] = ring + swz<C::kKChunks>(row0 + 8, e0);
  }
#pragma unroll
  for (int b = 0; b < kTB; ++b) {
    const int e0 = 32 * b + grp_ch + src_ch;
    const unsigned char* vr = ring + C::kKRing;
    const int o0 = swz<C::kVChunks>(rr0, e0);
    vp[b][0] = vr + o0 - (prv ? C::kVSlot : 0);
    vp[b][1] = vr + o0 + (prv ? (C::kSlots - 1) * C::kVSlot : 0);
    vp[b][2] = vr + swz<C::kVChunks>(row0 + 4, e0);
    vp[b][3] = vr + swz<C::kVChunks>(row0 + 8, e0);
  }
  const float* wl = wbuf + 8 * half;

  // One step: transposed reads of the twelve-row windows (dword m of read r
  // holds rows 8*half - 4 + 4r + 2m', +1), the operands, the products.
  auto step = [&](auto slot_c, int i) {
    constexpr int sl = decltype(slot_c)::value;
    u32x2_t wkr[3], wvr[kTB][3];
#pragma unroll
    for (int r = 0; r < 3; ++r) {
      const unsigned char* b = (r == 0 ? (sl == 0 ? kp[1] : kp[0]) : kp[r + 1]) + sl * C::kKSlot;
      wkr[r] = __builtin_bit_cast(u32x2_t, tr_read(b));
    }
#pragma unroll
    for (int bt = 0; bt < kTB; ++bt)
#pragma unroll
      for (int r = 0; r < 3; ++r) {
        const unsigned char* b = (r == 0 ? (sl == 0 ? vp[bt][1] : vp[bt][0]) : vp[bt][r + 1]) + sl * C::kVSlot;
        wvr[bt][r] = __builtin_bit_cast(u32x2_t, tr_read(b));
      }
    // gate weights of the lane's eight tokens
    const f32x4_t wa = *reinterpret_cast<const f32x4_t*>(wl + 16 * i);
    const f32x4_t wb = *reinterpret_cast<const f32x4_t*>(wl + 16 * i + 4);
    const float wj[8] = {wa[0], wa[1], wa[2], wa[3], wb[0], wb[1], wb[2], wb[3]};
    // A = w phi(kt) of key channel kch over the lane's eight tokens
    float xk[12];
#pragma unroll
    for (int r = 0; r < 3; ++r) {
      xk[4 * r + 0] = bf16_lo(wkr[r][0]); xk[4 * r + 1] = bf16_hi(wkr[r][0]);
      xk[4 * r + 2] = bf16_lo(wkr[r][1]); xk[4 * r + 3] = bf16_hi(wkr[r][1]);
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
    u32x4_t A;
#pragma unroll
    for (int p = 0; p < 4; ++p) A[p] = pack_bf16x2(kw[2 * p], kw[2 * p + 1]);
    // B[tau] = value rows of the lane's eight tokens shifted by tau - 3: the
    // window starts at row tau + 1 (odd shifts straddle two dwords)
#pragma unroll
    for (int bt = 0; bt < kTB; ++bt) {
      const uint32_t pv[6] = {wvr[bt][0][0], wvr[bt][0][1], wvr[bt][1][0],
                              wvr[bt][1][1], wvr[bt][2][0], wvr[bt][2][1]};
      u32x4_t B[4];
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        B[0][m] = __builtin_amdgcn_alignbit(pv[m + 1], pv[m], 16);
        B[1][m] = pv[m + 1];
        B[2][m] = __builtin_amdgcn_alignbit(pv[m + 2], pv[m + 1], 16);
        B[3][m] = pv[m + 2];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        acc[u][bt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8_t, A), __builtin_bit_cast(bf16x8_t, B[u]), acc[u][bt], 0, 0, 0);
    }
  };

  // Pipeline: at the top of step i, step i+1 is staged into its slot (the
  // slot of step i-3) and its registers are refilled with step i+3; then
  // step i is read back and computed.  The other wave on the SIMD covers the
  // read latency and overlaps its vector work with these MFMAs.  Loads and
  // stores run on every path, so the wait counts are the same everywhere;
  // steps past the end load only out-of-range rows (no traffic, zeros).
  using I0 = std::integral_constant<int, 0>;
  using I1 = std::integral_constant<int, 1>;
  using I2 = std::integral_constant<int, 2>;
  using I3 = std::integral_constant<int, 3>;
#pragma unroll
  for (int x = kXk; x < C::kKVec; ++x)
    *reinterpret_cast<u32x4_t*>(kwp[x] + (C::kSlots - 1) * C::kKSlot) = mk[x - kXk];
#pragma unroll
  for (int x = kXv; x < C::kVVec; ++x)
    *reinterpret_cast<u32x4_t*>(vwp[x] + (C::kSlots - 1) * C::kVSlot) = mv[x - kXv];
  commit(0, 0);
  issue(2, 0, nsteps > 2);
  for (int it = 0; it < nturns; ++it) {
    const int i = it * C::kSlots;
    commit(1, 1);
    issue(i + 3, 1, i + 3 < nsteps);
    step(I0{}, i);
    commit(2, 0);
    issue(i + 4, 0, i + 4 < nsteps);
    step(I1{}, i + 1);
    commit(3, 1);
    issue(i + 5, 1, i + 5 < nsteps);
    step(I2{}, i + 2);
    commit(0, 0);
    issue(i + 6, 0, i + 6 < nsteps);
    step(I3{}, i + 3);
  }

  // ---- merge: the waves of a part fill its D x D state, the parts are
  // rescaled to the chunk maximum and summed in a fixed order ----
  zacc += __shfl_xor(zacc, 32);
  __syncthreads();  // every wave is done with its rings
  float* Sp = reinterpret_cast<float*>(lds) + part * C::kPartFloats;
#pragma unroll
  for (int b = 0; b < kTB; ++b) {
    const int e = vc0 + 32 * b + (lane & 31);  // the channel of wv[b]
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int c = 32 * kh + 8 * (q / 4) + 4 * half + (q % 4);
      float sv = wv[b][0] * acc[0][b][q];
#pragma unroll
      for (int u = 1; u < 4; ++u) sv = fmaf(wv[b][u], acc[u][b][q], sv);
      Sp[c * D + e] = sv;
    }
  }
  if (vh == 0 && lane < 32) Sp[D * D + kch] = zacc;  // value slices repeat z, m, l
  if (vh == 0 && kh == 0 && lane == 0) {
    Sp[D * D + D] = mw;
    Sp[D * D + D + 1] = lw;
  }
  __syncthreads();
  const float* S0 = reinterpret_cast<const float*>(lds);
  float f[C::kParts];
  float M = -INFINITY;
#pragma unroll
  for (int p = 0; p < C::kParts; ++p) M = fmaxf(M, S0[p * C::kPartFloats + D * D + D]);
#pragma unroll
  for (int p = 0; p < C::kParts; ++p) {
    const float mp = S0[p * C::kPartFloats + D * D + D];
    f[p] = mp == -INFINITY ? 0.0f : __expf(mp - M);
  }
  for (int x = tid; x < D * D + D; x += C::kNT) {
    float v = 0.0f;
#pragma unroll
    for (int p = 0; p < C::kParts; ++p) v = fmaf(f[p], S0[p * C::kPartFloats + x], v);
    rec[x] = v;
  }
  if (tid == 0) {
    float l = 0.0f;
#pragma unroll
    for (int p = 0; p < C::kParts; ++p) l = fmaf(f[p], S0[p * C::kPartFloats + D * D + D + 1], l);
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
  static constexpr int kOcc = D == 128 ? 1 : 2;         // waves per SIMD (registers)
  static constexpr int kLds = 4 * kSlots * kSlotBytes;
};

template <int D, bool kNorm>
__global__ void __launch_bounds__(kThreads, RS<D>::kOcc)
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
  // At d = 128 a (sequence, head) reads 37 KB of operands, and each XCD
  // has its own L2: workgroups go to the eight XCDs in turn by linear id, so
  // XCD x is given one contiguous run of tiles (v below is a bijection of
  // the grid) and fetches a pair's operands once instead of all eight XCDs.
  int h = blockIdx.y, g = blockIdx.x;
  if constexpr (D == 128) {
    const int n = (int)(gridDim.x * gridDim.y), L = (int)(blockIdx.x + blockIdx.y * gridDim.x);
    const int q = n >> 3, r = n & 7, x = L & 7;
    const int v = x * q + min(x, r) + (L >> 3);
    g = v % (int)gridDim.x;
    h = v / (int)gridDim.x;
  }
  int s, tile;
  if (!unit_of(P, cu, P.rtile, P.rtiles_per_seq, g, &s, &tile)) return;
  s = __builtin_amdgcn_readfirstlane(s);
  tile = __builtin_amdgcn_readfirstlane(tile);
  // q taps and gamma of channel tid % D, loaded by every thread with no
  // branch around the loads, so that the tile's first loads below are issued
  // at once; the first D threads store them to LDS after those.
  float tq[4];
  load_taps4(conv_w, P.heads, h, 0, D, P.W, tid % D, tq);
  const __amdgpu_buffer_rsrc_t rg = make_rsrc(gamma ? gamma + (size_t)h * D : gamma, gamma ? 4u * D : 0u);
  const float graw = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rg, 4u * (tid % D), 0, 0));
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int64_t tt0 = (int64_t)tile * P.rtile;
  const int64_t tt1 = min(len, tt0 + (int64_t)P.rtile);
  const int per_wave = P.rtile >> 2;
  const int r0 = (int)(tt0 + (int64_t)wave * per_wave);  // slice-relative
  const int r1 = (int)min(tt1, (int64_t)r0 + per_wave);
  const int ngroups = (r1 - r0 + C::kGroup - 1) / C::kGroup;  // < 1: the wave has no rows
  unsigned char* ring = lds + wave * C::kSlots * C::kSlotBytes;

  const int n = lane & 15, gq = lane >> 4;
  const size_t sh = (size_t)s * P.heads + h;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(qin + base_row * D, (uint32_t)(len * C::kRowBytes));
  // kNorm false: out = o (no gated norm) and r is not read
  const __amdgpu_buffer_rsrc_t rr =
      kNorm ? make_rsrc(rin + base_row * D, (uint32_t)(len * C::kRowBytes)) : make_rsrc(qin, 0u);
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
  // Of the group before the wave's first token only rows 29..31 (the conv
  // window) are read; they sit in the vectors from kXh on.
  constexpr int kXh = (C::kGroup - 3) * C::kChunks / 64;
  u32x4_t qst[C::kVec], qhalo[C::kVec - kXh];
  u32x4_t rst[2][NKB];
  auto issue_q = [&](u32x4_t(&dst)[C::kVec], int grp, int first_row) {
#pragma unroll
    for (int x = 0; x < C::kVec; ++x) {
      const int u = x * 64 + lane;
      const int row = u / C::kChunks, ch = u % C::kChunks;
      const int tok = r0 + grp * C::kGroup + row;
      dst[x] = bload16(rq, row >= first_row ? (uint32_t)(tok * D + ch * 8) * 2u : kOutOfRange);
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
  auto commit_q = [&](const u32x4_t(&src)[C::kVec], int grp) {
    const int slot = (grp + C::kSlots) % C::kSlots;
#pragma unroll
    for (int x = 0; x < C::kVec; ++x) {
      const int u = x * 64 + lane;
      const int row = u / C::kChunks, ch = u % C::kChunks;
      *reinterpret_cast<u32x4_t*>(ring + slot * C::kSlotBytes + row * C::kRowBytes +
                                  ((ch ^ (row & (C::kChunks - 1))) << 4)) = src[x];
    }
  };

  // The conv window before the wave's first token, then group 0: both in
  // flight before the first wait.
#pragma unroll
  for (int x = kXh; x < C::kVec; ++x) {
    const int u = x * 64 + lane;
    const int row = u / C::kChunks, ch = u % C::kChunks;
    const int tok = r0 - C::kGroup + row;
    qhalo[x - kXh] = bload16(rq, row >= C::kGroup - 3 ? (uint32_t)(tok * D + ch * 8) * 2u : kOutOfRange);
  }
  issue_q(qst, 0, 0);
  if constexpr (kNorm) issue_r(0, true);
  if (tid < D) {
#pragma unroll
    for (int t = 0; t < 4; ++t) taps_q[tid][t] = tq[t];
    if constexpr (kNorm) gam[tid] = gamma ? graw : 1.0f;
  }
  __syncthreads();
  if (ngroups < 1) return;  // no block-wide synchronisation follows
#pragma unroll
  for (int x = kXh; x < C::kVec; ++x) {
    const int u = x * 64 + lane;
    const int row = u / C::kChunks, ch = u % C::kChunks;
    *reinterpret_cast<u32x4_t*>(ring + (C::kSlots - 1) * C::kSlotBytes + row * C::kRowBytes +
                                ((ch ^ (row & (C::kChunks - 1))) << 4)) = qhalo[x - kXh];
  }
  commit_q(qst, 0);
  issue_q(qst, 1, ngroups > 1 ? 0 : C::kGroup);

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
      const int tok = r0 + grp * C::kGroup + row;
      if constexpr (!kNorm) {  // out = o
#pragma unroll
        for (int qq = 0; qq < NKB; ++qq) {
          const f32x4_t y0 = acc[2 * qq], y1 = acc[2 * qq + 1];
          const uint32_t off = (uint32_t)(tok * D + 32 * qq + 8 * gq) * 4u;
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, y0), ro, off, 0, 0);
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, y1), ro, off + 16, 0, 0);
        }
        continue;
      }
      ss += __shfl_xor(ss, 16);
      ss += __shfl_xor(ss, 32);
      const float scale = __builtin_amdgcn_rsqf(ss * (1.0f / D) + P.eps);
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
    commit_q(qst, grp + 1);
    if constexpr (kNorm) issue_r(grp + 1, grp + 1 < ngroups);
    issue_q(qst, grp + 2, grp + 2 < ngroups ? 0 : C::kGroup);
  }
}

}  // namespace

bool stream_supported(const Plan& p) {
  // Every (sequence, head) slice must stay below 2^31 bytes for the 32-bit
  // buffer offsets; the fp32 output rows are the widest.
  return p.dtype == GBLA_BF16 && (p.d == 32 || p.d == 64 || p.d == 128) &&
         p.chunk <= SS<64>::kMaxChunk && p.chunk % (SS<32>::kStep * SS<32>::kParts) == 0 &&
         p.chunk % (SS<64>::kStep * SS<64>::kParts) == 0 &&
         p.chunk % (SS<128>::kStep * SS<128>::kParts) == 0 &&
         p.rtile % 128 == 0 && (int64_t)p.rows * p.d * 4 < (int64_t(1) << 31);
}

gbla_status launch_state_stream(const Plan& p, const void* k, const void* v, const void* a,
                                const float* conv_w, const int32_t* cu, float* partials,
                                hipStream_t st) {
  const dim3 grid(p.units, p.heads);
  if (p.d == 128) return launch_state128(p, k, v, a, conv_w, cu, partials, st);
  if (p.d == 64) return launch_state64(p, k, v, a, conv_w, cu, partials, st);
  hipLaunchKernelGGL((state_stream_kernel<32>), grid, dim3(SS<32>::kNT), 0, st, p,
                       (const uint16_t*)k, (const uint16_t*)v, (const uint16_t*)a, conv_w, cu, partials);
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}

gbla_status launch_readout_stream(const Plan& p, const void* q, const void* r, const float* conv_w,
                                  const float* gamma, const int32_t* cu, const unsigned char* frags,
                                  float* out, hipStream_t st, KernelEvents ev) {
  const dim3 grid(p.runits, p.heads);
  const uint16_t *qq = (const uint16_t*)q, *rr = (const uint16_t*)r;
#define GBLA_READOUT(DD, NORM)                                                                \
  do {                                                                                        \
    if (ev.any())                                                                             \
      hipExtLaunchKernelGGL((readout_stream_kernel<DD, NORM>), grid, dim3(kThreads), 0, st,   \
                            ev.start, ev.stop, 0, p, qq, rr, conv_w, gamma, cu, frags, out);  \
    else                                                                                      \
      hipLaunchKernelGGL((readout_stream_kernel<DD, NORM>), grid, dim3(kThreads), 0, st, p,   \
                         qq, rr, conv_w, gamma, cu, frags, out);                              \
  } while (0)
  const bool norm = gamma != nullptr;  // NULL gamma: the no-gated-norm switch
  if (p.d == 128) {
    if (norm) GBLA_READOUT(128, true); else GBLA_READOUT(128, false);
  } else if (p.d == 64) {
    if (norm) GBLA_READOUT(64, true); else GBLA_READOUT(64, false);
  } else {
    if (norm) GBLA_READOUT(32, true); else GBLA_READOUT(32, false);
  }
#undef GBLA_READOUT
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}

}  // namespace gbla
