// gbla_state128.hip -- the state reduction of the bf16 forward pass at head
// dim 128 (gfx950).
//
// One workgroup (8 waves) reduces one chunk of tokens of one (sequence, head)
// to a partial record [S_p | z_p | m_p | l_p] (Section 2.1, key-gating item:
// the matrix form K^T V and K^T 1 with K = g (.) phi(K)):
//     S_p = sum_j w_j phi(kt_j) vt_j^T,  z_p = sum_j w_j phi(kt_j),
//     w_j = exp(a_j - m_p),  m_p = max_j a_j,  l_p = sum_j w_j.
//
// At d = 128 the vector ALU is as busy as the matrix core: phi(kt) costs
// about a dozen vector instructions per (token, key channel).  So every
// (token, key channel) is formed exactly once per workgroup (wave w owns key
// channels 16 w .. 16 w + 15 and all 128 value channels, over every token of
// the chunk), and the value side takes no vector work at all.
//
//   * Staging: the chunk is streamed in steps of 32 tokens.  Each step goes
//     from HBM straight into one slot of an eight-slot LDS ring (buffer loads
//     with the LDS as destination), four steps ahead of the one being
//     multiplied; one barrier per step.  A slot holds 36 rows of keys and of
//     values: the step's 32 rows after the last 4 rows of the step before
//     (loaded a second time, from L2), so every conv window lies inside one
//     slot, and every slot is its own LDS array, so that the compiler tells
//     the slots apart and waits only for the step it reads.  Rows are 256
//     bytes; the 16-byte chunks of row r are stored at chunk ^ swz(r),
//     swz(r) = 2 (r & 3) + 8 (bit 3 of r + 7), so the four rows of a
//     transposed read fall on four different 32-byte bank groups, and the
//     lane groups served together (rows eight apart) on different halves of
//     the banks.  Rows outside the sequence read as zero (the buffer range),
//     which is also the conv's zero padding.
//   * Keys: ds_read_b64_tr_b16 hands each lane four consecutive tokens of one
//     channel; three reads give the twelve-row window of its eight tokens, so
//     the key conv, phi and the gate weight are applied in registers and the
//     result is the A operand of v_mfma_f32_16x16x32_bf16 (16 key channels x
//     32 tokens).
//   * Values: the conv is linear and per channel, so it is moved past the
//     token sum (taps u_tau, tap 3 on the current token).  With i = j - 3 + tau,
//         S_p[c][e] = sum_tau u_tau[e] M_tau[c][e],
//         M_tau     = sum_i w_{i+3-tau} phi(kt_{i+3-tau}) v_i^T,
//     so each M_tau multiplies the raw bf16 value rows with the gated keys
//     shifted back by tau tokens.  The shift is applied to A, once per step
//     (a lane's eight tokens, plus the last three of the lane group before it
//     via one cross-lane read), and is shared by all eight value tiles; the
//     value rows enter the products exactly as loaded, three tokens behind
//     the keys so that every shift looks back.  The taps are applied once,
//     in fp32, at the end.  z_p is summed in fp32 from the unrounded keys.
//   * Overlap: in step i a wave multiplies A(i - 1) with the value rows of
//     step i - 1 while it forms A(i) from the keys of step i; the two are
//     independent, so the matrix core runs while the vector unit works.
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
  static constexpr int kStep = 32;                       // tokens per step (MFMA K)
  static constexpr int kHalo = 4;                        // rows of the step before
  static constexpr int kRows = kHalo + kStep;
  static constexpr int kRowBytes = 2 * D;                // one bf16 row
  static constexpr int kHalf = kRows * kRowBytes;        // keys (or values) of a slot: 9 KB
  static constexpr int kSlotBytes = 2 * kHalf;
  static constexpr int kSlots = 8;
  static constexpr int kAhead = 4;                       // steps in flight past the current one
  static constexpr int kMaxChunk = 2048;
  static constexpr int kStepBytes = kStep * kRowBytes;   // bytes of one tensor per step in memory
};
static_assert(S128::kStep == S128::kWaves * 4, "one 1 KB load of four rows per wave and tensor");
static_assert(S128::kMaxChunk == S128::kWaves * 256, "gate pass: 256 tokens per wave");
static_assert(S128::kHalo == 4, "the halo is one 1 KB load per tensor");

// The ring: one array per slot (keys at 0, values at kHalf).
__shared__ __attribute__((aligned(16))) unsigned char st128_r0[S128::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st128_r1[S128::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st128_r2[S128::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st128_r3[S128::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st128_r4[S128::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st128_r5[S128::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st128_r6[S128::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st128_r7[S128::kSlotBytes];
__shared__ __attribute__((aligned(16))) float st128_wts[S128::kMaxChunk];  // gate weights
__shared__ __attribute__((aligned(16))) float st128_vtap[S128::D][4];      // value taps
__shared__ float st128_red[2 * S128::kWaves];                              // wave maxima and sums

template <int I>
__device__ __forceinline__ unsigned char* ring128() {
  static_assert(I >= 0 && I < S128::kSlots, "slot");
  if constexpr (I == 0) return st128_r0;
  else if constexpr (I == 1) return st128_r1;
  else if constexpr (I == 2) return st128_r2;
  else if constexpr (I == 3) return st128_r3;
  else if constexpr (I == 4) return st128_r4;
  else if constexpr (I == 5) return st128_r5;
  else if constexpr (I == 6) return st128_r6;
  else return st128_r7;
}

template <int I>
using IC = std::integral_constant<int, I>;

// The chunk swizzle of stored row r (see the file comment).  It only flips
// bits 1..3 of the chunk index, so in a row, XOR of a byte offset with 32 nb
// moves it from channel group 0 to channel group nb.
__device__ __forceinline__ int swz(int r) { return 2 * (r & 3) + 8 * (((r + 7) >> 3) & 1); }

__device__ __forceinline__ u32x2_t trr(const unsigned char* p) {
  return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                         (__attribute__((address_space(3))) i16x4_t*)(p)));
}

// A buffer resource over `bytes` bytes from `base`, as four scalar registers
// (the same descriptor as make_rsrc).
__device__ __forceinline__ u32x4_t rsrc_sgprs(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return u32x4_t{(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a),
                 (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32)),
                 (uint32_t)__builtin_amdgcn_readfirstlane((int)bytes), 0x00020000u};
}

// 16 bytes per lane from the buffer into LDS at base + 16 * lane: a buffer
// load with the LDS as destination (M0 = base; one wait state after writing
// M0).  Written as assembly so that the compiler does not track these loads:
// its wait-count pass loses track of which slot a load writes at the loop
// head and would then wait there for every load in flight.  The waits for
// these loads are the explicit vmcnt waits of the step loop, and no other
// vector-memory load is in flight while the ring is read.
__device__ __forceinline__ void dma16(const u32x4_t& r, unsigned char* base, uint32_t off) {
  const uint32_t m = (uint32_t)__builtin_amdgcn_readfirstlane(
      (int)(uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)base);
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(off), "s"(r), "s"(m)
               : "memory", "m0");
}

// s_waitcnt vmcnt(N), the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// The barrier of a step, with no fence.  Only the loads into LDS write the
// ring, and each wave has waited (vmcnt) for its own loads of the slot read
// next before it arrives, so after the barrier that slot is complete.  A
// workgroup fence here would make every wave wait for all of its loads in
// flight, the later steps' too, which ends the prefetch.  The clobber keeps
// the compiler from moving LDS accesses across the barrier.
__device__ __forceinline__ void ring_sync() { asm volatile("s_barrier" ::: "memory"); }

// Ragged batches are reduced longest unit first: lengths follow a wide
// distribution, and with one workgroup per CU the grid otherwise ends on a
// tail of long chunks that started last.  Rank r of a head takes, in order,
// every full chunk (sequence order), then the last, partial chunk of each
// sequence (an empty sequence counts as one of zero tokens) by its number of
// 32-token steps, most first, ties in sequence order.  Every thread of the
// block calls these helpers.

// The n-th unit in sequence order, where sequence s owns cnt(s) units:
// sets *s_out and *idx_out and returns true, or returns false and sets
// *total to the number of units when n is past them.
template <int NT, typename Cnt>
__device__ __forceinline__ bool locate_by(int nseq, int n, Cnt cnt, int* red, int* s_out,
                                          int* idx_out, int* total) {
  __shared__ int found[2];
  if (threadIdx.x == 0) found[0] = -1;
  int running = 0;
  for (int base = 0; base < nseq; base += NT) {
    const int sq = base + (int)threadIdx.x;
    const int c = sq < nseq ? cnt(sq) : 0;
    int all;
    const int incl = block_incl_scan<NT>(c, red, &all);
    if (sq < nseq && n >= running + incl - c && n < running + incl) {
      found[0] = sq;
      found[1] = n - running - (incl - c);
    }
    __syncthreads();
    if (found[0] >= 0) break;
    running += all;
  }
  *s_out = found[0];
  *idx_out = found[1];
  *total = running;
  __syncthreads();  // found[] is reused by the next call
  return *s_out >= 0;
}

// Rank r -> (sequence, chunk index, record slot units_before(s) + chunk).
template <int NT>
__device__ __forceinline__ bool lpt_unit(const int32_t* cu, int nseq, int unit, int r, int* s_out,
                                         int* idx_out, int* slot_out) {
  constexpr int kBuckets = S128::kMaxChunk / S128::kStep + 1;
  __shared__ int red[NT / 64];
  __shared__ int hist[kBuckets];
  __shared__ int pick[2];
  auto len = [&](int sq) { return (int64_t)cu[sq + 1] - cu[sq]; };
  auto full = [&](int sq) { return (int)(len(sq) / unit); };
  auto partial = [&](int sq) { const int64_t n = len(sq); return n == 0 || n % unit != 0; };
  auto bucket = [&](int sq) { return (int)((len(sq) % unit + S128::kStep - 1) / S128::kStep); };
  int s, idx, nfull;
  if (!locate_by<NT>(nseq, r, full, red, &s, &idx, &nfull)) {
    for (int b = threadIdx.x; b < kBuckets; b += NT) hist[b] = 0;
    __syncthreads();
    for (int sq = threadIdx.x; sq < nseq; sq += NT)
      if (partial(sq)) atomicAdd(&hist[bucket(sq)], 1);
    __syncthreads();
    if (threadIdx.x == 0) {
      int q = r - nfull;
      pick[0] = -1;
      for (int b = kBuckets - 1; b >= 0; --b) {
        if (q < hist[b]) {
          pick[0] = b;
          pick[1] = q;
          break;
        }
        q -= hist[b];
      }
    }
    __syncthreads();
    const int pb = pick[0], pq = pick[1];
    if (pb < 0) return false;  // past the last unit of the head
    int in_bucket, unused;
    if (!locate_by<NT>(nseq, pq, [&](int sq) { return partial(sq) && bucket(sq) == pb ? 1 : 0; },
                       red, &s, &in_bucket, &unused))
      return false;  // not reached: the histogram counted this unit
    idx = full(s);
  }
  int before = 0;
  for (int sq = threadIdx.x; sq < s; sq += NT) before += units_of(len(sq), unit);
  int all;
  (void)block_incl_scan<NT>(before, red, &all);
  *s_out = s;
  *idx_out = idx;
  *slot_out = all + idx;
  return true;
}

__global__ void __launch_bounds__(S128::kNT, 1)
state128_kernel(Plan P, const uint16_t* __restrict__ kin, const uint16_t* __restrict__ vin,
                const uint16_t* __restrict__ ain, const float* __restrict__ conv_w,
                const int32_t* __restrict__ cu, float* __restrict__ partials) {
  using C = S128;
  constexpr int D = C::D;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  // dense: grid (units, heads) in sequence order; ragged: one dimension,
  // heads innermost, longest unit first
  const int h = P.ragged ? (int)(blockIdx.x % P.heads) : (int)blockIdx.y;
  int s, chunk, g;
  if (P.ragged) {
    if (!lpt_unit<C::kNT>(cu, P.nseq, P.chunk, (int)(blockIdx.x / P.heads), &s, &chunk, &g)) return;
  } else {
    g = blockIdx.x;
    if (!unit_of<C::kNT>(P, cu, P.chunk, P.chunks_per_seq, g, &s, &chunk)) return;
  }
  s = __builtin_amdgcn_readfirstlane(s);
  chunk = __builtin_amdgcn_readfirstlane(chunk);
  g = __builtin_amdgcn_readfirstlane(g);
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int64_t t0 = (int64_t)chunk * P.chunk;
  const int64_t t1 = min(len, t0 + (int64_t)P.chunk);
  const int w0 = (int)t0;  // slice-relative first token
  const int ntok = t1 > t0 ? (int)(t1 - t0) : 0;
  const int nsteps = (ntok + C::kStep - 1) / C::kStep;
  float* rec = partials + ((size_t)h * P.units + g) * P.rec_floats;

  const u32x4_t rk = rsrc_sgprs(kin + base_row * D, (uint32_t)(len * 2 * D));
  const u32x4_t rv = rsrc_sgprs(vin + base_row * D, (uint32_t)(len * 2 * D));
  // no logits (uniform gates): an empty range, so every logit reads as 0
  const __amdgpu_buffer_rsrc_t ra =
      ain ? make_rsrc(ain + base_row, (uint32_t)(len * 2)) : make_rsrc(kin, 0u);

  // ---- loop-invariant loads first: taps, the wave's 256 gate logits ----
  constexpr float kLog2e = 1.4426950408889634f, kLn2 = 0.6931471805599453f;
  const int gq = lane >> 4, j = lane & 15;  // MFMA lane roles: token group, row/column
  float wk[4], vt[4];
  load_taps4(conv_w, P.heads, h, 1, D, P.W, 16 * wave + j, wk);  // key channel 16 wave + j
  load_taps4(conv_w, P.heads, h, 2, D, P.W, (64 * wave + lane) & (D - 1), vt);
  uint32_t abits[4];
  float amask[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int tok = 256 * wave + lane + 64 * i;
    const bool valid = tok < ntok;
    abits[i] = __builtin_amdgcn_raw_buffer_load_b16(ra, valid ? (uint32_t)(w0 + tok) * 2u : kOutOfRange,
                                                    0, 0);
    amask[i] = valid ? 0.0f : -INFINITY;
  }

  // ---- the ring.  Lane -> (token row 4 wave + lane / 16 of a step, 16-byte
  // chunk stored at lane % 16), which loads global chunk (lane % 16) ^ swz(row)
  // of the stored row.
  // Waves 0 and 1 also load the halo of the keys and of the values: rows
  // 28..31 of the step before, into stored rows 0..3, with the same lane
  // pattern. ----
  const int drow = lane >> 4;
  const int dch = (lane & 15) ^ swz(C::kHalo + 4 * wave + drow);
  const uint32_t dgoff = (uint32_t)((w0 + 4 * wave + drow) * C::kRowBytes + dch * 16);
  const int hch = (lane & 15) ^ swz(drow);
  // the halo rows of step `step` are rows step * 32 - 4 + lane / 16; for the
  // first step they precede the chunk (zero before the sequence start, where
  // the offset wraps out of range)
  const uint32_t hgoff = (uint32_t)((w0 - C::kHalo + drow) * C::kRowBytes + hch * 16);
  const bool halo = wave < 2;
  const u32x4_t rh = wave == 0 ? rk : rv;
  const int hdst = wave == 0 ? 0 : C::kHalf;
  // Step `step` into its slot: its rows while step < nsteps; its halo while
  // step <= nsteps (the step after the last still multiplies the last rows
  // of the chunk, see below); zeros otherwise.
  auto dma_step = [&](auto slot_c, int step) {
    unsigned char* sl = ring128<decltype(slot_c)::value>();
    const uint32_t o = step < nsteps ? dgoff + (uint32_t)step * C::kStepBytes : kOutOfRange;
    unsigned char* b = sl + (C::kHalo + 4 * wave) * C::kRowBytes;
    dma16(rk, b, o);
    dma16(rv, b + C::kHalf, o);
    if (halo) {
      const uint32_t oh = step <= nsteps ? hgoff + (uint32_t)step * C::kStepBytes : kOutOfRange;
      dma16(rh, sl + hdst, oh);
    }
  };
  // Slot 7 stands for the step before the first: zeros (its product, with
  // A = 0, adds nothing).
  dma_step(IC<7>{}, nsteps + 1);
  dma_step(IC<0>{}, 0);
  dma_step(IC<1>{}, 1);
  __builtin_amdgcn_sched_barrier(0);

  // ---- gate weights of the chunk: m, w_j = exp(a_j - m), l ----
  float av[4];
  float mloc = -INFINITY;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    av[i] = __uint_as_float(abits[i] << 16) + amask[i];
    mloc = fmaxf(mloc, av[i]);
  }
  mloc = wave_max(mloc);
  if (lane == 0) st128_red[wave] = mloc;
  if (wave < 2)
    *reinterpret_cast<f32x4_t*>(st128_vtap[64 * wave + lane]) = f32x4_t{vt[0], vt[1], vt[2], vt[3]};
  __syncthreads();
  float mw = st128_red[0];
#pragma unroll
  for (int w = 1; w < C::kWaves; ++w) mw = fmaxf(mw, st128_red[w]);
  float lsum = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float w = av[i] == -INFINITY ? 0.0f : __expf(av[i] - mw);
    st128_wts[256 * wave + lane + 64 * i] = w;
    lsum += w;
  }
  // The rest of the first kAhead steps: issuing them only now lets the
  // first two arrive sooner (the whole grid starts at once).
  dma_step(IC<2>{}, 2);
  dma_step(IC<3>{}, 3);
  static_assert(C::kAhead == 4, "the prologue issues steps 0..3");
  lsum = wave_sum(lsum);
  if (lane == 0) st128_red[C::kWaves + wave] = lsum;
  // The key taps carry a factor log2(e): the conv then gives kt * log2(e)
  // and phi needs only exp2.
#pragma unroll
  for (int tap = 0; tap < 4; ++tap) wk[tap] *= kLog2e;

  // ---- per-lane read offsets.  A transposed read hands the lane four
  // consecutive rows of one channel, the rows chosen by lanes j / 4.
  //   keys:   token rows 8 gq - 4 + j / 4 + 4 k (k = 0, 1, 2) of channels
  //           16 wave + 4 (j % 4) .. + 3: the conv window of tokens 8 gq .. + 7;
  //   values: token rows 8 gq - 3 + j / 4 + 4 k (k = 0, 1) of channels
  //           16 nb + 4 (j % 4) .. + 3; tile nb is the offset ^ 32 nb. ----
  auto roff = [&](int r, int cc) {  // stored row r, 16-byte channel chunk cc, lane's half
    return r * C::kRowBytes + ((cc ^ swz(r)) << 4) + ((j & 1) << 3);
  };
  const int kr0 = C::kHalo + 8 * gq - 4 + (j >> 2);
  const int kcc = 2 * wave + ((j & 3) >> 1);
  const int ko[3] = {roff(kr0, kcc), roff(kr0 + 4, kcc), roff(kr0 + 8, kcc)};
  const int vr0 = C::kHalo + 8 * gq - 3 + (j >> 2);
  // (rows vr0 and vr0 + 4 have the same swizzle: 1024 bytes apart)
  const int vo = C::kHalf + roff(vr0, (j & 3) >> 1);
  const int wlo = 32 * gq;  // byte offset of the lane's gate weights within a step

  f32x4_t acc[4][C::D / 16];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int b = 0; b < C::D / 16; ++b) acc[u][b] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
  float zacc = 0.0f;  // z of key channel 16 wave + j over the lane's tokens, fp32
  u32x4_t A = {0u, 0u, 0u, 0u};
  // A shifted back by tau = 0..3 tokens (the operands of the four products)
  // and the last two dwords of the step before's group 3 (for group 0).
  u32x4_t Ash[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) Ash[t] = u32x4_t{0u, 0u, 0u, 0u};
  uint32_t c2 = 0u, c3 = 0u;

  struct KeyIn {
    u32x2_t t[3];
    f32x4_t wa, wb;
  };
  // the twelve-row key window and the gate weights of step i (slot sl)
  auto kread = [&](auto slot_c, int i) {
    unsigned char* sl = ring128<decltype(slot_c)::value>();
    const int a0 = ko[0], a1 = ko[1], a2 = ko[2], aw = wlo + 128 * i;
    KeyIn r;
    r.t[0] = trr(sl + a0);
    r.t[1] = trr(sl + a1);
    r.t[2] = trr(sl + a2);
    const unsigned char* wb = reinterpret_cast<const unsigned char*>(st128_wts) + aw;
    r.wa = *reinterpret_cast<const f32x4_t*>(wb);
    r.wb = *reinterpret_cast<const f32x4_t*>(wb + 16);
    return r;
  };
  // A(i - 1) shifted back by tau = 0..3 tokens, from A and the last three
  // tokens of the lane group before (lane - 16), or, for group 0, of the step
  // before's group 3 (kept from the last step's cross-lane read).
  auto shifts = [&]() {
    const uint32_t r2 = (uint32_t)__shfl((int)A[2], lane + 48);
    const uint32_t r3 = (uint32_t)__shfl((int)A[3], lane + 48);
    const uint32_t p2 = gq == 0 ? c2 : r2, p3 = gq == 0 ? c3 : r3;
    c2 = r2;
    c3 = r3;
    const uint32_t s0 = __builtin_amdgcn_alignbit(A[0], p3, 16);
    const uint32_t s1 = __builtin_amdgcn_alignbit(A[1], A[0], 16);
    const uint32_t s2 = __builtin_amdgcn_alignbit(A[2], A[1], 16);
    const uint32_t s3 = __builtin_amdgcn_alignbit(A[3], A[2], 16);
    Ash[0] = A;
    Ash[1] = u32x4_t{s0, s1, s2, s3};
    Ash[2] = u32x4_t{p3, A[0], A[1], A[2]};
    Ash[3] = u32x4_t{__builtin_amdgcn_alignbit(p3, p2, 16), s0, s1, s2};
  };
  // The value rows of tile nb (value channels 16 nb .. + 15) of the lane's
  // eight tokens, three behind the keys, in slot sl: two transposed reads
  // form the B operand's four dwords.
  auto vread = [&](unsigned char* sl, int nb) {
    const int o = vo ^ (32 * nb);
    const u32x2_t x = trr(sl + o), y = trr(sl + o + 1024);
    return u32x4_t{x[0], x[1], y[0], y[1]};
  };
  // One step's arithmetic, as eight blocks: block nb reads the value rows of
  // tile nb + 2, multiplies tile nb with the four shifts of A(i - 1) (rows
  // in slot sp), and forms w phi(kt) of the lane's token nb of step i (key
  // channel 16 wave + j; the key conv window kr).  The blocks are kept in
  // this order (scheduling barriers), so that the matrix core, the vector
  // unit and the LDS all work at once and each read has a block to land in.
  // Then A(i) is packed to bf16 and shifted.  With A(i - 1) = 0 (the first
  // step) the products add nothing.
  auto step_work = [&](unsigned char* sp, const KeyIn& kr) {
    bf16x8_t a[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) a[t] = __builtin_bit_cast(bf16x8_t, Ash[t]);
    u32x4_t B = vread(sp, 0), B1 = vread(sp, 1);
    __builtin_amdgcn_sched_barrier(0);  // the step's first reads all issued before any wait
    const float wj[8] = {kr.wa[0], kr.wa[1], kr.wa[2], kr.wa[3],
                         kr.wb[0], kr.wb[1], kr.wb[2], kr.wb[3]};
    float xk[12];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
      xk[4 * q + 0] = bf16_lo(kr.t[q][0]); xk[4 * q + 1] = bf16_hi(kr.t[q][0]);
      xk[4 * q + 2] = bf16_lo(kr.t[q][1]); xk[4 * q + 3] = bf16_hi(kr.t[q][1]);
    }
    float kw[8];
#pragma unroll
    for (int nb = 0; nb < C::D / 16; ++nb) {
      u32x4_t B2;
      if (nb + 2 < C::D / 16) B2 = vread(sp, nb + 2);
      const bf16x8_t b = __builtin_bit_cast(bf16x8_t, B);
#pragma unroll
      for (int t = 0; t < 4; ++t)
        acc[t][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[t], b, acc[t][nb], 0, 0, 0);
      // token o = nb: kt * log2(e) from its window, then
      // phi(x) = max(x, 0) + exp(min(x, 0)) = ln2 max(x', 0) + 2^min(x', 0)
      const int o = nb;
      float kc = wk[0] * xk[o + 1];
#pragma unroll
      for (int tap = 1; tap < 4; ++tap) kc = fmaf(wk[tap], xk[o + 1 + tap], kc);
      const float ph = fmaf(kLn2, fmaxf(kc, 0.0f), __builtin_amdgcn_exp2f(fminf(kc, 0.0f)));
      kw[o] = wj[o] * ph;
      zacc += kw[o];
      // in the block, each product is followed by a few vector instructions,
      // which issue while the product runs
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 3, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      B = B1;
      if (nb + 2 < C::D / 16) B1 = B2;
    }
#pragma unroll
    for (int p = 0; p < 4; ++p) A[p] = pack_bf16x2(kw[2 * p], kw[2 * p + 1]);
    shifts();
  };
  // The last products (no keys to form): tile by tile, reads one tile ahead.
  auto values = [&](unsigned char* sp) {
    bf16x8_t a[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) a[t] = __builtin_bit_cast(bf16x8_t, Ash[t]);
    u32x4_t B = vread(sp, 0);
#pragma unroll
    for (int nb = 0; nb < C::D / 16; ++nb) {
      u32x4_t Bn;
      if (nb + 1 < C::D / 16) Bn = vread(sp, nb + 1);
      const bf16x8_t b = __builtin_bit_cast(bf16x8_t, B);
#pragma unroll
      for (int t = 0; t < 4; ++t)
        acc[t][nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[t], b, acc[t][nb], 0, 0, 0);
      if (nb + 1 < C::D / 16) B = Bn;
    }
  };

  // One step i in slot sl.  Every other step (i even): wait for this wave's
  // loads of steps i and i + 1, barrier, load steps i + kAhead and
  // i + kAhead + 1 into the slots of steps i - 4 and i - 3 (one barrier per
  // two steps halves the steps' fixed costs).  Then multiply the shifts of
  // A(i - 1) with the value rows of step i - 1 while A(i) is formed from the
  // keys of step i.
  auto step = [&](auto slot_c, int i) {
    constexpr int sl = decltype(slot_c)::value;
    if constexpr (sl % 2 == 0) {
      if (halo)
        wait_vm<3 * (C::kAhead - 2)>();
      else
        wait_vm<2 * (C::kAhead - 2)>();
      ring_sync();
      dma_step(IC<(sl + C::kAhead) % C::kSlots>{}, i + C::kAhead);
      dma_step(IC<(sl + C::kAhead + 1) % C::kSlots>{}, i + C::kAhead + 1);
    }
    const KeyIn kr = kread(slot_c, i);
    step_work(ring128<(sl + C::kSlots - 1) % C::kSlots>(), kr);
  };
  // the slot of step i, picked at run time (for the last products)
  auto slot_of = [&](int i) -> unsigned char* {
    switch (i & 7) {
      case 0: return ring128<0>();
      case 1: return ring128<1>();
      case 2: return ring128<2>();
      case 3: return ring128<3>();
      case 4: return ring128<4>();
      case 5: return ring128<5>();
      case 6: return ring128<6>();
      default: return ring128<7>();
    }
  };
  if (nsteps > 0) {
    for (int i = 0;; i += C::kSlots) {
      step(IC<0>{}, i);
      if (i + 1 >= nsteps) break;
      step(IC<1>{}, i + 1);
      if (i + 2 >= nsteps) break;
      step(IC<2>{}, i + 2);
      if (i + 3 >= nsteps) break;
      step(IC<3>{}, i + 3);
      if (i + 4 >= nsteps) break;
      step(IC<4>{}, i + 4);
      if (i + 5 >= nsteps) break;
      step(IC<5>{}, i + 5);
      if (i + 6 >= nsteps) break;
      step(IC<6>{}, i + 6);
      if (i + 7 >= nsteps) break;
      step(IC<7>{}, i + 7);
      if (i + 8 >= nsteps) break;
    }
    values(slot_of(nsteps - 1));
    // The value rows run three tokens behind the keys: the last three rows
    // of the chunk still meet the shifted keys of its last tokens, in the
    // slot of step nsteps (its halo; the rest reads as zero or meets A = 0).
    A = u32x4_t{0u, 0u, 0u, 0u};
    shifts();
  }
  wait_vm<0>();  // every load has landed, including the trailing ones
  __syncthreads();
  if (nsteps > 0) values(slot_of(nsteps));

  // ---- the record: S[c][e] = sum_tau u_tau[e] M_tau[c][e] for key channels
  // c = 16 wave + 4 gq + q and value channels e = 16 nb + j ----
#pragma unroll
  for (int nb = 0; nb < C::D / 16; ++nb) {
    const f32x4_t u = *reinterpret_cast<const f32x4_t*>(st128_vtap[16 * nb + j]);
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
  if (tid == 0) {
    float l = 0.0f;
#pragma unroll
    for (int w = 0; w < C::kWaves; ++w) l += st128_red[C::kWaves + w];
    rec[D * D + D] = mw;
    rec[D * D + D + 1] = l;
  }
}

}  // namespace

gbla_status launch_state128(const Plan& p, const void* k, const void* v, const void* a,
                            const float* conv_w, const int32_t* cu, float* partials, hipStream_t st) {
  if (p.d != S128::D || p.chunk > S128::kMaxChunk || p.chunk % S128::kStep != 0)
    return GBLA_ERR_UNSUPPORTED;  // the plan never asks for this
  const dim3 grid = p.ragged ? dim3((unsigned)p.units * (unsigned)p.heads) : dim3(p.units, p.heads);
  hipLaunchKernelGGL(state128_kernel, grid, dim3(S128::kNT), 0, st, p, (const uint16_t*)k,
                     (const uint16_t*)v, (const uint16_t*)a, conv_w, cu, partials);
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}

}  // namespace gbla
