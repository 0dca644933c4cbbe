// gbla_state64.hip -- the state reduction of the bf16 forward pass at head
// dim 64 (gfx950).
//
// One workgroup (8 waves) reduces one chunk of tokens of one (sequence, head)
// to a partial record [S_p | z_p | m_p | l_p] (Section 2.1, key-gating item:
// the matrix form K^T V and K^T 1 with K = g (.) phi(K)):
//     S_p = sum_j w_j phi(kt_j) vt_j^T,  z_p = sum_j w_j phi(kt_j),
//     w_j = exp(a_j - m_p),  m_p = max_j a_j,  l_p = sum_j w_j.
//
//   * Staging: the chunk is streamed in steps of 64 tokens.  Each step goes
//     from HBM straight into one slot of an eight-slot LDS ring (buffer loads
//     with the LDS as destination, no registers in between), four steps
//     ahead of the one being multiplied; one barrier per step.  (Deeper
//     prefetch measured slower: the whole grid's first requests then queue
//     behind each other and the first step starts later.)  A slot holds 72
//     rows of keys and of values: the step's 64 rows after the last 8 rows of
//     the step before (loaded a second time, from L2), so every conv window
//     lies inside one slot.  Every slot is its own LDS array, so the compiler
//     tells the slots apart and waits only for the step it reads.  Rows are
//     128 bytes; the 16-byte chunks of row r are stored at chunk ^ 2 (r & 3),
//     so the four rows of a transposed read fall on four different 32-byte
//     bank groups.  Rows outside the sequence read as zero (the buffer range),
//     which is also the conv's zero padding.
//   * Waves: wave w takes key channels 32 (w / 4) .. + 31 and the 16-token
//     part (w % 4) of every step, and holds the products with all 64 value
//     channels (two 32x32 tiles, v_mfma_f32_32x32x16_bf16).
//   * Keys: ds_read_b64_tr_b16 hands each lane four consecutive tokens of one
//     channel; three reads give the twelve-row window of its eight tokens, so
//     the key conv, phi and the gate weight are applied in registers and the
//     result is the A operand (32 key channels x 16 tokens).
//   * Values: the conv is linear and per channel, so it is moved past the
//     token sum (taps u_tau, tap 3 on the current token):
//         S_p[c][e] = sum_tau u_tau[e] M_tau[c][e],
//         M_tau     = sum_j w_j phi(kt_j) v_{j-3+tau}^T,
//     each M_tau an MFMA accumulator fed with raw bf16 value rows at a shift
//     of tau - 3 tokens (odd shifts take one alignbit per dword).  v enters
//     the products exactly; the taps are applied once, in fp32, at the end.
//   * Overlap: in step i a wave multiplies A(i - 1) with the value rows of
//     step i - 1 while it forms A(i) from the keys of step i; the two are
//     independent, so the matrix core runs while the vector unit works.
//   * One gate maximum m_p for the whole chunk, so the four parts' states
//     add without rescaling; they are summed in LDS in part order.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "gbla_device.h"
#include "gbla_plan.h"

namespace gbla {
namespace {

struct S64 {
  static constexpr int D = 64;
  static constexpr int kWaves = 8;
  static constexpr int kNT = 64 * kWaves;
  static constexpr int kStep = 64;                     // tokens per ring slot
  static constexpr int kPart = 16;                     // tokens of a wave per step (MFMA K)
  static constexpr int kHalo = 8;                      // rows of the step before
  static constexpr int kRows = kHalo + kStep;
  static constexpr int kRowBytes = 2 * D;              // one bf16 row
  static constexpr int kHalf = kRows * kRowBytes;      // keys (or values) of a slot: 9 KB
  static constexpr int kSlotBytes = 2 * kHalf;
  static constexpr int kSlots = 8;
  static constexpr int kAhead = 4;                     // steps in flight past the current one
  static constexpr int kMaxChunk = 2048;
  static constexpr int kStepBytes = kStep * kRowBytes;  // bytes of one tensor per step in memory
};
static_assert(S64::kStep == S64::kWaves * 8, "one 1 KB load of eight rows per wave and tensor");
static_assert(S64::kMaxChunk == S64::kWaves * 256, "gate pass: 256 tokens per wave");

// The ring: one array per slot (keys at 0, values at kHalf).
__shared__ __attribute__((aligned(16))) unsigned char st64_r0[S64::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st64_r1[S64::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st64_r2[S64::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st64_r3[S64::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st64_r4[S64::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st64_r5[S64::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st64_r6[S64::kSlotBytes];
__shared__ __attribute__((aligned(16))) unsigned char st64_r7[S64::kSlotBytes];
__shared__ __attribute__((aligned(16))) float st64_wts[S64::kMaxChunk];  // gate weights
__shared__ __attribute__((aligned(16))) float st64_vtap[S64::D][4];      // value taps
__shared__ __attribute__((aligned(16))) float st64_z[4 * S64::D];        // z of each part
__shared__ float st64_red[2 * S64::kWaves];                              // wave maxima and sums

template <int I>
__device__ __forceinline__ unsigned char* ring64() {
  static_assert(I >= 0 && I < S64::kSlots, "slot");
  if constexpr (I == 0) return st64_r0;
  else if constexpr (I == 1) return st64_r1;
  else if constexpr (I == 2) return st64_r2;
  else if constexpr (I == 3) return st64_r3;
  else if constexpr (I == 4) return st64_r4;
  else if constexpr (I == 5) return st64_r5;
  else if constexpr (I == 6) return st64_r6;
  else return st64_r7;
}

template <int I>
using IC = std::integral_constant<int, I>;

// Byte offset of (stored row r, element e) in a key or value half-slot; e a
// multiple of 4.  Token row t of the step is stored row t + kHalo.
__device__ __forceinline__ int roff(int r, int e) {
  const int c = e >> 3;
  return r * S64::kRowBytes + ((c ^ (2 * (r & 3))) << 4) + ((e & 4) << 1);
}

__device__ __forceinline__ u32x2_t trr(const unsigned char* p) {
  return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                                         (__attribute__((address_space(3))) i16x4_t*)(p)));
}

// 16 bytes per lane from the buffer into LDS at base + 16 * lane.
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, unsigned char* base, uint32_t off) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)base, 16,
                                           off, 0, 0, 0);
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

// Keeps the compiler from hoisting address arithmetic on x out of a step
// (one add per read is cheaper than eight slots' worth of live addresses).
__device__ __forceinline__ void opaque(int& x) { asm volatile("" : "+v"(x)); }

__global__ void __launch_bounds__(S64::kNT, 1)
state64_kernel(Plan P, const uint16_t* __restrict__ kin, const uint16_t* __restrict__ vin,
               const uint16_t* __restrict__ ain, const float* __restrict__ conv_w,
               const int32_t* __restrict__ cu, float* __restrict__ partials) {
  using C = S64;
  constexpr int D = C::D;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kh = wave >> 2;    // key channels 32 kh .. 32 kh + 31
  const int part = wave & 3;   // tokens 16 part .. 16 part + 15 of every step
  const bool halo = wave == C::kWaves - 1;  // also loads the next slot's halo rows
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

  // ---- loop-invariant loads first: taps, the wave's 256 gate logits ----
  constexpr float kLog2e = 1.4426950408889634f, kLn2 = 0.6931471805599453f;
  const int kch = 32 * kh + (lane & 31);  // the lane's key channel
  float wk[4], vt[4];
  load_taps4(conv_w, P.heads, h, 1, D, P.W, kch, wk);
  load_taps4(conv_w, P.heads, h, 2, D, P.W, lane, vt);  // value channel `lane`
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

  // ---- the ring.  Lane -> (token row 8 wave + lane / 8 of a step, 16-byte
  // chunk stored at lane % 8), which loads global chunk (lane % 8) ^ 2 (row & 3);
  // the halo load (last wave) puts rows 56..63 of the step before into
  // stored rows 0..7 with the same lane pattern. ----
  const int drow = 8 * wave + (lane >> 3);
  const int dch = (lane & 7) ^ (2 * ((lane >> 3) & 3));
  const uint32_t dgoff = (uint32_t)((w0 + drow) * C::kRowBytes + dch * 16);
  // the halo rows of step `step` are rows step * 64 - 8 + lane / 8; for the
  // first step they precede the chunk (zero before the sequence start, where
  // the offset wraps out of range)
  const uint32_t hgoff = (uint32_t)((w0 - 8 + (lane >> 3)) * C::kRowBytes + dch * 16);
  auto dma_step = [&](auto slot_c, int step) {
    unsigned char* sl = ring64<decltype(slot_c)::value>();
    const uint32_t o = step < nsteps ? dgoff + (uint32_t)step * C::kStepBytes : kOutOfRange;
    unsigned char* b = sl + (C::kHalo + 8 * wave) * C::kRowBytes;
    dma16(rk, b, o);
    dma16(rv, b + C::kHalf, o);
    if (halo) {
      const uint32_t oh = step < nsteps ? hgoff + (uint32_t)step * C::kStepBytes : kOutOfRange;
      dma16(rk, sl, oh);
      dma16(rv, sl + C::kHalf, oh);
    }
  };
  // Slot 7 stands for the step before the first: zeros (its product, with
  // A = 0, adds nothing).
  dma_step(IC<7>{}, nsteps);
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
  if (lane == 0) st64_red[wave] = mloc;
  if (wave == 0) *reinterpret_cast<f32x4_t*>(st64_vtap[lane]) = f32x4_t{vt[0], vt[1], vt[2], vt[3]};
  __syncthreads();
  float mw = st64_red[0];
#pragma unroll
  for (int w = 1; w < C::kWaves; ++w) mw = fmaxf(mw, st64_red[w]);
  float lsum = 0.0f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float w = av[i] == -INFINITY ? 0.0f : __expf(av[i] - mw);
    st64_wts[256 * wave + lane + 64 * i] = w;
    lsum += w;
  }
  // The rest of the first kAhead steps: issuing them only now lets the
  // first two arrive sooner (the whole grid starts at once).
  dma_step(IC<2>{}, 2);
  dma_step(IC<3>{}, 3);
  static_assert(C::kAhead == 4, "the prologue issues steps 0..3");
  lsum = wave_sum(lsum);
  if (lane == 0) st64_red[C::kWaves + wave] = lsum;
  // The key taps carry a factor log2(e): the conv then gives kt * log2(e)
  // and phi needs only exp2.
#pragma unroll
  for (int tap = 0; tap < 4; ++tap) wk[tap] *= kLog2e;

  // ---- per-lane read offsets.  A transposed read hands the lane four
  // consecutive rows of one channel; the lane's rows start at token row
  // 16 part + 8 half - 4 + (j / 4) (stored rows + kHalo).  Rows four apart
  // have the same swizzle, so +512 bytes is four rows further. ----
  const int half = lane >> 5;
  const int grp = (lane >> 4) & 1;
  const int j = lane & 15;
  const int srow0 = C::kHalo + C::kPart * part + 8 * half - 4 + (j >> 2);
  const int ke = 32 * kh + 16 * grp + 4 * (j & 3);  // first key channel the lane reads
  const int ve = 16 * grp + 4 * (j & 3);            // first value channel (tile 0)
  const int ko = roff(srow0, ke);
  // value window of shift tau: token rows 8 half - 3 + tau .. + 7
  int vo[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) vo[t] = C::kHalf + roff(srow0 + 1 + t, ve);
  const int wlo = (C::kPart * part + 8 * half) * 4;  // byte offset of the lane's gate weights

  f32x16_t acc[4][2];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[u][b][i] = 0.0f;
  float zacc = 0.0f;  // z of key channel kch over the lane's tokens, fp32 from the unrounded A
  u32x4_t A = {0u, 0u, 0u, 0u};

  struct KeyIn {
    u32x2_t t[3];
    f32x4_t wa, wb;
  };
  // the twelve-row key window and the gate weights of step i (slot sl)
  auto kread = [&](auto slot_c, int i) {
    unsigned char* sl = ring64<decltype(slot_c)::value>();
    int a0 = ko, aw = wlo + 256 * i;
    opaque(a0); opaque(aw);
    KeyIn r;
    r.t[0] = trr(sl + a0);
    r.t[1] = trr(sl + a0 + 512);
    r.t[2] = trr(sl + a0 + 1024);
    const unsigned char* wb = reinterpret_cast<const unsigned char*>(st64_wts) + aw;
    r.wa = *reinterpret_cast<const f32x4_t*>(wb);
    r.wb = *reinterpret_cast<const f32x4_t*>(wb + 16);
    return r;
  };
  // A = w phi(kt) of key channel kch over the lane's eight tokens; the
  // window holds token rows 8 half - 4 .. + 11, four per read.
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
  // The products of A with the value rows in slot sl, both 32-channel tiles:
  // B[tau] = value rows of the lane's eight tokens shifted by tau - 3, read
  // directly (two transposed reads form the operand's four dwords).  Tile 1
  // is 64 bytes further along the row, which XORs the chunk index by 4.
  auto values = [&](unsigned char* sl) {
    const bf16x8_t a = __builtin_bit_cast(bf16x8_t, A);
#pragma unroll
    for (int bt = 0; bt < 2; ++bt) {
      int off[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        off[t] = vo[t] ^ (64 * bt);
        opaque(off[t]);
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const u32x2_t x = trr(sl + off[t]), y = trr(sl + off[t] + 512);
        const u32x4_t B = {x[0], x[1], y[0], y[1]};
        acc[t][bt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, __builtin_bit_cast(bf16x8_t, B),
                                                             acc[t][bt], 0, 0, 0);
      }
    }
  };
  // values() on the rows in slot sl with the current A, and A formed anew
  // from the key window kr, the eight products spread through the vector
  // work of kcompute so that the matrix core and the vector unit overlap.
  auto values_keys = [&](unsigned char* sl, const KeyIn& kr) {
    values(sl);
    kcompute(kr);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
      __builtin_amdgcn_sched_group_barrier(0x002, 10, 0);  // ten vector ALU
    }
  };

  // One step i in slot sl: wait for this wave's loads of step i, barrier,
  // load step i + kAhead into the slot of step i - 4, then multiply A(i - 1)
  // with the value rows of step i - 1 while A(i) is formed from the keys of
  // step i (the products and the vector work are independent, so the matrix
  // core runs while the vector unit works).
  auto step = [&](auto slot_c, int i) {
    constexpr int sl = decltype(slot_c)::value;
    if (halo)
      wait_vm<4 * (C::kAhead - 1)>();
    else
      wait_vm<2 * (C::kAhead - 1)>();
    ring_sync();
    dma_step(IC<(sl + C::kAhead) % C::kSlots>{}, i + C::kAhead);
    const KeyIn kr = kread(slot_c, i);
    values_keys(ring64<(sl + C::kSlots - 1) % C::kSlots>(), kr);
  };
  // the slot of step i, picked at run time (for the last product)
  auto slot_of = [&](int i) -> unsigned char* {
    switch (i & 7) {
      case 0: return ring64<0>();
      case 1: return ring64<1>();
      case 2: return ring64<2>();
      case 3: return ring64<3>();
      case 4: return ring64<4>();
      case 5: return ring64<5>();
      case 6: return ring64<6>();
      default: return ring64<7>();
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
  }

  // ---- the record: part p's S[c][e] = sum_tau u_tau[e] M_tau[c][e] goes to
  // slot p (64 x 64 floats, row c = key channel), the parts are summed in
  // order ----
  wait_vm<0>();  // the trailing loads (out of range) land before the slots are reused
  zacc += __shfl_xor(zacc, 32);
  __syncthreads();
  {
    float* dst = reinterpret_cast<float*>(part == 0 ? ring64<0>()
                                          : part == 1 ? ring64<1>()
                                          : part == 2 ? ring64<2>() : ring64<3>());
#pragma unroll
    for (int b = 0; b < 2; ++b) {
      const int e = 32 * b + (lane & 31);
      const f32x4_t u = *reinterpret_cast<const f32x4_t*>(st64_vtap[e]);
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const int c = 32 * kh + 8 * (q / 4) + 4 * half + (q % 4);
        float sv = u[0] * acc[0][b][q];
#pragma unroll
        for (int t = 1; t < 4; ++t) sv = fmaf(u[t], acc[t][b][q], sv);
        dst[c * D + e] = sv;
      }
    }
    if (lane < 32) st64_z[part * D + kch] = zacc;
  }
  __syncthreads();
  {
    const f32x4_t* s0 = reinterpret_cast<const f32x4_t*>(ring64<0>());
    const f32x4_t* s1 = reinterpret_cast<const f32x4_t*>(ring64<1>());
    const f32x4_t* s2 = reinterpret_cast<const f32x4_t*>(ring64<2>());
    const f32x4_t* s3 = reinterpret_cast<const f32x4_t*>(ring64<3>());
#pragma unroll
    for (int x4 = tid; x4 < D * D / 4; x4 += C::kNT)
      reinterpret_cast<f32x4_t*>(rec)[x4] = ((s0[x4] + s1[x4]) + s2[x4]) + s3[x4];
    if (tid < D)
      rec[D * D + tid] = ((st64_z[tid] + st64_z[D + tid]) + st64_z[2 * D + tid]) + st64_z[3 * D + tid];
    if (tid == 0) {
      float l = 0.0f;
#pragma unroll
      for (int w = 0; w < C::kWaves; ++w) l += st64_red[C::kWaves + w];
      rec[D * D + D] = mw;
      rec[D * D + D + 1] = l;
    }
  }
}

}  // namespace

gbla_status launch_state64(const Plan& p, const void* k, const void* v, const void* a,
                           const float* conv_w, const int32_t* cu, float* partials, hipStream_t st) {
  if (p.d != S64::D || p.chunk > S64::kMaxChunk || p.chunk % S64::kStep != 0)
    return GBLA_ERR_UNSUPPORTED;  // the plan never asks for this
  const dim3 grid(p.units, p.heads);
  hipLaunchKernelGGL(state64_kernel, grid, dim3(S64::kNT), 0, st, p, (const uint16_t*)k,
                     (const uint16_t*)v, (const uint16_t*)a, conv_w, cu, partials);
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}

}  // namespace gbla
