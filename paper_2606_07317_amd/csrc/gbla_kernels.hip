// gbla_kernels.hip -- CDNA4 (gfx950) kernels of the GBLA forward pass.
//
// The pass (Section 2.1 of the paper, with phi = elu + 1 from Section 2):
//   Conv1D      qt, kt, vt = causal depthwise conv (width W <= 4) of q, k, v
//   key gating  g = softmax_j(a_j) over the tokens of one (sequence, head)
//   state       S = sum_j g_j phi(kt_j) vt_j^T,  z = sum_j g_j phi(kt_j)
//   readout     o_i = phi(qt_i)^T S / phi(qt_i)^T z
//   gated norm  y_i = o_i / sqrt(mean(o_i^2) + eps) * gamma * SiLU(r_i)
//
// Kernels:
//   conv_kernel           the Conv1D alone (test hook): a tile of rows plus a
//                         (W-1)-row halo is staged in LDS, fp32 out.
//   state_partial_kernel  one workgroup per (head, chunk of tokens): conv of
//                         k and v fused into the loads (a per-thread sliding
//                         window), phi, gate weights exp(a - m_chunk), then
//                         the chunk's partial S_p = sum (w phi(kt)) vt^T on
//                         bf16 MFMA (fp32 accumulate) through an LDS tile
//                         stored channel-major, plus z_p, m_p and l_p.
//   combine_kernel        fixed-order rescaled sum of the partials of one
//                         (sequence, head): S, z normalised by the softmax
//                         denominator, and the readout's MFMA A-operands.
//   readout_kernel        conv of q fused into the loads (DPP row rotates
//                         supply the three previous tokens), phi, the
//                         contraction with [S^T; z^T] on MFMA, and the gated
//                         RMSNorm epilogue with a cross-lane row reduction.
//
// Data types: activations are fp32 or bf16 (raw 16-bit patterns); all
// arithmetic is fp32 except the MFMA operands of the bf16 path, which are
// rounded to bf16 (round to nearest even) and accumulated in fp32.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "gbla_device.h"
#include "gbla_plan.h"

namespace gbla {
namespace {

constexpr int kConvRows = 64;  // rows per conv_kernel tile

template <typename T>
__device__ __forceinline__ float load_scalar(const T* p, int64_t i);
template <>
__device__ __forceinline__ float load_scalar<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float load_scalar<uint16_t>(const uint16_t* p, int64_t i) {
  return __uint_as_float((uint32_t)p[i] << 16);
}

// Key-gate logit of token i; a == NULL (uniform gates) reads as 0.
template <typename T>
__device__ __forceinline__ float gate_logit(const T* a, int64_t i) {
  return a ? load_scalar<T>(a, i) : 0.0f;
}

// Unpack the 16 bytes at one thread's slot: 8 bf16 or 4 fp32 channels.
template <typename T>
__device__ __forceinline__ void unpack16(const u32x4_t& u, float* x);
template <>
__device__ __forceinline__ void unpack16<float>(const u32x4_t& u, float* x) {
#pragma unroll
  for (int i = 0; i < 4; ++i) x[i] = __uint_as_float(u[i]);
}
template <>
__device__ __forceinline__ void unpack16<uint16_t>(const u32x4_t& u, float* x) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[2 * i] = bf16_lo(u[i]);
    x[2 * i + 1] = bf16_hi(u[i]);
  }
}

// exp for the gates, phi and SiLU: the hardware exp2 path for bf16 inputs,
// the library's full-accuracy expf for fp32 inputs.
template <typename T>
__device__ __forceinline__ float gexp(float x) {
  if constexpr (sizeof(T) == 4) return expf(x);
  else return __expf(x);
}

// phi(u) = elu(u) + 1 (Section 2, BLA paragraph).
template <typename T>
__device__ __forceinline__ float phi(float u) {
  return u > 0.0f ? u + 1.0f : gexp<T>(fminf(u, 0.0f));
}

// SiLU(x) = x * sigmoid(x).
template <typename T>
__device__ __forceinline__ float silu(float x) {
  return x * __builtin_amdgcn_rcpf(1.0f + gexp<T>(-x));
}

// ---------------------------------------------------------------------------
// conv_kernel: the Conv1D alone.  grid = (row tiles, slices, 3 tensors).
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(kThreads)
conv_kernel(Plan P, const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
            const float* __restrict__ conv_w, const int32_t* __restrict__ cu,
            float* __restrict__ qt, float* __restrict__ kt, float* __restrict__ vt) {
  constexpr int CPT = 16 / (int)sizeof(T);
  constexpr int VPR = D / CPT;  // 16-byte vectors per row
  __shared__ float tile[(kConvRows + 3) * D];
  const int tensor = blockIdx.z;
  const T* x = tensor == 0 ? q : (tensor == 1 ? k : v);
  float* y = tensor == 0 ? qt : (tensor == 1 ? kt : vt);
  const int slice = blockIdx.y;
  const int h = P.ragged ? slice : slice % P.heads;
  const int64_t r0 = (int64_t)blockIdx.x * kConvRows;
  const int64_t slice_row = (int64_t)slice * P.rows;

  // Stage rows r0-3 .. r0+63 (zero outside the slice) in fp32.
  for (int i = threadIdx.x; i < (kConvRows + 3) * VPR; i += kThreads) {
    const int rr = i / VPR, vi = i % VPR;
    const int64_t row = r0 - 3 + rr;
    float xs[CPT];
    if (row >= 0 && row < P.rows) {
      unpack16<T>(load16(x + (slice_row + row) * D + vi * CPT), xs);
    } else {
#pragma unroll
      for (int c = 0; c < CPT; ++c) xs[c] = 0.0f;
    }
#pragma unroll
    for (int c = 0; c < CPT; ++c) tile[rr * D + vi * CPT + c] = xs[c];
  }
  __syncthreads();

  for (int i = threadIdx.x; i < kConvRows * D; i += kThreads) {
    const int rr = i / D, c = i % D;
    const int64_t row = r0 + rr;
    if (row >= P.rows) break;
    int64_t start = 0;  // first row of the sequence that holds `row`
    if (P.ragged) {
      int lo = 0, hi = P.nseq;  // cu[lo] <= row < cu[hi]
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (cu[mid] <= row) lo = mid; else hi = mid;
      }
      start = cu[lo];
    }
    float w4[4];
    load_taps4(conv_w, P.heads, h, tensor, D, P.W, c, w4);
    float acc = 0.0f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int64_t src = row - 3 + t;
      if (src >= start) acc = fmaf(w4[t], tile[(rr + t) * D + c], acc);
    }
    y[(slice_row + row) * D + c] = acc;
  }
}

// ---------------------------------------------------------------------------
// state_partial_kernel
// ---------------------------------------------------------------------------
template <typename T, int D>
struct StateCfg {
  static constexpr int kCPT = 16 / (int)sizeof(T);          // channels per thread
  static constexpr int kCG = D / kCPT;                       // threads per token row
  static constexpr int kRG = kThreads / kCG;                 // strips per block
  static constexpr int kTP = kRG * 8;                        // tokens per pass
  static constexpr int kPitch = kTP * (int)sizeof(T) + 16;   // LDS bytes per channel row
  // bf16: gated keys, values rounded to bf16 (hi) and the rounding residue
  // (lo), so that S_p = A^T B_hi + A^T B_lo carries only the key rounding;
  // fp32: gated keys and values.
  static constexpr int kArrays = sizeof(T) == 2 ? 3 : 2;
  static constexpr int kLds = kArrays * D * kPitch;
  static constexpr int kTiles = (D / 32) * (D / 32);         // 32x32 output tiles of S_p
  static constexpr int kTilesPerWave = kTiles >= 4 ? kTiles / 4 : 1;
};

// One pass of MFMAs over the LDS tile: S_p[c][e] += sum_slot A[c][slot] B[e][slot].
template <typename T, int D>
__device__ __forceinline__ void state_mfma_pass(const unsigned char* lds, int wave, int lane,
                                                f32x16_t* acc) {
  using C = StateCfg<T, D>;
  if (C::kTiles < 4 && wave != 0) return;
  const unsigned char* A = lds;
  const unsigned char* B = lds + D * C::kPitch;
  const unsigned char* Bl = lds + 2 * D * C::kPitch;  // bf16 path only
  // Tile assignment: D=32 -> wave 0 owns the only tile; D=64 -> wave w owns
  // (w/2, w%2); D=128 -> wave w owns row block w and column blocks 0..3.
  const int tm = D == 128 ? wave : (D == 64 ? wave >> 1 : 0);
  const int row = lane & 31, half = lane >> 5;
  if constexpr (sizeof(T) == 2) {
#pragma unroll 4
    for (int ks = 0; ks < C::kTP / 16; ++ks) {
      const int byte = (16 * ks + 8 * half) * 2;
      const u32x4_t a = *reinterpret_cast<const u32x4_t*>(A + (32 * tm + row) * C::kPitch + byte);
#pragma unroll
      for (int t = 0; t < C::kTilesPerWave; ++t) {
        const int tn = D == 128 ? t : (D == 64 ? (wave & 1) : 0);
        const u32x4_t b = *reinterpret_cast<const u32x4_t*>(B + (32 * tn + row) * C::kPitch + byte);
        const u32x4_t bl = *reinterpret_cast<const u32x4_t*>(Bl + (32 * tn + row) * C::kPitch + byte);
        acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                         __builtin_bit_cast(bf16x8_t, b), acc[t],
                                                         0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                         __builtin_bit_cast(bf16x8_t, bl), acc[t],
                                                         0, 0, 0);
      }
    }
  } else {
#pragma unroll 4
    for (int ks = 0; ks < C::kTP / 2; ++ks) {
      const int byte = (2 * ks + half) * 4;
      const float a = *reinterpret_cast<const float*>(A + (32 * tm + row) * C::kPitch + byte);
#pragma unroll
      for (int t = 0; t < C::kTilesPerWave; ++t) {
        const int tn = D == 128 ? t : (D == 64 ? (wave & 1) : 0);
        const float b = *reinterpret_cast<const float*>(B + (32 * tn + row) * C::kPitch + byte);
        acc[t] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[t], 0, 0, 0);
      }
    }
  }
}

// Write 8 consecutive slots of one channel row: bf16 pairs or fp32.
template <typename T>
__device__ __forceinline__ void lds_store_slots(unsigned char* dst, const float* v8) {
  if constexpr (sizeof(T) == 2) {
    u32x4_t w;
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(v8[2 * i], v8[2 * i + 1]);
    *reinterpret_cast<u32x4_t*>(dst) = w;
  } else {
    f32x4_t lo = {v8[0], v8[1], v8[2], v8[3]};
    f32x4_t hi = {v8[4], v8[5], v8[6], v8[7]};
    reinterpret_cast<f32x4_t*>(dst)[0] = lo;
    reinterpret_cast<f32x4_t*>(dst)[1] = hi;
  }
}

// grid = (units per head, H).  Unit g of head h reduces tokens
// [chunk * P.chunk, min(len, (chunk + 1) * P.chunk)) of its sequence to
//   S_p[c][e] = sum_j w_j phi(kt_j)[c] vt_j[e],  z_p[c] = sum_j w_j phi(kt_j)[c],
//   w_j = exp(a_j - m_p),  m_p = max_j a_j,  l_p = sum_j w_j,
// stored as the record [S_p (d*d) | z_p (d) | m_p | l_p] of the workspace.
template <typename T, int D>
__global__ void __launch_bounds__(kThreads)
state_partial_kernel(Plan P, const T* __restrict__ kin, const T* __restrict__ vin,
                     const T* __restrict__ ain, const float* __restrict__ conv_w,
                     const int32_t* __restrict__ cu, float* __restrict__ partials) {
  using C = StateCfg<T, D>;
  constexpr int CPT = C::kCPT;
  __shared__ __attribute__((aligned(16))) unsigned char lds[C::kLds];
  __shared__ float red[4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = blockIdx.y, g = blockIdx.x;
  int s, chunk;
  if (P.ragged) {
    if (!locate_unit(cu, P.nseq, P.chunk, g, &s, &chunk)) return;
  } else {
    s = g / P.chunks_per_seq;
    chunk = g - s * P.chunks_per_seq;
  }
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int64_t t0 = (int64_t)chunk * P.chunk;
  const int64_t t1 = min(len, t0 + (int64_t)P.chunk);
  float* rec = partials + ((size_t)h * P.units + g) * P.rec_floats;

  // m_p: the chunk's largest gate logit.
  float mloc = -INFINITY;
  for (int64_t t = t0 + tid; t < t1; t += kThreads) mloc = fmaxf(mloc, gate_logit<T>(ain, base_row + t));
  const float m = block_max(mloc, red);

  const int cg = tid % C::kCG, rg = tid / C::kCG;
  const int c0 = cg * CPT;
  float wk[CPT][4], wv[CPT][4];
#pragma unroll
  for (int c = 0; c < CPT; ++c) {
    load_taps4(conv_w, P.heads, h, 1, D, P.W, c0 + c, wk[c]);
    load_taps4(conv_w, P.heads, h, 2, D, P.W, c0 + c, wv[c]);
  }

  // Each thread walks its own strip of consecutive tokens, 8 per pass, so
  // the conv window slides through registers.
  const int64_t span = t1 > t0 ? t1 - t0 : 0;
  const int64_t strip = ((span + C::kRG - 1) / C::kRG + 7) / 8 * 8;
  const int npass = (int)(strip / 8);
  const int64_t s0 = t0 + rg * strip;

  float xk[11][CPT], xv[11][CPT];  // rows s-3 .. s+7 of the current pass
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    const int64_t t = s0 - 3 + i;
    if (t >= 0 && t < len && npass > 0) {
      unpack16<T>(load16(kin + (base_row + t) * D + c0), xk[i]);
      unpack16<T>(load16(vin + (base_row + t) * D + c0), xv[i]);
    } else {
#pragma unroll
      for (int c = 0; c < CPT; ++c) xk[i][c] = xv[i][c] = 0.0f;
    }
  }

  f32x16_t acc[C::kTilesPerWave];
#pragma unroll
  for (int t = 0; t < C::kTilesPerWave; ++t)
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[t][i] = 0.0f;
  float zacc[CPT];
#pragma unroll
  for (int c = 0; c < CPT; ++c) zacc[c] = 0.0f;
  float lacc = 0.0f;

  unsigned char* ldsA = lds;
  unsigned char* ldsB = lds + D * C::kPitch;
  for (int pass = 0; pass < npass; ++pass) {
    float wj[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int64_t t = s0 + 8 * pass + j;
      if (t < t1) {
        unpack16<T>(load16(kin + (base_row + t) * D + c0), xk[3 + j]);
        unpack16<T>(load16(vin + (base_row + t) * D + c0), xv[3 + j]);
        wj[j] = gexp<T>(gate_logit<T>(ain, base_row + t) - m);
      } else {
#pragma unroll
        for (int c = 0; c < CPT; ++c) xk[3 + j][c] = xv[3 + j][c] = 0.0f;
        wj[j] = 0.0f;
      }
      lacc += wj[j];
    }
#pragma unroll
    for (int c = 0; c < CPT; ++c) {
      float kw[8], vv[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float kt = 0.0f, vt = 0.0f;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          kt = fmaf(wk[c][t], xk[j + t][c], kt);
          vt = fmaf(wv[c][t], xv[j + t][c], vt);
        }
        kw[j] = wj[j] * phi<T>(kt);
        vv[j] = vt;
        zacc[c] += kw[j];
      }
      const int slot_byte = (c0 + c) * C::kPitch + rg * 8 * (int)sizeof(T);
      lds_store_slots<T>(ldsA + slot_byte, kw);
      if constexpr (sizeof(T) == 2) {
        // values as bf16 hi + bf16 lo (lo = the residue of the first rounding)
        u32x4_t hi, lo;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          hi[i] = pack_bf16x2(vv[2 * i], vv[2 * i + 1]);
          lo[i] = pack_bf16x2(vv[2 * i] - bf16_lo(hi[i]), vv[2 * i + 1] - bf16_hi(hi[i]));
        }
        *reinterpret_cast<u32x4_t*>(ldsB + slot_byte) = hi;
        *reinterpret_cast<u32x4_t*>(ldsB + D * C::kPitch + slot_byte) = lo;
      } else {
        lds_store_slots<T>(ldsB + slot_byte, vv);
      }
    }
#pragma unroll
    for (int i = 0; i < 3; ++i)
#pragma unroll
      for (int c = 0; c < CPT; ++c) {
        xk[i][c] = xk[8 + i][c];
        xv[i][c] = xv[8 + i][c];
      }
    __syncthreads();
    state_mfma_pass<T, D>(lds, wave, lane, acc);
    __syncthreads();
  }

  // S_p from the MFMA accumulators: lane l, register i holds row
  // 8*(i/4) + 4*(l/32) + i%4 and column l%32 of its 32x32 tile.
  if (C::kTiles >= 4 || wave == 0) {
    const int tm = D == 128 ? wave : (D == 64 ? wave >> 1 : 0);
#pragma unroll
    for (int t = 0; t < C::kTilesPerWave; ++t) {
      const int tn = D == 128 ? t : (D == 64 ? (wave & 1) : 0);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int c = 32 * tm + 8 * (i / 4) + 4 * (lane / 32) + (i % 4);
        const int e = 32 * tn + (lane % 32);
        rec[c * D + e] = acc[t][i];
      }
    }
  }
  // z_p and l_p: fixed-order sums over the strips through LDS.
  float* zb = reinterpret_cast<float*>(lds);  // [kRG][D]
  float* lb = zb + C::kRG * D;                // [kRG]
#pragma unroll
  for (int c = 0; c < CPT; ++c) zb[rg * D + c0 + c] = zacc[c];
  if (cg == 0) lb[rg] = lacc;
  __syncthreads();
  if (tid < D) {
    float zs = 0.0f;
    for (int i = 0; i < C::kRG; ++i) zs += zb[i * D + tid];
    rec[D * D + tid] = zs;
  }
  if (tid == 0) {
    float ls = 0.0f;
    for (int i = 0; i < C::kRG; ++i) ls += lb[i];
    rec[D * D + D] = m;
    rec[D * D + D + 1] = ls;
  }
}

// ---------------------------------------------------------------------------
// combine_kernel: grid = (N sequences, H, element blocks).
// ---------------------------------------------------------------------------
// Readout operand layout (per sequence and head): the MFMA 16x16x32 A operand
// of block (mb, kb) for lane l = 16*gq + m holds 8 values v[j], j = 0..7:
//   mb < D/16:  v[j] = S[32*kb + 8*gq + j][e(mb, m)]
//   mb = D/16:  v[j] = z[32*kb + 8*gq + j]            (the denominator block)
// with e(mb, m) = 32*(mb/2) + 8*(m/4) + 4*(mb%2) + m%4, chosen so that one
// lane's accumulators cover 8 consecutive output channels per pair of blocks.
// bf16 path: 8 bf16 (16 bytes) per lane; fp32 path: 8 floats (32 bytes).
template <int D>
struct FragCfg {
  static constexpr int kNMB = D / 16 + 1;
  static constexpr int kNKB = D / 32;
  static constexpr int kSlots = kNMB * kNKB * 64;  // lane-slots of 8 values
};

template <typename T, int D>
__device__ __forceinline__ void frag_put(void* frag_sh, int mb, int kb, int lane, int j, float v) {
  const size_t slot = ((size_t)mb * FragCfg<D>::kNKB + kb) * 64 + lane;
  if constexpr (sizeof(T) == 2) {
    const uint32_t bits = pack_bf16x2(v, 0.0f) & 0xffffu;
    reinterpret_cast<uint16_t*>(frag_sh)[slot * 8 + j] = (uint16_t)bits;
  } else {
    reinterpret_cast<float*>(frag_sh)[slot * 8 + j] = v;
  }
}

// grid = (N * H, element slices of kThreads * E).  A block stages the chunk
// weights w_p = exp(m_p - M) of its (sequence, head) in LDS and forms
// Z = sum_p w_p l_p; each thread then sums element x of every partial in the
// order p = 0, 1, ... (compensated, so that thousands of chunks keep the sum
// to a few ulps), scales by 1/Z and writes S, z and the readout fragments.  Every reduction order is fixed by the shape alone (not by E or
// the grid), so every call gives the same bits.
constexpr int kCombineStage = 1024;  // chunk weights staged in LDS per round

template <typename T, int D, int E>
__global__ void __launch_bounds__(kThreads)
combine_kernel(Plan P, const int32_t* __restrict__ cu, const float* __restrict__ partials,
               float* __restrict__ S_out, float* __restrict__ z_out, unsigned char* __restrict__ frags,
               float* __restrict__ mz_out) {
  constexpr int kElems = D * D + D;
  __shared__ float red[kThreads / 64];
  __shared__ float wst[kCombineStage];
  const int tid = threadIdx.x;
  const int sh_idx = blockIdx.x;
  const int s = sh_idx / P.heads, h = sh_idx % P.heads;
  int first, count;
  if (P.ragged) {
    first = units_before(cu, s, P.chunk);
    count = units_of((int64_t)cu[s + 1] - cu[s], P.chunk);
  } else {
    first = s * P.chunks_per_seq;
    count = P.chunks_per_seq;
  }
  const size_t rf = P.rec_floats;
  const float* recs = partials + ((size_t)h * P.units + first) * rf;

  // M = max_p m_p and Z = sum_p exp(m_p - M) l_p: thread t takes p = t,
  // t + kThreads, ... in order; the waves' sums are added in wave order.
  // With at most kThreads partials, thread t loads (m_t, l_t) once and the
  // weights are staged from registers; the arithmetic is the same.
  const bool one = count <= kThreads;
  const int pc = tid < count ? tid : 0;
  const float m1 = recs[pc * rf + kElems], l1 = recs[pc * rf + kElems + 1];
  float ml = -INFINITY;
  if (one) {
    if (tid < count) ml = m1;
  } else {
    for (int p = tid; p < count; p += kThreads) ml = fmaxf(ml, recs[p * rf + kElems]);
  }
  const float M = block_max(ml, red);
  float zl = 0.0f;
  if (M != -INFINITY) {
    if (one) {
      if (tid < count) zl = gexp<T>(m1 - M) * l1;
    } else {
      for (int p = tid; p < count; p += kThreads) {
        const float* r = recs + p * rf + kElems;
        zl = fmaf(gexp<T>(r[0] - M), r[1], zl);
      }
    }
  }
  zl = wave_sum(zl);
  __syncthreads();
  if ((tid & 63) == 0) red[tid >> 6] = zl;
  __syncthreads();
  float Z = 0.0f;
#pragma unroll
  for (int w = 0; w < kThreads / 64; ++w) Z += red[w];
  const float invZ = Z > 0.0f ? 1.0f / Z : 0.0f;
  // (M, Z) of the sequence's softmax, for the backward pass
  if (mz_out && blockIdx.y == 0 && tid == 0) {
    mz_out[2 * (size_t)sh_idx] = M;
    mz_out[2 * (size_t)sh_idx + 1] = Z;
  }

  int xe[E];
  float v[E], cmp[E];  // compensated (Kahan) sums: sequences of thousands of chunks
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int x = (blockIdx.y * E + e) * kThreads + tid;
    xe[e] = x < kElems ? x : 0;  // a valid address for every thread
    v[e] = 0.0f;
    cmp[e] = 0.0f;
  }
  for (int p0 = 0; p0 < count; p0 += kCombineStage) {
    const int n = min(kCombineStage, count - p0);
    __syncthreads();
    if (one) {
      if (tid < n) wst[tid] = M == -INFINITY || m1 == -INFINITY ? 0.0f : gexp<T>(m1 - M);
    } else {
      for (int p = tid; p < n; p += kThreads) {
        const float mp = recs[(p0 + p) * rf + kElems];
        wst[p] = M == -INFINITY || mp == -INFINITY ? 0.0f : gexp<T>(mp - M);
      }
    }
    __syncthreads();
    // unrolled so that many partials' loads are in flight at once
#pragma unroll 16
    for (int p = 0; p < n; ++p) {
      const float w = wst[p];
      const float* r = recs + (p0 + p) * rf;
#pragma unroll
      for (int e = 0; e < E; ++e) kahan_add(v[e], cmp[e], w * r[xe[e]]);
    }
  }

  const size_t sh = (size_t)s * P.heads + h;
  unsigned char* fr = frags ? frags + sh * P.frag_bytes : nullptr;
  // bf16 fragments of a slice of S alone: the slice holds R whole rows c of S
  // (all D columns), so one lane can write the G <= 8 consecutive values j
  // of a fragment slot at once, through LDS, instead of one 2-byte store per
  // element (an L2 request each).
  constexpr int R = E * kThreads / D, G = R < 8 ? R : 8;
  if constexpr (sizeof(T) == 2 && R >= 2 && R % G == 0 && 8 % G == 0) {
    if (fr && (blockIdx.y + 1) * E * kThreads <= D * D) {  // uniform
      __shared__ float tr[E * kThreads];
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int x = (blockIdx.y * E + e) * kThreads + tid;
        const float val = v[e] * invZ;
        if (S_out) S_out[sh * D * D + x] = val;
        tr[e * kThreads + tid] = val;
      }
      __syncthreads();
      const int c0 = blockIdx.y * R;  // the slice's first row of S
      for (int it = tid; it < D * (R / G); it += kThreads) {
        const int ee = it % D, g = it / D, c = c0 + g * G;
        const int kb = c / 32, gq = (c % 32) / 8, j0 = c % 8;
        const int mb = 2 * (ee / 32) + (ee % 8) / 4, m = 4 * ((ee % 32) / 8) + ee % 4;
        const size_t slot = ((size_t)mb * FragCfg<D>::kNKB + kb) * 64 + 16 * gq + m;
        uint32_t w[G / 2];
#pragma unroll
        for (int i = 0; i < G / 2; ++i)
          w[i] = pack_bf16x2(tr[(g * G + 2 * i) * D + ee], tr[(g * G + 2 * i + 1) * D + ee]);
        unsigned char* dst = fr + (slot * 8 + j0) * 2;
        if constexpr (G == 8) {
          *reinterpret_cast<u32x4_t*>(dst) = u32x4_t{w[0], w[1], w[2], w[3]};
        } else if constexpr (G == 4) {
          *reinterpret_cast<u32x2_t*>(dst) = u32x2_t{w[0], w[1]};
        } else {
          *reinterpret_cast<uint32_t*>(dst) = w[0];
        }
      }
      return;
    }
  }
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int x = (blockIdx.y * E + e) * kThreads + tid;
    if (x >= kElems) continue;
    const float val = v[e] * invZ;
    if (x < D * D) {
      const int c = x / D, ee = x % D;
      if (S_out) S_out[sh * D * D + x] = val;
      const int kb = c / 32, gq = (c % 32) / 8, j = c % 8;
      const int mb = 2 * (ee / 32) + (ee % 8) / 4, m = 4 * ((ee % 32) / 8) + ee % 4;
      if (fr) frag_put<T, D>(fr, mb, kb, 16 * gq + m, j, val);
    } else {
      const int c = x - D * D;
      if (z_out) z_out[sh * D + c] = val;
      const int kb = c / 32, gq = (c % 32) / 8, j = c % 8;
      if (fr)
        for (int m = 0; m < 16; ++m) frag_put<T, D>(fr, D / 16, kb, 16 * gq + m, j, val);
    }
  }
}


// ---------------------------------------------------------------------------
// readout_kernel: grid = (readout units per head, H).
// ---------------------------------------------------------------------------
// Lane l = 16*gq + n of a wave handles tokens tb + 4n + j (j = 0..3) of a
// group of 64 tokens, channels 32*kb + 8*gq + [0, 8) of each.  The three
// tokens before tb + 4n are tokens j = 1..3 of lane n-1 (DPP row rotate by
// one inside the 16-lane row gq), or of lane 15 of the previous group.

// Row rotate right by one inside each row of 16 lanes: lane n receives the
// value of lane (n - 1) mod 16.
__device__ __forceinline__ uint32_t row_ror1(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)x, (int)x, 0x121, 0xf, 0xf, false);
}

template <typename T>
struct ChunkWords {
  static constexpr int kWords = 8 * (int)sizeof(T) / 4;  // 8 channels: 4 words bf16, 8 words fp32
};

template <typename T>
__device__ __forceinline__ void load_chunk(const T* base, bool valid, uint32_t* w) {
  constexpr int NW = ChunkWords<T>::kWords;
  if (valid) {
#pragma unroll
    for (int i = 0; i < NW / 4; ++i) {
      const u32x4_t u = load16(reinterpret_cast<const unsigned char*>(base) + 16 * i);
#pragma unroll
      for (int k = 0; k < 4; ++k) w[4 * i + k] = u[k];
    }
  } else {
#pragma unroll
    for (int i = 0; i < NW; ++i) w[i] = 0u;
  }
}

template <typename T>
__device__ __forceinline__ void unpack_chunk(const uint32_t* w, float* x8) {
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x8[2 * i] = bf16_lo(w[i]);
      x8[2 * i + 1] = bf16_hi(w[i]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 8; ++i) x8[i] = __uint_as_float(w[i]);
  }
}

template <typename T, int D>
__global__ void __launch_bounds__(kThreads)
readout_kernel(Plan P, const T* __restrict__ qin, const T* __restrict__ rin,
               const float* __restrict__ conv_w, const float* __restrict__ gamma,
               const int32_t* __restrict__ cu, const unsigned char* __restrict__ frags,
               float* __restrict__ out) {
  constexpr int NMB = FragCfg<D>::kNMB, NKB = FragCfg<D>::kNKB;
  constexpr int NW = ChunkWords<T>::kWords;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = blockIdx.y, g = blockIdx.x;
  int s, tile;
  if (P.ragged) {
    if (!locate_unit(cu, P.nseq, P.rtile, g, &s, &tile)) return;
  } else {
    s = g / P.rtiles_per_seq;
    tile = g - s * P.rtiles_per_seq;
  }
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int64_t tt0 = (int64_t)tile * P.rtile;
  const int64_t tt1 = min(len, tt0 + (int64_t)P.rtile);
  if (tt1 <= tt0) return;
  const int ngroups = (int)((tt1 - tt0 + 63) / 64);
  const int per_wave = (ngroups + 3) / 4;
  const int gbeg = wave * per_wave, gend = min(ngroups, gbeg + per_wave);
  if (gbeg >= gend) return;

  const int n = lane & 15, gq = lane >> 4;
  const size_t sh = (size_t)s * P.heads + h;

  // Readout operands [S^T; z^T] for this lane.
  const unsigned char* fr = frags + sh * P.frag_bytes;
  uint32_t A[NMB][NKB][NW];
#pragma unroll
  for (int mb = 0; mb < NMB; ++mb)
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
      const unsigned char* src = fr + (((size_t)mb * NKB + kb) * 64 + lane) * (NW * 4);
#pragma unroll
      for (int i = 0; i < NW / 4; ++i) {
        const u32x4_t u = load16(src + 16 * i);
#pragma unroll
        for (int k = 0; k < 4; ++k) A[mb][kb][4 * i + k] = u[k];
      }
    }
  float wq[NKB][8][4];
  float gm[NKB][8];
#pragma unroll
  for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int c = 32 * kb + 8 * gq + j;
      load_taps4(conv_w, P.heads, h, 0, D, P.W, c, wq[kb][j]);
      gm[kb][j] = gamma ? gamma[(size_t)h * D + c] : 1.0f;
    }

  // Rows tb-3 .. tb-1 of the wave's first group, as lane 15 of a virtual
  // previous group would hold them after the rotate (only lane n = 0 reads them).
  uint32_t prev[3][NKB][NW];
  {
    const int64_t tb = tt0 + 64 * (int64_t)gbeg;
#pragma unroll
    for (int jj = 0; jj < 3; ++jj) {
      const int64_t t = tb - 3 + jj;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
        load_chunk<T>(qin + (base_row + t) * D + 32 * kb + 8 * gq, t >= 0, prev[jj][kb]);
    }
  }

  for (int grp = gbeg; grp < gend; ++grp) {
    const int64_t tb = tt0 + 64 * (int64_t)grp;
    uint32_t raw[4][NKB][NW];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t t = tb + 4 * n + j;
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
        load_chunk<T>(qin + (base_row + t) * D + 32 * kb + 8 * gq, t < tt1, raw[j][kb]);
    }
    // hal[jj] = row (tb + 4n - 3 + jj), jj = 0..2
    uint32_t hal[3][NKB][NW];
#pragma unroll
    for (int jj = 0; jj < 3; ++jj)
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int i = 0; i < NW; ++i) {
          const uint32_t rot = row_ror1(raw[jj + 1][kb][i]);
          hal[jj][kb][i] = n == 0 ? prev[jj][kb][i] : rot;
          prev[jj][kb][i] = rot;
        }

#pragma unroll
    for (int j = 0; j < 4; ++j) {
      // B operand: phi(qt) of token tb + 4n + j, channels 32*kb + 8*gq + [0, 8).
      uint32_t Bw[NKB][NW];
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) {
        float x[4][8];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int r = j + t;  // window row r of 0..6: hal[0..2], raw[0..3]
          unpack_chunk<T>(r < 3 ? hal[r][kb] : raw[r - 3][kb], x[t]);
        }
        float f[8];
#pragma unroll
        for (int c = 0; c < 8; ++c) {
          float acc = 0.0f;
#pragma unroll
          for (int t = 0; t < 4; ++t) acc = fmaf(wq[kb][c][t], x[t][c], acc);
          f[c] = phi<T>(acc);
        }
        if constexpr (sizeof(T) == 2) {
#pragma unroll
          for (int i = 0; i < 4; ++i) Bw[kb][i] = pack_bf16x2(f[2 * i], f[2 * i + 1]);
        } else {
#pragma unroll
          for (int i = 0; i < 8; ++i) Bw[kb][i] = __float_as_uint(f[i]);
        }
      }
      f32x4_t acc[NMB];
#pragma unroll
      for (int mb = 0; mb < NMB; ++mb) acc[mb] = (f32x4_t){0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) {
          if constexpr (sizeof(T) == 2) {
            u32x4_t a4 = {A[mb][kb][0], A[mb][kb][1], A[mb][kb][2], A[mb][kb][3]};
            u32x4_t b4 = {Bw[kb][0], Bw[kb][1], Bw[kb][2], Bw[kb][3]};
            acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a4),
                                                              __builtin_bit_cast(bf16x8_t, b4),
                                                              acc[mb], 0, 0, 0);
          } else {
#pragma unroll
            for (int ss = 0; ss < 8; ++ss)
              acc[mb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(A[mb][kb][ss]),
                                                             __uint_as_float(Bw[kb][ss]),
                                                             acc[mb], 0, 0, 0);
          }
        }
      // Epilogue: lane holds num[e] for e = 32*q + 8*gq + [0, 8) (blocks 2q,
      // 2q+1) and the denominator in the last block.
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
      const int64_t t = tb + 4 * n + j;
      if (t < tt1 && !gamma) {  // out = o (no gated norm)
        const int64_t row = base_row + t;
#pragma unroll
        for (int qq = 0; qq < NKB; ++qq) {
          f32x4_t* dst = reinterpret_cast<f32x4_t*>(out + row * D + 32 * qq + 8 * gq);
          dst[0] = acc[2 * qq];
          dst[1] = acc[2 * qq + 1];
        }
      } else if (t < tt1) {
        const int64_t row = base_row + t;
#pragma unroll
        for (int qq = 0; qq < NKB; ++qq) {
          uint32_t rw[NW];
          load_chunk<T>(rin + row * D + 32 * qq + 8 * gq, true, rw);
          float rv[8];
          unpack_chunk<T>(rw, rv);
          f32x4_t y0, y1;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            y0[i] = acc[2 * qq][i] * scale * gm[qq][i] * silu<T>(rv[i]);
            y1[i] = acc[2 * qq + 1][i] * scale * gm[qq][4 + i] * silu<T>(rv[4 + i]);
          }
          f32x4_t* dst = reinterpret_cast<f32x4_t*>(out + row * D + 32 * qq + 8 * gq);
          dst[0] = y0;
          dst[1] = y1;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Dispatch.
// ---------------------------------------------------------------------------
template <template <typename, int> class Fn, typename... Args>
gbla_status dispatch(const Plan& p, Args&&... args) {
  if (p.dtype == GBLA_BF16) {
    if (p.d == 32) return Fn<uint16_t, 32>::run(p, args...);
    if (p.d == 64) return Fn<uint16_t, 64>::run(p, args...);
    if (p.d == 128) return Fn<uint16_t, 128>::run(p, args...);
  } else {
    if (p.d == 32) return Fn<float, 32>::run(p, args...);
    if (p.d == 64) return Fn<float, 64>::run(p, args...);
    if (p.d == 128) return Fn<float, 128>::run(p, args...);
  }
  return GBLA_ERR_UNSUPPORTED;
}

gbla_status last_launch_status() {
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}

template <typename T, int D>
struct ConvRun {
  static gbla_status run(const Plan& p, const void* q, const void* k, const void* v,
                         const float* w, const int32_t* cu, float* qt, float* kt, float* vt,
                         hipStream_t st) {
    const int64_t tiles = ((int64_t)p.rows + kConvRows - 1) / kConvRows;
    if (tiles == 0) return GBLA_OK;
    const int slices = p.ragged ? p.heads : p.nseq * p.heads;
    dim3 grid((unsigned)tiles, (unsigned)slices, 3);
    hipLaunchKernelGGL((conv_kernel<T, D>), grid, dim3(kThreads), 0, st, p,
                       (const T*)q, (const T*)k, (const T*)v, w, cu, qt, kt, vt);
    return last_launch_status();
  }
};

// One element per thread while the grid stays small, four or sixteen once
// there are many (sequence, head) pairs (fewer workgroups, each with more
// loads in flight).  The result does not depend on the choice.
template <typename T, int D>
gbla_status run_combine(const Plan& p, const int32_t* cu, const float* partials, float* S,
                        float* z, unsigned char* frags, float* mz, hipStream_t st) {
  constexpr int kElems = D * D + D;
  const int64_t pairs = (int64_t)p.nseq * p.heads;
  const int slices1 = (kElems + kThreads - 1) / kThreads;
  if (pairs * slices1 <= 4096) {
    hipLaunchKernelGGL((combine_kernel<T, D, 1>), dim3(pairs, slices1), dim3(kThreads), 0, st, p,
                       cu, partials, S, z, frags, mz);
  } else if (pairs * ((kElems + 4 * kThreads - 1) / (4 * kThreads)) <= 4096) {
    const int slices4 = (kElems + 4 * kThreads - 1) / (4 * kThreads);
    hipLaunchKernelGGL((combine_kernel<T, D, 4>), dim3(pairs, slices4), dim3(kThreads), 0, st, p,
                       cu, partials, S, z, frags, mz);
  } else {
    const int slices16 = (kElems + 16 * kThreads - 1) / (16 * kThreads);
    hipLaunchKernelGGL((combine_kernel<T, D, 16>), dim3(pairs, slices16), dim3(kThreads), 0, st, p,
                       cu, partials, S, z, frags, mz);
  }
  return last_launch_status();
}

template <typename T, int D>
struct StateRun {
  static gbla_status run(const Plan& p, const void* k, const void* v, const void* a,
                         const float* w, const int32_t* cu, void* ws, float* S, float* z,
                         float* mz, hipStream_t st) {
    unsigned char* base = static_cast<unsigned char*>(ws);
    float* partials = reinterpret_cast<float*>(base + p.off_partials);
    gbla_status e;
    if (stream_supported(p)) {
      e = launch_state_stream(p, k, v, a, w, cu, partials, st);
    } else {
      hipLaunchKernelGGL((state_partial_kernel<T, D>), dim3(p.units, p.heads), dim3(kThreads), 0,
                         st, p, (const T*)k, (const T*)v, (const T*)a, w, cu, partials);
      e = last_launch_status();
    }
    if (e != GBLA_OK) return e;
    return run_combine<T, D>(p, cu, partials, S, z, base + p.off_frags, mz, st);
  }
};

template <typename T, int D>
struct CombineF32Run {
  static gbla_status run(const Plan& p, const int32_t* cu, const float* partials, float* S,
                         float* z, float* mz, hipStream_t st) {
    return run_combine<float, D>(p, cu, partials, S, z, nullptr, mz, st);
  }
};

template <typename T, int D>
struct ReadoutRun {
  static gbla_status run(const Plan& p, const void* q, const void* r, const float* w,
                         const float* gamma, const int32_t* cu, const void* ws, float* out,
                         hipStream_t st, KernelEvents ev) {
    if (p.tokens == 0) {
      // nothing to launch: the events still mark this point of the stream
      if (ev.start && hipEventRecord(ev.start, st) != hipSuccess) return GBLA_ERR_HIP;
      if (ev.stop && hipEventRecord(ev.stop, st) != hipSuccess) return GBLA_ERR_HIP;
      return GBLA_OK;
    }
    const unsigned char* base = static_cast<const unsigned char*>(ws);
    if (stream_supported(p))
      return launch_readout_stream(p, q, r, w, gamma, cu, base + p.off_frags, out, st, ev);
    if (ev.any())
      hipExtLaunchKernelGGL((readout_kernel<T, D>), dim3(p.runits, p.heads), dim3(kThreads), 0, st,
                            ev.start, ev.stop, 0, p, (const T*)q, (const T*)r, w, gamma, cu,
                            base + p.off_frags, out);
    else
      hipLaunchKernelGGL((readout_kernel<T, D>), dim3(p.runits, p.heads), dim3(kThreads), 0, st,
                         p, (const T*)q, (const T*)r, w, gamma, cu, base + p.off_frags, out);
    return last_launch_status();
  }
};

}  // namespace

gbla_status launch_conv(const Plan& p, const void* q, const void* k, const void* v,
                        const float* conv_w, const int32_t* cu, float* qt, float* kt,
                        float* vt, hipStream_t stream) {
  return dispatch<ConvRun>(p, q, k, v, conv_w, cu, qt, kt, vt, stream);
}

gbla_status launch_state(const Plan& p, const void* k, const void* v, const void* a,
                         const float* conv_w, const int32_t* cu, void* workspace, float* S,
                         float* z, float* mz, hipStream_t stream) {
  return dispatch<StateRun>(p, k, v, a, conv_w, cu, workspace, S, z, mz, stream);
}

gbla_status launch_combine_f32(const Plan& p, const int32_t* cu, const float* partials,
                               float* S, float* z, float* mz, hipStream_t stream) {
  return dispatch<CombineF32Run>(p, cu, partials, S, z, mz, stream);
}

gbla_status launch_readout(const Plan& p, const void* q, const void* r, const float* conv_w,
                           const float* gamma, const int32_t* cu, const void* workspace,
                           float* out, hipStream_t stream, KernelEvents ev) {
  return dispatch<ReadoutRun>(p, q, r, conv_w, gamma, cu, workspace, out, stream, ev);
}

}  // namespace gbla
