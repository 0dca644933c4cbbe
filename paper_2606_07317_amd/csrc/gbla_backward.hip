// gbla_backward.hip -- the backward pass of GBLA (the chain rule through the
// forward pass of Section 2.1), fp32 arithmetic on bf16 or fp32 inputs.
//
// For one sequence and head, with the forward quantities recomputed
// (qt = Conv1D(q), Qh = phi(qt), P = phi(kt), g = softmax(a), S, z,
// num_i = Qh_i^T S, den_i = Qh_i^T z, o_i = num_i / den_i,
// rs_i = (mean o_i^2 + eps)^(-1/2), oh_i = rs_i o_i, y = oh gamma silu(r)):
//
//   query pass  doh = dy gamma silu(r), dgamma += dy oh silu(r),
//               dr = dy oh gamma silu'(r),
//               do = rs doh - rs^3/d (doh . o) o,
//               dnum = do / den, dden = -(do . o) / den,
//               dQh = S dnum + z dden, dqt = dQh phi'(qt),
//               dS = sum_i Qh_i dnum_i^T, dz = sum_i Qh_i dden_i
//   key pass    t_j = dS vt_j + dz, dkt = g_j t_j phi'(kt), dvt = g_j dS^T P_j,
//               da_j = g_j (P_j . t_j)
//   conv pass   dx_m = sum_t w_t dxt_{m+W-1-t}, dw_t = sum_i dxt_i x_{i-W+1+t}
//
// da has no softmax centering term: o does not change when every gate of a
// sequence is scaled by the same factor (the normaliser cancels between
// numerator and denominator), so sum_l g_l dL/dg_l = 0.
//
// Every reduction (dS, dz, dgamma, the tap gradients) runs in an order fixed
// by the shape, so the results are the same bits on every call.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gbla_device.h"
#include "gbla_ext.h"
#include "gbla_plan.h"

namespace gbla {
namespace {

template <typename T>
__device__ __forceinline__ float act(const T* p, int64_t i);
template <>
__device__ __forceinline__ float act<float>(const float* p, int64_t i) { return p[i]; }
template <>
__device__ __forceinline__ float act<uint16_t>(const uint16_t* p, int64_t i) {
  return __uint_as_float((uint32_t)p[i] << 16);
}

// Orders a wave's LDS stores before its later LDS loads of other lanes'
// slots (one wave's LDS operations complete in order; this keeps the
// compiler from moving them).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ float phi_f(float u) { return u > 0.0f ? u + 1.0f : expf(u); }

// Gate logit i, or 0 without gate logits (the no-key-gating switch: uniform
// gates, the softmax of constant logits).
template <typename T>
__device__ __forceinline__ float logit(const T* a, int64_t i) { return a ? act<T>(a, i) : 0.0f; }
// Hardware-exp forms for the matrix-core kernels (a few ulp; the gradients
// are held to fp32-sum accuracy, far above that).
__device__ __forceinline__ float phi_fast(float u) { return u > 0.0f ? u + 1.0f : __expf(u); }
__device__ __forceinline__ float sigmoid_fast(float x) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-x));
}
__device__ __forceinline__ float dphi_f(float u) { return u > 0.0f ? 1.0f : expf(u); }

template <int D>
struct BW {
  static constexpr int kWaves = 4;
  static constexpr int kTok = 16;                      // tokens per wave per block
  static constexpr int kBlk = kWaves * kTok;           // tokens per block of the query pass
  static constexpr int kSP = D + 1;                    // padded LDS row stride of S / dS
  static constexpr int kCPL = D > 64 ? D / 64 : 1;     // channels per lane
  static constexpr int kRS = kThreads / D;             // dS row stride between a thread's elements
  static constexpr int kEl = D / kRS;                  // dS elements per thread
};

// Channel of slot cc of a lane (may be >= D for d = 32: the lane is idle).
template <int D>
__device__ __forceinline__ int chan(int lane, int cc) { return lane + 64 * cc; }

// ---------------------------------------------------------------------------
// State recomputed in fp32: grid (units, H); a unit is the forward's chunk of
// tokens.  Writes the record [S_p | z_p | m_p | l_p] of the chunk with
//   w_j = exp(a_j - m_p), m_p = max_j a_j, l_p = sum_j w_j,
//   S_p = sum_j w_j phi(kt_j) vt_j^T, z_p = sum_j w_j phi(kt_j),
// every product in fp32 (the forward's bf16 path rounds the gated keys to
// bf16 for its MFMAs; the gradients read S and z without that rounding).
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(kThreads)
bwd_state_kernel(Plan P, const T* __restrict__ kin, const T* __restrict__ vin,
                 const T* __restrict__ ain, const float* __restrict__ conv_w,
                 const int32_t* __restrict__ cu, float* __restrict__ partials) {
  using C = BW<D>;
  constexpr int CPL = C::kCPL, kEl = C::kEl;
  __shared__ float kb[C::kBlk][D];
  __shared__ float vb[C::kBlk][D];
  __shared__ float red[C::kWaves];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.y, g = blockIdx.x;
  int s, chunk;
  if (!unit_of(P, cu, P.chunk, P.chunks_per_seq, g, &s, &chunk)) return;
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int64_t t0 = (int64_t)chunk * P.chunk;
  const int64_t t1 = min(len, t0 + (int64_t)P.chunk);

  float ml = -INFINITY;
  for (int64_t j = t0 + tid; j < t1; j += kThreads) ml = fmaxf(ml, logit<T>(ain, base_row + j));
  const float m = block_max(ml, red);

  float wk[CPL][4], wv[CPL][4];
#pragma unroll
  for (int cc = 0; cc < CPL; ++cc) {
    const int e = min(chan<D>(lane, cc), D - 1);
    load_taps4(conv_w, P.heads, h, 1, D, P.W, e, wk[cc]);
    load_taps4(conv_w, P.heads, h, 2, D, P.W, e, wv[cc]);
  }
  const int ds_e = tid % D, ds_c0 = tid / D;
  float S_acc[kEl];
#pragma unroll
  for (int i = 0; i < kEl; ++i) S_acc[i] = 0.0f;
  float z_acc = 0.0f, l_acc = 0.0f;

  for (int64_t b0 = t0; b0 < t1; b0 += C::kBlk) {
    for (int k = 0; k < C::kTok; ++k) {
      const int slot = wave * C::kTok + k;
      const int64_t j = b0 + slot;
      const bool live = j < t1;  // wave-uniform
      const float w = live ? expf(logit<T>(ain, base_row + j) - m) : 0.0f;
      if (lane == 0) l_acc += w;
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int e = chan<D>(lane, cc);
        if (e < D) {
          float ka = 0.0f, va = 0.0f;
          if (live) {
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              const int64_t src = j - 3 + t;
              if (src >= 0) {
                ka = fmaf(wk[cc][t], act<T>(kin, (base_row + src) * D + e), ka);
                va = fmaf(wv[cc][t], act<T>(vin, (base_row + src) * D + e), va);
              }
            }
          }
          kb[slot][e] = w * phi_f(ka);
          vb[slot][e] = va;
        }
      }
    }
    __syncthreads();
    // S_p += sum over the block's tokens in token order; thread tid owns
    // column e = tid % D and rows c0 + kRS * i.
#pragma unroll 2
    for (int slot = 0; slot < C::kBlk; ++slot) {
      const float vv = vb[slot][ds_e];
#pragma unroll
      for (int i = 0; i < kEl; ++i) S_acc[i] = fmaf(kb[slot][ds_c0 + C::kRS * i], vv, S_acc[i]);
    }
    if (tid < D)
      for (int slot = 0; slot < C::kBlk; ++slot) z_acc += kb[slot][tid];
    __syncthreads();
  }

  float* rec = partials + ((size_t)h * P.units + g) * P.rec_floats;
#pragma unroll
  for (int i = 0; i < kEl; ++i) rec[(ds_c0 + C::kRS * i) * D + ds_e] = S_acc[i];
  if (tid < D) rec[D * D + tid] = z_acc;
  __syncthreads();  // every wave has read red in block_max (the loop may not run)
  if (lane == 0) red[wave] = l_acc;
  __syncthreads();
  if (tid == 0) {
    float l = 0.0f;
#pragma unroll
    for (int w = 0; w < C::kWaves; ++w) l += red[w];
    rec[D * D + D] = m;
    rec[D * D + D + 1] = l;
  }
}

// ---------------------------------------------------------------------------
// Query pass: grid (units, H).
// ---------------------------------------------------------------------------
template <typename T, int D, bool kNorm>
__global__ void __launch_bounds__(kThreads)
bwd_query_kernel(Plan P, const T* __restrict__ qin, const T* __restrict__ rin,
                 const float* __restrict__ dy, const float* __restrict__ conv_w,
                 const float* __restrict__ gamma, const int32_t* __restrict__ cu,
                 const float* __restrict__ Sg, const float* __restrict__ zg,
                 float* __restrict__ dqt, float* __restrict__ dr, float* __restrict__ dsp,
                 float* __restrict__ dgp) {
  using C = BW<D>;
  constexpr int CPL = C::kCPL, kEl = C::kEl;
  __shared__ float Ss[D * C::kSP];
  __shared__ float zs[D];
  __shared__ float qh_b[C::kBlk][D];
  __shared__ float dn_b[C::kBlk][D];
  __shared__ float dd_b[C::kBlk];
  __shared__ float red[C::kWaves][D];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.y, g = blockIdx.x;
  int s, chunk;
  if (!unit_of(P, cu, P.chunk, P.chunks_per_seq, g, &s, &chunk)) return;
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int64_t t0 = (int64_t)chunk * P.chunk;
  const int64_t t1 = min(len, t0 + (int64_t)P.chunk);
  const size_t sh = (size_t)s * P.heads + h;
  for (int x = tid; x < D * D; x += kThreads) Ss[(x / D) * C::kSP + x % D] = Sg[sh * D * D + x];
  if (tid < D) zs[tid] = zg[sh * D + tid];

  float wq[CPL][4], gm[CPL], dg_acc[CPL];
#pragma unroll
  for (int cc = 0; cc < CPL; ++cc) {
    const int e = min(chan<D>(lane, cc), D - 1);
    load_taps4(conv_w, P.heads, h, 0, D, P.W, e, wq[cc]);
    gm[cc] = kNorm ? gamma[(size_t)h * D + e] : 1.0f;
    dg_acc[cc] = 0.0f;
  }
  const int ds_e = tid % D, ds_c0 = tid / D;
  float dS_acc[kEl];
#pragma unroll
  for (int m = 0; m < kEl; ++m) dS_acc[m] = 0.0f;
  float dz_acc = 0.0f;
  __syncthreads();

  for (int64_t b0 = t0; b0 < t1; b0 += C::kBlk) {
    for (int k = 0; k < C::kTok; ++k) {
      const int slot = wave * C::kTok + k;
      const int64_t i = b0 + slot;  // token of the sequence
      if (i >= t1) {                // wave-uniform: contributes nothing
#pragma unroll
        for (int cc = 0; cc < CPL; ++cc) {
          const int e = chan<D>(lane, cc);
          if (e < D) {
            qh_b[slot][e] = 0.0f;
            dn_b[slot][e] = 0.0f;
          }
        }
        if (lane == 0) dd_b[slot] = 0.0f;
        continue;
      }
      const int64_t row = base_row + i;
      float qt[CPL], qh[CPL];
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int e = chan<D>(lane, cc);
        float acc = 0.0f;
        if (e < D) {
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const int64_t src = i - 3 + t;
            if (src >= 0) acc = fmaf(wq[cc][t], act<T>(qin, (base_row + src) * D + e), acc);
          }
          qh_b[slot][e] = phi_f(acc);
        }
        qt[cc] = acc;
        qh[cc] = phi_f(acc);
      }
      wave_lds_sync();
      // num and den (z dotted with Qh over the wave)
      float num[CPL], zd = 0.0f;
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int e = chan<D>(lane, cc);
        float acc = 0.0f;
        if (e < D) {
#pragma unroll 8
          for (int c = 0; c < D; ++c) acc = fmaf(qh_b[slot][c], Ss[c * C::kSP + e], acc);
          zd = fmaf(qh[cc], zs[e], zd);
        }
        num[cc] = acc;
      }
      const float den = wave_sum(zd);
      float o[CPL], ss = 0.0f;
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        o[cc] = num[cc] / den;
        if (chan<D>(lane, cc) < D) ss = fmaf(o[cc], o[cc], ss);
      }
      float dnum[CPL], dden;
      if constexpr (kNorm) {
        const float rs = 1.0f / sqrtf(wave_sum(ss) / D + P.eps);
        float doh[CPL], s1 = 0.0f;
#pragma unroll
        for (int cc = 0; cc < CPL; ++cc) {
          const int e = chan<D>(lane, cc);
          doh[cc] = 0.0f;
          if (e < D) {
            const float rv = act<T>(rin, row * D + e), dyv = dy[row * D + e];
            const float sig = 1.0f / (1.0f + expf(-rv)), silu = rv * sig;
            const float oh = o[cc] * rs;
            doh[cc] = dyv * gm[cc] * silu;
            dg_acc[cc] = fmaf(dyv * oh, silu, dg_acc[cc]);
            dr[row * D + e] = dyv * oh * gm[cc] * sig * (1.0f + rv * (1.0f - sig));
            s1 = fmaf(doh[cc], o[cc], s1);
          }
        }
        s1 = wave_sum(s1);
#pragma unroll
        for (int cc = 0; cc < CPL; ++cc) dnum[cc] = (rs * doh[cc] - rs * rs * rs / D * s1 * o[cc]) / den;
        // do . o = eps rs^3 s1 exactly (rs^-2 = |o|^2/d + eps); see the matrix-core kernel
        dden = -P.eps * rs * rs * rs * s1 / den;
      } else {  // y = o: do = dy
        float s2 = 0.0f;
#pragma unroll
        for (int cc = 0; cc < CPL; ++cc) {
          const int e = chan<D>(lane, cc);
          const float dyv = e < D ? dy[row * D + e] : 0.0f;
          dnum[cc] = dyv / den;
          s2 = fmaf(dyv, o[cc], s2);
        }
        dden = -wave_sum(s2) / den;
      }
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int e = chan<D>(lane, cc);
        if (e < D) dn_b[slot][e] = dnum[cc];
      }
      if (lane == 0) dd_b[slot] = dden;
      wave_lds_sync();
      // dQh[c] = sum_e S[c][e] dnum[e] + z[c] dden (lane owns c)
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const int c = chan<D>(lane, cc);
        if (c < D) {
          float acc = zs[c] * dden;
#pragma unroll 8
          for (int e = 0; e < D; ++e) acc = fmaf(Ss[c * C::kSP + e], dn_b[slot][e], acc);
          dqt[row * D + c] = acc * dphi_f(qt[cc]);
        }
      }
    }
    __syncthreads();
    // dS += sum over the block's tokens (in token order) of Qh_i dnum_i^T.
    // Thread tid owns column e = tid % D and rows c0 + kRS * m of dS.
#pragma unroll 2
    for (int slot = 0; slot < C::kBlk; ++slot) {
      const float dn = dn_b[slot][ds_e];
#pragma unroll
      for (int m = 0; m < kEl; ++m) dS_acc[m] = fmaf(qh_b[slot][ds_c0 + C::kRS * m], dn, dS_acc[m]);
    }
    if (tid < D)
      for (int slot = 0; slot < C::kBlk; ++slot) dz_acc = fmaf(qh_b[slot][tid], dd_b[slot], dz_acc);
    __syncthreads();
  }

  float* rec = dsp + ((size_t)h * P.units + g) * P.rec_floats;
#pragma unroll
  for (int m = 0; m < kEl; ++m) rec[(ds_c0 + C::kRS * m) * D + ds_e] = dS_acc[m];
  if (tid < D) rec[D * D + tid] = dz_acc;
  // dgamma partial of the unit: the four waves' sums in wave order
#pragma unroll
  for (int cc = 0; cc < CPL; ++cc) {
    const int e = chan<D>(lane, cc);
    if (e < D) red[wave][e] = dg_acc[cc];
  }
  __syncthreads();
  if (tid < D) {
    float acc = 0.0f;
#pragma unroll
    for (int w = 0; w < C::kWaves; ++w) acc += red[w][tid];
    dgp[((size_t)h * P.units + g) * D + tid] = acc;
  }
}

// ---------------------------------------------------------------------------
// dS, dz of each (sequence, head): the fixed-order sum of its units' partials.
// grid (N * H, element slices of kThreads).
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(kThreads)
bwd_dscombine_kernel(Plan P, const int32_t* __restrict__ cu, const float* __restrict__ dsp,
                     float* __restrict__ dS) {
  constexpr int kElems = D * D + D;
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
  const int x = blockIdx.y * kThreads + threadIdx.x;
  if (x >= kElems) return;
  const float* recs = dsp + ((size_t)h * P.units + first) * P.rec_floats + x;
  const size_t rf = P.rec_floats;
  // in unit order (compensated); eight loads in flight per group
  float acc = 0.0f, cmp = 0.0f;
  int p = 0;
  for (; p + 8 <= count; p += 8) {
    float v[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) v[i] = recs[(size_t)(p + i) * rf];
#pragma unroll
    for (int i = 0; i < 8; ++i) kahan_add(acc, cmp, v[i]);
  }
  for (; p < count; ++p) kahan_add(acc, cmp, recs[(size_t)p * rf]);
  dS[(size_t)sh_idx * kElems + x] = acc;
}

// ---------------------------------------------------------------------------
// Key pass: grid (units, H).
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(kThreads)
bwd_key_kernel(Plan P, const T* __restrict__ kin, const T* __restrict__ vin,
               const T* __restrict__ ain, const float* __restrict__ conv_w,
               const int32_t* __restrict__ cu, const float* __restrict__ dSg,
               const float* __restrict__ mz, float* __restrict__ dkt, float* __restrict__ dvt,
               float* __restrict__ da) {
  using C = BW<D>;
  constexpr int CPL = C::kCPL;
  __shared__ float dSs[D * C::kSP];
  __shared__ float dzs[D];
  __shared__ float vb[C::kWaves][D];
  __shared__ float pb[C::kWaves][D];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.y, g = blockIdx.x;
  int s, chunk;
  if (!unit_of(P, cu, P.chunk, P.chunks_per_seq, g, &s, &chunk)) return;
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int64_t t0 = (int64_t)chunk * P.chunk;
  const int64_t t1 = min(len, t0 + (int64_t)P.chunk);
  const size_t sh = (size_t)s * P.heads + h;
  const float* dsrc = dSg + sh * (D * D + D);
  for (int x = tid; x < D * D; x += kThreads) dSs[(x / D) * C::kSP + x % D] = dsrc[x];
  if (tid < D) dzs[tid] = dsrc[D * D + tid];
  const float M = mz[2 * sh], Z = mz[2 * sh + 1];
  const float invZ = Z > 0.0f ? 1.0f / Z : 0.0f;
  float wk[CPL][4], wv[CPL][4];
#pragma unroll
  for (int cc = 0; cc < CPL; ++cc) {
    const int e = min(chan<D>(lane, cc), D - 1);
    load_taps4(conv_w, P.heads, h, 1, D, P.W, e, wk[cc]);
    load_taps4(conv_w, P.heads, h, 2, D, P.W, e, wv[cc]);
  }
  __syncthreads();

  for (int64_t j = t0 + wave; j < t1; j += C::kWaves) {
    const int64_t row = base_row + j;
    wave_lds_sync();  // the previous token's reads of vb, pb are done
    float kt[CPL], pv[CPL];
#pragma unroll
    for (int cc = 0; cc < CPL; ++cc) {
      const int e = chan<D>(lane, cc);
      float ka = 0.0f, va = 0.0f;
      if (e < D) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const int64_t src = j - 3 + t;
          if (src >= 0) {
            ka = fmaf(wk[cc][t], act<T>(kin, (base_row + src) * D + e), ka);
            va = fmaf(wv[cc][t], act<T>(vin, (base_row + src) * D + e), va);
          }
        }
        vb[wave][e] = va;
        pb[wave][e] = phi_f(ka);
      }
      kt[cc] = ka;
      pv[cc] = phi_f(ka);
    }
    wave_lds_sync();
    const float alog = ain ? act<T>(ain, row) : 0.0f;
    const float gj = M == -INFINITY ? 0.0f : expf(alog - M) * invZ;
    // t[c] = sum_e dS[c][e] vt[e] + dz[c]; dkt = g t phi'(kt); dg = P . t
    float dgl = 0.0f;
#pragma unroll
    for (int cc = 0; cc < CPL; ++cc) {
      const int c = chan<D>(lane, cc);
      if (c < D) {
        float acc = dzs[c];
#pragma unroll 8
        for (int e = 0; e < D; ++e) acc = fmaf(dSs[c * C::kSP + e], vb[wave][e], acc);
        dkt[row * D + c] = gj * acc * dphi_f(kt[cc]);
        dgl = fmaf(pv[cc], acc, dgl);
      }
    }
    const float dg = wave_sum(dgl);
    if (da && lane == 0) da[row] = gj * dg;
    // dvt[e] = g sum_c dS[c][e] P[c]
#pragma unroll
    for (int cc = 0; cc < CPL; ++cc) {
      const int e = chan<D>(lane, cc);
      if (e < D) {
        float acc = 0.0f;
#pragma unroll 8
        for (int c = 0; c < D; ++c) acc = fmaf(dSs[c * C::kSP + e], pb[wave][c], acc);
        dvt[row * D + e] = gj * acc;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Conv1D backward: grid (units, H, 3 tensors).  Thread (grp, e) handles
// channel e of tokens t0 + grp, t0 + grp + kThreads / D, ...; the tap
// gradients of the unit are summed over the groups in group order.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(kThreads)
bwd_conv_kernel(Plan P, const T* __restrict__ qin, const T* __restrict__ kin,
                const T* __restrict__ vin, const float* __restrict__ dxt_all,
                const float* __restrict__ conv_w, const int32_t* __restrict__ cu,
                float* __restrict__ dq, float* __restrict__ dk, float* __restrict__ dv,
                float* __restrict__ dcp, size_t act_elems) {
  constexpr int kG = kThreads / D;
  __shared__ float red[kG][D][4];
  const int tid = threadIdx.x, e = tid % D, grp = tid / D;
  const int h = blockIdx.y, g = blockIdx.x, tensor = blockIdx.z;
  int s, chunk;
  if (!unit_of(P, cu, P.chunk, P.chunks_per_seq, g, &s, &chunk)) return;
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int64_t t0 = (int64_t)chunk * P.chunk;
  const int64_t t1 = min(len, t0 + (int64_t)P.chunk);
  const T* x = tensor == 0 ? qin : tensor == 1 ? kin : vin;
  float* out = tensor == 0 ? dq : tensor == 1 ? dk : dv;
  const float* dxt = dxt_all + (size_t)tensor * act_elems;
  float w4[4];
  load_taps4(conv_w, P.heads, h, tensor, D, P.W, e, w4);
  float dc[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int64_t i = t0 + grp; i < t1; i += kG) {
    float acc = 0.0f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int64_t m = i + 3 - t;  // the output that tap t reads token i into
      if (m < len) acc = fmaf(w4[t], dxt[(base_row + m) * D + e], acc);
    }
    out[(base_row + i) * D + e] = acc;
    const float d0 = dxt[(base_row + i) * D + e];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int64_t src = i - 3 + t;
      if (src >= 0) dc[t] = fmaf(d0, act<T>(x, (base_row + src) * D + e), dc[t]);
    }
  }
#pragma unroll
  for (int t = 0; t < 4; ++t) red[grp][e][t] = dc[t];
  __syncthreads();
  if (grp == 0) {
    float* rec = dcp + (((size_t)h * P.units + g) * 3 + tensor) * D * 4;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      float acc = 0.0f;
      for (int gg = 0; gg < kG; ++gg) acc += red[gg][e][t];
      rec[e * 4 + t] = acc;
    }
  }
}

// ---------------------------------------------------------------------------
// dgamma and the tap gradients: per head, the fixed-order sum over the head's
// units (every sequence of the batch).  grid (H, slices of 64 outputs); the
// outputs of a head are dgamma[0 .. d) then the taps in [3, d, W] order.
// Wave w sums a quarter of the units in unit order; the four quarter sums
// are added in wave order.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(kThreads)
bwd_param_kernel(Plan P, const int32_t* __restrict__ cu, const float* __restrict__ dgp,
                 const float* __restrict__ dcp, float* __restrict__ dgamma,
                 float* __restrict__ dconv) {
  __shared__ float red[4][64];
  const int h = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int total = P.ragged ? units_before(cu, P.nseq, P.chunk) : P.chunks_per_seq * P.nseq;
  const int nout = D + (dconv ? 3 * D * P.W : 0);
  const int e = blockIdx.y * 64 + lane;
  const bool live = e < nout;
  size_t off = 0, stride = 0;
  if (e < D) {
    off = (size_t)h * P.units * D + e;
    stride = D;
  } else if (live) {
    const int x = e - D, tensor = x / (D * P.W), rem = x % (D * P.W);
    const int c = rem / P.W, t4 = rem % P.W + (4 - P.W);  // right-aligned slot of the tap
    off = ((size_t)h * P.units * 3 + tensor) * D * 4 + c * 4 + t4;
    stride = (size_t)3 * D * 4;
  }
  const float* src = e < D ? dgp : dcp;
  const int u0 = (int)((int64_t)total * wave / 4), u1 = (int)((int64_t)total * (wave + 1) / 4);
  float acc = 0.0f, cmp = 0.0f;  // compensated: a quarter can hold thousands of units
  if (live) {
    int u = u0;
    for (; u + 8 <= u1; u += 8) {
      float v[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = src[off + (size_t)(u + i) * stride];
#pragma unroll
      for (int i = 0; i < 8; ++i) kahan_add(acc, cmp, v[i]);
    }
    for (; u < u1; ++u) kahan_add(acc, cmp, src[off + (size_t)u * stride]);
  }
  red[wave][lane] = acc;
  __syncthreads();
  if (tid < 64 && live) {
    const float sum = (red[0][tid] + red[1][tid]) + (red[2][tid] + red[3][tid]);
    if (e < D) {
      if (dgamma) dgamma[(size_t)h * D + e] = sum;
    } else {
      const int x = e - D, tensor = x / (D * P.W), rem = x % (D * P.W);
      dconv[((size_t)tensor * P.heads + h) * D * P.W + rem] = sum;
    }
  }
}

// ===========================================================================
// Matrix-core path (every head dim; at d = 128 one workgroup per CU).
//
// Every contraction runs on v_mfma_f32_16x16x4_f32: fp32 operands, exact
// products, fp32 accumulation, so the results carry fp32 rounding only (the
// gradients cancel strongly -- dQh = S dnum + z dden, t = dS vt + dz -- and
// a bf16 split of the operands would show through that cancellation).
//
// Lane layout.  A wave works on 16 tokens at a time; lane (n, g) = (lane &
// 15, lane >> 4) holds token n and the channel set
//     Sigma(g) = { 16 kq + 4 g + i : kq < d/16, i < 4 },
// which is the row set that a 16x16 MFMA output hands lane (n, g) when the M
// index is the channel.  The K index of every channel contraction is ordered
// the same way (K step 4 kq + i gives lane group g channel 16 kq + 4 g + i),
// so a lane's Sigma(g) values are directly its B operands and the outputs
// land where the next step needs them.  The constant A operands (S^T, S,
// dS, dS^T) are laid out once per workgroup in LDS in that K order, four K
// steps per 16-byte lane vector.
//
// Token sums (S_p and dS) contract over tokens: a wave stages its 16 tokens'
// fp32 rows in its own LDS area and reads them back as K steps of four
// tokens, accumulating its own d x d partial; the four waves' partials are
// added in wave order at the end.  Waves never wait for each other inside
// the token loop, and each one loads its next 16-token block before working
// on the current one.
// ===========================================================================
template <int D>
struct MF {
  static constexpr int NMB = D / 16;          // 16-channel blocks
  // staging row stride (floats): the four lane groups' rows start 16 banks apart
  static constexpr int kRow = D + 16;
  static constexpr int kStage = 16 * kRow;    // one wave's 16-token array
  static constexpr int kBlocks = NMB * NMB;   // 16x16 blocks of a d x d result
  static constexpr int kStep = 64;            // tokens between a wave's blocks
};

__device__ __forceinline__ f32x4_t mfma4(float a, float b, f32x4_t acc) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc, 0, 0, 0);
}

// acc[mb] += A_mb v over the d channels: A fragments f32x4 at
// frag[(mb * NMB + kq) * 64 + lane] (K steps 4 kq .. 4 kq + 3), B = the
// lane's Sigma values v[kq][i].
template <int D, int NM>
__device__ __forceinline__ void contract(const f32x4_t* __restrict__ frag, int lane,
                                         const float (*v)[4], f32x4_t* acc) {
  constexpr int NMB = D / 16;
#pragma unroll
  for (int kq = 0; kq < NMB; ++kq)
#pragma unroll
    for (int mb = 0; mb < NM; ++mb) {
      const f32x4_t a = frag[(mb * NMB + kq) * 64 + lane];
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[mb] = mfma4(a[i], v[kq][i], acc[mb]);
    }
}

// Sum over the four lane groups (the lanes n, n+16, n+32, n+48 of one token).
__device__ __forceinline__ float sum_groups(float x) {
  x += __shfl_xor(x, 16);
  return x + __shfl_xor(x, 32);
}

// Sum over the 16 lanes of a lane group (fixed tree), result in every lane.
__device__ __forceinline__ float sum_tokens(float x) {
  x += __shfl_xor(x, 8);
  x += __shfl_xor(x, 4);
  x += __shfl_xor(x, 2);
  return x + __shfl_xor(x, 1);
}

// A-operand fragments of the d x d matrix X in the K order above:
// X[row][k] = src[k * D + row] (kTrans) or src[row * D + k].  Every thread of
// the block takes part.
template <int D, bool kTrans>
__device__ __forceinline__ void build_frags(const float* __restrict__ src, f32x4_t* frag) {
  constexpr int NMB = D / 16;
  for (int idx = threadIdx.x; idx < NMB * NMB * 64; idx += kThreads) {
    const int f = idx >> 6, l = idx & 63;
    const int mb = f / NMB, kq = f % NMB;
    const int row = 16 * mb + (l & 15), k0 = 16 * kq + 4 * (l >> 4);
    f32x4_t v;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      v[i] = kTrans ? src[(size_t)(k0 + i) * D + row] : src[(size_t)row * D + k0 + i];
    frag[idx] = v;
  }
}

// The fragments of build_frags<D, false> for S' = S - z m^T: X[row][k] =
// src[row * D + k] - zv[row] mv[k] (zv, mv in LDS).
template <int D>
__device__ __forceinline__ void build_frags_centred(const float* __restrict__ src, const float* zv,
                                                    const float* mv, f32x4_t* frag) {
  constexpr int NMB = D / 16;
  for (int idx = threadIdx.x; idx < NMB * NMB * 64; idx += kThreads) {
    const int f = idx >> 6, l = idx & 63;
    const int mb = f / NMB, kq = f % NMB;
    const int row = 16 * mb + (l & 15), k0 = 16 * kq + 4 * (l >> 4);
    f32x4_t v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = fmaf(-zv[row], mv[k0 + i], src[(size_t)row * D + k0 + i]);
    frag[idx] = v;
  }
}

// Loads four consecutive channels of one row (element offset `off` of a
// buffer resource; out of range reads 0) as fp32.
template <typename T>
__device__ __forceinline__ f32x4_t load4(__amdgpu_buffer_rsrc_t r, uint32_t off);
template <>
__device__ __forceinline__ f32x4_t load4<float>(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(f32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, off * 4u, 0, 0));
}
template <>
__device__ __forceinline__ f32x4_t load4<uint16_t>(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  const u32x2_t w = __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(r, off * 2u, 0, 0));
  return (f32x4_t){bf16_lo(w[0]), bf16_hi(w[0]), bf16_lo(w[1]), bf16_hi(w[1])};
}
template <typename T>
__device__ __forceinline__ float load1(__amdgpu_buffer_rsrc_t r, uint32_t off);
template <>
__device__ __forceinline__ float load1<float>(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off * 4u, 0, 0));
}
template <>
__device__ __forceinline__ float load1<uint16_t>(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return bf16_lo((uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, off * 2u, 0, 0));
}
__device__ __forceinline__ void store4(__amdgpu_buffer_rsrc_t r, uint32_t off, const float* v) {
  const f32x4_t x = {v[0], v[1], v[2], v[3]};
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, x), r, off * 4u, 0, 0);
}

// Slice-relative element offset of channel c of token `tok` (tok may be
// negative: the unsigned offset is then past any range and reads 0).
template <int D>
__device__ __forceinline__ uint32_t eoff(int tok, int c) {
  return (uint32_t)(tok * D + c);
}

// Four consecutive channels as loaded (raw bf16 pairs or fp32), widened only
// where they are used, so that loads issued a block ahead stay in flight.
template <typename T>
struct Raw;
template <>
struct Raw<uint16_t> {
  using type = u32x2_t;
  static __device__ __forceinline__ type load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_bit_cast(u32x2_t, __builtin_amdgcn_raw_buffer_load_b64(r, off * 2u, 0, 0));
  }
  static __device__ __forceinline__ f32x4_t widen(type w) {
    return (f32x4_t){bf16_lo(w[0]), bf16_hi(w[0]), bf16_lo(w[1]), bf16_hi(w[1])};
  }
};
template <>
struct Raw<float> {
  using type = u32x4_t;
  static __device__ __forceinline__ type load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off * 4u, 0, 0);
  }
  static __device__ __forceinline__ f32x4_t widen(type w) { return __builtin_bit_cast(f32x4_t, w); }
};

// Value of token n - K for lane n of a 16-lane row: lane n - K of `cur`, or
// lane n - K + 16 of `prev` (the preceding 16 tokens) when n < K.  DPP
// row_shr:K moves cur up by K lanes inside each row; the lanes it leaves
// empty keep the row_ror:K rotation of prev.
template <int K>
__device__ __forceinline__ float shifted(float cur, float prev) {
  const int old = __builtin_amdgcn_mov_dpp(__float_as_int(prev), 0x120 + K, 0xF, 0xF, false);
  return __int_as_float(
      __builtin_amdgcn_update_dpp(old, __float_as_int(cur), 0x110 + K, 0xF, 0xF, false));
}

// One input tensor streamed 16 tokens at a time along a wave's contiguous
// token range: lane (n, g) loads only its own row (its Sigma(g) channels)
// one block ahead; the conv window's three earlier tokens come from the
// neighbouring lanes and, across the block edge, from the previous block.
template <typename T, int D>
struct RowStream {
  static constexpr int NMB = D / 16;
  typename Raw<T>::type nxt[NMB];  // raw row of the block to come (in flight)
  float prev[NMB][4];              // rows of the previous block
  __device__ __forceinline__ void issue(__amdgpu_buffer_rsrc_t r, int tok, int g) {
#pragma unroll
    for (int kq = 0; kq < NMB; ++kq) nxt[kq] = Raw<T>::load(r, eoff<D>(tok, 16 * kq + 4 * g));
  }
  // prev <- the 16 tokens before `tok` (row tok - 16 of the lane), then the
  // first block's rows are issued.
  __device__ __forceinline__ void start(__amdgpu_buffer_rsrc_t r, int tok, int g) {
#pragma unroll
    for (int kq = 0; kq < NMB; ++kq) {
      const f32x4_t p = Raw<T>::widen(Raw<T>::load(r, eoff<D>(tok - 16, 16 * kq + 4 * g)));
#pragma unroll
      for (int i = 0; i < 4; ++i) prev[kq][i] = p[i];
    }
    issue(r, tok, g);
  }
  // Consumes the issued rows: out[kq][i] = sum_t taps[c][t] x_{tok - 3 + t}[c]
  // (c = 16 kq + 4 g + i); they become prev.
  __device__ __forceinline__ void conv(const f32x4_t* taps, int g, float (*out)[4]) {
#pragma unroll
    for (int kq = 0; kq < NMB; ++kq) {
      const f32x4_t c = Raw<T>::widen(nxt[kq]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const f32x4_t w = taps[16 * kq + 4 * g + i];
        float acc = w[0] * shifted<3>(c[i], prev[kq][i]);
        acc = fmaf(w[1], shifted<2>(c[i], prev[kq][i]), acc);
        acc = fmaf(w[2], shifted<1>(c[i], prev[kq][i]), acc);
        out[kq][i] = fmaf(w[3], c[i], acc);
        prev[kq][i] = c[i];
      }
    }
  }
};

// Writes a lane's Sigma values as row n of a wave's fp32 staging array.
template <int D>
__device__ __forceinline__ void stage_sigma(float* arr, int n, int g, const float (*v)[4]) {
#pragma unroll
  for (int kq = 0; kq < D / 16; ++kq)
    *reinterpret_cast<f32x4_t*>(arr + n * MF<D>::kRow + 16 * kq + 4 * g) =
        (f32x4_t){v[kq][0], v[kq][1], v[kq][2], v[kq][3]};
}

// acc[mb * NMB + nb] += sum over the wave's 16 staged tokens of X[tok][c]
// Y[tok][e] for c block mb, e block nb (K step kk is token 4 kk + g of lane
// group g).
// With zpart, also zpart[b] += X[tok][16 b + j] over the lane's tokens
// (tokens g, g + 4, ... of lane (j, g)): the column sums of X.
template <int D>
__device__ __forceinline__ void token_product(const float* X, const float* Y, int lane,
                                              f32x4_t* acc, float* zpart = nullptr) {
  using C = MF<D>;
  const int j = lane & 15, g = lane >> 4;
  // at d = 128 (64 products per K step) the K steps are not unrolled, so that
  // their reads are not all hoisted into registers at once
#pragma unroll(D >= 128 ? 1 : 4)
  for (int kk = 0; kk < 4; ++kk) {
    const int row = (4 * kk + g) * C::kRow;
    float xv[C::NMB], yv[C::NMB];
#pragma unroll
    for (int b = 0; b < C::NMB; ++b) {
      xv[b] = X[row + 16 * b + j];
      yv[b] = Y[row + 16 * b + j];
    }
#pragma unroll
    for (int mb = 0; mb < C::NMB; ++mb)
#pragma unroll
      for (int nb = 0; nb < C::NMB; ++nb)
        acc[mb * C::NMB + nb] = mfma4(xv[mb], yv[nb], acc[mb * C::NMB + nb]);
    if (zpart) {
#pragma unroll
      for (int b = 0; b < C::NMB; ++b) zpart[b] += xv[b];
    }
  }
}

// Adds the four waves' d x d accumulators in wave order (through `buf`, d*d
// floats of LDS) and writes the sum to dst[c * D + e].  Every thread calls.
template <int D>
__device__ __forceinline__ void wave_ordered_sum(const f32x4_t* acc, float* buf, float* dst) {
  using C = MF<D>;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, n = lane & 15, g = lane >> 4;
  for (int w = 0; w < 4; ++w) {
    if (wave == w) {
#pragma unroll
      for (int mb = 0; mb < C::NMB; ++mb)
#pragma unroll
        for (int nb = 0; nb < C::NMB; ++nb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int x = (16 * mb + 4 * g + i) * D + 16 * nb + n;
            const float v = acc[mb * C::NMB + nb][i];
            buf[x] = w == 0 ? v : buf[x] + v;
          }
    }
    __syncthreads();
  }
  for (int x = threadIdx.x; x < D * D; x += kThreads) dst[x] = buf[x];
  __syncthreads();
}

// Copies the d x d matrix src (global) to buf (LDS) with 16-byte loads.
template <int D>
__device__ __forceinline__ void stage_matrix(const float* __restrict__ src, float* buf) {
  for (int x = 4 * threadIdx.x; x < D * D; x += 4 * kThreads)
    *reinterpret_cast<f32x4_t*>(buf + x) = *reinterpret_cast<const f32x4_t*>(src + x);
}

// Sums per-lane Sigma accumulators over the tokens (lanes) and the waves in
// a fixed order and writes the d sums to dst (every thread must call).
template <int D>
__device__ __forceinline__ void reduce_sigma(const float (*v)[4], float (*red)[D], float* dst) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, n = lane & 15, g = lane >> 4;
#pragma unroll
  for (int kq = 0; kq < D / 16; ++kq)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float s = sum_tokens(v[kq][i]);
      if (n == 0) red[wave][16 * kq + 4 * g + i] = s;
    }
  __syncthreads();
  if (threadIdx.x < D) {
    float acc = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) acc += red[w][threadIdx.x];
    dst[threadIdx.x] = acc;
  }
  __syncthreads();
}

// ---------------------------------------------------------------------------
// State, matrix-core version: the record [S_p | z_p | m_p | l_p] of a unit.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(kThreads, D >= 128 ? 1 : 2)
bwd_state_mfma_kernel(Plan P, const T* __restrict__ kin, const T* __restrict__ vin,
                      const T* __restrict__ ain, const float* __restrict__ conv_w,
                      const int32_t* __restrict__ cu, float* __restrict__ partials) {
  using C = MF<D>;
  constexpr int NMB = C::NMB;
  __shared__ __attribute__((aligned(16))) float stg[4][2][C::kStage];  // [wave][kt or vt]
  __shared__ f32x4_t tk[D], tv[D];
  __shared__ float red[4][D];
  __shared__ float red4[4];
  const int tid = threadIdx.x, lane = tid & 63, n = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.y, unit = blockIdx.x;
  int s, chunk;
  if (!unit_of(P, cu, P.chunk, P.chunks_per_seq, unit, &s, &chunk)) return;
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int t0 = chunk * P.chunk;
  const int t1 = (int)min(len, (int64_t)t0 + P.chunk);
  if (tid < D) {
    float w4[4];
    load_taps4(conv_w, P.heads, h, 1, D, P.W, tid, w4);
    tk[tid] = (f32x4_t){w4[0], w4[1], w4[2], w4[3]};
    load_taps4(conv_w, P.heads, h, 2, D, P.W, tid, w4);
    tv[tid] = (f32x4_t){w4[0], w4[1], w4[2], w4[3]};
  }
  float ml = -INFINITY;
  for (int j = t0 + tid; j < t1; j += kThreads) ml = fmaxf(ml, logit<T>(ain, base_row + j));
  const float m = block_max(ml, red4);  // its barriers also publish tk, tv

  const uint32_t rows = (uint32_t)len * D;
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(kin + base_row * D, rows * sizeof(T));
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vin + base_row * D, rows * sizeof(T));
  // no gate logits: an empty range, so every logit reads as 0
  const __amdgpu_buffer_rsrc_t ra =
      ain ? make_rsrc(ain + base_row, (uint32_t)len * sizeof(T)) : make_rsrc(kin, 0u);
  f32x4_t acc[C::kBlocks];
#pragma unroll
  for (int k = 0; k < C::kBlocks; ++k) acc[k] = (f32x4_t){0.0f, 0.0f, 0.0f, 0.0f};
  // z: the column sums of the staged gated keys, per lane (channel 16 b + j,
  // tokens g, g + 4, ...), summed over the lane groups and waves at the end
  float zpart[NMB];
#pragma unroll
  for (int b = 0; b < NMB; ++b) zpart[b] = 0.0f;
  float lacc = 0.0f;
  float* X = stg[wave][0];
  float* Y = stg[wave][1];

  // the wave's contiguous quarter of the unit, 16 tokens at a time
  const int q4 = P.chunk / 4, w0 = t0 + wave * q4, w1 = min(t1, w0 + q4);
  RowStream<T, D> sk, sv;
  int tok = w0 + n;
  sk.start(rk, tok, g);
  sv.start(rv, tok, g);
  float al = load1<T>(ra, (uint32_t)tok);
  for (int b0 = w0; b0 < w1; b0 += 16) {
    float kt[NMB][4], vt[NMB][4];
    __asm__ volatile("" ::: "memory");  // taps are re-read from LDS, not held
    sk.conv(tk, g, kt);
    sv.conv(tv, g, vt);
    const float w = tok < t1 ? __expf(al - m) : 0.0f;
    // the next block's rows (out of range past the slice: read as 0, unused)
    tok += 16;
    sk.issue(rk, tok, g);
    sv.issue(rv, tok, g);
    al = load1<T>(ra, (uint32_t)tok);
    if (g == 0) lacc += w;
#pragma unroll
    for (int kq = 0; kq < NMB; ++kq)
#pragma unroll
      for (int i = 0; i < 4; ++i) kt[kq][i] = w * phi_fast(kt[kq][i]);
    wave_lds_sync();  // the previous block's reads of X, Y are done
    stage_sigma<D>(X, n, g, kt);
    stage_sigma<D>(Y, n, g, vt);
    wave_lds_sync();
    token_product<D>(X, Y, lane, acc, zpart);
  }

  float* rec = partials + ((size_t)h * P.units + unit) * P.rec_floats;
  __syncthreads();  // every wave is done with its staging area
  wave_ordered_sum<D>(acc, &stg[0][0][0], rec);
#pragma unroll
  for (int b = 0; b < NMB; ++b) {
    const float zs = sum_groups(zpart[b]);
    if (g == 0) red[wave][16 * b + n] = zs;
  }
  __syncthreads();
  if (tid < D) rec[D * D + tid] = ((red[0][tid] + red[1][tid]) + red[2][tid]) + red[3][tid];
  const float lsum = sum_tokens(lacc);  // lanes of group 0 hold the weights
  if (lane == 0) red4[wave] = lsum;
  __syncthreads();
  if (tid == 0) {
    rec[D * D + D] = m;
    rec[D * D + D + 1] = (red4[0] + red4[1]) + (red4[2] + red4[3]);
  }
}

// ---------------------------------------------------------------------------
// Query pass, matrix-core version.
// ---------------------------------------------------------------------------
// kDS: the unit's dS partial is summed here (d <= 64).  At d = 128 the
// token-sum accumulators and the two d x d operand layouts do not fit one
// CU together, so this kernel writes dnum (to dnum_out, the layout of dy)
// and bwd_dsum_mfma_kernel forms dS from it.
template <typename T, int D, bool kNorm, bool kDS>
__global__ void __launch_bounds__(kThreads, D >= 128 ? 1 : 2)
bwd_query_mfma_kernel(Plan P, const T* __restrict__ qin, const T* __restrict__ rin,
                      const float* __restrict__ dy, const float* __restrict__ conv_w,
                      const float* __restrict__ gamma, const int32_t* __restrict__ cu,
                      const float* __restrict__ Sg, const float* __restrict__ zg,
                      float* __restrict__ dqt, float* __restrict__ dr, float* __restrict__ dsp,
                      float* __restrict__ dgp, float* __restrict__ dnum_out) {
  using C = MF<D>;
  constexpr int NMB = C::NMB;
  __shared__ f32x4_t a1[NMB * NMB * 64];  // num: A[e][c] = S[c][e]
  __shared__ f32x4_t a2[NMB * NMB * 64];  // dQh: A[c][e] = S[c][e]
  __shared__ __attribute__((aligned(16))) float stg[4][2][kDS ? C::kStage : 4];  // [wave][Qh or dnum]
  __shared__ f32x4_t tq[D];
  __shared__ __attribute__((aligned(16))) float zs[D], gs[D], ms[D];
  __shared__ float red[4][D];
  static_assert(!kDS || sizeof(stg) >= D * D * sizeof(float), "staging holds a d x d matrix");
  const int tid = threadIdx.x, lane = tid & 63, n = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.y, unit = blockIdx.x;
  int s, chunk;
  if (!unit_of(P, cu, P.chunk, P.chunks_per_seq, unit, &s, &chunk)) return;
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int t0 = chunk * P.chunk;
  const int t1 = (int)min(len, (int64_t)t0 + P.chunk);
  const size_t sh = (size_t)s * P.heads + h;
  const float* z = zg + sh * D;
  float* sbuf = &stg[0][0][0];
  if constexpr (kDS) stage_matrix<D>(Sg + sh * D * D, sbuf);
  if (tid < D) {
    float w4[4];
    load_taps4(conv_w, P.heads, h, 0, D, P.W, tid, w4);
    tq[tid] = (f32x4_t){w4[0], w4[1], w4[2], w4[3]};
    zs[tid] = z[tid];
    gs[tid] = kNorm ? gamma[(size_t)h * D + tid] : 1.0f;
  }
  float dzacc[NMB][4], dgacc[NMB][4];
#pragma unroll
  for (int kq = 0; kq < NMB; ++kq)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      dzacc[kq][i] = 0.0f;
      dgacc[kq][i] = 0.0f;
    }
  __syncthreads();
  // dQh = S dnum + z dden is formed as S' dnum + z (dden + m . dnum) with
  // S' = S - z m^T, m = (sum_c S[c][.]) / (sum_c z[c]) (the gate-weighted
  // mean value row): the same quantity, but without the cancellation
  // between the two terms when the value rows share a mean (then
  // S dnum ~ z (m . dnum) and o ~ m, and the no-norm dden + m . dnum is
  // formed as -((o - m) . dy) / den directly).
  const float* Ssrc = kDS ? sbuf : Sg + sh * D * D;
  if (tid < D) {
    float cs = 0.0f, zsum = 0.0f;
    for (int c = 0; c < D; ++c) {
      cs += Ssrc[(size_t)c * D + tid];
      zsum += zs[c];
    }
    ms[tid] = zsum > 0.0f ? cs / zsum : 0.0f;
  }
  __syncthreads();
  // the operand layouts, from the staged S, or at d = 128 straight from memory
  build_frags<D, true>(Ssrc, a1);
  build_frags_centred<D>(Ssrc, zs, ms, a2);
  f32x4_t acc3[kDS ? C::kBlocks : 1];
#pragma unroll
  for (int k = 0; k < (kDS ? C::kBlocks : 1); ++k) acc3[k] = (f32x4_t){0.0f, 0.0f, 0.0f, 0.0f};

  const uint32_t rows = (uint32_t)len * D;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(qin + base_row * D, rows * sizeof(T));
  // without the gated norm r is not read (an empty range) and dr not written
  const __amdgpu_buffer_rsrc_t rr =
      kNorm ? make_rsrc(rin + base_row * D, rows * sizeof(T)) : make_rsrc(qin, 0u);
  const __amdgpu_buffer_rsrc_t rdy = make_rsrc(dy + base_row * D, rows * 4u);
  const __amdgpu_buffer_rsrc_t rdq = make_rsrc(dqt + base_row * D, rows * 4u);
  const __amdgpu_buffer_rsrc_t rdr =
      kNorm ? make_rsrc(dr + base_row * D, rows * 4u) : make_rsrc(dqt, 0u);
  const __amdgpu_buffer_rsrc_t rdn =
      kDS ? make_rsrc(dqt, 0u) : make_rsrc(dnum_out + base_row * D, rows * 4u);
  float* X = stg[wave][0];
  float* Y = stg[wave][1];
  __syncthreads();  // fragments built; the staging area is free again

  // the wave's contiguous quarter of the unit, 16 tokens at a time
  const int q4 = P.chunk / 4, w0 = t0 + wave * q4, w1 = min(t1, w0 + q4);
  RowStream<T, D> sq;
  typename Raw<T>::type rraw[NMB];
  u32x4_t dyraw[NMB];
  int tok = w0 + n;
  auto issue_rd = [&](int tk) {
#pragma unroll
    for (int kq = 0; kq < NMB; ++kq) {
      rraw[kq] = Raw<T>::load(rr, eoff<D>(tk, 16 * kq + 4 * g));
      dyraw[kq] = Raw<float>::load(rdy, eoff<D>(tk, 16 * kq + 4 * g));
    }
  };
  sq.start(rq, tok, g);
  issue_rd(tok);
  for (int b0 = w0; b0 < w1; b0 += 16) {
    float qh[NMB][4];
    f32x4_t rv[NMB], dyv[NMB];
    // the A fragments and taps are re-read from LDS each block rather than
    // held in registers across the loop
    __asm__ volatile("" ::: "memory");
    sq.conv(tq, g, qh);
#pragma unroll
    for (int kq = 0; kq < NMB; ++kq) {
      rv[kq] = Raw<T>::widen(rraw[kq]);
      dyv[kq] = Raw<float>::widen(dyraw[kq]);
    }
    const int cur = tok;
    tok += 16;
    sq.issue(rq, tok, g);  // the next block's rows (out of range past the slice: 0, unused)
    issue_rd(tok);
    float zd = 0.0f;
#pragma unroll
    for (int kq = 0; kq < NMB; ++kq) {
      const f32x4_t zr = *reinterpret_cast<const f32x4_t*>(&zs[16 * kq + 4 * g]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        qh[kq][i] = phi_fast(qh[kq][i]);
        zd = fmaf(qh[kq][i], zr[i], zd);
      }
    }
    // num = S^T Qh (MFMA), den = z . Qh
    f32x4_t acc1[NMB];
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) acc1[mb] = (f32x4_t){0.0f, 0.0f, 0.0f, 0.0f};
    contract<D, NMB>(a1, lane, qh, acc1);
    const float inv_den = 1.0f / sum_groups(zd);
    float o[NMB][4], ss = 0.0f;
#pragma unroll
    for (int kq = 0; kq < NMB; ++kq)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        o[kq][i] = acc1[kq][i] * inv_den;
        ss = fmaf(o[kq][i], o[kq][i], ss);
      }
    float dnum[NMB][4], dden, dcen;  // dcen = dden + m . dnum
    if constexpr (kNorm) {
      const float rs = 1.0f / sqrtf(sum_groups(ss) / D + P.eps);
      // gated RMSNorm backward
      float doh[NMB][4], s1 = 0.0f;
#pragma unroll
      for (int kq = 0; kq < NMB; ++kq) {
        const f32x4_t gm = *reinterpret_cast<const f32x4_t*>(&gs[16 * kq + 4 * g]);
        float drv[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float r = rv[kq][i], d = dyv[kq][i];
          const float sig = sigmoid_fast(r), silu = r * sig;
          const float oh = o[kq][i] * rs;
          doh[kq][i] = d * gm[i] * silu;
          dgacc[kq][i] = fmaf(d * oh, silu, dgacc[kq][i]);
          drv[i] = d * oh * gm[i] * sig * (1.0f + r * (1.0f - sig));
          s1 = fmaf(doh[kq][i], o[kq][i], s1);
        }
        store4(rdr, eoff<D>(cur, 16 * kq + 4 * g), drv);
      }
      s1 = sum_groups(s1);
      const float c3 = rs * rs * rs / D * s1;
#pragma unroll
      for (int kq = 0; kq < NMB; ++kq)
#pragma unroll
        for (int i = 0; i < 4; ++i) dnum[kq][i] = (rs * doh[kq][i] - c3 * o[kq][i]) * inv_den;
      // do . o = rs s1 (1 - rs^2 |o|^2 / d) = eps rs^3 s1 exactly (rs^-2 = |o|^2/d + eps):
      // the RMSNorm leaves almost nothing along o, and summing do . o would
      // return mostly the rounding of its terms.
      dden = -P.eps * rs * rs * rs * s1 * inv_den;
      float md = 0.0f;
#pragma unroll
      for (int kq = 0; kq < NMB; ++kq) {
        const f32x4_t mr = *reinterpret_cast<const f32x4_t*>(&ms[16 * kq + 4 * g]);
#pragma unroll
        for (int i = 0; i < 4; ++i) md = fmaf(mr[i], dnum[kq][i], md);
      }
      dcen = dden + sum_groups(md);
    } else {  // y = o: do = dy
      float s2 = 0.0f, s2c = 0.0f;
#pragma unroll
      for (int kq = 0; kq < NMB; ++kq) {
        const f32x4_t mr = *reinterpret_cast<const f32x4_t*>(&ms[16 * kq + 4 * g]);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          dnum[kq][i] = dyv[kq][i] * inv_den;
          s2 = fmaf(dyv[kq][i], o[kq][i], s2);
          s2c = fmaf(dyv[kq][i], o[kq][i] - mr[i], s2c);
        }
      }
      dden = -sum_groups(s2) * inv_den;
      dcen = -sum_groups(s2c) * inv_den;
    }
    // dQh = S' dnum + z (dden + m . dnum)
    f32x4_t acc2[NMB];
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) acc2[mb] = (f32x4_t){0.0f, 0.0f, 0.0f, 0.0f};
    contract<D, NMB>(a2, lane, dnum, acc2);
#pragma unroll
    for (int kq = 0; kq < NMB; ++kq) {
      const f32x4_t zr = *reinterpret_cast<const f32x4_t*>(&zs[16 * kq + 4 * g]);
      float dq[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        // phi'(u) = 1 for u > 0 and e^u = phi(u) <= 1 otherwise: min(phi(u), 1)
        dq[i] = fmaf(zr[i], dcen, acc2[kq][i]) * fminf(qh[kq][i], 1.0f);
        dzacc[kq][i] = fmaf(qh[kq][i], dden, dzacc[kq][i]);
      }
      store4(rdq, eoff<D>(cur, 16 * kq + 4 * g), dq);
    }
    if constexpr (kDS) {
      // dS += sum over the block's tokens of Qh dnum^T
      wave_lds_sync();  // the previous block's reads of X, Y are done
      stage_sigma<D>(X, n, g, qh);
      stage_sigma<D>(Y, n, g, dnum);
      wave_lds_sync();
      token_product<D>(X, Y, lane, acc3);
    } else {
#pragma unroll
      for (int kq = 0; kq < NMB; ++kq) store4(rdn, eoff<D>(cur, 16 * kq + 4 * g), dnum[kq]);
    }
  }

  float* rec = dsp + ((size_t)h * P.units + unit) * P.rec_floats;
  __syncthreads();  // every wave is done with its staging area
  if constexpr (kDS) wave_ordered_sum<D>(acc3, sbuf, rec);
  reduce_sigma<D>(dzacc, red, rec + D * D);
  reduce_sigma<D>(dgacc, red, dgp + ((size_t)h * P.units + unit) * D);
}

// ---------------------------------------------------------------------------
// dS of a unit from the query pass's dnum (d = 128): dS_p = sum_i Qh_i dnum_i^T
// with Qh recomputed exactly as the query pass forms it, the tokens taken in
// the same order (each wave its contiguous quarter, 16 at a time; the four
// waves' partials added in wave order).  Writes S-part of the unit's record;
// the query pass wrote its dz part.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(kThreads, 1)
bwd_dsum_mfma_kernel(Plan P, const T* __restrict__ qin, const float* __restrict__ dnum,
                     const float* __restrict__ conv_w, const int32_t* __restrict__ cu,
                     float* __restrict__ dsp) {
  using C = MF<D>;
  constexpr int NMB = C::NMB;
  __shared__ __attribute__((aligned(16))) float stg[4][2][C::kStage];  // [wave][Qh or dnum]
  __shared__ f32x4_t tq[D];
  static_assert(sizeof(stg) >= D * D * sizeof(float), "staging holds a d x d matrix");
  const int tid = threadIdx.x, lane = tid & 63, n = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.y, unit = blockIdx.x;
  int s, chunk;
  if (!unit_of(P, cu, P.chunk, P.chunks_per_seq, unit, &s, &chunk)) return;
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int t0 = chunk * P.chunk;
  const int t1 = (int)min(len, (int64_t)t0 + P.chunk);
  if (tid < D) {
    float w4[4];
    load_taps4(conv_w, P.heads, h, 0, D, P.W, tid, w4);
    tq[tid] = (f32x4_t){w4[0], w4[1], w4[2], w4[3]};
  }
  __syncthreads();
  const uint32_t rows = (uint32_t)len * D;
  const __amdgpu_buffer_rsrc_t rq = make_rsrc(qin + base_row * D, rows * sizeof(T));
  const __amdgpu_buffer_rsrc_t rdn = make_rsrc(dnum + base_row * D, rows * 4u);
  f32x4_t acc[C::kBlocks];
#pragma unroll
  for (int k = 0; k < C::kBlocks; ++k) acc[k] = (f32x4_t){0.0f, 0.0f, 0.0f, 0.0f};
  float* X = stg[wave][0];
  float* Y = stg[wave][1];

  const int q4 = P.chunk / 4, w0 = t0 + wave * q4, w1 = min(t1, w0 + q4);
  RowStream<T, D> sq;
  u32x4_t dnraw[NMB];
  int tok = w0 + n;
  auto issue_dn = [&](int tk) {
#pragma unroll
    for (int kq = 0; kq < NMB; ++kq) dnraw[kq] = Raw<float>::load(rdn, eoff<D>(tk, 16 * kq + 4 * g));
  };
  sq.start(rq, tok, g);
  issue_dn(tok);
  for (int b0 = w0; b0 < w1; b0 += 16) {
    float qh[NMB][4], dn[NMB][4];
    __asm__ volatile("" ::: "memory");  // taps are re-read from LDS, not held
    sq.conv(tq, g, qh);
#pragma unroll
    for (int kq = 0; kq < NMB; ++kq) {
      const f32x4_t d = Raw<float>::widen(dnraw[kq]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        qh[kq][i] = phi_fast(qh[kq][i]);
        dn[kq][i] = d[i];
      }
    }
    tok += 16;
    sq.issue(rq, tok, g);  // the next block's rows (out of range past the slice: 0, unused)
    issue_dn(tok);
    wave_lds_sync();  // the previous block's reads of X, Y are done
    stage_sigma<D>(X, n, g, qh);
    stage_sigma<D>(Y, n, g, dn);
    wave_lds_sync();
    token_product<D>(X, Y, lane, acc);
  }
  float* rec = dsp + ((size_t)h * P.units + unit) * P.rec_floats;
  __syncthreads();  // every wave is done with its staging area
  wave_ordered_sum<D>(acc, &stg[0][0][0], rec);
}

// ---------------------------------------------------------------------------
// Key pass, matrix-core version: no token sums, so the waves run their
// 16-token blocks independently.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(kThreads, D >= 128 ? 1 : 2)
bwd_key_mfma_kernel(Plan P, const T* __restrict__ kin, const T* __restrict__ vin,
                    const T* __restrict__ ain, const float* __restrict__ conv_w,
                    const int32_t* __restrict__ cu, const float* __restrict__ dSg,
                    const float* __restrict__ mz, float* __restrict__ dkt,
                    float* __restrict__ dvt, float* __restrict__ da) {
  using C = MF<D>;
  constexpr int NMB = C::NMB;
  __shared__ f32x4_t a4[NMB * NMB * 64];  // t = dS vt: A[c][e] = dS[c][e]
  __shared__ f32x4_t a5[NMB * NMB * 64];  // dvt = dS^T P: A[e][c] = dS[c][e]
  // dS staged for the layouts (d <= 64; at d = 128 they are built from memory)
  constexpr bool kStaged = D <= 64;
  __shared__ __attribute__((aligned(16))) float sbuf[kStaged ? D * D : 4];
  __shared__ f32x4_t tk[D], tv[D];
  __shared__ __attribute__((aligned(16))) float dzs[D];
  const int tid = threadIdx.x, lane = tid & 63, n = lane & 15, g = lane >> 4;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = blockIdx.y, unit = blockIdx.x;
  int s, chunk;
  if (!unit_of(P, cu, P.chunk, P.chunks_per_seq, unit, &s, &chunk)) return;
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int t0 = chunk * P.chunk;
  const int t1 = (int)min(len, (int64_t)t0 + P.chunk);
  const size_t sh = (size_t)s * P.heads + h;
  const float* dS = dSg + sh * (D * D + D);
  if constexpr (kStaged) stage_matrix<D>(dS, sbuf);
  if (tid < D) {
    float w4[4];
    load_taps4(conv_w, P.heads, h, 1, D, P.W, tid, w4);
    tk[tid] = (f32x4_t){w4[0], w4[1], w4[2], w4[3]};
    load_taps4(conv_w, P.heads, h, 2, D, P.W, tid, w4);
    tv[tid] = (f32x4_t){w4[0], w4[1], w4[2], w4[3]};
    dzs[tid] = dS[D * D + tid];
  }
  const float M = mz[2 * sh], Z = mz[2 * sh + 1];
  const float invZ = Z > 0.0f ? 1.0f / Z : 0.0f;
  __syncthreads();
  build_frags<D, false>(kStaged ? sbuf : dS, a4);
  build_frags<D, true>(kStaged ? sbuf : dS, a5);
  __syncthreads();

  const uint32_t rows = (uint32_t)len * D;
  const __amdgpu_buffer_rsrc_t rk = make_rsrc(kin + base_row * D, rows * sizeof(T));
  const __amdgpu_buffer_rsrc_t rv = make_rsrc(vin + base_row * D, rows * sizeof(T));
  // absent gate logits read as 0 and an absent da is not written (empty ranges)
  const __amdgpu_buffer_rsrc_t ra =
      ain ? make_rsrc(ain + base_row, (uint32_t)len * sizeof(T)) : make_rsrc(kin, 0u);
  const __amdgpu_buffer_rsrc_t rdk = make_rsrc(dkt + base_row * D, rows * 4u);
  const __amdgpu_buffer_rsrc_t rdv = make_rsrc(dvt + base_row * D, rows * 4u);
  const __amdgpu_buffer_rsrc_t rda =
      da ? make_rsrc(da + base_row, (uint32_t)t1 * 4u) : make_rsrc(dkt, 0u);

  // the wave's contiguous quarter of the unit, 16 tokens at a time
  const int q4 = P.chunk / 4, w0 = t0 + wave * q4, w1 = min(t1, w0 + q4);
  RowStream<T, D> sk, sv;
  int tok = w0 + n;
  sk.start(rk, tok, g);
  sv.start(rv, tok, g);
  float al = load1<T>(ra, (uint32_t)tok);
  for (int b0 = w0; b0 < w1; b0 += 16) {
    float kt[NMB][4], vt[NMB][4];
    // the A fragments are re-read from LDS each block rather than held in
    // registers across the loop
    __asm__ volatile("" ::: "memory");
    sk.conv(tk, g, kt);
    sv.conv(tv, g, vt);
    const float gj = __expf(al - M) * invZ;
    const int cur = tok;
    tok += 16;
    sk.issue(rk, tok, g);  // the next block's rows (out of range past the slice: 0, unused)
    sv.issue(rv, tok, g);
    al = load1<T>(ra, (uint32_t)tok);
    // t = dS vt + dz
    f32x4_t acc4[NMB];
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) acc4[mb] = (f32x4_t){0.0f, 0.0f, 0.0f, 0.0f};
    contract<D, NMB>(a4, lane, vt, acc4);
    float pk[NMB][4], dgl = 0.0f;
#pragma unroll
    for (int kq = 0; kq < NMB; ++kq) {
      const f32x4_t dzr = *reinterpret_cast<const f32x4_t*>(&dzs[16 * kq + 4 * g]);
      float dk[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float u = kt[kq][i];
        const float p = phi_fast(u);
        const float t = acc4[kq][i] + dzr[i];
        dk[i] = gj * t * (u > 0.0f ? 1.0f : p);
        dgl = fmaf(p, t, dgl);
        pk[kq][i] = p;
      }
      store4(rdk, eoff<D>(cur, 16 * kq + 4 * g), dk);
    }
    const float dg = sum_groups(dgl);
    if (g == 0)
      __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, gj * dg), rda,
                                            (uint32_t)cur * 4u, 0, 0);
    // dvt = g dS^T P
    f32x4_t acc5[NMB];
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) acc5[mb] = (f32x4_t){0.0f, 0.0f, 0.0f, 0.0f};
    contract<D, NMB>(a5, lane, pk, acc5);
#pragma unroll
    for (int kq = 0; kq < NMB; ++kq) {
      float dv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) dv[i] = gj * acc5[kq][i];
      store4(rdv, eoff<D>(cur, 16 * kq + 4 * g), dv);
    }
  }
}

// ---------------------------------------------------------------------------
// Conv1D backward, streaming version: grid (units, H, 3 tensors).  Thread
// (run, c4) handles channels 4 c4 .. 4 c4 + 3 of runs of 8 consecutive
// tokens; the run's dxt rows m .. m + 10 and x rows m - 3 .. m + 7 are loaded
// at once (out-of-range rows read 0).  The tap gradients of the unit are
// summed over the runs in run order.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(kThreads)
bwd_conv_stream_kernel(Plan P, const T* __restrict__ qin, const T* __restrict__ kin,
                       const T* __restrict__ vin, const float* __restrict__ dxt_all,
                       const float* __restrict__ conv_w, const int32_t* __restrict__ cu,
                       float* __restrict__ dq, float* __restrict__ dk, float* __restrict__ dv,
                       float* __restrict__ dcp, size_t act_elems) {
  constexpr int CG = D / 4, RUNS = kThreads / CG, RL = 8;
  __shared__ f32x4_t red[RUNS][D];
  const int tid = threadIdx.x, c4 = tid % CG, run = tid / CG, c0 = 4 * c4;
  const int h = blockIdx.y, unit = blockIdx.x, tensor = blockIdx.z;
  int s, chunk;
  if (!unit_of(P, cu, P.chunk, P.chunks_per_seq, unit, &s, &chunk)) return;
  int64_t len, base_row;
  seq_geometry(P, cu, s, h, &len, &base_row);
  const int t0 = chunk * P.chunk;
  const int t1 = (int)min(len, (int64_t)t0 + P.chunk);
  const T* x = tensor == 0 ? qin : tensor == 1 ? kin : vin;
  float* out = tensor == 0 ? dq : tensor == 1 ? dk : dv;
  const uint32_t rows = (uint32_t)len * D;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x + base_row * D, rows * sizeof(T));
  const __amdgpu_buffer_rsrc_t rd =
      make_rsrc(dxt_all + (size_t)tensor * act_elems + base_row * D, rows * 4u);
  const __amdgpu_buffer_rsrc_t ro = make_rsrc(out + base_row * D, (uint32_t)t1 * D * 4u);
  float w4[4][4];
#pragma unroll
  for (int c = 0; c < 4; ++c) load_taps4(conv_w, P.heads, h, tensor, D, P.W, c0 + c, w4[c]);
  float dc[4][4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int t = 0; t < 4; ++t) dc[c][t] = 0.0f;
  for (int b = t0 + run * RL; b < t1; b += RUNS * RL) {
    f32x4_t d[RL + 3], xx[RL + 3];
#pragma unroll
    for (int r = 0; r < RL + 3; ++r) {
      d[r] = load4<float>(rd, eoff<D>(b + r, c0));
      xx[r] = load4<T>(rx, eoff<D>(b - 3 + r, c0));
    }
#pragma unroll
    for (int j = 0; j < RL; ++j) {
      // tokens past t1: their dxt rows read 0 (past len) or belong to the
      // next unit, and their stores fall outside the range; no tap sums
      const bool live = b + j < t1;
      float y[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        float acc = w4[c][3] * d[j][c];
        acc = fmaf(w4[c][2], d[j + 1][c], acc);
        acc = fmaf(w4[c][1], d[j + 2][c], acc);
        y[c] = fmaf(w4[c][0], d[j + 3][c], acc);
        const float dd = live ? d[j][c] : 0.0f;
#pragma unroll
        for (int t = 0; t < 4; ++t) dc[c][t] = fmaf(dd, xx[j + t][c], dc[c][t]);
      }
      store4(ro, eoff<D>(b + j, c0), y);
    }
  }
#pragma unroll
  for (int c = 0; c < 4; ++c) red[run][c0 + c] = (f32x4_t){dc[c][0], dc[c][1], dc[c][2], dc[c][3]};
  __syncthreads();
  if (tid < D) {
    f32x4_t acc = red[0][tid];
    for (int r = 1; r < RUNS; ++r) acc += red[r][tid];
    *reinterpret_cast<f32x4_t*>(dcp + (((size_t)h * P.units + unit) * 3 + tensor) * D * 4 + tid * 4) = acc;
  }
}

template <typename T, int D>
gbla_status run_backward(const Plan& p, const BwdLayout& L, const void* q, const void* k,
                         const void* v, const void* a, const void* r, const float* conv_w,
                         const float* gamma, const int32_t* cu, const float* dy, void* ws,
                         float* dq, float* dk, float* dv, float* da, float* dr, float* dconv,
                         float* dgamma, hipStream_t st) {
  unsigned char* base = static_cast<unsigned char*>(ws);
  float* S = reinterpret_cast<float*>(base + L.off_S);
  float* z = reinterpret_cast<float*>(base + L.off_z);
  float* mz = reinterpret_cast<float*>(base + L.off_mz);
  float* dsp = reinterpret_cast<float*>(base + L.off_dsp);
  float* dS = reinterpret_cast<float*>(base + L.off_dS);
  float* dgp = reinterpret_cast<float*>(base + L.off_dgp);
  float* dxt = reinterpret_cast<float*>(base + L.off_dxt);
  float* dcp = reinterpret_cast<float*>(base + L.off_dcp);
  const size_t act_elems = (size_t)p.tokens * p.heads * D;
  const dim3 grid(p.units, p.heads);
  // Matrix-core kernels for every head dim; 32-bit buffer offsets need every
  // fp32 (sequence, head) slice below 2^31 bytes.
  const bool small_slices = (int64_t)p.rows * D * 4 < (int64_t(1) << 31);
  constexpr int kElems = D * D + D;
  const dim3 cgrid((unsigned)((int64_t)p.nseq * p.heads), (kElems + kThreads - 1) / kThreads);
  bool mfma = small_slices;
  if (mfma) {
    // d = 128: the query pass writes dnum into the third dxt slot (the key
    // pass fills it only afterwards) and bwd_dsum_mfma_kernel sums dS from it
    constexpr bool kDS = D <= 64;
    float* dnum = dxt + 2 * act_elems;
    hipLaunchKernelGGL((bwd_state_mfma_kernel<T, D>), grid, dim3(kThreads), 0, st, p,
                       (const T*)k, (const T*)v, (const T*)a, conv_w, cu, dsp);
    gbla_status e = launch_combine_f32(p, cu, dsp, S, z, mz, st);
    if (e != GBLA_OK) return e;
    if (gamma)
      hipLaunchKernelGGL((bwd_query_mfma_kernel<T, D, true, kDS>), grid, dim3(kThreads), 0, st, p,
                         (const T*)q, (const T*)r, dy, conv_w, gamma, cu, (const float*)S,
                         (const float*)z, dxt, dr, dsp, dgp, dnum);
    else
      hipLaunchKernelGGL((bwd_query_mfma_kernel<T, D, false, kDS>), grid, dim3(kThreads), 0, st, p,
                         (const T*)q, (const T*)r, dy, conv_w, gamma, cu, (const float*)S,
                         (const float*)z, dxt, dr, dsp, dgp, dnum);
    if constexpr (!kDS)
      hipLaunchKernelGGL((bwd_dsum_mfma_kernel<T, D>), grid, dim3(kThreads), 0, st, p,
                         (const T*)q, (const float*)dnum, conv_w, cu, dsp);
    hipLaunchKernelGGL((bwd_dscombine_kernel<D>), cgrid, dim3(kThreads), 0, st, p, cu,
                       (const float*)dsp, dS);
    hipLaunchKernelGGL((bwd_key_mfma_kernel<T, D>), grid, dim3(kThreads), 0, st, p,
                       (const T*)k, (const T*)v, (const T*)a, conv_w, cu, (const float*)dS,
                       (const float*)mz, dxt + act_elems, dxt + 2 * act_elems, da);
  }
  if (!mfma) {
    hipLaunchKernelGGL((bwd_state_kernel<T, D>), grid, dim3(kThreads), 0, st, p, (const T*)k,
                       (const T*)v, (const T*)a, conv_w, cu, dsp);
    gbla_status e = launch_combine_f32(p, cu, dsp, S, z, mz, st);
    if (e != GBLA_OK) return e;
    if (gamma)
      hipLaunchKernelGGL((bwd_query_kernel<T, D, true>), grid, dim3(kThreads), 0, st, p,
                         (const T*)q, (const T*)r, dy, conv_w, gamma, cu, S, z, dxt, dr, dsp, dgp);
    else
      hipLaunchKernelGGL((bwd_query_kernel<T, D, false>), grid, dim3(kThreads), 0, st, p,
                         (const T*)q, (const T*)r, dy, conv_w, gamma, cu, S, z, dxt, dr, dsp, dgp);
    hipLaunchKernelGGL((bwd_dscombine_kernel<D>), cgrid, dim3(kThreads), 0, st, p, cu,
                       (const float*)dsp, dS);
    hipLaunchKernelGGL((bwd_key_kernel<T, D>), grid, dim3(kThreads), 0, st, p, (const T*)k,
                       (const T*)v, (const T*)a, conv_w, cu, (const float*)dS, (const float*)mz,
                       dxt + act_elems, dxt + 2 * act_elems, da);
  }
  if (small_slices)
    hipLaunchKernelGGL((bwd_conv_stream_kernel<T, D>), dim3(p.units, p.heads, 3), dim3(kThreads),
                       0, st, p, (const T*)q, (const T*)k, (const T*)v, (const float*)dxt, conv_w,
                       cu, dq, dk, dv, dcp, act_elems);
  else
    hipLaunchKernelGGL((bwd_conv_kernel<T, D>), dim3(p.units, p.heads, 3), dim3(kThreads), 0, st,
                       p, (const T*)q, (const T*)k, (const T*)v, (const float*)dxt, conv_w, cu,
                       dq, dk, dv, dcp, act_elems);
  const int nout = D + 3 * D * p.W;
  hipLaunchKernelGGL((bwd_param_kernel<D>), dim3(p.heads, (nout + 63) / 64), dim3(kThreads), 0, st, p, cu,
                     (const float*)dgp, (const float*)dcp, dgamma, dconv);
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}

}  // namespace

gbla_status launch_backward(const Plan& p, const BwdLayout& L, const void* q, const void* k,
                            const void* v, const void* a, const void* r, const float* conv_w,
                            const float* gamma, const int32_t* cu, const float* dy, void* ws,
                            float* dq, float* dk, float* dv, float* da, float* dr, float* dconv,
                            float* dgamma, hipStream_t st) {
#define GBLA_BWD(TT, DD)                                                                      \
  return run_backward<TT, DD>(p, L, q, k, v, a, r, conv_w, gamma, cu, dy, ws, dq, dk, dv, da, \
                              dr, dconv, dgamma, st)
  if (p.dtype == GBLA_BF16) {
    if (p.d == 32) GBLA_BWD(uint16_t, 32);
    if (p.d == 64) GBLA_BWD(uint16_t, 64);
    if (p.d == 128) GBLA_BWD(uint16_t, 128);
  } else {
    if (p.d == 32) GBLA_BWD(float, 32);
    if (p.d == 64) GBLA_BWD(float, 64);
    if (p.d == 128) GBLA_BWD(float, 128);
  }
#undef GBLA_BWD
  return GBLA_ERR_UNSUPPORTED;
}

}  // namespace gbla
