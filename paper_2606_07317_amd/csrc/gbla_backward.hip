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
  for (int64_t j = t0 + tid; j < t1; j += kThreads) ml = fmaxf(ml, act<T>(ain, base_row + j));
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
      const float w = live ? expf(act<T>(ain, base_row + j) - m) : 0.0f;
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
template <typename T, int D>
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
    gm[cc] = gamma[(size_t)h * D + e];
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
      float dnum[CPL], s2 = 0.0f;
#pragma unroll
      for (int cc = 0; cc < CPL; ++cc) {
        const float dov = rs * doh[cc] - rs * rs * rs / D * s1 * o[cc];
        dnum[cc] = dov / den;
        if (chan<D>(lane, cc) < D) s2 = fmaf(dov, o[cc], s2);
      }
      const float dden = -wave_sum(s2) / den;
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
  const float* recs = dsp + ((size_t)h * P.units + first) * P.rec_floats;
  float acc = 0.0f;
  for (int p = 0; p < count; ++p) acc += recs[(size_t)p * P.rec_floats + x];
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
    if (lane == 0) da[row] = gj * dg;
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
// dgamma and the tap gradients: per head, the fixed-order sum over the
// head's units (every sequence of the batch).  grid (H).
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(kThreads)
bwd_param_kernel(Plan P, const int32_t* __restrict__ cu, const float* __restrict__ dgp,
                 const float* __restrict__ dcp, float* __restrict__ dgamma,
                 float* __restrict__ dconv) {
  const int h = blockIdx.x, tid = threadIdx.x;
  const int total = P.ragged ? units_before(cu, P.nseq, P.chunk) : P.chunks_per_seq * P.nseq;
  if (tid < D) {
    float acc = 0.0f;
    for (int u = 0; u < total; ++u) acc += dgp[((size_t)h * P.units + u) * D + tid];
    dgamma[(size_t)h * D + tid] = acc;
  }
  if (!dconv) return;
  for (int idx = tid; idx < 3 * D * P.W; idx += kThreads) {
    const int tensor = idx / (D * P.W), rem = idx % (D * P.W);
    const int e = rem / P.W, tw = rem % P.W;
    const int t4 = tw + (4 - P.W);  // right-aligned slot of tap tw
    float acc = 0.0f;
    for (int u = 0; u < total; ++u)
      acc += dcp[(((size_t)h * P.units + u) * 3 + tensor) * D * 4 + e * 4 + t4];
    dconv[(((size_t)tensor * P.heads + h) * D + e) * P.W + tw] = acc;
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
  hipLaunchKernelGGL((bwd_state_kernel<T, D>), grid, dim3(kThreads), 0, st, p, (const T*)k,
                     (const T*)v, (const T*)a, conv_w, cu, dsp);
  gbla_status e = launch_combine_f32(p, cu, dsp, S, z, mz, st);
  if (e != GBLA_OK) return e;
  hipLaunchKernelGGL((bwd_query_kernel<T, D>), grid, dim3(kThreads), 0, st, p, (const T*)q,
                     (const T*)r, dy, conv_w, gamma, cu, S, z, dxt, dr, dsp, dgp);
  constexpr int kElems = D * D + D;
  hipLaunchKernelGGL((bwd_dscombine_kernel<D>),
                     dim3((unsigned)((int64_t)p.nseq * p.heads), (kElems + kThreads - 1) / kThreads),
                     dim3(kThreads), 0, st, p, cu, (const float*)dsp, dS);
  hipLaunchKernelGGL((bwd_key_kernel<T, D>), grid, dim3(kThreads), 0, st, p, (const T*)k,
                     (const T*)v, (const T*)a, conv_w, cu, (const float*)dS, (const float*)mz,
                     dxt + act_elems, dxt + 2 * act_elems, da);
  hipLaunchKernelGGL((bwd_conv_kernel<T, D>), dim3(p.units, p.heads, 3), dim3(kThreads), 0, st, p,
                     (const T*)q, (const T*)k, (const T*)v, (const float*)dxt, conv_w, cu, dq, dk,
                     dv, dcp, act_elems);
  hipLaunchKernelGGL((bwd_param_kernel<D>), dim3(p.heads), dim3(kThreads), 0, st, p, cu,
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
