// gbla_layer.hip -- the projections of the full GBLA layer (Section 2.1):
//     Xt = Conv1D(X),  [Q | K | V | R | a] = Xt Wp^T
//
// conv_x_kernel  streams X once: causal depthwise conv in fp32, Xt rounded
//                to bf16 into the workspace (a bf16 layer stores it so).
// proj_kernel    P = Xt Wp^T on v_mfma_f32_32x32x16_bf16 (fp32 accumulation):
//                a workgroup of 4 waves (2 x 2, 64 x 64 each) computes a
//                128-token x 128-feature tile, 64 model channels per K step,
//                the next step's rows loaded into registers while the
//                current step's products run.  The epilogue rounds P to bf16
//                and scatters every feature to the head-major layout the
//                attention kernels read ([B, H, n, d] / [B, H, n]), through
//                LDS so that each lane writes 16-byte pieces.
// The conv is a separate pass rather than part of the tile staging: redone
// for every feature tile, its vector work would compete with the products
// (measured: 0.36 against 0.54 PFLOP/s for the GEMM), while the pass itself
// costs one read and one write of X.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gbla_device.h"
#include "gbla_ext.h"
#include "gbla_plan.h"

namespace gbla {
namespace {

constexpr int kBM = 128, kBN = 128, kBK = 64;
constexpr int kRowBytes = kBK * 2;           // one tile row of bf16
constexpr int kTileBytes = 128 * kRowBytes;  // 16 KB

// Byte offset of 16-byte chunk `c` of row `r` in a tile (chunks XOR-swizzled
// by the row, so the MFMA operand reads of 32 rows spread over the banks).
__device__ __forceinline__ int tile_off(int r, int c) { return r * kRowBytes + ((c ^ (r & 7)) << 4); }

__device__ __forceinline__ u32x4_t bload(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

// First token of the sequence that holds token m (global token index).
__device__ __forceinline__ int seq_start(const LayerPlan& P, const int32_t* cu, int m) {
  if (!P.ragged) return m - m % P.rows;
  int lo = 0, hi = P.nseq;  // cu[lo] <= m < cu[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (cu[mid] <= m) lo = mid; else hi = mid;
  }
  return cu[lo];
}

// One past the last token of the sequence that holds token m (packed batch).
__device__ __forceinline__ int seq_end(const LayerPlan& P, const int32_t* cu, int m) {
  int lo = 0, hi = P.nseq;  // cu[lo] <= m < cu[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (cu[mid] <= m) lo = mid; else hi = mid;
  }
  return cu[hi];
}

// ---------------------------------------------------------------------------
// conv_x_kernel: Xt = Conv1D(X) in fp32, rounded to bf16, into the
// workspace.  grid (d_model / 128, tokens / 256): thread (run, chunk) takes
// eight channels of 16 consecutive tokens from the 19 rows covering their
// windows (the three rows before the run come from the previous run's
// tokens, or read as zero before the sequence start).
// ---------------------------------------------------------------------------
constexpr int kConvRun = 16;

__global__ void __launch_bounds__(kThreads)
conv_x_kernel(LayerPlan P, const uint16_t* __restrict__ x, const float* __restrict__ conv_x,
              const int32_t* __restrict__ cu, uint16_t* __restrict__ xt) {
  const int tid = threadIdx.x, chunk = tid & 15, run = tid >> 4;
  const int c0 = blockIdx.x * 128 + 8 * chunk;
  const int t0 = blockIdx.y * (16 * kConvRun) + run * kConvRun;
  const int K = P.d_model, M = P.tokens;
  if (t0 >= M || c0 >= K) return;  // no barrier follows
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, (uint32_t)((int64_t)M * K * 2));
  float w[8][4];
#pragma unroll
  for (int j = 0; j < 8; ++j)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int ti = t - (4 - P.W);
      w[j][t] = ti >= 0 ? conv_x[(size_t)(c0 + j) * P.W + ti] : 0.0f;
    }
  u32x4_t raw[kConvRun + 3];
#pragma unroll
  for (int u = 0; u < kConvRun + 3; ++u)
    raw[u] = bload(rx, (uint32_t)(((int64_t)(t0 - 3 + u) * K + c0) * 2));
  int start = seq_start(P, cu, t0), next = P.ragged ? seq_end(P, cu, t0) : start + P.rows;
#pragma unroll
  for (int i = 0; i < kConvRun; ++i) {
    const int m = t0 + i;
    if (m >= M) break;
    if (m >= next) {  // a new sequence starts inside the run
      start = seq_start(P, cu, m);
      next = P.ragged ? seq_end(P, cu, m) : start + P.rows;
    }
    const int back = m - start;
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.0f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      if (3 - t > back) continue;  // row before the sequence start
      const u32x4_t v = raw[i + t];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[2 * q] = fmaf(w[2 * q][t], bf16_lo(v[q]), acc[2 * q]);
        acc[2 * q + 1] = fmaf(w[2 * q + 1][t], bf16_hi(v[q]), acc[2 * q + 1]);
      }
    }
    u32x4_t o;
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = pack_bf16x2(acc[2 * q], acc[2 * q + 1]);
    *reinterpret_cast<u32x4_t*>(xt + (size_t)m * K + c0) = o;
  }
}

// ---------------------------------------------------------------------------
// proj_kernel: P = Xt Wp^T on bf16 MFMA, scattered to the attention layout.
// grid (features / 128, tokens / 128); 4 waves (2 x 2) of 64 x 64.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kThreads, 2)
proj_kernel(LayerPlan P, const uint16_t* __restrict__ xt, const uint16_t* __restrict__ wp,
            uint16_t* __restrict__ q, uint16_t* __restrict__ k, uint16_t* __restrict__ v,
            uint16_t* __restrict__ r, uint16_t* __restrict__ a) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[2][2][kTileBytes];  // [buf][Xt or W]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int n0 = blockIdx.x * kBN, m0 = blockIdx.y * kBM;
  const int K = P.d_model, M = P.tokens, N = P.features;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(xt, (uint32_t)((int64_t)M * K * 2));
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(wp, (uint32_t)((int64_t)N * K * 2));

  u32x4_t xraw[4], wraw[4];
  auto issue = [&](int kt) {
    const int k0 = kt * kBK;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = tid + 256 * j, row = c >> 3, ch = c & 7;
      xraw[j] = bload(rx, (uint32_t)(((int64_t)(m0 + row) * K + k0 + 8 * ch) * 2));
      wraw[j] = bload(rw, (uint32_t)(((int64_t)(n0 + row) * K + k0 + 8 * ch) * 2));
    }
  };
  auto commit = [&](int buf) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = tid + 256 * j, row = c >> 3, ch = c & 7;
      *reinterpret_cast<u32x4_t*>(&lds[buf][0][tile_off(row, ch)]) = xraw[j];
      *reinterpret_cast<u32x4_t*>(&lds[buf][1][tile_off(row, ch)]) = wraw[j];
    }
  };

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;

  const int nk = K / kBK;
  const int half = lane >> 5, l32 = lane & 31;
  issue(0);
  commit(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) issue(kt + 1);  // in flight during the products
    const unsigned char* A = lds[buf][0];
    const unsigned char* B = lds[buf][1];
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      const int c = 2 * ks + half;
      u32x4_t af[2], bf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) af[i] = *reinterpret_cast<const u32x4_t*>(A + tile_off(64 * wm + 32 * i + l32, c));
#pragma unroll
      for (int j = 0; j < 2; ++j) bf[j] = *reinterpret_cast<const u32x4_t*>(B + tile_off(64 * wn + 32 * j + l32, c));
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, af[i]),
                                                              __builtin_bit_cast(bf16x8_t, bf[j]),
                                                              acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) commit(buf ^ 1);
    __syncthreads();
  }

  // Epilogue.  The wave's 64 x 64 tile goes through LDS as bf16 rows
  // (stride 72 elements), then each lane writes 16-byte pieces: eight
  // consecutive features of one token, which are eight consecutive channels
  // of one head (d is a multiple of 8).  Gate-logit features, whose
  // destinations are H rows apart, are written one by one.
  constexpr int kEpRow = 72;
  uint16_t* ep = reinterpret_cast<uint16_t*>(&lds[0][0][0]) + wave * 64 * kEpRow;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int row = 32 * i + 8 * (rr >> 2) + 4 * half + (rr & 3);
        ep[row * kEpRow + 32 * j + l32] = (uint16_t)(pack_bf16x2(acc[i][j][rr], 0.0f) & 0xffffu);
      }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const int Hd = P.heads * P.d;
  const int piece = lane & 7;              // eight features 8 piece .. 8 piece + 7
  const int nb = n0 + 64 * wn + 8 * piece;  // first feature of the piece
#pragma unroll
  for (int pass = 0; pass < 8; ++pass) {
    const int row = 8 * pass + (lane >> 3);
    const int m = m0 + 64 * wm + row;
    if (m >= M || nb >= N) continue;
    // token m: dense slice (b, position) or packed row
    int64_t b = 0, pos = m;
    if (!P.ragged) {
      b = m / P.rows;
      pos = m - b * P.rows;
    }
    const uint16_t* src = ep + row * kEpRow + 8 * piece;
    if (nb + 8 <= 4 * Hd) {
      const int blk = nb / Hd, h = (nb % Hd) / P.d, e = nb % P.d;
      uint16_t* dst = blk == 0 ? q : blk == 1 ? k : blk == 2 ? v : r;
      const int64_t orow = P.ragged ? (int64_t)h * M + m : (b * P.heads + h) * P.rows + pos;
      *reinterpret_cast<u32x4_t*>(dst + orow * P.d + e) = *reinterpret_cast<const u32x4_t*>(src);
    } else {
#pragma unroll
      for (int f = 0; f < 8; ++f) {
        const int n = nb + f;
        if (n >= N) break;
        const int h = n - 4 * Hd;  // gate logits (every earlier feature is in a 16-byte piece)
        const int64_t orow = P.ragged ? (int64_t)h * M + m : (b * P.heads + h) * P.rows + pos;
        a[orow] = src[f];
      }
    }
  }
}

}  // namespace

gbla_status launch_project(const LayerPlan& p, const void* x, const float* conv_x,
                           const void* w_proj, const int32_t* cu, void* xt, void* q, void* k,
                           void* v, void* r, void* a, hipStream_t st) {
  if (p.tokens == 0) return GBLA_OK;
  hipLaunchKernelGGL(conv_x_kernel, dim3((p.d_model + 127) / 128, (p.tokens + 16 * kConvRun - 1) / (16 * kConvRun)),
                     dim3(kThreads), 0, st, p, (const uint16_t*)x, conv_x, cu, (uint16_t*)xt);
  const dim3 grid((p.features + kBN - 1) / kBN, (p.tokens + kBM - 1) / kBM);
  hipLaunchKernelGGL(proj_kernel, grid, dim3(kThreads), 0, st, p, (const uint16_t*)xt,
                     (const uint16_t*)w_proj, (uint16_t*)q, (uint16_t*)k, (uint16_t*)v,
                     (uint16_t*)r, (uint16_t*)a);
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}

}  // namespace gbla
