// gbla_layer.hip -- the projections of the full GBLA layer (Section 2.1):
//     Xt = Conv1D(X),  [Q | K | V | R | a] = Xt Wp^T
// as one bf16 MFMA GEMM with the conv fused into the staging of the X tile
// and an epilogue that scatters every output feature to the head-major
// layout the attention kernels read ([B, H, n, d] / [B, H, n]).
//
// Tiles: a workgroup of 256 threads (4 waves, 2 x 2) computes a 128-token x
// 128-feature tile of P = Xt Wp^T, 64 model channels per K step, with
// v_mfma_f32_32x32x16_bf16 (fp32 accumulation).  Each K step's X rows (plus
// the W-1 rows before the tile) and Wp rows are loaded into registers one
// step ahead, then the conv is applied in fp32 while the X tile is written
// to LDS: thread (strip, chunk) convolves four consecutive tokens of eight
// channels from the seven rows that cover their windows, so each element is
// convolved once per tile and the conv never reaches HBM.  Xt is rounded to
// bf16 there, and P to bf16 in the epilogue: a bf16 layer keeps both in
// bf16.  The conv stops at each sequence start (cu_seqlens for packed
// batches).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gbla_device.h"
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

__global__ void __launch_bounds__(kThreads, 2)
proj_kernel(LayerPlan P, const uint16_t* __restrict__ x, const float* __restrict__ conv_x,
            const uint16_t* __restrict__ wp, const int32_t* __restrict__ cu,
            uint16_t* __restrict__ q, uint16_t* __restrict__ k, uint16_t* __restrict__ v,
            uint16_t* __restrict__ r, uint16_t* __restrict__ a) {
  __shared__ __attribute__((aligned(16))) unsigned char lds[2][2][kTileBytes];  // [buf][X or W]
  __shared__ __attribute__((aligned(16))) f32x4_t taps[2][kBK];                // [buf][channel]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int n0 = blockIdx.x * kBN, m0 = blockIdx.y * kBM;
  const int K = P.d_model, M = P.tokens, N = P.features;

  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, (uint32_t)((int64_t)M * K * 2));
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(wp, (uint32_t)((int64_t)N * K * 2));

  // X staging role: strip of 4 tokens, chunk of 8 channels.
  const int chunk = tid & 7, strip = tid >> 3;
  const int xr0 = 4 * strip;  // first tile row of the strip
  // valid[i] bit t: tap t of output row i reads a row of its own sequence
  uint32_t valid = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + xr0 + i;
    if (m < M) {
      const int back = m - seq_start(P, cu, m);  // rows available before m
#pragma unroll
      for (int t = 0; t < 4; ++t)
        if (3 - t <= back && t >= 4 - P.W) valid |= 1u << (4 * i + t);
    }
  }

  u32x4_t xraw[7], wraw[4];
  f32x4_t tapraw = {0.0f, 0.0f, 0.0f, 0.0f};
  auto issue = [&](int kt) {
    const int k0 = kt * kBK;
#pragma unroll
    for (int u = 0; u < 7; ++u) {
      const int m = m0 + xr0 - 3 + u;
      xraw[u] = bload(rx, (uint32_t)(((int64_t)m * K + k0 + 8 * chunk) * 2));
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = tid + 256 * j, row = c >> 3, ch = c & 7;
      wraw[j] = bload(rw, (uint32_t)(((int64_t)(n0 + row) * K + k0 + 8 * ch) * 2));
    }
    if (tid < kBK) {
      float w4[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int ti = t - (4 - P.W);
        w4[t] = ti >= 0 ? conv_x[(size_t)(k0 + tid) * P.W + ti] : 0.0f;
      }
      tapraw = (f32x4_t){w4[0], w4[1], w4[2], w4[3]};
    }
  };
  auto commit = [&](int buf) {
    if (tid < kBK) taps[buf][tid] = tapraw;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int c = tid + 256 * j, row = c >> 3, ch = c & 7;
      *reinterpret_cast<u32x4_t*>(&lds[buf][1][tile_off(row, ch)]) = wraw[j];
    }
  };
  // The conv of the strip's rows (taps of this step must be in LDS).
  auto commit_x = [&](int buf) {
    float xs[7][8];
#pragma unroll
    for (int u = 0; u < 7; ++u)
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        xs[u][2 * w] = bf16_lo(xraw[u][w]);
        xs[u][2 * w + 1] = bf16_hi(xraw[u][w]);
      }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float acc[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[j] = 0.0f;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const bool on = (valid >> (4 * i + t)) & 1u;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const float w = taps[buf][8 * chunk + j][t];
          acc[j] = fmaf(on ? w : 0.0f, xs[i + t][j], acc[j]);
        }
      }
      u32x4_t o;
#pragma unroll
      for (int w = 0; w < 4; ++w) o[w] = pack_bf16x2(acc[2 * w], acc[2 * w + 1]);
      *reinterpret_cast<u32x4_t*>(&lds[buf][0][tile_off(xr0 + i, chunk)]) = o;
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
  issue(0);
  commit(0);
  __syncthreads();
  commit_x(0);
  __syncthreads();
  const int half = lane >> 5, l32 = lane & 31;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) issue(kt + 1);
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
    if (kt + 1 < nk) {
      commit(buf ^ 1);
      __syncthreads();  // taps of the next step published
      commit_x(buf ^ 1);
    }
    __syncthreads();
  }

  // Epilogue: element (m, n) of P to its projection, head and channel.
  const int Hd = P.heads * P.d;
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int n = n0 + 64 * wn + 32 * j + l32;
    if (n >= N) continue;
    const int blk = n / Hd;  // 0..3: Q, K, V, R; 4: gate logits
    uint16_t* dst = blk == 0 ? q : blk == 1 ? k : blk == 2 ? v : blk == 3 ? r : a;
    const int h = blk < 4 ? (n % Hd) / P.d : n - 4 * Hd;
    const int e = blk < 4 ? n % P.d : 0;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int m = m0 + 64 * wm + 32 * i + 8 * (rr >> 2) + 4 * half + (rr & 3);
        if (m >= M) continue;
        // token m -> (sequence slice row): dense [B, H, n, .], ragged [H, T, .]
        int64_t row;
        if (P.ragged) {
          row = (int64_t)h * M + m;
        } else {
          const int b = m / P.rows, i2 = m - b * P.rows;
          row = ((int64_t)b * P.heads + h) * P.rows + i2;
        }
        const uint32_t bits = pack_bf16x2(acc[i][j][rr], 0.0f) & 0xffffu;
        if (blk < 4) dst[row * P.d + e] = (uint16_t)bits;
        else dst[row] = (uint16_t)bits;
      }
  }
}

}  // namespace

gbla_status launch_project(const LayerPlan& p, const void* x, const float* conv_x,
                           const void* w_proj, const int32_t* cu, void* q, void* k, void* v,
                           void* r, void* a, hipStream_t st) {
  if (p.tokens == 0) return GBLA_OK;
  const dim3 grid((p.features + kBN - 1) / kBN, (p.tokens + kBM - 1) / kBM);
  hipLaunchKernelGGL(proj_kernel, grid, dim3(kThreads), 0, st, p, (const uint16_t*)x, conv_x,
                     (const uint16_t*)w_proj, cu, (uint16_t*)q, (uint16_t*)k, (uint16_t*)v,
                     (uint16_t*)r, (uint16_t*)a);
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}

}  // namespace gbla
