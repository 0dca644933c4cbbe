// gbla_layer.hip -- the projections of the full GBLA layer (Section 2.1):
//     Xt = Conv1D(X),  [Q | K | V | R | a] = Xt Wp^T
//
// conv_x_kernel  streams X once: causal depthwise conv in fp32, Xt rounded
//                to bf16 into the workspace (a bf16 layer stores it so).
// proj_kernel    P = Xt Wp^T on v_mfma_f32_32x32x16_bf16 (fp32 accumulation):
//                a workgroup of 8 waves (2 x 4, 128 x 64 each) computes a
//                256-token x 256-feature tile, 64 model channels per K step,
//                the next steps' rows loaded into registers while the
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

constexpr int kBM = 256, kBN = 256, kBK = 32;
constexpr int kProjWaves = 8, kProjThreads = 64 * kProjWaves;  // 2 x 4 waves
constexpr int kProjGrid = 256;                                  // persistent workgroups
constexpr int kWaveM = kBM / 2, kWaveN = kBN / 4;               // 128 x 64 per wave
constexpr int kRowBytes = kBK * 2;           // one tile row of bf16: four 16-byte chunks
constexpr int kTileBytes = 256 * kRowBytes;  // 16 KB
// LDS: two K steps of both tiles, or in the epilogue a 64 x 64 half of
// every wave's tile in bf16, rows padded to 72 elements
constexpr int kEpRow = 72;
constexpr int kLdsBytes = 4 * kTileBytes > kProjWaves * 64 * kEpRow * 2 ? 4 * kTileBytes
                                                                         : kProjWaves * 64 * kEpRow * 2;

// Byte offset of 16-byte chunk `c` of row `r` in a tile.  The chunks are
// XOR-swizzled by r / 4: a 16-byte operand read serves 16 lanes (16
// consecutive rows) per cycle from 64 banks (256 bytes), and four rows share
// a 256-byte bank row, so the four rows of a bank row take its four chunks
// and the swizzle gives the four groups of four rows different chunks.  (The
// signed division, rather than a shift, keeps the compiler from holding a
// precomputed address per operand across the loop, which made it spill.)
__device__ __forceinline__ int tile_off(int r, int c) { return r * kRowBytes + ((c ^ ((r / 4) & 3)) << 4); }

__device__ __forceinline__ u32x4_t bload(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}

// fp32 -> bf16 bits, round to nearest even, in integer arithmetic.  In the
// projection epilogue, the hardware pack conversion or any per-element NaN
// select made the register allocator spill the main loop's accumulators.
// No select is needed there: the only NaNs an accumulator can hold are the
// default NaN or NaNs carried from bf16 inputs, whose low 16 bits are zero,
// and for those the rounding sum cannot carry into bit 16, so they keep
// their upper half (a NaN).
__device__ __forceinline__ uint16_t bf16_bits_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
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
// (features / 256) x (tokens / 256) tiles, numbered L, owned by persistent
// workgroups (tiles blockIdx.x, blockIdx.x + gridDim.x, ...); 8 waves
// (2 x 4) of 128 x 64, two per SIMD, so one workgroup per CU (244 VGPRs a
// wave).  A wave tile of 128 x 64 reads 0.75 KB of LDS operands per 32x32x16
// product, against 1 KB for 64 x 64, and the larger workgroup tile halves
// the L2 reads per product.  The dispatcher places workgroup b on XCD b % 8;
// with a grid that is a multiple of 8, tile L therefore runs on XCD L % 8.
// When the token tiles come in multiples of 64, each XCD takes every eighth
// token tile in groups of eight, walking all feature tiles of a group before
// the next, so that the workgroups an XCD holds at once share a few token
// and feature tiles in its L2, where the plain order made every XCD stream
// all of Wp.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(kProjThreads, 1)
proj_kernel(LayerPlan P, const uint16_t* __restrict__ xt, const uint16_t* __restrict__ wp,
            uint16_t* __restrict__ q, uint16_t* __restrict__ k, uint16_t* __restrict__ v,
            uint16_t* __restrict__ r, uint16_t* __restrict__ a) {
  // two K steps of both tiles ([buf][Xt or W]); the epilogue reuses it
  __shared__ __attribute__((aligned(16))) unsigned char lds_raw[kLdsBytes];
  auto tile = [&](int buf, int which) { return lds_raw + (2 * buf + which) * kTileBytes; };
  constexpr int TM = kWaveM / 32, TN = kWaveN / 32;   // 32 x 32 products per wave and K slice
  constexpr int kLoads = kBM * (kBK / 8) / kProjThreads;  // 16-byte pieces per thread and tile
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 2, wn = wave & 3;
  const int tiles_n = (P.features + kBN - 1) / kBN, tiles_m = (P.tokens + kBM - 1) / kBM;
  const int tiles = tiles_n * tiles_m;
  // token and feature tile bases of tile L
  auto tile_of = [&](int L, int& m0_, int& n0_) {
    int tm, tn;
    if (tiles_m % 64 == 0) {
      const int x = L % 8, j = L / 8, per = 8 * tiles_n;
      const int grp = j / per, rr = j % per;
      tn = rr / 8;
      tm = (grp * 8 + rr % 8) * 8 + x;
    } else {
      tn = L % tiles_n;
      tm = L / tiles_n;
    }
    m0_ = tm * kBM;
    n0_ = tn * kBN;
  };
  const int K = P.d_model, M = P.tokens, N = P.features;
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(xt, (uint32_t)((int64_t)M * K * 2));
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(wp, (uint32_t)((int64_t)N * K * 2));

  const int nk = K / kBK;
  // Register staging, two K steps ahead: set s holds the rows of every
  // other step, so a step's rows have two steps of products to arrive.
  u32x4_t xraw[2][kLoads], wraw[2][kLoads];
  // Steps past the last load out of range (zeros, no traffic): the loads are
  // never behind a branch, so the compiler's waits stay exact (a branch made
  // it drain every load before each commit).
  auto issue = [&](int set, int kt, int m0, int n0, bool tile_live) {
    const int k0 = kt * kBK;
    const bool live = tile_live && kt < nk;
    // 32-bit offsets: tokens * d_model * 2 < 2^31 (the plan checks it), so
    // even a row up to 255 past the last token stays below 2^32
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int c = tid + kProjThreads * j, row = c >> 2, ch = c & 3;
      xraw[set][j] = bload(rx, live ? ((uint32_t)(m0 + row) * (uint32_t)K + (uint32_t)(k0 + 8 * ch)) * 2u : kOutOfRange);
    }
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int c = tid + kProjThreads * j, row = c >> 2, ch = c & 3;
      wraw[set][j] = bload(rw, live ? ((uint32_t)(n0 + row) * (uint32_t)K + (uint32_t)(k0 + 8 * ch)) * 2u : kOutOfRange);
    }
  };
  auto commit = [&](int set, int buf) {
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int c = tid + kProjThreads * j, row = c >> 2, ch = c & 3;
      *reinterpret_cast<u32x4_t*>(tile(buf, 0) + tile_off(row, ch)) = xraw[set][j];
    }
#pragma unroll
    for (int j = 0; j < kLoads; ++j) {
      const int c = tid + kProjThreads * j, row = c >> 2, ch = c & 3;
      *reinterpret_cast<u32x4_t*>(tile(buf, 1) + tile_off(row, ch)) = wraw[set][j];
    }
  };

  f32x16_t acc[TM][TN];
  const int half = lane >> 5, l32 = lane & 31;
  auto products = [&](int buf) {
    const unsigned char* A = tile(buf, 0);
    const unsigned char* B = tile(buf, 1);
#pragma unroll
    for (int ks = 0; ks < kBK / 16; ++ks) {
      const int c = 2 * ks + half;
      u32x4_t bf[TN];
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bf[j] = *reinterpret_cast<const u32x4_t*>(B + tile_off(kWaveN * wn + 32 * j + l32, c));
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const u32x4_t af = *reinterpret_cast<const u32x4_t*>(A + tile_off(kWaveM * wm + 32 * i + l32, c));
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, af),
                                                              __builtin_bit_cast(bf16x8_t, bf[j]),
                                                              acc[i][j], 0, 0, 0);
      }
    }
  };
  // A workgroup owns tiles blockIdx.x, blockIdx.x + gridDim.x, ...; the
  // first two K steps of its next tile are loaded while the current tile's
  // epilogue writes (out of range, no traffic, after its last tile).
  int m0, n0;
  tile_of(blockIdx.x, m0, n0);
  issue(0, 0, m0, n0, true);
  issue(1, 1, m0, n0, true);
  for (int64_t L = blockIdx.x; L < tiles; L += gridDim.x) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.0f;
    // Step kt's rows sit in set kt % 2 and LDS buffer kt % 2; the loop runs two
    // steps per turn so that every staging index is a constant.
    commit(0, 0);
    __syncthreads();
    for (int kt = 0; kt < nk; kt += 2) {
      issue(0, kt + 2, m0, n0, true);  // set 0 is free: step kt is in LDS
      products(0);
      commit(1, 1);      // zeros past the last step, never read
      __syncthreads();
      if (kt + 1 >= nk) break;
      issue(1, kt + 3, m0, n0, true);
      products(1);
      commit(0, 0);
      __syncthreads();
    }
    int m1 = 0, n1 = 0;
    const bool has_next = L + gridDim.x < tiles;
    tile_of((int)(has_next ? L + gridDim.x : L), m1, n1);
    issue(0, 0, m1, n1, has_next);
    issue(1, 1, m1, n1, has_next);

    // Epilogue, per 64 x 64 half of the wave's tile: through LDS as bf16 rows
    // (stride 72 elements), then each lane writes 16-byte pieces: eight
    // consecutive features of one token, which are eight consecutive channels
    // of one head (d is a multiple of 8).  Gate-logit features, whose
    // destinations are H rows apart, are written one by one.
    uint16_t* ep = reinterpret_cast<uint16_t*>(lds_raw) + wave * 64 * kEpRow;
    const int Hd = P.heads * P.d;
    const int piece = lane & 7;                     // eight features 8 piece .. 8 piece + 7
    const int nb = n0 + kWaveN * wn + 8 * piece;    // first feature of the piece
    const bool in_proj = nb + 8 <= 4 * Hd;          // else gate logits (or past N)
    const int blk = in_proj ? nb / Hd : 0, h = in_proj ? (nb % Hd) / P.d : 0, e = in_proj ? nb % P.d : 0;
    uint16_t* const dst = blk == 0 ? q : blk == 1 ? k : blk == 2 ? v : r;
    // Destination rows are linear in the token within a tile when its tokens
    // are packed rows or lie in one dense sequence: then one row index per lane
    // (for the tile's first token) and an offset per pass, with no division.
    const bool linear = P.ragged || P.rows % kBM == 0;
    int64_t b0 = 0, pos0 = m0;
    if (!P.ragged) {
      b0 = m0 / P.rows;
      pos0 = m0 - b0 * P.rows;
    }
    auto out_row = [&](int head, int m) -> int64_t {  // row of (head, token m) in [.., n, d] / [H, T, d]
      if (P.ragged) return (int64_t)head * M + m;
      if (linear) return (b0 * P.heads + head) * P.rows + pos0 + (m - m0);
      const int64_t b = m / P.rows;
      return (b * P.heads + head) * P.rows + (m - b * P.rows);
    };
#pragma unroll
    for (int si = 0; si < TM / 2; ++si) {
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
#pragma unroll
          for (int rr = 0; rr < 16; ++rr) {
            const int row = 32 * i + 8 * (rr >> 2) + 4 * half + (rr & 3);
            ep[row * kEpRow + 32 * j + l32] = bf16_bits_rne(acc[2 * si + i][j][rr]);
          }
        }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
      for (int pass = 0; pass < 8; ++pass) {
        const int row = 8 * pass + (lane >> 3);
        const int m = m0 + kWaveM * wm + 64 * si + row;
        if (m >= M || nb >= N) continue;
        const uint16_t* src = ep + row * kEpRow + 8 * piece;
        if (in_proj) {
          *reinterpret_cast<u32x4_t*>(dst + out_row(h, m) * P.d + e) = *reinterpret_cast<const u32x4_t*>(src);
        } else {
#pragma unroll
          for (int f = 0; f < 8; ++f) {
            const int n = nb + f;
            if (n >= N) break;
            // gate logits (every earlier feature is in a 16-byte piece)
            a[out_row(n - 4 * Hd, m)] = src[f];
          }
        }
      }
      // the next half reuses this wave's staging rows
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    m0 = m1;
    n0 = n1;
    __syncthreads();  // every wave is done with the staging area before the next commit
  }
}

}  // namespace

gbla_status launch_project(const LayerPlan& p, const void* x, const float* conv_x,
                           const void* w_proj, const int32_t* cu, void* xt, void* q, void* k,
                           void* v, void* r, void* a, hipStream_t st) {
  if (p.tokens == 0) return GBLA_OK;
  const int64_t tiles = (int64_t)((p.features + kBN - 1) / kBN) * ((p.tokens + kBM - 1) / kBM);
  if (tiles > 2147483647LL) return GBLA_ERR_UNSUPPORTED;  // the grid's x extent; nothing enqueued
  hipLaunchKernelGGL(conv_x_kernel, dim3((p.d_model + 127) / 128, (p.tokens + 16 * kConvRun - 1) / (16 * kConvRun)),
                     dim3(kThreads), 0, st, p, (const uint16_t*)x, conv_x, cu, (uint16_t*)xt);
  // one workgroup per CU (256 on MI355X), each owning every 256th tile; a
  // multiple of 8 keeps tile L on XCD L % 8
  const dim3 grid((unsigned)(tiles < kProjGrid ? tiles : kProjGrid));
  hipLaunchKernelGGL(proj_kernel, grid, dim3(kProjThreads), 0, st, p, (const uint16_t*)xt,
                     (const uint16_t*)w_proj, (uint16_t*)q, (uint16_t*)k, (uint16_t*)v,
                     (uint16_t*)r, (uint16_t*)a);
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}

}  // namespace gbla
