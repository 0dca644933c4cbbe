// gbla_layer.hip -- the projections of the full GBLA layer (Section 2.1):
//     Xt = Conv1D(X),  [Q | K | V | R | a] = Xt Wp^T
//
// conv_x_kernel  streams X once: causal depthwise conv in fp32, Xt rounded
//                to bf16 into the workspace (a bf16 layer stores it so).
// proj_kernel    P = Xt Wp^T on v_mfma_f32_32x32x16_bf16 (fp32 accumulation):
//                a workgroup of 4 waves (2 x 2, 128 x 128 each, one per
//                SIMD, accumulators in AGPRs) computes a 256-token x
//                256-feature tile, 64 model channels per K step, the
//                operand rows loaded straight into a two-step LDS ring one
//                step ahead.  The output is rounded to bf16 and
//                scattered to the head-major layout the attention kernels
//                read ([B, H, n, d] / [B, H, n]), written under the next
//                tile's products where the shape allows.
// The conv is a separate pass rather than part of the tile staging: redone
// for every feature tile, its vector work would compete with the products
// (measured: 0.36 against 0.54 PFLOP/s for the GEMM), while the pass itself
// costs one read and one write of X.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "gbla_device.h"
#include "gbla_ext.h"
#include "gbla_plan.h"

namespace gbla {
namespace {

constexpr int kBM = 256, kBN = 256, kBK = 64;
constexpr int kProjWaves = 4, kProjThreads = 64 * kProjWaves;  // 2 x 2 waves
constexpr int kProjGrid = 256;                                  // persistent workgroups
constexpr int kWaveM = kBM / 2, kWaveN = kBN / 2;               // 128 x 128 per wave
constexpr int kRowBytes = kBK * 2;           // one tile row of bf16: eight 16-byte chunks
constexpr int kTileBytes = 256 * kRowBytes;  // 32 KB
constexpr int kStages = 2;                   // K steps held in LDS at once
constexpr int kStageBytes = 2 * kTileBytes;  // both tiles of one K step
// the ring, then a spare 32 KB: one 32-token block of every wave's staged
// output (the deferred stores' first eight)
constexpr int kSpareBytes = 32768;
constexpr int kLdsBytes = kStages * kStageBytes + kSpareBytes;
// per wave and K step: 16-byte loads into LDS, 1 KB (64 lanes) each
constexpr int kDmaPerTile = kTileBytes / (kProjThreads * 16);

// Byte offset of 16-byte chunk `c` of row `r` in a tile (128-byte rows, eight
// chunks).  A 16-byte operand read serves 16 lanes (16 consecutive rows) from
// 64 banks (256 bytes: the even rows' chunks in one half, the odd rows' in
// the other), so the eight even (odd) rows of 16 need eight different chunk
// positions: the chunks are XOR-swizzled by (r / 2) % 8.  (Swizzled by r % 8,
// rows r and r + 8 collided, and 49% of the LDS cycles were conflicts.)
__device__ __forceinline__ int tile_off(int r, int c) { return r * kRowBytes + ((c ^ ((r >> 1) & 7)) << 4); }

// A buffer resource over `bytes` bytes from `base`, as four scalar registers
// for the assembly loads below (the same descriptor as make_rsrc).
__device__ __forceinline__ u32x4_t rsrc_sgprs(const void* base, uint32_t bytes) {
  const uint64_t ad = reinterpret_cast<uint64_t>(base);
  return u32x4_t{(uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)ad),
                 (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(ad >> 32)),
                 (uint32_t)__builtin_amdgcn_readfirstlane((int)bytes), 0x00020000u};
}

// 16 bytes per lane from the buffer into LDS at base + 16 * lane (M0 = base;
// one wait state after writing M0).  Assembly, so that the compiler neither
// tracks these loads (the step loop waits for them explicitly, by count) nor
// moves LDS accesses across them.
// M is the LDS byte address (wave-uniform).
__device__ __forceinline__ void dma16(const u32x4_t& r, uint32_t m, uint32_t off) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(off), "s"(r), "s"(m)
               : "memory", "m0");
}

// The lane index, computed where it is used: a volatile statement cannot be
// hoisted, so addresses formed from it are not held (and spilled) across
// the tile loop, where each reload's wait would drain the loads in flight.
__device__ __forceinline__ int lane_now() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}

// s_waitcnt lgkmcnt(0), the other counters left alone (gfx9 encoding).
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// s_waitcnt vmcnt(N), the other counters left alone (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}

// Workgroup barrier with no fence: a fence would make each wave wait for all
// of its loads in flight, the later K steps' too.  Each wave has waited for
// its own loads of the step it reads next, and every LDS read of a stage is
// consumed (so complete) before the barrier after which that stage is
// refilled.  The clobber keeps the compiler from moving LDS accesses across.
__device__ __forceinline__ void step_sync() { asm volatile("s_barrier" ::: "memory"); }

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
  // taps: one 16-byte load per channel at W = 4, else one load per tap (an
  // out-of-range offset, read as zero, for the taps before the first)
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(conv_x, (uint32_t)(K * P.W * 4));
  float w[8][4];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t row = (uint32_t)((c0 + j) * P.W) * 4u;
    if (P.W == 4) {
      const u32x4_t t4 = __builtin_amdgcn_raw_buffer_load_b128(rw, row, 0, 0);
#pragma unroll
      for (int t = 0; t < 4; ++t) w[j][t] = __uint_as_float(t4[t]);
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int ti = t - (4 - P.W);
        w[j][t] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rw, ti >= 0 ? row + 4u * ti : kOutOfRange, 0, 0));
      }
    }
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
// workgroups (tiles blockIdx.x, blockIdx.x + gridDim.x, ...).  Four waves
// (2 x 2) of 128 x 128, one per SIMD: a wave's accumulators fill its 256
// AGPRs, and a 128 x 128 wave tile reads 0.5 KB of LDS operands per
// 32x32x16 product.
//
// The K steps (64 channels) of all the workgroup's tiles form one stream,
// numbered g: step g sits in LDS stage g % 2, loaded by buffer loads that
// write LDS directly (no staging registers, no LDS stores) one step ahead.
// At the top of step g every wave waits for its own loads of step g and the
// workgroup meets at a barrier; the loads of step g + 1 then refill the
// stage of step g - 1, issued between the step's first products.  Eight
// lanes load a row's 128 bytes, whole lines: with 32-channel steps (64
// bytes a row, a four-stage ring three steps ahead) every line took two L2
// requests, and the kernel ran 3% slower.  Within a step, each of the four
// 16-channel slices is read while the previous slice's products run.
//
// Output: the products are formed as P^T (Wp rows as the first operand),
// so lane l of a 32 x 32 block holds token l % 32 and, in elements
// 4 g .. 4 g + 3, the four consecutive features 8 g + 4 (l / 32) .. + 3.
// Stores must cover whole lines: 16 bytes per lane at different tokens'
// rows cost an L2 request each, which made the output as slow as the
// products.  So with DEFER (d_model a multiple of 1024, i.e. at least 16 K
// steps per tile; a tile's features in one of q, k, v, r; its tokens' rows
// linear) each wave stages its block through LDS at the tile's end and
// reads it back as 16-byte pieces, eight lanes to a 128-byte row, which go
// out two per K step of the next tile, under its products (to an
// out-of-range offset when none is pending), ahead of the step's loads.
// Without DEFER the tile is written from the accumulators at once (eight
// bytes per lane).
//
// The dispatcher places workgroup b on XCD b % 8; with a grid that is a
// multiple of 8, tile L therefore runs on XCD L % 8.  When the token tiles
// come in multiples of 64, each XCD takes every eighth token tile in groups
// of eight, walking all feature tiles of a group before the next, so that
// the workgroups an XCD holds at once share a few token and feature tiles
// in its L2, where the plain order made every XCD stream all of Wp.
// ---------------------------------------------------------------------------
template <int... U, class F>
__device__ __forceinline__ void unrolled(std::integer_sequence<int, U...>, F&& f) {
  (f(std::integral_constant<int, U>{}), ...);
}

template <bool DEFER>
__global__ void __launch_bounds__(kProjThreads, 1)
proj_kernel(LayerPlan P, const uint16_t* __restrict__ xt, const uint16_t* __restrict__ wp,
            uint16_t* __restrict__ q, uint16_t* __restrict__ k, uint16_t* __restrict__ v,
            uint16_t* __restrict__ r) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[kLdsBytes];
  constexpr int TM = kWaveM / 32, TN = kWaveN / 32;  // 32 x 32 products per wave and K slice
  constexpr int kStoresPerStep = 2;  // deferred 16-byte stores per lane and K step
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;
  const int tiles_n = (4 * P.heads * P.d + kBN - 1) / kBN, tiles_m = (P.tokens + kBM - 1) / kBM;
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
  const int Hd = P.heads * P.d;
  const int K = P.d_model, M = P.tokens, N = 4 * Hd;  // Q, K, V, R features (the gates: gate_kernel)
  const int nk = K / kBK;
  const int64_t hstride = P.ragged ? (int64_t)M : (int64_t)P.rows;  // rows between heads
  const int half = lane >> 5, l32 = lane & 31;

  // ---- the load stream ----
  // Load j of a wave covers tile rows 8 (kDmaPerTile wave + j) .. + 7: lane
  // l writes row (l / 8), stored chunk l % 8, which holds source chunk
  // (l % 8) ^ (row / 2 % 8) (the swizzle of tile_off), i.e. (l % 8) ^
  // ((l / 16 + 4 (j % 2)) % 8): two lane offsets, by the parity of j.  The offsets within the
  // tile are the same for Xt and Wp; the tile's first row and the K step go
  // into the descriptor, whose extent ends at the last token (feature), so
  // rows past it read zeros.
  // the lane's part of the offsets (row lane / 8, its source chunk); each
  // load adds its first row through an opaque row pitch, so that the eight
  // sums are formed at the loads rather than held in registers
  const uint32_t lbase0 = (uint32_t)(((lane >> 3) * K + 8 * ((lane & 7) ^ ((lane >> 4) & 7))) * 2);
  const uint32_t lbase1 = (uint32_t)(((lane >> 3) * K + 8 * ((lane & 7) ^ (((lane >> 4) + 4) & 7))) * 2);
  int dL = blockIdx.x, ds = 0, dm0 = 0, dn0 = 0;  // the next step to load
  if (dL < tiles) tile_of(dL, dm0, dn0);
  // the LDS byte address of the ring (wave-uniform)
  const uint32_t lds_addr = (uint32_t)__builtin_amdgcn_readfirstlane(
      (int)(uint32_t)(uintptr_t)(__attribute__((address_space(3))) void*)lds);
  u32x4_t lrx, lrw;
  uint32_t lst;
  auto load_prep = [&](int stage) {
    const bool live = dL < tiles;
    const int k0 = ds * kBK;
    const uint32_t xb = live && dm0 < M ? (uint32_t)(((int64_t)(M - dm0) * K - k0) * 2) : 0u;
    const uint32_t wb = live ? (uint32_t)(((int64_t)(N - dn0) * K - k0) * 2) : 0u;
    lrx = rsrc_sgprs(xt + ((int64_t)dm0 * K + k0), xb);
    lrw = rsrc_sgprs(wp + ((int64_t)dn0 * K + k0), wb);
    lst = lds_addr + stage * kStageBytes + wave * (kDmaPerTile * 1024);
  };
  auto load_part = [&](int j) {
    int pitch = 2 * K;
    asm volatile("" : "+s"(pitch));
    const uint32_t off = ((j & 1) ? lbase1 : lbase0) + (uint32_t)(8 * (kDmaPerTile * wave + j) * pitch);
    dma16(lrx, lst + 1024 * j, off);
    dma16(lrw, lst + kTileBytes + 1024 * j, off);
  };
  auto load_advance = [&]() {
    if (++ds == nk) {
      ds = 0;
      dL += gridDim.x;
      if (dL < tiles) tile_of(dL, dm0, dn0);
    }
  };

  // ---- operand reads and products ----
  // The operand of lane l in K slice ks: row l % 32 of a 32-row block, chunk
  // 2 ks + l / 32.  Blocks start at multiples of 32 rows, so the swizzle
  // depends on the lane only: one offset per slice, the block and stage
  // added.
  int roff[4];
#pragma unroll
  for (int ks = 0; ks < 4; ++ks) roff[ks] = tile_off(l32, 2 * ks + half);
  u32x4_t fa[2][TM], fb[2][TN];  // [slice % 2][block]
  // (the stage's offset passes through an empty asm statement, so that the
  // addresses are formed at each read rather than held for every stage and
  // slice, eight registers the epilogue pushed into scratch)
  auto read_slice = [&](int stage, int ks) {
    int so = stage * kStageBytes;
    asm volatile("" : "+s"(so));
    const unsigned char* A = lds + so + kWaveM * wm * kRowBytes + roff[ks];
    const unsigned char* B = lds + so + kTileBytes + kWaveN * wn * kRowBytes + roff[ks];
#pragma unroll
    for (int i = 0; i < TM; ++i) fa[ks & 1][i] = *reinterpret_cast<const u32x4_t*>(A + 32 * i * kRowBytes);
#pragma unroll
    for (int j = 0; j < TN; ++j) fb[ks & 1][j] = *reinterpret_cast<const u32x4_t*>(B + 32 * j * kRowBytes);
  };
  f32x16_t acc[TM][TN];
  // FRESH: the tile's first product of this block, accumulating onto zero
  // (no separate clearing of the 256 accumulator registers)
  auto mfma = [&](int ks, int i, int j, bool fresh) {
    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, fb[ks & 1][j]),
                                                        __builtin_bit_cast(bf16x8_t, fa[ks & 1][i]),
                                                        fresh ? f32x16_t{} : acc[i][j], 0, 0, 0);
  };

  // ---- output ----
  // Token row of (head 0, this lane's token m): [B, H, L, .] or [H, T, .].
  // (The divisor goes through an empty asm statement so that its reciprocal
  // is formed at each use rather than once before the tile loop, where it
  // was spilled; a reload's wait would drain the loads in flight.)
  auto token_row = [&](int m) -> int64_t {
    if (P.ragged) return m;
    int rows = P.rows;
    asm volatile("" : "+s"(rows));
    const int b = m / rows;
    return (int64_t)b * P.heads * rows + (m - b * rows);
  };
  // The whole tile at once (every tile without DEFER), eight bytes per lane.
  auto write_now = [&](int m0, int n0) {
    int64_t tokrow[TM];
    bool tok_ok[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = m0 + kWaveM * wm + 32 * i + l32;
      tok_ok[i] = m < M;
      tokrow[i] = token_row(m);
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int nf = n0 + kWaveN * wn + 32 * j + 8 * gq;  // first feature of the group (uniform)
        if (nf >= N) continue;
        const int blk = nf / Hd, h = (nf % Hd) / P.d, e = nf % P.d;
        uint16_t* const dst = blk == 0 ? q : blk == 1 ? k : blk == 2 ? v : r;
        // the group's part of the address, the same for every lane
        unsigned char* const gbase = reinterpret_cast<unsigned char*>(dst) + ((int64_t)h * hstride * P.d + e) * 2;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          if (!tok_ok[i]) continue;
          const u32x2_t o{pack_bf16x2(acc[i][j][4 * gq], acc[i][j][4 * gq + 1]),
                          pack_bf16x2(acc[i][j][4 * gq + 2], acc[i][j][4 * gq + 3])};
          *reinterpret_cast<u32x2_t*>(gbase + (tokrow[i] * P.d + 4 * half) * 2) = o;
        }
      }
    }
  };
  // Deferred output.  At a tile's end each wave stages its 128 x 128 bf16
  // block, 32 tokens at a time, in LDS as rows of 256 bytes (16-byte chunks
  // XOR-swizzled by the row) and reads it back as 16-byte pieces: piece
  // (i, pass) holds token 32 i + 4 pass + l / 16 and features 8 (l % 16) ..
  // + 7, so eight lanes write one token's 128-byte row of a head (d = 64),
  // whole lines.  Token block 0 stays in the spare LDS region and is read
  // piece by piece as its stores go out (the next tile's first four steps);
  // blocks 1..3 go through the stage of the tile's last step into registers.
  // The features lie in one of q, k, v, r (H d is a multiple of 256) and the
  // tile's tokens in one sequence or in the packed rows (token rows linear
  // in the token); the targets' extents, tokens * H * d * 2 bytes, are
  // below 2^31 (the launcher checks all three).
  const uint32_t act_bytes = (uint32_t)((int64_t)M * Hd * 2);
  u32x4_t ob[TM - 1][8];  // token blocks 1..3 (rotating into ob[0])
  uint32_t obase = 0;     // byte offset of (this lane's first token, its features)
  int mfirst = 0;         // this lane's first token
  uint32_t tokstep = 0;   // bytes between consecutive tokens' rows
  __amdgpu_buffer_rsrc_t rcur = make_rsrc(q, 0u);
  bool ob_live = false;
  unsigned char* const spare = lds + kStages * kStageBytes + wave * 8192;
  if constexpr (DEFER) {
#pragma unroll
    for (int i = 0; i + 1 < TM; ++i)
#pragma unroll
      for (int ps = 0; ps < 8; ++ps) ob[i][ps] = u32x4_t{0u, 0u, 0u, 0u};
  }
  // byte offset of piece PS in a wave's staged 32-token block
  auto piece_off = [&](int ps, int el) {
    const int row = 4 * ps + (el >> 4);
    return row * 256 + (((el & 15) ^ (row & 15)) * 16);
  };
  auto defer_tile = [&](int m0, int n0, unsigned char* stage) {
    const int el = lane_now();
    const int e32 = el & 31, ehalf = el >> 5;
    unsigned char* const wst = stage + wave * 8192;  // this wave's 32 x 256-byte rows
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      unsigned char* const buf = i == 0 ? spare : wst;
      // lane (token e32, half) writes features 32 j + 8 gq + 4 half .. + 3
      // (one 32 x 32 block at a time: scheduled freely, the conversions held
      // enough registers to push the loop's addresses into scratch)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
#pragma unroll
        for (int gq = 0; gq < 4; ++gq) {
          const int ch = (4 * j + gq) ^ (e32 & 15);
          *reinterpret_cast<u32x2_t*>(buf + e32 * 256 + ch * 16 + 8 * ehalf) =
              u32x2_t{pack_bf16x2(acc[i][j][4 * gq], acc[i][j][4 * gq + 1]),
                      pack_bf16x2(acc[i][j][4 * gq + 2], acc[i][j][4 * gq + 3])};
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      if (i == 0) continue;
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
      for (int ps = 0; ps < 8; ++ps) ob[i - 1][ps] = *reinterpret_cast<const u32x4_t*>(wst + piece_off(ps, el));
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    // The staging's LDS writes and read-backs complete before the next step's
    // barrier, after which another wave's loads refill this stage (the
    // read-backs' results are used only later, by the stores, so nothing
    // else would wait for them).
    wait_lgkm0();
    int hd = Hd, dd = P.d;
    asm volatile("" : "+s"(hd), "+s"(dd));
    const int nf = n0 + kWaveN * wn, blk = nf / hd;
    const int c = nf % hd + 8 * (el & 15), h = c / dd, e = c % dd;
    uint16_t* const dst = blk == 0 ? q : blk == 1 ? k : blk == 2 ? v : r;
    rcur = make_rsrc(dst, act_bytes);
    mfirst = m0 + kWaveM * wm + (el >> 4);
    obase = (uint32_t)(((token_row(mfirst) + (int64_t)h * hstride) * P.d + e) * 2);
    tokstep = (uint32_t)(P.d * 2);
  };
  // Store piece PS of token block SB, DATA; nothing pending past the fourth
  // block.
  auto store_piece = [&](const u32x4_t& data, int ps, int sb) {
    const int dm = 32 * sb + 4 * ps;
    const bool live = ob_live && sb < TM && mfirst + dm < M;
    __builtin_amdgcn_raw_buffer_store_b128(data, rcur, live ? obase + dm * tokstep : kOutOfRange, 0, 0);
  };
  auto spare_piece = [&](int ps) {  // piece PS of token block 0
    return *reinterpret_cast<const u32x4_t*>(spare + piece_off(ps, lane_now()));
  };

  // ---- one K step ----
  // With DEFER, steps come in blocks of four from a step that is a multiple
  // of 4, so step gg's stage is u % 2.
  // BLK0: the tile's first block of four steps (its stores read block 0 from
  // the spare region).
  auto step = [&](int gg, auto u_c, int sb, auto first_c, auto blk0_c) {
    constexpr int u = decltype(u_c)::value;
    constexpr bool fresh = decltype(first_c)::value && u == 0;  // the tile's first step
    constexpr bool blk0 = decltype(blk0_c)::value;
    const int st = DEFER ? (u & (kStages - 1)) : (gg & (kStages - 1));
    // Own loads of step gg in.  Everything in flight is waited for: loads and
    // stores share the counter and need not complete in order, so a count
    // that leaves the last stores out would not prove the loads complete.
    // The step's stores therefore go out before its loads, under its first
    // products, and have a whole step to finish.
    wait_vm<0>();
    step_sync();  // everyone's; the stage of step gg - 1 is free
    read_slice(st, 0);
    u32x4_t sp[2] = {};
    if constexpr (DEFER && blk0) {
      sp[0] = spare_piece(2 * u);
      sp[1] = spare_piece(2 * u + 1);
    }
    load_prep((st + 1) & (kStages - 1));
    __builtin_amdgcn_sched_barrier(0);
    // slices 0..3, each slice's products under the next slice's reads; the
    // deferred stores after the first row of products, then the step's loads
    // (step gg + 1), two per row of products in slices 0 and 1
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      if (ks < 3) read_slice(st, ks + 1);
#pragma unroll
      for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j) mfma(ks, i, j, fresh && ks == 0);
        if constexpr (DEFER) {
          if (ks == 0 && i == 0) {
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int h2 = 0; h2 < kStoresPerStep; ++h2) {
              if constexpr (blk0)
                store_piece(sp[h2], 2 * u + h2, 0);
              else
                store_piece(ob[0][2 * u + h2], 2 * u + h2, sb);
            }
          }
        }
        if (ks < 2) {
          __builtin_amdgcn_sched_barrier(0);
          load_part(4 * ks + i);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    load_advance();
  };

  // ---- prologue: step 0 in flight ----
  load_prep(0);
#pragma unroll
  for (int j = 0; j < kDmaPerTile; ++j) load_part(j);
  load_advance();

  int g = 0;  // the step being multiplied
  for (int L = blockIdx.x; L < tiles; L += gridDim.x) {
    int m0, n0;
    tile_of(L, m0, n0);
    if constexpr (DEFER) {
      // the first block of four steps, its first step accumulating onto zero
      step(g, std::integral_constant<int, 0>{}, 0, std::true_type{}, std::true_type{});
      unrolled(std::make_integer_sequence<int, 3>{}, [&](auto v_c) {
        step(g + decltype(v_c)::value + 1, std::integral_constant<int, decltype(v_c)::value + 1>{}, 0,
             std::false_type{}, std::true_type{});
      });
      g += 4;
      for (int s = 4, sb = 1; s < nk; s += 4, ++sb) {
        unrolled(std::make_integer_sequence<int, 4>{},
                 [&](auto u_c) { step(g + decltype(u_c)::value, u_c, sb, std::false_type{}, std::false_type{}); });
        g += 4;
#pragma unroll
        for (int i = 0; i + 2 < TM; ++i)  // the next token block's pieces
#pragma unroll
          for (int ps = 0; ps < 8; ++ps) ob[i][ps] = ob[i + 1][ps];
      }
      step_sync();  // every wave done reading the stage of the tile's last step
      defer_tile(m0, n0, lds + ((g - 1) & (kStages - 1)) * kStageBytes);
      ob_live = true;
    } else {
      step(g++, std::integral_constant<int, 0>{}, 0, std::true_type{}, std::false_type{});
      for (int s = 1; s < nk; ++s, ++g)
        step(g, std::integral_constant<int, 0>{}, 0, std::false_type{}, std::false_type{});
      write_now(m0, n0);
    }
  }
  if constexpr (DEFER) {  // the last tile's stores
    if (ob_live) {
      unrolled(std::make_integer_sequence<int, 8>{},
               [&](auto ps_c) { store_piece(spare_piece(decltype(ps_c)::value), decltype(ps_c)::value, 0); });
#pragma unroll
      for (int sb = 1; sb < TM; ++sb)
#pragma unroll
        for (int ps = 0; ps < 8; ++ps) store_piece(ob[sb - 1][ps], ps, sb);
    }
  }
  // drain: every load into LDS (the steps past the last tile read zeros)
  // has landed before the workgroup ends
  wait_vm<0>();
}

// ---------------------------------------------------------------------------
// gate_kernel: the gate logits a = Xt w_g^T (the last H rows of Wp), rounded
// to bf16, in the [B, H, L] / [H, T] layout.  H outputs per token make this a
// pass over Xt rather than a GEMM tile: in the projection kernel they would
// fill a 256-feature tile for 16 features.  A workgroup takes 128 tokens; per
// step of 128 model channels its threads load the 128 x 256-byte slab with
// 16 lanes to a row (whole lines; one lane per row, as the MFMA operand
// layout would have it, cost an L2 request per 16 bytes), store it to LDS
// (16-byte chunks XOR-swizzled by the row), together with the same channels
// of up to 32 gate rows, and each wave multiplies its 32 tokens by the gates
// on v_mfma_f32_32x32x16_bf16, the gate rows as the first operand: lane l
// holds token l % 32, so a gate's 32 consecutive tokens are written
// together.  The next step's slabs are loaded into registers while the
// current ones are multiplied, into one LDS buffer of 40 KB (a second
// buffer, or W read through the cache, measured no faster).
// ---------------------------------------------------------------------------
constexpr int kGateTokens = 128;  // per workgroup (4 waves of 32)

__global__ void __launch_bounds__(kThreads)
gate_kernel(LayerPlan P, const uint16_t* __restrict__ xt, const uint16_t* __restrict__ wp,
            uint16_t* __restrict__ a) {
  __shared__ __attribute__((aligned(16))) unsigned char slab[kGateTokens * 256];
  __shared__ __attribute__((aligned(16))) unsigned char wslab[32 * 256];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;
  const int K = P.d_model, M = P.tokens, H = P.heads;
  const int tb = blockIdx.x * kGateTokens;
  const int64_t grow0 = (int64_t)4 * H * P.d;  // first gate row of Wp
  // rows past the last token (gate) read zeros: their offsets pass the extent
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(xt, (uint32_t)((int64_t)M * K * 2));
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(wp + grow0 * K, (uint32_t)((int64_t)H * K * 2));
  // slab loads: thread t takes chunk t % 16 of rows t / 16 + 16 j
  const int lc = tid & 15, lr = tid >> 4;
  auto load = [&](int k0, int g0, u32x4_t (&x)[10]) {
    const bool in = k0 + 8 * lc < K;
#pragma unroll
    for (int j = 0; j < 8; ++j)
      x[j] = bload(rx, in ? ((uint32_t)(tb + lr + 16 * j) * (uint32_t)K + (uint32_t)(k0 + 8 * lc)) * 2u : kOutOfRange);
#pragma unroll
    for (int j = 0; j < 2; ++j)
      x[8 + j] = bload(rw, in ? ((uint32_t)(g0 + lr + 16 * j) * (uint32_t)K + (uint32_t)(k0 + 8 * lc)) * 2u : kOutOfRange);
  };
  auto put = [&](const u32x4_t (&x)[10]) {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int row = lr + 16 * j;
      *reinterpret_cast<u32x4_t*>(&slab[row * 256 + ((lc ^ (row & 15)) << 4)]) = x[j];
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int row = lr + 16 * j;
      *reinterpret_cast<u32x4_t*>(&wslab[row * 256 + ((lc ^ (row & 15)) << 4)]) = x[8 + j];
    }
  };
  const int m = tb + 32 * wave + l32;  // this lane's token in the products
  const int srow = 32 * wave + l32;
  // d_model is a multiple of 64: the last step may be half empty, its
  // channels past d_model read as zeros (out-of-range offsets)
  const int nk = (K + 127) / 128;
  for (int g0 = 0; g0 < H; g0 += 32) {
    f32x16_t acc = {};
    u32x4_t x[10];
    load(0, g0, x);
    put(x);
    __syncthreads();
    for (int s = 0; s < nk; ++s) {
      if (s + 1 < nk) load(128 * (s + 1), g0, x);
      u32x4_t wa[8], xa[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int ch = 2 * u + half;
        wa[u] = *reinterpret_cast<const u32x4_t*>(&wslab[l32 * 256 + ((ch ^ (l32 & 15)) << 4)]);
        xa[u] = *reinterpret_cast<const u32x4_t*>(&slab[srow * 256 + ((ch ^ (srow & 15)) << 4)]);
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, wa[u]),
                                                      __builtin_bit_cast(bf16x8_t, xa[u]), acc, 0, 0, 0);
      __syncthreads();  // every wave done reading the slabs
      if (s + 1 < nk) {
        put(x);
        __syncthreads();
      }
    }
    if (m < M) {
      int64_t arow = m;  // row of (gate 0, token m) in a
      if (!P.ragged) {
        const int b = m / P.rows;
        arow = (int64_t)b * H * P.rows + (m - b * P.rows);
      }
      const int64_t hstride = P.ragged ? (int64_t)M : (int64_t)P.rows;
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int gi = g0 + 8 * (rr >> 2) + 4 * half + (rr & 3);
        if (gi < H) a[arow + gi * hstride] = (uint16_t)pack_bf16x2(acc[rr], 0.0f);
      }
    }
  }
}

}  // namespace

gbla_status launch_project(const LayerPlan& p, const void* x, const float* conv_x,
                           const void* w_proj, const int32_t* cu, void* xt, void* q, void* k,
                           void* v, void* r, void* a, hipStream_t st) {
  if (p.tokens == 0) return GBLA_OK;
  const int64_t tiles = (int64_t)((4 * p.heads * p.d + kBN - 1) / kBN) * ((p.tokens + kBM - 1) / kBM);
  if (tiles > 2147483647LL) return GBLA_ERR_UNSUPPORTED;  // the grid's x extent; nothing enqueued
  hipLaunchKernelGGL(conv_x_kernel, dim3((p.d_model + 127) / 128, (p.tokens + 16 * kConvRun - 1) / (16 * kConvRun)),
                     dim3(kThreads), 0, st, p, (const uint16_t*)x, conv_x, cu, (uint16_t*)xt);
  // one workgroup per CU (256 on MI355X), each owning every 256th tile; a
  // multiple of 8 keeps tile L on XCD L % 8
  const dim3 grid((unsigned)(tiles < kProjGrid ? tiles : kProjGrid));
  // deferred stores: at least 32 K steps per tile, a tile's features in one
  // target, its tokens' rows linear, and 32-bit offsets into q, k, v, r
  const bool defer = p.d_model % 1024 == 0 && (p.heads * p.d) % 256 == 0 &&
                     (p.ragged || p.rows % kBM == 0) &&
                     (int64_t)p.tokens * p.heads * p.d * 2 < (int64_t(1) << 31);
  hipLaunchKernelGGL(defer ? proj_kernel<true> : proj_kernel<false>, grid, dim3(kProjThreads), 0, st, p,
                     (const uint16_t*)xt, (const uint16_t*)w_proj, (uint16_t*)q, (uint16_t*)k,
                     (uint16_t*)v, (uint16_t*)r);
  hipLaunchKernelGGL(gate_kernel, dim3((unsigned)((p.tokens + kGateTokens - 1) / kGateTokens)), dim3(kThreads), 0,
                     st, p, (const uint16_t*)xt, (const uint16_t*)w_proj, (uint16_t*)a);
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}

}  // namespace gbla
