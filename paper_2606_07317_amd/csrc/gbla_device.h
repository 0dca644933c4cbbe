// gbla_device.h -- device helpers shared by the kernel sources of libgbla.so.
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "gbla_plan.h"

namespace gbla {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

// bf16 <-> fp32 (bf16 held as raw 16-bit patterns).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Two fp32 -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2_t f = {lo, hi};
  bf16x2_t b = __builtin_convertvector(f, bf16x2_t);
  return __builtin_bit_cast(uint32_t, b);
}

__device__ __forceinline__ u32x4_t load16(const void* p) {
  return *reinterpret_cast<const u32x4_t*>(p);
}

// Raw buffer resource over `bytes` bytes from `base` (gfx9 dword-3 format
// bits).  Loads past the range read 0 and stores past it are dropped, which
// is how the streaming kernels mask sequence edges without branches.  Byte
// offsets are 32-bit: callers keep every slice under 2^31 bytes, so a
// negative offset (a row before the sequence start) is out of range too.
// The caller passes wave-uniform values; they are moved to scalar registers
// here so the descriptor never lives in vector registers.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
  const int n = __builtin_amdgcn_readfirstlane((int)bytes);
  void* p = reinterpret_cast<void*>(((uint64_t)hi << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(p, 0, n, 0x00020000);
}
constexpr uint32_t kOutOfRange = 0x80000000u;

// Taps of one tensor (0 = q, 1 = k, 2 = v), head h, channel c, right-aligned
// to four taps: tap 3 multiplies the current token, taps before 4 - W are 0.
// conv_w == NULL is the identity conv (the no-Conv1D switch).  The loads go
// through a buffer range over the taps (empty when conv_w is NULL), so there
// is no branch around them: a branch would make the compiler wait for each
// group of taps before issuing the loads that follow.
__device__ __forceinline__ void load_taps4(const float* conv_w, int H, int h, int tensor, int D,
                                           int W, int c, float* w4) {
  const __amdgpu_buffer_rsrc_t r =
      make_rsrc(conv_w, conv_w ? (uint32_t)(3 * H * D * W) * 4u : 0u);
  const uint32_t row = (uint32_t)(((tensor * H + h) * D + c) * W) * 4u;
  if (W == 4) {  // one 16-byte load (W is wave-uniform)
    const u32x4_t x = __builtin_amdgcn_raw_buffer_load_b128(r, row, 0, 0);
#pragma unroll
    for (int t = 0; t < 4; ++t) w4[t] = __uint_as_float(x[t]);
  } else {
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int ti = t - (4 - W);
      w4[t] = __uint_as_float(
          __builtin_amdgcn_raw_buffer_load_b32(r, ti >= 0 ? row + 4u * ti : kOutOfRange, 0, 0));
    }
  }
  w4[3] = conv_w ? w4[3] : 1.0f;
}

// sum += x with Kahan's compensation: c carries the low-order bits that the
// rounded sum lost, so a sum of n terms keeps an error of a few ulps instead
// of growing with n.  Used for the fixed-order sums over chunks, which run to
// thousands of terms on long sequences.
__device__ __forceinline__ void kahan_add(float& sum, float& c, float x) {
  const float y = x - c;
  const float t = sum + y;
  c = (t - sum) - y;
  sum = t;
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

__device__ __forceinline__ int wave_incl_scan(int x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  return x;
}

// Block-wide reductions for blocks of NT threads (NT / 64 waves); `red`
// holds NT / 64 entries.
template <int NT = kThreads>
__device__ __forceinline__ float block_max(float x, float* red) {
  x = wave_max(x);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
  float m = red[0];
#pragma unroll
  for (int i = 1; i < NT / 64; ++i) m = fmaxf(m, red[i]);
  return m;
}

// Inclusive scan over the block; *total receives the block sum.
template <int NT = kThreads>
__device__ __forceinline__ int block_incl_scan(int x, int* red, int* total) {
  x = wave_incl_scan(x);
  __syncthreads();
  if ((threadIdx.x & 63) == 63) red[threadIdx.x >> 6] = x;
  __syncthreads();
  const int w = threadIdx.x >> 6;
  int before = 0, all = 0;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) {
    before += i < w ? red[i] : 0;
    all += red[i];
  }
  *total = all;
  return x + before;
}

__device__ __forceinline__ int units_of(int64_t len, int unit) {
  const int64_t c = (len + unit - 1) / unit;
  return c < 1 ? 1 : (int)c;
}

// Ragged batches: find the sequence s and the unit index inside it of the
// g-th unit of a head, where sequence s owns max(1, ceil(len_s / unit))
// consecutive units.  Every thread of the block must call it; returns false
// (for the whole block) when g is past the last unit.
template <int NT = kThreads>
__device__ __forceinline__ bool locate_unit(const int32_t* cu, int nseq, int unit, int g,
                                            int* s_out, int* idx_out) {
  __shared__ int red[NT / 64];
  __shared__ int found[2];
  if (threadIdx.x == 0) found[0] = -1;
  int running = 0;
  for (int base = 0; base < nseq; base += NT) {
    const int s = base + threadIdx.x;
    int cnt = 0;
    if (s < nseq) cnt = units_of((int64_t)cu[s + 1] - cu[s], unit);
    int total;
    const int incl = block_incl_scan<NT>(cnt, red, &total);
    const int excl = incl - cnt;
    if (s < nseq && g >= running + excl && g < running + incl) {
      found[0] = s;
      found[1] = g - running - excl;
    }
    __syncthreads();
    if (found[0] >= 0) break;
    running += total;
  }
  const int s = found[0];
  *s_out = s;
  *idx_out = found[1];
  return s >= 0;
}

// Number of units of the sequences before s, summed over the block.
__device__ __forceinline__ int units_before(const int32_t* cu, int s, int unit) {
  __shared__ int red[4];
  int acc = 0;
  for (int i = threadIdx.x; i < s; i += kThreads) acc += units_of((int64_t)cu[i + 1] - cu[i], unit);
  int total;
  (void)block_incl_scan(acc, red, &total);
  return total;
}

// Length of sequence s and the row (token index in the [*, rows, d] slice
// layout) of its token 0 for head h.
__device__ __forceinline__ void seq_geometry(const Plan& P, const int32_t* cu, int s, int h,
                                             int64_t* len, int64_t* base_row) {
  if (P.ragged) {
    const int64_t c0 = cu[s];
    *len = (int64_t)cu[s + 1] - c0;
    *base_row = (int64_t)h * P.rows + c0;
  } else {
    *len = P.rows;
    *base_row = ((int64_t)s * P.heads + h) * P.rows;
  }
}

// Find (sequence, unit index) of unit g of a head, dense or ragged.
template <int NT = kThreads>
__device__ __forceinline__ bool unit_of(const Plan& P, const int32_t* cu, int unit, int per_seq,
                                        int g, int* s, int* idx) {
  if (P.ragged) return locate_unit<NT>(cu, P.nseq, unit, g, s, idx);
  *s = g / per_seq;
  *idx = g - *s * per_seq;
  return true;
}

}  // namespace gbla
