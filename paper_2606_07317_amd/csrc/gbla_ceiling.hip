// gbla_ceiling.hip -- a measurement aid, not part of the method: one launch
// that moves exactly the forward pass's bytes with none of its arithmetic,
// the practical ceiling that the forward's time is compared with.
//
// Per token and head it reads q, k, v and r (d elements each, 16-byte
// loads) and the one gate logit, and writes d fp32 values (16-byte stores):
// the (4d + 1) e + 4d bytes the forward must move at least once.  The
// written values combine the loaded bits, so no load can be dropped.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "gbla.h"
#include "gbla_device.h"

namespace gbla {
namespace {

constexpr int kCeilBlocks = 4096;  // grid of the grid-stride loop (measured best of 1024..8192)

// bf16 inputs: 16 bytes = 8 elements of one token; a token has 2^shift of
// them (d / 8).
__global__ void __launch_bounds__(kThreads)
stream_ceiling_kernel(const u32x4_t* __restrict__ q, const u32x4_t* __restrict__ k,
                      const u32x4_t* __restrict__ v, const u32x4_t* __restrict__ r,
                      const uint16_t* __restrict__ a, u32x4_t* __restrict__ y, int64_t units,
                      int shift) {
  const int64_t mask = (int64_t(1) << shift) - 1;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < units; i += stride) {
    u32x4_t x = q[i] ^ k[i] ^ v[i] ^ r[i];
    if ((i & mask) == 0) x[0] += a[i >> shift];  // the token's logit, once
    y[2 * i] = x;
    y[2 * i + 1] = x;
  }
}

}  // namespace
}  // namespace gbla

extern "C" gbla_status gbla_stream_ceiling(const void* q, const void* k, const void* v,
                                           const void* gate_logits, const void* out_gate,
                                           int64_t token_heads, int32_t head_dim, float* out,
                                           void* stream) {
  if (!q || !k || !v || !gate_logits || !out_gate || !out || token_heads < 0)
    return GBLA_ERR_INVALID_ARGUMENT;
  if (head_dim != 32 && head_dim != 64 && head_dim != 128) return GBLA_ERR_UNSUPPORTED;
  for (const void* p : {q, k, v, out_gate, static_cast<const void*>(out)})
    if (reinterpret_cast<uintptr_t>(p) % 16 != 0) return GBLA_ERR_MISALIGNED;
  if (reinterpret_cast<uintptr_t>(gate_logits) % 2 != 0) return GBLA_ERR_MISALIGNED;
  const int shift = head_dim == 32 ? 2 : head_dim == 64 ? 3 : 4;  // log2(d / 8)
  const int64_t units = token_heads << shift;
  if (units == 0) return GBLA_OK;
  const int64_t want = (units + gbla::kThreads - 1) / gbla::kThreads;
  const unsigned blocks = (unsigned)(want < gbla::kCeilBlocks ? want : gbla::kCeilBlocks);
  hipLaunchKernelGGL(gbla::stream_ceiling_kernel, dim3(blocks), dim3(gbla::kThreads), 0,
                     static_cast<hipStream_t>(stream), static_cast<const gbla::u32x4_t*>(q),
                     static_cast<const gbla::u32x4_t*>(k), static_cast<const gbla::u32x4_t*>(v),
                     static_cast<const gbla::u32x4_t*>(out_gate),
                     static_cast<const uint16_t*>(gate_logits), reinterpret_cast<gbla::u32x4_t*>(out),
                     units, shift);
  return hipGetLastError() == hipSuccess ? GBLA_OK : GBLA_ERR_HIP;
}
