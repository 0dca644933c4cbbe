// gbla_plan.h -- host-side launch plan shared by the C ABI and the kernel
// launchers.  Internal to libgbla.so; not part of the public boundary.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "gbla.h"

namespace gbla {

// Everything a launch needs that depends only on the shape (never on the
// contents of cu_seqlens), so that gbla_workspace_bytes and the entry points
// always agree, and the split structure -- hence the summation order of the
// state reduction -- is a function of the shape alone.
struct Plan {
  int32_t nseq;        // B (dense) or N_s (ragged)
  int32_t heads;       // H
  int32_t rows;        // n (dense) or T (ragged): tokens per head slice
  int32_t d;           // head dim
  int32_t W;           // conv width
  int32_t dtype;       // gbla_dtype
  int32_t ragged;      // 1 when cu_seqlens describes packed sequences
  float eps;
  uint32_t flags;      // GBLA_NO_* switches
  int64_t tokens;      // sum of sequence lengths (B*n or T)

  // State reduction: the tokens of one (sequence, head) are cut into chunks
  // of `chunk` tokens; one workgroup reduces one chunk to a partial state.
  int32_t chunk;
  int32_t chunks_per_seq;  // dense only: ceil(n / chunk), at least 1
  int32_t units;           // state workgroups per head (dense exact, ragged bound)

  // Readout: one workgroup handles `rtile` tokens of one (sequence, head).
  int32_t rtile;
  int32_t rtiles_per_seq;  // dense only
  int32_t runits;          // readout workgroups per head (dense exact, ragged bound)

  // Workspace layout (bytes from the workspace base).
  int32_t rec_floats;      // floats per partial record: S_p, z_p, m_p, l_p, padding
  size_t off_partials;
  size_t off_frags;
  size_t frag_bytes;       // bytes of readout operands per (sequence, head)
  size_t total_bytes;
};

// Fills `p` from the public shape; returns GBLA_OK or the error the shape
// deserves.  `ragged` says whether cu_seqlens will be given.
gbla_status make_plan(const gbla_shape* s, bool ragged, Plan* p);

// Host helpers shared by the plans and the entry points.
size_t align_up(size_t x, size_t a);
bool aligned(const void* p, size_t a);

// Optional kernel-duration events for the readout launch.  When either is
// set, the kernel goes through hipExtLaunchKernel, which records `start` as
// the kernel begins executing and `stop` as it ends, so their elapsed time is
// the kernel's own duration, without the launch gaps around it.
struct KernelEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
  bool any() const { return start != nullptr || stop != nullptr; }
};

// The forward pass behind gbla_forward, gbla_forward_timed and
// gbla_forward_noalloc (gbla_api.cpp): checks, then the kernels.
gbla_status forward_entry(const gbla_shape* shape, const void* q, const void* k, const void* v,
                          const void* gate_logits, const void* out_gate, const float* conv_w,
                          const float* norm_w, const int32_t* cu_seqlens, void* workspace,
                          size_t workspace_bytes, float* out, void* stream, KernelEvents ev);

// Kernel launchers (gbla_kernels.hip).  Arguments were validated by the
// caller; these only enqueue work on `stream`.
gbla_status launch_conv(const Plan& p, const void* q, const void* k, const void* v,
                        const float* conv_w, const int32_t* cu, float* qt, float* kt,
                        float* vt, hipStream_t stream);
// S, z (normalised state) and mz (the softmax's max and sum per (sequence,
// head)) are optional fp32 outputs; NULL skips them.
gbla_status launch_state(const Plan& p, const void* k, const void* v, const void* a,
                         const float* conv_w, const int32_t* cu, void* workspace,
                         float* S, float* z, float* mz, hipStream_t stream);
gbla_status launch_readout(const Plan& p, const void* q, const void* r, const float* conv_w,
                           const float* gamma, const int32_t* cu, const void* workspace,
                           float* out, hipStream_t stream, KernelEvents ev = {});
// The fixed-order combine of partial records [S_p | z_p | m_p | l_p] laid out
// like the forward's (rec_floats apart, [H, units]), with full-accuracy expf
// for every dtype and no readout operands: S, z, mz as in launch_state.
gbla_status launch_combine_f32(const Plan& p, const int32_t* cu, const float* partials,
                               float* S, float* z, float* mz, hipStream_t stream);

// Streaming kernels (gbla_stream.hip): bf16 inputs, head dim 32, 64 or 128.
bool stream_supported(const Plan& p);
gbla_status launch_state_stream(const Plan& p, const void* k, const void* v, const void* a,
                                const float* conv_w, const int32_t* cu, float* partials,
                                hipStream_t stream);
// Head dim 64 (gbla_state64.hip): same partial records as launch_state_stream.
gbla_status launch_state64(const Plan& p, const void* k, const void* v, const void* a,
                           const float* conv_w, const int32_t* cu, float* partials,
                           hipStream_t stream);
// Head dim 128 (gbla_state128.hip): same partial records as launch_state_stream.
gbla_status launch_state128(const Plan& p, const void* k, const void* v, const void* a,
                            const float* conv_w, const int32_t* cu, float* partials,
                            hipStream_t stream);
gbla_status launch_readout_stream(const Plan& p, const void* q, const void* r, const float* conv_w,
                                  const float* gamma, const int32_t* cu, const unsigned char* frags,
                                  float* out, hipStream_t stream, KernelEvents ev = {});

}  // namespace gbla
