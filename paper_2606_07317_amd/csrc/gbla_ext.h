// gbla_ext.h -- host-side plans and launchers of the backward pass and of the
// full layer.  Internal to libgbla.so; not part of the public boundary.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "gbla.h"
#include "gbla_plan.h"

namespace gbla {

// Workspace of the backward pass (bytes from the workspace base), all fp32.
struct BwdLayout {
  size_t off_S;     // [N, H, d, d] normalised state
  size_t off_z;     // [N, H, d]
  size_t off_mz;    // [N, H, 2] softmax max and sum of the gate logits
  size_t off_dsp;   // [H, units, rec_floats] per-unit state partials, then
                    // per-unit dS, dz partials
  size_t off_dS;    // [N, H, d*d + d] dS, dz
  size_t off_dgp;   // [H, units, d] per-unit dgamma partials
  size_t off_dxt;   // [3, tokens * H * d] gradients of the convolved q, k, v
  size_t off_dcp;   // [H, units, 3, d, 4] per-unit tap-gradient partials
  size_t total_bytes;
};
// The backward's plan: the forward's with its own unit size (the state
// partials, dS partials and tap partials are per unit of this plan).
gbla_status backward_plan(const Plan& p, Plan* out);
BwdLayout make_bwd_layout(const Plan& p);

// Backward launcher (gbla_backward.hip); dconv may be NULL (no Conv1D).
gbla_status launch_backward(const Plan& p, const BwdLayout& L, const void* q, const void* k,
                            const void* v, const void* a, const void* r, const float* conv_w,
                            const float* gamma, const int32_t* cu, const float* dy, void* ws,
                            float* dq, float* dk, float* dv, float* da, float* dr, float* dconv,
                            float* dgamma, hipStream_t st);

// The full layer from X (gbla_layer.hip): the conv on X and the stacked
// projections, then the attention core with its own conv switched off.
struct LayerPlan {
  int32_t nseq;       // B or N_s
  int32_t rows;       // L (dense) or T (ragged)
  int32_t d_model;
  int32_t heads;
  int32_t d;
  int32_t W;
  int32_t ragged;
  int32_t tokens;     // B * L or T
  int32_t features;   // 4 * H * d + H, the rows of the stacked projection weights
  Plan core;          // plan of the attention core (flags GBLA_NO_CONV)
  size_t off_xt, off_q, off_k, off_v, off_r, off_a, off_core, total_bytes;
};
gbla_status make_layer_plan(const gbla_layer_shape* s, bool ragged, LayerPlan* p);
// xt: tokens x d_model bf16 scratch for the convolved embeddings.
gbla_status launch_project(const LayerPlan& p, const void* x, const float* conv_x,
                           const void* w_proj, const int32_t* cu, void* xt, void* q, void* k,
                           void* v, void* r, void* a, hipStream_t stream);

}  // namespace gbla
