/*
 * gbla.h -- C ABI of the MI355X (gfx950) GBLA forward pass.
 *
 * Gated Bidirectional Linear Attention (Section 2.1 of the paper) over the
 * projected tensors of every head:
 *
 *   qt, kt, vt = causal depthwise Conv1D of q, k, v        (item "Conv1D")
 *   g          = softmax over the tokens of the sequence of a   (item "Key gating")
 *   S = sum_j g_j phi(kt_j) vt_j^T,  z = sum_j g_j phi(kt_j)    (its matrix form)
 *   o_i = phi(qt_i)^T S / phi(qt_i)^T z                          (same display)
 *   y_i = RmsNorm(o_i) * gamma * SiLU(r_i)                   (item "RMSNorm with gating")
 *
 * with phi(x) = elu(x) + 1 (Section 2, Bidirectional Linear Attention
 * paragraph).  The Conv1D is applied to the projected q, k, v of each head
 * (depthwise: separate taps per tensor, head and channel; tap W-1 multiplies
 * the current token; no bias); it does not cross sequence starts.  The key
 * gate logits a and the output-gate input r are taken as given.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Every array argument is a DEVICE pointer owned by the caller.  The
 *   library never allocates, frees or synchronizes device memory and keeps
 *   no mutable global state; calls on different streams are independent as
 *   long as each stream uses its own workspace.
 * - Layouts are contiguous, row-major, head_dim fastest:
 *     dense  (cu_seqlens == NULL): activations [B, H, n, d], logits [B, H, n]
 *     ragged (cu_seqlens != NULL): activations [H, T, d],    logits [H, T]
 *   where T = cu_seqlens[N_s] is the packed token count.  In both cases
 *   shape->seqlen is n (dense) or T (ragged) and shape->batch is B or N_s.
 * - Base pointers of activations, outputs, weights and the workspace must be
 *   16-byte aligned (the workspace 256-byte aligned); the logits need only
 *   their element alignment.  Otherwise GBLA_ERR_MISALIGNED.
 * - cu_seqlens (int32, device, N_s + 1 entries) is a precondition, not
 *   checked on the host: cu[0] = 0, non-decreasing, cu[N_s] = T.  Empty
 *   sequences are allowed (they produce no rows and a zero state).
 * - All argument checks run on the host before anything is enqueued; on an
 *   error nothing is launched.  A failed launch returns GBLA_ERR_HIP.
 *   Device faults surface at the caller's next synchronization.  Nothing is
 *   thrown across the ABI.  The calls do not synchronize the stream.
 * - stream is a hipStream_t (NULL = the null stream).
 */
#ifndef GBLA_H
#define GBLA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GBLA_OK = 0,
  GBLA_ERR_INVALID_ARGUMENT = 1, /* null pointer, negative size, bad eps     */
  GBLA_ERR_UNSUPPORTED = 2,      /* head_dim, conv_width or dtype not built   */
  GBLA_ERR_MISALIGNED = 3,       /* a base pointer breaks the alignment rule  */
  GBLA_ERR_WORKSPACE = 4,        /* workspace missing or too small            */
  GBLA_ERR_HIP = 5               /* the HIP runtime reported an error         */
} gbla_status;

typedef enum { GBLA_F32 = 0, GBLA_BF16 = 1 } gbla_dtype;

/*
 * Ablation switches, the rows of the paper's ablation table (Section 3,
 * "Ablation", Table 4; "W/o Key gating", "W/o Conv1D", "W/o Gated RMSNorm", and all
 * three, which is plain bidirectional linear attention, Eq. (1)).  OR them
 * into shape->flags.  An input that a switch removes may be NULL and is
 * ignored if given.
 *   GBLA_NO_GATE  uniform key gates, g_j = 1/n over each sequence (the
 *                 softmax of constant logits); gate_logits is not read.
 *                 The scale cancels in o; gbla_state exports S and z with it.
 *   GBLA_NO_CONV  identity Conv1D: qt = q, kt = k, vt = v; conv_w is not read.
 *   GBLA_NO_NORM  out = o (no RMSNorm, gamma or SiLU gate); out_gate and
 *                 norm_w are not read.
 */
enum {
  GBLA_NO_GATE = 1,
  GBLA_NO_CONV = 2,
  GBLA_NO_NORM = 4,
  GBLA_BLA = 7
};

typedef struct {
  int32_t batch;      /* B (dense) or N_s, the number of sequences (ragged)      */
  int32_t heads;      /* H >= 1                                                  */
  int32_t seqlen;     /* n (dense) or T = cu_seqlens[N_s] (ragged), >= 0          */
  int32_t head_dim;   /* d in {32, 64, 128}                                      */
  int32_t conv_width; /* W in [1, 4]                                             */
  int32_t max_seqlen; /* ragged: an upper bound of the lengths (>= 0); dense: 0  */
  int32_t dtype;      /* gbla_dtype of q, k, v, gate_logits and out_gate         */
  float eps;          /* RMSNorm epsilon, finite and >= 0                        */
  uint32_t flags;     /* OR of GBLA_NO_* switches; 0 is the full GBLA layer      */
} gbla_shape;

/*
 * Bytes of device scratch that gbla_forward / gbla_state need for this
 * shape: the larger of the dense and the ragged reading, taking only a
 * reading the entry points accept.  Pure host arithmetic; returns 0 when the
 * shape is invalid in both readings.  The caller allocates it once (any
 * contents): the entry points initialise what they use on every call.
 */
size_t gbla_workspace_bytes(const gbla_shape* shape);

/*
 * The whole forward pass (Section 2.1: Conv1D, key gating, the global state,
 * the readout and the gated RMSNorm).
 *   q, k, v      [B,H,n,d] or [H,T,d], dtype = shape->dtype; pre-conv projections
 *   gate_logits  [B,H,n]   or [H,T],   dtype = shape->dtype; a = X~ w_g per head
 *   out_gate     [B,H,n,d] or [H,T,d], dtype = shape->dtype; r = X~ W_R per head
 *   conv_w       [3,H,d,W] fp32, taps of q, k, v in that order
 *   norm_w       [H,d] fp32, the RMSNorm weight gamma
 *   cu_seqlens   NULL (dense) or int32 [N_s + 1] (ragged)
 *   workspace    >= gbla_workspace_bytes(shape) bytes of device scratch
 *   out          [B,H,n,d] or [H,T,d] fp32, y (o under GBLA_NO_NORM)
 * gate_logits, conv_w and out_gate / norm_w may be NULL under the switch
 * that removes them (see GBLA_NO_*).
 */
gbla_status gbla_forward(const gbla_shape* shape, const void* q, const void* k,
                         const void* v, const void* gate_logits, const void* out_gate,
                         const float* conv_w, const float* norm_w,
                         const int32_t* cu_seqlens, void* workspace,
                         size_t workspace_bytes, float* out, void* stream);

/*
 * gbla_forward, timed on the GPU: start_event and stop_event (hipEvent_t,
 * created by the caller, either may be NULL) are recorded on the stream
 * just before the pass's first kernel and as its last kernel ends
 * (hipExtLaunchKernel), so hipEventElapsedTime gives the pass's time on the
 * GPU without the launch gap that follows it.  Results, argument checks and
 * errors are gbla_forward's.
 */
gbla_status gbla_forward_timed(const gbla_shape* shape, const void* q, const void* k,
                               const void* v, const void* gate_logits, const void* out_gate,
                               const float* conv_w, const float* norm_w,
                               const int32_t* cu_seqlens, void* workspace,
                               size_t workspace_bytes, float* out, void* stream,
                               void* start_event, void* stop_event);

/*
 * gbla_forward for callers that cannot allocate device memory (code under
 * graph capture, tight serving loops, harnesses that forbid allocation): no
 * workspace argument; the scratch (partial states and readout operands)
 * lives in a fixed array of GBLA_NOALLOC_SCRATCH_BYTES in device memory that
 * each GPU holds from its first such call until the process ends.  Nothing
 * is allocated or freed by this call.  Shapes whose gbla_forward scratch
 * (the plan's size for the reading in use, dense or ragged) exceeds that
 * size are refused with GBLA_ERR_WORKSPACE before anything is launched;
 * about 4.5 MB serve B=1, H=8, n=32768, d=64.  The GPU is the stream's
 * (the current device for the null stream).  Every call on one GPU uses that
 * GPU's one array: calls that overlap in time on one GPU (different streams,
 * or the same array captured into graphs replayed concurrently) race and
 * must be serialised by the caller.  The array keeps the last call's
 * contents; every call initialises what it reads.  Other arguments, results
 * and errors are gbla_forward's; GBLA_ERR_HIP also if the array's device
 * address cannot be looked up.
 */
#define GBLA_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
gbla_status gbla_forward_noalloc(const gbla_shape* shape, const void* q, const void* k,
                                 const void* v, const void* gate_logits, const void* out_gate,
                                 const float* conv_w, const float* norm_w,
                                 const int32_t* cu_seqlens, float* out, void* stream);

/*
 * The Conv1D alone (Section 2.1, item "Conv1D"): writes the convolved
 * q_t, k_t, v_t (fp32, same layout as q) of every token.  Test hook; the
 * forward pass fuses the conv into its loads and never writes these.
 */
gbla_status gbla_conv1d(const gbla_shape* shape, const void* q, const void* k,
                        const void* v, const float* conv_w, const int32_t* cu_seqlens,
                        float* q_t, float* k_t, float* v_t, void* stream);

/*
 * The global state alone (Section 2.1, key-gating item, matrix form):
 *   S [N,H,d,d] fp32 with S[c][e] = sum_j g_j phi(kt_j)[c] vt_j[e],
 *   z [N,H,d]   fp32 with z[c]    = sum_j g_j phi(kt_j)[c],
 * N = B (dense) or N_s (ragged), g the softmax-normalised gates (sum 1).
 * Leaves the readout operands in the workspace for gbla_readout.
 */
gbla_status gbla_state(const gbla_shape* shape, const void* k, const void* v,
                       const void* gate_logits, const float* conv_w,
                       const int32_t* cu_seqlens, void* workspace, size_t workspace_bytes,
                       float* S, float* z, void* stream);

/*
 * The readout and gated RMSNorm alone (o_i = phi(qt_i)^T S / phi(qt_i)^T z,
 * then y), reading the state that the last gbla_state call with the same
 * shape left in this workspace.  Stage hook for tests and timing; the
 * result equals gbla_forward's.
 */
gbla_status gbla_readout(const gbla_shape* shape, const void* q, const void* out_gate,
                         const float* conv_w, const float* norm_w,
                         const int32_t* cu_seqlens, void* workspace,
                         size_t workspace_bytes, float* out, void* stream);

/*
 * gbla_readout, with the readout kernel's own duration: start_event and
 * stop_event (hipEvent_t, created by the caller, either may be NULL) are
 * recorded when the kernel begins executing and when it ends, as
 * hipExtLaunchKernel does, so hipEventElapsedTime gives the kernel's time
 * without the launch gaps that events recorded around the call would add.
 * With no tokens nothing is launched and both events are recorded on the
 * stream.  Results, argument checks and errors are gbla_readout's.
 */
gbla_status gbla_readout_timed(const gbla_shape* shape, const void* q, const void* out_gate,
                               const float* conv_w, const float* norm_w,
                               const int32_t* cu_seqlens, void* workspace,
                               size_t workspace_bytes, float* out, void* stream,
                               void* start_event, void* stop_event);

/*
 * Bytes of device scratch that gbla_backward needs for this shape (the
 * larger of the accepted dense and ragged readings; 0 if neither is).  About 12 * tokens * H * d bytes (fp32
 * gradients of the convolved q, k, v) plus per-chunk partials.
 */
size_t gbla_backward_workspace_bytes(const gbla_shape* shape);

/*
 * Gradients of L = sum(out * dy) with respect to every input of gbla_forward:
 * the chain rule through the forward pass of Section 2.1 (Conv1D, key gating,
 * the global state, the readout, the gated RMSNorm), the forward quantities
 * recomputed from the inputs.  The paper defines the forward only; the
 * backward is its exact derivative (the gates need no softmax centering
 * term: the output does not change when every gate of a sequence is scaled
 * by one factor).
 *   q ... cu_seqlens  the inputs of the gbla_forward call, same layouts
 *   dy               [B,H,n,d] or [H,T,d] fp32, dL/dout
 *   workspace        >= gbla_backward_workspace_bytes(shape) bytes
 *   dq, dk, dv       [B,H,n,d] or [H,T,d] fp32
 *   d_gate_logits    [B,H,n]   or [H,T]   fp32
 *   d_out_gate       [B,H,n,d] or [H,T,d] fp32
 *   d_conv_w         [3,H,d,W] fp32, summed over the batch
 *   d_norm_w         [H,d]     fp32, summed over the batch
 * Every output is overwritten (not accumulated).  Reductions run in an order
 * fixed by the shape: repeated calls give the same bits.  Under the ablation
 * switches (GBLA_NO_*) the inputs a switch removes, and their gradients, may
 * be NULL and are neither read nor written.
 */
gbla_status gbla_backward(const gbla_shape* shape, const void* q, const void* k,
                          const void* v, const void* gate_logits, const void* out_gate,
                          const float* conv_w, const float* norm_w,
                          const int32_t* cu_seqlens, const float* dy, void* workspace,
                          size_t workspace_bytes, float* dq, float* dk, float* dv,
                          float* d_gate_logits, float* d_out_gate, float* d_conv_w,
                          float* d_norm_w, void* stream);

/*
 * The full GBLA layer from the input embeddings X (Section 2.1, the paper's
 * own placement of the conv):
 *   Xt = Conv1D(X)  (causal, depthwise over the d_model channels)
 *   Q = Xt W_Q, K = Xt W_K, V = Xt W_V, a = Xt w_g, R = Xt W_R  (per head)
 *   y  = the attention and gated RMSNorm of gbla_forward on (Q, K, V, a, R)
 *        with no further conv.
 * bf16 only: Xt and the projections are rounded to bf16 (fp32
 * accumulation), as a bf16 layer stores them.
 */
typedef struct {
  int32_t batch;      /* B (dense) or N_s (ragged)                              */
  int32_t seqlen;     /* L (dense) or T = cu_seqlens[N_s] (ragged), >= 0         */
  int32_t d_model;    /* model width: a multiple of 64, at most 16384            */
  int32_t heads;      /* H >= 1                                                  */
  int32_t head_dim;   /* d in {32, 64, 128}                                      */
  int32_t conv_width; /* W in [1, 4]                                             */
  int32_t max_seqlen; /* ragged: an upper bound of the lengths; dense: 0         */
  int32_t dtype;      /* GBLA_BF16                                               */
  float eps;          /* RMSNorm epsilon                                         */
} gbla_layer_shape;

/* Scratch bytes of gbla_layer_forward (the projections and the core's
 * workspace): the larger of the accepted dense and ragged readings; 0 if
 * neither is accepted. */
size_t gbla_layer_workspace_bytes(const gbla_layer_shape* shape);

/*
 * The conv and the projections alone (test and stage hook):
 *   x        [B, L, d_model] or [T, d_model] bf16 (token-major embeddings)
 *   conv_x   [d_model, W] fp32, tap W-1 on the current token
 *   w_proj   [4*H*d + H, d_model] bf16: the output features' weight rows,
 *            W_Q's columns (h, e) at rows h*d + e, then W_K, W_V, W_R at
 *            offsets H*d, 2*H*d, 3*H*d, then w_g's H columns
 *   workspace >= gbla_layer_workspace_bytes(shape) bytes (holds Xt)
 *   q, k, v, r  [B, H, L, d] or [H, T, d] bf16 outputs; a [B, H, L] or [H, T]
 * Base pointers 16-byte aligned (a: 2 bytes, workspace: 256).  Does not
 * synchronize.
 */
gbla_status gbla_layer_project(const gbla_layer_shape* shape, const void* x,
                               const float* conv_x, const void* w_proj,
                               const int32_t* cu_seqlens, void* workspace,
                               size_t workspace_bytes, void* q, void* k, void* v, void* r,
                               void* a, void* stream);

/*
 * The whole layer: out [B, H, L, d] or [H, T, d] fp32 (the layout of
 * gbla_forward's output), norm_w [H, d] fp32 gamma.
 */
gbla_status gbla_layer_forward(const gbla_layer_shape* shape, const void* x,
                               const float* conv_x, const void* w_proj, const float* norm_w,
                               const int32_t* cu_seqlens, void* workspace,
                               size_t workspace_bytes, float* out, void* stream);

/* A static, human-readable name of a status code (never NULL). */
const char* gbla_status_string(gbla_status status);

/*
 * Measurement aid, not part of the method: one launch that moves exactly the
 * bytes gbla_forward must move for `token_heads` (token, head) pairs of bf16
 * inputs at head_dim d, with none of its arithmetic.  It reads q, k, v and
 * out_gate (d bf16 each per pair, 16-byte loads) and one gate logit per pair,
 * and writes d fp32 values per pair to out (16-byte stores): (4d + 1) * 2 +
 * 4d bytes per pair, 770 at d = 64.  The written values are a function of
 * the loaded bits, not GBLA.  Layouts are flat (pair-major, d contiguous).
 * The benchmark times it beside the forward as the practical ceiling of a
 * single pass over the same bytes.  Errors: GBLA_ERR_INVALID_ARGUMENT for a
 * NULL pointer or negative count, GBLA_ERR_UNSUPPORTED for d not in {32, 64,
 * 128}, GBLA_ERR_MISALIGNED unless q, k, v, out_gate, out are 16-byte and
 * gate_logits 2-byte aligned, GBLA_ERR_HIP for a failed launch.
 */
gbla_status gbla_stream_ceiling(const void* q, const void* k, const void* v,
                                const void* gate_logits, const void* out_gate,
                                int64_t token_heads, int32_t head_dim, float* out, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* GBLA_H */
