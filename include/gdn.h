/*
 * gdn.h - C ABI of the MI355X (gfx950) chunkwise gated delta rule.
 *
 * The operation (Gated DeltaNet, Sec. 3.1, Eq. "gated_delta_rule"): for each
 * sequence and head, with the state stored as a dk x dv matrix S (the
 * transpose of the paper's dv x dk state),
 *
 *     S_t = alpha_t (I - beta_t k_t k_t^T) S_{t-1} + beta_t k_t v_t^T,
 *     o_t = S_t^T q_t,              alpha_t = exp(log_alpha_t),
 *
 * evaluated chunk by chunk (64 tokens) through the gate-decayed UT transform
 * of Sec. 3.3 ("Hardware-efficient chunkwise training").  No query scale is
 * applied (the paper's o_t = S_t q_t has none).  The backward returns the
 * exact gradients of  L = sum_t <dO_t, o_t> + <dS_final, S_final>  with
 * respect to q, k, v, beta, log_alpha and the initial state (the paper gives
 * no backward; the gradient of the forward map is unique).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All tensor pointers are DEVICE pointers, contiguous, innermost dim last:
 *      q, k, dq, dk        [B, T, H, dk]   (dtype of the problem)
 *      v, o, dO, dv        [B, T, H, dv]   (dtype of the problem)
 *      beta, log_alpha,
 *      dbeta, dlog_alpha   [B, T, H]       float32 always
 *      h0, ht, dht, dh0    [Nseq, H, dk, dv] float32 always
 *    Packed variable-length input: B == 1, T = total tokens, and
 *    cu_seqlens[0..num_seqs] (int32, 0 = cu[0] <= ... <= cu[num_seqs] = T)
 *    delimit the sequences; the state restarts at every sequence start
 *    (h0[n] or zero) and chunks restart there too.  Dense input: Nseq = B.
 *  - log_alpha == NULL means alpha == 1 for every token: the ungated delta
 *    rule of DeltaNet (Sec. 2.2), without any decay arithmetic.  A NULL
 *    dlog_alpha skips the gate gradient (and the work only it needs); with
 *    log_alpha == NULL and a non-NULL dlog_alpha, it receives the gradient at
 *    log_alpha = 0.
 *  - Value preconditions (not checked on the device): log_alpha <= 0
 *    (alpha in (0, 1]); beta finite (nominally (0, 1); (0, 2) also works,
 *    nothing is clamped); q and k are already L2-normalised if the caller
 *    wants the paper's block semantics (the library does not normalise).
 *  - Pointers must be 16-byte aligned.
 *  - The library never allocates, frees or synchronises and keeps no state
 *    between calls: the caller owns every buffer, including the workspace,
 *    whose size the *_workspace_size queries return.  (One exception:
 *    gdn_chunk_fwd_noalloc uses a static device array of the library.)  All work is enqueued on
 *    `stream` (a hipStream_t; NULL = the default stream); outputs are valid
 *    when the stream reaches them.  Calls on different streams with distinct
 *    workspaces are independent.
 *  - Every argument check runs on the host before the first launch; a failed
 *    check returns its status and launches nothing.  A launch failure returns
 *    GDN_ERR_HIP.  No C++ exception crosses this boundary.
 *  - Supported head dims: (dk, dv) in {(64, 64), (128, 128), (256, 512)},
 *    in bfloat16 (fp32 accumulation) and in float32.  The block prologue and
 *    epilogue take the dims of these pairs; the fused block is bfloat16 only.
 */
#ifndef GDN_H_
#define GDN_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum { GDN_F32 = 0, GDN_BF16 = 1 } gdn_dtype;

typedef enum {
  GDN_OK = 0,
  GDN_ERR_NULL = 1,        /* a required pointer is NULL                     */
  GDN_ERR_SHAPE = 2,       /* B, T, H < 1, or packed input with B != 1      */
  GDN_ERR_UNSUPPORTED = 3, /* (dtype, dk, dv) combination not built         */
  GDN_ERR_CU_SEQLENS = 4,  /* cu_seqlens_host malformed, or device copy NULL */
  GDN_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than the query      */
  GDN_ERR_HIP = 6,         /* a kernel launch failed                         */
  GDN_ERR_ALIGN = 7,       /* a pointer is not 16-byte aligned               */
  GDN_ERR_SAVED = 8,       /* saved buffer NULL or smaller than the query    */
  GDN_ERR_VALUE = 9        /* a scalar argument (width, eps) out of range    */
} gdn_status;

typedef struct {
  int32_t B, T, H, dk, dv;
  /* Packed input: number of sequences N.  Ignored for dense input. */
  int32_t num_seqs;
  /* Packed input: device int32[N+1], or NULL for dense input.             */
  const int32_t *cu_seqlens;
  /* Packed input: the same N+1 values in host memory (used for validation
   * and grid sizing without a device-to-host copy).  Required when
   * cu_seqlens != NULL.                                                    */
  const int32_t *cu_seqlens_host;
  gdn_dtype dtype;
} gdn_problem;

/* Workspace bytes gdn_chunk_fwd / gdn_chunk_bwd need for this problem
 * (0 if the problem itself is invalid). */
size_t gdn_chunk_fwd_workspace_size(const gdn_problem *p);
size_t gdn_chunk_bwd_workspace_size(const gdn_problem *p);

/* Forward.  Sec. 3.3, the gated chunk state update and output equations
 * (output mask read as the decay mask Gamma, with its diagonal).
 *   in : q, k, v, beta; log_alpha or NULL (alpha == 1); h0 = initial
 *        states or NULL (zero)
 *   out: o; ht = final states, or NULL to skip. */
gdn_status gdn_chunk_fwd(const gdn_problem *p, const void *q, const void *k,
                         const void *v, const float *beta,
                         const float *log_alpha, const float *h0, void *o,
                         float *ht, void *workspace, size_t workspace_bytes,
                         void *stream);

/* Forward without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same operation, arguments (minus the workspace),
 * outputs, checks and statuses as gdn_chunk_fwd, and the same kernels.  The
 * workspace is a static device array of GDN_NOALLOC_SCRATCH_BYTES bytes inside
 * the library, one per GPU, held until the process ends; the call allocates
 * nothing.  Problems whose gdn_chunk_fwd_workspace_size exceeds it return
 * GDN_ERR_WORKSPACE before any HIP call (about 390 chunk-heads at
 * dk = 256, dv = 512; 900 at dk = dv = 128).  The array belongs to the
 * calling thread's current device (hipGetDevice), which must be the device of
 * the pointers and of `stream`.  All calls on one GPU share the array:
 * calls that overlap in time on that GPU (other streams, other threads) race
 * and give wrong results; serialise them.  Nothing in the array needs to
 * start at zero. */
#define GDN_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)
gdn_status gdn_chunk_fwd_noalloc(const gdn_problem *p, const void *q,
                                 const void *k, const void *v,
                                 const float *beta, const float *log_alpha,
                                 const float *h0, void *o, float *ht,
                                 void *stream);

/* Backward (stateless: recomputes the forward's chunk states itself).
 *   in : the forward's inputs; dO = gradient of o; dht = gradient of the
 *        final states or NULL (zero)
 *   out: dq, dk, dv, dbeta; dlog_alpha, or NULL to skip; dh0 = gradient
 *        of the initial states, or NULL to skip.  Every output is
 *        overwritten. */
gdn_status gdn_chunk_bwd(const gdn_problem *p, const void *q, const void *k,
                         const void *v, const float *beta,
                         const float *log_alpha, const float *h0,
                         const void *dO, const float *dht, void *dq, void *dk,
                         void *dv, float *dbeta, float *dlog_alpha, float *dh0,
                         void *workspace, size_t workspace_bytes, void *stream);

/* Forward that keeps what the backward needs (training).  Same operation
 * and outputs as gdn_chunk_fwd (Sec. 3.3), and in addition fills `saved`
 * (device memory of gdn_chunk_saved_size bytes, owned by the caller, opaque
 * to it) with the per-chunk quantities the backward reads: the cumulative
 * log-gates, each chunk's entry state S_[t], the pseudo-values
 * V' = U~ - W~ S_[t] of the UT transform, and the chunk-local operands built
 * from q, k, beta and the gates (P, T = (I + A)^-1, W~, their transposes).
 * The layout of `saved` depends only on the problem; its content is valid
 * for the inputs the call was made with until the caller overwrites it.
 * `workspace` (gdn_chunk_fwd_save_workspace_size bytes) holds the call's
 * temporaries only and may be reused as soon as the call has run. */
size_t gdn_chunk_saved_size(const gdn_problem *p);
size_t gdn_chunk_fwd_save_workspace_size(const gdn_problem *p);
gdn_status gdn_chunk_fwd_save(const gdn_problem *p, const void *q,
                              const void *k, const void *v, const float *beta,
                              const float *log_alpha, const float *h0, void *o,
                              float *ht, void *saved, size_t saved_bytes,
                              void *workspace, size_t workspace_bytes,
                              void *stream);

/* Backward from a saving forward's buffer: the same gradients as
 * gdn_chunk_bwd for the inputs gdn_chunk_fwd_save was called with, without
 * rebuilding the chunk operands or recomputing the chunk states.  Reads q,
 * k, v and beta (the same tensors the saving forward read), dO, dht (or
 * NULL) and `saved`, which it leaves unchanged; log_alpha and h0 enter
 * through `saved`.  Same outputs as gdn_chunk_bwd.  `workspace` holds
 * gdn_chunk_bwd_saved_workspace_size bytes. */
size_t gdn_chunk_bwd_saved_workspace_size(const gdn_problem *p);
gdn_status gdn_chunk_bwd_saved(const gdn_problem *p, const void *q,
                               const void *k, const void *v,
                               const float *beta, const void *dO,
                               const float *dht, const void *saved,
                               size_t saved_bytes, void *dq, void *dk,
                               void *dv, float *dbeta, float *dlog_alpha,
                               float *dh0, void *workspace,
                               size_t workspace_bytes, void *stream);

/* Token-by-token (recurrent) form, for inference: Sec. 3.1, Eq.
 * gated_delta_rule applied one token at a time,
 *     S <- alpha_t (I - beta_t k_t k_t^T) S + beta_t k_t v_t^T,   o_t = S^T q_t,
 * for every sequence and head, over all T tokens of the call (T = 1 is one
 * decode step).  Same problem description, inputs, outputs, value
 * conventions and statuses as gdn_chunk_fwd; the result equals the chunked
 * forward's up to rounding.  No workspace.  The state may be updated in
 * place: h0 == ht is allowed (h0 NULL still means a zero initial state).
 * The state is read once and written once per call, whatever T; per token
 * the call is latency-bound, so long prompts belong on gdn_chunk_fwd. */
gdn_status gdn_recurrent_fwd(const gdn_problem *p, const void *q,
                             const void *k, const void *v, const float *beta,
                             const float *log_alpha, const float *h0, void *o,
                             float *ht, void *stream);

/* Block prologue (Sec. 3.4 and the block-design figure): what turns the
 * projections into the rule's q, k, v.  Per channel c of x [B, T, H, dim]
 * (the problem's layout, dtype and sequences):
 *     u_t[c] = sum_{i < width} w[c][i] * x_{t - width + 1 + i}[c]
 * (a causal depthwise convolution over time that restarts with zeros at
 * every sequence start), z_t = silu(u_t), and with l2norm != 0
 * y_t = z_t / sqrt(|z_t|^2 + eps) over the dim channels of each (token, head)
 * (q and k), else y_t = z_t (v).  dim is the problem's dk or dv; width is
 * 1..4 (the paper says only "short"); w is fp32 [H * dim][width], tap
 * width-1 multiplying the current token.  The backward returns dx and the
 * weight gradient dw (fp32 [H * dim][width], summed over all tokens in a
 * fixed order: deterministic).  Both need gdn_conv_silu_workspace_size
 * bytes of workspace.  Errors as elsewhere; GDN_ERR_VALUE for width or eps
 * out of range. */
size_t gdn_conv_silu_workspace_size(const gdn_problem *p, int dim, int width);
gdn_status gdn_conv_silu_fwd(const gdn_problem *p, int dim, int width,
                             int l2norm, float eps, const void *x,
                             const float *w, void *y, void *workspace,
                             size_t workspace_bytes, void *stream);
gdn_status gdn_conv_silu_bwd(const gdn_problem *p, int dim, int width,
                             int l2norm, float eps, const void *x,
                             const float *w, const void *dy, void *dx,
                             float *dw, void *workspace,
                             size_t workspace_bytes, void *stream);

/* Block epilogue (Sec. 3.4: the output is normalised and gated before the
 * output projection; the figure's caption gives the gate a SiLU).  Per
 * (token, head) row of o [B, T, H, dv]:
 *     y = o / sqrt(mean(o^2) + eps) * w * silu(g)
 * with g [B, T, H, dv] (the gate projection, dtype of the problem) and w
 * fp32 [dv] shared by the heads.  The backward returns dout (the gradient
 * of o), dg and dw (fp32 [dv], deterministic); it needs
 * gdn_norm_gate_workspace_size bytes of workspace, the forward none. */
size_t gdn_norm_gate_workspace_size(const gdn_problem *p);
gdn_status gdn_norm_gate_fwd(const gdn_problem *p, float eps, const void *o,
                             const void *g, const float *w, void *y,
                             void *stream);
gdn_status gdn_norm_gate_bwd(const gdn_problem *p, float eps, const void *o,
                             const void *g, const float *w, const void *dy,
                             void *dout, void *dg, float *dw, void *workspace,
                             size_t workspace_bytes, void *stream);

/* Fused block: the prologue above run inside the chunked rule's own kernels
 * (Sec. 3.4 and the block-design figure: the projections of q, k and v pass
 * through the short convolution and SiLU, q and k through the L2
 * normalisation, before the gated delta rule).  The result is that of
 * gdn_conv_silu_fwd (l2norm 1 for q and k, 0 for v) followed by the chunked
 * rule on its outputs, up to rounding, without the rule's q, k and v making
 * a round trip through memory between the prologue and the rule: the prep
 * kernel forms them from the projections as it loads its chunk's rows, and
 * in the backward the gradient kernel applies the prologue's backward to its
 * own dq and dk (recomputing the convolution from the projections) before
 * anything is stored.
 * bf16 problems only (GDN_ERR_UNSUPPORTED otherwise), any dk, dv the rule
 * supports; dense or packed sequences as for the rule.
 *
 * The prologue is described by gdn_block_prologue: width 1..4 and eps >= 0
 * (finite) as for gdn_conv_silu_fwd (GDN_ERR_VALUE otherwise), the
 * projections xq, xk [B, T, H, dk] and xv [B, T, H, dv] (bf16, the
 * problem's layout and sequences), and the fp32 weights wq, wk [H * dk][width]
 * and wv [H * dv][width] (tap width-1 multiplies the current token).  All six
 * pointers are required and 16-byte aligned. */
typedef struct {
  int32_t width;            /* convolution taps, 1..4             */
  float eps;                /* L2 epsilon of q and k              */
  const void *xq, *xk, *xv; /* projections, bf16                  */
  const float *wq, *wk, *wv;/* convolution weights, fp32          */
} gdn_block_prologue;

/* Forward of the fused block: o and ht as gdn_chunk_fwd computes them from
 * the rule's q, k, v; beta, log_alpha, h0, o, ht and the workspace
 * (gdn_chunk_fwd_workspace_size bytes) as there.  q, k, v (optional, NULL
 * to skip) receive the rule's inputs the prologue formed, [B, T, H, d]
 * bf16. */
gdn_status gdn_block_fwd(const gdn_problem *p, const gdn_block_prologue *pro,
                         const float *beta, const float *log_alpha,
                         const float *h0, void *o, float *ht, void *q, void *k,
                         void *v, void *workspace, size_t workspace_bytes,
                         void *stream);

/* Saving forward of the fused block (training): as gdn_block_fwd, and fills
 * `saved` (gdn_chunk_saved_size bytes) as gdn_chunk_fwd_save does, with
 * gdn_chunk_fwd_save_workspace_size bytes of workspace.  q, k and v are
 * required here: the backward reads the rule's q, k, v. */
gdn_status gdn_block_fwd_save(const gdn_problem *p,
                              const gdn_block_prologue *pro, const float *beta,
                              const float *log_alpha, const float *h0, void *o,
                              float *ht, void *q, void *k, void *v, void *saved,
                              size_t saved_bytes, void *workspace,
                              size_t workspace_bytes, void *stream);

/* Backward of the fused block from a saving fused forward: the gradients
 * with respect to the block's inputs, dxq, dxk [B, T, H, dk] and dxv
 * [B, T, H, dv] (bf16), dwq, dwk, dwv (fp32, shaped as the weights, summed
 * over all tokens in a fixed order: deterministic), and dbeta, dlog_alpha
 * (optional), dh0 (optional) as gdn_chunk_bwd_saved returns them.  Reads
 * the same prologue, the rule's q, k, v that gdn_block_fwd_save wrote, beta,
 * dO, dht (or NULL) and `saved` (unchanged).  `workspace` holds
 * gdn_block_bwd_saved_workspace_size(p, width) bytes.  At dk = 64 the
 * prologue's backward of q and k runs inside the gradient kernel; at
 * dk >= 128, where that kernel holds one workgroup per CU, the gradient
 * kernel writes the rule's dq, dk into the workspace and the convolution
 * backward of q and k follows (the faster of the two forms measured at each
 * size; the results agree to rounding). */
size_t gdn_block_bwd_saved_workspace_size(const gdn_problem *p, int width);
gdn_status gdn_block_bwd_saved(const gdn_problem *p,
                               const gdn_block_prologue *pro, const void *q,
                               const void *k, const void *v,
                               const float *beta, const void *dO,
                               const float *dht, const void *saved,
                               size_t saved_bytes, void *dxq, void *dxk,
                               void *dxv, float *dwq, float *dwk, float *dwv,
                               float *dbeta, float *dlog_alpha, float *dh0,
                               void *workspace, size_t workspace_bytes,
                               void *stream);

/* Optional launch timing, for benchmarks and profilers.  The caller creates
 * and owns the events (hipEvent_t handles, e.g. from hipEventCreate).  A
 * *_timed call records events[2i] just before and events[2i+1] just after
 * its i-th kernel launch on `stream`, for the first capacity/2 launches, and
 * reports how many launches it made and their kernel names (static strings
 * owned by the library).  Durations are read with hipEventElapsedTime once
 * the stream has passed the events.  With timing == NULL a *_timed call is
 * exactly the plain call.  Same arguments, checks and statuses otherwise. */
typedef struct {
  void **events;        /* in : hipEvent_t handles                */
  int32_t capacity;     /* in : number of handles in `events`     */
  int32_t launched;     /* out: kernel launches made by the call  */
  const char *names[8]; /* out: kernel name of launch i           */
} gdn_timing;

gdn_status gdn_chunk_fwd_timed(const gdn_problem *p, const void *q,
                               const void *k, const void *v, const float *beta,
                               const float *log_alpha, const float *h0, void *o,
                               float *ht, void *workspace,
                               size_t workspace_bytes, void *stream,
                               gdn_timing *timing);
gdn_status gdn_chunk_bwd_timed(const gdn_problem *p, const void *q,
                               const void *k, const void *v, const float *beta,
                               const float *log_alpha, const float *h0,
                               const void *dO, const float *dht, void *dq,
                               void *dk, void *dv, float *dbeta,
                               float *dlog_alpha, float *dh0, void *workspace,
                               size_t workspace_bytes, void *stream,
                               gdn_timing *timing);
gdn_status gdn_chunk_fwd_save_timed(const gdn_problem *p, const void *q,
                                    const void *k, const void *v,
                                    const float *beta, const float *log_alpha,
                                    const float *h0, void *o, float *ht,
                                    void *saved, size_t saved_bytes,
                                    void *workspace, size_t workspace_bytes,
                                    void *stream, gdn_timing *timing);
gdn_status gdn_chunk_bwd_saved_timed(const gdn_problem *p, const void *q,
                                     const void *k, const void *v,
                                     const float *beta, const void *dO,
                                     const float *dht, const void *saved,
                                     size_t saved_bytes, void *dq, void *dk,
                                     void *dv, float *dbeta, float *dlog_alpha,
                                     float *dh0, void *workspace,
                                     size_t workspace_bytes, void *stream,
                                     gdn_timing *timing);

gdn_status gdn_block_fwd_timed(const gdn_problem *p,
                               const gdn_block_prologue *pro, const float *beta,
                               const float *log_alpha, const float *h0, void *o,
                               float *ht, void *q, void *k, void *v,
                               void *workspace, size_t workspace_bytes,
                               void *stream, gdn_timing *timing);
gdn_status gdn_block_fwd_save_timed(const gdn_problem *p,
                                    const gdn_block_prologue *pro,
                                    const float *beta, const float *log_alpha,
                                    const float *h0, void *o, float *ht, void *q,
                                    void *k, void *v, void *saved,
                                    size_t saved_bytes, void *workspace,
                                    size_t workspace_bytes, void *stream,
                                    gdn_timing *timing);
gdn_status gdn_block_bwd_saved_timed(
    const gdn_problem *p, const gdn_block_prologue *pro, const void *q,
    const void *k, const void *v, const float *beta, const void *dO, const float *dht, const void *saved,
    size_t saved_bytes, void *dxq, void *dxk, void *dxv, float *dwq, float *dwk,
    float *dwv, float *dbeta, float *dlog_alpha, float *dh0, void *workspace,
    size_t workspace_bytes, void *stream, gdn_timing *timing);

gdn_status gdn_recurrent_fwd_timed(const gdn_problem *p, const void *q,
                                   const void *k, const void *v,
                                   const float *beta, const float *log_alpha,
                                   const float *h0, void *o, float *ht,
                                   void *stream, gdn_timing *timing);

/* Diagnostics, for tests of the library itself.  Before its first launch
 * every call checks that each device pointer its kernels dereference is set
 * (an internal consistency check behind the argument checks above; a failure
 * is GDN_ERR_HIP).  gdn_debug_audit runs that check for launch sequence
 * `sequence` (0 forward, 1 stateless backward, 2 saving forward, 3 saved
 * backward, 4 token-by-token forward, 5 fused block forward, 6 its saving
 * forward, 7 its saved backward) on a description in which exactly the
 * pointer fields whose bit is set in `present` are non-null (field i is
 * named by gdn_debug_audit_field(i), NULL past the last; the field log_alpha
 * also switches the gate arithmetic on, cu the packed layout).  It returns
 * the index of the first required field that is missing, -1 if none is, -2
 * for an unknown sequence.  Nothing is launched or dereferenced. */
int32_t gdn_debug_audit(int32_t sequence, uint64_t present);
const char *gdn_debug_audit_field(int32_t index);

/* Which form gdn_block_bwd_saved runs, for tests of both at every size:
 * 0 by dk (the default), 1 the prologue's backward inside the gradient
 * kernel, 2 the gradient kernel then the convolution backward of q and k.
 * Process-wide; returns the previous mode, or -1 for an unknown one. */
int32_t gdn_debug_block_bwd(int32_t mode);

/* Human-readable name of a status. */
const char *gdn_status_string(gdn_status s);

#ifdef __cplusplus
}
#endif
#endif /* GDN_H_ */
