/*
 * lce.h -- C ABI of the fused linear + cross-entropy (LCE) step for MI355X (gfx950).
 *
 * The operation is the output layer of a language model and its loss:
 *
 *     logits   z_i = W x_i                       (x_i = row i of hidden[N,H], W = weight[V,H])
 *     lse_i    = log sum_v exp(z_iv)
 *     l_i      = lse_i - z_{i,y_i}  for y_i != ignore_index, else 0
 *     loss     = sum_i l_i / n_valid   (MEAN; n_valid = number of non-ignored tokens)
 *              | sum_i l_i             (SUM)
 *              | l                     (NONE, forward only)
 *     dZ_i     = g_i (softmax(z_i) - onehot(y_i)),  g_i = [y_i != ignore_index] / n_valid (MEAN) or 1 (SUM)
 *     dH = grad_hidden = dZ W,   dW = grad_weight = dZ^T X
 *
 * This is the paper's fused LinearCrossEntropy kernel (Section 3.3, "Integrated I/O and Compute
 * Co-Design", paragraph "Optimized Triton Kernels"): the projection is fused with the loss and the
 * gradients are produced chunk by chunk over the tokens, so that the N x V logits tensor is never
 * held in memory. The mixed-precision convention (bf16 or fp16 tensors on the GPU, fp32 where
 * precision matters) follows Section 2.1 ("Static footprints") and Section 3.2 ("Optimized CPU
 * Memory Layout with Shared Buffers": parameters and gradients in BF16/FP16 on the GPU).
 *
 * Conventions for every entry point
 *   - All tensor pointers are DEVICE pointers owned by the caller, row-major and contiguous:
 *     hidden [N,H], weight [V,H], labels [N] (int64), grad_hidden [N,H], grad_weight [V,H].
 *     hidden, weight, grad_hidden and grad_weight have the element type `dtype`.
 *     Pointers must be 16-byte aligned.
 *   - The library never allocates, frees or synchronises. Scratch memory comes from the caller
 *     (`workspace`, device memory of at least lce_workspace_size(...) bytes, 256-byte aligned).
 *   - Work is enqueued in order on `stream` (a hipStream_t; NULL = the default stream) and the call
 *     returns without waiting. Outputs are overwritten, never accumulated into.
 *   - Arguments are validated before anything is enqueued; on any error nothing is launched.
 *   - Results are deterministic: the same inputs on the same device give bitwise equal outputs
 *     (no atomics; every reduction has a fixed order).
 *   - Arithmetic: bf16 or fp16 operands with fp32 accumulation (dtype BF16, FP16) or fp32
 *     throughout (FP32). loss and lse are fp32; grad_hidden and grad_weight have the input dtype.
 *     With FP16 the library keeps its intermediate per-logit values in fp16 under fixed power-of-two
 *     scales, so that the 1/n_valid-sized gradient entries do not underflow fp16's exponent range;
 *     the results carry the precision of fp16 outputs. With BF16 and FP32 the backward keeps each
 *     token's exp(z - z_target) in the input dtype (the softmax gradient then factors into a
 *     per-token scale); a chunk holding a token whose loss exceeds 60 is redone with per-slice
 *     maxima instead, so no intermediate value overflows.
 *   - A non-ignored label outside [0, V) is not an error the call can report (labels live on the
 *     device); its token's loss becomes NaN (and so does a MEAN or SUM loss). With BF16 and FP32
 *     the token contributes nothing to the gradients; with FP16 it contributes its softmax without
 *     a one-hot term. The gradients stay finite either way.
 *   - MEAN with no valid token gives loss 0 and zero gradients.
 *   - Supported shapes: N, H, V >= 1 and below 2^30; H a multiple of 8 (BF16, FP16) or 4 (FP32);
 *     256 x max(H, V rounded up to 256) elements below 2^31 bytes; a chunk's blocked copies of X
 *     below 2^31 bytes and a chunk of at most 2,097,088 tokens (65534 blocks of 32); with the
 *     RMSNorm backward, N at most 4,194,240 (65535 blocks of 64 rows). Other sizes give
 *     LCE_ERR_UNSUPPORTED.
 */
#ifndef LCE_H_
#define LCE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  LCE_OK = 0,
  LCE_ERR_INVALID_ARGUMENT = 1,    /* null pointer, size < 1, unknown enum, NONE with backward */
  LCE_ERR_UNSUPPORTED = 2,         /* valid but outside the supported shapes (see above)      */
  LCE_ERR_WORKSPACE_TOO_SMALL = 3, /* workspace_bytes < lce_workspace_size(...)               */
  LCE_ERR_HIP = 4                  /* the HIP runtime reported an error while enqueueing      */
} lce_status_t;

typedef enum { LCE_DTYPE_FP32 = 0, LCE_DTYPE_BF16 = 1, LCE_DTYPE_FP16 = 2 } lce_dtype_t;

/* Same order as torch's reduction enum. */
typedef enum { LCE_REDUCTION_NONE = 0, LCE_REDUCTION_MEAN = 1, LCE_REDUCTION_SUM = 2 } lce_reduction_t;

/*
 * Bytes of device workspace needed by lce_forward (with_backward = 0) or lce_forward_backward
 * (with_backward = 1) for these sizes. chunk_tokens is the number of tokens processed per chunk
 * (0 = automatic: with backward, the largest multiple of 64 not above min(H, ceil(N/2)), at least
 * 64, raised to ceil(N / limit) rounded up to 64 when that keeps the chunk count within dW's carry
 * limit (BF16 4, FP16 9; see lce_plan_info) and is at most 2 H; forward only, all N tokens up to
 * 16384, else chunks of 16384 or the backward size if larger;
 * a nonzero value smaller than N must be a multiple of 64). The workspace holds
 * O(chunk_tokens * (V + H) + N) elements with backward (one chunk's logits-shaped buffer, two
 * rearranged copies of the chunk's hidden rows, per-token vectors), plus V x H fp32 when dW is
 * carried across chunks in fp32 (see lce_plan_info), and O(chunk_tokens * (V / 64 + H) + N)
 * forward only (per-slice partials instead); the N x V logits never exist. Returns 0 for
 * invalid arguments.
 */
size_t lce_workspace_size(int64_t N, int64_t H, int64_t V, int dtype, int with_backward,
                          int64_t chunk_tokens);

/*
 * How a call with these arguments will run (host-side planning only: nothing is launched), for
 * callers and tests that need to know which path the step takes.
 *   chunk_tokens, chunks     : tokens per chunk and number of chunks.
 *   dh_splits                : backward only: the vocabulary is split this many ways in each chunk's
 *                              dH contraction when its tile grid would not fill the device (the splits'
 *                              fp32 partials are then summed in a fixed order); 1 = the contraction
 *                              stores dH directly. 0 for a forward-only plan.
 *   target_referenced        : backward with BF16 or FP32: exp(z - z_target) is kept per logit (the
 *                              slice-maximum path is taken only by chunks whose fallback flag is set).
 *   dw_fp32_carry            : backward with BF16 / FP16 and more chunks than the type's carry limit
 *                              (BF16 4, FP16 9): dW's sum over chunks is carried in an fp32 accumulator
 *                              of V x H in the workspace instead of in dW itself. Each chunk boundary
 *                              rounds a 16-bit running sum once (at most the unit roundoff u relative),
 *                              so c chunks add up to (c - 1) u; the limits keep that, with the rounding
 *                              of the stored exponentials and of the output, within 2e-2 (BF16,
 *                              u = 2^-8) and 5e-3 (FP16, u = 2^-11) of max|dW|.
 *   workspace_bytes          : lce_workspace_size(...) of the same arguments.
 *   fallback_flags_offset    : backward only: byte offset in the workspace of `chunks` int32 flags.
 *                              After a call has completed, flag c is nonzero if and only if chunk c
 *                              was redone with slice-maximum references (some token's loss above 60,
 *                              or inputs that are not finite); each call clears them first.
 * Returns LCE_ERR_INVALID_ARGUMENT for a null `info` and otherwise the status lce_forward /
 * lce_forward_backward would return for these sizes (info untouched unless LCE_OK).
 */
typedef struct {
  int64_t chunk_tokens;
  int64_t chunks;
  int32_t dh_splits;
  int32_t target_referenced;
  int32_t dw_fp32_carry;
  int32_t reserved;
  size_t workspace_bytes;
  size_t fallback_flags_offset;
} lce_plan_info_t;
lce_status_t lce_plan_info(int64_t N, int64_t H, int64_t V, int dtype, int with_backward,
                           int64_t chunk_tokens, lce_plan_info_t* info);

/* The chunk size lce_forward_backward uses for chunk_tokens = 0 (automatic), or 0 if invalid. */
int64_t lce_auto_chunk_tokens(int64_t N, int64_t H, int64_t V, int dtype);

/*
 * Forward only: the loss, and optionally each token's log-sum-exp. The projection fused with the
 * loss without the N x V logits (Section 3.3, paragraph "Optimized Triton Kernels"); the per-token
 * loss and lse serve evaluation, where no gradient is wanted.
 *   dtype      : an lce_dtype_t value; reduction: an lce_reduction_t value (NONE, MEAN or SUM). Both
 *                are passed as int throughout this header so that any value a caller passes is
 *                well defined and an unknown one is rejected (LCE_ERR_INVALID_ARGUMENT).
 *   loss : device fp32, [1] for MEAN/SUM, [N] for NONE (per-token losses, 0 for ignored tokens).
 *   lse  : device fp32 [N], or NULL. Filled for every token, ignored ones included.
 * Performs 2*N*H*V flops of contraction.
 */
lce_status_t lce_forward(const void* hidden, const void* weight, const int64_t* labels,
                         int64_t N, int64_t H, int64_t V, int dtype,
                         int64_t ignore_index, int reduction,
                         float* loss, float* lse,
                         void* workspace, size_t workspace_bytes, void* stream);

/*
 * lce_forward without a workspace argument and without allocating, for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc. Same arguments, results and errors as lce_forward, except:
 *   - Scratch is a static device array of LCE_NO_ALLOC_SCRATCH_BYTES (64 MiB) inside the library,
 *     one per device, held from the library's first use on that device until the process ends.
 *     The call picks the largest chunk of tokens whose workspace fits it (the results do not depend
 *     on the chunk) and returns LCE_ERR_WORKSPACE_TOO_SMALL, before anything is enqueued, when even
 *     64 tokens per chunk need more (the per-token part is 12 N bytes: N up to about 5 million at
 *     H = 4096, V = 128256).
 *   - The array is shared by every call on a device and keeps the last call's contents (nothing in
 *     it has to start at zero). Calls that overlap on one device -- on different streams, or from
 *     different threads without ordering -- race on it: the caller orders them (one stream, or
 *     events). `stream` must belong to the current device.
 *   - The first call on a device looks up the array's address (hipGetSymbolAddress); no call
 *     allocates or frees memory (no hipMalloc, hipFree or allocating library routine).
 */
#define LCE_NO_ALLOC_SCRATCH_BYTES (64u << 20)
lce_status_t lce_forward_no_alloc(const void* hidden, const void* weight, const int64_t* labels,
                                  int64_t N, int64_t H, int64_t V, int dtype,
                                  int64_t ignore_index, int reduction,
                                  float* loss, float* lse, void* stream);

/*
 * Forward and backward: the reduced loss and its gradients with respect to hidden and weight
 * (upstream gradient 1; scale both outputs for another upstream value). This is the fused step of
 * Section 3.3 (paragraph "Optimized Triton Kernels"): the gradients are produced token chunk by
 * token chunk in the same call, so that only one chunk's logits-shaped buffer ever exists.
 * chunk_tokens is the chunk size (the paper fixes none; 0 picks it automatically, see
 * lce_workspace_size): a memory-for-time knob for the caller.
 *   reduction   : MEAN or SUM (NONE returns LCE_ERR_INVALID_ARGUMENT).
 *   loss        : device fp32 [1].
 *   grad_hidden : device [N,H] of dtype; grad_weight: device [V,H] of dtype.
 *   chunk_tokens: as for lce_workspace_size (pass the same value).
 * Performs 6*N*H*V flops of contraction.
 */
lce_status_t lce_forward_backward(const void* hidden, const void* weight, const int64_t* labels,
                                  int64_t N, int64_t H, int64_t V, int dtype,
                                  int64_t ignore_index, int reduction,
                                  float* loss, void* grad_hidden, void* grad_weight,
                                  int64_t chunk_tokens,
                                  void* workspace, size_t workspace_bytes, void* stream);

/*
 * The final RMSNorm fused into the step. Section 3.3 ("Optimized Triton Kernels") names RMSNorm
 * among the fused kernels; the normalisation right before the output layer is applied here,
 * in the same call and on the same stream:
 *
 *     r_i = 1 / sqrt(mean_j h_ij^2 + eps),   x_ij = gamma_j h_ij r_i
 *
 * then the LCE step above on x. The backward adds the normalisation's Jacobian:
 *     grad_hidden_ij = r_i gamma_j dX_ij - r_i^3 h_ij (1/H) sum_k h_ik gamma_k dX_ik
 *     grad_gamma_j   = sum_i dX_ij h_ij r_i            (dX = d loss / d x)
 *
 *   hidden      : device [N,H] of dtype, the rows BEFORE normalisation.
 *   gamma       : device [H] of dtype (the learned gain).
 *   eps         : >= 0 and finite, else LCE_ERR_INVALID_ARGUMENT.
 *   normed      : forward only, optional device [N,H] of dtype that receives x (NULL: x stays in
 *                 the workspace).
 *   grad_hidden : device [N,H] of dtype, gradient with respect to the pre-norm rows;
 *   grad_gamma  : device [H] of dtype;  grad_weight: device [V,H] of dtype.
 * Every other argument, convention and error is that of lce_forward / lce_forward_backward. The
 * workspace is lce_rmsnorm_workspace_size(...) bytes: the step's own plus x [N,H] (dtype), r [N]
 * and, with backward, dX [N,H] in fp32 (dX never passes through the input dtype), the dH GEMM's
 * fp32 partials for one chunk, s [N] and [ceil(N/64), H] fp32 partials of grad_gamma (summed in a
 * fixed order): O(N H), no N x V term.
 */
size_t lce_rmsnorm_workspace_size(int64_t N, int64_t H, int64_t V, int dtype, int with_backward,
                                  int64_t chunk_tokens);
lce_status_t lce_rmsnorm_forward(const void* hidden, const void* gamma, const void* weight,
                                 const int64_t* labels, int64_t N, int64_t H, int64_t V, int dtype,
                                 float eps, int64_t ignore_index, int reduction,
                                 float* loss, float* lse, void* normed,
                                 void* workspace, size_t workspace_bytes, void* stream);
lce_status_t lce_rmsnorm_forward_backward(const void* hidden, const void* gamma, const void* weight,
                                          const int64_t* labels, int64_t N, int64_t H, int64_t V,
                                          int dtype, float eps, int64_t ignore_index, int reduction,
                                          float* loss, void* grad_hidden, void* grad_gamma,
                                          void* grad_weight, int64_t chunk_tokens,
                                          void* workspace, size_t workspace_bytes, void* stream);

/*
 * Host optimizer step for the output layer's FP32 master weights (Section 3.2, "Layer-Adam
 * Optimizer"; schedule in Section 3.1, "Asynchronous Parameter Updating"). AdamW with bias
 * correction, t = step (from 1):
 *     m = b1 m + (1 - b1) g;  v = b2 v + (1 - b2) g^2
 *     p = p - lr ( (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps) + weight_decay p )
 * in fp32, updating param, exp_avg and exp_avg_sq in place (all HOST memory, n elements). grad has
 * the element type `dtype` (BF16, FP16 or FP32), typically the pinned buffer a gradient was copied
 * into from the GPU. If param16 is not NULL (16-bit dtypes only) the updated parameters are also
 * written there, rounded to `dtype` (the shared conversion buffer of Section 3.2, "Optimized CPU
 * Memory Layout with Shared Buffers", ready for the next h2d copy). n_threads: CPU threads to split
 * the range over (0 = all hardware threads). Returns after the update (no GPU work; no allocation
 * beyond the threads). Errors: LCE_ERR_INVALID_ARGUMENT for a null pointer, n < 0, step < 1,
 * an unknown dtype, param16 with FP32, or lr < 0, beta outside [0, 1), eps <= 0, weight_decay < 0
 * or any non-finite setting.
 */
typedef struct {
  float lr, beta1, beta2, eps, weight_decay;
} lce_adam_config_t;
lce_status_t lce_host_adam_step(float* param, const void* grad, int dtype, float* exp_avg,
                                float* exp_avg_sq, int64_t n, const lce_adam_config_t* cfg,
                                int64_t step, void* param16, int n_threads);

/*
 * One training step of the output layer with its FP32 master weights, Adam states and 16-bit
 * gradient/parameter buffers in host memory: the layer-sliding schedule of Section 3.1
 * ("Asynchronous Parameter Updating", "Thread-Based Lightweight Engine") and the buffers of
 * Section 3.2 ("Optimized CPU Memory Layout with Shared Buffers", "Layer-Adam Optimizer"), applied
 * to blocks of vocabulary rows of this one layer.
 *
 * On `stream`: lce_forward_backward on `weight`, with the last chunk's dW contraction run as
 * `vocab_blocks` launches over consecutive row blocks. With overlap = 1, each block's gradient is
 * copied into grad_host on a side stream as soon as it is computed; the calling thread updates that
 * block (lce_host_adam_step with n_threads threads, writing the 16-bit result into param_host) as
 * soon as its copy has landed, and copies it back into `weight` on a second side stream (after the
 * last dH contraction, the last reader of `weight`). With overlap = 0 the same work runs one phase
 * after the other (all copies out, the whole update, all copies in) as a reference schedule; both
 * give bitwise identical results.
 *
 *   hidden, labels, N, H, V, dtype (BF16 or FP16; FP32 gives LCE_ERR_UNSUPPORTED), ignore_index,
 *   reduction (MEAN/SUM), chunk_tokens, workspace: as for lce_forward_backward.
 *   weight      : device [V,H] dtype: this step's weights; updated in place (rounded from master).
 *   grad_hidden : device [N,H] dtype (dH, as in lce_forward_backward); loss: device fp32 [1].
 *   grad_weight : device [V,H] dtype: receives this step's dW.
 *   master, exp_avg, exp_avg_sq: HOST fp32 [V,H], updated in place (AdamW, see lce_host_adam_step).
 *   grad_host, param_host: HOST [V,H] dtype, pinned for asynchronous copies (page-locked memory from
 *                 hipHostMalloc); receive dW and the rounded updated weights.
 *   step        : Adam step count (>= 1); vocab_blocks in [1, 256].
 *   timing      : optional; receives the phases of this call (milliseconds).
 * Unlike the other entry points this call synchronises: it returns when the update and the copies
 * are complete (and `stream` is ordered after them). Its two side streams (non-blocking, default
 * priority) are created on the first call on a device and kept until the process ends; calls on one
 * device share them. It creates and destroys its events per call and allocates no memory. Errors as for lce_forward_backward and
 * lce_host_adam_step; LCE_ERR_HIP if a copy or stream operation fails.
 */
typedef struct {
  double step_ms;    /* wall time of the call                                               */
  double gpu_ms;     /* the forward + backward contractions on `stream`                     */
  double d2h_ms;     /* sum over blocks of the gradient copies                              */
  double update_ms;  /* host time inside the optimizer                                      */
  double h2d_ms;     /* sum over blocks of the parameter copies                             */
  double tail_ms;    /* from the end of the GPU work to the end of the last parameter copy  */
} lce_head_step_timing_t;
lce_status_t lce_head_train_step(const void* hidden, const int64_t* labels, int64_t N, int64_t H,
                                 int64_t V, int dtype, int64_t ignore_index, int reduction,
                                 int64_t chunk_tokens, void* weight, void* grad_hidden,
                                 void* grad_weight, float* loss, float* master, float* exp_avg,
                                 float* exp_avg_sq, void* grad_host, void* param_host,
                                 const lce_adam_config_t* adam, int64_t step, int vocab_blocks,
                                 int n_threads, int overlap, void* workspace,
                                 size_t workspace_bytes, void* stream,
                                 lce_head_step_timing_t* timing);

/*
 * Per-kernel timing, for measurement tools (not for concurrent use). While enabled, every launch of
 * lce_forward / lce_forward_backward (and of their RMSNorm variants) is bracketed by two hipEvents
 * recorded on the call's stream.
 * lce_timing_read waits for the recorded events and returns, per kernel kind, the total elapsed
 * milliseconds and the number of launches since the last enable; the events are then released.
 * Kinds: 0 logits GEMM + log-sum-exp, 1 dH GEMM (with its split reduction), 2 dW GEMM,
 * 3 dlogits, 4 (unused), 5 the remaining small kernels (including the RMSNorm ones).
 * lce_timing_enable(1) resets the totals; (0) stops recording. Returns LCE_OK or LCE_ERR_HIP.
 */
#define LCE_TIMING_KINDS 6
lce_status_t lce_timing_enable(int enable);
lce_status_t lce_timing_read(double* ms, int64_t* launches, int n_kinds);

/* A static, human-readable name for a status code. */
const char* lce_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* LCE_H_ */
