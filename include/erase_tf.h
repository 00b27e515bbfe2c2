/*
 * erase_tf.h -- C ABI of the detached small-transformer training step.
 *
 * The operation: the paper splits NanoChat's attention stack into detached
 * pieces that each learn from their own objective and send no gradient to
 * the piece before them (Section 3.1, with Eq. 1 and Eq. 2 of Section 2).
 * Here every layer is one detached block with its own local next-token
 * head, on token ids uniform over the vocabulary:
 *
 *   a0_1 = E[tokens[:, :-1]]            (block 1 owns the embedding E)
 *   a0_b = sg[z_{b-1}]                  (b > 1)
 *   n1 = rms(a0);  [q | k | v] = n1 Wqkv^T
 *   o  = causal softmax attention of every head (head size 64, scale 1/8)
 *   a1 = a0 + o Wo^T;  n2 = rms(a1);  z = a1 + gelu(n2 W1^T) W2^T
 *   l_b = mean over the B*T positions of -log softmax(rms(z) Wh_b^T)[next token]
 *
 * with rms(x) = x / sqrt(mean(x^2) + 1e-6) per row (no gain), gelu in its
 * tanh form, no biases, and L = lambda * sum_b l_b.  Block b's backward needs
 * only its own forward and local loss; ERASE (Section 2.2) launches it early
 * on a second stream.  Block 1 also updates the embedding rows its tokens
 * selected (dense Adam over the whole table, as with a dense gradient).
 *
 * The conventions of erase.h hold: erase_status results, caller-owned device
 * memory and streams (distinct, default priority), host validation before
 * anything is enqueued, deferred device errors at erase_tf_sync() that stay
 * sticky, one context per host thread, no device allocation after init.
 * bf16 GEMM operands and stored activations, fp32 accumulation, fp32 master
 * parameters, moments, gradients, statistics and losses.
 */
#ifndef ERASE_TF_H_
#define ERASE_TF_H_

#include "erase.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Opaque transformer-step context: created by erase_tf_init(), owned by
 * the library, released by erase_tf_destroy(). */
typedef struct erase_tf_ctx erase_tf_ctx;

typedef struct {
  int32_t vocab;     /* V: multiple of 64, 64..1048576 */
  int32_t d_model;   /* d = 64 * n_heads, at most 4096 */
  int32_t n_heads;   /* head size is 64 */
  int32_t n_layers;  /* detached blocks, 1..64 */
  int32_t seq_len;   /* T >= 1 */
  int32_t batch;     /* B >= 1, B * T <= 2^24 */
  float lr, beta1, beta2, eps;  /* Adam as in erase_config */
  float lambda;      /* weight of every local loss (finite) */
} erase_tf_config;

/* Per-block fp32 parameters (erase_block_buffers of erase.h), in this flat
 * order: block 0 only: E[V][d]; then every block: Wqkv[3d][d], Wo[d][d],
 * W1[4d][d], W2[d][4d], Wh[V][d] (row-major, torch nn.Linear layout).
 * Host only; no HIP call. */
ERASE_API erase_status erase_tf_param_count(const erase_tf_config* cfg, int32_t block, int64_t* count);

/* Bytes of device workspace for `cfg`: per block the activations, the
 * vocabulary logits [B T][V] (bf16, overwritten in place by their
 * gradient), softmax statistics, activation gradients, weight-gradient
 * partials and the bf16 weight copies.  Host only; no HIP call. */
ERASE_API erase_status erase_tf_workspace_bytes(const erase_tf_config* cfg, size_t* bytes);

/* Validate, carve `workspace` (device, 256-byte aligned) and create the
 * context.  Enqueues on s_fwd the zeroing of the workspace and the weight
 * copies; resets the step counter to 0; does not synchronize.  `bufs` is a
 * host array of n_layers entries (param, m, v required, grad optional; all
 * 4-byte aligned) that must stay valid for the context's life. */
ERASE_API erase_status erase_tf_init(const erase_tf_config* cfg, const erase_block_buffers* bufs, void* workspace,
                           size_t ws_bytes, void* s_fwd, void* s_bwd, erase_tf_ctx** ctx_out);

/* Enqueue one training step and return without waiting.
 *   tokens: device int32 [batch][seq_len + 1]; position t of row b reads
 *           tokens[b][t] and predicts tokens[b][t + 1].  An id outside
 *           [0, V) reads a zero embedding row and is never a target; the
 *           step completes and erase_tf_sync() returns
 *           ERASE_ERR_INVALID_ARG (sticky).
 *   schedule: ERASE_SCHED_SERIAL (everything on s_fwd: forward and local
 *           loss of blocks 1..B, backward of B..1, Adam of 1..B) or
 *           ERASE_SCHED_OVERLAP (block b's body forward on s_fwd; its head,
 *           loss, backward and Adam on s_bwd after an event, overlapping
 *           block b+1's forward; the step ends with s_fwd joined on s_bwd).
 *           Both run identical kernels and give bit-identical results.
 *           Other schedules: ERASE_ERR_UNSUPPORTED.
 *   losses: device fp32 [n_layers], receives the unweighted l_b.
 * tokens and losses must stay valid and unmodified until erase_tf_sync(). */
ERASE_API erase_status erase_tf_step(erase_tf_ctx* ctx, const int32_t* tokens, int32_t schedule, float* losses);

/* Wait for the context's work; report deferred errors (HIP errors,
 * ERASE_ERR_NONFINITE for a non-finite loss, ERASE_ERR_INVALID_ARG for an
 * out-of-range token id), all sticky. */
ERASE_API erase_status erase_tf_sync(erase_tf_ctx* ctx);

/* Step counter (synchronizes s_fwd), weight-copy refresh after the caller
 * changed `param`, as in erase.h. */
ERASE_API erase_status erase_tf_get_step(erase_tf_ctx* ctx, int64_t* t);
ERASE_API erase_status erase_tf_set_step(erase_tf_ctx* ctx, int64_t t);
ERASE_API erase_status erase_tf_refresh_weights(erase_tf_ctx* ctx);

/* Per-launch timing as in erase.h (erase_kernel_time records; record 0 is
 * the empty interval, kind 7).  Kinds of this step: 0 prologue, 1 forward
 * GEMM (layer: 0 qkv, 1 output projection, 2 MLP up, 3 MLP down, 4
 * vocabulary logits), 3 weight-grad GEMM and 4 input-grad GEMM (layer as for
 * 1), 6 both gradient GEMMs of one weight in one launch (layer as for 1),
 * 5 Adam, 11 embedding gather, 12 RMSNorm forward, 13 RMSNorm backward,
 * 14 attention forward, 15 attention backward (layer 1 row sums, 2 dK/dV,
 * 3 dQ), 16 softmax normaliser of the vocabulary head (layer 0 every row,
 * 1 the recomputation of out-of-range rows), 17 embedding gradient (four
 * launches, bracketed by stream events rather than kernel-stamped ones). */
ERASE_API erase_status erase_tf_set_timing(erase_tf_ctx* ctx, int32_t enable);
ERASE_API erase_status erase_tf_read_timing(erase_tf_ctx* ctx, erase_kernel_time* out, int32_t cap, int32_t* n);

/* Device address and row pitch (elements) of a stored tensor of block
 * `block`, for inspection after erase_tf_sync():
 *   0 a0, 1 n1, 2 qkv [.][3d], 3 o, 4 a1, 5 n2, 6 u [.][4d] (MLP
 *   pre-activation), 7 gelu(u), 8 z, 9 hn, 10 the head's exponentials
 *   e[n][v] = exp(logit - target logit) [.][V] (bf16; after a step the
 *   target entry holds e - S_n, S_n the row's sum, so that rowscale[n] e[n]
 *   is the logit gradient lam (softmax - onehot) / N), 11 lse (fp32
 *   [B][H][T], pitch T), 12 dqkv, 13 dz, 14 rowscale (fp32 [B T], pitch
 *   B T: lam / (N S_n)), 15 hns = rowscale hn (bf16 unless noted; rows are
 *   positions b T + t).  ERASE_ERR_INVALID_ARG for an unknown id or block. */
ERASE_API erase_status erase_tf_tensor(erase_tf_ctx* ctx, int32_t block, int32_t which, void** ptr, int64_t* ld);

/* Destroy (waits for the streams; frees events).  NULL is accepted. */
ERASE_API erase_status erase_tf_destroy(erase_tf_ctx* ctx);

/* Last error message recorded on the context ("" if none). */
ERASE_API const char* erase_tf_last_error(erase_tf_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* ERASE_TF_H_ */
