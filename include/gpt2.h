/*
 * gpt2.h - C ABI of the MI355X (gfx950) GPT-2 training-step library.
 *
 * The library runs one GPU's share of a GPT-2 training step as described in
 * arXiv 2609.28568: the forward and backward pass of every pre-LayerNorm
 * block, the LM head tied to the token table (vocabulary padded to a multiple
 * of 64, softmax over the real tokens only), softmax cross-entropy, global-norm
 * clipping and an AdamW update of fp32 master weights (section "Model",
 * Figure 1; section "Optimisation and precision"; section "Batch geometry").
 * Precision follows the paper's statement: bf16 activations; fp32 master
 * weights, gradients and optimizer state; fp32 normalisation statistics and
 * loss.
 *
 * Conventions common to every call
 *  - Plain C types only; nothing here throws. Every call returns a status:
 *      GPT2_ERR_INVALID_ARG  malformed request (bad config, NULL pointer,
 *                            shape beyond what was sized); nothing launched;
 *      GPT2_ERR_STATE        calls out of order (backward without a forward
 *                            that had targets, accumulate with no gradient,
 *                            optimizer step with no gradient);
 *      GPT2_ERR_DEVICE       a HIP runtime or launch error.
 *    gpt2_last_error() gives a human-readable reason for the last failure.
 *  - Ownership: the caller allocates every device buffer (sizes from
 *    gpt2_query_sizes) and owns the HIP stream; the library never allocates
 *    device memory and owns only the host-side handle. Buffers must outlive
 *    the handle and must not be used by other work while a call's kernels run.
 *  - Asynchrony: calls enqueue kernels on the stream given to gpt2_init and
 *    return without synchronising, except gpt2_loss and gpt2_probe_read.
 *  - Pointers named d_* are device pointers; others are host pointers.
 *  - Parameter layout: one flat fp32 buffer grouped by kind, each kind stacked
 *    over layers: wte [Vp,C], wpe [Tmax,C], ln1w [L,C], ln1b [L,C],
 *    qkvw [L,3C,C], qkvb [L,3C], attprojw [L,C,C], attprojb [L,C], ln2w [L,C],
 *    ln2b [L,C], fcw [L,F,C], fcb [L,F], fcprojw [L,C,F], fcprojb [L,C],
 *    lnfw [C], lnfb [C]. Matrices are row-major [out, in]; q|k|v are stacked in
 *    that order along qkvw's rows, head h on rows [h*hd, (h+1)*hd) of each.
 *    Gradients, Adam m and v mirror this layout (fp32); the bf16 weight copy
 *    mirrors it in bf16.
 */
#ifndef GPT2_MI355X_H
#define GPT2_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gpt2_status {
  GPT2_OK = 0,
  GPT2_ERR_INVALID_ARG = 1,
  GPT2_ERR_STATE = 2,
  GPT2_ERR_DEVICE = 3
} gpt2_status;

/* Model, batch and optimiser description ("Model"; "Optimisation and
 * precision"). Validated by gpt2_query_sizes and gpt2_init:
 *   n_layer >= 1; d_model % n_head == 0; head_dim in {16, 32, 64, 128};
 *   d_model and d_ff multiples of 64; vocab_padded >= vocab, a multiple of 64
 *   and <= 65536; 1 <= T <= max_seq_len; B >= 1; grad_accum >= 1;
 *   warmup_steps >= 1; total_steps > warmup_steps; 0 <= beta < 1;
 *   (B*T + 256) * max(vocab_padded, 3*d_model, d_ff) * 2 < 2^32, since the
 *   kernels address each token-major bf16 operand with 32-bit byte offsets
 *   (at vocab_padded 50304 that is B*T <= 42436). */
typedef struct gpt2_config {
  int32_t n_layer, n_head, d_model, d_ff;
  int32_t vocab, vocab_padded, max_seq_len;
  int32_t B, T, grad_accum;
  float ln_eps;                         /* LayerNorm epsilon (1e-5) */
  float lr_max, lr_min;                 /* schedule peak and floor */
  int32_t warmup_steps, total_steps;    /* linear warmup, then cosine */
  float beta1, beta2, adam_eps, weight_decay, grad_clip;
} gpt2_config;

/* Byte sizes of the caller-owned buffers, plus the parameter count. */
typedef struct gpt2_sizes {
  size_t params_f32, grads_f32, adam_m, adam_v, params_bf16;
  size_t activations;   /* forward state kept for the backward pass */
  size_t workspace;     /* backward and optimizer scratch */
  size_t n_params;      /* number of scalar parameters (padded vocabulary) */
} gpt2_sizes;

/* Device buffers, each at least the size gpt2_query_sizes reports and
 * 256-byte aligned. */
typedef struct gpt2_buffers {
  void *params_f32, *grads_f32, *adam_m, *adam_v, *params_bf16;
  void *activations, *workspace;
} gpt2_buffers;

typedef struct gpt2_model gpt2_model;   /* opaque host-side handle */

/* Sizes for cfg (the model of section "Model" at the micro-batch geometry
 * of "Batch geometry"; fp32 master weights, gradients and moments and a bf16
 * copy, "Optimisation and precision"). out (host) receives byte sizes.
 * Returns INVALID_ARG for a config that fails validation or a NULL pointer. */
gpt2_status gpt2_query_sizes(const gpt2_config* cfg, gpt2_sizes* out);

/* Number of parameter tensors: 2 + 12*n_layer + 2 (148 for 12 layers, the
 * count of gradient tensors the paper checks against its reference dump,
 * section "What is checked before training starts"). 0 for an invalid cfg. */
int32_t gpt2_num_tensors(const gpt2_config* cfg);

/* Describe parameter tensor idx (0 <= idx < gpt2_num_tensors): name in
 * GPT-2's flat naming (e.g. "h.10.ln_2.weight"), element offset into the flat
 * buffer, shape (ndim 1 or 2) and whether weight decay applies to it (2-D
 * weights only, "Optimisation and precision"). name must hold 64 bytes. */
gpt2_status gpt2_tensor_info(const gpt2_config* cfg, int32_t idx, char* name,
                             size_t* offset, int32_t* shape, int32_t* ndim,
                             int32_t* decay);

/* Create a handle over caller-owned buffers (bufs, host struct of device
 * pointers; the library keeps the pointers, never the memory) and enqueue the
 * initial state on hip_stream (a hipStream_t, NULL for the default stream).
 *   init_mode 0: the caller has filled params_f32 (and adam_m, adam_v: zero
 *     for a fresh run); init writes the bf16 weight copy. seed is unused.
 *   init_mode 1: seeded initialisation of section "Model": every 2-D weight
 *     (both embedding tables included) N(0, 0.02), the attention and MLP
 *     output projections (the two that write into the residual stream)
 *     N(0, 0.02/sqrt(2 n_layer)), biases and LayerNorm shifts 0, gains 1, the
 *     padding rows vocab..vocab_padded-1 of the token table exactly 0; adam_m
 *     and adam_v cleared; bf16 copy written. Element i of the flat buffer
 *     takes the Box-Muller normal (fp64) of the first two words of
 *     Philox4x32-10 (Salmon et al., SC 2011) at counter (i mod 2^32,
 *     i div 2^32, 0, 0) and key (seed mod 2^32, seed div 2^32), multiplied by
 *     its standard deviation in fp64 and rounded once to fp32, so a given seed
 *     gives the same weights on every device.
 * *out (host) receives the handle. INVALID_ARG for a bad config, a NULL or
 * unaligned buffer, or an init_mode other than 0 and 1 (nothing enqueued). */
gpt2_status gpt2_init(const gpt2_config* cfg, const gpt2_buffers* bufs,
                      void* hip_stream, uint64_t seed, int32_t init_mode,
                      gpt2_model** out);

/* Refresh the bf16 weight copy ("Optimisation and precision": bf16 compute
 * from fp32 master weights) after the caller changed params_f32. */
gpt2_status gpt2_sync_weights(gpt2_model* m);

/* Forward pass (section "Model", Figure 1): embedding, n_layer blocks, final
 * LayerNorm, tied LM head over all vocab_padded columns. d_inputs: int32
 * [B*T] token ids in [0, vocab), row-major [B, T]. d_targets: int32 [B*T]
 * next-token ids in [0, vocab), or NULL. With targets the softmax
 * cross-entropy over the first vocab columns runs too: per-token losses are
 * kept and the logits buffer is overwritten by dlogits = (softmax - onehot) /
 * (B*T*grad_accum), exactly 0 on padding columns. Without targets the logits
 * are kept. Ids outside [0, vocab) are a contract violation: the kernels
 * read row (or column) 0 in their place, so nothing is read out of bounds,
 * and note it on the device; the next gpt2_loss or gpt2_evaluate returns
 * GPT2_ERR_INVALID_ARG for it (a malformed request, told apart from a
 * failed run, section "The stack under test"). */
gpt2_status gpt2_forward(gpt2_model* m, const int32_t* d_inputs,
                         const int32_t* d_targets);

/* Backward pass (the analytic gradient of the forward of section "Model")
 * for the last forward, which must have had targets (STATE otherwise).
 * accumulate = 0 overwrites the fp32 gradients, 1 adds to them (micro-steps
 * of gradient accumulation, "Batch geometry"; STATE when there is no
 * gradient to add to). */
gpt2_status gpt2_backward(gpt2_model* m, int32_t accumulate);

/* Optimiser step ("Optimisation and precision"), 0-based step index >= 0:
 * global gradient norm over all tensors, clip coefficient grad_clip/norm when
 * the norm exceeds grad_clip, then AdamW (betas, eps, bias correction with
 * t = step + 1, decoupled decay on the 2-D weights only) at the scheduled
 * learning rate gpt2_lr_at(cfg, step); the bf16 weight copy is refreshed.
 * *lr_out (host, optional) receives the rate used; d_grad_norm_out (device
 * fp32, optional) receives the pre-clip norm. STATE when no backward has run
 * since the last step. */
gpt2_status gpt2_adamw_step(gpt2_model* m, int64_t step, float* lr_out,
                            float* d_grad_norm_out);

/* The optimizer step of gpt2_adamw_step, for callers that cannot allocate
 * memory (code under HIP graph capture, tight serving or training loops,
 * harnesses that forbid allocation): same arguments, same results, same
 * kernels, but its scratch (the sum-of-squares partials, the norm and the
 * clip coefficient) lives in a static device array of the library (16 KiB,
 * one copy per GPU, held until the process ends) instead of the caller's
 * workspace. Nothing is allocated: the array's device address is looked up
 * once per device on the first call (which must run with the model's device
 * current). The scratch does not grow with the model, so no model is too
 * large for it (INVALID_ARG would name the two sizes otherwise). Calls that
 * overlap on one GPU share the array and race; the array keeps the last
 * call's contents, every one of which a call writes before it reads it. */
gpt2_status gpt2_adamw_step_noalloc(gpt2_model* m, int64_t step, float* lr_out,
                                    float* d_grad_norm_out);

/* Loss of the last forward with targets ("Optimisation and precision": loss
 * in fp32, the mean over the B*T positions): *loss_out (host) receives the
 * mean; d_token_losses (device fp32 [B*T], row-major [B, T], optional)
 * receives each position's loss. Synchronises the stream. STATE before any
 * forward with targets; INVALID_ARG, with the loss still written, when a
 * forward since the last report was given ids outside [0, vocab). */
gpt2_status gpt2_loss(gpt2_model* m, float* loss_out, float* d_token_losses);

/* Forward-only evaluation of held-out tokens (the held-out loss of section
 * "Batch geometry" and the evaluation cadence of "Method"): the same blocks
 * as gpt2_forward, keeping one block's activations at a time, and the head
 * and cross-entropy of GPT2_FUSION_HEAD_CE mode 1 without its gradient pass:
 * the logits are never stored, only each row's softmax statistics. Its
 * per-token losses equal those of a training forward in that mode bit for
 * bit (mode 0 works from bf16-rounded logits instead of fp32 ones).
 * d_inputs, d_targets: int32 [B*T] as for gpt2_forward (targets required).
 * *loss_out (host) receives the mean loss; d_token_losses (device fp32
 * [B*T], optional) the per-token losses. It reuses the activation buffer, so
 * a following gpt2_backward needs a new gpt2_forward first (GPT2_ERR_STATE
 * otherwise); gradients and optimiser state are untouched. Synchronises the
 * stream. */
gpt2_status gpt2_evaluate(gpt2_model* m, const int32_t* d_inputs, const int32_t* d_targets, float* loss_out,
                          float* d_token_losses);

/* Learning rate at a 0-based step ("Optimisation and precision": linear
 * warmup, then cosine decay): lr_max*(step+1)/warmup for step < warmup, then
 * lr_min + (lr_max-lr_min)*(1+cos(pi*f))/2 with f the fraction of the
 * remaining steps elapsed, clamped to [0,1]. Pure function; 0 for a NULL cfg
 * or a negative step. */
float gpt2_lr_at(const gpt2_config* cfg, int64_t step);

/* Free the host handle (device buffers stay the caller's); m may be NULL. */
void gpt2_destroy(gpt2_model* m);
/* Reason for the last failure of a call on m, or of a call that had no
 * handle when m is NULL ("The stack under test": typed diagnostics). The
 * string lives until the next failing call. */
const char* gpt2_last_error(const gpt2_model* m);

/* Saved forward state, for inspection: the per-layer activations of Figure 1
 * that the paper compares against a reference dump (section "What is checked
 * before training starts"). which: one of gpt2_act; layer selects the block
 * for per-block entries. Reports (host pointers) the byte offset into the
 * activations buffer, the element count and the element type (0 = fp32,
 * 1 = bf16, 2 = int32). INVALID_ARG for an unknown entry or layer. */
typedef enum gpt2_act {
  GPT2_ACT_RESIDUAL = 0,  /* bf16 [BT,C]: block input (layer 0 = embedding
                             output; layer n_layer = last block's output) */
  GPT2_ACT_LN1 = 1,       /* bf16 [BT,C] */
  GPT2_ACT_LN1_MEAN = 2,  /* fp32 [BT] */
  GPT2_ACT_LN1_RSTD = 3,  /* fp32 [BT] */
  GPT2_ACT_QKV = 4,       /* bf16 [BT,3C] */
  GPT2_ACT_ATT = 5,       /* bf16 [BT,C], heads concatenated */
  GPT2_ACT_ATT_LSE = 6,   /* fp32 [B,H,T]: log-sum-exp of scaled scores */
  GPT2_ACT_X_MID = 7,     /* bf16 [BT,C]: residual after attention */
  GPT2_ACT_LN2 = 8,       /* bf16 [BT,C] */
  GPT2_ACT_LN2_MEAN = 9,
  GPT2_ACT_LN2_RSTD = 10,
  GPT2_ACT_FC = 11,       /* bf16 [BT,F]: MLP pre-activation */
  GPT2_ACT_GELU = 12,     /* bf16 [BT,F] */
  GPT2_ACT_LNF = 13,      /* bf16 [BT,C] */
  GPT2_ACT_LNF_MEAN = 14,
  GPT2_ACT_LNF_RSTD = 15,
  GPT2_ACT_LOGITS = 16,   /* bf16 [BT,Vp]: logits, or dlogits after a
                             forward with targets */
  GPT2_ACT_LOSSES = 17,   /* fp32 [BT]: per-token loss */
  GPT2_ACT_COUNT = 18
} gpt2_act;

gpt2_status gpt2_activation_info(const gpt2_model* m, int32_t which,
                                 int32_t layer, size_t* offset_bytes,
                                 size_t* numel, int32_t* dtype);

/* One block of section "Model" (pre-LayerNorm attention and MLP with their
 * residual connections) in isolation, used to measure and check one block:
 * d_x_in bf16 [BT,C] is copied into the residual slot of `layer`, the block
 * runs, and its output is copied to d_x_out (bf16 [BT,C], optional). The
 * backward takes the upstream gradient d_dx_out (bf16 [BT,C]), writes the
 * layer's parameter gradients (overwrite or accumulate) and the gradient
 * with respect to the block input to d_dx_in (bf16 [BT,C], optional). */
gpt2_status gpt2_block_forward(gpt2_model* m, int32_t layer,
                               const void* d_x_in, void* d_x_out);
gpt2_status gpt2_block_backward(gpt2_model* m, int32_t layer,
                                const void* d_dx_out, void* d_dx_in,
                                int32_t accumulate);

/* Embedding backward (the stage table's "embedding backward" row, section
 * "Speed") in isolation, used to check its index handling: the
 * token-table gradient receives, for each position r, the row d_dx[r] (bf16
 * [B*T, C]) at row d_ids[r] (int32 [B*T], in [0, vocab)), and the position
 * table gradient receives the batch sum per position. accumulate = 0 first
 * clears both gradients; 1 adds to them. Rows of the token table that no id
 * names are left untouched (exactly 0 after a clear). */
gpt2_status gpt2_embedding_backward(gpt2_model* m, const int32_t* d_ids,
                                    const void* d_dx, int32_t accumulate);

/* Alternative kernel arrangements of the same computation, for measuring
 * the fusions the paper reports trying (section "Speed", table of levers),
 * each checked against the arrangement it replaces:
 *   GPT2_FUSION_RESIDUAL_NORM, how a residual connection meets the pre-norm
 *   after it (the paper's fused residual-and-pre-norm lever):
 *     0 (default) the projection GEMM's epilogue adds the residual and the
 *       LayerNorm reads the sum;
 *     1 the projection writes its branch, one kernel forms the rounded sum
 *       and normalises it;
 *     2 the composed path: a separate addition kernel, then the LayerNorm.
 *     Modes 1 and 2 give bit-identical activations (the paper's gate: the
 *     fused residual sum must equal the composed addition exactly).
 *   GPT2_FUSION_HEAD_CE, the tied LM head and the cross-entropy (the stage
 *   table's cross-entropy row, section "Speed"):
 *     0 (default) the head GEMM writes the bf16 logits, one kernel reads
 *       them and writes loss and dlogits;
 *     1 the logits are never stored: a first head GEMM writes only each
 *       row's softmax statistics per tile slice and its target logit, a
 *       kernel combines them into the log-sum-exp and the loss, and a second
 *       head GEMM's epilogue writes dlogits from the fp32 logits.
 * The mode applies from the next forward pass on; the backward reads only the
 * saved activations. INVALID_ARG for an unknown fusion or mode. */
typedef enum gpt2_fusion {
  GPT2_FUSION_RESIDUAL_NORM = 0,
  GPT2_FUSION_HEAD_CE = 1
} gpt2_fusion;
gpt2_status gpt2_set_fusion(gpt2_model* m, int32_t fusion, int32_t mode);

/* Kernel timing probes for measurement, per stage in the manner of the
 * paper's stage table (section "Speed"). Kernels are grouped in classes; for
 * classes in the enabled mask, every launch is bracketed by HIP events on
 * the model's stream and its algorithmic work (flops or bytes) is counted.
 * gpt2_probe_read synchronises and reports (host pointers, each optional)
 * totals since the last reset. */
typedef enum gpt2_kclass {
  GPT2_K_GEMM_FWD = 0,       /* x W^T + bias (+ residual): one kernel */
  GPT2_K_GEMM_FWD_GELU = 1,  /* x W^T + bias with the GELU epilogue */
  GPT2_K_GEMM_DX = 2,        /* dY W */
  GPT2_K_GEMM_DX_GELU = 3,   /* dY W times GELU'(pre-activation) */
  GPT2_K_GEMM_DW = 4,        /* dY^T X into fp32 gradients (or split slices);
                                the LM head's, and the single-block path's */
  GPT2_K_ATTN_FWD = 5,
  GPT2_K_ATTN_BWD = 6,       /* dQ (which also computes D), then dK/dV */
  GPT2_K_LAYERNORM = 7,      /* forward and backward */
  GPT2_K_CROSS_ENTROPY = 8,
  GPT2_K_OPTIMIZER = 9,      /* norm, clip coefficient and AdamW */
  GPT2_K_OTHER = 10,         /* embedding, reductions, casts */
  GPT2_K_GEMM_DW_GROUPED = 11, /* every block weight gradient of a backward
                                  pass in one grouped launch */
  GPT2_K_COUNT = 12
} gpt2_kclass;

gpt2_status gpt2_probe_enable(gpt2_model* m, uint32_t class_mask);
gpt2_status gpt2_probe_reset(gpt2_model* m);
gpt2_status gpt2_probe_read(gpt2_model* m, int32_t kclass, double* total_ms,
                            int64_t* launches, double* flops, double* bytes);

#ifdef __cplusplus
}
#endif

#endif /* GPT2_MI355X_H */
