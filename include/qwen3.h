/*
 * qwen3.h - C ABI of the Qwen3-shaped adapter fine-tuning step (MI355X, gfx950).
 *
 * The step of the paper's clinical stage (arXiv 2609.28568, section "The
 * clinical stage"): a frozen bf16 Qwen3-shaped decoder adapted with
 * rank-stabilised low-rank adapters (output scaled by alpha / sqrt(rank)),
 * loss taken on the answer part of every sequence only, AdamW with
 * global-norm clipping on the adapter parameters alone (section
 * "Optimisation and precision"). Architecture: pre-RMSNorm layers;
 * grouped-query attention with an RMSNorm over the head dimension on every
 * query and key head and a rotary embedding (split-half pairs); a SwiGLU MLP;
 * a final RMSNorm; the token table tied to the LM head; no biases.
 *
 * Shares the status codes and the conventions of gpt2.h: plain C types,
 * nothing throws, caller-owned device buffers and stream, calls enqueue
 * asynchronously except qwen3_loss, d_* pointers are device pointers.
 *
 * Buffer layouts (element offsets and shapes also from qwen3_tensor_info):
 *  - base_bf16, frozen, in this order, matrices row-major [out, in], stacked
 *    over the L layers: embed [V,C]; in_norm [L,C]; qkv [L, (H+2Hkv)*hd, C]
 *    (query rows, then key rows, then value rows, head h on rows
 *    [h*hd, (h+1)*hd) of each); q_norm [L,hd]; k_norm [L,hd]; o [L,C,H*hd];
 *    post_norm [L,C]; gate_up [L,2F,C] (gate rows, then up rows);
 *    down [L,C,F]; final_norm [C].
 *  - lora_f32 (fp32 master), lora_grads, adam_m, adam_v (fp32) and lora_bf16
 *    (bf16 copy the GEMMs read) share one layout: for every enabled group in
 *    the order q|k|v, o, gate|up, down: A [L, n*RP, in] then B [L, out, RP],
 *    where RP = 64 is the padded rank, n the projections of the group (3, 1,
 *    2, 1) and out the group's total output width (its projections' rows
 *    stacked as in base_bf16). A projection's A occupies rows [j*RP, j*RP+r)
 *    of its group's A, its B columns [0, r); the padding rows and columns are
 *    zero and stay zero (their gradients are exactly zero).
 */
#ifndef QWEN3_MI355X_H
#define QWEN3_MI355X_H

#include <stddef.h>
#include <stdint.h>

#include "gpt2.h"

#ifdef __cplusplus
extern "C" {
#endif

/* adapter groups (lora_groups bit mask) */
enum { QWEN3_LORA_QKV = 1, QWEN3_LORA_O = 2, QWEN3_LORA_GATE_UP = 4, QWEN3_LORA_DOWN = 8 };

typedef struct qwen3_config {
  int32_t n_layer, d_model, n_head, n_kv_head, head_dim, d_ff, vocab, max_seq_len;
  int32_t B, T;              /* micro-batch geometry, T <= max_seq_len */
  float rms_eps;             /* 1e-6 */
  float rope_theta;          /* 1e6 */
  int32_t lora_rank;         /* r, 1..32 */
  float lora_alpha;          /* adapter output scaled by alpha / sqrt(r) */
  int32_t lora_groups;       /* QWEN3_LORA_* bits; q|k|v and o: 3 */
  float loss_from;           /* loss on positions t >= floor(loss_from * T) of every sequence */
  float lr, beta1, beta2, adam_eps, weight_decay, grad_clip;   /* adapter AdamW */
} qwen3_config;

typedef struct qwen3_sizes {
  size_t base_bf16, lora_f32, lora_grads, adam_m, adam_v, lora_bf16, activations, workspace;   /* bytes */
} qwen3_sizes;

typedef struct qwen3_buffers {
  void *base_bf16, *lora_f32, *lora_grads, *adam_m, *adam_v, *lora_bf16, *activations, *workspace;
} qwen3_buffers;

typedef struct qwen3_model qwen3_model;

/* Validation: head_dim == 128; n_head a multiple of n_kv_head; d_model and
 * d_ff multiples of 128, vocab and B*T multiples of 64 (every contraction is
 * a whole number of GEMM k-tiles); T <= max_seq_len; 1 <= lora_rank <= 32;
 * every buffer a kernel addresses below 4 GiB (32-bit offsets). Failures
 * return GPT2_ERR_INVALID_ARG. */
gpt2_status qwen3_query_sizes(const qwen3_config* cfg, qwen3_sizes* out);

/* Tensor idx of the base (which = 0) or adapter (which = 1) layout: name,
 * element offset, shape (ndim <= 3). GPT2_ERR_INVALID_ARG past the last one. */
gpt2_status qwen3_tensor_info(const qwen3_config* cfg, int32_t which, int32_t idx, char name[64], size_t* offset,
                              int32_t shape[3], int32_t* ndim);

/* Bind the buffers and stream; the caller fills base_bf16 and lora_f32 and
 * zeroes adam_m and adam_v. Writes lora_bf16 from lora_f32. */
gpt2_status qwen3_init(const qwen3_config* cfg, const qwen3_buffers* bufs, void* hip_stream, qwen3_model** out);

/* Re-derive lora_bf16 from lora_f32 (after the caller changed lora_f32). */
gpt2_status qwen3_sync_weights(qwen3_model* m);

/* Forward over d_inputs [B*T] (int32 token ids in [0, vocab)); with d_targets
 * [B*T] also the masked loss and the logit gradient the backward needs. The
 * final norm and the LM head run on the positions that carry loss only (the
 * others' logits enter neither the loss nor any gradient). */
gpt2_status qwen3_forward(qwen3_model* m, const int32_t* d_inputs, const int32_t* d_targets);

/* Adapter gradients of the masked mean loss into lora_grads (overwritten).
 * GPT2_ERR_STATE unless the last forward had targets. */
gpt2_status qwen3_backward(qwen3_model* m);

/* Clip the adapter gradients to global norm grad_clip and apply one AdamW
 * step (step counted from 0) to lora_f32, m, v; rewrites lora_bf16. The norm
 * before clipping goes to d_grad_norm_out if given. GPT2_ERR_STATE without a
 * backward since the last step. */
gpt2_status qwen3_adamw_step(qwen3_model* m, int64_t step, float* d_grad_norm_out);

/* Masked mean loss of the last forward with targets (synchronises the stream);
 * the per-position losses [B*T] (0 on positions without loss) are copied to
 * d_token_losses if given. */
gpt2_status qwen3_loss(qwen3_model* m, float* loss_out, float* d_token_losses);

/* Alternative kernel arrangements, for measurement and for the tests that
 * compare them (the paper's fusion levers, section "Speed"):
 *   QWEN3_FUSION_SWIGLU, where the SwiGLU of the MLP runs:
 *     1 (default) in the GEMM epilogues: the gate|up projection writes its
 *       pre-activation and silu(gate) up; the input gradient of the down
 *       projection writes the gate and up gradients from the saved
 *       pre-activation, and its own output is never stored (a projection
 *       with an adapter keeps the separate kernels);
 *     0 separate SwiGLU forward and backward kernels between the GEMMs.
 *   Both compute the same bits. GPT2_ERR_INVALID_ARG for an unknown
 *   arrangement or mode. */
enum { QWEN3_FUSION_SWIGLU = 0 };
gpt2_status qwen3_set_fusion(qwen3_model* m, int32_t fusion, int32_t mode);

void qwen3_destroy(qwen3_model* m);
const char* qwen3_last_error(const qwen3_model* m);

/* Kernel timing probes for measurement, as gpt2_probe_*: launches of the
 * enabled classes are bracketed with HIP events on the model's stream, and
 * their algorithmic FLOPs (GEMMs: 2 M N K at the true adapter rank;
 * attention: the causal half) and bytes are summed per class.
 * qwen3_probe_read synchronises and reports totals since the last reset. */
enum {
  QWEN3_K_GEMM_FWD = 0,      /* frozen projections (with the adapter's u B^T as a second contraction
                                segment of the same GEMM) and the LM head, forward */
  QWEN3_K_GEMM_DX = 1,       /* their input gradients (with du A likewise; the LM head's included) */
  QWEN3_K_GEMM_ADAPTER = 2,  /* the other adapter products: s x A^T, s dy B, and the adapter gradients */
  QWEN3_K_ATTN_FWD = 3,
  QWEN3_K_ATTN_BWD = 4,
  QWEN3_K_NORM = 5,          /* RMSNorm forward/backward, q/k head norm + rotary forward/backward */
  QWEN3_K_CROSS_ENTROPY = 6,
  QWEN3_K_OPTIMIZER = 7,     /* norm, clip coefficient and AdamW */
  QWEN3_K_OTHER = 8,         /* embedding gather, SwiGLU, scales, reductions */
  QWEN3_K_COUNT = 9
};
gpt2_status qwen3_probe_enable(qwen3_model* m, uint32_t class_mask);
gpt2_status qwen3_probe_reset(qwen3_model* m);
gpt2_status qwen3_probe_read(qwen3_model* m, int32_t kclass, double* total_ms, int64_t* launches, double* flops,
                             double* bytes);

#ifdef __cplusplus
}
#endif

#endif
