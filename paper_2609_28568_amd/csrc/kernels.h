// Internal launcher interface between the host library and the HIP kernels.
// Every launcher enqueues on the given stream and returns hipGetLastError().
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;

// ---------------------------------------------------------------- GEMM
enum GemmEpilogue {
  EPI_BF16 = 0,      // C = bf16(acc + bias? + residual?)
  EPI_GELU = 1,      // C = bf16(acc + bias) (pre-activation), C2 = bf16(gelu(acc + bias))
  EPI_GELU_BWD = 2,  // C = bf16(acc * gelu'(aux))
  EPI_F32 = 3,       // C (fp32, one slice per split) = acc (+ C if accumulate)
  EPI_CE_STATS = 7,  // softmax statistics of each row, see GemmArgs
  EPI_CE_GRAD = 8,   // softmax cross-entropy gradient of each row, see GemmArgs
  // SwiGLU fused into the gate|up projection (B = [gate rows; up rows], N =
  // 2F output columns, no second segment, tiles 128 columns wide): a tile's
  // B rows alternate 32 gate rows and the 32 up rows of the same features, so
  // C = the pre-activation [M][2F] (gate columns, then up columns, row stride
  // ldc) and C2 = silu(gate) up [M][F] (row stride F), computed from the
  // bf16-rounded pre-activation as the separate kernel does
  EPI_SWIGLU = 9,
  // SwiGLU backward fused into the input gradient of the down projection
  // (N = F): the product, rounded to bf16, is the gradient of silu(gate) up;
  // with aux = the saved pre-activation [M][2F] (row stride ldc) the epilogue
  // writes C = [gate gradient | up gradient] [M][2F] (row stride ldc)
  EPI_SWIGLU_BWD = 10
};

struct GemmArgs {
  const bf16_t* A;
  const bf16_t* B;
  int M, N, K;
  int lda, ldb;
  void* C;
  int ldc;
  const float* bias;       // [N] or null
  const bf16_t* residual;  // [M][ldc] or null
  bf16_t* C2;              // second output of EPI_GELU
  const bf16_t* aux;       // pre-activation for EPI_GELU_BWD
  int accumulate;
  int splits;              // split of the contraction over grid.z (EPI_F32 only)
  long split_stride;       // elements between split output slices
  int k_chunk;             // contraction length per split (from gemm_split_plan)
  // EPI_F32 with A read transposed (a weight gradient dY^T X): when set, the
  // GEMM also writes partial sums of A's rows over the contraction (the bias
  // gradient, sum over tokens of dY) into [gemm_bias_parts(M, N, splits)][M];
  // summing those rows gives the bias gradient
  float* bsum;
  // EPI_BF16 without residual: the accumulator is multiplied by alpha before
  // the bias (0 or 1: no scaling)
  float alpha;
  // Optional second contraction segment (K2 > 0; A not transposed, no split,
  // K and K2 multiples of 64): C += A2 B2 over K2 more indices, A2 [M][lda2]
  // and B2 in B's orientation (row stride ldb2). Output columns n >=
  // a2_bound[i] (for each non-zero bound, multiples of 128) read A2 from K2
  // columns further right per bound passed, so column blocks of the output
  // can contract with different column blocks of A2.
  const bf16_t* A2;
  const bf16_t* B2;
  int K2, lda2, ldb2;
  int a2_bound[2];
  // Output rows m >= b_bound[i] (for each non-zero bound, multiples of 128)
  // read B from b_step columns further right per bound passed, so row blocks
  // of the output can contract with different column blocks of B.
  int b_bound[2], b_step;
  // row stride of the bsum partial rows (0: M)
  int bsum_ld;
  // Softmax cross-entropy over the output rows (the tied LM head, rows =
  // token positions, columns = vocabulary entries; only columns < ce_V count,
  // targets outside [0, ce_V) read column 0):
  //   EPI_CE_STATS writes no C: for each row, per wave-column slice of each
  //     tile, the max and the sum of exp(logit - max) over its real columns
  //     into ce_stats [M][gemm_ce_parts(N)] (float2), and the target's logit
  //     into ce_tlogit [M];
  //   EPI_CE_GRAD writes C = bf16((exp(logit - ce_lse[m]) - [n == target])
  //     * ce_scale) on real columns, 0 on the others.
  const int32_t* ce_targets;
  float* ce_stats;
  float* ce_tlogit;
  const float* ce_lse;
  int ce_V;
  float ce_scale;
};

// Grouped weight gradients: launch_gemm_grouped runs, in one launch, every
// tile of up to GEMM_GROUPS groups of products C_p[m][n] (=|+=) sum_k A_p[k][m]
// B_p[k][n] (A and B read transposed, fp32 output, contraction length K
// shared by all). Group i holds `count` products of the same M x N whose
// operands and outputs sit at fixed element strides from the group's first
// one (C_p row stride N). With bsum, product p also writes the partial sums of
// A_p's rows (its bias gradient) into rows [slot][p][M] of bsum, slot <
// gemm_bias_parts(M, N, 1); summing over slots gives the bias gradients of
// the group's products, stored one after another.
// A group with splits > 1 divides its contraction into `splits` chunks of
// k_chunk tokens (a multiple of 64): product p's chunk z writes the plain sum
// (never accumulating) to C_p + z * split_stride, for the caller to reduce;
// such a group carries no bsum. With nfull > 0 the groups before the last
// one hold nfull tiles and the last one the rest (both multiples of 8), and
// each of the 8 XCDs takes an equal share of both (the last group's tiles
// filling the final round).
constexpr int GEMM_GROUPS = 5;
struct GemmGroup {
  const bf16_t* A;
  const bf16_t* B;
  float* C;
  float* bsum;
  long a_stride, b_stride, c_stride;
  int M, N, lda, ldb;
  int count;
  int splits, k_chunk;   // contraction split (splits <= 1: none)
  long split_stride;
};
struct GemmGroupedArgs {
  GemmGroup grp[GEMM_GROUPS];
  int ngroups;
  int K;
  int accumulate;
  int nfull;   // tiles before the last group when its tiles fill the final round (0: no such plan)
};
hipError_t launch_gemm_grouped(const GemmGroupedArgs& g, hipStream_t s);
// Partial rows (slots) a grouped launch writes for group i's bias sums; it
// depends only on the groups' M and N
int gemm_grouped_bias_parts(const GemmGroupedArgs& g, int i);

// Block tile (bm x bn, contraction depth bk per stage) the GEMM uses for an
// M x N product with the given operand orientation and epilogue.
struct GemmConfig { int bm, bn, bk; };
GemmConfig gemm_config(int M, int N, int a_t, int b_t, int epi);
// Plan a contraction split of K into about `want` pieces: writes the chunk
// length (a multiple of the 64-wide k tile) and returns the split count.
int gemm_split_plan(int K, int want, int* k_chunk);
// Partial rows a weight-gradient GEMM writes into GemmArgs::bsum
int gemm_bias_parts(int M, int N, int splits);
hipError_t launch_gemm(const GemmArgs& g, int a_t, int b_t, int epi, hipStream_t s);
// float2 partials per row that EPI_CE_STATS writes for an M x N product
int gemm_ce_parts(int M, int N);
// Combine the EPI_CE_STATS partials of each row: lse[r] = log-sum-exp of the
// real columns, losses[r] = lse[r] - tlogit[r]; targets outside [0, V) set
// bit ID_BAD_TARGET of *bad (when not null).
hipError_t launch_ce_combine(const float* stats, int nparts, const float* tlogit, const int32_t* targets, int V,
                             float* lse, float* losses, int rows, uint32_t* bad, hipStream_t s);

// ---------------------------------------------------------------- attention
// Grouped-query attention: H query heads, Hkv key/value heads (0: Hkv = H),
// query head h reading key/value head h / (H / Hkv). q|k|v rows hold the H
// query heads, then the Hkv key heads, then the Hkv value heads, hd channels
// each: row stride W = (H + 2 Hkv) hd. C = H hd.
struct AttnArgs {
  int B, T, H, hd;
  const bf16_t* qkv;   // [B*T, W]
  bf16_t* out;         // [B*T, C]
  float* lse;          // [B, H, T]
  // backward
  const bf16_t* dout;  // [B*T, C]
  float* dsum;         // [B, H, T] rowsum(dout * out)
  bf16_t* dqkv;        // [B*T, W]; a key/value head's gradient sums over its query heads
  int Hkv;
};
hipError_t launch_attention_fwd(const AttnArgs& a, hipStream_t s);
hipError_t launch_attention_bwd(const AttnArgs& a, hipStream_t s);

// ---------------------------------------------------------------- layernorm
hipError_t launch_layernorm_fwd(const bf16_t* x, const float* w, const float* b, bf16_t* y,
                                float* mean, float* rstd, int rows, int C, float eps, hipStream_t s);
// The residual connection and the following pre-norm in one pass: xsum =
// bf16(res + x) (fp32 sum, rounded to nearest even), then y = LayerNorm(xsum)
// read from those rounded values, bit for bit what launch_residual_add
// followed by launch_layernorm_fwd gives. res == nullptr: plain LayerNorm of x.
hipError_t launch_add_layernorm_fwd(const bf16_t* x, const bf16_t* res, bf16_t* xsum, const float* w, const float* b,
                                    bf16_t* y, float* mean, float* rstd, int rows, int C, float eps, hipStream_t s);
// out = bf16(res + x) elementwise (n % 4 == 0)
hipError_t launch_residual_add(const bf16_t* res, const bf16_t* x, bf16_t* out, long n, hipStream_t s);
// dres_out = (has_res ? dres_in : 0) + dx (dres_in may be dres_out; it is not
// read when has_res == 0).
// Each block writes one row of partials part[blk][3][C]: sums over its rows of
// dy*xhat (gain gradient), dy (shift gradient) and the new dres (the bias
// gradient of the linear layer whose output gradient dres is).
int layernorm_bwd_blocks(int rows);
hipError_t launch_layernorm_bwd(const bf16_t* dy, const bf16_t* x, const float* mean,
                                const float* rstd, const float* w, const bf16_t* dres_in, bf16_t* dres_out,
                                int has_res, float* part, int rows, int C, hipStream_t s);

// ---------------------------------------------------------------- misc
// dst[i] (fp32, n elements) = (accumulate ? dst[i] : 0) + sum_s src[s*n + i]
hipError_t launch_reduce_slices(const float* src, int nslices, long n, float* dst, int accumulate,
                                hipStream_t s);
// dst[i] (bf16, n elements, n % 4 == 0) = scale * sum_s src[s*n + i]
hipError_t launch_reduce_slices_bf16(const float* src, int nslices, long n, float scale, bf16_t* dst, hipStream_t s);
// The same for two independent segments in one launch (n and n2 multiples of 4)
hipError_t launch_reduce_slices2(const float* src, int nslices, long n, float* dst, const float* src2,
                                 int nslices2, long n2, float* dst2, int accumulate, hipStream_t s);
// Sum over S slices of partial rows, for narrow rows and many slices:
// dst_j[c] (=|+=) sum_s part[s*stride + j*n + c], for j < nd (up to 3
// destinations, null ones skipped) and c < n. Fixed summation order.
hipError_t launch_reduce_parts(const float* part, int S, long stride, int n, int nd, float* d0, float* d1,
                               float* d2, int accumulate, hipStream_t s);
// Up to REDUCE_JOBS such reductions of one shape (S slices of stride floats,
// nd outputs of n) in one launch: job j sums part[j] into d[j][0..nd-1]
// (null destinations skipped).
constexpr int REDUCE_JOBS = 32;
struct ReducePartsJobs {
  int count;
  const float* part[REDUCE_JOBS];
  float* d[REDUCE_JOBS][3];
};
hipError_t launch_reduce_parts_multi(const ReducePartsJobs& J, int S, long stride, int n, int nd, int accumulate,
                                     hipStream_t s);
// Token ids outside [0, V) are a caller's contract violation: the kernels
// that read ids (embedding forward, cross-entropy target gather) read row 0
// in their place and set bit ID_BAD_INPUT or ID_BAD_TARGET of *bad (when bad
// is not null); the embedding backward skips them.
constexpr uint32_t ID_BAD_INPUT = 1u, ID_BAD_TARGET = 2u;
hipError_t launch_embed_fwd(const int32_t* ids, const float* wte, const float* wpe, bf16_t* x, int B,
                            int T, int C, int V, uint32_t* bad, hipStream_t s);
// dwte[ids[r]] += dx[r] (fp32 atomics; adds to what is there)
hipError_t launch_embed_bwd(const int32_t* ids, const bf16_t* dx, float* dwte, int B, int T, int C, int V,
                            hipStream_t s);
// dwpe[t] = (accumulate ? dwpe[t] : 0) + sum_b dx[b, t] for t < T; rows T..Tmax-1 get 0 added
hipError_t launch_embed_bwd_pos(const bf16_t* dx, float* dwpe, int B, int T, int Tmax, int C,
                                int accumulate, hipStream_t s);

// fused softmax cross-entropy over the first V of Vp columns; dlogits
// (scaled) overwrite the logits; losses fp32 [rows]
// write_grad: overwrite the logits with dlogits (training) or leave them
hipError_t launch_cross_entropy(bf16_t* logits, const int32_t* targets, float* losses, int rows, int V, int Vp,
                                float grad_scale, int write_grad, uint32_t* bad, hipStream_t s);
// mean of n floats into out[0] (single block, fixed order); with flag (not
// null), also moves *flag into out[1] (its bits) and clears *flag
hipError_t launch_mean(const float* x, int n, float* out, hipStream_t s, uint32_t* flag = nullptr);
// out[0] = scale * sum of x[0..n)
hipError_t launch_sum_scaled(const float* x, int n, float scale, float* out, hipStream_t s);
// Cross-entropy over the rows of the positions that carry loss (t >= mask_from
// of every T): logits row i (of rows = B (T - mask_from)) belongs to position
// p = (i / n) T + mask_from + i % n, n = T - mask_from, whose target and loss
// are targets[p] and losses[p]; the losses of the other positions are set to 0.
hipError_t launch_cross_entropy_masked(bf16_t* logits, const int32_t* targets, float* losses, int rows, int V, int Vp,
                                       float grad_scale, int write_grad, int T, int mask_from, hipStream_t s,
                                       uint32_t* bad = nullptr);

// ---------------------------------------------------------------- Qwen3-shaped adapter step
hipError_t launch_embed_gather(const int32_t* ids, const bf16_t* table, bf16_t* x, long rows, int C, hipStream_t s);
// y = x / sqrt(mean(x^2) + eps) * w per row; rstd [rows] saved. Only the rows
// of positions t >= mask_from of every T are normalised: output row i (of
// rows = B (T - mask_from)) is input row (i / n) T + mask_from + i % n,
// n = T - mask_from (mask_from = 0: every row, in place order).
hipError_t launch_rmsnorm_fwd(const bf16_t* x, const bf16_t* w, bf16_t* y, float* rstd, int rows, int C, float eps,
                              int T, int mask_from, hipStream_t s);
// dres (=|+=) the RMSNorm input gradient (the gain is frozen) over all rows of
// x; dy and rstd hold only the rows of positions t >= mask_from, compacted as
// launch_rmsnorm_fwd writes them; the other rows get a zero gradient
hipError_t launch_rmsnorm_bwd(const bf16_t* dy, const bf16_t* x, const float* rstd, const bf16_t* w, bf16_t* dres,
                              int accumulate, int rows, int C, int T, int mask_from, hipStream_t s);
// raw q|k|v [BT][(H + 2 Hkv) hd] -> packed q|k|v in the same layout for the
// grouped-query attention kernels: query and key heads RMS-normalised and
// rotated, value heads copied; rstd of every q and k head saved
hipError_t launch_qknorm_rope_fwd(const bf16_t* raw, const bf16_t* qn_w, const bf16_t* kn_w, const float* cosT,
                                  const float* sinT, bf16_t* packed, float* rq, float* rk, int BT, int T, int H, int Hkv,
                                  int hd, float eps, hipStream_t s);
hipError_t launch_qknorm_rope_bwd(const bf16_t* dpacked, const bf16_t* raw, const bf16_t* qn_w, const bf16_t* kn_w,
                                  const float* cosT, const float* sinT, const float* rq, const float* rk, bf16_t* draw,
                                  int BT, int T, int H, int Hkv, int hd, hipStream_t s);
// m = silu(g) * u over gu = [g | u] ([rows][2F]); and the gradient pair
hipError_t launch_swiglu_fwd(const bf16_t* gu, bf16_t* m, long rows, int F, hipStream_t s);
hipError_t launch_swiglu_bwd(const bf16_t* dm, const bf16_t* gu, bf16_t* dgu, long rows, int F, hipStream_t s);
// Adapter products that stream a tall operand once (lora.hip): for segments
// q < nseg and tiles t < nts of 16 columns,
//   y[m][col[q] + tr(t) + c] = s * sum_{k < klen[q]} x[m][k0[q] + k] * w[q][(tr(t) + c) * ldw + k]
// with tr(t) = (t / ntp) * tstride + 16 * (t % ntp), m < M, c < 16; every
// other column of y's rows [0, ldy) is written as 0. klen multiples of 64,
// ntp 1 or 2, nseg <= 3, nts / ntp <= 3.
struct LoraRowArgs {
  const bf16_t* x;
  long ldx;
  int M;
  int nseg, nts, ntp, tstride;
  int k0[3], klen[3], col[3];
  const bf16_t* w[3];
  long ldw;
  float s;
  bf16_t* y;
  int ldy;
};
hipError_t launch_lora_rows(const LoraRowArgs& a, hipStream_t s);
// Bt[l][c][k] = B[l][k][c] for l < L, c < 32, k < out (B rows of rp >= 32
// elements, out a multiple of 64): the adapter B matrices with the
// contraction index contiguous, for launch_lora_rows.
hipError_t launch_lora_bt(const bf16_t* B, bf16_t* Bt, int L, int out, int rp, hipStream_t s);
// x[r][c] *= sc for r < rows, c < cols (row stride ld)
hipError_t launch_scale_bf16(bf16_t* x, long rows, int cols, int ld, float sc, hipStream_t s);

// fp32 -> bf16 copy of n elements (n % 4 == 0)
hipError_t launch_cast_bf16(const float* src, bf16_t* dst, long n, hipStream_t s);

// Seeded initialisation of a flat fp32 parameter buffer from the counter-based
// generator Philox4x32-10 (Salmon et al., SC 2011): element i takes counter
// (i mod 2^32, i div 2^32, 0, 0) and key (key0, key1); its first two output
// words give a standard normal by the Box-Muller transform (in fp64). Element
// i of segment k (ending at end[k], exclusive) becomes std[k] * normal when
// std[k] > 0, else fill[k]; elements in [zero_lo, zero_hi) become 0. Adam
// moments m, v are cleared and the bf16 copy written. n % 4 == 0.
struct InitArgs {
  float* p;
  float* m;
  float* v;
  bf16_t* p_bf16;
  long n;
  long end[16];
  double std[16];
  float fill[16];
  int count;
  long zero_lo, zero_hi;
  uint32_t key0, key1;
};
hipError_t launch_init_params(const InitArgs& a, hipStream_t s);

// ---------------------------------------------------------------- optimizer
int sumsq_parts();
hipError_t launch_sumsq(const float* g, long n, float* parts, hipStream_t s);
// norm = sqrt(sum parts); coef = clip/norm if norm > clip else 1
hipError_t launch_clip_coef(const float* parts, int nparts, float clip, float* norm_coef,
                            hipStream_t s);

struct AdamSegments {
  long end[16];    // exclusive end offset (elements) of each segment
  int decay[16];   // 1 where weight decay applies
  int count;
};
struct AdamArgs {
  float* p;
  const float* g;
  float* m;
  float* v;
  bf16_t* p_bf16;
  const float* norm_coef;  // [0] norm, [1] clip coefficient
  long n;
  float lr, beta1, beta2, eps, weight_decay;
  float bc1, bc2;          // 1 - beta^t
  AdamSegments seg;
};
hipError_t launch_adamw(const AdamArgs& a, hipStream_t s);

// ---------------------------------------------------------------- no-alloc scratch
// Floats of the static scratch array the allocation-free entry points use
// (the optimizer's sum-of-squares partials, then its norm and clip
// coefficient): 16 KiB per GPU.
constexpr int NOALLOC_SCRATCH_FLOATS = 4096;
// Device address of the current device's copy of the array (looked up on the
// first call per device, with that device current).
hipError_t noalloc_scratch(float** out);
