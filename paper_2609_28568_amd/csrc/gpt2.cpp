// Host side of the GPT-2 training-step library: configuration checks, the
// layout of the caller-owned buffers, and the per-layer launch sequence of the
// forward pass, the backward pass and the optimizer step. Every launch goes
// to the stream given at init; nothing here allocates device memory.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <algorithm>
#include <string>
#include <vector>

#include "../../include/gpt2.h"
#include "kernels.h"
#include "probe.h"

namespace {

enum Kind {
  K_WTE, K_WPE, K_LN1W, K_LN1B, K_QKVW, K_QKVB, K_ATTPROJW, K_ATTPROJB,
  K_LN2W, K_LN2B, K_FCW, K_FCB, K_FCPROJW, K_FCPROJB, K_LNFW, K_LNFB, K_NKIND
};

constexpr size_t ALIGN = 256;
size_t align_up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

struct Dims {
  int L, H, C, F, V, Vp, Tmax, B, T, hd, accum;
  long BT;
};

Dims dims_of(const gpt2_config& c) {
  Dims d;
  d.L = c.n_layer; d.H = c.n_head; d.C = c.d_model; d.F = c.d_ff; d.V = c.vocab;
  d.Vp = c.vocab_padded; d.Tmax = c.max_seq_len; d.B = c.B; d.T = c.T;
  d.hd = c.n_head > 0 ? c.d_model / c.n_head : 0; d.accum = c.grad_accum;
  d.BT = (long)c.B * c.T;
  return d;
}

const char* validate(const gpt2_config* c) {
  if (!c) return "config is NULL";
  if (c->n_layer < 1) return "n_layer must be >= 1";
  if (c->n_head < 1 || c->d_model % c->n_head) return "d_model must be a multiple of n_head";
  int hd = c->d_model / c->n_head;
  if (hd != 16 && hd != 32 && hd != 64 && hd != 128) return "head_dim must be 16, 32, 64 or 128";
  if (c->d_model % 64 || c->d_model > 2048) return "d_model must be a multiple of 64 and <= 2048";
  if (c->d_ff % 64 || c->d_ff < 64) return "d_ff must be a positive multiple of 64";
  if (c->vocab < 1 || c->vocab_padded < c->vocab) return "need 1 <= vocab <= vocab_padded";
  if (c->vocab_padded % 64 || c->vocab_padded > 65536) return "vocab_padded must be a multiple of 64, <= 65536";
  if (c->max_seq_len < 1 || c->T < 1 || c->T > c->max_seq_len) return "need 1 <= T <= max_seq_len";
  if (c->B < 1) return "B must be >= 1";
  if ((long)c->B * c->T > (1L << 26)) return "B*T too large";
  {
    // kernels address each [B*T, width] operand (plus up to 256 rows of tile
    // overhang) with 32-bit byte offsets
    const long wide = std::max({(long)c->vocab_padded, 3L * c->d_model, (long)c->d_ff});
    if (((long)c->B * c->T + 256) * wide * 2 >= (1L << 32))
      return "B*T too large: a [B*T, max(vocab_padded, 3*d_model, d_ff)] bf16 operand must stay below 4 GiB";
  }
  if (c->grad_accum < 1) return "grad_accum must be >= 1";
  if (!(c->ln_eps > 0.0f)) return "ln_eps must be > 0";
  if (c->warmup_steps < 1 || c->total_steps <= c->warmup_steps) return "need 1 <= warmup_steps < total_steps";
  if (!(c->beta1 >= 0.0f && c->beta1 < 1.0f && c->beta2 >= 0.0f && c->beta2 < 1.0f)) return "betas must be in [0,1)";
  if (!(c->adam_eps > 0.0f) || !(c->grad_clip > 0.0f)) return "adam_eps and grad_clip must be > 0";
  return nullptr;
}

// element counts of each parameter kind, in flat-buffer order
void kind_sizes(const Dims& d, size_t n[K_NKIND]) {
  size_t L = d.L, C = d.C, F = d.F;
  n[K_WTE] = (size_t)d.Vp * C; n[K_WPE] = (size_t)d.Tmax * C;
  n[K_LN1W] = n[K_LN1B] = L * C;
  n[K_QKVW] = L * 3 * C * C; n[K_QKVB] = L * 3 * C;
  n[K_ATTPROJW] = L * C * C; n[K_ATTPROJB] = L * C;
  n[K_LN2W] = n[K_LN2B] = L * C;
  n[K_FCW] = L * F * C; n[K_FCB] = L * F;
  n[K_FCPROJW] = L * C * F; n[K_FCPROJB] = L * C;
  n[K_LNFW] = n[K_LNFB] = C;
}
const bool kDecay[K_NKIND] = {true, true, false, false, true, false, true, false,
                              false, false, true, false, true, false, false, false};

// contraction splits for a weight-gradient GEMM with an M x N output
// output tiles of the weight-gradient GEMM (the tile shape gemm.hip picks)
long dw_tiles(int M, int N) {
  const GemmConfig c = gemm_config(M, N, 1, 1, EPI_F32);
  return (long)((M + c.bm - 1) / c.bm) * ((N + c.bn - 1) / c.bn);
}

// Split the token contraction of a weight gradient when its tiles alone
// would leave CUs idle: 8 splits (one per XCD) or 16, each at least 512
// tokens long.
int dw_want(const Dims& d, int M, int N) {
  const long tiles = dw_tiles(M, N);
  if (tiles >= 256) return 1;
  int want = tiles * 8 >= 256 ? 8 : 16;
  while (want > 1 && d.BT / want < 512) want /= 2;
  return want;
}

int dw_splits(const Dims& d, int M, int N) {
  return gemm_split_plan((int)d.BT, dw_want(d, M, N), nullptr);
}

int dw_chunk(const Dims& d, int M, int N) {
  int kc = 0;
  gemm_split_plan((int)d.BT, dw_want(d, M, N), &kc);
  return kc;
}

// An unsplit weight gradient runs in rounds of 512 tiles (two workgroups per
// CU). When its last round would be at most half full, only the whole rounds
// (the first m_main rows) run unsplit, and the remaining rows take a
// contraction split sized to fill the chip, reduced afterwards. Used only
// when the remaining rows are a whole number of their own tiles, so no
// operand read leaves the matrices.
struct DwTail {
  int m_main;   // rows computed unsplit (M when there is no tail split)
  int splits;   // contraction splits of rows [m_main, M)
  int chunk;    // tokens per split
};

DwTail dw_tail(const Dims& d, int M, int N) {
  DwTail t{M, 1, 0};
  constexpr long ROUND = 512;
  const GemmConfig c = gemm_config(M, N, 1, 1, EPI_F32);
  const long tm = (M + c.bm - 1) / c.bm, tn = (N + c.bn - 1) / c.bn, tiles = tm * tn;
  if (tiles < ROUND || tiles % ROUND == 0 || tiles % ROUND > ROUND / 2 || ROUND % tn != 0) return t;
  if (M % c.bm != 0 || N % c.bn != 0) return t;
  const int m_main = (int)(tiles / ROUND * ROUND / tn) * c.bm;
  const int m_rest = M - m_main;
  const GemmConfig cr = gemm_config(m_rest, N, 1, 1, EPI_F32);
  if (m_rest % cr.bm != 0 || N % cr.bn != 0) return t;
  const long rest_tiles = (long)(m_rest / cr.bm) * (N / cr.bn);
  int want = (int)(ROUND / rest_tiles);
  while (want > 1 && d.BT / want < 512) --want;
  if (want < 2) return t;
  t.m_main = m_main;
  t.splits = gemm_split_plan((int)d.BT, want, &t.chunk);
  return t;
}

struct ActLayout {
  size_t residual, ln1, ln1_mean, ln1_rstd, qkv, att, lse, x_mid, ln2, ln2_mean, ln2_rstd, fc, gelu;
  size_t lnf, lnf_mean, lnf_rstd, logits, losses, loss_mean, ids, total;
  // per-layer strides in bytes
  size_t s_act, s_qkv, s_ff, s_row, s_lse;
};

struct WsLayout {
  size_t dres, dh, datt, dbig, dsum, splitk, bsum, lnpart, sumsq, normcoef, total;
  size_t splitk_elems, bsum_elems, s_lnpart;
  // the training backward keeps every layer's output gradients until one
  // grouped launch computes all block weight gradients: residual-stream
  // gradients [2L+1][BT][C] (slot 2l+2 enters block l, 2l+1 is after its MLP
  // branch, 2l leaves it), MLP pre-activation gradients [L][BT][F], q|k|v
  // gradients [L][BT][3C], and the bias partial sums of the q|k|v and MLP-up
  // groups
  size_t dres_l, dfc_l, dqkv_l, gbs_qkv, gbs_fc;
  size_t s_dres, s_dfc, s_dqkv;
  // the two-pass head + cross-entropy: per-row softmax statistics of every
  // head tile slice, the target logits and the log-sum-exp of each row
  size_t ce_stats, ce_tlogit, ce_lse;
};

ActLayout act_layout(const Dims& d) {
  ActLayout a{};
  const size_t BT = d.BT, C = d.C, L = d.L;
  a.s_act = align_up(BT * C * 2);
  a.s_qkv = align_up(BT * 3 * C * 2);
  a.s_ff = align_up(BT * d.F * 2);
  a.s_row = align_up(BT * 4);
  a.s_lse = align_up((size_t)d.B * d.H * d.T * 4);
  size_t o = 0;
  a.residual = o; o += (L + 1) * a.s_act;
  a.ln1 = o; o += L * a.s_act;
  a.ln1_mean = o; o += L * a.s_row;
  a.ln1_rstd = o; o += L * a.s_row;
  a.qkv = o; o += L * a.s_qkv;
  a.att = o; o += L * a.s_act;
  a.lse = o; o += L * a.s_lse;
  a.x_mid = o; o += L * a.s_act;
  a.ln2 = o; o += L * a.s_act;
  a.ln2_mean = o; o += L * a.s_row;
  a.ln2_rstd = o; o += L * a.s_row;
  a.fc = o; o += L * a.s_ff;
  a.gelu = o; o += L * a.s_ff;
  a.lnf = o; o += a.s_act;
  a.lnf_mean = o; o += a.s_row;
  a.lnf_rstd = o; o += a.s_row;
  a.logits = o; o += align_up(BT * (size_t)d.Vp * 2);
  a.losses = o; o += a.s_row;
  a.loss_mean = o; o += ALIGN;
  a.ids = o; o += a.s_row;
  a.total = o;
  return a;
}

// The four groups of the grouped weight-gradient launch, shapes only (the
// pointers are filled in by the backward): q|k|v [3C, C], attention
// projection [C, C], MLP up [F, C], MLP down [C, F], each over the L layers.
enum { G_QKV, G_ATTPROJ, G_FC, G_FCPROJ };
GemmGroupedArgs dw_groups(const Dims& d) {
  GemmGroupedArgs g{};
  g.ngroups = 4;
  g.K = (int)d.BT;
  const int mn[4][2] = {{3 * d.C, d.C}, {d.C, d.C}, {d.F, d.C}, {d.C, d.F}};
  for (int i = 0; i < 4; ++i) {
    g.grp[i].M = mn[i][0];
    g.grp[i].N = mn[i][1];
    g.grp[i].count = d.L;
  }
  return g;
}

// The grouped weight-gradient launch runs in rounds of 512 tiles (two
// workgroups on each of the 256 CUs). When its last round would be at most
// half full and consists of whole MLP-down products (the last group), those
// products split their token contraction into `splits` chunks, so that the
// final round is full of shorter work items; their fp32 slices are reduced
// afterwards. np = 0: no such plan.
struct DwGroupedTail {
  int np = 0, splits = 1, chunk = 0;
  long nfull = 0;
};

DwGroupedTail dw_grouped_tail(const Dims& d) {
  DwGroupedTail t;
  constexpr long ROUND = 512;
  const GemmGroupedArgs g = dw_groups(d);
  int bm = 192;
  for (int i = 0; i < g.ngroups; ++i)
    if (g.grp[i].M % 192 || g.grp[i].N % 192) bm = 128;
  long total = 0;
  for (int i = 0; i < g.ngroups; ++i) total += (long)((g.grp[i].M + bm - 1) / bm) * ((g.grp[i].N + bm - 1) / bm) * g.grp[i].count;
  const GemmGroup& last = g.grp[G_FCPROJ];
  const long tpp = (long)((last.M + bm - 1) / bm) * ((last.N + bm - 1) / bm);
  const long tail = total % ROUND;
  if (total < ROUND || tail == 0 || tail > ROUND / 2 || tail % tpp || tail / tpp > last.count) return t;
  int splits = (int)(ROUND / tail);
  if (splits > 4) splits = 4;
  int chunk = 0;
  splits = gemm_split_plan((int)d.BT, splits, &chunk);
  if (splits < 2 || ((tail * splits) % 8) != 0) return t;
  t.np = (int)(tail / tpp);
  t.splits = splits;
  t.chunk = chunk;
  t.nfull = total - tail;
  return t;
}

WsLayout ws_layout(const Dims& d) {
  WsLayout w{};
  const size_t BT = d.BT, C = d.C, F = d.F;
  size_t wide = F > 3 * C ? F : 3 * C;
  size_t sk = 0;
  auto upd = [&](int M, int N) {
    int s = dw_splits(d, M, N);
    if (s > 1) sk = std::max(sk, (size_t)s * M * N);
    const DwTail t = dw_tail(d, M, N);
    if (t.splits > 1) sk = std::max(sk, (size_t)t.splits * (M - t.m_main) * N);
  };
  upd(3 * d.C, d.C); upd(d.C, d.C); upd(d.F, d.C); upd(d.C, d.F); upd(d.Vp, d.C);
  const DwGroupedTail gt = dw_grouped_tail(d);
  if (gt.np > 0) sk = std::max(sk, (size_t)gt.splits * gt.np * d.C * d.F);
  w.splitk_elems = sk;
  // bias partial sums of the weight gradients that carry a bias gradient
  size_t bs = 0;
  auto bupd = [&](int M, int N) {
    const int s = dw_splits(d, M, N);
    bs = std::max(bs, (size_t)gemm_bias_parts(M, N, s) * M);
  };
  bupd(3 * d.C, d.C); bupd(d.F, d.C); bupd(d.C, d.F);
  w.bsum_elems = bs;
  size_t o = 0;
  w.dres = o; o += align_up(BT * C * 2);
  w.dh = o; o += align_up(BT * C * 2);
  w.datt = o; o += align_up(BT * C * 2);
  w.dbig = o; o += align_up(BT * wide * 2);
  w.dsum = o; o += align_up((size_t)d.B * d.H * d.T * 4);
  w.splitk = o; o += align_up(sk * 4);
  w.bsum = o; o += align_up(w.bsum_elems * 4);
  // LayerNorm backward partial sums: one slot per LayerNorm of the model
  // (2L + 1), so that the training backward reduces them all in one launch
  w.s_lnpart = align_up((size_t)layernorm_bwd_blocks((int)BT) * 3 * C * 4);
  w.lnpart = o; o += (2 * (size_t)d.L + 1) * w.s_lnpart;
  w.sumsq = o; o += align_up((size_t)sumsq_parts() * 4);
  w.normcoef = o; o += ALIGN;
  w.s_dres = align_up(BT * C * 2);
  w.s_dfc = align_up(BT * F * 2);
  w.s_dqkv = align_up(BT * 3 * C * 2);
  w.dres_l = o; o += (2 * (size_t)d.L + 1) * w.s_dres;
  w.dfc_l = o; o += (size_t)d.L * w.s_dfc;
  w.dqkv_l = o; o += (size_t)d.L * w.s_dqkv;
  const GemmGroupedArgs gg = dw_groups(d);
  w.gbs_qkv = o; o += align_up((size_t)gemm_grouped_bias_parts(gg, G_QKV) * d.L * 3 * C * 4);
  w.gbs_fc = o; o += align_up((size_t)gemm_grouped_bias_parts(gg, G_FC) * d.L * F * 4);
  w.ce_stats = o; o += align_up(BT * (size_t)gemm_ce_parts((int)BT, d.Vp) * 8);
  w.ce_tlogit = o; o += align_up(BT * 4);
  w.ce_lse = o; o += align_up(BT * 4);
  w.total = o;
  return w;
}

}  // namespace

struct gpt2_model {
  gpt2_config cfg;
  Dims d;
  gpt2_buffers buf;
  hipStream_t stream;
  size_t kn[K_NKIND], koff[K_NKIND], n_params;
  ActLayout act;
  WsLayout ws;
  bool have_dlogits = false;   // last forward had targets
  bool have_grads = false;     // gradients hold a backward result
  bool have_loss = false;
  // how a residual connection meets the following pre-norm (gpt2_fusion):
  // 0 the projection's epilogue adds the residual, the LayerNorm reads the
  // sum; 1 the projection writes its branch and one kernel adds and
  // normalises; 2 a separate addition kernel, then the LayerNorm (the
  // composed path that 1 must match bit for bit)
  int residual_norm = 0;
  // the LM head and the cross-entropy (gpt2_fusion): 0 the head GEMM writes
  // the logits and one kernel computes loss and dlogits over them; 1 the head
  // GEMM runs twice, first writing only each row's softmax statistics and
  // target logit, then writing dlogits from the combined log-sum-exp
  int head_ce = 0;
  // LayerNorm backward reductions left for one launch at the end of the
  // training backward (their partial sums each in a slot of their own)
  ReducePartsJobs ln_jobs{};
  int ln_jobs_acc = 0;
  std::string err;
  ProbeSet<GPT2_K_COUNT> probes;

  // typed pointers
  float* pf(int k) { return static_cast<float*>(buf.params_f32) + koff[k]; }
  float* gf(int k) { return static_cast<float*>(buf.grads_f32) + koff[k]; }
  bf16_t* pb(int k) { return static_cast<bf16_t*>(buf.params_bf16) + koff[k]; }
  char* A(size_t off) { return static_cast<char*>(buf.activations) + off; }
  char* W(size_t off) { return static_cast<char*>(buf.workspace) + off; }
  bf16_t* res(int l) { return reinterpret_cast<bf16_t*>(A(act.residual + l * act.s_act)); }
  bf16_t* ln1(int l) { return reinterpret_cast<bf16_t*>(A(act.ln1 + l * act.s_act)); }
  float* ln1m(int l) { return reinterpret_cast<float*>(A(act.ln1_mean + l * act.s_row)); }
  float* ln1r(int l) { return reinterpret_cast<float*>(A(act.ln1_rstd + l * act.s_row)); }
  bf16_t* qkv(int l) { return reinterpret_cast<bf16_t*>(A(act.qkv + l * act.s_qkv)); }
  bf16_t* att(int l) { return reinterpret_cast<bf16_t*>(A(act.att + l * act.s_act)); }
  float* lse(int l) { return reinterpret_cast<float*>(A(act.lse + l * act.s_lse)); }
  bf16_t* xmid(int l) { return reinterpret_cast<bf16_t*>(A(act.x_mid + l * act.s_act)); }
  bf16_t* ln2(int l) { return reinterpret_cast<bf16_t*>(A(act.ln2 + l * act.s_act)); }
  float* ln2m(int l) { return reinterpret_cast<float*>(A(act.ln2_mean + l * act.s_row)); }
  float* ln2r(int l) { return reinterpret_cast<float*>(A(act.ln2_rstd + l * act.s_row)); }
  bf16_t* fc(int l) { return reinterpret_cast<bf16_t*>(A(act.fc + l * act.s_ff)); }
  bf16_t* gelu(int l) { return reinterpret_cast<bf16_t*>(A(act.gelu + l * act.s_ff)); }
  bf16_t* lnf() { return reinterpret_cast<bf16_t*>(A(act.lnf)); }
  float* lnfm() { return reinterpret_cast<float*>(A(act.lnf_mean)); }
  float* lnfr() { return reinterpret_cast<float*>(A(act.lnf_rstd)); }
  bf16_t* logits() { return reinterpret_cast<bf16_t*>(A(act.logits)); }
  float* losses() { return reinterpret_cast<float*>(A(act.losses)); }
  // loss_mean()[0]: mean loss; [1]: the id-range flag bits moved there with it
  float* loss_mean() { return reinterpret_cast<float*>(A(act.loss_mean)); }
  // live id-range flag (bits ID_BAD_INPUT, ID_BAD_TARGET), in the same slot
  uint32_t* id_flag() { return reinterpret_cast<uint32_t*>(A(act.loss_mean + 64)); }
  int32_t* ids() { return reinterpret_cast<int32_t*>(A(act.ids)); }
  bf16_t* wsb(size_t off) { return reinterpret_cast<bf16_t*>(W(off)); }
  float* wsf(size_t off) { return reinterpret_cast<float*>(W(off)); }

  gpt2_status fail(gpt2_status s, const std::string& msg) {
    err = msg;
    return s;
  }

  // Launch through f(); optionally bracket it with events for the probes.
  template <class Fn>
  hipError_t run(int cls, double fl, double by, Fn f) {
    return probes.run(stream, cls, fl, by, f);
  }
};

namespace {

#define TRY(expr)                                                                     \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess)                                                             \
      return m->fail(GPT2_ERR_DEVICE, std::string("HIP error at ") + #expr + ": " +  \
                                          hipGetErrorString(e_));                     \
  } while (0)

using Model = gpt2_model;

int gemm_class(int a_t, int b_t, int epi) {
  if (a_t) return GPT2_K_GEMM_DW;
  if (b_t) return epi == EPI_GELU_BWD ? GPT2_K_GEMM_DX_GELU : GPT2_K_GEMM_DX;
  return epi == EPI_GELU ? GPT2_K_GEMM_FWD_GELU : GPT2_K_GEMM_FWD;
}

hipError_t gemm(Model* m, int cls, int M, int N, int K, const bf16_t* A, int lda, int a_t, const bf16_t* B,
                int ldb, int b_t, int epi, void* C, int ldc, const float* bias = nullptr,
                const bf16_t* residual = nullptr, bf16_t* C2 = nullptr, const bf16_t* aux = nullptr,
                int accumulate = 0, int splits = 1, long split_stride = 0, int k_chunk = 0, double alg_flops = 0.0,
                float* bsum = nullptr) {
  GemmArgs g{};
  g.A = A; g.B = B; g.M = M; g.N = N; g.K = K; g.lda = lda; g.ldb = ldb;
  g.C = C; g.ldc = ldc; g.bias = bias; g.residual = residual; g.C2 = C2; g.aux = aux;
  g.accumulate = accumulate; g.splits = splits; g.split_stride = split_stride; g.k_chunk = k_chunk;
  g.bsum = bsum;
  // algorithmic FLOPs: the tied head passes its count over the real vocabulary
  // only (the padded columns are computed but carry no probability)
  const double fl = alg_flops > 0.0 ? alg_flops : 2.0 * M * N * K;
  (void)cls;
  return m->run(gemm_class(a_t, b_t, epi), fl, 0.0, [&] { return launch_gemm(g, a_t, b_t, epi, m->stream); });
}

// weight gradient dW[M][N] (=|+=) sum_t A[t][m] * X[t][n] (fp32); with db,
// also the bias gradient db[M] (=|+=) sum_t A[t][m], summed by the GEMM from
// the A fragments it reads and reduced together with its contraction split
hipError_t weight_grad(Model* m, int M, int N, const bf16_t* dy, const bf16_t* x, float* dW, int accumulate,
                       int m_real = 0, float* db = nullptr) {
  const int BT = (int)m->d.BT;
  const int mr = m_real ? m_real : M;
  const double fl = 2.0 * mr * (double)N * BT;
  int s = dw_splits(m->d, M, N);
  float* bp = db ? m->wsf(m->ws.bsum) : nullptr;
  if (s <= 1) {
    const DwTail t = dw_tail(m->d, M, N);
    if (t.splits <= 1 || db) {
      hipError_t e = gemm(m, GPT2_K_GEMM_DW, M, N, BT, dy, M, 1, x, N, 1, EPI_F32, dW, N, nullptr, nullptr, nullptr,
                          nullptr, accumulate, 1, 0, 0, fl, bp);
      if (e != hipSuccess || !db) return e;
      const int np = gemm_bias_parts(M, N, 1);
      return m->run(GPT2_K_OTHER, 0.0, 4.0 * (double)M * (np + 1 + accumulate),
                    [&] { return launch_reduce_slices(bp, np, M, db, accumulate, m->stream); });
    }
    // whole rounds unsplit, the rest split over tokens and reduced
    const int m0 = t.m_main, m1 = M - t.m_main;
    const double fl0 = 2.0 * std::min(mr, m0) * (double)N * BT, fl1 = fl - fl0;
    hipError_t e = gemm(m, GPT2_K_GEMM_DW, m0, N, BT, dy, M, 1, x, N, 1, EPI_F32, dW, N, nullptr, nullptr, nullptr,
                        nullptr, accumulate, 1, 0, 0, fl0);
    if (e != hipSuccess) return e;
    float* part = m->wsf(m->ws.splitk);
    e = gemm(m, GPT2_K_GEMM_DW, m1, N, BT, dy + m0, M, 1, x, N, 1, EPI_F32, part, N, nullptr, nullptr, nullptr,
             nullptr, 0, t.splits, (long)m1 * N, t.chunk, fl1);
    if (e != hipSuccess) return e;
    float* dW1 = dW + (size_t)m0 * N;
    return m->run(GPT2_K_OTHER, 0.0, 4.0 * (double)m1 * N * (t.splits + 1 + accumulate),
                  [&] { return launch_reduce_slices(part, t.splits, (long)m1 * N, dW1, accumulate, m->stream); });
  }
  float* part = m->wsf(m->ws.splitk);
  hipError_t e = gemm(m, GPT2_K_GEMM_DW, M, N, BT, dy, M, 1, x, N, 1, EPI_F32, part, N, nullptr, nullptr, nullptr,
                      nullptr, 0, s, (long)M * N, dw_chunk(m->d, M, N), fl, bp);
  if (e != hipSuccess) return e;
  if (!db)
    return m->run(GPT2_K_OTHER, 0.0, 4.0 * (double)M * N * (s + 1 + accumulate),
                  [&] { return launch_reduce_slices(part, s, (long)M * N, dW, accumulate, m->stream); });
  const int np = gemm_bias_parts(M, N, s);
  return m->run(GPT2_K_OTHER, 0.0, 4.0 * ((double)M * N * (s + 1 + accumulate) + (double)M * (np + 1 + accumulate)),
                [&] {
                  return launch_reduce_slices2(part, s, (long)M * N, dW, bp, np, M, db, accumulate, m->stream);
                });
}

hipError_t ln_fwd(Model* m, const bf16_t* x, const float* w, const float* b, bf16_t* y, float* mean, float* rstd) {
  const int BT = (int)m->d.BT, C = m->d.C;
  return m->run(GPT2_K_LAYERNORM, 0.0, 4.0 * BT * C + 8.0 * BT + 8.0 * C,
                [&] { return launch_layernorm_fwd(x, w, b, y, mean, rstd, BT, C, m->cfg.ln_eps, m->stream); });
}

// LayerNorm backward into the residual-stream gradient: dres_out = (has_res ?
// dres_in : 0) + dx; also writes the gain and shift gradients and, when dbias
// is given, the column sum of the new residual gradient (the bias gradient of
// the projection that produced it).
// The queued LayerNorm backward reductions, in one launch.
hipError_t reduce_ln_parts(Model* m) {
  ReducePartsJobs& J = m->ln_jobs;
  if (J.count == 0) return hipSuccess;
  const int C = m->d.C, nb = layernorm_bwd_blocks((int)m->d.BT), acc = m->ln_jobs_acc;
  hipError_t e = m->run(GPT2_K_OTHER, 0.0, 4.0 * 3 * C * (double)J.count * (nb + 1 + acc), [&] {
    return launch_reduce_parts_multi(J, nb, 3L * C, C, 3, acc, m->stream);
  });
  J.count = 0;
  return e;
}

// With slot >= 0 the partial sums go to that slot and their reduction is
// queued for reduce_ln_parts; otherwise they are reduced at once.
hipError_t ln_bwd(Model* m, const bf16_t* dy, const bf16_t* x, const float* mean, const float* rstd, const float* w,
                  const bf16_t* dres_in, bf16_t* dres_out, int has_res, float* dw, float* db, float* dbias,
                  int accumulate, int slot = -1) {
  const int BT = (int)m->d.BT, C = m->d.C;
  float* part = m->wsf(m->ws.lnpart + (size_t)(slot < 0 ? 0 : slot) * m->ws.s_lnpart);
  hipError_t e = m->run(GPT2_K_LAYERNORM, 0.0, 2.0 * BT * C * (3 + has_res) + 8.0 * BT, [&] {
    return launch_layernorm_bwd(dy, x, mean, rstd, w, dres_in, dres_out, has_res, part, BT, C, m->stream);
  });
  if (e != hipSuccess) return e;
  if (slot >= 0) {
    ReducePartsJobs& J = m->ln_jobs;
    if (J.count == REDUCE_JOBS || (J.count > 0 && m->ln_jobs_acc != accumulate)) {
      e = reduce_ln_parts(m);
      if (e != hipSuccess) return e;
    }
    J.part[J.count] = part;
    J.d[J.count][0] = dw;
    J.d[J.count][1] = db;
    J.d[J.count][2] = dbias;
    ++J.count;
    m->ln_jobs_acc = accumulate;
    return hipSuccess;
  }
  int nb = layernorm_bwd_blocks(BT);
  return m->run(GPT2_K_OTHER, 0.0, 4.0 * 3 * C * (nb + 1 + accumulate), [&] {
    return launch_reduce_parts(part, nb, 3L * C, C, 3, dw, db, dbias, accumulate, m->stream);
  });
}


AttnArgs attn_args(Model* m, int slot, bf16_t* dqkv = nullptr) {
  AttnArgs a{};
  a.B = m->d.B; a.T = m->d.T; a.H = m->d.H; a.hd = m->d.hd;
  a.qkv = m->qkv(slot); a.out = m->att(slot); a.lse = m->lse(slot);
  a.dout = m->wsb(m->ws.datt); a.dsum = m->wsf(m->ws.dsum); a.dqkv = dqkv ? dqkv : m->wsb(m->ws.dbig);
  return a;
}

double attn_fwd_flops(const Dims& d) {
  // causal: q.k and p.v over the key positions j <= i only
  return 4.0 * d.B * d.H * d.hd * ((double)d.T * (d.T + 1) / 2.0);
}

// The tied LM head and the softmax cross-entropy over the real vocabulary
// (sections "Model" and "Optimisation and precision"), with targets:
// per-token losses, and (write_grad) dlogits scaled by grad_scale in the
// logits buffer. mode 0: the head writes the logits, the cross-entropy
// kernel reads them and writes dlogits over them; mode 1: a statistics pass
// of the head GEMM, a combine kernel, and (write_grad) a second head GEMM
// whose epilogue writes dlogits; the logits are never stored. Training takes
// the configured head_ce; the forward-only evaluation always takes mode 1,
// which needs only the statistics pass there.
gpt2_status head_and_loss(Model* m, const int32_t* d_targets, float grad_scale, int write_grad, int mode) {
  const Dims& d = m->d;
  const int BT = (int)d.BT, C = d.C;
  const double head_fl = 2.0 * BT * (double)d.V * C;
  if (mode == 0) {
    TRY(gemm(m, GPT2_K_GEMM_FWD, BT, d.Vp, C, m->lnf(), C, 0, m->pb(K_WTE), C, 0, EPI_BF16, m->logits(), d.Vp,
             nullptr, nullptr, nullptr, nullptr, 0, 1, 0, 0, head_fl));
    TRY(m->run(GPT2_K_CROSS_ENTROPY, 0.0, (2.0 + 2.0 * write_grad) * BT * d.Vp + 8.0 * BT, [&] {
      return launch_cross_entropy(m->logits(), d_targets, m->losses(), BT, d.V, d.Vp, grad_scale, write_grad,
                                  m->id_flag(), m->stream);
    }));
  } else {
    GemmArgs g{};
    g.A = m->lnf(); g.B = m->pb(K_WTE); g.M = BT; g.N = d.Vp; g.K = C; g.lda = C; g.ldb = C;
    g.C = m->logits(); g.ldc = d.Vp;
    g.ce_targets = d_targets; g.ce_stats = m->wsf(m->ws.ce_stats); g.ce_tlogit = m->wsf(m->ws.ce_tlogit);
    g.ce_lse = m->wsf(m->ws.ce_lse); g.ce_V = d.V; g.ce_scale = grad_scale;
    TRY(m->run(GPT2_K_GEMM_FWD, head_fl, 0.0, [&] { return launch_gemm(g, 0, 0, EPI_CE_STATS, m->stream); }));
    const int parts = gemm_ce_parts(BT, d.Vp);
    TRY(m->run(GPT2_K_CROSS_ENTROPY, 0.0, 8.0 * BT * parts + 16.0 * BT, [&] {
      return launch_ce_combine(g.ce_stats, parts, g.ce_tlogit, d_targets, d.V, m->wsf(m->ws.ce_lse), m->losses(), BT,
                               m->id_flag(), m->stream);
    }));
    if (write_grad)
      TRY(m->run(GPT2_K_GEMM_FWD, head_fl, 0.0, [&] { return launch_gemm(g, 0, 0, EPI_CE_GRAD, m->stream); }));
  }
  TRY(m->run(GPT2_K_OTHER, 0.0, 4.0 * BT,
             [&] { return launch_mean(m->losses(), BT, m->loss_mean(), m->stream, m->id_flag()); }));
  return GPT2_OK;
}

// The pre-norm that follows a residual connection: xsum = bf16(res +
// branch), y = LayerNorm(xsum), by the configured path (Model::residual_norm,
// modes 1 and 2; branch is the projection's output without the residual).
// With w == nullptr only the sum is formed.
hipError_t add_norm(Model* m, const bf16_t* res, const bf16_t* branch, bf16_t* xsum, const float* w, const float* b,
                    bf16_t* y, float* mean, float* rstd) {
  const int BT = (int)m->d.BT, C = m->d.C;
  if (m->residual_norm == 2 || !w) {
    hipError_t e = m->run(GPT2_K_OTHER, 0.0, 6.0 * BT * C,
                          [&] { return launch_residual_add(res, branch, xsum, (long)BT * C, m->stream); });
    if (e != hipSuccess || !w) return e;
    return ln_fwd(m, xsum, w, b, y, mean, rstd);
  }
  return m->run(GPT2_K_LAYERNORM, 0.0, 8.0 * BT * C + 8.0 * BT + 8.0 * C, [&] {
    return launch_add_layernorm_fwd(branch, res, xsum, w, b, y, mean, rstd, BT, C, m->cfg.ln_eps, m->stream);
  });
}

// The pre-norm that follows block l's output: the next block's LN1 (into
// activation slot a_next), or the final LayerNorm after the last block.
struct NextNorm {
  const float *w, *b;
  bf16_t* y;
  float *mean, *rstd;
};
NextNorm next_norm(Model* m, int l, int a_next) {
  if (l + 1 < m->d.L) {
    const size_t oC = (size_t)(l + 1) * m->d.C;
    return {m->pf(K_LN1W) + oC, m->pf(K_LN1B) + oC, m->ln1(a_next), m->ln1m(a_next), m->ln1r(a_next)};
  }
  return {m->pf(K_LNFW), m->pf(K_LNFB), m->lnf(), m->lnfm(), m->lnfr()};
}

// Forward of block l (its weights) from residual slot `in` to slot `out`,
// keeping the block's activations in activation slot `a`. Training uses
// in = a = l, out = l + 1 (everything kept for the backward); evaluation
// reuses slot 0 and two residual slots. When ln1_done, the block's LN1 was
// already computed together with the residual sum that forms its input.
// With residual_norm 1 or 2 and next_a >= 0 the block also forms the next
// pre-norm (next_norm) with its output and sets *next_done.
gpt2_status block_fwd(Model* m, int l, int in, int out, int a, int next_a = -1, bool ln1_done = false,
                      bool* next_done = nullptr) {
  const Dims& d = m->d;
  const int BT = (int)d.BT, C = d.C, F = d.F;
  const size_t oC = (size_t)l * C, o3C = (size_t)l * 3 * C, oF = (size_t)l * F;
  const bool fused = m->residual_norm != 0;
  bf16_t* branch = m->wsb(m->ws.datt);   // free during the forward pass
  if (next_done) *next_done = false;
  if (!ln1_done)
    TRY(ln_fwd(m, m->res(in), m->pf(K_LN1W) + oC, m->pf(K_LN1B) + oC, m->ln1(a), m->ln1m(a), m->ln1r(a)));
  TRY(gemm(m, GPT2_K_GEMM_FWD, BT, 3 * C, C, m->ln1(a), C, 0, m->pb(K_QKVW) + o3C * C, C, 0, EPI_BF16, m->qkv(a),
           3 * C, m->pf(K_QKVB) + o3C));
  AttnArgs aa = attn_args(m, a);
  TRY(m->run(GPT2_K_ATTN_FWD, attn_fwd_flops(d), 0.0, [&] { return launch_attention_fwd(aa, m->stream); }));
  if (!fused) {
    TRY(gemm(m, GPT2_K_GEMM_FWD, BT, C, C, m->att(a), C, 0, m->pb(K_ATTPROJW) + oC * C, C, 0, EPI_BF16, m->xmid(a),
             C, m->pf(K_ATTPROJB) + oC, m->res(in)));
    TRY(ln_fwd(m, m->xmid(a), m->pf(K_LN2W) + oC, m->pf(K_LN2B) + oC, m->ln2(a), m->ln2m(a), m->ln2r(a)));
  } else {
    TRY(gemm(m, GPT2_K_GEMM_FWD, BT, C, C, m->att(a), C, 0, m->pb(K_ATTPROJW) + oC * C, C, 0, EPI_BF16, branch, C,
             m->pf(K_ATTPROJB) + oC));
    TRY(add_norm(m, m->res(in), branch, m->xmid(a), m->pf(K_LN2W) + oC, m->pf(K_LN2B) + oC, m->ln2(a), m->ln2m(a),
                 m->ln2r(a)));
  }
  TRY(gemm(m, GPT2_K_GEMM_FWD, BT, F, C, m->ln2(a), C, 0, m->pb(K_FCW) + oF * C, C, 0, EPI_GELU, m->fc(a), F,
           m->pf(K_FCB) + oF, nullptr, m->gelu(a)));
  if (!fused) {
    TRY(gemm(m, GPT2_K_GEMM_FWD, BT, C, F, m->gelu(a), F, 0, m->pb(K_FCPROJW) + oC * F, F, 0, EPI_BF16, m->res(out),
             C, m->pf(K_FCPROJB) + oC, m->xmid(a)));
  } else {
    TRY(gemm(m, GPT2_K_GEMM_FWD, BT, C, F, m->gelu(a), F, 0, m->pb(K_FCPROJW) + oC * F, F, 0, EPI_BF16, branch, C,
             m->pf(K_FCPROJB) + oC));
    if (next_a >= 0) {
      const NextNorm nn = next_norm(m, l, next_a);
      TRY(add_norm(m, m->xmid(a), branch, m->res(out), nn.w, nn.b, nn.y, nn.mean, nn.rstd));
      if (next_done) *next_done = true;
    } else {
      TRY(add_norm(m, m->xmid(a), branch, m->res(out), nullptr, nullptr, nullptr, nullptr, nullptr));
    }
  }
  return GPT2_OK;
}

// Gradient buffers of one block's backward: the residual-stream gradient
// entering the block (at its output), after its MLP branch, and leaving it
// (at its input); the MLP pre-activation gradient and the q|k|v gradient.
// They may alias (the single-block path runs in place).
struct BlockGrads {
  bf16_t *dres_out, *dres_mid, *dres_in, *dfc, *dqkv;
};

BlockGrads grads_in_place(Model* m) {
  bf16_t* dres = m->wsb(m->ws.dres);
  bf16_t* dbig = m->wsb(m->ws.dbig);
  return {dres, dres, dres, dbig, dbig};
}

// the per-layer buffers the training backward keeps for the grouped
// weight-gradient launch
BlockGrads grads_of_layer(Model* m, int l) {
  const WsLayout& w = m->ws;
  return {m->wsb(w.dres_l + (size_t)(2 * l + 2) * w.s_dres), m->wsb(w.dres_l + (size_t)(2 * l + 1) * w.s_dres),
          m->wsb(w.dres_l + (size_t)(2 * l) * w.s_dres), m->wsb(w.dfc_l + (size_t)l * w.s_dfc),
          m->wsb(w.dqkv_l + (size_t)l * w.s_dqkv)};
}

// Backward of block l from the residual-stream gradient in gb.dres_out. When
// fcproj_bias_done, the MLP output bias gradient (the column sum of dres_out)
// was already produced by the LayerNorm backward that wrote it. When
// write_prev_bias, the column sum of the outgoing gradient is the MLP output
// bias gradient of block l-1. With defer_dw the four weight gradients (and
// the q|k|v and MLP-up bias gradients) are left to the grouped launch.
gpt2_status block_bwd(Model* m, int l, int acc, bool fcproj_bias_done, bool write_prev_bias, const BlockGrads& gb,
                      bool defer_dw) {
  const Dims& d = m->d;
  const int BT = (int)d.BT, C = d.C, F = d.F;
  const size_t oC = (size_t)l * C, o3C = (size_t)l * 3 * C, oF = (size_t)l * F;
  bf16_t* dh = m->wsb(m->ws.dh);
  bf16_t* datt = m->wsb(m->ws.datt);
  // MLP down projection; GELU backward fused into the input-gradient epilogue
  TRY(gemm(m, GPT2_K_GEMM_DX, BT, F, C, gb.dres_out, C, 0, m->pb(K_FCPROJW) + oC * F, F, 1, EPI_GELU_BWD, gb.dfc, F,
           nullptr, nullptr, nullptr, m->fc(l)));
  if (!defer_dw)
    TRY(weight_grad(m, C, F, gb.dres_out, m->gelu(l), m->gf(K_FCPROJW) + oC * F, acc, 0,
                    fcproj_bias_done ? nullptr : m->gf(K_FCPROJB) + oC));
  // MLP up projection
  TRY(gemm(m, GPT2_K_GEMM_DX, BT, C, F, gb.dfc, F, 0, m->pb(K_FCW) + oF * C, C, 1, EPI_BF16, dh, C));
  if (!defer_dw) TRY(weight_grad(m, F, C, gb.dfc, m->ln2(l), m->gf(K_FCW) + oF * C, acc, 0, m->gf(K_FCB) + oF));
  TRY(ln_bwd(m, dh, m->xmid(l), m->ln2m(l), m->ln2r(l), m->pf(K_LN2W) + oC, gb.dres_out, gb.dres_mid, 1,
             m->gf(K_LN2W) + oC, m->gf(K_LN2B) + oC, m->gf(K_ATTPROJB) + oC, acc, defer_dw ? 2 * l + 1 : -1));
  // attention output projection (its bias gradient came from the LayerNorm above)
  TRY(gemm(m, GPT2_K_GEMM_DX, BT, C, C, gb.dres_mid, C, 0, m->pb(K_ATTPROJW) + oC * C, C, 1, EPI_BF16, datt, C));
  if (!defer_dw) TRY(weight_grad(m, C, C, gb.dres_mid, m->att(l), m->gf(K_ATTPROJW) + oC * C, acc));
  // attention
  AttnArgs aa = attn_args(m, l, gb.dqkv);
  TRY(m->run(GPT2_K_ATTN_BWD, 2.0 * attn_fwd_flops(d), 0.0, [&] { return launch_attention_bwd(aa, m->stream); }));
  // q|k|v projection
  TRY(gemm(m, GPT2_K_GEMM_DX, BT, C, 3 * C, gb.dqkv, 3 * C, 0, m->pb(K_QKVW) + o3C * C, C, 1, EPI_BF16, dh, C));
  if (!defer_dw)
    TRY(weight_grad(m, 3 * C, C, gb.dqkv, m->ln1(l), m->gf(K_QKVW) + o3C * C, acc, 0, m->gf(K_QKVB) + o3C));
  float* prev_bias = (write_prev_bias && l > 0) ? m->gf(K_FCPROJB) + (size_t)(l - 1) * C : nullptr;
  TRY(ln_bwd(m, dh, m->res(l), m->ln1m(l), m->ln1r(l), m->pf(K_LN1W) + oC, gb.dres_mid, gb.dres_in, 1,
             m->gf(K_LN1W) + oC, m->gf(K_LN1B) + oC, prev_bias, acc, defer_dw ? 2 * l : -1));
  return GPT2_OK;
}

// Every block weight gradient in one launch, from the layers' kept gradients
// and saved activations: no contraction split, so no partial slices; then the
// q|k|v and MLP-up bias gradients from the launch's partial sums.
gpt2_status grouped_weight_grads(Model* m, int acc) {
  const Dims& d = m->d;
  const WsLayout& w = m->ws;
  const ActLayout& a = m->act;
  const size_t C = d.C, F = d.F;
  GemmGroupedArgs g = dw_groups(d);
  g.accumulate = acc;
  GemmGroup* q = &g.grp[G_QKV];
  q->A = m->wsb(w.dqkv_l); q->a_stride = (long)(w.s_dqkv / 2); q->lda = (int)(3 * C);
  q->B = m->ln1(0); q->b_stride = (long)(a.s_act / 2); q->ldb = (int)C;
  q->C = m->gf(K_QKVW); q->c_stride = (long)(3 * C * C);
  q->bsum = m->wsf(w.gbs_qkv);
  GemmGroup* ap = &g.grp[G_ATTPROJ];
  ap->A = m->wsb(w.dres_l + w.s_dres); ap->a_stride = (long)(w.s_dres); ap->lda = (int)C;   // slots 2l+1
  ap->B = m->att(0); ap->b_stride = (long)(a.s_act / 2); ap->ldb = (int)C;
  ap->C = m->gf(K_ATTPROJW); ap->c_stride = (long)(C * C);
  GemmGroup* fc = &g.grp[G_FC];
  fc->A = m->wsb(w.dfc_l); fc->a_stride = (long)(w.s_dfc / 2); fc->lda = (int)F;
  fc->B = m->ln2(0); fc->b_stride = (long)(a.s_act / 2); fc->ldb = (int)C;
  fc->C = m->gf(K_FCW); fc->c_stride = (long)(F * C);
  fc->bsum = m->wsf(w.gbs_fc);
  GemmGroup* fp = &g.grp[G_FCPROJ];
  fp->A = m->wsb(w.dres_l + 2 * w.s_dres); fp->a_stride = (long)(w.s_dres); fp->lda = (int)C;   // slots 2l+2
  fp->B = m->gelu(0); fp->b_stride = (long)(a.s_ff / 2); fp->ldb = (int)F;
  fp->C = m->gf(K_FCPROJW); fp->c_stride = (long)(C * F);
  // the last np MLP-down products as a fifth group with a split contraction
  // (slices in the split-K buffer)
  const DwGroupedTail gt = dw_grouped_tail(d);
  float* tail_dst = nullptr;
  if (gt.np > 0) {
    const int keep = (int)d.L - gt.np;
    GemmGroup* tl = &g.grp[g.ngroups++];
    *tl = *fp;
    fp->count = keep;
    tl->count = gt.np;
    tl->A = fp->A + (size_t)keep * fp->a_stride;
    tl->B = fp->B + (size_t)keep * fp->b_stride;
    tl->C = m->wsf(w.splitk);
    tl->splits = gt.splits;
    tl->k_chunk = gt.chunk;
    tl->split_stride = (long)gt.np * (long)(C * F);
    g.nfull = gt.nfull;
    tail_dst = m->gf(K_FCPROJW) + (size_t)keep * C * F;
  }
  double fl = 0.0;
  for (int i = 0; i < g.ngroups; ++i) fl += 2.0 * g.grp[i].M * (double)g.grp[i].N * d.BT * g.grp[i].count;
  TRY(m->run(GPT2_K_GEMM_DW_GROUPED, fl, 0.0, [&] { return launch_gemm_grouped(g, m->stream); }));
  if (tail_dst) {
    const long n = (long)gt.np * (long)(C * F);
    TRY(m->run(GPT2_K_OTHER, 0.0, 4.0 * n * (gt.splits + 1 + acc), [&] {
      return launch_reduce_slices2(m->wsf(w.splitk), gt.splits, n, tail_dst, nullptr, 0, 0, nullptr, acc, m->stream);
    }));
  }
  const int pq = gemm_grouped_bias_parts(g, G_QKV), pf = gemm_grouped_bias_parts(g, G_FC);
  const long nq = (long)d.L * 3 * C, nf = (long)d.L * F;
  TRY(m->run(GPT2_K_OTHER, 0.0, 4.0 * nq * (pq + 1 + acc), [&] {
    return launch_reduce_parts(m->wsf(w.gbs_qkv), pq, nq, (int)nq, 1, m->gf(K_QKVB), nullptr, nullptr, acc,
                               m->stream);
  }));
  TRY(m->run(GPT2_K_OTHER, 0.0, 4.0 * nf * (pf + 1 + acc), [&] {
    return launch_reduce_parts(m->wsf(w.gbs_fc), pf, nf, (int)nf, 1, m->gf(K_FCB), nullptr, nullptr, acc, m->stream);
  }));
  return GPT2_OK;
}

double lr_schedule(const gpt2_config& c, int64_t step) {
  if (step < c.warmup_steps) return (double)c.lr_max * (double)(step + 1) / c.warmup_steps;
  double frac = (double)(step - c.warmup_steps) / (double)(c.total_steps - c.warmup_steps);
  if (frac < 0) frac = 0;
  if (frac > 1) frac = 1;
  return (double)c.lr_min + 0.5 * (1.0 + std::cos(M_PI * frac)) * ((double)c.lr_max - (double)c.lr_min);
}

thread_local std::string g_last_error;

// Seeded initialisation on the device (section "Model": N(0, 0.02), the two
// projections that write into the residual stream scaled by 1/sqrt(2L);
// biases and LayerNorm shifts 0, gains 1, padding rows of the token table 0);
// the Adam moments are cleared and the bf16 copy written in the same pass.
gpt2_status seeded_init(Model* m, uint64_t seed) {
  InitArgs a{};
  a.p = static_cast<float*>(m->buf.params_f32);
  a.m = static_cast<float*>(m->buf.adam_m);
  a.v = static_cast<float*>(m->buf.adam_v);
  a.p_bf16 = static_cast<bf16_t*>(m->buf.params_bf16);
  a.n = (long)m->n_params;
  a.count = K_NKIND;
  const double std = 0.02, rstd = 0.02 / std::sqrt(2.0 * m->d.L);
  for (int k = 0; k < K_NKIND; ++k) {
    a.end[k] = (long)(m->koff[k] + m->kn[k]);
    const bool weight = k == K_WTE || k == K_WPE || k == K_QKVW || k == K_FCW;
    const bool resid = k == K_ATTPROJW || k == K_FCPROJW;
    a.std[k] = weight ? std : resid ? rstd : 0.0;
    a.fill[k] = (k == K_LN1W || k == K_LN2W || k == K_LNFW) ? 1.0f : 0.0f;
  }
  a.zero_lo = (long)m->koff[K_WTE] + (long)m->d.V * m->d.C;
  a.zero_hi = (long)m->koff[K_WTE] + (long)m->d.Vp * m->d.C;
  a.key0 = (uint32_t)seed;
  a.key1 = (uint32_t)(seed >> 32);
  TRY(m->run(GPT2_K_OTHER, 0.0, 14.0 * m->n_params, [&] { return launch_init_params(a, m->stream); }));
  return GPT2_OK;
}

// Copy the mean loss and the id-range flag moved next to it, synchronise, and
// report ids outside [0, vocab) seen since the last report.
gpt2_status read_loss(Model* m, float* loss_out) {
  float host[2];
  TRY(hipMemcpyAsync(host, m->loss_mean(), sizeof(host), hipMemcpyDeviceToHost, m->stream));
  TRY(hipStreamSynchronize(m->stream));
  *loss_out = host[0];
  uint32_t bad;
  std::memcpy(&bad, &host[1], 4);
  if (bad)
    return m->fail(GPT2_ERR_INVALID_ARG, std::string("token ids outside [0, vocab) in the ") +
                                             ((bad & ID_BAD_INPUT) && (bad & ID_BAD_TARGET) ? "inputs and targets"
                                              : (bad & ID_BAD_INPUT)                         ? "inputs"
                                                                                             : "targets") +
                                             " of a forward pass since the last loss: the loss is not meaningful");
  return GPT2_OK;
}

}  // namespace

extern "C" {

gpt2_status gpt2_query_sizes(const gpt2_config* cfg, gpt2_sizes* out) {
  if (const char* why = validate(cfg)) {
    g_last_error = why;
    return GPT2_ERR_INVALID_ARG;
  }
  if (!out) {
    g_last_error = "out is NULL";
    return GPT2_ERR_INVALID_ARG;
  }
  Dims d = dims_of(*cfg);
  size_t kn[K_NKIND];
  kind_sizes(d, kn);
  size_t n = 0;
  for (int k = 0; k < K_NKIND; ++k) n += kn[k];
  out->n_params = n;
  out->params_f32 = out->grads_f32 = out->adam_m = out->adam_v = align_up(n * 4);
  out->params_bf16 = align_up(n * 2);
  out->activations = act_layout(d).total;
  out->workspace = ws_layout(d).total;
  return GPT2_OK;
}

int32_t gpt2_num_tensors(const gpt2_config* cfg) {
  if (!cfg || cfg->n_layer < 1) return 0;
  return 2 + 12 * cfg->n_layer + 2;
}

gpt2_status gpt2_tensor_info(const gpt2_config* cfg, int32_t idx, char* name, size_t* offset, int32_t* shape,
                             int32_t* ndim, int32_t* decay) {
  if (const char* why = validate(cfg)) {
    g_last_error = why;
    return GPT2_ERR_INVALID_ARG;
  }
  if (!name || !offset || !shape || !ndim || !decay || idx < 0 || idx >= gpt2_num_tensors(cfg)) {
    g_last_error = "bad tensor_info argument";
    return GPT2_ERR_INVALID_ARG;
  }
  Dims d = dims_of(*cfg);
  size_t kn[K_NKIND], ko[K_NKIND], o = 0;
  kind_sizes(d, kn);
  for (int k = 0; k < K_NKIND; ++k) {
    ko[k] = o;
    o += kn[k];
  }
  static const char* per_layer[12] = {"ln_1.weight", "ln_1.bias", "attn.c_attn.weight", "attn.c_attn.bias",
                                      "attn.c_proj.weight", "attn.c_proj.bias", "ln_2.weight", "ln_2.bias",
                                      "mlp.c_fc.weight", "mlp.c_fc.bias", "mlp.c_proj.weight", "mlp.c_proj.bias"};
  static const int per_layer_kind[12] = {K_LN1W, K_LN1B, K_QKVW, K_QKVB, K_ATTPROJW, K_ATTPROJB,
                                         K_LN2W, K_LN2B, K_FCW, K_FCB, K_FCPROJW, K_FCPROJB};
  const int C = d.C, F = d.F;
  if (idx == 0) {
    snprintf(name, 64, "wte");
    *offset = ko[K_WTE]; shape[0] = d.Vp; shape[1] = C; *ndim = 2; *decay = 1;
    return GPT2_OK;
  }
  if (idx == 1) {
    snprintf(name, 64, "wpe");
    *offset = ko[K_WPE]; shape[0] = d.Tmax; shape[1] = C; *ndim = 2; *decay = 1;
    return GPT2_OK;
  }
  int last = gpt2_num_tensors(cfg);
  if (idx >= last - 2) {
    bool w = idx == last - 2;
    snprintf(name, 64, w ? "ln_f.weight" : "ln_f.bias");
    *offset = ko[w ? K_LNFW : K_LNFB]; shape[0] = C; shape[1] = 0; *ndim = 1; *decay = 0;
    return GPT2_OK;
  }
  int l = (idx - 2) / 12, j = (idx - 2) % 12;
  int k = per_layer_kind[j];
  snprintf(name, 64, "h.%d.%s", l, per_layer[j]);
  size_t per = kn[k] / d.L;
  *offset = ko[k] + (size_t)l * per;
  *decay = kDecay[k] ? 1 : 0;
  switch (k) {
    case K_QKVW: shape[0] = 3 * C; shape[1] = C; *ndim = 2; break;
    case K_QKVB: shape[0] = 3 * C; shape[1] = 0; *ndim = 1; break;
    case K_ATTPROJW: shape[0] = C; shape[1] = C; *ndim = 2; break;
    case K_FCW: shape[0] = F; shape[1] = C; *ndim = 2; break;
    case K_FCB: shape[0] = F; shape[1] = 0; *ndim = 1; break;
    case K_FCPROJW: shape[0] = C; shape[1] = F; *ndim = 2; break;
    default: shape[0] = C; shape[1] = 0; *ndim = 1; break;
  }
  return GPT2_OK;
}

gpt2_status gpt2_init(const gpt2_config* cfg, const gpt2_buffers* bufs, void* hip_stream, uint64_t seed,
                      int32_t init_mode, gpt2_model** out) {
  if (const char* why = validate(cfg)) {
    g_last_error = why;
    return GPT2_ERR_INVALID_ARG;
  }
  if (!bufs || !out) {
    g_last_error = "bufs or out is NULL";
    return GPT2_ERR_INVALID_ARG;
  }
  if (init_mode != 0 && init_mode != 1) {
    g_last_error = "init_mode must be 0 (caller-filled weights) or 1 (seeded initialisation)";
    return GPT2_ERR_INVALID_ARG;
  }
  const void* ptrs[7] = {bufs->params_f32, bufs->grads_f32, bufs->adam_m, bufs->adam_v,
                         bufs->params_bf16, bufs->activations, bufs->workspace};
  for (const void* p : ptrs) {
    if (!p || (reinterpret_cast<uintptr_t>(p) % ALIGN)) {
      g_last_error = "a buffer is NULL or not 256-byte aligned";
      return GPT2_ERR_INVALID_ARG;
    }
  }
  Model* m = new (std::nothrow) Model();
  if (!m) {
    g_last_error = "out of host memory";
    return GPT2_ERR_INVALID_ARG;
  }
  m->cfg = *cfg;
  m->d = dims_of(*cfg);
  m->buf = *bufs;
  m->stream = static_cast<hipStream_t>(hip_stream);
  kind_sizes(m->d, m->kn);
  size_t o = 0;
  for (int k = 0; k < K_NKIND; ++k) {
    m->koff[k] = o;
    o += m->kn[k];
  }
  m->n_params = o;
  m->act = act_layout(m->d);
  m->ws = ws_layout(m->d);
  gpt2_status st = init_mode == 1 ? seeded_init(m, seed) : gpt2_sync_weights(m);
  // the id-range flag starts clear (a fill kernel, not a memset, so the
  // enqueued work stays capturable)
  if (st == GPT2_OK &&
      launch_reduce_slices(nullptr, 0, 4, reinterpret_cast<float*>(m->id_flag()), 0, m->stream) != hipSuccess)
    st = m->fail(GPT2_ERR_DEVICE, "clearing the id-range flag failed");
  if (st != GPT2_OK) {
    g_last_error = m->err;
    delete m;
    return st;
  }
  *out = m;
  return GPT2_OK;
}

gpt2_status gpt2_sync_weights(gpt2_model* m) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  TRY(m->run(GPT2_K_OTHER, 0.0, 6.0 * m->n_params, [&] {
    return launch_cast_bf16(static_cast<float*>(m->buf.params_f32), static_cast<bf16_t*>(m->buf.params_bf16),
                            (long)m->n_params, m->stream);
  }));
  return GPT2_OK;
}

gpt2_status gpt2_forward(gpt2_model* m, const int32_t* d_inputs, const int32_t* d_targets) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  if (!d_inputs) return m->fail(GPT2_ERR_INVALID_ARG, "inputs is NULL");
  const Dims& d = m->d;
  const int BT = (int)d.BT, C = d.C;
  m->have_dlogits = false;
  m->have_loss = false;
  // keep the ids for the embedding backward
  TRY(hipMemcpyAsync(m->ids(), d_inputs, (size_t)BT * 4, hipMemcpyDeviceToDevice, m->stream));
  TRY(m->run(GPT2_K_OTHER, 0.0, 4.0 * BT + 8.0 * BT * C + 2.0 * BT * C,
             [&] {
               return launch_embed_fwd(d_inputs, m->pf(K_WTE), m->pf(K_WPE), m->res(0), d.B, d.T, C, d.V, m->id_flag(),
                                       m->stream);
             }));
  bool ln_done = false;
  for (int l = 0; l < d.L; ++l) {
    gpt2_status s = block_fwd(m, l, l, l + 1, l, l + 1, ln_done, &ln_done);
    if (s != GPT2_OK) return s;
  }
  if (!ln_done) TRY(ln_fwd(m, m->res(d.L), m->pf(K_LNFW), m->pf(K_LNFB), m->lnf(), m->lnfm(), m->lnfr()));
  if (!d_targets) {
    // logits only
    TRY(gemm(m, GPT2_K_GEMM_FWD, BT, d.Vp, C, m->lnf(), C, 0, m->pb(K_WTE), C, 0, EPI_BF16, m->logits(), d.Vp,
             nullptr, nullptr, nullptr, nullptr, 0, 1, 0, 0, 2.0 * BT * (double)d.V * C));
    return GPT2_OK;
  }
  {
    gpt2_status st = head_and_loss(m, d_targets, (float)(1.0 / ((double)BT * d.accum)), 1, m->head_ce);
    if (st != GPT2_OK) return st;
  }
  m->have_dlogits = true;
  m->have_loss = true;
  return GPT2_OK;
}

gpt2_status gpt2_evaluate(gpt2_model* m, const int32_t* d_inputs, const int32_t* d_targets, float* loss_out,
                          float* d_token_losses) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  if (!d_inputs || !d_targets || !loss_out) return m->fail(GPT2_ERR_INVALID_ARG, "inputs, targets or loss_out is NULL");
  const Dims& d = m->d;
  const int BT = (int)d.BT, C = d.C;
  // the activation buffer is reused: the last training forward is gone
  m->have_dlogits = false;
  m->have_loss = false;
  TRY(m->run(GPT2_K_OTHER, 0.0, 4.0 * BT + 8.0 * BT * C + 2.0 * BT * C,
             [&] {
               return launch_embed_fwd(d_inputs, m->pf(K_WTE), m->pf(K_WPE), m->res(0), d.B, d.T, C, d.V, m->id_flag(),
                                       m->stream);
             }));
  bool ln_done = false;
  for (int l = 0; l < d.L; ++l) {
    gpt2_status s = block_fwd(m, l, l & 1, (l + 1) & 1, 0, 0, ln_done, &ln_done);
    if (s != GPT2_OK) return s;
  }
  if (!ln_done) TRY(ln_fwd(m, m->res(d.L & 1), m->pf(K_LNFW), m->pf(K_LNFB), m->lnf(), m->lnfm(), m->lnfr()));
  {
    gpt2_status st = head_and_loss(m, d_targets, 0.0f, 0, 1);
    if (st != GPT2_OK) return st;
  }
  if (d_token_losses)
    TRY(hipMemcpyAsync(d_token_losses, m->losses(), (size_t)BT * 4, hipMemcpyDeviceToDevice, m->stream));
  return read_loss(m, loss_out);
}

gpt2_status gpt2_backward(gpt2_model* m, int32_t accumulate) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  if (!m->have_dlogits) return m->fail(GPT2_ERR_STATE, "backward needs a forward with targets first");
  if (accumulate && !m->have_grads) return m->fail(GPT2_ERR_STATE, "accumulate with no gradient to add to");
  const Dims& d = m->d;
  const int BT = (int)d.BT, C = d.C;
  const int acc = accumulate ? 1 : 0;
  bf16_t* dh = m->wsb(m->ws.dh);
  m->ln_jobs.count = 0;   // nothing queued from a pass that failed part-way
  // tied LM head: input gradient and the head's share of the token-table gradient
  TRY(gemm(m, GPT2_K_GEMM_DX, BT, C, d.Vp, m->logits(), d.Vp, 0, m->pb(K_WTE), C, 1, EPI_BF16, dh, C, nullptr,
           nullptr, nullptr, nullptr, 0, 1, 0, 0, 2.0 * BT * (double)d.V * C));
  TRY(weight_grad(m, d.Vp, C, m->logits(), m->lnf(), m->gf(K_WTE), acc, d.V));
  bf16_t* dres_top = grads_of_layer(m, d.L - 1).dres_out;   // written, not read (has_res 0)
  TRY(ln_bwd(m, dh, m->res(d.L), m->lnfm(), m->lnfr(), m->pf(K_LNFW), dres_top, dres_top, 0, m->gf(K_LNFW),
             m->gf(K_LNFB), m->gf(K_FCPROJB) + (size_t)(d.L - 1) * C, acc, 2 * d.L));
  for (int l = d.L - 1; l >= 0; --l) {
    gpt2_status s = block_bwd(m, l, acc, true, true, grads_of_layer(m, l), true);
    if (s != GPT2_OK) return s;
  }
  const bf16_t* dres = grads_of_layer(m, 0).dres_in;
  // embedding: scatter into the token table (after the head's share), sum into positions
  TRY(m->run(GPT2_K_OTHER, 0.0, 4.0 * BT + 2.0 * BT * C + 8.0 * BT * C,
             [&] { return launch_embed_bwd(m->ids(), dres, m->gf(K_WTE), d.B, d.T, C, d.V, m->stream); }));
  TRY(m->run(GPT2_K_OTHER, 0.0, 2.0 * BT * C + 4.0 * d.Tmax * C * (1 + acc),
             [&] { return launch_embed_bwd_pos(dres, m->gf(K_WPE), d.B, d.T, d.Tmax, C, acc, m->stream); }));
  {
    gpt2_status s = grouped_weight_grads(m, acc);
    if (s != GPT2_OK) return s;
  }
  // every LayerNorm's gain, shift and following-bias gradients
  TRY(reduce_ln_parts(m));
  m->have_grads = true;
  return GPT2_OK;
}

}  // extern "C"

namespace {

// The optimizer step with its scratch (sum-of-squares partials, norm and clip
// coefficient) at the given device addresses.
gpt2_status adamw_step_with(gpt2_model* m, int64_t step, float* lr_out, float* d_grad_norm_out, float* parts,
                            float* nc) {
  const gpt2_config& c = m->cfg;
  const long n = (long)m->n_params;
  float* grads = static_cast<float*>(m->buf.grads_f32);
  TRY(m->run(GPT2_K_OPTIMIZER, 0.0, 4.0 * n, [&] { return launch_sumsq(grads, n, parts, m->stream); }));
  TRY(m->run(GPT2_K_OPTIMIZER, 0.0, 4.0 * sumsq_parts(),
             [&] { return launch_clip_coef(parts, sumsq_parts(), c.grad_clip, nc, m->stream); }));
  if (d_grad_norm_out)
    TRY(hipMemcpyAsync(d_grad_norm_out, nc, sizeof(float), hipMemcpyDeviceToDevice, m->stream));
  const double lr = lr_schedule(c, step);
  AdamArgs a{};
  a.p = static_cast<float*>(m->buf.params_f32);
  a.g = grads;
  a.m = static_cast<float*>(m->buf.adam_m);
  a.v = static_cast<float*>(m->buf.adam_v);
  a.p_bf16 = static_cast<bf16_t*>(m->buf.params_bf16);
  a.norm_coef = nc;
  a.n = n;
  a.lr = (float)lr;
  a.beta1 = c.beta1; a.beta2 = c.beta2; a.eps = c.adam_eps; a.weight_decay = c.weight_decay;
  a.bc1 = (float)(1.0 - std::pow((double)c.beta1, (double)(step + 1)));
  a.bc2 = (float)(1.0 - std::pow((double)c.beta2, (double)(step + 1)));
  a.seg.count = K_NKIND;
  for (int k = 0; k < K_NKIND; ++k) {
    a.seg.end[k] = (long)(m->koff[k] + m->kn[k]);
    a.seg.decay[k] = kDecay[k] ? 1 : 0;
  }
  TRY(m->run(GPT2_K_OPTIMIZER, 0.0, 30.0 * n, [&] { return launch_adamw(a, m->stream); }));
  if (lr_out) *lr_out = (float)lr;
  m->have_grads = false;
  return GPT2_OK;
}

}  // namespace

extern "C" {

gpt2_status gpt2_adamw_step(gpt2_model* m, int64_t step, float* lr_out, float* d_grad_norm_out) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  if (step < 0) return m->fail(GPT2_ERR_INVALID_ARG, "step must be >= 0");
  if (!m->have_grads) return m->fail(GPT2_ERR_STATE, "optimizer step with no gradient");
  return adamw_step_with(m, step, lr_out, d_grad_norm_out, m->wsf(m->ws.sumsq), m->wsf(m->ws.normcoef));
}

gpt2_status gpt2_adamw_step_noalloc(gpt2_model* m, int64_t step, float* lr_out, float* d_grad_norm_out) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  if (step < 0) return m->fail(GPT2_ERR_INVALID_ARG, "step must be >= 0");
  if (!m->have_grads) return m->fail(GPT2_ERR_STATE, "optimizer step with no gradient");
  // partials, then the norm and coefficient at the next 64-float boundary
  const int parts = sumsq_parts();
  const int nc_off = (parts + 63) / 64 * 64;
  if (nc_off + 2 > NOALLOC_SCRATCH_FLOATS)
    return m->fail(GPT2_ERR_INVALID_ARG, "the optimizer's scratch (" + std::to_string(nc_off + 2) +
                                             " floats) exceeds the static scratch array (" +
                                             std::to_string(NOALLOC_SCRATCH_FLOATS) + " floats)");
  float* scratch = nullptr;
  TRY(noalloc_scratch(&scratch));
  return adamw_step_with(m, step, lr_out, d_grad_norm_out, scratch, scratch + nc_off);
}

gpt2_status gpt2_loss(gpt2_model* m, float* loss_out, float* d_token_losses) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  if (!loss_out) return m->fail(GPT2_ERR_INVALID_ARG, "loss_out is NULL");
  if (!m->have_loss) return m->fail(GPT2_ERR_STATE, "no forward with targets yet");
  if (d_token_losses)
    TRY(hipMemcpyAsync(d_token_losses, m->losses(), (size_t)m->d.BT * 4, hipMemcpyDeviceToDevice, m->stream));
  return read_loss(m, loss_out);
}

float gpt2_lr_at(const gpt2_config* cfg, int64_t step) {
  if (!cfg || step < 0) return 0.0f;
  return (float)lr_schedule(*cfg, step);
}

void gpt2_destroy(gpt2_model* m) {
  if (!m) return;
  delete m;
}

const char* gpt2_last_error(const gpt2_model* m) {
  if (m && !m->err.empty()) return m->err.c_str();
  return g_last_error.c_str();
}

gpt2_status gpt2_activation_info(const gpt2_model* mc, int32_t which, int32_t layer, size_t* offset_bytes,
                                 size_t* numel, int32_t* dtype) {
  gpt2_model* m = const_cast<gpt2_model*>(mc);
  if (!m || !offset_bytes || !numel || !dtype) return GPT2_ERR_INVALID_ARG;
  const Dims& d = m->d;
  const size_t BT = d.BT, C = d.C;
  const ActLayout& a = m->act;
  const bool per_layer = which >= GPT2_ACT_LN1 && which <= GPT2_ACT_GELU;
  const int lmax = which == GPT2_ACT_RESIDUAL ? d.L : (per_layer ? d.L - 1 : 0);
  if (layer < 0 || layer > lmax) return m->fail(GPT2_ERR_INVALID_ARG, "layer out of range");
  const size_t l = layer;
  switch (which) {
    case GPT2_ACT_RESIDUAL: *offset_bytes = a.residual + l * a.s_act; *numel = BT * C; *dtype = 1; break;
    case GPT2_ACT_LN1: *offset_bytes = a.ln1 + l * a.s_act; *numel = BT * C; *dtype = 1; break;
    case GPT2_ACT_LN1_MEAN: *offset_bytes = a.ln1_mean + l * a.s_row; *numel = BT; *dtype = 0; break;
    case GPT2_ACT_LN1_RSTD: *offset_bytes = a.ln1_rstd + l * a.s_row; *numel = BT; *dtype = 0; break;
    case GPT2_ACT_QKV: *offset_bytes = a.qkv + l * a.s_qkv; *numel = BT * 3 * C; *dtype = 1; break;
    case GPT2_ACT_ATT: *offset_bytes = a.att + l * a.s_act; *numel = BT * C; *dtype = 1; break;
    case GPT2_ACT_ATT_LSE: *offset_bytes = a.lse + l * a.s_lse; *numel = (size_t)d.B * d.H * d.T; *dtype = 0; break;
    case GPT2_ACT_X_MID: *offset_bytes = a.x_mid + l * a.s_act; *numel = BT * C; *dtype = 1; break;
    case GPT2_ACT_LN2: *offset_bytes = a.ln2 + l * a.s_act; *numel = BT * C; *dtype = 1; break;
    case GPT2_ACT_LN2_MEAN: *offset_bytes = a.ln2_mean + l * a.s_row; *numel = BT; *dtype = 0; break;
    case GPT2_ACT_LN2_RSTD: *offset_bytes = a.ln2_rstd + l * a.s_row; *numel = BT; *dtype = 0; break;
    case GPT2_ACT_FC: *offset_bytes = a.fc + l * a.s_ff; *numel = BT * d.F; *dtype = 1; break;
    case GPT2_ACT_GELU: *offset_bytes = a.gelu + l * a.s_ff; *numel = BT * d.F; *dtype = 1; break;
    case GPT2_ACT_LNF: *offset_bytes = a.lnf; *numel = BT * C; *dtype = 1; break;
    case GPT2_ACT_LNF_MEAN: *offset_bytes = a.lnf_mean; *numel = BT; *dtype = 0; break;
    case GPT2_ACT_LNF_RSTD: *offset_bytes = a.lnf_rstd; *numel = BT; *dtype = 0; break;
    case GPT2_ACT_LOGITS: *offset_bytes = a.logits; *numel = BT * d.Vp; *dtype = 1; break;
    case GPT2_ACT_LOSSES: *offset_bytes = a.losses; *numel = BT; *dtype = 0; break;
    default: return m->fail(GPT2_ERR_INVALID_ARG, "unknown activation");
  }
  return GPT2_OK;
}

gpt2_status gpt2_block_forward(gpt2_model* m, int32_t layer, const void* d_x_in, void* d_x_out) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  if (!d_x_in || layer < 0 || layer >= m->d.L) return m->fail(GPT2_ERR_INVALID_ARG, "bad block_forward argument");
  const size_t bytes = (size_t)m->d.BT * m->d.C * 2;
  TRY(hipMemcpyAsync(m->res(layer), d_x_in, bytes, hipMemcpyDeviceToDevice, m->stream));
  gpt2_status s = block_fwd(m, layer, layer, layer + 1, layer);
  if (s != GPT2_OK) return s;
  if (d_x_out) TRY(hipMemcpyAsync(d_x_out, m->res(layer + 1), bytes, hipMemcpyDeviceToDevice, m->stream));
  return GPT2_OK;
}

gpt2_status gpt2_block_backward(gpt2_model* m, int32_t layer, const void* d_dx_out, void* d_dx_in,
                                int32_t accumulate) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  if (!d_dx_out || layer < 0 || layer >= m->d.L) return m->fail(GPT2_ERR_INVALID_ARG, "bad block_backward argument");
  const size_t bytes = (size_t)m->d.BT * m->d.C * 2;
  bf16_t* dres = m->wsb(m->ws.dres);
  TRY(hipMemcpyAsync(dres, d_dx_out, bytes, hipMemcpyDeviceToDevice, m->stream));
  gpt2_status s = block_bwd(m, layer, accumulate ? 1 : 0, false, false, grads_in_place(m), false);
  if (s != GPT2_OK) return s;
  if (d_dx_in) TRY(hipMemcpyAsync(d_dx_in, dres, bytes, hipMemcpyDeviceToDevice, m->stream));
  return GPT2_OK;
}

gpt2_status gpt2_embedding_backward(gpt2_model* m, const int32_t* d_ids, const void* d_dx, int32_t accumulate) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  if (!d_ids || !d_dx) return m->fail(GPT2_ERR_INVALID_ARG, "ids or dx is NULL");
  const Dims& d = m->d;
  const bf16_t* dx = static_cast<const bf16_t*>(d_dx);
  const int acc = accumulate ? 1 : 0;
  if (!acc)  // zero-slice reduction writes zeros
    TRY(launch_reduce_slices(nullptr, 0, (long)m->kn[K_WTE], m->gf(K_WTE), 0, m->stream));
  TRY(m->run(GPT2_K_OTHER, 0.0, 4.0 * d.BT + 10.0 * d.BT * d.C,
             [&] { return launch_embed_bwd(d_ids, dx, m->gf(K_WTE), d.B, d.T, d.C, d.V, m->stream); }));
  TRY(m->run(GPT2_K_OTHER, 0.0, 2.0 * d.BT * d.C + 4.0 * d.Tmax * d.C * (1 + acc),
             [&] { return launch_embed_bwd_pos(dx, m->gf(K_WPE), d.B, d.T, d.Tmax, d.C, acc, m->stream); }));
  return GPT2_OK;
}

gpt2_status gpt2_set_fusion(gpt2_model* m, int32_t fusion, int32_t mode) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  if (fusion == GPT2_FUSION_RESIDUAL_NORM) {
    if (mode < 0 || mode > 2) return m->fail(GPT2_ERR_INVALID_ARG, "residual-norm mode must be 0, 1 or 2");
    m->residual_norm = mode;
    return GPT2_OK;
  }
  if (fusion == GPT2_FUSION_HEAD_CE) {
    if (mode < 0 || mode > 1) return m->fail(GPT2_ERR_INVALID_ARG, "head-cross-entropy mode must be 0 or 1");
    m->head_ce = mode;
    return GPT2_OK;
  }
  return m->fail(GPT2_ERR_INVALID_ARG, "unknown fusion");
}

gpt2_status gpt2_probe_enable(gpt2_model* m, uint32_t class_mask) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  m->probes.mask = class_mask;
  return GPT2_OK;
}

gpt2_status gpt2_probe_reset(gpt2_model* m) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  if (m->probes.reset() != hipSuccess) return m->fail(GPT2_ERR_DEVICE, "event sync failed");
  return GPT2_OK;
}

gpt2_status gpt2_probe_read(gpt2_model* m, int32_t kclass, double* total_ms, int64_t* launches, double* flops,
                            double* bytes) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  if (kclass < 0 || kclass >= GPT2_K_COUNT) return m->fail(GPT2_ERR_INVALID_ARG, "bad kernel class");
  if (m->probes.collect() != hipSuccess) return m->fail(GPT2_ERR_DEVICE, "event timing failed");
  if (total_ms) *total_ms = m->probes.ms[kclass];
  if (launches) *launches = m->probes.launches[kclass];
  if (flops) *flops = m->probes.flops[kclass];
  if (bytes) *bytes = m->probes.bytes[kclass];
  return GPT2_OK;
}

}  // extern "C"
