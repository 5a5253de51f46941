// Host side of the Qwen3-shaped adapter fine-tuning step: configuration
// checks, the layout of the caller-owned buffers, and the launch sequence of
// the forward pass, the backward pass (adapter gradients, with input
// gradients through the frozen base) and the adapter optimizer step. Every
// launch goes to the stream given at init; nothing here allocates device
// memory.
//
// Adapters: the down products u = s x A^T and, backward, du = s dy B run in
// one pass over x or dy each (lora.hip, n*RP columns with the rank padding
// written as zeros); the up products ride on the base projections' GEMMs as
// a second contraction segment, y += u B^T and dx += du A; dA = du^T x and
// dB = dy^T u contract over the tokens, split and reduced.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/qwen3.h"
#include "kernels.h"
#include "probe.h"

namespace {

// Padded adapter rank: every contraction the GEMMs run must be a whole
// number of their 32- or 64-deep k-tiles (a tile reads past a sub-matrix's
// last column into its neighbour, and only the buffer's end reads as zero),
// so the rank is padded to 64 and B*T, the vocabulary and all widths are
// multiples of 64.
constexpr int RP = 64;
constexpr size_t ALIGN = 256;
constexpr size_t TAIL = 1 << 20;   // slack after each arena: operand tiles of
                                   // column-offset sub-matrices may address
                                   // up to a tile row past the last element
size_t align_up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

enum Group { G_QKV, G_O, G_GU, G_DN, G_N };

struct Dims {
  int L, C, H, Hkv, hd, F, V, Tmax, B, T, r, groups;
  long BT;
  int QD, KVD, QKVD;   // H*hd, Hkv*hd, (H+2Hkv)*hd
  float s;             // alpha / sqrt(r)
  int mask_from;       // first position with loss
  int nl;              // positions with loss per sequence, T - mask_from
  long BTL;            // rows with loss, B * nl
};

Dims dims_of(const qwen3_config& c) {
  Dims d{};
  d.L = c.n_layer; d.C = c.d_model; d.H = c.n_head; d.Hkv = c.n_kv_head; d.hd = c.head_dim; d.F = c.d_ff;
  d.V = c.vocab; d.Tmax = c.max_seq_len; d.B = c.B; d.T = c.T; d.r = c.lora_rank; d.groups = c.lora_groups;
  d.BT = (long)c.B * c.T;
  d.QD = d.H * d.hd; d.KVD = d.Hkv * d.hd; d.QKVD = d.QD + 2 * d.KVD;
  d.s = c.lora_alpha / std::sqrt((float)c.lora_rank);
  d.mask_from = (int)std::floor((double)c.loss_from * c.T);
  d.nl = d.T - d.mask_from;
  d.BTL = (long)d.B * d.nl;
  return d;
}

// Group geometry: projections, input width, output widths of the projections.
struct GroupGeom { int n, in; int out[3]; int out_total; };
GroupGeom group_geom(const Dims& d, int g) {
  switch (g) {
    case G_QKV: return {3, d.C, {d.QD, d.KVD, d.KVD}, d.QKVD};
    case G_O: return {1, d.QD, {d.C, 0, 0}, d.C};
    case G_GU: return {2, d.C, {d.F, d.F, 0}, 2 * d.F};
    default: return {1, d.F, {d.C, 0, 0}, d.C};
  }
}
const char* group_name(int g) {
  static const char* n[] = {"qkv", "o", "gate_up", "down"};
  return n[g];
}

// ---------------------------------------------------------------- layouts
enum BaseKind { B_EMBED, B_IN_NORM, B_QKV, B_QNORM, B_KNORM, B_O, B_POST_NORM, B_GU, B_DOWN, B_FINAL_NORM, B_NKIND };
const char* base_name(int k) {
  static const char* n[] = {"embed", "in_norm", "qkv", "q_norm", "k_norm", "o", "post_norm", "gate_up", "down",
                            "final_norm"};
  return n[k];
}

struct Shape { int nd; int s[3]; };
Shape base_shape(const Dims& d, int k) {
  switch (k) {
    case B_EMBED: return {2, {d.V, d.C, 0}};
    case B_IN_NORM: return {2, {d.L, d.C, 0}};
    case B_QKV: return {3, {d.L, d.QKVD, d.C}};
    case B_QNORM: return {2, {d.L, d.hd, 0}};
    case B_KNORM: return {2, {d.L, d.hd, 0}};
    case B_O: return {3, {d.L, d.C, d.QD}};
    case B_POST_NORM: return {2, {d.L, d.C, 0}};
    case B_GU: return {3, {d.L, 2 * d.F, d.C}};
    case B_DOWN: return {3, {d.L, d.C, d.F}};
    default: return {1, {d.C, 0, 0}};
  }
}
size_t numel(const Shape& s) {
  size_t n = 1;
  for (int i = 0; i < s.nd; ++i) n *= (size_t)s.s[i];
  return n;
}

struct LoraTensor { int group; bool is_b; Shape shape; size_t off; };

std::vector<LoraTensor> lora_layout(const Dims& d, size_t* total) {
  std::vector<LoraTensor> t;
  size_t o = 0;
  for (int g = 0; g < G_N; ++g) {
    if (!(d.groups & (1 << g))) continue;
    const GroupGeom gg = group_geom(d, g);
    Shape a{3, {d.L, gg.n * RP, gg.in}}, b{3, {d.L, gg.out_total, RP}};
    t.push_back({g, false, a, o});
    o += numel(a);
    t.push_back({g, true, b, o});
    o += numel(b);
  }
  if (total) *total = o;
  return t;
}

struct ActLayout {
  size_t res, h, r1, raw, rq, rk, packed, lse, att, xmid, h2, r2, gu, m, u[G_N];
  size_t xf, rf, logits, losses, loss, total;
  size_t s_act, s_row, s_raw, s_rq, s_rk, s_packed, s_lse, s_att, s_gu, s_m, s_u[G_N];
};

ActLayout act_layout(const Dims& d) {
  ActLayout a{};
  const size_t BT = d.BT, L = d.L;
  a.s_act = align_up(BT * d.C * 2);
  a.s_row = align_up(BT * 4);
  a.s_raw = align_up(BT * d.QKVD * 2);
  a.s_rq = align_up(BT * d.H * 4);
  a.s_rk = align_up(BT * d.Hkv * 4);
  a.s_packed = align_up(BT * d.QKVD * 2);
  a.s_lse = align_up((size_t)d.B * d.H * d.T * 4);
  a.s_att = align_up(BT * d.QD * 2);
  a.s_gu = align_up(BT * 2 * d.F * 2);
  a.s_m = align_up(BT * d.F * 2);
  size_t o = 0;
  a.res = o; o += (L + 1) * a.s_act;
  a.h = o; o += L * a.s_act;
  a.r1 = o; o += L * a.s_row;
  a.raw = o; o += L * a.s_raw;
  a.rq = o; o += L * a.s_rq;
  a.rk = o; o += L * a.s_rk;
  a.packed = o; o += L * a.s_packed;
  a.lse = o; o += L * a.s_lse;
  a.att = o; o += L * a.s_att;
  a.xmid = o; o += L * a.s_act;
  a.h2 = o; o += L * a.s_act;
  a.r2 = o; o += L * a.s_row;
  a.gu = o; o += L * a.s_gu;
  a.m = o; o += L * a.s_m;
  for (int g = 0; g < G_N; ++g) {
    a.s_u[g] = 0;
    if (d.groups & (1 << g)) a.s_u[g] = align_up(BT * group_geom(d, g).n * RP * 2);
    a.u[g] = o; o += L * a.s_u[g];
  }
  // final norm output and logits: rows of the positions that carry loss only
  a.xf = o; o += align_up((size_t)d.BTL * d.C * 2);
  a.rf = o; o += align_up((size_t)d.BTL * 4);
  a.logits = o; o += align_up((size_t)d.BTL * d.V * 2);
  a.losses = o; o += a.s_row;
  a.loss = o; o += ALIGN;
  a.total = o + TAIL;
  return a;
}

constexpr int DW_SPLITS = 16;   // token-contraction split of the adapter gradients
constexpr int HEAD_SPLITS = 4;  // vocabulary-contraction split of the LM head's input gradient
constexpr int BT_ROWS = 32;     // rows of the transposed B copies: the largest rank

struct WsLayout {
  size_t dres, dh, datt, dpacked, draw, dgu, dm, du, dsum, cosT, sinT, part, part2, sumsq, normcoef, total;
  size_t bt[G_N];   // per adapted group: B transposed, [L][BT_ROWS][out_total] bf16
};

WsLayout ws_layout(const Dims& d) {
  WsLayout w{};
  const size_t BT = d.BT;
  // split partial slices: adapter B gradients [split][out][RP] (or the LM
  // head's input gradient [split][BTL][C]) and adapter A gradients
  // [split][n RP][in]
  size_t part = (size_t)d.BTL * d.C * HEAD_SPLITS, part2 = 0;
  for (int g = 0; g < G_N; ++g) {
    if (!(d.groups & (1 << g))) continue;
    const GroupGeom gg = group_geom(d, g);
    part = std::max(part, (size_t)DW_SPLITS * gg.out_total * RP);
    part2 = std::max(part2, (size_t)DW_SPLITS * gg.n * RP * gg.in);
  }
  size_t o = 0;
  w.dres = o; o += align_up(BT * d.C * 2);
  w.dh = o; o += align_up(BT * d.C * 2);   // also the LM head's input gradient (loss rows)
  w.datt = o; o += align_up(BT * d.QD * 2);
  w.dpacked = o; o += align_up(BT * d.QKVD * 2);
  w.draw = o; o += align_up(BT * d.QKVD * 2);
  w.dgu = o; o += align_up(BT * 2 * d.F * 2);
  w.dm = o; o += align_up(BT * d.F * 2);
  w.du = o; o += align_up(BT * 3 * RP * 2);
  w.dsum = o; o += align_up((size_t)d.B * d.H * d.T * 4);
  w.cosT = o; o += align_up((size_t)d.T * (d.hd / 2) * 4);
  w.sinT = o; o += align_up((size_t)d.T * (d.hd / 2) * 4);
  w.part = o; o += align_up(part * 4);
  w.part2 = o; o += align_up(part2 * 4);
  w.sumsq = o; o += align_up((size_t)sumsq_parts() * 4);
  w.normcoef = o; o += ALIGN;
  for (int g = 0; g < G_N; ++g) {
    w.bt[g] = o;
    if (d.groups & (1 << g)) o += align_up((size_t)d.L * BT_ROWS * group_geom(d, g).out_total * 2);
  }
  w.total = o + TAIL;
  return w;
}

const char* validate(const qwen3_config* c) {
  if (!c) return "null config";
  if (c->n_layer < 1 || c->d_model < 8 || c->n_head < 1 || c->n_kv_head < 1 || c->d_ff < 8 || c->vocab < 8)
    return "non-positive dimension";
  if (c->head_dim != 128) return "head_dim must be 128";
  if (c->n_head % c->n_kv_head) return "n_head must be a multiple of n_kv_head";
  if (c->d_model % 128 || c->d_ff % 128) return "d_model and d_ff must be multiples of 128";
  if (c->vocab % 64) return "vocab must be a multiple of 64";
  if (((long)c->B * c->T) % 64) return "B*T must be a multiple of 64";
  if (c->B < 1 || c->T < 2 || c->T > c->max_seq_len) return "bad B, T or max_seq_len";
  if (c->lora_rank < 1 || c->lora_rank > 32) return "lora_rank must be in 1..32";
  if (c->lora_groups <= 0 || c->lora_groups > 15) return "lora_groups must select at least one adapter group";
  if (!(c->loss_from >= 0.0f && c->loss_from < 1.0f)) return "loss_from must be in [0, 1)";
  if (c->d_model > 2048) return "d_model above 2048";
  const Dims d = dims_of(*c);
  if (d.mask_from >= d.T) return "no position carries loss";
  // 32-bit byte offsets: the largest operands the kernels address
  const size_t big = std::max({(size_t)d.BTL * d.V, (size_t)d.BT * d.QKVD, (size_t)d.V * d.C,
                               (size_t)d.BT * 2 * d.F});
  if ((big + 512 * (size_t)std::max(d.V, 2 * d.F)) * 2 >= (1ull << 32)) return "a buffer exceeds 32-bit offsets";
  return nullptr;
}

}  // namespace

struct qwen3_model {
  qwen3_config cfg;
  Dims d;
  qwen3_buffers buf;
  hipStream_t stream;
  ActLayout act;
  WsLayout ws;
  std::vector<LoraTensor> lt;
  size_t n_lora;
  size_t base_off[B_NKIND];
  bool have_targets = false, have_grads = false;
  int swiglu_fused = 1;   // QWEN3_FUSION_SWIGLU mode
  std::string err;
  ProbeSet<QWEN3_K_COUNT> probes;

  // Launch through f(); bracketed with events when the class's probe is on.
  template <class Fn>
  hipError_t run(int cls, double fl, double by, Fn f) {
    return probes.run(stream, cls, fl, by, f);
  }

  bf16_t* base(int k) { return static_cast<bf16_t*>(buf.base_bf16) + base_off[k]; }
  char* A() { return static_cast<char*>(buf.activations); }
  char* W() { return static_cast<char*>(buf.workspace); }
  bf16_t* ab(size_t off) { return reinterpret_cast<bf16_t*>(A() + off); }
  float* af(size_t off) { return reinterpret_cast<float*>(A() + off); }
  bf16_t* wb(size_t off) { return reinterpret_cast<bf16_t*>(W() + off); }
  float* wf(size_t off) { return reinterpret_cast<float*>(W() + off); }
  bf16_t* res(int l) { return ab(act.res + l * act.s_act); }
  // adapter tensors of a group in a buffer with the adapter layout
  const LoraTensor* lora_t(int g, bool b) const {
    for (const auto& t : lt)
      if (t.group == g && t.is_b == b) return &t;
    return nullptr;
  }
  bool has(int g) const { return d.groups & (1 << g); }
};

namespace {

thread_local std::string g_err;

#define TRY(expr)                                                                     \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess) {                                                           \
      m->err = std::string(#expr) + ": " + hipGetErrorString(e_);                     \
      g_err = m->err;                                                                 \
      return GPT2_ERR_DEVICE;                                                         \
    }                                                                                 \
  } while (0)

// C[M,N] (row stride ldc) = A B with A [M,K] (or [K,M] when a_t) and B [N,K]
// (or [K,N] when b_t), bf16 in, epilogue as in the GPT-2 step. `fl` is the
// product's algorithmic FLOP count for the probes (2 M N K unless the
// contraction or an output dimension is padded).
hipError_t gemm(qwen3_model* m, int cls, double fl, int M, int N, int K, const bf16_t* A, int lda, int a_t,
                const bf16_t* B, int ldb, int b_t, int epi, void* C, int ldc, const bf16_t* residual = nullptr,
                int splits = 1, int k_chunk = 0, long split_stride = 0) {
  GemmArgs g{};
  g.A = A; g.B = B; g.M = M; g.N = N; g.K = K; g.lda = lda; g.ldb = ldb; g.C = C; g.ldc = ldc;
  g.residual = residual; g.splits = splits; g.k_chunk = k_chunk; g.split_stride = split_stride;
  return m->run(cls, fl, 0.0, [&] { return launch_gemm(g, a_t, b_t, epi, m->stream); });
}

double mnk2(double M, double N, double K) { return 2.0 * M * N * K; }

hipError_t run_gemm(qwen3_model* m, int cls, double fl, const GemmArgs& g, int a_t, int b_t, int epi) {
  return m->run(cls, fl, 0.0, [&] { return launch_gemm(g, a_t, b_t, epi, m->stream); });
}

// Frozen projection of group g at layer l: y (row stride ldy) = x W^T
// (+ residual). When the group is adapted, u = s x A^T first (its own small
// GEMM, kept for the backward), and the adapter's up-projection u B^T rides
// in the same GEMM as a second contraction segment, projection j's output
// columns contracting with u's j-th block of RP columns.
hipError_t proj_fwd(qwen3_model* m, int g, int l, const bf16_t* x, const bf16_t* W, bf16_t* y, int ldy,
                    const bf16_t* residual) {
  const Dims& d = m->d;
  const GroupGeom gg = group_geom(d, g);
  GemmArgs a{};
  a.A = x; a.lda = gg.in; a.B = W; a.ldb = gg.in; a.M = (int)d.BT; a.N = gg.out_total; a.K = gg.in;
  a.C = y; a.ldc = ldy; a.residual = residual;
  double fl = mnk2(d.BT, gg.out_total, gg.in);
  if (m->has(g)) {
    const LoraTensor* ta = m->lora_t(g, false);
    const LoraTensor* tb = m->lora_t(g, true);
    const bf16_t* wa = static_cast<const bf16_t*>(m->buf.lora_bf16) + ta->off + (size_t)l * gg.n * RP * gg.in;
    const bf16_t* wb = static_cast<const bf16_t*>(m->buf.lora_bf16) + tb->off + (size_t)l * gg.out_total * RP;
    bf16_t* u = m->ab(m->act.u[g] + l * m->act.s_u[g]);
    const int nu = gg.n * RP;
    // u = s x A^T, one pass over x: the 16-row tiles of each projection's
    // real rank rows of A, padding columns of u written as zeros
    const int ntp = (d.r + 15) / 16;
    LoraRowArgs ra{};
    ra.x = x; ra.ldx = gg.in; ra.M = (int)d.BT; ra.nseg = 1; ra.nts = gg.n * ntp; ra.ntp = ntp; ra.tstride = RP;
    ra.k0[0] = 0; ra.klen[0] = gg.in; ra.col[0] = 0; ra.w[0] = wa; ra.ldw = gg.in;
    ra.s = d.s; ra.y = u; ra.ldy = nu;
    hipError_t e = m->run(QWEN3_K_GEMM_ADAPTER, mnk2(d.BT, gg.n * d.r, gg.in), 0.0,
                          [&] { return launch_lora_rows(ra, m->stream); });
    if (e != hipSuccess) return e;
    a.A2 = u; a.lda2 = nu; a.B2 = wb; a.ldb2 = RP; a.K2 = RP;
    // projection j + 1 starts at output column out[0] + ... + out[j]
    int bound = 0;
    for (int j = 0; j + 1 < gg.n; ++j) {
      bound += gg.out[j];
      a.a2_bound[j] = bound;
    }
    fl += mnk2(d.BT, gg.out_total, d.r);
  }
  return run_gemm(m, QWEN3_K_GEMM_FWD, fl, a, 0, 0, EPI_BF16);
}

// Backward of proj_fwd given the output gradient dy (row stride ldy) and the
// input x: the adapter gradients (when adapted) and, unless dx is null,
// dx = dy W (+ du A with du = s dy_j B_j per projection, as a second
// contraction segment of the same GEMM). The adapter gradients contract over
// the tokens, split DW_SPLITS ways into the partial areas and summed by one
// launch: dB_j = dy_j^T u_j, dA = du^T x.
hipError_t proj_bwd(qwen3_model* m, int g, int l, const bf16_t* dy, int ldy, const bf16_t* x, const bf16_t* W,
                    bf16_t* dx) {
  const Dims& d = m->d;
  const GroupGeom gg = group_geom(d, g);
  const int BT = (int)d.BT, nu = gg.n * RP;
  GemmArgs a{};
  a.A = dy; a.lda = ldy; a.B = W; a.ldb = gg.in; a.M = BT; a.N = gg.in; a.K = gg.out_total;
  a.C = dx; a.ldc = gg.in;
  double fl = mnk2(d.BT, gg.in, gg.out_total);
  if (m->has(g)) {
    const int AD = QWEN3_K_GEMM_ADAPTER;
    const LoraTensor* ta = m->lora_t(g, false);
    const LoraTensor* tb = m->lora_t(g, true);
    const size_t oa = ta->off + (size_t)l * gg.n * RP * gg.in, ob = tb->off + (size_t)l * gg.out_total * RP;
    const bf16_t* wa = static_cast<const bf16_t*>(m->buf.lora_bf16) + oa;
    const bf16_t* u = m->ab(m->act.u[g] + l * m->act.s_u[g]);
    bf16_t* du = m->wb(m->ws.du);
    float* pb = m->wf(m->ws.part);
    float* pa = m->wf(m->ws.part2);
    hipError_t e;
    // du_j = s dy_j B_j ([BT, RP] blocks of du), all projections in one
    // pass over dy: segment j contracts dy's columns of projection j with the
    // transposed copy of B_j (rows = rank, contraction index contiguous)
    {
      const int ntp = (d.r + 15) / 16;
      const bf16_t* bt = m->wb(m->ws.bt[g]) + (size_t)l * BT_ROWS * gg.out_total;
      LoraRowArgs ra{};
      ra.x = dy; ra.ldx = ldy; ra.M = BT; ra.nseg = gg.n; ra.nts = ntp; ra.ntp = ntp; ra.tstride = RP;
      ra.ldw = gg.out_total; ra.s = d.s; ra.y = du; ra.ldy = nu;
      double dfl = 0.0;
      for (int j = 0, col = 0; j < gg.n; col += gg.out[j], ++j) {
        ra.k0[j] = col; ra.klen[j] = gg.out[j]; ra.col[j] = j * RP; ra.w[j] = bt + col;
        dfl += mnk2(d.BT, d.r, gg.out[j]);
      }
      e = m->run(AD, dfl, 0.0, [&] { return launch_lora_rows(ra, m->stream); });
      if (e != hipSuccess) return e;
    }
    int kc = 0;
    const int splits = gemm_split_plan(BT, DW_SPLITS, &kc);
    {
      // dB_j = dy_j^T u_j for every projection in one product over all
      // out_total rows: projection j's rows read u's j-th block of RP columns
      GemmArgs r{};
      r.A = dy; r.lda = ldy; r.B = u; r.ldb = nu; r.M = gg.out_total; r.N = RP; r.K = BT;
      r.C = pb; r.ldc = RP; r.splits = splits; r.k_chunk = kc; r.split_stride = (long)gg.out_total * RP;
      r.b_step = RP;
      int bound = 0;
      for (int j = 0; j + 1 < gg.n; ++j) {
        bound += gg.out[j];
        r.b_bound[j] = bound;
      }
      e = run_gemm(m, AD, mnk2(gg.out_total, d.r, d.BT), r, 1, 1, EPI_F32);
      if (e != hipSuccess) return e;
    }
    // dA = du^T x
    GemmArgs r{};
    r.A = du; r.lda = nu; r.B = x; r.ldb = gg.in; r.M = nu; r.N = gg.in; r.K = BT;
    r.C = pa; r.ldc = gg.in; r.splits = splits; r.k_chunk = kc; r.split_stride = (long)nu * gg.in;
    e = run_gemm(m, AD, mnk2(gg.n * d.r, gg.in, d.BT), r, 1, 1, EPI_F32);
    if (e != hipSuccess) return e;
    const long nb = (long)gg.out_total * RP, na = (long)nu * gg.in;
    e = m->run(QWEN3_K_OTHER, 0.0, 4.0 * (double)(nb + na) * (splits + 1), [&] {
      return launch_reduce_slices2(pb, splits, nb, static_cast<float*>(m->buf.lora_grads) + ob, pa, splits, na,
                                   static_cast<float*>(m->buf.lora_grads) + oa, 0, m->stream);
    });
    if (e != hipSuccess || !dx) return e;
    a.A2 = du; a.lda2 = nu; a.B2 = wa; a.ldb2 = gg.in; a.K2 = nu;
    fl += mnk2(d.BT, gg.in, gg.n * d.r);
  }
  if (!dx) return hipSuccess;
  return run_gemm(m, QWEN3_K_GEMM_DX, fl, a, 0, 1, EPI_BF16);
}

AttnArgs attn_args(qwen3_model* m, int l) {
  const Dims& d = m->d;
  AttnArgs a{};
  a.B = d.B; a.T = d.T; a.H = d.H; a.Hkv = d.Hkv; a.hd = d.hd;
  a.qkv = m->ab(m->act.packed + l * m->act.s_packed);
  a.out = m->ab(m->act.att + l * m->act.s_att);
  a.lse = m->af(m->act.lse + l * m->act.s_lse);
  a.dout = m->wb(m->ws.datt);
  a.dsum = m->wf(m->ws.dsum);
  a.dqkv = m->wb(m->ws.dpacked);
  return a;
}

double attn_fwd_flops(const Dims& d) {
  // causal: q.k and p.v over the key positions j <= i only
  return 4.0 * d.B * d.H * d.hd * ((double)d.T * (d.T + 1) / 2.0);
}

gpt2_status fail(qwen3_model* m, gpt2_status st, const std::string& why) {
  if (m) m->err = why;
  g_err = why;
  return st;
}

}  // namespace

extern "C" {

gpt2_status qwen3_query_sizes(const qwen3_config* cfg, qwen3_sizes* out) {
  if (const char* why = validate(cfg)) return fail(nullptr, GPT2_ERR_INVALID_ARG, why);
  if (!out) return fail(nullptr, GPT2_ERR_INVALID_ARG, "null sizes");
  const Dims d = dims_of(*cfg);
  size_t nb = 0;
  for (int k = 0; k < B_NKIND; ++k) nb += numel(base_shape(d, k));
  size_t nl = 0;
  lora_layout(d, &nl);
  out->base_bf16 = align_up(nb * 2) + TAIL;
  out->lora_f32 = align_up(nl * 4);
  out->lora_grads = align_up(nl * 4);
  out->adam_m = align_up(nl * 4);
  out->adam_v = align_up(nl * 4);
  out->lora_bf16 = align_up(nl * 2) + TAIL;
  out->activations = act_layout(d).total;
  out->workspace = ws_layout(d).total;
  return GPT2_OK;
}

gpt2_status qwen3_tensor_info(const qwen3_config* cfg, int32_t which, int32_t idx, char name[64], size_t* offset,
                              int32_t shape[3], int32_t* ndim) {
  if (const char* why = validate(cfg)) return fail(nullptr, GPT2_ERR_INVALID_ARG, why);
  const Dims d = dims_of(*cfg);
  Shape s{};
  size_t off = 0;
  std::string nm;
  if (which == 0) {
    if (idx < 0 || idx >= B_NKIND) return fail(nullptr, GPT2_ERR_INVALID_ARG, "tensor index out of range");
    for (int k = 0; k < idx; ++k) off += numel(base_shape(d, k));
    s = base_shape(d, idx);
    nm = base_name(idx);
  } else if (which == 1) {
    const auto lt = lora_layout(d, nullptr);
    if (idx < 0 || idx >= (int)lt.size()) return fail(nullptr, GPT2_ERR_INVALID_ARG, "tensor index out of range");
    s = lt[idx].shape;
    off = lt[idx].off;
    nm = std::string(group_name(lt[idx].group)) + (lt[idx].is_b ? "_B" : "_A");
  } else {
    return fail(nullptr, GPT2_ERR_INVALID_ARG, "which must be 0 (base) or 1 (adapters)");
  }
  if (name) std::snprintf(name, 64, "%s", nm.c_str());
  if (offset) *offset = off;
  if (shape)
    for (int i = 0; i < 3; ++i) shape[i] = i < s.nd ? s.s[i] : 0;
  if (ndim) *ndim = s.nd;
  return GPT2_OK;
}

gpt2_status qwen3_init(const qwen3_config* cfg, const qwen3_buffers* bufs, void* hip_stream, qwen3_model** out) {
  if (const char* why = validate(cfg)) return fail(nullptr, GPT2_ERR_INVALID_ARG, why);
  if (!bufs || !out || !bufs->base_bf16 || !bufs->lora_f32 || !bufs->lora_grads || !bufs->adam_m || !bufs->adam_v ||
      !bufs->lora_bf16 || !bufs->activations || !bufs->workspace)
    return fail(nullptr, GPT2_ERR_INVALID_ARG, "null buffer");
  qwen3_model* m = new (std::nothrow) qwen3_model();
  if (!m) return fail(nullptr, GPT2_ERR_DEVICE, "host allocation failed");
  m->cfg = *cfg;
  m->d = dims_of(*cfg);
  m->buf = *bufs;
  m->stream = static_cast<hipStream_t>(hip_stream);
  m->act = act_layout(m->d);
  m->ws = ws_layout(m->d);
  m->lt = lora_layout(m->d, &m->n_lora);
  size_t o = 0;
  for (int k = 0; k < B_NKIND; ++k) {
    m->base_off[k] = o;
    o += numel(base_shape(m->d, k));
  }
  // rotary tables in fp64, stored fp32: angle t * theta^(-2i/hd)
  const Dims& d = m->d;
  std::vector<float> ct((size_t)d.T * (d.hd / 2)), st(ct.size());
  for (int t = 0; t < d.T; ++t)
    for (int i = 0; i < d.hd / 2; ++i) {
      const double ang = (double)t * std::pow((double)cfg->rope_theta, -2.0 * i / d.hd);
      ct[(size_t)t * (d.hd / 2) + i] = (float)std::cos(ang);
      st[(size_t)t * (d.hd / 2) + i] = (float)std::sin(ang);
    }
  hipError_t e = hipMemcpyAsync(m->wf(m->ws.cosT), ct.data(), ct.size() * 4, hipMemcpyHostToDevice, m->stream);
  if (e == hipSuccess)
    e = hipMemcpyAsync(m->wf(m->ws.sinT), st.data(), st.size() * 4, hipMemcpyHostToDevice, m->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(m->stream);   // the host vectors go out of scope
  if (e != hipSuccess) {
    g_err = std::string("rotary tables: ") + hipGetErrorString(e);
    delete m;
    return GPT2_ERR_DEVICE;
  }
  gpt2_status st2 = qwen3_sync_weights(m);
  if (st2 != GPT2_OK) {
    delete m;
    return st2;
  }
  *out = m;
  return GPT2_OK;
}

gpt2_status qwen3_sync_weights(qwen3_model* m) {
  if (!m) return fail(nullptr, GPT2_ERR_INVALID_ARG, "null model");
  TRY(launch_cast_bf16(static_cast<const float*>(m->buf.lora_f32), static_cast<bf16_t*>(m->buf.lora_bf16),
                       (long)m->n_lora, m->stream));
  return GPT2_OK;
}

gpt2_status qwen3_forward(qwen3_model* m, const int32_t* d_inputs, const int32_t* d_targets) {
  if (!m || !d_inputs) return fail(m, GPT2_ERR_INVALID_ARG, "null argument");
  const Dims& d = m->d;
  const int BT = (int)d.BT, BTL = (int)d.BTL;
  const int FWD = QWEN3_K_GEMM_FWD, NORM = QWEN3_K_NORM, OTHER = QWEN3_K_OTHER;
  const double rowb = 2.0 * d.BT * d.C;   // bytes of one bf16 [BT, C] activation
  TRY(m->run(OTHER, 0.0, 2.0 * rowb + 4.0 * d.BT,
             [&] { return launch_embed_gather(d_inputs, m->base(B_EMBED), m->res(0), d.BT, d.C, m->stream); }));
  for (int l = 0; l < d.L; ++l) {
    bf16_t* h = m->ab(m->act.h + l * m->act.s_act);
    float* r1 = m->af(m->act.r1 + l * m->act.s_row);
    bf16_t* raw = m->ab(m->act.raw + l * m->act.s_raw);
    bf16_t* xmid = m->ab(m->act.xmid + l * m->act.s_act);
    bf16_t* h2 = m->ab(m->act.h2 + l * m->act.s_act);
    float* r2 = m->af(m->act.r2 + l * m->act.s_row);
    bf16_t* gu = m->ab(m->act.gu + l * m->act.s_gu);
    bf16_t* mm = m->ab(m->act.m + l * m->act.s_m);
    // attention sub-layer
    TRY(m->run(NORM, 0.0, 2.0 * rowb + 4.0 * d.BT, [&] {
      return launch_rmsnorm_fwd(m->res(l), m->base(B_IN_NORM) + (size_t)l * d.C, h, r1, BT, d.C, m->cfg.rms_eps, 1, 0,
                                m->stream);
    }));
    TRY(proj_fwd(m, G_QKV, l, h, m->base(B_QKV) + (size_t)l * d.QKVD * d.C, raw, d.QKVD, nullptr));
    AttnArgs aa = attn_args(m, l);
    TRY(m->run(NORM, 0.0, 4.0 * d.BT * d.QKVD + 4.0 * d.BT * (d.H + d.Hkv), [&] {
      return launch_qknorm_rope_fwd(raw, m->base(B_QNORM) + (size_t)l * d.hd, m->base(B_KNORM) + (size_t)l * d.hd,
                                    m->wf(m->ws.cosT), m->wf(m->ws.sinT), const_cast<bf16_t*>(aa.qkv),
                                    m->af(m->act.rq + l * m->act.s_rq), m->af(m->act.rk + l * m->act.s_rk), BT, d.T,
                                    d.H, d.Hkv, d.hd, m->cfg.rms_eps, m->stream);
    }));
    TRY(m->run(QWEN3_K_ATTN_FWD, attn_fwd_flops(d), 0.0, [&] { return launch_attention_fwd(aa, m->stream); }));
    TRY(proj_fwd(m, G_O, l, aa.out, m->base(B_O) + (size_t)l * d.C * d.QD, xmid, d.C, m->res(l)));
    // MLP sub-layer
    TRY(m->run(NORM, 0.0, 2.0 * rowb + 4.0 * d.BT, [&] {
      return launch_rmsnorm_fwd(xmid, m->base(B_POST_NORM) + (size_t)l * d.C, h2, r2, BT, d.C, m->cfg.rms_eps, 1, 0,
                                m->stream);
    }));
    if (m->swiglu_fused && !m->has(G_GU)) {
      // gate|up projection with the SwiGLU in its epilogue: writes the
      // pre-activation (kept for the backward) and the output
      GemmArgs a{};
      a.A = h2; a.lda = d.C; a.B = m->base(B_GU) + (size_t)l * 2 * d.F * d.C; a.ldb = d.C;
      a.M = BT; a.N = 2 * d.F; a.K = d.C; a.C = gu; a.ldc = 2 * d.F; a.C2 = mm;
      TRY(run_gemm(m, FWD, mnk2(d.BT, 2 * d.F, d.C), a, 0, 0, EPI_SWIGLU));
    } else {
      TRY(proj_fwd(m, G_GU, l, h2, m->base(B_GU) + (size_t)l * 2 * d.F * d.C, gu, 2 * d.F, nullptr));
      TRY(m->run(OTHER, 0.0, 6.0 * d.BT * d.F, [&] { return launch_swiglu_fwd(gu, mm, d.BT, d.F, m->stream); }));
    }
    TRY(proj_fwd(m, G_DN, l, mm, m->base(B_DOWN) + (size_t)l * d.C * d.F, m->res(l + 1), d.C, xmid));
  }
  // final norm and LM head on the positions that carry loss (compacted rows)
  bf16_t* xf = m->ab(m->act.xf);
  TRY(m->run(NORM, 0.0, 4.0 * d.BTL * d.C + 4.0 * d.BTL, [&] {
    return launch_rmsnorm_fwd(m->res(d.L), m->base(B_FINAL_NORM), xf, m->af(m->act.rf), BTL, d.C, m->cfg.rms_eps, d.T,
                              d.mask_from, m->stream);
  }));
  bf16_t* logits = m->ab(m->act.logits);
  TRY(gemm(m, FWD, mnk2(BTL, d.V, d.C), BTL, d.V, d.C, xf, d.C, 0, m->base(B_EMBED), d.C, 0, EPI_BF16, logits, d.V));
  m->have_targets = d_targets != nullptr;
  if (d_targets) {
    const float inv_n = 1.0f / (float)d.BTL;   // mean over the positions with loss
    TRY(m->run(QWEN3_K_CROSS_ENTROPY, 0.0, 4.0 * d.BTL * d.V + 12.0 * d.BT, [&] {
      return launch_cross_entropy_masked(logits, d_targets, m->af(m->act.losses), BTL, d.V, d.V, inv_n, 1, d.T,
                                         d.mask_from, m->stream);
    }));
    TRY(m->run(OTHER, 0.0, 4.0 * d.BT,
               [&] { return launch_sum_scaled(m->af(m->act.losses), BT, inv_n, m->af(m->act.loss), m->stream); }));
  }
  return GPT2_OK;
}

gpt2_status qwen3_backward(qwen3_model* m) {
  if (!m) return fail(nullptr, GPT2_ERR_INVALID_ARG, "null model");
  if (!m->have_targets) return fail(m, GPT2_ERR_STATE, "backward needs a forward with targets");
  const Dims& d = m->d;
  const int BT = (int)d.BT, BTL = (int)d.BTL;
  const int DX = QWEN3_K_GEMM_DX, NORM = QWEN3_K_NORM;
  const double rowb = 2.0 * d.BT * d.C;
  bf16_t* dres = m->wb(m->ws.dres);
  bf16_t* dh = m->wb(m->ws.dh);
  // transposed copies of every adapted group's B (all layers), read by the
  // du products
  for (int g = 0; g < G_N; ++g) {
    if (!m->has(g)) continue;
    const int out = group_geom(d, g).out_total;
    const bf16_t* b = static_cast<const bf16_t*>(m->buf.lora_bf16) + m->lora_t(g, true)->off;
    TRY(m->run(QWEN3_K_OTHER, 0.0, 4.0 * d.L * BT_ROWS * out,
               [&] { return launch_lora_bt(b, m->wb(m->ws.bt[g]), d.L, out, RP, m->stream); }));
  }
  // LM head: dxf = dlogits embed over the loss rows, the long vocabulary
  // contraction split so that the few output tiles fill the GPU, then the
  // final RMSNorm (rows without loss get a zero gradient)
  {
    int kc = 0;
    const int splits = gemm_split_plan(d.V, HEAD_SPLITS, &kc);
    float* part = m->wf(m->ws.part);
    TRY(gemm(m, DX, mnk2(BTL, d.C, d.V), BTL, d.C, d.V, m->ab(m->act.logits), d.V, 0, m->base(B_EMBED), d.C, 1,
             EPI_F32, part, d.C, nullptr, splits, kc, (long)d.BTL * d.C));
    TRY(m->run(QWEN3_K_OTHER, 0.0, (4.0 * splits + 2.0) * d.BTL * d.C,
               [&] { return launch_reduce_slices_bf16(part, splits, d.BTL * d.C, 1.0f, dh, m->stream); }));
  }
  TRY(m->run(NORM, 0.0, 2.0 * rowb + 4.0 * d.BTL * d.C + 4.0 * d.BTL, [&] {
    return launch_rmsnorm_bwd(dh, m->res(d.L), m->af(m->act.rf), m->base(B_FINAL_NORM), dres, 0, BT, d.C, d.T,
                              d.mask_from, m->stream);
  }));
  for (int l = d.L - 1; l >= 0; --l) {
    const bf16_t* h = m->ab(m->act.h + l * m->act.s_act);
    const float* r1 = m->af(m->act.r1 + l * m->act.s_row);
    const bf16_t* raw = m->ab(m->act.raw + l * m->act.s_raw);
    const bf16_t* xmid = m->ab(m->act.xmid + l * m->act.s_act);
    const bf16_t* h2 = m->ab(m->act.h2 + l * m->act.s_act);
    const float* r2 = m->af(m->act.r2 + l * m->act.s_row);
    const bf16_t* gu = m->ab(m->act.gu + l * m->act.s_gu);
    const bf16_t* mm = m->ab(m->act.m + l * m->act.s_m);
    bf16_t* dm = m->wb(m->ws.dm);
    bf16_t* dgu = m->wb(m->ws.dgu);
    // down projection: res(l+1) = xmid + m down^T (+ adapter)
    if (m->swiglu_fused && !m->has(G_DN)) {
      // no adapter: only its input gradient, with the SwiGLU backward in the
      // epilogue (dgu from the gradient of m and the saved pre-activation)
      GemmArgs a{};
      a.A = dres; a.lda = d.C; a.B = m->base(B_DOWN) + (size_t)l * d.C * d.F; a.ldb = d.F;
      a.M = BT; a.N = d.F; a.K = d.C; a.C = dgu; a.ldc = 2 * d.F; a.aux = gu;
      TRY(run_gemm(m, DX, mnk2(d.BT, d.F, d.C), a, 0, 1, EPI_SWIGLU_BWD));
    } else {
      TRY(proj_bwd(m, G_DN, l, dres, d.C, mm, m->base(B_DOWN) + (size_t)l * d.C * d.F, dm));
      TRY(m->run(QWEN3_K_OTHER, 0.0, 10.0 * d.BT * d.F,
                 [&] { return launch_swiglu_bwd(dm, gu, dgu, d.BT, d.F, m->stream); }));
    }
    TRY(proj_bwd(m, G_GU, l, dgu, 2 * d.F, h2, m->base(B_GU) + (size_t)l * 2 * d.F * d.C, dh));
    TRY(m->run(NORM, 0.0, 4.0 * rowb + 4.0 * d.BT, [&] {
      return launch_rmsnorm_bwd(dh, xmid, r2, m->base(B_POST_NORM) + (size_t)l * d.C, dres, 1, BT, d.C, 1, 0,
                                m->stream);
    }));
    // attention output projection: xmid = res(l) + att o^T (+ adapter)
    AttnArgs aa = attn_args(m, l);
    bf16_t* datt = m->wb(m->ws.datt);
    TRY(proj_bwd(m, G_O, l, dres, d.C, aa.out, m->base(B_O) + (size_t)l * d.C * d.QD, datt));
    TRY(m->run(QWEN3_K_ATTN_BWD, 2.0 * attn_fwd_flops(d), 0.0, [&] { return launch_attention_bwd(aa, m->stream); }));
    bf16_t* draw = m->wb(m->ws.draw);
    TRY(m->run(NORM, 0.0, 6.0 * d.BT * d.QKVD + 4.0 * d.BT * (d.H + d.Hkv), [&] {
      return launch_qknorm_rope_bwd(m->wb(m->ws.dpacked), raw, m->base(B_QNORM) + (size_t)l * d.hd,
                                    m->base(B_KNORM) + (size_t)l * d.hd, m->wf(m->ws.cosT), m->wf(m->ws.sinT),
                                    m->af(m->act.rq + l * m->act.s_rq), m->af(m->act.rk + l * m->act.s_rk), draw, BT,
                                    d.T, d.H, d.Hkv, d.hd, m->stream);
    }));
    // the first layer's input gradient would only reach the frozen token
    // table: its q|k|v input gradient and the norm behind it are skipped
    const bool need_dx = l > 0;
    TRY(proj_bwd(m, G_QKV, l, draw, d.QKVD, h, m->base(B_QKV) + (size_t)l * d.QKVD * d.C, need_dx ? dh : nullptr));
    if (need_dx)
      TRY(m->run(NORM, 0.0, 4.0 * rowb + 4.0 * d.BT, [&] {
        return launch_rmsnorm_bwd(dh, m->res(l), r1, m->base(B_IN_NORM) + (size_t)l * d.C, dres, 1, BT, d.C, 1, 0,
                                  m->stream);
      }));
  }
  m->have_grads = true;
  return GPT2_OK;
}

gpt2_status qwen3_adamw_step(qwen3_model* m, int64_t step, float* d_grad_norm_out) {
  if (!m) return fail(nullptr, GPT2_ERR_INVALID_ARG, "null model");
  if (!m->have_grads) return fail(m, GPT2_ERR_STATE, "optimizer step needs a backward");
  if (step < 0) return fail(m, GPT2_ERR_INVALID_ARG, "negative step");
  const qwen3_config& c = m->cfg;
  const long n = (long)m->n_lora;
  float* grads = static_cast<float*>(m->buf.lora_grads);
  float* parts = m->wf(m->ws.sumsq);
  float* nc = m->wf(m->ws.normcoef);
  const int OPT = QWEN3_K_OPTIMIZER;
  TRY(m->run(OPT, 0.0, 4.0 * n, [&] { return launch_sumsq(grads, n, parts, m->stream); }));
  TRY(m->run(OPT, 0.0, 4.0 * sumsq_parts(),
             [&] { return launch_clip_coef(parts, sumsq_parts(), c.grad_clip, nc, m->stream); }));
  if (d_grad_norm_out) TRY(hipMemcpyAsync(d_grad_norm_out, nc, sizeof(float), hipMemcpyDeviceToDevice, m->stream));
  AdamArgs a{};
  a.p = static_cast<float*>(m->buf.lora_f32);
  a.g = grads;
  a.m = static_cast<float*>(m->buf.adam_m);
  a.v = static_cast<float*>(m->buf.adam_v);
  a.p_bf16 = static_cast<bf16_t*>(m->buf.lora_bf16);
  a.norm_coef = nc;
  a.n = n;
  a.lr = c.lr;
  a.beta1 = c.beta1; a.beta2 = c.beta2; a.eps = c.adam_eps; a.weight_decay = c.weight_decay;
  a.bc1 = (float)(1.0 - std::pow((double)c.beta1, (double)(step + 1)));
  a.bc2 = (float)(1.0 - std::pow((double)c.beta2, (double)(step + 1)));
  a.seg.count = 1;
  a.seg.end[0] = n;
  a.seg.decay[0] = 1;   // the configured decay applies to every adapter tensor (all are 2-D)
  TRY(m->run(OPT, 0.0, 30.0 * n, [&] { return launch_adamw(a, m->stream); }));
  m->have_grads = false;
  return GPT2_OK;
}

gpt2_status qwen3_loss(qwen3_model* m, float* loss_out, float* d_token_losses) {
  if (!m || !loss_out) return fail(m, GPT2_ERR_INVALID_ARG, "null argument");
  if (!m->have_targets) return fail(m, GPT2_ERR_STATE, "no forward with targets");
  if (d_token_losses)
    TRY(hipMemcpyAsync(d_token_losses, m->af(m->act.losses), (size_t)m->d.BT * 4, hipMemcpyDeviceToDevice,
                       m->stream));
  TRY(hipMemcpyAsync(loss_out, m->af(m->act.loss), 4, hipMemcpyDeviceToHost, m->stream));
  TRY(hipStreamSynchronize(m->stream));
  return GPT2_OK;
}

gpt2_status qwen3_set_fusion(qwen3_model* m, int32_t fusion, int32_t mode) {
  if (!m) return GPT2_ERR_INVALID_ARG;
  if (fusion == QWEN3_FUSION_SWIGLU) {
    if (mode < 0 || mode > 1) return fail(m, GPT2_ERR_INVALID_ARG, "SwiGLU mode must be 0 or 1");
    m->swiglu_fused = mode;
    return GPT2_OK;
  }
  return fail(m, GPT2_ERR_INVALID_ARG, "unknown fusion");
}

void qwen3_destroy(qwen3_model* m) { delete m; }

const char* qwen3_last_error(const qwen3_model* m) { return m ? m->err.c_str() : g_err.c_str(); }

gpt2_status qwen3_probe_enable(qwen3_model* m, uint32_t class_mask) {
  if (!m) return fail(nullptr, GPT2_ERR_INVALID_ARG, "null model");
  m->probes.mask = class_mask;
  return GPT2_OK;
}

gpt2_status qwen3_probe_reset(qwen3_model* m) {
  if (!m) return fail(nullptr, GPT2_ERR_INVALID_ARG, "null model");
  if (m->probes.reset() != hipSuccess) return fail(m, GPT2_ERR_DEVICE, "event sync failed");
  return GPT2_OK;
}

gpt2_status qwen3_probe_read(qwen3_model* m, int32_t kclass, double* total_ms, int64_t* launches, double* flops,
                             double* bytes) {
  if (!m) return fail(nullptr, GPT2_ERR_INVALID_ARG, "null model");
  if (kclass < 0 || kclass >= QWEN3_K_COUNT) return fail(m, GPT2_ERR_INVALID_ARG, "bad kernel class");
  if (m->probes.collect() != hipSuccess) return fail(m, GPT2_ERR_DEVICE, "event timing failed");
  if (total_ms) *total_ms = m->probes.ms[kclass];
  if (launches) *launches = m->probes.launches[kclass];
  if (flops) *flops = m->probes.flops[kclass];
  if (bytes) *bytes = m->probes.bytes[kclass];
  return GPT2_OK;
}

}  // extern "C"
