// Causal multi-head attention for gfx950, flash style: the score matrix never
// leaves the chip; softmax is computed online in the forward pass and
// recomputed from the saved log-sum-exp in the backward pass.
//
// Layout: q|k|v packed per token [B*T, 3C], head h on channels
// [h*hd, (h+1)*hd) of each third; output [B*T, C]; log-sum-exp of the scaled
// scores [B, H, T] in fp32.
//
// Every product is v_mfma_f32_32x32x16_bf16. Tiles of 64 rows x hd move from
// HBM straight into LDS (buffer_load ... lds, double-buffered: the next tile
// loads while the current one is used) and stay in their natural row-major
// layout; operands that need the other orientation are read with
// ds_read_b64_tr_b16. Scores are arranged so that probabilities (and their
// gradients) are consumed by the next MFMA straight from the accumulator
// registers: an MFMA only needs its two operands to agree on which
// contraction index sits in each of a lane's 8 slots, and the register order
// of a 32x32 accumulator (rows 8*(r/4) + 4*(lane/32) + r%4) is matched by
// reading the other operand in that order.
//
//   forward: per 128 queries (4 waves x 32), walk key tiles: S^T = K Q^T
//            (one query per lane, so the running max and sum are lane-local up
//            to an exchange with lane^32), O^T += V^T P^T. The softmax takes
//            the max over the raw scores and folds the scale into the
//            exponential's argument (one fma, one exp2 per score); the shift
//            it subtracts only moves when a lane's tile max exceeds it by more
//            than RESCALE_SLACK (log2 units), so the output accumulators are
//            rescaled on few tiles. Softmax does not depend on the shift, and
//            probabilities stay below 2^RESCALE_SLACK.
//   dQ:      per 128 queries, walk key tiles: recompute P^T, dP^T = V dO^T,
//            dS^T = P^T (dP^T - D), dQ^T += K^T dS^T. D = rowsum(dO * O) is
//            computed here from the query's dO and O rows and stored.
//   dK, dV:  per 128 keys (4 waves x 32), walk query tiles from the diagonal:
//            S = Q K^T, dP = dO V^T (one key per lane), dV^T += dO^T P,
//            dK^T += Q^T dS; runs after dQ, reading the stored D.
// Grouped-query attention: a key/value head serves H / Hkv query heads; the
// forward and dQ kernels read the key/value head of their query head, and a
// dK/dV workgroup walks the query tiles of every query head of its group.
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "lds_dma.h"

namespace {

constexpr int TILE = 64;    // rows per LDS tile (keys or queries)
typedef float v4f32 __attribute__((ext_vector_type(4)));
typedef LDS_AS v4f32 lds_v4f32_t;
constexpr int BQ = 128;     // rows owned by one workgroup (4 waves x 32)
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
constexpr float RESCALE_SLACK = 8.0f;

// 2^x with the bare hardware instruction: softmax arguments are at most
// RESCALE_SLACK (forward) or 0 (backward), and results below 2^-126 are
// negligible against the row maximum's term of at least 1
DEV float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

DEV int bitrev3(int x) { return ((x & 1) << 2) | (x & 2) | ((x >> 2) & 1); }
DEV int bitrev4(int x) { return ((x & 1) << 3) | ((x & 2) << 1) | ((x >> 1) & 2) | ((x >> 3) & 1); }

// Physical 16-byte unit of (row, chunk) in a [64][HD] tile. The XOR keeps
// both access patterns free of bank conflicts: 32 lanes reading 16 bytes of
// 32 consecutive rows at one chunk, and 32 lanes of transposed reads covering
// 4 consecutive rows x 4 chunks.
template <int HD>
DEV int unit(int row, int c) {
  constexpr int U = HD / 8;
  int f = 0;
  if constexpr (U == 16) f = bitrev4(row & 15);
  else if constexpr (U == 8) f = bitrev3((row >> 1) & 7);
  else if constexpr (U == 4) f = (row >> 2) & 3;
  return row * U + (c ^ f);
}

// Loads rows [r0, r0+64) of one head's slice (row stride ld elements) of a
// buffer into an LDS tile. Instruction i of the tile goes to bytes
// [1024 i, 1024 i + 1024); waves take instructions in turn. A lane's byte
// offset within the tile's rows is the same for every tile, so it is
// computed once; a tile adds only its (scalar) starting offset.
template <int HD>
struct RowLoader {
  static constexpr int U = HD / 8, UNITS = TILE * U, INSTR = (UNITS + 63) / 64, PER = (INSTR + 3) / 4;
  uint32_t rel[PER];

  DEV void init(int ld, int wave, int lane) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int u = (wave + 4 * i) * 64 + lane;
      const int row = u / U, p = u % U;
      const int c = unit<HD>(row, p) - row * U;   // the XOR is its own inverse
      rel[i] = ((uint32_t)row * (uint32_t)ld + (uint32_t)(c * 8)) * 2u;
    }
  }

  // off: byte offset in the buffer of row r0 of the head's slice
  DEV void issue(v4i32 rs, uint32_t off, lds_char_t* dst, int wave, int lane) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int ins = wave + 4 * i;
      if (ins < INSTR && (UNITS % 64 == 0 || ins * 64 + lane < UNITS))
        dma16(rs, off + rel[i], lds_addr(dst + ins * 1024));
    }
  }
};

// The same load with the lane offsets recomputed per tile (for kernels whose
// registers are at the limit). src: row 0 of the head's slice.
template <int HD>
DEV void issue_rows(v4i32 rs, const bf16_t* base_of_buffer, const bf16_t* src, int r0, int ld, lds_char_t* dst,
                    int wave, int lane) {
  constexpr int U = HD / 8, UNITS = TILE * U, INSTR = (UNITS + 63) / 64;
  const uint32_t src_off = (uint32_t)((src - base_of_buffer) * 2);
  for (int ins = wave; ins < INSTR; ins += 4) {
    const int u = ins * 64 + lane;
    const int row = u / U, p = u % U;
    const int c = unit<HD>(row, p) - row * U;   // the XOR is its own inverse
    const uint32_t off = src_off + ((uint32_t)(r0 + row) * (uint32_t)ld + (uint32_t)(c * 8)) * 2u;
    if (UNITS % 64 == 0 || u < UNITS) dma16(rs, off, lds_addr(dst + ins * 1024));
  }
}

// 8 contraction values of tile row (row) at chunk c (a natural-layout operand).
template <int HD>
DEV bf16x8 read_row(const lds_char_t* t, int row, int c) {
  return lds_read16(t + unit<HD>(row, c) * 16);
}

// Transposed operand from a [64][HD] tile: lane gets column n = d0 +
// lane%32 at tile rows kb + {0..3} (slots 0..3) and kb + 8 + {0..3} (slots
// 4..7), where kb = rbase + 4*(lane/32) -- the register order of a 32x32
// accumulator over rows rbase..rbase+15.
template <int HD>
DEV bf16x8 read_tr(const lds_char_t* t, int d0, int rbase, int lane) {
  const int s = lane & 15, h = (lane >> 4) & 1, g = lane >> 5;
  // for hd 16 the upper 16 output rows of the 32-row MFMA tile are never
  // stored; their columns are folded back into the tile
  const int n = (d0 + 16 * h + 4 * (s & 3)) & (HD < 32 ? HD - 1 : 0x7fffffff);
  const int kb = rbase + 4 * g + (s >> 2);
  const int c = n >> 3, sub = (n & 7) * 2;
  const uint2 a = lds_read_tr(t + unit<HD>(kb, c) * 16 + sub);
  const uint2 b = lds_read_tr(t + unit<HD>(kb + 8, c) * 16 + sub);
  return as_bf16x8(make_uint4(a.x, a.y, b.x, b.y));
}

// Registers 8h..8h+7 of a 32x32 fp32 accumulator as a bf16 operand.
DEV bf16x8 acc_slots(const floatx16& x, int h) {
  return as_bf16x8(make_uint4(pack2(x[8 * h + 0], x[8 * h + 1]), pack2(x[8 * h + 2], x[8 * h + 3]),
                              pack2(x[8 * h + 4], x[8 * h + 5]), pack2(x[8 * h + 6], x[8 * h + 7])));
}

// accumulator register r of lane group g sits at row 8*(r/4) + 4g + r%4
DEV int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

DEV void zero(floatx16& x) {
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] = 0.0f;
}

template <int HD>
struct Shape {
  static constexpr int KS = HD / 16;                 // k-steps over the head dim
  static constexpr int DT = HD < 32 ? 1 : HD / 32;   // 32-row tiles over the head dim
  static constexpr int TB = TILE * HD * 2;           // bytes of one tile
  static constexpr int TBA = (TB + 1023) / 1024 * 1024;
};

// ------------------------------------------------------------------ forward

template <int HD>
__global__ __launch_bounds__(256, 2) void attn_fwd_kernel(AttnArgs a) {
  using S = Shape<HD>;
  __shared__ __attribute__((aligned(1024))) char smem_raw[2 * 2 * S::TBA];   // 2 stages x (K, V)
  lds_char_t* smem = (lds_char_t*)smem_raw;
  const int T = a.T, H = a.H, C = H * HD, Hkv = a.Hkv > 0 ? a.Hkv : H, ld = (H + 2 * Hkv) * HD;
  // 1-D grid, head fastest: every head's heaviest (last) query block is
  // dispatched first, then the next heaviest of every head, and so on, so the
  // causal imbalance leaves no long blocks for the end; and with B*H a
  // multiple of 8 all blocks of a head land on one XCD (blocks are dealt to
  // the 8 XCDs round-robin)
  const int BH = a.B * H, nqb = (T + BQ - 1) / BQ;
  const int bh = blockIdx.x % BH, b = bh / H, h = bh % H;
  const int qb = nqb - 1 - (int)(blockIdx.x / BH);
  // the wave index is uniform across the wave: say so, so that per-wave
  // conditions compile to scalar branches
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lq = lane & 31, g = lane >> 5;
  const int q0w = qb * BQ + wave * 32;
  const int q = q0w + lq;
  const bf16_t* base = a.qkv + (size_t)b * T * ld + h * HD;
  const bf16_t* kbase = a.qkv + (size_t)b * T * ld + (H + h / (H / Hkv)) * HD;
  const v4i32 rs = make_rsrc(a.qkv, (uint32_t)((size_t)a.B * T * ld * 2));

  bf16x8 qf[S::KS];
#pragma unroll
  for (int s = 0; s < S::KS; ++s) {
    uint4 v = make_uint4(0, 0, 0, 0);
    if (q < T) v = *reinterpret_cast<const uint4*>(base + (size_t)q * ld + 16 * s + 8 * g);
    qf[s] = as_bf16x8(v);
  }
  floatx16 o[S::DT];
#pragma unroll
  for (int d = 0; d < S::DT; ++d) zero(o[d]);
  float m_run = -INFINITY, l_run = 0.0f;
  const float sc = LOG2E / sqrtf((float)HD);

  const int kv_end = min(T, qb * BQ + BQ);
  const int ntiles = (kv_end + TILE - 1) / TILE;
  // the lane offsets of the K/V loads computed once (at hd 128 the registers
  // they take cost more than recomputing them per tile)
  RowLoader<HD> kvl;
  if constexpr (HD < 128) kvl.init(ld, wave, lane);
  const uint32_t koff = (uint32_t)((kbase - a.qkv) * 2), voff = koff + (uint32_t)(Hkv * HD * 2);
  auto issue = [&](int it) {
    lds_char_t* st = smem + (it & 1) * 2 * S::TBA;
    if constexpr (HD < 128) {
      const uint32_t r = (uint32_t)(it * TILE) * (uint32_t)ld * 2u;
      kvl.issue(rs, koff + r, st, wave, lane);
      kvl.issue(rs, voff + r, st + S::TBA, wave, lane);
    } else {
      issue_rows<HD>(rs, a.qkv, kbase, it * TILE, ld, st, wave, lane);
      issue_rows<HD>(rs, a.qkv, kbase + Hkv * HD, it * TILE, ld, st + S::TBA, wave, lane);
    }
  };
  issue(0);
  for (int it = 0; it < ntiles; ++it) {
    wait_vmcnt<0>();
    block_barrier();
    if (it + 1 < ntiles) issue(it + 1);
    const int kv0 = it * TILE;
    if (kv0 > q0w + 31) continue;   // every query of this wave precedes the tile
    const lds_char_t* Ks = smem + (it & 1) * 2 * S::TBA;
    const lds_char_t* Vs = Ks + S::TBA;

    floatx16 s[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      zero(s[t]);
#pragma unroll
      for (int k = 0; k < S::KS; ++k) s[t] = mfma32(read_row<HD>(Ks, 32 * t + lq, 2 * k + g), qf[k], s[t]);
    }
    // only tiles that straddle the diagonal or the sequence end are masked
    const bool diag = kv0 + TILE - 1 > q0w || kv0 + TILE > T;
    float mt = -INFINITY;
    auto mask_max = [&](auto masked) {
      const int jmax = min(q, T - 1) - kv0 - 4 * g;   // key j = kv0 + 4g + offset is kept if offset <= jmax
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float x = s[t][r];
          if constexpr (decltype(masked)::value) x = (32 * t + acc_row(r, 0) <= jmax) ? x : -INFINITY;
          s[t][r] = x;
          mt = fmaxf(mt, x);
        }
    };
    if (diag) mask_max(std::true_type{});
    else mask_max(std::false_type{});
    mt = fmaxf(mt, __shfl_xor(mt, 32, WAVE)) * sc;
    // key 0 is visible to every query, so after tile 0 the shift is finite
    const bool grow = mt > m_run + RESCALE_SLACK;
    if (__ballot(grow) != 0) {
      const float alpha = grow ? fast_exp2(m_run - mt) : 1.0f;
      m_run = grow ? mt : m_run;
      l_run *= alpha;
#pragma unroll
      for (int d = 0; d < S::DT; ++d)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[d][r] *= alpha;
    }
    float rsum = 0.0f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = fast_exp2(fmaf(s[t][r], sc, -m_run));
        s[t][r] = p;
        rsum += p;
      }
    l_run += rsum + __shfl_xor(rsum, 32, WAVE);
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const bf16x8 pf = acc_slots(s[t], hh);
#pragma unroll
        for (int d = 0; d < S::DT; ++d) o[d] = mfma32(read_tr<HD>(Vs, 32 * d, 32 * t + 16 * hh, lane), pf, o[d]);
      }
  }

  if (q < T) {
    const float inv = 1.0f / l_run;
    bf16_t* out = a.out + ((size_t)b * T + q) * C + h * HD;
#pragma unroll
    for (int d = 0; d < S::DT; ++d)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int dd = 32 * d + 8 * c + 4 * g;
        if (dd < HD)
          *reinterpret_cast<uint2*>(out + dd) = make_uint2(pack2(o[d][4 * c] * inv, o[d][4 * c + 1] * inv),
                                                           pack2(o[d][4 * c + 2] * inv, o[d][4 * c + 3] * inv));
      }
    if (g == 0) a.lse[(size_t)bh * T + q] = (m_run + log2f(l_run)) * LN2;
  }
}

// ------------------------------------------------------------------ backward

// D[b,h,t] = sum_d dO * O, one thread per (token, head)
// dK, dV for 128 keys (4 waves x 32), walking query tiles of 64 from the
// diagonal to the end.
// At hd 128 one workgroup per CU: the K/V fragments and the dK/dV
// accumulators alone take 192 registers per lane, so the kernel needs the
// accumulation registers that a single wave per SIMD may use (with two per
// SIMD it spilled to scratch and ran 2.5x slower).
template <int HD>
__global__ __launch_bounds__(256, HD >= 128 ? 1 : 2) void attn_bwd_dkdv_kernel(AttnArgs a) {
  using S = Shape<HD>;
  constexpr int STAGE = 2 * S::TBA + 1024;   // Q tile, dO tile, lse and D rows
  __shared__ __attribute__((aligned(1024))) char smem_raw[2 * STAGE];
  lds_char_t* smem = (lds_char_t*)smem_raw;
  const int T = a.T, H = a.H, C = H * HD, Hkv = a.Hkv > 0 ? a.Hkv : H, ld = (H + 2 * Hkv) * HD;
  const int G = H / Hkv;   // query heads per key/value head
  // 1-D grid over (sequence, key/value head) pairs, head fastest: the
  // heaviest (first) key blocks of every head are dispatched first (see the
  // forward kernel)
  const int BH = a.B * Hkv;
  const int bj = blockIdx.x % BH, b = bj / Hkv, j = bj % Hkv;
  const int kb = (int)(blockIdx.x / BH);
  // the wave index is uniform across the wave: say so, so that per-wave
  // conditions compile to scalar branches
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lk = lane & 31, g = lane >> 5;
  const int kv0w = kb * BQ + wave * 32;
  const int kv = kv0w + lk;
  const bf16_t* kbase = a.qkv + (size_t)b * T * ld + (H + j) * HD;   // key head j; value head j at + Hkv HD
  const v4i32 rq = make_rsrc(a.qkv, (uint32_t)((size_t)a.B * T * ld * 2));
  const v4i32 rd = make_rsrc(a.dout, (uint32_t)((size_t)a.B * T * C * 2));
  const v4i32 rl = make_rsrc(a.lse, (uint32_t)((size_t)a.B * H * T * 4));
  const v4i32 rD = make_rsrc(a.dsum, (uint32_t)((size_t)a.B * H * T * 4));

  bf16x8 kf[S::KS], vf[S::KS];
#pragma unroll
  for (int s = 0; s < S::KS; ++s) {
    uint4 k4 = make_uint4(0, 0, 0, 0), v4 = make_uint4(0, 0, 0, 0);
    if (kv < T) {
      k4 = *reinterpret_cast<const uint4*>(kbase + (size_t)kv * ld + 16 * s + 8 * g);
      v4 = *reinterpret_cast<const uint4*>(kbase + (size_t)kv * ld + Hkv * HD + 16 * s + 8 * g);
    }
    kf[s] = as_bf16x8(k4);
    vf[s] = as_bf16x8(v4);
  }
  floatx16 dk[S::DT], dv[S::DT];
#pragma unroll
  for (int d = 0; d < S::DT; ++d) {
    zero(dk[d]);
    zero(dv[d]);
  }
  const float scale = 1.0f / sqrtf((float)HD);
  const float sc = scale * LOG2E;

  // query tiles from the diagonal to the end, for each query head h = j G + gi
  // of the group in turn: step it is tile it % nt of head gi = it / nt
  const int qstart = kb * BQ;
  const int nt = qstart < T ? (T - qstart + TILE - 1) / TILE : 0;
  const int ntiles = nt * G;
  auto issue = [&](int it) {
    lds_char_t* st = smem + (it & 1) * STAGE;
    const int h = j * G + it / nt;
    const int q0 = qstart + (it % nt) * TILE;
    issue_rows<HD>(rq, a.qkv, a.qkv + (size_t)b * T * ld + h * HD, q0, ld, st, wave, lane);
    issue_rows<HD>(rd, a.dout, a.dout + (size_t)b * T * C + h * HD, q0, C, st + S::TBA, wave, lane);
    // the tile's 64 log-sum-exp and D values (256 bytes each): 16 lanes
    if (wave == 0 && lane < 16) {
      const uint32_t off = ((uint32_t)(b * H + h) * (uint32_t)T + (uint32_t)q0) * 4u + 16u * lane;
      dma16(rl, off, lds_addr(st + 2 * S::TBA));
      dma16(rD, off, lds_addr(st + 2 * S::TBA + 256));
    }
  };
  if (ntiles > 0) issue(0);
  for (int it = 0; it < ntiles; ++it) {
    wait_vmcnt<0>();
    block_barrier();
    if (it + 1 < ntiles) issue(it + 1);
    const int q0 = qstart + (it % nt) * TILE;
    if (q0 + TILE - 1 < kv0w) continue;   // every query precedes this wave's keys
    const lds_char_t* Qs = smem + (it & 1) * STAGE;
    const lds_char_t* Ds = Qs + S::TBA;
    const lds_char_t* lr = Qs + 2 * S::TBA;   // lse [64] then D [64], fp32
    const bool diag = q0 < kv0w + 32 || q0 + TILE > T || kv0w + 32 > T;

    // Query halves t (rows 32t..32t+31 of the tile) against this wave's keys:
    // scores and score gradients, then their contributions to dV and dK. At
    // hd 128 the halves run one after the other (the K/V fragments and the
    // dK/dV accumulators already take 192 registers); smaller heads keep both
    // halves in flight.
    constexpr int NT = HD >= 128 ? 1 : 2;
#pragma unroll(HD >= 128 ? 1 : 2)
    for (int t0 = 0; t0 < 2; t0 += NT) {
      floatx16 p[NT], ds[NT];
#pragma unroll
      for (int i = 0; i < NT; ++i) {
        const int t = t0 + i;
        zero(p[i]);
        zero(ds[i]);
#pragma unroll
        for (int k = 0; k < S::KS; ++k) {
          p[i] = mfma32(read_row<HD>(Qs, 32 * t + lk, 2 * k + g), kf[k], p[i]);
          ds[i] = mfma32(read_row<HD>(Ds, 32 * t + lk, 2 * k + g), vf[k], ds[i]);
        }
      }
      // probabilities and their score gradients, masked only on tiles that
      // straddle the diagonal or the sequence end
      auto probs = [&](auto masked) {
#pragma unroll
        for (int i = 0; i < NT; ++i)
#pragma unroll
          for (int c4 = 0; c4 < 4; ++c4) {
            // keep the per-group reads of lse and D next to their use
            // (hoisting them all would run out of registers)
            __builtin_amdgcn_sched_barrier(0);
            const int qi = 32 * (t0 + i) + 8 * c4 + 4 * g;   // 4 consecutive queries
            const v4f32 l4 = *reinterpret_cast<const lds_v4f32_t*>(lr + 4 * qi);
            const v4f32 d4 = *reinterpret_cast<const lds_v4f32_t*>(lr + 256 + 4 * qi);
            const float lv[4] = {l4.x * LOG2E, l4.y * LOG2E, l4.z * LOG2E, l4.w * LOG2E};
            const float dvv[4] = {d4.x, d4.y, d4.z, d4.w};
            // query qq = q0 + qi + e sees key kv if kv <= qq < T (and kv < T)
            const int qlo = kv - q0 - qi, qhi = T - q0 - qi;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int r = 4 * c4 + e;
              float pv = fast_exp2(p[i][r] * sc - lv[e]);
              if constexpr (decltype(masked)::value) pv = (e >= qlo && e < qhi && kv < T) ? pv : 0.0f;
              p[i][r] = pv;
              ds[i][r] = pv * (ds[i][r] - dvv[e]);
            }
          }
      };
      if (diag) probs(std::true_type{});
      else probs(std::false_type{});
#pragma unroll
      for (int i = 0; i < NT; ++i)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const bf16x8 pf = acc_slots(p[i], hh), sf = acc_slots(ds[i], hh);
#pragma unroll
          for (int d = 0; d < S::DT; ++d) {
            dv[d] = mfma32(read_tr<HD>(Ds, 32 * d, 32 * (t0 + i) + 16 * hh, lane), pf, dv[d]);
            dk[d] = mfma32(read_tr<HD>(Qs, 32 * d, 32 * (t0 + i) + 16 * hh, lane), sf, dk[d]);
          }
        }
    }
  }

  if (kv < T) {
    bf16_t* dst = a.dqkv + ((size_t)b * T + kv) * ld + (H + j) * HD;
#pragma unroll
    for (int d = 0; d < S::DT; ++d)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int dd = 32 * d + 8 * c + 4 * g;
        if (dd < HD) {
          *reinterpret_cast<uint2*>(dst + dd) =
              make_uint2(pack2(dk[d][4 * c] * scale, dk[d][4 * c + 1] * scale),
                         pack2(dk[d][4 * c + 2] * scale, dk[d][4 * c + 3] * scale));
          *reinterpret_cast<uint2*>(dst + Hkv * HD + dd) =
              make_uint2(pack2(dv[d][4 * c], dv[d][4 * c + 1]), pack2(dv[d][4 * c + 2], dv[d][4 * c + 3]));
        }
      }
  }
}

// dQ for 128 queries (4 waves x 32), walking key tiles of 64.
template <int HD>
__global__ __launch_bounds__(256, 2) void attn_bwd_dq_kernel(AttnArgs a) {
  using S = Shape<HD>;
  __shared__ __attribute__((aligned(1024))) char smem_raw[2 * 2 * S::TBA];   // 2 stages x (K, V)
  lds_char_t* smem = (lds_char_t*)smem_raw;
  const int T = a.T, H = a.H, C = H * HD, Hkv = a.Hkv > 0 ? a.Hkv : H, ld = (H + 2 * Hkv) * HD;
  // 1-D grid, head fastest, heaviest (last) query blocks first, as in the
  // forward pass
  const int BH = a.B * H, nqb = (T + BQ - 1) / BQ;
  const int bh = blockIdx.x % BH, b = bh / H, h = bh % H;
  const int qb = nqb - 1 - (int)(blockIdx.x / BH);
  // the wave index is uniform across the wave: say so, so that per-wave
  // conditions compile to scalar branches
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lq = lane & 31, g = lane >> 5;
  const int q0w = qb * BQ + wave * 32;
  const int q = q0w + lq;
  const bf16_t* base = a.qkv + (size_t)b * T * ld + h * HD;
  const bf16_t* kbase = a.qkv + (size_t)b * T * ld + (H + h / (H / Hkv)) * HD;
  const bf16_t* dob = a.dout + (size_t)b * T * C + h * HD;
  const v4i32 rs = make_rsrc(a.qkv, (uint32_t)((size_t)a.B * T * ld * 2));

  const bf16_t* ob = a.out + (size_t)b * T * C + h * HD;
  bf16x8 qf[S::KS], df[S::KS];
  // all of the query's loads first (rows past T read row T-1 and are unused),
  // then the arithmetic, so no load waits behind another's use
  uint4 q4[S::KS], d4[S::KS], o4[S::KS];
  const int qr = min(q, T - 1);
#pragma unroll
  for (int s = 0; s < S::KS; ++s) {
    q4[s] = *reinterpret_cast<const uint4*>(base + (size_t)qr * ld + 16 * s + 8 * g);
    d4[s] = *reinterpret_cast<const uint4*>(dob + (size_t)qr * C + 16 * s + 8 * g);
    o4[s] = *reinterpret_cast<const uint4*>(ob + (size_t)qr * C + 16 * s + 8 * g);
  }
  const float lse_q = a.lse[(size_t)bh * T + qr];
  float dpart = 0.0f;
#pragma unroll
  for (int s = 0; s < S::KS; ++s) {
    if (q >= T) q4[s] = d4[s] = o4[s] = make_uint4(0, 0, 0, 0);
    qf[s] = as_bf16x8(q4[s]);
    df[s] = as_bf16x8(d4[s]);
    const uint4 dd = d4[s], oo = o4[s];
    dpart += lo_f(dd.x) * lo_f(oo.x) + hi_f(dd.x) * hi_f(oo.x) + lo_f(dd.y) * lo_f(oo.y) + hi_f(dd.y) * hi_f(oo.y);
    dpart += lo_f(dd.z) * lo_f(oo.z) + hi_f(dd.z) * hi_f(oo.z) + lo_f(dd.w) * lo_f(oo.w) + hi_f(dd.w) * hi_f(oo.w);
  }
  const float lse2 = q < T ? lse_q * LOG2E : 0.0f;
  // D = rowsum(dO * O) of query q: lanes lq and lq + 32 hold the two halves of
  // its row. Stored for the dK/dV kernel, which runs after this one.
  const float dsum = dpart + __shfl_xor(dpart, 32);
  if (g == 0 && q < T) a.dsum[(size_t)bh * T + q] = dsum;
  floatx16 dq[S::DT];
#pragma unroll
  for (int d = 0; d < S::DT; ++d) zero(dq[d]);
  const float scale = 1.0f / sqrtf((float)HD);
  const float sc = scale * LOG2E;

  const int kv_end = min(T, qb * BQ + BQ);
  const int ntiles = (kv_end + TILE - 1) / TILE;
  RowLoader<HD> kvl;
  kvl.init(ld, wave, lane);
  const uint32_t koff = (uint32_t)((kbase - a.qkv) * 2), voff = koff + (uint32_t)(Hkv * HD * 2);
  auto issue = [&](int it) {
    lds_char_t* st = smem + (it & 1) * 2 * S::TBA;
    const uint32_t r = (uint32_t)(it * TILE) * (uint32_t)ld * 2u;
    kvl.issue(rs, koff + r, st, wave, lane);
    kvl.issue(rs, voff + r, st + S::TBA, wave, lane);
  };
  issue(0);
  for (int it = 0; it < ntiles; ++it) {
    wait_vmcnt<0>();
    block_barrier();
    if (it + 1 < ntiles) issue(it + 1);
    const int kv0 = it * TILE;
    if (kv0 > q0w + 31) continue;
    const lds_char_t* Ks = smem + (it & 1) * 2 * S::TBA;
    const lds_char_t* Vs = Ks + S::TBA;
    const bool diag = kv0 + TILE - 1 > q0w || kv0 + TILE > T || q0w + 32 > T;

    floatx16 p[2], ds[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      zero(p[t]);
      zero(ds[t]);
#pragma unroll
      for (int k = 0; k < S::KS; ++k) {
        p[t] = mfma32(read_row<HD>(Ks, 32 * t + lq, 2 * k + g), qf[k], p[t]);
        ds[t] = mfma32(read_row<HD>(Vs, 32 * t + lq, 2 * k + g), df[k], ds[t]);
      }
      auto probs = [&](auto masked) {
        // key j = kv0 + 32t + 4g + offset is seen if j <= q, j < T, and q < T
        const int jmax = (q < T ? min(q, T - 1) : -1) - kv0 - 32 * t - 4 * g;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float pv = fast_exp2(p[t][r] * sc - lse2);
          if constexpr (decltype(masked)::value) pv = (acc_row(r, 0) <= jmax) ? pv : 0.0f;
          ds[t][r] = pv * (ds[t][r] - dsum);
        }
      };
      if (diag) probs(std::true_type{});
      else probs(std::false_type{});
    }
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const bf16x8 sf = acc_slots(ds[t], hh);
#pragma unroll
        for (int d = 0; d < S::DT; ++d) dq[d] = mfma32(read_tr<HD>(Ks, 32 * d, 32 * t + 16 * hh, lane), sf, dq[d]);
      }
  }

  if (q < T) {
    bf16_t* dst = a.dqkv + ((size_t)b * T + q) * ld + h * HD;
#pragma unroll
    for (int d = 0; d < S::DT; ++d)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const int dd = 32 * d + 8 * c + 4 * g;
        if (dd < HD)
          *reinterpret_cast<uint2*>(dst + dd) =
              make_uint2(pack2(dq[d][4 * c] * scale, dq[d][4 * c + 1] * scale),
                         pack2(dq[d][4 * c + 2] * scale, dq[d][4 * c + 3] * scale));
      }
  }
}

// Row loads for an eight-wave workgroup: instruction i of the 64-row tile
// goes to bytes [1024 i, 1024 i + 1024), waves taking instructions in turn.
// off: byte offset in the buffer of row 0 of the head's slice.
template <int HD>
DEV void issue_rows8(v4i32 rs, uint32_t off, int r0, int ld, lds_char_t* dst, int wave, int lane) {
  constexpr int U = HD / 8, INSTR = TILE * U / 64;
  static_assert(INSTR % 8 == 0, "tile must split evenly over 8 waves");
#pragma unroll
  for (int i = 0; i < INSTR / 8; ++i) {
    const int ins = wave + 8 * i;
    const int u = ins * 64 + lane;
    const int row = u / U, p = u % U;
    const int c = unit<HD>(row, p) - row * U;   // the XOR is its own inverse
    dma16(rs, off + ((uint32_t)(r0 + row) * (uint32_t)ld + (uint32_t)(c * 8)) * 2u, lds_addr(dst + ins * 1024));
  }
}

// dK, dV at hd 128 with eight waves per 128 keys: wave w owns keys
// 32 (w % 4) .. +31 of the block and the query half w / 4 (rows 32 (w / 4)
// .. +31) of every 64-query tile, so each SIMD runs two waves (the four-wave
// form needs more registers than two waves per SIMD allow: its K/V fragments
// live in registers). The block's K and V rows stay in LDS for the whole walk
// and are read per k-step; at the end the two waves of a key group add their
// dK/dV partial sums through LDS.
template <int HD>
__global__ __launch_bounds__(512, 1) void attn_bwd_dkdv8_kernel(AttnArgs a) {
  using S = Shape<HD>;
  constexpr int KVB = BQ * HD * 2;             // one 128-row block of K or V
  constexpr int STAGE = 2 * S::TBA + 1024;     // Q tile, dO tile, lse and D rows
  constexpr int SMEM = 2 * KVB + 2 * STAGE;
  constexpr int NACC = 2 * S::DT * 16;         // dK and dV registers per lane
  static_assert(4 * NACC * 64 * 4 <= SMEM, "dK/dV exchange fits the tiles' space");
  __shared__ __attribute__((aligned(1024))) char smem_raw[SMEM];
  lds_char_t* smem = (lds_char_t*)smem_raw;
  lds_char_t* Ks = smem;
  lds_char_t* Vs = smem + KVB;
  lds_char_t* stages = smem + 2 * KVB;
  const int T = a.T, H = a.H, C = H * HD, Hkv = a.Hkv > 0 ? a.Hkv : H, ld = (H + 2 * Hkv) * HD;
  const int G = H / Hkv;
  const int BH = a.B * Hkv;
  const int bj = blockIdx.x % BH, b = bj / Hkv, j = bj % Hkv;
  const int kb = (int)(blockIdx.x / BH);
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kw = wave & 3, th = wave >> 2;   // key group, query half
  const int lk = lane & 31, g = lane >> 5;
  const int kv0w = kb * BQ + kw * 32;
  const int kv = kv0w + lk;
  const v4i32 rq = make_rsrc(a.qkv, (uint32_t)((size_t)a.B * T * ld * 2));
  const v4i32 rd = make_rsrc(a.dout, (uint32_t)((size_t)a.B * T * C * 2));
  const v4i32 rl = make_rsrc(a.lse, (uint32_t)((size_t)a.B * H * T * 4));
  const v4i32 rD = make_rsrc(a.dsum, (uint32_t)((size_t)a.B * H * T * 4));
  const uint32_t seq_q = (uint32_t)b * (uint32_t)T * (uint32_t)ld * 2u;   // byte offset of the sequence's qkv rows
  const uint32_t seq_d = (uint32_t)b * (uint32_t)T * (uint32_t)C * 2u;

  floatx16 dk[S::DT], dv[S::DT];
#pragma unroll
  for (int d = 0; d < S::DT; ++d) {
    zero(dk[d]);
    zero(dv[d]);
  }
  const float scale = 1.0f / sqrtf((float)HD);
  const float sc = scale * LOG2E;

  const int qstart = kb * BQ;
  const int nt = qstart < T ? (T - qstart + TILE - 1) / TILE : 0;
  const int ntiles = nt * G;
  auto issue = [&](int it) {
    lds_char_t* st = stages + (it & 1) * STAGE;
    const int h = j * G + it / nt;
    const int q0 = qstart + (it % nt) * TILE;
    issue_rows8<HD>(rq, seq_q + (uint32_t)(h * HD) * 2u, q0, ld, st, wave, lane);
    issue_rows8<HD>(rd, seq_d + (uint32_t)(h * HD) * 2u, q0, C, st + S::TBA, wave, lane);
    if (wave == 0 && lane < 16) {
      const uint32_t off = ((uint32_t)(b * H + h) * (uint32_t)T + (uint32_t)q0) * 4u + 16u * lane;
      dma16(rl, off, lds_addr(st + 2 * S::TBA));
      dma16(rD, off, lds_addr(st + 2 * S::TBA + 256));
    }
  };
  if (ntiles > 0) {
    // the block's key and value rows (key head j; value head j at + Hkv hd)
    const uint32_t koff = seq_q + (uint32_t)((H + j) * HD) * 2u, voff = koff + (uint32_t)(Hkv * HD) * 2u;
    issue_rows8<HD>(rq, koff, qstart, ld, Ks, wave, lane);
    issue_rows8<HD>(rq, koff, qstart + TILE, ld, Ks + S::TB, wave, lane);
    issue_rows8<HD>(rq, voff, qstart, ld, Vs, wave, lane);
    issue_rows8<HD>(rq, voff, qstart + TILE, ld, Vs + S::TB, wave, lane);
    issue(0);
  }
  for (int it = 0; it < ntiles; ++it) {
    wait_vmcnt<0>();
    block_barrier();
    if (it + 1 < ntiles) issue(it + 1);
    const int qh0 = qstart + (it % nt) * TILE + 32 * th;   // this wave's first query
    if (qh0 + 31 < kv0w) continue;   // every query of the half precedes this wave's keys
    const lds_char_t* Qs = stages + (it & 1) * STAGE;
    const lds_char_t* Ds = Qs + S::TBA;
    const lds_char_t* lr = Qs + 2 * S::TBA;   // lse [64] then D [64], fp32
    const bool diag = qh0 < kv0w + 32 || qh0 + 32 > T || kv0w + 32 > T;

    // S = Q K^T and dP = dO V^T for the half's 32 queries x the wave's 32 keys
    floatx16 p, ds;
    zero(p);
    zero(ds);
#pragma unroll
    for (int k = 0; k < S::KS; ++k) {
      p = mfma32(read_row<HD>(Qs, 32 * th + lk, 2 * k + g), read_row<HD>(Ks, 32 * kw + lk, 2 * k + g), p);
      ds = mfma32(read_row<HD>(Ds, 32 * th + lk, 2 * k + g), read_row<HD>(Vs, 32 * kw + lk, 2 * k + g), ds);
    }
    auto probs = [&](auto masked) {
#pragma unroll
      for (int c4 = 0; c4 < 4; ++c4) {
        const int qi = 32 * th + 8 * c4 + 4 * g;   // 4 consecutive queries of the tile
        const v4f32 l4 = *reinterpret_cast<const lds_v4f32_t*>(lr + 4 * qi);
        const v4f32 d4 = *reinterpret_cast<const lds_v4f32_t*>(lr + 256 + 4 * qi);
        const float lv[4] = {l4.x * LOG2E, l4.y * LOG2E, l4.z * LOG2E, l4.w * LOG2E};
        const float dvv[4] = {d4.x, d4.y, d4.z, d4.w};
        // query qh0 - 32 th + qi + e sees key kv if kv <= query < T (and kv < T)
        const int qlo = kv - (qh0 - 32 * th) - qi, qhi = T - (qh0 - 32 * th) - qi;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = 4 * c4 + e;
          float pv = fast_exp2(p[r] * sc - lv[e]);
          if constexpr (decltype(masked)::value) pv = (e >= qlo && e < qhi && kv < T) ? pv : 0.0f;
          p[r] = pv;
          ds[r] = pv * (ds[r] - dvv[e]);
        }
      }
    };
    if (diag) probs(std::true_type{});
    else probs(std::false_type{});
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      const bf16x8 pf = acc_slots(p, hh), sf = acc_slots(ds, hh);
#pragma unroll
      for (int d = 0; d < S::DT; ++d) {
        dv[d] = mfma32(read_tr<HD>(Ds, 32 * d, 32 * th + 16 * hh, lane), pf, dv[d]);
        dk[d] = mfma32(read_tr<HD>(Qs, 32 * d, 32 * th + 16 * hh, lane), sf, dk[d]);
      }
    }
  }

  // the second query half's waves hand their partial sums to the first's
  __syncthreads();
  lds_v4f32_t* red = (lds_v4f32_t*)smem_raw + kw * (NACC / 4) * 64 + lane;
  if (th == 1) {
#pragma unroll
    for (int d = 0; d < S::DT; ++d)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        red[((2 * d) * 4 + c) * 64] = v4f32{dk[d][4 * c], dk[d][4 * c + 1], dk[d][4 * c + 2], dk[d][4 * c + 3]};
        red[((2 * d + 1) * 4 + c) * 64] = v4f32{dv[d][4 * c], dv[d][4 * c + 1], dv[d][4 * c + 2], dv[d][4 * c + 3]};
      }
  }
  __syncthreads();
  if (th == 1 || kv >= T) return;
  bf16_t* dst = a.dqkv + ((size_t)b * T + kv) * ld + (H + j) * HD;
#pragma unroll
  for (int d = 0; d < S::DT; ++d)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const v4f32 ok = red[((2 * d) * 4 + c) * 64], ov = red[((2 * d + 1) * 4 + c) * 64];
      const int dd = 32 * d + 8 * c + 4 * g;
      *reinterpret_cast<uint2*>(dst + dd) =
          make_uint2(pack2((dk[d][4 * c] + ok.x) * scale, (dk[d][4 * c + 1] + ok.y) * scale),
                     pack2((dk[d][4 * c + 2] + ok.z) * scale, (dk[d][4 * c + 3] + ok.w) * scale));
      *reinterpret_cast<uint2*>(dst + Hkv * HD + dd) =
          make_uint2(pack2(dv[d][4 * c] + ov.x, dv[d][4 * c + 1] + ov.y), pack2(dv[d][4 * c + 2] + ov.z, dv[d][4 * c + 3] + ov.w));
    }
}

template <int HD>
hipError_t fwd_t(const AttnArgs& a, hipStream_t s) {
  dim3 grid(((a.T + BQ - 1) / BQ) * a.B * a.H);
  hipLaunchKernelGGL(attn_fwd_kernel<HD>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int HD>
hipError_t bwd_t(const AttnArgs& a, hipStream_t s) {
  // dQ first: it also computes D = rowsum(dO * O), which dK/dV reads
  const int nb = (a.T + BQ - 1) / BQ, Hkv = a.Hkv > 0 ? a.Hkv : a.H;
  hipLaunchKernelGGL(attn_bwd_dq_kernel<HD>, dim3(nb * a.B * a.H), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if constexpr (HD == 128)
    hipLaunchKernelGGL(attn_bwd_dkdv8_kernel<HD>, dim3(nb * a.B * Hkv), dim3(512), 0, s, a);
  else
    hipLaunchKernelGGL(attn_bwd_dkdv_kernel<HD>, dim3(nb * a.B * Hkv), dim3(256), 0, s, a);
  return hipGetLastError();
}

// Shapes the kernels support: head sizes 16..128, H a multiple of Hkv, and
// every byte offset into q|k|v (rows of (H + 2 Hkv) hd) within 32 bits.
bool attn_ok(const AttnArgs& a) {
  const int Hkv = a.Hkv > 0 ? a.Hkv : a.H;
  if (a.H < 1 || Hkv < 1 || a.H % Hkv) return false;
  return (size_t)a.B * a.T * (a.H + 2 * Hkv) * a.hd * 2 < (1ull << 32);
}

}  // namespace

hipError_t launch_attention_fwd(const AttnArgs& a, hipStream_t s) {
  if (!attn_ok(a)) return hipErrorInvalidValue;
  switch (a.hd) {
    case 16: return fwd_t<16>(a, s);
    case 32: return fwd_t<32>(a, s);
    case 64: return fwd_t<64>(a, s);
    case 128: return fwd_t<128>(a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_attention_bwd(const AttnArgs& a, hipStream_t s) {
  if (!attn_ok(a)) return hipErrorInvalidValue;
  switch (a.hd) {
    case 16: return bwd_t<16>(a, s);
    case 32: return bwd_t<32>(a, s);
    case 64: return bwd_t<64>(a, s);
    case 128: return bwd_t<128>(a, s);
  }
  return hipErrorInvalidValue;
}
