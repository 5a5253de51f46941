// bf16 MFMA GEMM with fp32 accumulation for gfx950.
//
//   C[m][n] = sum_k A(m,k) * B(n,k)
//
// A(m,k) is A[m*lda + k] (contraction contiguous) or, with A_T, A[k*lda + m]
// (contraction strided); likewise B. One template covers the three products
// of a linear layer y = x W^T + b with W stored [out, in]:
//   forward  y[t][o]  = sum_i x[t][i] W[o][i]        A = x,  B = W   (A_T=0, B_T=0)
//   input    dx[t][i] = sum_o dy[t][o] W[o][i]       A = dy, B = W   (A_T=0, B_T=1)
//   weight   dW[o][i] = sum_t dy[t][o] x[t][i]       A = dy, B = x   (A_T=1, B_T=1)
//
// Data movement: operand tiles go from HBM straight into LDS with
// buffer_load ... lds (no staging registers; the buffer descriptor's range
// check turns reads past the end of a matrix into zeros), through a ring of
// NS stages of BK contraction steps each, so later tiles are in flight while
// the MFMAs of the current one run. Each wave waits only for its own loads
// (vmcnt) before the block barrier that publishes a stage. With BK = 64 a
// contraction-contiguous operand is fetched in whole 128-byte row segments.
//
// LDS layouts, both in 16-byte units with an XOR swizzle against bank
// conflicts:
//   contraction-contiguous operand: [rows][BK]; an MFMA fragment (8
//     consecutive k of one row) is one ds_read_b128;
//   contraction-strided operand: [BK][rows], the operand's natural layout;
//     a fragment is two ds_read_b64_tr_b16, which hand each lane four
//     consecutive k of one row gathered from four other lanes' reads.
// The fragments of the next k-step are read while the MFMAs of the current
// one run.
//
// MFMA: v_mfma_f32_32x32x16_bf16 with its row index i mapped to n and its
// column index j to m. The epilogue goes through LDS so that every output row
// segment of a wave is written (and any residual or pre-activation read) as
// one contiguous run instead of 16-byte pieces of 32 rows.
#include <type_traits>

#include "common.h"
#include "kernels.h"
#include "lds_dma.h"

namespace {

typedef float v4f32_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4f32_t lds_v4f32_t;
typedef __attribute__((address_space(3))) float lds_f32_t;

// Epilogues of the kernel: the four of GemmEpilogue, plus the two variants
// that read global memory (residual add; fp32 accumulation), kept separate so
// the others do not reserve registers for those reads.
constexpr int EPI_BF16_RES = 4;
constexpr int EPI_F32_ACC = 5;
constexpr int EPI_BF16_SCALE = 6;   // EPI_BF16 with the accumulator scaled by alpha

DEV int bitrev3(int x) { return ((x & 1) << 2) | (x & 2) | ((x >> 2) & 1); }

// Physical 16-byte unit of logical (row, chunk) in a contraction-contiguous
// tile [R][BK]. 32 lanes read 32 consecutive rows at one chunk; the XOR
// spreads them over all 64 banks.
template <int BK>
DEV int unit_n(int row, int c) {
  if constexpr (BK == 32) return row * 4 + (c ^ ((row >> 2) & 3));
  else return row * 8 + (c ^ bitrev3((row >> 1) & 7));
}
// ... in a contraction-strided tile [BK][R]: R/8 units per k-row. A
// transposed fragment read touches 4 consecutive k-rows x 4 units per
// 32 lanes; the chunk XOR spreads those 16 units over all 64 banks:
// 4*(k%4) when a row is a multiple of 16 units (256 B), 4*((k/2)%2) for
// 192-wide tiles (24 units, so consecutive rows already sit 8 units apart).
// Both stay inside aligned groups of 8 or 16 units, hence inside the row.
template <int R>
DEV int unit_t(int k, int c) {
  if constexpr ((R / 8) % 16 == 0) return k * (R / 8) + (c ^ ((k & 3) << 2));
  else return k * (R / 8) + (c ^ (((k >> 1) & 1) << 2));
}

// Waves per workgroup: 4 in a 2 x 2 arrangement; 8 (4 x 2) for 256-row tiles
// with 64-deep stages, whose two 128-row halves share each B tile in LDS
// (one workgroup per CU, two waves per SIMD).
constexpr int gemm_waves(int bm, int bk) { return bm >= 256 && bk >= 64 ? 8 : 4; }

// Issue the direct-to-LDS loads of one operand tile (R rows of the operand,
// BK contraction steps starting at k0) into the stage at `dst`. Wave w of NW
// issues instructions w, w+NW, ...; each instruction moves 64 units (1 KB),
// unit u of the tile going to byte 16*u.
// With PAIRS (a contraction-contiguous operand only), tile row r reads
// operand row r0 + 32 (r / 64) + r % 32, plus alt for the odd 32-row groups:
// 32 rows of one block of the operand, then the same 32 rows of the block
// alt rows further on, and so on.
template <int R, int BK, bool TR, int NW, bool PAIRS = false>
DEV void issue_tile(v4i32 rs, int ld, int r0, int k0, lds_char_t* dst, int wave, int lane, int alt = 0) {
  static_assert(!PAIRS || (!TR && R % 64 == 0), "paired rows: contraction-contiguous tiles of whole 64-row pairs");
  constexpr int UNITS = R * BK / 8;
  constexpr int INSTR = UNITS / 64;
  static_assert(UNITS % (64 * NW) == 0, "tile must split evenly over the waves");
#pragma unroll
  for (int i = 0; i < INSTR / NW; ++i) {
    const int ins = wave + NW * i;
    const int u = ins * 64 + lane;   // physical unit written by this lane
    uint32_t off;
    if constexpr (!TR) {
      constexpr int U = BK / 8;
      const int row = u / U, p = u % U;
      const int c = unit_n<BK>(row, p) - row * U;   // the XOR is its own inverse
      const int grow = PAIRS ? r0 + 32 * (row >> 6) + (row & 31) + ((row >> 5) & 1) * alt : r0 + row;
      off = ((uint32_t)grow * (uint32_t)ld + (uint32_t)(k0 + c * 8)) * 2u;
    } else {
      const int k = u / (R / 8), p = u % (R / 8);
      const int c = unit_t<R>(k, p) - k * (R / 8);
      off = ((uint32_t)(k0 + k) * (uint32_t)ld + (uint32_t)(r0 + c * 8)) * 2u;
    }
    dma16(rs, off, lds_addr(dst + ins * 1024));
  }
}

// MFMA fragment: 8 consecutive k (k-step s, lane group lane/32) of row
// row_base + lane%32 of the tile.
template <int R, int BK, bool TR>
DEV bf16x8 read_frag(const lds_char_t* stage, int row_base, int s, int lane) {
  if constexpr (!TR) {
    const int row = row_base + (lane & 31), c = 2 * s + (lane >> 5);
    return lds_read16(stage + unit_n<BK>(row, c) * 16);
  } else {
    // lane t of each 16-lane group names k-row kb + t/4 and columns
    // n + 4*(t%4)..+3; it receives column n + t at k-rows kb..kb+3
    const int t = lane & 15, h = (lane >> 4) & 1, g = lane >> 5;
    const int n = row_base + 16 * h + 4 * (t & 3);
    const int kb = 16 * s + 8 * g + (t >> 2);
    const int c = n >> 3, sub = (n & 7) * 2;   // byte offset 0 or 8 in the unit
    const uint2 a = lds_read_tr(stage + unit_t<R>(kb, c) * 16 + sub);
    const uint2 b = lds_read_tr(stage + unit_t<R>(kb + 4, c) * 16 + sub);
    return as_bf16x8(make_uint4(a.x, a.y, b.x, b.y));
  }
}

// Kernel parameters: the product's arguments, plus the group table of a
// grouped launch
struct GroupedParams {
  GemmArgs g;
  GemmGroupedArgs gg;
};
template <bool GROUPED>
using KParams = std::conditional_t<GROUPED, GroupedParams, GemmArgs>;
DEV const GemmArgs& args_of(const GemmArgs& p) { return p; }
DEV const GemmArgs& args_of(const GroupedParams& p) { return p.g; }

// Tiles of one product of group gr (the grouped launch's tile shape)
template <int BM, int BN>
DEV int group_tiles(const GemmGroup& gr) {
  return ((gr.M + BM - 1) / BM) * ((gr.N + BN - 1) / BN);
}

template <int BM, int BN, int BK, int NS, bool A_T, bool B_T, int EPI, bool SEG2 = false, bool GROUPED = false>
__global__ __launch_bounds__(64 * gemm_waves(BM, BK), (NS <= 2 ? 2 : 1)) void gemm_kernel(KParams<GROUPED> P) {
  GemmArgs g = args_of(P);
  constexpr int NW = gemm_waves(BM, BK), WM = NW / 2;
  constexpr int WTM = BM / WM, WTN = BN / 2;   // WM x 2 waves
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int KSTEPS = BK / 16;
  constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int LOADS = (BM + BN) * BK / (512 * NW);   // load instructions per wave per stage
  // epilogue staging: per wave 32 rows x WTN fp32 (row stride padded by 4)
  constexpr int EP_LD = WTN + 4;
  constexpr int EP_BYTES = NW * 32 * EP_LD * 4;
  constexpr int SMEM = NS * STAGE > EP_BYTES ? NS * STAGE : EP_BYTES;
  static_assert(KSTEPS % 2 == 0, "fragment double buffer alternates per k-step");
  static_assert(NS >= 2 && NS - 2 <= 3 && (NS - 2) * LOADS < 64, "ring depth / vmcnt range");
  __shared__ __attribute__((aligned(1024))) char smem_raw[SMEM];
  lds_char_t* smem = (lds_char_t*)smem_raw;

  // the wave index is uniform across the wave: say so, so that LDS addresses
  // and per-wave conditions are computed on the scalar unit
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave >> 1, wn = wave & 1;

  // Blocks are dealt round-robin to the 8 XCDs; renumber them so each XCD
  // works through a contiguous run of tiles (n fastest), which keeps the row
  // panel of A it reads in its own L2.
  // With a contraction split over 8k blocks the grid is 1-D: block b works on
  // split b % splits... arranged so that split z always lands on XCD z % 8 and
  // each XCD's L2 serves one contraction range for all of its tiles.
  int bid = 0, split = 0;
  if constexpr (GROUPED) {
    // one tile of one product of one group: the 1-D grid runs through the
    // groups in order, each group's products in order, each product's tiles
    // n fastest; every XCD takes a contiguous run of that order
    int b = blockIdx.x;
    const int tot = gridDim.x, nfull = P.gg.nfull;
    if (nfull > 0) {
      // XCD x takes full tiles [x nfull/8, (x+1) nfull/8), then its eighth
      // of the last group's tiles
      const int f8 = nfull >> 3, x = b & 7, loc = b >> 3;
      b = loc < f8 ? x * f8 + loc : nfull + x * ((tot - nfull) >> 3) + (loc - f8);
    } else if ((tot & 7) == 0) {
      b = (b & 7) * (tot >> 3) + (b >> 3);
    }
    int k = 0;
#pragma unroll
    for (int i = 0; i + 1 < GEMM_GROUPS; ++i) {
      const GemmGroup& gr = P.gg.grp[i];
      const int t = group_tiles<BM, BN>(gr) * gr.count * (gr.splits > 1 ? gr.splits : 1);
      if (k == i && i + 1 < P.gg.ngroups && b >= t) {
        b -= t;
        k = i + 1;
      }
    }
#pragma unroll
    for (int i = 0; i < GEMM_GROUPS; ++i) {
      if (i == k) {
        const GemmGroup& gr = P.gg.grp[i];
        const int tpp = group_tiles<BM, BN>(gr);
        // a product's tiles, each tile's contraction chunks adjacent
        const int sp = gr.splits > 1 ? gr.splits : 1;
        const int pidx = b / (tpp * sp);
        const int rem = b - pidx * tpp * sp;
        bid = rem / sp;
        split = rem - bid * sp;
        g.A = gr.A + (size_t)pidx * gr.a_stride;
        g.B = gr.B + (size_t)pidx * gr.b_stride;
        g.C = gr.C + (size_t)pidx * gr.c_stride;
        g.M = gr.M;
        g.N = gr.N;
        g.lda = gr.lda;
        g.ldb = gr.ldb;
        g.ldc = gr.N;
        g.bsum = gr.bsum ? gr.bsum + (size_t)pidx * gr.M : nullptr;
        g.bsum_ld = gr.count * gr.M;
        if (sp > 1) {
          g.k_chunk = gr.k_chunk;
          g.split_stride = gr.split_stride;
          g.accumulate = 0;   // slices hold plain sums
        }
      }
    }
  }
  const int ntn = (g.N + BN - 1) / BN, ntiles = ntn * ((g.M + BM - 1) / BM);
  if constexpr (GROUPED) {
  } else if (g.splits > 1) {
    split = blockIdx.x % g.splits;
    bid = blockIdx.x / g.splits;
  } else {
    split = 0;
    bid = blockIdx.y * gridDim.x + blockIdx.x;
    if ((ntiles & 7) == 0) bid = (bid & 7) * (ntiles >> 3) + (bid >> 3);
  }
  const int m0 = (bid / ntn) * BM, n0 = (bid % ntn) * BN;

  const int kbeg = split * g.k_chunk;
  const int kend = min(g.K, kbeg + g.k_chunk);
  // k-tiles of the first segment, then (SEG2) those of the second
  const int nk1 = (kend - kbeg + BK - 1) / BK;
  const int nk = SEG2 ? nk1 + g.K2 / BK : nk1;

  // buffer ranges: the whole operand matrices; reads past the end return 0
  const uint32_t a_rows = A_T ? (uint32_t)g.K : (uint32_t)g.M;
  const uint32_t b_rows = B_T ? (uint32_t)g.K : (uint32_t)g.N;
  const v4i32 ra = make_rsrc(g.A, a_rows * (uint32_t)g.lda * 2u);
  const v4i32 rb = make_rsrc(g.B, b_rows * (uint32_t)g.ldb * 2u);

  // second segment: A2 column offset of this tile's output column block
  v4i32 ra2 = ra, rb2 = rb;
  int a2col = 0;
  if constexpr (SEG2) {
    static_assert(!A_T, "second segment with a non-transposed A only");
    ra2 = make_rsrc(g.A2, (uint32_t)g.M * (uint32_t)g.lda2 * 2u);
    rb2 = make_rsrc(g.B2, (B_T ? (uint32_t)g.K2 : (uint32_t)g.N) * (uint32_t)g.ldb2 * 2u);
    a2col = g.K2 * ((g.a2_bound[0] > 0 && n0 >= g.a2_bound[0]) + (g.a2_bound[1] > 0 && n0 >= g.a2_bound[1]));
  }

  // B column offset of this tile's output row block
  const int bcol = g.b_step * ((g.b_bound[0] > 0 && m0 >= g.b_bound[0]) + (g.b_bound[1] > 0 && m0 >= g.b_bound[1]));

  auto stage = [&](int kt) { return smem + (kt % NS) * STAGE; };
  auto issue = [&](int kt) {
    lds_char_t* st = stage(kt);
    if (!SEG2 || kt < nk1) {
      const int k0 = kbeg + kt * BK;
      issue_tile<BM, BK, A_T, NW>(ra, g.lda, m0, k0, st, wave, lane);
      if constexpr (EPI == EPI_SWIGLU)
        issue_tile<BN, BK, B_T, NW, true>(rb, g.ldb, n0 / 2, k0, st + A_BYTES, wave, lane, g.N / 2);
      else
        issue_tile<BN, BK, B_T, NW>(rb, g.ldb, n0 + bcol, k0, st + A_BYTES, wave, lane);
    } else {
      const int k2 = (kt - nk1) * BK;
      issue_tile<BM, BK, A_T, NW>(ra2, g.lda2, m0, a2col + k2, st, wave, lane);
      issue_tile<BN, BK, B_T, NW>(rb2, g.ldb2, n0, k2, st + A_BYTES, wave, lane);
    }
  };
  auto load = [&](bf16x8* fa, bf16x8* fb, int kt, int s) {
    const lds_char_t* st = stage(kt);
#pragma unroll
    for (int i = 0; i < TM; ++i) fa[i] = read_frag<BM, BK, A_T>(st, wm * WTM + i * 32, s, lane);
#pragma unroll
    for (int j = 0; j < TN; ++j) fb[j] = read_frag<BN, BK, B_T>(st + A_BYTES, wn * WTN + j * 32, s, lane);
  };

  floatx16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
  auto mma = [&](const bf16x8* fa, const bf16x8* fb) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) acc[i][j] = mfma32(fb[j], fa[i], acc[i][j]);
  };
  // a tile has landed once at most the loads of the `later` tiles issued
  // after it are outstanding (loads complete in issue order)
  auto wait_later = [&](int later) {
    constexpr int L3 = NS - 2 >= 3 ? 3 : 0, L2 = NS - 2 >= 2 ? 2 : 0;
    if (L3 && later >= 3) wait_vmcnt<L3 * LOADS>();
    else if (L2 && later >= 2) wait_vmcnt<L2 * LOADS>();
    else if (later >= 1) wait_vmcnt<LOADS>();
    else wait_vmcnt<0>();
  };

  // Bias-gradient partial sums of a weight gradient: row m of A (dY^T) summed
  // over this workgroup's share of the contraction, from the A fragments the
  // MFMAs consume. The ntn workgroups of a row of tiles take alternate
  // k-tiles, and the two waves reading the same A fragments alternate
  // k-steps, so each wave adds up 1/(2 ntn) of its fragments. Lane l holds
  // row l%32 of each 32-row fragment at k-slots 8*(l/32)..+7.
  constexpr bool BSUM = A_T && (EPI == EPI_F32 || EPI == EPI_F32_ACC);
  const bool bsum_on = BSUM && g.bsum != nullptr;
  const int tn = n0 / BN;
  float bs[BSUM ? TM : 1];
#pragma unroll
  for (int i = 0; i < (BSUM ? TM : 1); ++i) bs[i] = 0.0f;
  auto bias_sums = [&](const bf16x8* f) {
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const uint4 u = __builtin_bit_cast(uint4, f[i]);
      bs[i] += ((lo_f(u.x) + hi_f(u.x)) + (lo_f(u.y) + hi_f(u.y))) + ((lo_f(u.z) + hi_f(u.z)) + (lo_f(u.w) + hi_f(u.w)));
    }
  };

  // Tile kt: wait for it, publish it with the barrier (which also frees the
  // stage of tile kt-1 for tile kt+NS-1), then walk its k-steps reading the
  // fragments of step s+1 while the MFMAs of step s run. Left to itself the
  // compiler sinks each fragment read next to its first MFMA and waits for
  // it there; the schedule fences below keep a whole step's reads ahead of
  // the previous step's MFMAs. Chosen per product from timings of the GPT-2
  // step (tiles up to 192 x 192; the larger ones would spill):
  //   weight gradients: fences only (-3 %);
  //   input gradients: fences, and the last k-step of a tile deferred past
  //     the next tile's barrier so that its MFMAs cover the latency of that
  //     tile's first reads (-1 to -1.5 %);
  //   forward products: the compiler's own schedule.
  bf16x8 fa[2][TM], fb[2][TN];
#pragma unroll
  for (int s = 0; s < NS - 1; ++s)
    if (s < nk) issue(s);
  constexpr int KL = WTM * WTN > 96 * 96 ? 0 : A_T ? 1 : B_T ? 2 : 0;
  if constexpr (KL == 2) {
  for (int kt = 0; kt < nk; ++kt) {
    // issued so far: tiles up to kt + NS - 2
    wait_later(min(NS - 2, nk - 1 - kt));
    __builtin_amdgcn_s_waitcnt(0xC07F);   // this wave's reads of the stage the DMA below may overwrite are done
    block_barrier();
    if (kt + NS - 1 < nk) issue(kt + NS - 1);
    load(fa[0], fb[0], kt, 0);
    __builtin_amdgcn_sched_barrier(0);
    if (kt > 0) {
      // the last k-step of the previous tile, deferred past the barrier so
      // that its MFMAs cover the latency of this tile's first reads
      mma(fa[1], fb[1]);
      if constexpr (BSUM) {
        if (bsum_on && ((KSTEPS - 1) & 1) == wn && (kt - 1) % ntn == tn) bias_sums(fa[1]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int s = 0; s + 1 < KSTEPS; ++s) {
      load(fa[(s + 1) & 1], fb[(s + 1) & 1], kt, s + 1);
      __builtin_amdgcn_sched_barrier(0);
      mma(fa[s & 1], fb[s & 1]);
      if constexpr (BSUM) {
        if (bsum_on && (s & 1) == wn && kt % ntn == tn) bias_sums(fa[s & 1]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  if (nk > 0) {
    mma(fa[1], fb[1]);
    if constexpr (BSUM) {
      if (bsum_on && ((KSTEPS - 1) & 1) == wn && (nk - 1) % ntn == tn) bias_sums(fa[1]);
    }
  }
  } else {
  for (int kt = 0; kt < nk; ++kt) {
    // issued so far: tiles up to kt + NS - 2
    wait_later(min(NS - 2, nk - 1 - kt));
    block_barrier();
    if (kt + NS - 1 < nk) issue(kt + NS - 1);
    load(fa[0], fb[0], kt, 0);
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      if (s + 1 < KSTEPS) load(fa[(s + 1) & 1], fb[(s + 1) & 1], kt, s + 1);
      if constexpr (KL == 1) __builtin_amdgcn_sched_barrier(0);
      mma(fa[s & 1], fb[s & 1]);
      if constexpr (BSUM) {
        if (bsum_on && (s & 1) == wn && kt % ntn == tn) bias_sums(fa[s & 1]);
      }
      if constexpr (KL == 1) __builtin_amdgcn_sched_barrier(0);
    }
  }
  }
  if constexpr (BSUM) {
    // lanes l and l+32 hold the two k-halves of row l; each wave writes its
    // own partial row, slot (split, tile column, wave column)
    if (bsum_on) {
      const size_t slot = ((size_t)split * ntn + tn) * 2 + wn;
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const float v = bs[i] + __shfl_xor(bs[i], 32);
        const int m = m0 + wm * WTM + 32 * i + (lane & 31);
        if (lane < 32 && m < g.M) g.bsum[slot * (g.bsum_ld ? g.bsum_ld : g.M) + m] = v;
      }
    }
  }

  // ---------------------------------------------------------------- softmax cross-entropy
  // Lane l holds row l%32 of each 32-row block i and, of fragment j, the
  // columns 32j + 8q + 4(l/32) + e (acc[i][j][4q + e]), so a row's values sit
  // in lanes l and l^32 only.
  if constexpr (EPI == EPI_CE_STATS || EPI == EPI_CE_GRAD) {
    const int lg = lane >> 5;
    const int nb = n0 + wn * WTN + 4 * lg;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int mrow = m0 + wm * WTM + 32 * i + (lane & 31);
      const bool row_ok = mrow < g.M;
      int t = row_ok ? g.ce_targets[mrow] : 0;
      if ((unsigned)t >= (unsigned)g.ce_V) t = 0;
      if constexpr (EPI == EPI_CE_STATS) {
        float mx = -INFINITY;
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (nb + 32 * j + 8 * (r >> 2) + (r & 3) < g.ce_V) mx = fmaxf(mx, acc[i][j][r]);
        float se = 0.0f;
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int n = nb + 32 * j + 8 * (r >> 2) + (r & 3);
            if (n < g.ce_V) se += __expf(acc[i][j][r] - mx);
            if (n == t && row_ok) g.ce_tlogit[mrow] = acc[i][j][r];
          }
        const float m2 = __shfl_xor(mx, 32, WAVE), s2 = __shfl_xor(se, 32, WAVE);
        const float mn = fmaxf(mx, m2);
        se = (mx == -INFINITY ? 0.0f : se * __expf(mx - mn)) + (m2 == -INFINITY ? 0.0f : s2 * __expf(m2 - mn));
        if (lg == 0 && row_ok) {
          const int parts = ((g.N + BN - 1) / BN) * 2;
          reinterpret_cast<float2*>(g.ce_stats)[(size_t)mrow * parts + (n0 / BN) * 2 + wn] = make_float2(mn, se);
        }
      } else {
        const float lse = row_ok ? g.ce_lse[mrow] : 0.0f;
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int n = nb + 32 * j + 8 * (r >> 2) + (r & 3);
            float v = n < g.ce_V ? __expf(acc[i][j][r] - lse) * g.ce_scale : 0.0f;
            if (n == t) v -= g.ce_scale;
            acc[i][j][r] = v;
          }
      }
    }
    if constexpr (EPI == EPI_CE_STATS) return;
  }

  // ---------------------------------------------------------------- epilogue
  // Each wave writes its tile 32 rows at a time: accumulators go to LDS, come
  // back as whole row segments, and are stored with the bias, residual,
  // GELU, GELU derivative or fp32 accumulation applied. Every global read an
  // output block needs (residual, pre-activation, previous fp32 value) is
  // issued before its LDS round trip, so its latency is paid once per block
  // of 32 rows instead of once per chunk. Addresses are the block's origin
  // (uniform across the wave) plus a per-lane 32-bit offset computed once;
  // a tile lying wholly inside C (every tile when M and N are multiples of
  // the tile) runs a copy of the loop without bounds checks.
  constexpr int CPR = WTN / 4;                 // 4-column chunks per row
  constexpr int CHUNKS = 32 * CPR / 64;        // chunks per lane per 32-row block
  static_assert((32 * CPR) % 64 == 0, "epilogue chunking");
  // a lane's chunk cc sits at column ((lane + 64 cc) % CPR) * 4, which takes
  // NB = CPR / gcd(64, CPR) distinct values, repeating with period NB in cc
  constexpr int G64 = (CPR % 64 == 0) ? 64 : (CPR % 32 == 0) ? 32 : (CPR % 16 == 0) ? 16 : (CPR % 8 == 0) ? 8
                    : (CPR % 4 == 0) ? 4 : (CPR % 2 == 0) ? 2 : 1;
  constexpr int NB = CPR / G64;
  const int lrow = lane & 31, lg = lane >> 5;
  float* Cf = static_cast<float*>(g.C) + (size_t)split * g.split_stride;
  bf16_t* Cb = static_cast<bf16_t*>(g.C);
  const int ncol0 = n0 + wn * WTN;
  float4 bias4[NB];
  if constexpr (EPI == EPI_BF16 || EPI == EPI_BF16_RES || EPI == EPI_GELU || EPI == EPI_BF16_SCALE ||
                EPI == EPI_CE_GRAD) {
#pragma unroll
    for (int q = 0; q < NB; ++q) {
      const int n = ncol0 + ((lane + 64 * q) % CPR) * 4;
      bias4[q] = (g.bias && n < g.N) ? *reinterpret_cast<const float4*>(g.bias + n) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
  // chunk cc of this lane: row idx / CPR of a 32-row block, columns
  // (idx % CPR) * 4 .. +3 of the wave's WTN, idx = lane + 64 cc; its offset
  // from the block's origin (computed where used: kept in registers across
  // the blocks it would cost the largest tiles spills)
  auto co = [&](int cc) -> uint32_t {
    const int idx = lane + 64 * cc;
    return (uint32_t)(idx / CPR) * (uint32_t)g.ldc + (uint32_t)((idx % CPR) * 4);
  };
  const bool interior = m0 + BM <= g.M && n0 + BN <= g.N;
  auto in_c = [&](auto checked, int mrow0, int cc) -> bool {
    if constexpr (!decltype(checked)::value) return true;
    const int idx = lane + 64 * cc;
    return mrow0 + idx / CPR < g.M && ncol0 + (idx % CPR) * 4 < g.N;
  };

  // every wave is done with the ring before it is reused for staging
  block_barrier();
  lds_f32_t* ep = (lds_f32_t*)smem_raw + wave * 32 * EP_LD;
  constexpr int CG = 4;   // chunks per group read back from LDS together
  static_assert(CHUNKS % CG == 0, "epilogue groups");
  // bf16 inputs of a chunk (residual or pre-activation) are read for the
  // whole 32-row block before its LDS round trip; fp32 values to accumulate
  // onto, four times larger, a group at a time
  constexpr bool RD16 = EPI == EPI_BF16_RES || EPI == EPI_GELU_BWD;
  // with at most two 32-row blocks per wave the bf16 inputs of the whole tile
  // are read up front; otherwise block by block
  constexpr int RD_AHEAD = TM <= 2 ? TM : 1;
  const bf16_t* rd_src = (EPI == EPI_GELU_BWD || EPI == EPI_SWIGLU_BWD) ? g.aux : g.residual;
  uint2 rd_all[RD16 ? TM : 1][RD16 ? CHUNKS : 1];
  auto read_block = [&](int i, auto checked) {
    const int mrow0 = m0 + wm * WTM + i * 32;
    const bf16_t* src = rd_src + ((size_t)mrow0 * g.ldc + ncol0);
#pragma unroll
    for (int cc = 0; cc < CHUNKS; ++cc)
      rd_all[i][cc] = in_c(checked, mrow0, cc) ? *reinterpret_cast<const uint2*>(src + co(cc)) : make_uint2(0, 0);
  };
  auto store_tile = [&](auto checked) {
    if constexpr (RD16) {
#pragma unroll
      for (int i = 0; i < RD_AHEAD; ++i) read_block(i, checked);
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int mrow0 = m0 + wm * WTM + i * 32;
      if constexpr (RD16) {
        if (i >= RD_AHEAD) read_block(i, checked);
      }
      uint2 (&rd)[RD16 ? CHUNKS : 1] = rd_all[RD16 ? i : 0];
      // lane holds, for row lrow of this 32-row block, columns
      // 32j + 8q + 4*lg .. +3 of the wave's WTN columns
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int col = 32 * j + 8 * q + 4 * lg;
          const v4f32_t v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
          *reinterpret_cast<lds_v4f32_t*>(ep + lrow * EP_LD + col) = v;
        }
      __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): this wave's LDS writes are done
      __builtin_amdgcn_wave_barrier();
      // the bias and bf16 inputs read above have landed: one explicit wait here
      // (otherwise the compiler waits before every store that follows a read)
      if (i == 0 || (RD16 && i >= RD_AHEAD)) wait_vmcnt<0>();
      const size_t bo = (size_t)mrow0 * g.ldc + ncol0;
      float* Cfi = Cf + bo;
      bf16_t* Cbi = Cb + bo;
      if constexpr (EPI == EPI_SWIGLU) {
        // The wave's 64 staged columns are the gate values of features
        // f0..f0+31, then the up values of the same features (the B rows were
        // loaded in such pairs). Lane slot pi = lane + 64 pp takes row pi / 8
        // and features f0 + 4 (pi % 8) .. +3 of both halves: the
        // pre-activation (gate columns, then up columns) and silu(gate) up,
        // from the bf16-rounded values as the separate kernel computes it;
        // eight lanes write 64 contiguous bytes of a row.
        static_assert(TN == 2 && !A_T && !B_T && !SEG2, "SwiGLU: 64 columns per wave, no second segment");
        const int F = g.N / 2, f0 = ncol0 / 2;
#pragma unroll
        for (int pp = 0; pp < 4; ++pp) {
          const int pi = lane + 64 * pp, row = pi >> 3, k = pi & 7;
          const int m = mrow0 + row, f = f0 + 4 * k;
          const v4f32_t gv = *reinterpret_cast<const lds_v4f32_t*>(ep + row * EP_LD + 4 * k);
          const v4f32_t uv = *reinterpret_cast<const lds_v4f32_t*>(ep + row * EP_LD + 32 + 4 * k);
          if (decltype(checked)::value && (m >= g.M || f >= F)) continue;
          const uint2 gw = make_uint2(pack2(gv.x, gv.y), pack2(gv.z, gv.w));
          const uint2 uw = make_uint2(pack2(uv.x, uv.y), pack2(uv.z, uv.w));
          bf16_t* pre = Cb + (size_t)m * g.ldc;
          *reinterpret_cast<uint2*>(pre + f) = gw;
          *reinterpret_cast<uint2*>(pre + F + f) = uw;
          *reinterpret_cast<uint2*>(g.C2 + (size_t)m * F + f) =
              make_uint2(pack2(swiglu1(lo_f(gw.x), lo_f(uw.x)), swiglu1(hi_f(gw.x), hi_f(uw.x))),
                         pack2(swiglu1(lo_f(gw.y), lo_f(uw.y)), swiglu1(hi_f(gw.y), hi_f(uw.y))));
        }
      } else {
      // read back row segments a group at a time, apply and store
#pragma unroll
      for (int c0 = 0; c0 < CHUNKS; c0 += CG) {
        v4f32_t vals[CG];
        float4 prev[EPI == EPI_F32_ACC ? CG : 1];
        // SwiGLU backward: the saved gate and up values of the chunk's features
        uint2 gx[EPI == EPI_SWIGLU_BWD ? CG : 1], ux[EPI == EPI_SWIGLU_BWD ? CG : 1];
#pragma unroll
        for (int c = 0; c < CG; ++c) {
          const int idx = lane + 64 * (c0 + c);
          if constexpr (EPI == EPI_F32_ACC)
            prev[c] = (g.accumulate && in_c(checked, mrow0, c0 + c))
                          ? *reinterpret_cast<const float4*>(Cfi + co(c0 + c))
                          : make_float4(0.f, 0.f, 0.f, 0.f);
          if constexpr (EPI == EPI_SWIGLU_BWD) {
            const bool ok = in_c(checked, mrow0, c0 + c);
            const bf16_t* src = rd_src + bo + co(c0 + c);
            gx[c] = ok ? *reinterpret_cast<const uint2*>(src) : make_uint2(0, 0);
            ux[c] = ok ? *reinterpret_cast<const uint2*>(src + g.N) : make_uint2(0, 0);
          }
          vals[c] = *reinterpret_cast<const lds_v4f32_t*>(ep + (idx / CPR) * EP_LD + (idx % CPR) * 4);
        }
#pragma unroll
        for (int c = 0; c < CG; ++c) {
          const int cc = c0 + c;
          if (!in_c(checked, mrow0, cc)) continue;
          float v0 = vals[c].x, v1 = vals[c].y, v2 = vals[c].z, v3 = vals[c].w;
          const uint32_t off = co(cc);
          if constexpr (EPI == EPI_F32 || EPI == EPI_F32_ACC) {
            if constexpr (EPI == EPI_F32_ACC) {
              v0 += prev[c].x; v1 += prev[c].y; v2 += prev[c].z; v3 += prev[c].w;
            }
            *reinterpret_cast<float4*>(Cfi + off) = make_float4(v0, v1, v2, v3);
          } else if constexpr (EPI == EPI_SWIGLU_BWD) {
            // the output gradient rounded to bf16, as the separate kernel reads it
            const uint32_t d01 = pack2(v0, v1), d23 = pack2(v2, v3);
            float dg[4], du[4];
            swiglu1_bwd(lo_f(d01), lo_f(gx[c].x), lo_f(ux[c].x), dg[0], du[0]);
            swiglu1_bwd(hi_f(d01), hi_f(gx[c].x), hi_f(ux[c].x), dg[1], du[1]);
            swiglu1_bwd(lo_f(d23), lo_f(gx[c].y), lo_f(ux[c].y), dg[2], du[2]);
            swiglu1_bwd(hi_f(d23), hi_f(gx[c].y), hi_f(ux[c].y), dg[3], du[3]);
            *reinterpret_cast<uint2*>(Cbi + off) = make_uint2(pack2(dg[0], dg[1]), pack2(dg[2], dg[3]));
            *reinterpret_cast<uint2*>(Cbi + off + g.N) = make_uint2(pack2(du[0], du[1]), pack2(du[2], du[3]));
          } else if constexpr (EPI == EPI_GELU_BWD) {
            v0 *= gelu_tanh_grad(lo_f(rd[cc].x)); v1 *= gelu_tanh_grad(hi_f(rd[cc].x));
            v2 *= gelu_tanh_grad(lo_f(rd[cc].y)); v3 *= gelu_tanh_grad(hi_f(rd[cc].y));
            *reinterpret_cast<uint2*>(Cbi + off) = make_uint2(pack2(v0, v1), pack2(v2, v3));
          } else {
            if constexpr (EPI == EPI_BF16_SCALE) {
              v0 *= g.alpha; v1 *= g.alpha; v2 *= g.alpha; v3 *= g.alpha;
            }
            const float4 bb = bias4[cc % NB];
            v0 += bb.x; v1 += bb.y; v2 += bb.z; v3 += bb.w;
            if constexpr (EPI == EPI_GELU) {
              *reinterpret_cast<uint2*>(Cbi + off) = make_uint2(pack2(v0, v1), pack2(v2, v3));
              *reinterpret_cast<uint2*>(g.C2 + bo + off) =
                  make_uint2(pack2(gelu_tanh(v0), gelu_tanh(v1)), pack2(gelu_tanh(v2), gelu_tanh(v3)));
            } else {
              if constexpr (EPI == EPI_BF16_RES) {
                v0 += lo_f(rd[cc].x); v1 += hi_f(rd[cc].x); v2 += lo_f(rd[cc].y); v3 += hi_f(rd[cc].y);
              }
              *reinterpret_cast<uint2*>(Cbi + off) = make_uint2(pack2(v0, v1), pack2(v2, v3));
            }
          }
        }
      }
      }
      __builtin_amdgcn_s_waitcnt(0xC07F);   // reads done before the next block overwrites
      __builtin_amdgcn_wave_barrier();
    }
  };
  if (interior) store_tile(std::false_type{});
  else store_tile(std::true_type{});
}

template <int BM, int BN, int BK, int NS, bool A_T, bool B_T, int EPI, bool SEG2 = false>
hipError_t launch_t(const GemmArgs& g, hipStream_t s) {
  const unsigned tn = (g.N + BN - 1) / BN, tm = (g.M + BM - 1) / BM;
  dim3 grid = g.splits > 1 ? dim3(tn * tm * g.splits) : dim3(tn, tm);
  hipLaunchKernelGGL((gemm_kernel<BM, BN, BK, NS, A_T, B_T, EPI, SEG2>), grid, dim3(64 * gemm_waves(BM, BK)), 0, s, g);
  return hipGetLastError();
}

// Grouped weight gradients: every tile of every product in one 1-D grid.
template <int BM, int BN, int BK>
hipError_t launch_grouped_t(const GemmGroupedArgs& gg, hipStream_t s) {
  GroupedParams P{};
  P.gg = gg;
  GemmArgs& g = P.g;
  g.K = gg.K;
  g.splits = 1;
  g.k_chunk = (gg.K + 63) / 64 * 64;
  g.accumulate = gg.accumulate;
  // fields the kernel sets per product; these keep the shared code's reads in range
  g.A = gg.grp[0].A; g.B = gg.grp[0].B; g.C = gg.grp[0].C; g.M = gg.grp[0].M; g.N = gg.grp[0].N;
  long tiles = 0;
  for (int i = 0; i < gg.ngroups; ++i)
    tiles += (long)((gg.grp[i].M + BM - 1) / BM) * ((gg.grp[i].N + BN - 1) / BN) * gg.grp[i].count *
             (gg.grp[i].splits > 1 ? gg.grp[i].splits : 1);
  if (tiles < 1 || tiles > (1L << 30)) return hipErrorInvalidValue;
  if (gg.accumulate)
    hipLaunchKernelGGL((gemm_kernel<BM, BN, BK, 2, true, true, EPI_F32_ACC, false, true>), dim3((unsigned)tiles),
                       dim3(64 * gemm_waves(BM, BK)), 0, s, P);
  else
    hipLaunchKernelGGL((gemm_kernel<BM, BN, BK, 2, true, true, EPI_F32, false, true>), dim3((unsigned)tiles),
                       dim3(64 * gemm_waves(BM, BK)), 0, s, P);
  return hipGetLastError();
}

// Non-transposed A with an optional second contraction segment and output scale.
template <int BM, int BN, int BK, bool B_T>
hipError_t launch_bf16(const GemmArgs& g, hipStream_t s) {
  const bool scale = g.alpha != 0.0f && g.alpha != 1.0f;
  if (g.K2 > 0) {
    if (scale) return hipErrorInvalidValue;
    return g.residual ? launch_t<BM, BN, BK, 2, false, B_T, EPI_BF16_RES, true>(g, s)
                      : launch_t<BM, BN, BK, 2, false, B_T, EPI_BF16, true>(g, s);
  }
  if (g.residual) return scale ? hipErrorInvalidValue : launch_t<BM, BN, BK, 2, false, B_T, EPI_BF16_RES>(g, s);
  return scale ? launch_t<BM, BN, BK, 2, false, B_T, EPI_BF16_SCALE>(g, s)
               : launch_t<BM, BN, BK, 2, false, B_T, EPI_BF16>(g, s);
}

template <int BM, int BN, int BK>
hipError_t launch_cfg(const GemmArgs& g, int a_t, int b_t, int epi, hipStream_t s) {
  if (g.K2 > 0 && (a_t || epi != EPI_BF16)) return hipErrorInvalidValue;
  if (!a_t && !b_t && epi == EPI_BF16) return launch_bf16<BM, BN, BK, false>(g, s);
  if (!a_t && !b_t && epi == EPI_GELU) return launch_t<BM, BN, BK, 2, false, false, EPI_GELU>(g, s);
  if (!a_t && !b_t && epi == EPI_CE_STATS) return launch_t<BM, BN, BK, 2, false, false, EPI_CE_STATS>(g, s);
  if (!a_t && !b_t && epi == EPI_CE_GRAD) return launch_t<BM, BN, BK, 2, false, false, EPI_CE_GRAD>(g, s);
  if (!a_t && b_t && epi == EPI_BF16) return launch_bf16<BM, BN, BK, true>(g, s);
  if (!a_t && b_t && epi == EPI_GELU_BWD) return launch_t<BM, BN, BK, 2, false, true, EPI_GELU_BWD>(g, s);
  if (!a_t && b_t && epi == EPI_SWIGLU_BWD) return launch_t<BM, BN, BK, 2, false, true, EPI_SWIGLU_BWD>(g, s);
  if (!a_t && !b_t && epi == EPI_SWIGLU) {
    if constexpr (BN == 128) return launch_t<BM, BN, BK, 2, false, false, EPI_SWIGLU>(g, s);
    return hipErrorInvalidValue;
  }
  // products with few output tiles and a long contraction, split into fp32 slices
  if (!a_t && b_t && epi == EPI_F32 && !g.accumulate) return launch_t<BM, BN, BK, 2, false, true, EPI_F32>(g, s);
  if (!a_t && !b_t && epi == EPI_F32 && !g.accumulate) return launch_t<BM, BN, BK, 2, false, false, EPI_F32>(g, s);
  if (a_t && b_t && epi == EPI_F32)
    return g.accumulate ? launch_t<BM, BN, BK, 2, true, true, EPI_F32_ACC>(g, s)
                        : launch_t<BM, BN, BK, 2, true, true, EPI_F32>(g, s);
  return hipErrorInvalidValue;
}

}  // namespace

// Tile configuration per product, chosen from timings of every GPT-2 124M
// product on the MI355X (all with two blocks per CU and a 2-stage ring):
//   weight gradients: 192 x 192 tiles, 32-deep stages;
//   forward MLP-up with GELU, and products with at least 8192 such tiles
//   (the tied head): 256 x 192 x 32, whose rounds of 512 tiles fill the chip;
//   input gradients without the GELU derivative, and forward products of
//   1024 to 8191 such tiles (the Qwen3-shaped gate/up projection): 256 x 192
//   x 64 with eight waves, the two 128-row halves sharing each B tile (-2 to
//   -3 % on the GPT-2 input gradients, -3.5 % on the gate/up product, against
//   two four-wave 128 x 192 workgroups per CU; slower for the GPT-2 forward
//   and GELU-derivative products);
//   other forward and input-gradient products, the GELU-derivative input
//   gradient included: 128 x 192, 64-deep stages (-5 % on the latter
//   against 32-deep stages since the k-loop schedule fences).
// Widths that are not multiples of 192 (the Qwen3-shaped model, small test
// models) take 256 x 128 tiles when they give at least 512 of them, else
// 128 x 128, 64-deep except for weight gradients (the Qwen3-shaped step:
// input gradients -17 %, forward products -4 % against 32-deep stages).
GemmConfig gemm_config(int M, int N, int a_t, int b_t, int epi) {
  // the fused SwiGLU pairs the two 32-column fragments of a wave: 128-wide tiles
  if (epi == EPI_SWIGLU)
    return (M >= 256 && (long)((M + 255) / 256) * (N / 128) >= 512) ? GemmConfig{256, 128, 32} : GemmConfig{128, 128, 64};
  if (N >= 192 && N % 192 == 0) {
    if (a_t) {
      if (M >= 192 && M % 192 == 0) return {192, 192, 32};
      if (M >= 128) return {128, 192, 32};
    } else {
      if (M >= 256 && b_t && epi == EPI_BF16) return {256, 192, 64};
      const long tiles256 = (long)((M + 255) / 256) * (N / 192);
      if (M >= 256 && epi == EPI_BF16 && tiles256 >= 1024 && tiles256 < 8192) return {256, 192, 64};
      if (M >= 256 && (epi == EPI_GELU || tiles256 >= 8192)) return {256, 192, 32};
      if (M >= 128) return {128, 192, 64};
    }
  }
  // 256-row tiles only when they still give two workgroups per CU (a
  // workgroup alone on a CU keeps its MFMA pipe about half busy)
  if (M >= 256 && N >= 128 && N % 128 == 0 && (long)((M + 255) / 256) * (N / 128) >= 512) return {256, 128, 32};
  return {128, 128, a_t ? 32 : 64};
}

int gemm_ce_parts(int M, int N) {
  const GemmConfig c = gemm_config(M, N, 0, 0, EPI_CE_STATS);
  return ((N + c.bn - 1) / c.bn) * 2;
}

int gemm_bias_parts(int M, int N, int splits) {
  const GemmConfig c = gemm_config(M, N, 1, 1, EPI_F32);
  return (splits < 1 ? 1 : splits) * ((N + c.bn - 1) / c.bn) * 2;
}

int gemm_split_plan(int K, int want, int* k_chunk) {
  if (want < 1) want = 1;
  int kc = (K + want - 1) / want;
  kc = (kc + 63) / 64 * 64;
  if (kc < 64) kc = 64;
  if (k_chunk) *k_chunk = kc;
  int n = (K + kc - 1) / kc;
  return n < 1 ? 1 : n;
}

hipError_t launch_gemm(const GemmArgs& g0, int a_t, int b_t, int epi, hipStream_t s) {
  GemmArgs g = g0;
  // byte offsets are 32-bit: the operand matrices, plus the up to 256 rows a
  // tile may address past their end, must stay below 4 GiB
  if ((size_t)((a_t ? g.K : g.M) + 256) * g.lda * 2 >= (1ull << 32) ||
      (size_t)((b_t ? g.K : g.N) + 256) * g.ldb * 2 >= (1ull << 32))
    return hipErrorInvalidValue;
  if (g.splits <= 1 || g.k_chunk <= 0) {
    g.splits = 1;
    g.k_chunk = (g.K + 63) / 64 * 64;
    if (g.k_chunk < 64) g.k_chunk = 64;
  } else {
    // the caller's plan: k_chunk a multiple of 64 and splits = ceil(K / k_chunk)
    if (g.k_chunk % 64 || (long)g.k_chunk * g.splits < g.K || (long)g.k_chunk * (g.splits - 1) >= g.K)
      return hipErrorInvalidValue;
    if (epi != EPI_F32) return hipErrorInvalidValue;
  }
  if (epi == EPI_SWIGLU || epi == EPI_SWIGLU_BWD) {
    // one contraction, A not transposed; SwiGLU: B not transposed, gate and up
    // rows in 64-row pairs of tiles, both outputs given; its backward: the
    // pre-activation to read and room for both gradients in each row
    if (a_t || g.K2 > 0 || g.splits > 1 || g.bias || g.residual) return hipErrorInvalidValue;
    if (epi == EPI_SWIGLU && (b_t || g.N % 128 || !g.C2 || g.ldc < g.N)) return hipErrorInvalidValue;
    if (epi == EPI_SWIGLU_BWD && (!b_t || g.N % 4 || !g.aux || g.ldc < 2 * g.N)) return hipErrorInvalidValue;
  }
  if (g.K2 > 0) {
    if (g.splits > 1 || g.K % 64 || g.K2 % 64 || !g.A2 || !g.B2 || a_t) return hipErrorInvalidValue;
    if ((size_t)(g.M + 256) * g.lda2 * 2 >= (1ull << 32) ||
        (size_t)((b_t ? g.K2 : g.N) + 256) * g.ldb2 * 2 >= (1ull << 32))
      return hipErrorInvalidValue;
  }
  if (g.b_step != 0) {
    // row blocks must not straddle a bound; B must be read transposed ([K][N])
    if (!b_t || g.b_step < 0) return hipErrorInvalidValue;
    for (int i = 0; i < 2; ++i)
      if (g.b_bound[i] < 0 || g.b_bound[i] % 128) return hipErrorInvalidValue;
  }
  GemmConfig c = gemm_config(g.M, g.N, a_t, b_t, epi);
  // a tile's output columns must lie within one block of the second segment
  const bool bounded = g.K2 > 0 && (g.a2_bound[0] > 0 || g.a2_bound[1] > 0);
  if (bounded) {
    for (int i = 0; i < 2; ++i)
      if (g.a2_bound[i] < 0 || g.a2_bound[i] % 128) return hipErrorInvalidValue;
    if ((g.a2_bound[0] % c.bn) || (g.a2_bound[1] % c.bn))
      c = (g.M >= 256 && (long)((g.M + 255) / 256) * ((g.N + 127) / 128) >= 512) ? GemmConfig{256, 128, 32}
                                                                                  : GemmConfig{128, 128, 64};
  }
  // an output row block must not straddle a B column-offset bound
  if (g.b_step != 0 && ((g.b_bound[0] % c.bm) || (g.b_bound[1] % c.bm))) return hipErrorInvalidValue;
  if (c.bm == 192) return launch_cfg<192, 192, 32>(g, a_t, b_t, epi, s);
  if (c.bm == 256 && c.bn == 192) {
    if (c.bk == 64) return launch_cfg<256, 192, 64>(g, a_t, b_t, epi, s);
    return launch_cfg<256, 192, 32>(g, a_t, b_t, epi, s);
  }
  if (c.bm == 128 && c.bn == 192) {
    if (c.bk == 64) return launch_cfg<128, 192, 64>(g, a_t, b_t, epi, s);
    return launch_cfg<128, 192, 32>(g, a_t, b_t, epi, s);
  }
  if (c.bm == 256) return launch_cfg<256, 128, 32>(g, a_t, b_t, epi, s);
  if (c.bk == 64) return launch_cfg<128, 128, 64>(g, a_t, b_t, epi, s);
  return launch_cfg<128, 128, 32>(g, a_t, b_t, epi, s);
}

// One tile shape for every group: 192 x 192 when all of them are multiples of
// 192 in both output dimensions (the weight-gradient tile of gemm_config),
// else 128 x 128. Each group's operands (plus the up to 256 rows a tile may
// address past their end) must stay within 32-bit byte offsets.
static bool grouped_uses_192(const GemmGroupedArgs& gg) {
  for (int i = 0; i < gg.ngroups; ++i)
    if (gg.grp[i].M % 192 || gg.grp[i].N % 192) return false;
  return true;
}

int gemm_grouped_bias_parts(const GemmGroupedArgs& gg, int i) {
  const int bn = grouped_uses_192(gg) ? 192 : 128;
  return ((gg.grp[i].N + bn - 1) / bn) * 2;
}

hipError_t launch_gemm_grouped(const GemmGroupedArgs& gg, hipStream_t s) {
  if (gg.ngroups < 1 || gg.ngroups > GEMM_GROUPS || gg.K < 1) return hipErrorInvalidValue;
  long tiles = 0, last = 0;
  const bool g192 = grouped_uses_192(gg);
  for (int i = 0; i < gg.ngroups; ++i) {
    const GemmGroup& gr = gg.grp[i];
    if (!gr.A || !gr.B || !gr.C || gr.M < 1 || gr.N < 1 || gr.count < 1 || gr.N % 4) return hipErrorInvalidValue;
    if (gr.splits > 1) {
      // chunks of whole 64-token steps covering K; slices of plain sums
      if (gr.bsum || gr.k_chunk < 64 || gr.k_chunk % 64 || (long)gr.k_chunk * gr.splits < gg.K ||
          (long)gr.k_chunk * (gr.splits - 1) >= gg.K || gr.split_stride < (long)gr.count * gr.c_stride)
        return hipErrorInvalidValue;
    }
    const int bm = g192 ? 192 : 128;
    last = (long)((gr.M + bm - 1) / bm) * ((gr.N + bm - 1) / bm) * gr.count * (gr.splits > 1 ? gr.splits : 1);
    tiles += last;
    if ((size_t)(gg.K + 256) * gr.lda * 2 >= (1ull << 32) || (size_t)(gg.K + 256) * gr.ldb * 2 >= (1ull << 32))
      return hipErrorInvalidValue;
  }
  if (gg.nfull != 0 && (gg.nfull < 0 || gg.nfull % 8 || gg.nfull != tiles - last || last % 8)) return hipErrorInvalidValue;
  return g192 ? launch_grouped_t<192, 192, 32>(gg, s) : launch_grouped_t<128, 128, 32>(gg, s);
}
