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
// NSTAGE stages of 32 contraction steps each, so several tiles are in flight
// while the MFMAs of the current one run. Each wave waits only for its own
// loads (vmcnt) before the block barrier that publishes a stage.
//
// LDS layouts, both in 16-byte units with an XOR swizzle against bank
// conflicts:
//   contraction-contiguous operand: [rows][32] (4 units per row); an MFMA
//     fragment (8 consecutive k of one row) is one ds_read_b128;
//   contraction-strided operand: [32][rows], the operand's natural layout;
//     a fragment is two ds_read_b64_tr_b16, which hand each lane four
//     consecutive k of one row gathered from four other lanes' reads.
//
// MFMA: v_mfma_f32_32x32x16_bf16 with its row index i mapped to n and its
// column index j to m, so each lane ends up holding four consecutive n of one
// output row (8-byte bf16 / 16-byte fp32 stores in the epilogue).
#include "common.h"
#include "kernels.h"
#include "lds_dma.h"

namespace {

constexpr int BK = 32;        // contraction steps per stage
constexpr int NSTAGE = 4;     // LDS ring depth

// Physical 16-byte unit of logical (row, chunk) in a contraction-contiguous
// tile [R][32]: 4 units per row, chunk XOR (row/4)%4.
DEV int unit_n(int row, int c) { return row * 4 + (c ^ ((row >> 2) & 3)); }
// ... in a contraction-strided tile [32][R]: R/8 units per k-row. A
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

// Issue the direct-to-LDS loads of one operand tile (R rows of the operand,
// 32 contraction steps starting at k0) into the stage at `dst`. Wave w issues
// instructions w, w+4, ...; each instruction moves 64 units (1 KB), unit u of
// the tile going to byte 16*u.
template <int R, bool TR>
DEV void issue_tile(v4i32 rs, int ld, int r0, int k0, lds_char_t* dst, int wave, int lane) {
  constexpr int UNITS = R * BK / 8;
  constexpr int INSTR = UNITS / 64;
  static_assert(UNITS % 256 == 0, "tile must split evenly over 4 waves");
#pragma unroll
  for (int i = 0; i < INSTR / 4; ++i) {
    const int ins = wave + 4 * i;
    const int u = ins * 64 + lane;   // physical unit written by this lane
    uint32_t off;
    if constexpr (!TR) {
      const int row = u >> 2, p = u & 3;
      const int c = p ^ ((row >> 2) & 3);
      off = ((uint32_t)(r0 + row) * (uint32_t)ld + (uint32_t)(k0 + c * 8)) * 2u;
    } else {
      const int k = u / (R / 8), p = u % (R / 8);
      const int c = unit_t<R>(k, p) - k * (R / 8);   // the XOR is its own inverse
      off = ((uint32_t)(k0 + k) * (uint32_t)ld + (uint32_t)(r0 + c * 8)) * 2u;
    }
    dma16(rs, off, lds_addr(dst + ins * 1024));
  }
}

// MFMA fragment: 8 consecutive k (k-step s, lane group lane/32) of row
// row_base + lane%32 of the tile.
template <int R, bool TR>
DEV bf16x8 read_frag(const lds_char_t* stage, int row_base, int s, int lane) {
  if constexpr (!TR) {
    const int row = row_base + (lane & 31), c = 2 * s + (lane >> 5);
    return lds_read16(stage + unit_n(row, c) * 16);
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

template <int BM, int BN, bool A_T, bool B_T, int EPI>
__global__ __launch_bounds__(256, 1) void gemm_kernel(GemmArgs g) {
  constexpr int WTM = BM / 2, WTN = BN / 2;   // 2 x 2 waves
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int LOADS = (BM + BN) / 64;       // load instructions per wave per stage
  // one array per ring stage: with the loop unrolled by NSTAGE every LDS read
  // and every in-flight load names its stage statically, so the compiler
  // knows the reads of one stage do not wait on the loads into another
  static_assert(NSTAGE == 4, "ring of four stages");
  __shared__ __attribute__((aligned(1024))) char st0[STAGE];
  __shared__ __attribute__((aligned(1024))) char st1[STAGE];
  __shared__ __attribute__((aligned(1024))) char st2[STAGE];
  __shared__ __attribute__((aligned(1024))) char st3[STAGE];
  auto stage = [&](int s) -> lds_char_t* {
    return (lds_char_t*)(s == 0 ? st0 : (s == 1 ? st1 : (s == 2 ? st2 : st3)));
  };

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // Blocks are dealt round-robin to the 8 XCDs; renumber them so each XCD
  // works through a contiguous run of tiles (n fastest), which keeps the row
  // panel of A it reads in its own L2.
  const int ntn = gridDim.x, ntiles = gridDim.x * gridDim.y;
  int bid = blockIdx.y * gridDim.x + blockIdx.x;
  if ((ntiles & 7) == 0) bid = (bid & 7) * (ntiles >> 3) + (bid >> 3);
  const int m0 = (bid / ntn) * BM, n0 = (bid % ntn) * BN;

  const int kbeg = blockIdx.z * g.k_chunk;
  const int kend = min(g.K, kbeg + g.k_chunk);
  const int nk = (kend - kbeg + BK - 1) / BK;

  // buffer ranges: the whole operand matrices; reads past the end return 0
  const uint32_t a_rows = A_T ? (uint32_t)g.K : (uint32_t)g.M;
  const uint32_t b_rows = B_T ? (uint32_t)g.K : (uint32_t)g.N;
  const v4i32 ra = make_rsrc(g.A, a_rows * (uint32_t)g.lda * 2u);
  const v4i32 rb = make_rsrc(g.B, b_rows * (uint32_t)g.ldb * 2u);

  auto issue = [&](int kt, lds_char_t* st) {
    const int k0 = kbeg + kt * BK;
    issue_tile<BM, A_T>(ra, g.lda, m0, k0, st, wave, lane);
    issue_tile<BN, B_T>(rb, g.ldb, n0, k0, st + A_BYTES, wave, lane);
  };

  floatx16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

#pragma unroll
  for (int s = 0; s < NSTAGE - 1; ++s)
    if (s < nk) issue(s, stage(s));

  for (int kt0 = 0; kt0 < nk; kt0 += NSTAGE) {
#pragma unroll
    for (int S = 0; S < NSTAGE; ++S) {
      const int kt = kt0 + S;
      if (kt < nk) {
        // tile kt has landed once at most the loads of the tiles issued
        // after it are outstanding
        if (kt + NSTAGE - 2 < nk) wait_vmcnt<(NSTAGE - 2) * LOADS>();
        else wait_vmcnt<0>();
        block_barrier();
        // the stage read in the previous step now takes tile kt+NSTAGE-1
        if (kt + NSTAGE - 1 < nk) issue(kt + NSTAGE - 1, stage((S + NSTAGE - 1) % NSTAGE));

        const lds_char_t* a_s = stage(S);
        const lds_char_t* b_s = a_s + A_BYTES;
#pragma unroll
        for (int s = 0; s < BK / 16; ++s) {
          bf16x8 fa[TM], fb[TN];
#pragma unroll
          for (int i = 0; i < TM; ++i) fa[i] = read_frag<BM, A_T>(a_s, wm * WTM + i * 32, s, lane);
#pragma unroll
          for (int j = 0; j < TN; ++j) fb[j] = read_frag<BN, B_T>(b_s, wn * WTN + j * 32, s, lane);
#pragma unroll
          for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) acc[i][j] = mfma32(fb[j], fa[i], acc[i][j]);
        }
      }
    }
  }

  // epilogue: lane holds, for output row m, n = nb + 8*(r/4) + (r%4)
  const int lrow = lane & 31;
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = m0 + wm * WTM + i * 32 + lrow;
    if (m >= g.M) continue;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = n0 + wn * WTN + j * 32 + q * 8 + (lane >> 5) * 4;
        if (n >= g.N) continue;
        float v0 = acc[i][j][q * 4 + 0], v1 = acc[i][j][q * 4 + 1];
        float v2 = acc[i][j][q * 4 + 2], v3 = acc[i][j][q * 4 + 3];
        const size_t off = (size_t)m * g.ldc + n;
        if constexpr (EPI == EPI_F32) {
          float* C = static_cast<float*>(g.C) + (size_t)blockIdx.z * g.split_stride;
          float4* p = reinterpret_cast<float4*>(C + off);
          if (g.accumulate) {
            float4 o = *p;
            v0 += o.x; v1 += o.y; v2 += o.z; v3 += o.w;
          }
          *p = make_float4(v0, v1, v2, v3);
        } else if constexpr (EPI == EPI_GELU_BWD) {
          uint2 u = *reinterpret_cast<const uint2*>(g.aux + off);
          v0 *= gelu_tanh_grad(lo_f(u.x)); v1 *= gelu_tanh_grad(hi_f(u.x));
          v2 *= gelu_tanh_grad(lo_f(u.y)); v3 *= gelu_tanh_grad(hi_f(u.y));
          *reinterpret_cast<uint2*>(static_cast<bf16_t*>(g.C) + off) = make_uint2(pack2(v0, v1), pack2(v2, v3));
        } else {
          if (g.bias) {
            float4 b = *reinterpret_cast<const float4*>(g.bias + n);
            v0 += b.x; v1 += b.y; v2 += b.z; v3 += b.w;
          }
          if constexpr (EPI == EPI_GELU) {
            *reinterpret_cast<uint2*>(static_cast<bf16_t*>(g.C) + off) = make_uint2(pack2(v0, v1), pack2(v2, v3));
            *reinterpret_cast<uint2*>(g.C2 + off) =
                make_uint2(pack2(gelu_tanh(v0), gelu_tanh(v1)), pack2(gelu_tanh(v2), gelu_tanh(v3)));
          } else {
            if (g.residual) {
              uint2 r = *reinterpret_cast<const uint2*>(g.residual + off);
              v0 += lo_f(r.x); v1 += hi_f(r.x); v2 += lo_f(r.y); v3 += hi_f(r.y);
            }
            *reinterpret_cast<uint2*>(static_cast<bf16_t*>(g.C) + off) = make_uint2(pack2(v0, v1), pack2(v2, v3));
          }
        }
      }
    }
  }
}

template <int BM, int BN, bool A_T, bool B_T, int EPI>
hipError_t launch_t(const GemmArgs& g, hipStream_t s) {
  dim3 grid((g.N + BN - 1) / BN, (g.M + BM - 1) / BM, g.splits);
  hipLaunchKernelGGL((gemm_kernel<BM, BN, A_T, B_T, EPI>), grid, dim3(256), 0, s, g);
  return hipGetLastError();
}

// Tile shape per problem (see gemm_tile_shape): 256 x 192 tiles (4 waves of
// 128 x 96) when N is a multiple of 192, which holds for every GPT-2 width
// (768, 2304, 3072 and the padded vocabulary 50304) and makes the 16384-row
// GEMMs fill the 256 CUs in whole rounds; 256 x 128 otherwise; 128 x 128 for
// small problems.
template <bool A_T, bool B_T, int EPI>
hipError_t launch_shape(const GemmArgs& g, hipStream_t s) {
  int bm = 0, bn = 0;
  gemm_tile_shape(g.M, g.N, &bm, &bn);
  if (bm == 256 && bn == 192) return launch_t<256, 192, A_T, B_T, EPI>(g, s);
  if (bm == 256) return launch_t<256, 128, A_T, B_T, EPI>(g, s);
  return launch_t<128, 128, A_T, B_T, EPI>(g, s);
}

}  // namespace

void gemm_tile_shape(int M, int N, int* bm, int* bn) {
  if (M >= 256 && N >= 192 && N % 192 == 0) {
    *bm = 256; *bn = 192;
  } else if (M >= 256 && N >= 128 && N % 128 == 0) {
    *bm = 256; *bn = 128;
  } else {
    *bm = 128; *bn = 128;
  }
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
  if (!a_t && !b_t) {
    switch (epi) {
      case EPI_BF16: return launch_shape<false, false, EPI_BF16>(g, s);
      case EPI_GELU: return launch_shape<false, false, EPI_GELU>(g, s);
      default: break;
    }
  } else if (!a_t && b_t) {
    switch (epi) {
      case EPI_BF16: return launch_shape<false, true, EPI_BF16>(g, s);
      case EPI_GELU_BWD: return launch_shape<false, true, EPI_GELU_BWD>(g, s);
      default: break;
    }
  } else if (a_t && b_t) {
    if (epi == EPI_F32) return launch_shape<true, true, EPI_F32>(g, s);
  }
  return hipErrorInvalidValue;
}
