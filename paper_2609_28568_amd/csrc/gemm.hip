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
// Tiles of BM x BN x 64 are staged through LDS, double-buffered: the global
// loads of tile k+1 are in flight while the MFMAs of tile k run. LDS keeps
// every operand contraction-contiguous ([row][k], padded rows), so each MFMA
// operand is one 16-byte LDS read. Strided operands are transposed in
// registers on the way in: a thread loads a 4(k) x 8(row) block with four
// 16-byte loads and writes eight 8-byte rows.
//
// The MFMA is v_mfma_f32_32x32x16_bf16 with its row index i mapped to n and
// its column index j to m, so each lane ends up holding four consecutive n
// of one output row (8-byte bf16 / 16-byte fp32 stores).
#include "common.h"
#include "kernels.h"

namespace {

constexpr int BK = 64;
constexpr int LDK = BK + 8;   // padded LDS row (144 bytes) to spread banks

template <int R, bool TR, int NT>
struct TileLoader {
  // contraction-contiguous: R rows x 64 k as 16-byte chunks
  static constexpr int CH = TR ? 0 : (R * BK / 8) / NT;
  // contraction-strided: (64/4) x (R/8) blocks of 4 k x 8 rows
  static constexpr int UN = TR ? ((BK / 4) * (R / 8)) / NT : 0;
  static_assert(TR ? (((BK / 4) * (R / 8)) % NT == 0) : ((R * BK / 8) % NT == 0), "tile/threads");
  static constexpr int NREG = TR ? UN * 4 : CH;
  uint4 v[NREG];

  // rows: [r0, r0+R) of Rtot; contraction: [k0, k0+64) of kend
  DEV void load(const bf16_t* __restrict__ X, int ld, int r0, int Rtot, int k0, int kend, int tid) {
    if constexpr (!TR) {
#pragma unroll
      for (int i = 0; i < CH; ++i) {
        int c = tid + NT * i;
        int row = c >> 3, kc = (c & 7) * 8;
        int gr = r0 + row, gk = k0 + kc;
        if (gr < Rtot && gk < kend)
          v[i] = *reinterpret_cast<const uint4*>(X + (size_t)gr * ld + gk);
        else
          v[i] = make_uint4(0, 0, 0, 0);
      }
    } else {
#pragma unroll
      for (int i = 0; i < UN; ++i) {
        int u = tid + NT * i;
        int rc = u % (R / 8), kq = u / (R / 8);
        int gr = r0 + rc * 8;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          int gk = k0 + kq * 4 + q;
          if (gr < Rtot && gk < kend)
            v[i * 4 + q] = *reinterpret_cast<const uint4*>(X + (size_t)gk * ld + gr);
          else
            v[i * 4 + q] = make_uint4(0, 0, 0, 0);
        }
      }
    }
  }

  DEV void store(bf16_t* __restrict__ S, int tid) const {
    if constexpr (!TR) {
#pragma unroll
      for (int i = 0; i < CH; ++i) {
        int c = tid + NT * i;
        int row = c >> 3, kc = (c & 7) * 8;
        *reinterpret_cast<uint4*>(S + row * LDK + kc) = v[i];
      }
    } else {
#pragma unroll
      for (int i = 0; i < UN; ++i) {
        int u = tid + NT * i;
        int rc = u % (R / 8), kq = u / (R / 8);
        const uint4 w0 = v[i * 4 + 0], w1 = v[i * 4 + 1], w2 = v[i * 4 + 2], w3 = v[i * 4 + 3];
        const uint32_t a0[4] = {w0.x, w0.y, w0.z, w0.w};
        const uint32_t a1[4] = {w1.x, w1.y, w1.z, w1.w};
        const uint32_t a2[4] = {w2.x, w2.y, w2.z, w2.w};
        const uint32_t a3[4] = {w3.x, w3.y, w3.z, w3.w};
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          uint2 even = make_uint2(lo_pair(a0[p], a1[p]), lo_pair(a2[p], a3[p]));
          uint2 odd = make_uint2(hi_pair(a0[p], a1[p]), hi_pair(a2[p], a3[p]));
          *reinterpret_cast<uint2*>(S + (rc * 8 + 2 * p) * LDK + kq * 4) = even;
          *reinterpret_cast<uint2*>(S + (rc * 8 + 2 * p + 1) * LDK + kq * 4) = odd;
        }
      }
    }
  }
};

template <int BM, int BN, int WGM, int WGN, bool A_T, bool B_T, int EPI>
__global__ __launch_bounds__(WGM* WGN * 64) void gemm_kernel(GemmArgs g) {
  constexpr int NT = WGM * WGN * 64;
  constexpr int WTM = BM / WGM, WTN = BN / WGN;   // wave tile
  constexpr int TM = WTM / 32, TN = WTN / 32;     // 32x32 MFMA tiles per wave
  static_assert(WTM % 32 == 0 && WTN % 32 == 0, "wave tile");

  __shared__ __attribute__((aligned(16))) bf16_t smem[2 * (BM + BN) * LDK];
  constexpr int STAGE = (BM + BN) * LDK;   // one buffer: A rows then B rows

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WGN, wn = wave % WGN;
  const int m0 = blockIdx.y * BM, n0 = blockIdx.x * BN;

  // contraction range of this split
  const int kchunk = g.k_chunk;
  const int kbeg = blockIdx.z * kchunk;
  const int kend = min(g.K, kbeg + kchunk);
  const int nk = (kend - kbeg + BK - 1) / BK;

  TileLoader<BM, A_T, NT> la;
  TileLoader<BN, B_T, NT> lb;

  floatx16 acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  if (nk > 0) {
    la.load(g.A, g.lda, m0, g.M, kbeg, kend, tid);
    lb.load(g.B, g.ldb, n0, g.N, kbeg, kend, tid);
    la.store(smem, tid);
    lb.store(smem + BM * LDK, tid);
  }
  __syncthreads();

  const int lrow = lane & 31, lk = (lane >> 5) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) {
      la.load(g.A, g.lda, m0, g.M, kbeg + (kt + 1) * BK, kend, tid);
      lb.load(g.B, g.ldb, n0, g.N, kbeg + (kt + 1) * BK, kend, tid);
    }
    const bf16_t* a_s = smem + cur * STAGE + (wm * WTM + lrow) * LDK + lk;
    const bf16_t* b_s = smem + cur * STAGE + BM * LDK + (wn * WTN + lrow) * LDK + lk;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      uint4 fa[TM], fb[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) fa[i] = *reinterpret_cast<const uint4*>(a_s + i * 32 * LDK + kk);
#pragma unroll
      for (int j = 0; j < TN; ++j) fb[j] = *reinterpret_cast<const uint4*>(b_s + j * 32 * LDK + kk);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = mfma32(as_bf16x8(fb[j]), as_bf16x8(fa[i]), acc[i][j]);
    }
    if (kt + 1 < nk) {
      la.store(smem + (cur ^ 1) * STAGE, tid);
      lb.store(smem + (cur ^ 1) * STAGE + BM * LDK, tid);
    }
    __syncthreads();
  }

  // epilogue: lane holds, for output row m, n = nb + 8*(r/4) + (r%4)
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

template <int BM, int BN, int WGM, int WGN, bool A_T, bool B_T, int EPI>
hipError_t launch_t(const GemmArgs& g, hipStream_t s) {
  dim3 grid((g.N + BN - 1) / BN, (g.M + BM - 1) / BM, g.splits);
  hipLaunchKernelGGL((gemm_kernel<BM, BN, WGM, WGN, A_T, B_T, EPI>), grid, dim3(WGM * WGN * 64), 0, s, g);
  return hipGetLastError();
}

template <bool A_T, bool B_T, int EPI>
hipError_t launch_shape(const GemmArgs& g, hipStream_t s) {
  return launch_t<128, 128, 2, 2, A_T, B_T, EPI>(g, s);
}

}  // namespace

int gemm_split_plan(int K, int want, int* k_chunk) {
  if (want < 1) want = 1;
  int kc = (K + want - 1) / want;
  kc = (kc + BK - 1) / BK * BK;
  if (kc < BK) kc = BK;
  if (k_chunk) *k_chunk = kc;
  int n = (K + kc - 1) / kc;
  return n < 1 ? 1 : n;
}

hipError_t launch_gemm(const GemmArgs& g0, int a_t, int b_t, int epi, hipStream_t s) {
  GemmArgs g = g0;
  if (g.splits <= 1 || g.k_chunk <= 0) {
    g.splits = 1;
    g.k_chunk = (g.K + BK - 1) / BK * BK;
    if (g.k_chunk < BK) g.k_chunk = BK;
  } else {
    // the caller's plan: k_chunk a multiple of 64 and splits = ceil(K / k_chunk)
    if (g.k_chunk % BK || (long)g.k_chunk * g.splits < g.K || (long)g.k_chunk * (g.splits - 1) >= g.K)
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
