// Row-streaming products of the low-rank adapters (section "The clinical
// stage": adapters of rank r <= 32 on the projections): the down product
// u = s x A^T of the forward pass and du_j = s dy_j B_j of the backward pass.
// Each reads one tall operand once (x: tokens x in, dy: tokens x out) and
// contracts it with at most 32 weight rows per projection, so it is bound by
// the HBM stream of that operand, not by arithmetic.
//
// One workgroup per 16 rows of the tall operand. Its four waves take
// interleaved 64-wide contraction steps, so that together they read 512
// contiguous bytes of each of the 16 rows at a time. A lane loads 32
// contiguous bytes of one row (the A operand of two 16x16x32 MFMAs) and the
// same 32 contraction positions of one weight row (the B operand): both
// operands carry the same positions, so which positions an MFMA pairs up is
// immaterial. The four waves' fp32 sums meet in LDS, are added in a fixed
// order, scaled by s and rounded to bf16 once. Output columns that no weight
// row covers are written as zeros, so the padded-rank layout the consumers
// read is complete.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int LR_WAVES = 4;
constexpr int LR_STEP = 64;   // contraction positions per wave step

DEV floatx4 mfma16(bf16x8 a, bf16x8 b, floatx4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// row offset of tile t inside a segment's weight rows and output columns
DEV int tile_row(const LoraRowArgs& a, int t) { return (t / a.ntp) * a.tstride + 16 * (t % a.ntp); }

// NSEG contraction segments, NTS 16-column tiles per segment, RING steps per
// batch of loads (two batches in flight per wave).
template <int NSEG, int NTS, int RING>
__global__ __launch_bounds__(256, 2) void lora_rows_kernel(LoraRowArgs a) {
  constexpr int NT = NSEG * NTS;
  __shared__ float red[LR_WAVES][NT][16][16];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g = lane >> 4;
  const long m0 = (long)blockIdx.x * 16;
  const long mrow = min(m0 + r16, (long)a.M - 1);   // rows past M read row M-1 and are not stored
  const bf16_t* xrow = a.x + mrow * a.ldx + 16 * g;
  int nst[NSEG], S = 0;
#pragma unroll
  for (int q = 0; q < NSEG; ++q) {
    nst[q] = a.klen[q] / LR_STEP;
    S += nst[q];
  }
  // this wave's steps are wave, wave + 4, ... below S
  const int mine = S > wave ? (S - wave + LR_WAVES - 1) / LR_WAVES : 0;
  long wro[NTS];
#pragma unroll
  for (int t = 0; t < NTS; ++t) wro[t] = (long)(tile_row(a, t) + r16) * a.ldw + 16 * g;

  floatx4 acc[NT];
#pragma unroll
  for (int j = 0; j < NT; ++j) acc[j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

  // step i of this wave -> segment (-1 past the end) and contraction offset
  auto decode = [&](int i, int& p, int& kr) {
    p = -1;
    kr = 0;
    if (i >= mine) return;
    int s = wave + LR_WAVES * i;
#pragma unroll
    for (int q = 0; q < NSEG; ++q) {
      if (p < 0) {
        if (s < nst[q]) {
          p = q;
          kr = s * LR_STEP;
        } else {
          s -= nst[q];
        }
      }
    }
  };
  auto load = [&](uint4 (&xv)[RING][2], uint4 (&wv)[RING][NTS][2], int (&pv)[RING], int i0) {
#pragma unroll
    for (int r = 0; r < RING; ++r) {
      int p, kr;
      decode(i0 + r, p, kr);
      pv[r] = p;
#pragma unroll
      for (int q = 0; q < NSEG; ++q) {
        if (p == q) {
          const bf16_t* xp = xrow + a.k0[q] + kr;
          xv[r][0] = *reinterpret_cast<const uint4*>(xp);
          xv[r][1] = *reinterpret_cast<const uint4*>(xp + 8);
#pragma unroll
          for (int t = 0; t < NTS; ++t) {
            const bf16_t* wp = a.w[q] + wro[t] + kr;
            wv[r][t][0] = *reinterpret_cast<const uint4*>(wp);
            wv[r][t][1] = *reinterpret_cast<const uint4*>(wp + 8);
          }
        }
      }
    }
  };
  auto compute = [&](const uint4 (&xv)[RING][2], const uint4 (&wv)[RING][NTS][2], const int (&pv)[RING]) {
#pragma unroll
    for (int r = 0; r < RING; ++r) {
#pragma unroll
      for (int q = 0; q < NSEG; ++q) {
        if (pv[r] == q) {
#pragma unroll
          for (int t = 0; t < NTS; ++t) {
            acc[q * NTS + t] = mfma16(as_bf16x8(xv[r][0]), as_bf16x8(wv[r][t][0]), acc[q * NTS + t]);
            acc[q * NTS + t] = mfma16(as_bf16x8(xv[r][1]), as_bf16x8(wv[r][t][1]), acc[q * NTS + t]);
          }
        }
      }
    }
  };

  uint4 xa[RING][2], wa[RING][NTS][2], xb[RING][2], wb[RING][NTS][2];
  int pa[RING], pb[RING];
  load(xa, wa, pa, 0);
  for (int i0 = 0; i0 < mine; i0 += 2 * RING) {
    load(xb, wb, pb, i0 + RING);
    compute(xa, wa, pa);
    load(xa, wa, pa, i0 + 2 * RING);
    compute(xb, wb, pb);
  }

  // lane holds rows 4g..4g+3 of column r16 of each 16x16 tile
#pragma unroll
  for (int j = 0; j < NT; ++j)
#pragma unroll
    for (int e = 0; e < 4; ++e) red[wave][j][4 * g + e][r16] = acc[j][e];
  __syncthreads();

  // 4 output columns per thread and pass: the tile covering them (if any)
  // summed over the waves in order, scaled, rounded; zeros elsewhere
  const int nq = a.ldy / 4;
  for (int idx = tid; idx < 16 * nq; idx += 256) {
    const int rr = idx / nq, c = (idx - rr * nq) * 4;
    const long m = m0 + rr;
    if (m >= a.M) continue;
    float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int q = 0; q < NSEG; ++q)
#pragma unroll
      for (int t = 0; t < NTS; ++t) {
        const int c0 = a.col[q] + tile_row(a, t);
        if (c >= c0 && c < c0 + 16) {
          const int cc = c - c0;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int j = q * NTS + t;
            const float sum = ((red[0][j][rr][cc + e] + red[1][j][rr][cc + e]) + red[2][j][rr][cc + e]) +
                              red[3][j][rr][cc + e];
            v[e] = sum * a.s;
          }
        }
      }
    *reinterpret_cast<uint2*>(a.y + m * a.ldy + c) = make_uint2(pack2(v[0], v[1]), pack2(v[2], v[3]));
  }
}

template <int NSEG, int NTS>
hipError_t rows_t(const LoraRowArgs& a, hipStream_t s) {
  constexpr int RING = NTS == 1 ? 4 : NTS == 2 ? 2 : 1;
  hipLaunchKernelGGL((lora_rows_kernel<NSEG, NTS, RING>), dim3((a.M + 15) / 16), dim3(256), 0, s, a);
  return hipGetLastError();
}

// Bt[l][c][k] = B[l][k][c] for the first 32 columns c of B's rows (rp
// elements each), k < out: 64 rows of B per workgroup through LDS.
__global__ __launch_bounds__(256) void lora_bt_kernel(const bf16_t* __restrict__ B, bf16_t* __restrict__ Bt,
                                                      int out, int rp) {
  __shared__ bf16_t tile[64][32 + 2];
  const int tid = threadIdx.x, k0 = blockIdx.x * 64, l = blockIdx.y;
  const bf16_t* src = B + ((size_t)l * out + k0) * rp;
  bf16_t* dst = Bt + (size_t)l * 32 * out + k0;
  {
    const int row = tid >> 2, q = (tid & 3) * 8;
    const uint4 v = *reinterpret_cast<const uint4*>(src + (size_t)row * rp + q);
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      tile[row][q + 2 * e] = (bf16_t)(w[e] & 0xffffu);
      tile[row][q + 2 * e + 1] = (bf16_t)(w[e] >> 16);
    }
  }
  __syncthreads();
  const int c = tid >> 3, kq = (tid & 7) * 8;
  uint32_t w[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) w[e] = (uint32_t)tile[kq + 2 * e][c] | ((uint32_t)tile[kq + 2 * e + 1][c] << 16);
  *reinterpret_cast<uint4*>(dst + (size_t)c * out + kq) = make_uint4(w[0], w[1], w[2], w[3]);
}

}  // namespace

hipError_t launch_lora_rows(const LoraRowArgs& a, hipStream_t s) {
  if (a.M < 1 || a.nseg < 1 || a.nseg > 3 || a.ntp < 1 || a.ntp > 2 || a.nts < a.ntp || a.nts % a.ntp ||
      a.ldy % 4 || a.ldx % 8 || a.ldw % 8 || a.tstride % 16)
    return hipErrorInvalidValue;
  for (int q = 0; q < a.nseg; ++q)
    if (a.klen[q] < 0 || a.klen[q] % LR_STEP || a.k0[q] % 8 || a.k0[q] + a.klen[q] > a.ldx || a.col[q] % 4 ||
        a.col[q] + (a.nts / a.ntp - 1) * a.tstride + 16 * a.ntp > a.ldy)
      return hipErrorInvalidValue;
  switch (a.nseg * 8 + a.nts) {
    case 9: return rows_t<1, 1>(a, s);
    case 10: return rows_t<1, 2>(a, s);
    case 11: return rows_t<1, 3>(a, s);
    case 12: return rows_t<1, 4>(a, s);
    case 14: return rows_t<1, 6>(a, s);
    case 17: return rows_t<2, 1>(a, s);
    case 18: return rows_t<2, 2>(a, s);
    case 25: return rows_t<3, 1>(a, s);
    case 26: return rows_t<3, 2>(a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_lora_bt(const bf16_t* B, bf16_t* Bt, int L, int out, int rp, hipStream_t s) {
  if (L < 1 || out < 64 || out % 64 || rp < 32 || rp % 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(lora_bt_kernel, dim3(out / 64, L), dim3(256), 0, s, B, Bt, out, rp);
  return hipGetLastError();
}
