// Causal multi-head attention for gfx950, flash style (online softmax, the
// score matrix never leaves the chip).
//
// Layout: q|k|v packed per token [B*T, 3C], head h on channels
// [h*hd, (h+1)*hd) of each third; output [B*T, C]; log-sum-exp of the scaled
// scores [B, H, T] in fp32 for the backward pass.
//
// All products use v_mfma_f32_32x32x16_bf16. Scores are computed transposed
// (keys along the MFMA row index i, queries along the column index j) so that
// one lane holds 16 scores of a single query: softmax statistics then need a
// reduction over the lane's own registers plus one exchange with lane ^ 32.
// The probabilities feed the next product straight from registers: an MFMA
// only needs A and B to agree on which contraction index sits in each of the
// lane's 8 slots, so the value operand is read from LDS in the order the
// score accumulator already has (two 8-byte reads per operand).
//
// Backward: dK/dV by a kernel that owns a key block and walks query tiles,
// dQ by a kernel that owns a query block and walks key tiles; both recompute
// P from the saved log-sum-exp and D = rowsum(dO * O) from a small pre-pass.
#include "common.h"
#include "kernels.h"

namespace {

constexpr int BKV = 64;     // keys (or queries) per LDS tile
constexpr int BQ = 128;     // rows owned by one workgroup (4 waves x 32)
constexpr int LDT = BKV + 8;
constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

// rows [r0, r0+64) of one head's slice of a q/k/v section -> S[64][HD+8]
template <int HD>
DEV void load_rows(bf16_t* S, const bf16_t* src, int r0, int T, int ld, int tid) {
  constexpr int CPR = HD / 8;
  for (int c = tid; c < BKV * CPR; c += 256) {
    int r = c / CPR, cc = (c % CPR) * 8;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (r0 + r < T) v = *reinterpret_cast<const uint4*>(src + (size_t)(r0 + r) * ld + cc);
    *reinterpret_cast<uint4*>(S + r * (HD + 8) + cc) = v;
  }
}

// same rows, transposed: St[d][r] (rows of 64+8)
template <int HD>
DEV void load_rows_t(bf16_t* St, const bf16_t* src, int r0, int T, int ld, int tid) {
  constexpr int CPR = HD / 8;
  for (int u = tid; u < (BKV / 4) * CPR; u += 256) {
    int dc = (u % CPR) * 8, rq = (u / CPR) * 4;
    uint32_t w[4][4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (r0 + rq + q < T) v = *reinterpret_cast<const uint4*>(src + (size_t)(r0 + rq + q) * ld + dc);
      w[q][0] = v.x; w[q][1] = v.y; w[q][2] = v.z; w[q][3] = v.w;
    }
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      *reinterpret_cast<uint2*>(St + (dc + 2 * p) * LDT + rq) =
          make_uint2(lo_pair(w[0][p], w[1][p]), lo_pair(w[2][p], w[3][p]));
      *reinterpret_cast<uint2*>(St + (dc + 2 * p + 1) * LDT + rq) =
          make_uint2(hi_pair(w[0][p], w[1][p]), hi_pair(w[2][p], w[3][p]));
    }
  }
}

// Operand read from a transposed tile St[d][r] in the slot order of a
// 32x32 accumulator: k-step (t, h) covers rows 32t+16h + {4g..4g+3, 8+4g..8+4g+3}.
DEV bf16x8 read_t_slots(const bf16_t* St, int drow, int t, int h, int g) {
  const bf16_t* p = St + drow * LDT + 32 * t + 16 * h + 4 * g;
  uint2 a = *reinterpret_cast<const uint2*>(p);
  uint2 b = *reinterpret_cast<const uint2*>(p + 8);
  return as_bf16x8(make_uint4(a.x, a.y, b.x, b.y));
}

// Registers 8h..8h+7 of a 32x32 fp32 accumulator as a bf16 operand.
DEV bf16x8 acc_slots(const floatx16& x, int h) {
  return as_bf16x8(make_uint4(pack2(x[8 * h + 0], x[8 * h + 1]), pack2(x[8 * h + 2], x[8 * h + 3]),
                              pack2(x[8 * h + 4], x[8 * h + 5]), pack2(x[8 * h + 6], x[8 * h + 7])));
}

// row offset of accumulator register r for lane group g: 8*(r/4) + 4g + r%4
DEV int acc_row(int r, int g) { return 8 * (r >> 2) + 4 * g + (r & 3); }

template <int HD>
__global__ __launch_bounds__(256) void attn_fwd_kernel(AttnArgs a) {
  constexpr int HDP = HD < 32 ? 32 : HD;
  constexpr int KS = HD / 16;     // k-steps over the head dimension
  constexpr int DT = HDP / 32;    // 32-row tiles over the head dimension
  __shared__ __attribute__((aligned(16))) bf16_t Ks[BKV * (HD + 8)];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[HDP * LDT];

  const int T = a.T, H = a.H, C = H * HD, ld = 3 * C;
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int qb = gridDim.x - 1 - blockIdx.x;   // heaviest blocks first
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lq = lane & 31, g = lane >> 5;
  const int q0w = qb * BQ + wave * 32;
  const int q = q0w + lq;
  const bf16_t* base = a.qkv + (size_t)b * T * ld + h * HD;

  if (HD < 32)
    for (int i = tid; i < (HDP - HD) * LDT; i += 256) Vt[HD * LDT + i] = 0;

  bf16x8 qf[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    uint4 v = make_uint4(0, 0, 0, 0);
    if (q < T) v = *reinterpret_cast<const uint4*>(base + (size_t)q * ld + 16 * s + 8 * g);
    qf[s] = as_bf16x8(v);
  }

  floatx16 o[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) o[d][r] = 0.0f;
  float m_run = -INFINITY, l_run = 0.0f;
  const float sc = LOG2E / sqrtf((float)HD);

  const int kv_end = min(T, qb * BQ + BQ);
  for (int kv0 = 0; kv0 < kv_end; kv0 += BKV) {
    __syncthreads();
    load_rows<HD>(Ks, base + C, kv0, T, ld, tid);
    load_rows_t<HD>(Vt, base + 2 * C, kv0, T, ld, tid);
    __syncthreads();
    if (kv0 > q0w + 31) continue;   // every query of this wave precedes the tile

    floatx16 s[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[t][r] = 0.0f;
#pragma unroll
      for (int k = 0; k < KS; ++k) {
        uint4 kv = *reinterpret_cast<const uint4*>(Ks + (32 * t + lq) * (HD + 8) + 16 * k + 8 * g);
        s[t] = mfma32(as_bf16x8(kv), qf[k], s[t]);
      }
    }
    float mt = -INFINITY;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int j = kv0 + 32 * t + acc_row(r, g);
        float x = (j <= q && j < T) ? s[t][r] * sc : -INFINITY;
        s[t][r] = x;
        mt = fmaxf(mt, x);
      }
    mt = fmaxf(mt, __shfl_xor(mt, 32, WAVE));
    const float m_new = fmaxf(m_run, mt);
    const float alpha = exp2f(m_run - m_new);
    float rs = 0.0f;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float p = exp2f(s[t][r] - m_new);
        s[t][r] = p;
        rs += p;
      }
    rs += __shfl_xor(rs, 32, WAVE);
    l_run = l_run * alpha + rs;
    m_run = m_new;
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[d][r] *= alpha;
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        bf16x8 pf = acc_slots(s[t], hh);
#pragma unroll
        for (int d = 0; d < DT; ++d) o[d] = mfma32(read_t_slots(Vt, 32 * d + lq, t, hh, g), pf, o[d]);
      }
  }

  if (q < T) {
    const float inv = 1.0f / l_run;
    bf16_t* out = a.out + ((size_t)b * T + q) * C + h * HD;
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        int dd = 32 * d + 8 * c + 4 * g;
        if (dd < HD)
          *reinterpret_cast<uint2*>(out + dd) =
              make_uint2(pack2(o[d][4 * c] * inv, o[d][4 * c + 1] * inv),
                         pack2(o[d][4 * c + 2] * inv, o[d][4 * c + 3] * inv));
      }
    if (g == 0) a.lse[(size_t)bh * T + q] = (m_run + log2f(l_run)) * LN2;
  }
}

// D[b,h,t] = sum_d dO * O, one thread per (token, head)
template <int HD>
__global__ void attn_dsum_kernel(AttnArgs a) {
  const int C = a.H * HD;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)a.B * a.T * a.H) return;
  const int h = idx % a.H;
  const long tok = idx / a.H;
  const int b = tok / a.T, t = tok % a.T;
  const bf16_t* o = a.out + tok * C + h * HD;
  const bf16_t* d = a.dout + tok * C + h * HD;
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < HD; i += 8) {
    uint4 x = *reinterpret_cast<const uint4*>(o + i), y = *reinterpret_cast<const uint4*>(d + i);
    acc += lo_f(x.x) * lo_f(y.x) + hi_f(x.x) * hi_f(y.x) + lo_f(x.y) * lo_f(y.y) + hi_f(x.y) * hi_f(y.y);
    acc += lo_f(x.z) * lo_f(y.z) + hi_f(x.z) * hi_f(y.z) + lo_f(x.w) * lo_f(y.w) + hi_f(x.w) * hi_f(y.w);
  }
  a.dsum[((size_t)b * a.H + h) * a.T + t] = acc;
}

// dK, dV for a block of 128 keys (4 waves x 32), walking query tiles of 64.
template <int HD>
__global__ __launch_bounds__(256) void attn_bwd_dkdv_kernel(AttnArgs a) {
  constexpr int HDP = HD < 32 ? 32 : HD;
  constexpr int KS = HD / 16, DT = HDP / 32;
  __shared__ __attribute__((aligned(16))) bf16_t Qs[BKV * (HD + 8)];
  __shared__ __attribute__((aligned(16))) bf16_t Qt[HDP * LDT];
  __shared__ __attribute__((aligned(16))) bf16_t Ds[BKV * (HD + 8)];
  __shared__ __attribute__((aligned(16))) bf16_t Dt[HDP * LDT];
  __shared__ float lse_s[BKV], dsum_s[BKV];

  const int T = a.T, H = a.H, C = H * HD, ld = 3 * C;
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int kb = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lq = lane & 31, g = lane >> 5;
  const int kv0w = kb * BQ + wave * 32;
  const int kv = kv0w + lq;
  const bf16_t* base = a.qkv + (size_t)b * T * ld + h * HD;
  const bf16_t* dob = a.dout + (size_t)b * T * C + h * HD;

  if (HD < 32)
    for (int i = tid; i < (HDP - HD) * LDT; i += 256) {
      Qt[HD * LDT + i] = 0;
      Dt[HD * LDT + i] = 0;
    }

  bf16x8 kf[KS], vf[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    uint4 k4 = make_uint4(0, 0, 0, 0), v4 = make_uint4(0, 0, 0, 0);
    if (kv < T) {
      k4 = *reinterpret_cast<const uint4*>(base + (size_t)kv * ld + C + 16 * s + 8 * g);
      v4 = *reinterpret_cast<const uint4*>(base + (size_t)kv * ld + 2 * C + 16 * s + 8 * g);
    }
    kf[s] = as_bf16x8(k4);
    vf[s] = as_bf16x8(v4);
  }
  floatx16 dk[DT], dv[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) dk[d][r] = dv[d][r] = 0.0f;
  const float scale = 1.0f / sqrtf((float)HD);
  const float sc = scale * LOG2E;

  for (int q0 = kb * BQ; q0 < T; q0 += BKV) {
    __syncthreads();
    load_rows<HD>(Qs, base, q0, T, ld, tid);
    load_rows_t<HD>(Qt, base, q0, T, ld, tid);
    load_rows<HD>(Ds, dob, q0, T, C, tid);
    load_rows_t<HD>(Dt, dob, q0, T, C, tid);
    if (tid < BKV) {
      int qq = q0 + tid;
      lse_s[tid] = qq < T ? a.lse[(size_t)bh * T + qq] * LOG2E : 0.0f;
      dsum_s[tid] = qq < T ? a.dsum[(size_t)bh * T + qq] : 0.0f;
    }
    __syncthreads();
    if (q0 + BKV - 1 < kv0w) continue;   // every query of the tile precedes this wave's keys

    floatx16 p[2], ds[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int r = 0; r < 16; ++r) p[t][r] = ds[t][r] = 0.0f;
#pragma unroll
      for (int k = 0; k < KS; ++k) {
        uint4 qa = *reinterpret_cast<const uint4*>(Qs + (32 * t + lq) * (HD + 8) + 16 * k + 8 * g);
        uint4 da = *reinterpret_cast<const uint4*>(Ds + (32 * t + lq) * (HD + 8) + 16 * k + 8 * g);
        p[t] = mfma32(as_bf16x8(qa), kf[k], p[t]);
        ds[t] = mfma32(as_bf16x8(da), vf[k], ds[t]);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int qi = 32 * t + acc_row(r, g);
        int qq = q0 + qi;
        float pv = (kv <= qq && qq < T && kv < T) ? exp2f(p[t][r] * sc - lse_s[qi]) : 0.0f;
        p[t][r] = pv;
        ds[t][r] = pv * (ds[t][r] - dsum_s[qi]);
      }
    }
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        bf16x8 pf = acc_slots(p[t], hh), sf = acc_slots(ds[t], hh);
#pragma unroll
        for (int d = 0; d < DT; ++d) {
          dv[d] = mfma32(read_t_slots(Dt, 32 * d + lq, t, hh, g), pf, dv[d]);
          dk[d] = mfma32(read_t_slots(Qt, 32 * d + lq, t, hh, g), sf, dk[d]);
        }
      }
  }

  if (kv < T) {
    bf16_t* dst = a.dqkv + ((size_t)b * T + kv) * ld + h * HD;
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        int dd = 32 * d + 8 * c + 4 * g;
        if (dd < HD) {
          *reinterpret_cast<uint2*>(dst + C + dd) =
              make_uint2(pack2(dk[d][4 * c] * scale, dk[d][4 * c + 1] * scale),
                         pack2(dk[d][4 * c + 2] * scale, dk[d][4 * c + 3] * scale));
          *reinterpret_cast<uint2*>(dst + 2 * C + dd) =
              make_uint2(pack2(dv[d][4 * c], dv[d][4 * c + 1]), pack2(dv[d][4 * c + 2], dv[d][4 * c + 3]));
        }
      }
  }
}

// dQ for a block of 128 queries (4 waves x 32), walking key tiles of 64.
template <int HD>
__global__ __launch_bounds__(256) void attn_bwd_dq_kernel(AttnArgs a) {
  constexpr int HDP = HD < 32 ? 32 : HD;
  constexpr int KS = HD / 16, DT = HDP / 32;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[BKV * (HD + 8)];
  __shared__ __attribute__((aligned(16))) bf16_t Kt[HDP * LDT];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[BKV * (HD + 8)];

  const int T = a.T, H = a.H, C = H * HD, ld = 3 * C;
  const int bh = blockIdx.y, b = bh / H, h = bh % H;
  const int qb = gridDim.x - 1 - blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lq = lane & 31, g = lane >> 5;
  const int q0w = qb * BQ + wave * 32;
  const int q = q0w + lq;
  const bf16_t* base = a.qkv + (size_t)b * T * ld + h * HD;
  const bf16_t* dob = a.dout + (size_t)b * T * C + h * HD;

  if (HD < 32)
    for (int i = tid; i < (HDP - HD) * LDT; i += 256) Kt[HD * LDT + i] = 0;

  bf16x8 qf[KS], df[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    uint4 q4 = make_uint4(0, 0, 0, 0), d4 = make_uint4(0, 0, 0, 0);
    if (q < T) {
      q4 = *reinterpret_cast<const uint4*>(base + (size_t)q * ld + 16 * s + 8 * g);
      d4 = *reinterpret_cast<const uint4*>(dob + (size_t)q * C + 16 * s + 8 * g);
    }
    qf[s] = as_bf16x8(q4);
    df[s] = as_bf16x8(d4);
  }
  const float lse2 = q < T ? a.lse[(size_t)bh * T + q] * LOG2E : 0.0f;
  const float dsum = q < T ? a.dsum[(size_t)bh * T + q] : 0.0f;
  floatx16 dq[DT];
#pragma unroll
  for (int d = 0; d < DT; ++d)
#pragma unroll
    for (int r = 0; r < 16; ++r) dq[d][r] = 0.0f;
  const float scale = 1.0f / sqrtf((float)HD);
  const float sc = scale * LOG2E;

  const int kv_end = min(T, qb * BQ + BQ);
  for (int kv0 = 0; kv0 < kv_end; kv0 += BKV) {
    __syncthreads();
    load_rows<HD>(Ks, base + C, kv0, T, ld, tid);
    load_rows_t<HD>(Kt, base + C, kv0, T, ld, tid);
    load_rows<HD>(Vs, base + 2 * C, kv0, T, ld, tid);
    __syncthreads();
    if (kv0 > q0w + 31) continue;

    floatx16 p[2], ds[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
#pragma unroll
      for (int r = 0; r < 16; ++r) p[t][r] = ds[t][r] = 0.0f;
#pragma unroll
      for (int k = 0; k < KS; ++k) {
        uint4 ka = *reinterpret_cast<const uint4*>(Ks + (32 * t + lq) * (HD + 8) + 16 * k + 8 * g);
        uint4 va = *reinterpret_cast<const uint4*>(Vs + (32 * t + lq) * (HD + 8) + 16 * k + 8 * g);
        p[t] = mfma32(as_bf16x8(ka), qf[k], p[t]);
        ds[t] = mfma32(as_bf16x8(va), df[k], ds[t]);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        int j = kv0 + 32 * t + acc_row(r, g);
        float pv = (j <= q && j < T && q < T) ? exp2f(p[t][r] * sc - lse2) : 0.0f;
        ds[t][r] = pv * (ds[t][r] - dsum);
      }
    }
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        bf16x8 sf = acc_slots(ds[t], hh);
#pragma unroll
        for (int d = 0; d < DT; ++d) dq[d] = mfma32(read_t_slots(Kt, 32 * d + lq, t, hh, g), sf, dq[d]);
      }
  }

  if (q < T) {
    bf16_t* dst = a.dqkv + ((size_t)b * T + q) * ld + h * HD;
#pragma unroll
    for (int d = 0; d < DT; ++d)
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        int dd = 32 * d + 8 * c + 4 * g;
        if (dd < HD)
          *reinterpret_cast<uint2*>(dst + dd) =
              make_uint2(pack2(dq[d][4 * c] * scale, dq[d][4 * c + 1] * scale),
                         pack2(dq[d][4 * c + 2] * scale, dq[d][4 * c + 3] * scale));
      }
  }
}

template <int HD>
hipError_t fwd_t(const AttnArgs& a, hipStream_t s) {
  dim3 grid((a.T + BQ - 1) / BQ, a.B * a.H);
  hipLaunchKernelGGL(attn_fwd_kernel<HD>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int HD>
hipError_t bwd_t(const AttnArgs& a, hipStream_t s) {
  long n = (long)a.B * a.T * a.H;
  hipLaunchKernelGGL(attn_dsum_kernel<HD>, dim3((n + 255) / 256), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 grid((a.T + BQ - 1) / BQ, a.B * a.H);
  hipLaunchKernelGGL(attn_bwd_dkdv_kernel<HD>, grid, dim3(256), 0, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(attn_bwd_dq_kernel<HD>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_fwd(const AttnArgs& a, hipStream_t s) {
  switch (a.hd) {
    case 16: return fwd_t<16>(a, s);
    case 32: return fwd_t<32>(a, s);
    case 64: return fwd_t<64>(a, s);
    case 128: return fwd_t<128>(a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_attention_bwd(const AttnArgs& a, hipStream_t s) {
  switch (a.hd) {
    case 16: return bwd_t<16>(a, s);
    case 32: return bwd_t<32>(a, s);
    case 64: return bwd_t<64>(a, s);
    case 128: return bwd_t<128>(a, s);
  }
  return hipErrorInvalidValue;
}
