// Elementwise and normalisation kernels of the Qwen3-shaped adapter step:
// token gather from a bf16 table, RMSNorm forward and backward over rows, the
// per-head RMSNorm + rotary embedding of queries and keys (output in the same
// q|k|v layout, which the grouped-query attention kernels read in place), the
// SwiGLU gate and its derivative, and an in-place scale.
#include "common.h"
#include "kernels.h"

namespace {

// x[row] = table[id[row]] (bf16 rows of C elements, C a multiple of 8)
__global__ void embed_gather_kernel(const int32_t* __restrict__ ids, const bf16_t* __restrict__ table,
                                    bf16_t* __restrict__ x, long rows, int C) {
  const long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 8;
  if (i >= rows * C) return;
  const long row = i / C;
  const int c = (int)(i % C);
  *reinterpret_cast<uint4*>(x + i) = *reinterpret_cast<const uint4*>(table + (size_t)ids[row] * C + c);
}

// Row maps of the positions that carry loss: of every T rows (one sequence)
// the last T - mask_from do. Compact row i (over those rows only) is input
// row loss_row(i); input row p has compact index loss_index(p) when
// p % T >= mask_from. With mask_from = 0 both maps are the identity.
DEV int loss_row(int i, int T, int mask_from) {
  const int n = T - mask_from;
  return (i / n) * T + mask_from + i % n;
}
DEV int loss_index(int p, int T, int mask_from) {
  return (p / T) * (T - mask_from) + p % T - mask_from;
}

// One row per wave; lane owns 4-channel chunks c = 4*(lane + 64*i). Loads of
// a row are issued at once from clamped addresses and masked afterwards.
// Output row i normalises input row loss_row(i) (rows = output rows).
template <int MAXCH>
__global__ __launch_bounds__(256) void rmsnorm_fwd_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ w,
                                                          bf16_t* __restrict__ y, float* __restrict__ rstd_out,
                                                          int rows, int C, float eps, int T, int mask_from) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const bf16_t* xr = x + (size_t)loss_row(row, T, mask_from) * C;
  uint2 xu[MAXCH], wu[MAXCH];
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const int c = min(4 * (lane + 64 * i), C - 4);
    xu[i] = *reinterpret_cast<const uint2*>(xr + c);
    wu[i] = *reinterpret_cast<const uint2*>(w + c);
  }
  float v[MAXCH][4];
  float ss = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const bool in = 4 * (lane + 64 * i) < C;
    v[i][0] = in ? lo_f(xu[i].x) : 0.0f;
    v[i][1] = in ? hi_f(xu[i].x) : 0.0f;
    v[i][2] = in ? lo_f(xu[i].y) : 0.0f;
    v[i][3] = in ? hi_f(xu[i].y) : 0.0f;
    ss += v[i][0] * v[i][0] + v[i][1] * v[i][1] + v[i][2] * v[i][2] + v[i][3] * v[i][3];
  }
  const float rstd = 1.0f / sqrtf(wave_sum(ss) / C + eps);
  bf16_t* yr = y + (size_t)row * C;
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const int c = 4 * (lane + 64 * i);
    if (c < C) {
      const float o0 = v[i][0] * rstd * lo_f(wu[i].x), o1 = v[i][1] * rstd * hi_f(wu[i].x);
      const float o2 = v[i][2] * rstd * lo_f(wu[i].y), o3 = v[i][3] * rstd * hi_f(wu[i].y);
      *reinterpret_cast<uint2*>(yr + c) = make_uint2(pack2(o0, o1), pack2(o2, o3));
    }
  }
  if (lane == 0) rstd_out[row] = rstd;
}

// dres (=|+=) rstd (g - xhat mean(g xhat)), g = dy w, xhat = x rstd (gain frozen).
// dy and rstd hold compact rows (loss_index); rows p with p % T < mask_from
// have no upstream gradient: dres is left as is (accumulate) or zeroed.
template <int MAXCH>
__global__ __launch_bounds__(256) void rmsnorm_bwd_kernel(const bf16_t* __restrict__ dy, const bf16_t* __restrict__ x,
                                                          const float* __restrict__ rstd_in,
                                                          const bf16_t* __restrict__ w, bf16_t* __restrict__ dres,
                                                          int accumulate, int rows, int C, int T, int mask_from) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  bf16_t* rr = dres + (size_t)row * C;
  if (row % T < mask_from) {
    if (!accumulate)
      for (int c = 4 * lane; c < C; c += 256) *reinterpret_cast<uint2*>(rr + c) = make_uint2(0, 0);
    return;
  }
  const int ci = loss_index(row, T, mask_from);
  const bf16_t* xr = x + (size_t)row * C;
  const bf16_t* dr = dy + (size_t)ci * C;
  uint2 xu[MAXCH], du[MAXCH], wu[MAXCH], ru[MAXCH];
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const int c = min(4 * (lane + 64 * i), C - 4);
    xu[i] = *reinterpret_cast<const uint2*>(xr + c);
    du[i] = *reinterpret_cast<const uint2*>(dr + c);
    wu[i] = *reinterpret_cast<const uint2*>(w + c);
    ru[i] = accumulate ? *reinterpret_cast<const uint2*>(rr + c) : make_uint2(0, 0);
  }
  const float rstd = rstd_in[ci];
  float xh[MAXCH][4], g[MAXCH][4];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const bool in = 4 * (lane + 64 * i) < C;
    const float xv[4] = {lo_f(xu[i].x), hi_f(xu[i].x), lo_f(xu[i].y), hi_f(xu[i].y)};
    const float dv[4] = {lo_f(du[i].x), hi_f(du[i].x), lo_f(du[i].y), hi_f(du[i].y)};
    const float wv[4] = {lo_f(wu[i].x), hi_f(wu[i].x), lo_f(wu[i].y), hi_f(wu[i].y)};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      xh[i][e] = in ? xv[e] * rstd : 0.0f;
      g[i][e] = in ? dv[e] * wv[e] : 0.0f;
      s += g[i][e] * xh[i][e];
    }
  }
  const float m = wave_sum(s) / C;
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const int c = 4 * (lane + 64 * i);
    if (c < C) {
      float o[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) o[e] = rstd * (g[i][e] - xh[i][e] * m);
      o[0] += lo_f(ru[i].x); o[1] += hi_f(ru[i].x); o[2] += lo_f(ru[i].y); o[3] += hi_f(ru[i].y);
      *reinterpret_cast<uint2*>(rr + c) = make_uint2(pack2(o[0], o[1]), pack2(o[2], o[3]));
    }
  }
}

// Per (token, head slot) item of width 128: 16 lanes, lane i of the group
// holding elements 8i..8i+7, four items per wave; the rotary pair (e, e + 64)
// is lanes (i, i ^ 8) of the group. Query heads 0..H-1 and key heads
// 0..Hkv-1 are RMS-normalised with their gains and rotated by the token's
// angles (cos/sin tables [T][64] in fp32); value heads are copied. The output
// has the input's layout, q [H*128] | k [Hkv*128] | v [Hkv*128] per token,
// which the grouped-query attention kernels read directly. Items are whole
// 16-lane groups, so a group that runs past the end exits as a whole and
// every shuffle stays inside a group.
constexpr int QK_HD = 128;

DEV float group16_sum(float v) {
  v += __shfl_xor(v, 8);
  v += __shfl_xor(v, 4);
  v += __shfl_xor(v, 2);
  v += __shfl_xor(v, 1);
  return v;
}

DEV void unpack8(const uint4& u, float* v) {
  v[0] = lo_f(u.x); v[1] = hi_f(u.x); v[2] = lo_f(u.y); v[3] = hi_f(u.y);
  v[4] = lo_f(u.z); v[5] = hi_f(u.z); v[6] = lo_f(u.w); v[7] = hi_f(u.w);
}

DEV uint4 pack8(const float* v) {
  return make_uint4(pack2(v[0], v[1]), pack2(v[2], v[3]), pack2(v[4], v[5]), pack2(v[6], v[7]));
}

// the 8 cos and sin values of elements 8i..8i+7 (frequency index (8i) mod 64)
DEV void rope_coefs(const float* __restrict__ cosT, const float* __restrict__ sinT, int t, int sub, float* c,
                    float* sn) {
  const int p = (8 * sub) & 63;
  const float4 c0 = *reinterpret_cast<const float4*>(cosT + (size_t)t * 64 + p);
  const float4 c1 = *reinterpret_cast<const float4*>(cosT + (size_t)t * 64 + p + 4);
  const float4 s0 = *reinterpret_cast<const float4*>(sinT + (size_t)t * 64 + p);
  const float4 s1 = *reinterpret_cast<const float4*>(sinT + (size_t)t * 64 + p + 4);
  c[0] = c0.x; c[1] = c0.y; c[2] = c0.z; c[3] = c0.w; c[4] = c1.x; c[5] = c1.y; c[6] = c1.z; c[7] = c1.w;
  sn[0] = s0.x; sn[1] = s0.y; sn[2] = s0.z; sn[3] = s0.w; sn[4] = s1.x; sn[5] = s1.y; sn[6] = s1.z; sn[7] = s1.w;
}

__global__ __launch_bounds__(256) void qknorm_rope_fwd_kernel(const bf16_t* __restrict__ raw, const bf16_t* __restrict__ qn_w,
                                                              const bf16_t* __restrict__ kn_w, const float* __restrict__ cosT,
                                                              const float* __restrict__ sinT, bf16_t* __restrict__ packed,
                                                              float* __restrict__ rq, float* __restrict__ rk, int BT, int T,
                                                              int H, int Hkv, float eps) {
  const int sub = threadIdx.x & 15;
  const long item = ((long)blockIdx.x * blockDim.x + threadIdx.x) >> 4;   // (token, head slot) over H + 2 Hkv slots
  const int slots = H + 2 * Hkv;
  if (item >= (long)BT * slots) return;
  const int tok = (int)(item / slots), hs = (int)(item % slots);
  const int t = tok % T;
  const size_t off = (size_t)tok * slots * QK_HD + hs * QK_HD + 8 * sub;
  const uint4 u = *reinterpret_cast<const uint4*>(raw + off);
  if (hs >= H + Hkv) {   // value head: copied
    *reinterpret_cast<uint4*>(packed + off) = u;
    return;
  }
  const bool isq = hs < H;
  float x[8];
  unpack8(u, x);
  float ss = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) ss += x[e] * x[e];
  const float rstd = 1.0f / sqrtf(group16_sum(ss) / QK_HD + eps);
  const uint4 wu = *reinterpret_cast<const uint4*>((isq ? qn_w : kn_w) + 8 * sub);
  float w[8];
  unpack8(wu, w);
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = x[e] * rstd * w[e];
  // rotate: first half x1 cos - x2 sin, second half x2 cos + x1 sin
  float c[8], sn[8];
  rope_coefs(cosT, sinT, t, sub, c, sn);
  const float sgn = sub < 8 ? -1.0f : 1.0f;
  float y[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) y[e] = x[e] * c[e] + sgn * __shfl_xor(x[e], 8) * sn[e];
  *reinterpret_cast<uint4*>(packed + off) = pack8(y);
  if (sub == 0) {
    if (isq) rq[(size_t)tok * H + hs] = rstd;
    else rk[(size_t)tok * Hkv + (hs - H)] = rstd;
  }
}

// Backward of qknorm_rope_fwd_kernel: dpacked -> draw, both in the q|k|v
// layout (the attention backward has already summed a key/value head's
// gradient over its query heads); queries and keys go back through the
// rotation (its transpose) and the RMSNorm, values pass through. Same item
// layout.
__global__ __launch_bounds__(256) void qknorm_rope_bwd_kernel(const bf16_t* __restrict__ dpacked, const bf16_t* __restrict__ raw,
                                                              const bf16_t* __restrict__ qn_w, const bf16_t* __restrict__ kn_w,
                                                              const float* __restrict__ cosT, const float* __restrict__ sinT,
                                                              const float* __restrict__ rq, const float* __restrict__ rk,
                                                              bf16_t* __restrict__ draw, int BT, int T, int H, int Hkv) {
  const int sub = threadIdx.x & 15;
  const long item = ((long)blockIdx.x * blockDim.x + threadIdx.x) >> 4;
  const int slots = H + 2 * Hkv;
  if (item >= (long)BT * slots) return;
  const int tok = (int)(item / slots), hs = (int)(item % slots);
  const int t = tok % T;
  const size_t off = (size_t)tok * slots * QK_HD + hs * QK_HD + 8 * sub;
  const uint4 du = *reinterpret_cast<const uint4*>(dpacked + off);
  if (hs >= H + Hkv) {   // value head: passes through
    *reinterpret_cast<uint4*>(draw + off) = du;
    return;
  }
  float d[8];
  unpack8(du, d);
  // transposed rotation: first half d1 cos + d2 sin, second half d2 cos - d1 sin
  float c[8], sn[8];
  rope_coefs(cosT, sinT, t, sub, c, sn);
  const float sgn = sub < 8 ? 1.0f : -1.0f;
  float n[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) n[e] = d[e] * c[e] + sgn * __shfl_xor(d[e], 8) * sn[e];
  // RMSNorm backward over the head (gain frozen)
  const bool isq = hs < H;
  float x[8], w[8];
  unpack8(*reinterpret_cast<const uint4*>(raw + off), x);
  unpack8(*reinterpret_cast<const uint4*>((isq ? qn_w : kn_w) + 8 * sub), w);
  const float rstd = isq ? rq[(size_t)tok * H + hs] : rk[(size_t)tok * Hkv + (hs - H)];
  float dot = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    x[e] *= rstd;          // xhat
    n[e] *= w[e];          // g
    dot += n[e] * x[e];
  }
  const float m = group16_sum(dot) / QK_HD;
  float o[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = rstd * (n[e] - x[e] * m);
  *reinterpret_cast<uint4*>(draw + off) = pack8(o);
}


// m[r][c] = silu(gu[r][c]) * gu[r][F + c]; 4 columns per thread
__global__ void swiglu_fwd_kernel(const bf16_t* __restrict__ gu, bf16_t* __restrict__ m, long rows, int F) {
  const long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= rows * F) return;
  const long r = i / F;
  const int c = (int)(i % F);
  const uint2 g = *reinterpret_cast<const uint2*>(gu + (size_t)r * 2 * F + c);
  const uint2 u = *reinterpret_cast<const uint2*>(gu + (size_t)r * 2 * F + F + c);
  const float gv[4] = {lo_f(g.x), hi_f(g.x), lo_f(g.y), hi_f(g.y)};
  const float uv[4] = {lo_f(u.x), hi_f(u.x), lo_f(u.y), hi_f(u.y)};
  float o[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = swiglu1(gv[e], uv[e]);
  *reinterpret_cast<uint2*>(m + i) = make_uint2(pack2(o[0], o[1]), pack2(o[2], o[3]));
}

// dgu = [dm * u * silu'(g) | dm * silu(g)], silu'(g) = s (1 + g (1 - s))
__global__ void swiglu_bwd_kernel(const bf16_t* __restrict__ dm, const bf16_t* __restrict__ gu, bf16_t* __restrict__ dgu,
                                  long rows, int F) {
  const long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= rows * F) return;
  const long r = i / F;
  const int c = (int)(i % F);
  const uint2 d = *reinterpret_cast<const uint2*>(dm + i);
  const uint2 g = *reinterpret_cast<const uint2*>(gu + (size_t)r * 2 * F + c);
  const uint2 u = *reinterpret_cast<const uint2*>(gu + (size_t)r * 2 * F + F + c);
  const float dv[4] = {lo_f(d.x), hi_f(d.x), lo_f(d.y), hi_f(d.y)};
  const float gv[4] = {lo_f(g.x), hi_f(g.x), lo_f(g.y), hi_f(g.y)};
  const float uv[4] = {lo_f(u.x), hi_f(u.x), lo_f(u.y), hi_f(u.y)};
  float dg[4], du[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    swiglu1_bwd(dv[e], gv[e], uv[e], dg[e], du[e]);
  }
  *reinterpret_cast<uint2*>(dgu + (size_t)r * 2 * F + c) = make_uint2(pack2(dg[0], dg[1]), pack2(dg[2], dg[3]));
  *reinterpret_cast<uint2*>(dgu + (size_t)r * 2 * F + F + c) = make_uint2(pack2(du[0], du[1]), pack2(du[2], du[3]));
}

// x[r][c] *= s for rows x cols (row stride ld), bf16 in place
__global__ void scale_bf16_kernel(bf16_t* __restrict__ x, long rows, int cols, int ld, float s) {
  const long i = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= rows * cols) return;
  const long r = i / cols;
  const int c = (int)(i % cols);
  bf16_t* p = x + (size_t)r * ld + c;
  *p = f2bf(bf2f(*p) * s);
}

inline unsigned nblocks(long n, int nt) { return (unsigned)((n + nt - 1) / nt); }

}  // namespace

hipError_t launch_embed_gather(const int32_t* ids, const bf16_t* table, bf16_t* x, long rows, int C, hipStream_t s) {
  if (C % 8) return hipErrorInvalidValue;
  hipLaunchKernelGGL(embed_gather_kernel, dim3(nblocks(rows * C / 8, 256)), dim3(256), 0, s, ids, table, x, rows, C);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_fwd(const bf16_t* x, const bf16_t* w, bf16_t* y, float* rstd, int rows, int C, float eps,
                              int T, int mask_from, hipStream_t s) {
  if (C % 4 || T < 1 || mask_from < 0 || mask_from >= T) return hipErrorInvalidValue;
  const dim3 g((rows + 3) / 4), b(256);
  if (C <= 256) hipLaunchKernelGGL(rmsnorm_fwd_kernel<1>, g, b, 0, s, x, w, y, rstd, rows, C, eps, T, mask_from);
  else if (C <= 512) hipLaunchKernelGGL(rmsnorm_fwd_kernel<2>, g, b, 0, s, x, w, y, rstd, rows, C, eps, T, mask_from);
  else if (C <= 1024) hipLaunchKernelGGL(rmsnorm_fwd_kernel<4>, g, b, 0, s, x, w, y, rstd, rows, C, eps, T, mask_from);
  else if (C <= 2048) hipLaunchKernelGGL(rmsnorm_fwd_kernel<8>, g, b, 0, s, x, w, y, rstd, rows, C, eps, T, mask_from);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_rmsnorm_bwd(const bf16_t* dy, const bf16_t* x, const float* rstd, const bf16_t* w, bf16_t* dres,
                              int accumulate, int rows, int C, int T, int mask_from, hipStream_t s) {
  if (C % 4 || T < 1 || mask_from < 0 || mask_from >= T) return hipErrorInvalidValue;
  const dim3 g((rows + 3) / 4), b(256);
  if (C <= 256)
    hipLaunchKernelGGL(rmsnorm_bwd_kernel<1>, g, b, 0, s, dy, x, rstd, w, dres, accumulate, rows, C, T, mask_from);
  else if (C <= 512)
    hipLaunchKernelGGL(rmsnorm_bwd_kernel<2>, g, b, 0, s, dy, x, rstd, w, dres, accumulate, rows, C, T, mask_from);
  else if (C <= 1024)
    hipLaunchKernelGGL(rmsnorm_bwd_kernel<4>, g, b, 0, s, dy, x, rstd, w, dres, accumulate, rows, C, T, mask_from);
  else if (C <= 2048)
    hipLaunchKernelGGL(rmsnorm_bwd_kernel<8>, g, b, 0, s, dy, x, rstd, w, dres, accumulate, rows, C, T, mask_from);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_qknorm_rope_fwd(const bf16_t* raw, const bf16_t* qn_w, const bf16_t* kn_w, const float* cosT,
                                  const float* sinT, bf16_t* packed, float* rq, float* rk, int BT, int T, int H, int Hkv,
                                  int hd, float eps, hipStream_t s) {
  if (hd != QK_HD || Hkv < 1 || H % Hkv) return hipErrorInvalidValue;
  const long items = (long)BT * (H + 2 * Hkv);
  hipLaunchKernelGGL(qknorm_rope_fwd_kernel, dim3(nblocks(items, 16)), dim3(256), 0, s, raw, qn_w, kn_w, cosT, sinT,
                     packed, rq, rk, BT, T, H, Hkv, eps);
  return hipGetLastError();
}

hipError_t launch_qknorm_rope_bwd(const bf16_t* dpacked, const bf16_t* raw, const bf16_t* qn_w, const bf16_t* kn_w,
                                  const float* cosT, const float* sinT, const float* rq, const float* rk, bf16_t* draw,
                                  int BT, int T, int H, int Hkv, int hd, hipStream_t s) {
  if (hd != QK_HD || Hkv < 1 || H % Hkv) return hipErrorInvalidValue;
  const long items = (long)BT * (H + 2 * Hkv);
  hipLaunchKernelGGL(qknorm_rope_bwd_kernel, dim3(nblocks(items, 16)), dim3(256), 0, s, dpacked, raw, qn_w, kn_w, cosT,
                     sinT, rq, rk, draw, BT, T, H, Hkv);
  return hipGetLastError();
}

hipError_t launch_swiglu_fwd(const bf16_t* gu, bf16_t* m, long rows, int F, hipStream_t s) {
  if (F % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(swiglu_fwd_kernel, dim3(nblocks(rows * F / 4, 256)), dim3(256), 0, s, gu, m, rows, F);
  return hipGetLastError();
}

hipError_t launch_swiglu_bwd(const bf16_t* dm, const bf16_t* gu, bf16_t* dgu, long rows, int F, hipStream_t s) {
  if (F % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(swiglu_bwd_kernel, dim3(nblocks(rows * F / 4, 256)), dim3(256), 0, s, dm, gu, dgu, rows, F);
  return hipGetLastError();
}

hipError_t launch_scale_bf16(bf16_t* x, long rows, int cols, int ld, float sc, hipStream_t s) {
  hipLaunchKernelGGL(scale_bf16_kernel, dim3(nblocks(rows * cols, 256)), dim3(256), 0, s, x, rows, cols, ld, sc);
  return hipGetLastError();
}
