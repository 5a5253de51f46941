// LayerNorm forward and backward over rows of C channels (pre-LN blocks and
// the final norm, Figure 1). Statistics in fp32, biased variance, eps from the
// config. One wavefront per row; each lane owns channels {4*(lane + 64*i)..+3},
// read as 8-byte bf16 chunks.
#include "common.h"
#include "kernels.h"

namespace {

// Sum of two bf16 rows in fp32, rounded to bf16 (to nearest even): the
// residual connection's addition
DEV uint2 add_rows(uint2 r, uint2 a) {
  return make_uint2(pack2(lo_f(r.x) + lo_f(a.x), hi_f(r.x) + hi_f(a.x)),
                    pack2(lo_f(r.y) + lo_f(a.y), hi_f(r.y) + hi_f(a.y)));
}

// MAXCH: 4-channel chunks per lane, C <= 256*MAXCH. With RES the row is first
// formed as the residual sum x = bf16(res + x) (stored to xsum), and the
// normalisation then reads those rounded values, exactly as a separate
// addition followed by this kernel would.
template <int MAXCH, bool RES = false>
__global__ __launch_bounds__(256) void ln_fwd_kernel(const bf16_t* __restrict__ x, const bf16_t* __restrict__ res,
                                                     bf16_t* __restrict__ xsum, const float* __restrict__ w,
                                                     const float* __restrict__ b, bf16_t* __restrict__ y,
                                                     float* __restrict__ mean_out, float* __restrict__ rstd_out,
                                                     int rows, int C, float eps) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const bf16_t* xr = x + (size_t)row * C;
  // Every lane issues all its loads at once: chunks past C read the row's
  // last chunk (an in-range address) and are masked out of the arithmetic,
  // so no load waits behind a branch.
  uint2 xu[MAXCH], ru[MAXCH];
  float4 wv[MAXCH], bv[MAXCH];
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const int c = min(4 * (lane + 64 * i), C - 4);
    xu[i] = *reinterpret_cast<const uint2*>(xr + c);
    if constexpr (RES) ru[i] = *reinterpret_cast<const uint2*>(res + (size_t)row * C + c);
    wv[i] = *reinterpret_cast<const float4*>(w + c);
    bv[i] = *reinterpret_cast<const float4*>(b + c);
  }
  if constexpr (RES) {
#pragma unroll
    for (int i = 0; i < MAXCH; ++i) {
      xu[i] = add_rows(ru[i], xu[i]);
      const int c = 4 * (lane + 64 * i);
      if (c < C) *reinterpret_cast<uint2*>(xsum + (size_t)row * C + c) = xu[i];
    }
  }
  float v[MAXCH][4];
  float s = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const bool in = 4 * (lane + 64 * i) < C;
    v[i][0] = in ? lo_f(xu[i].x) : 0.0f;
    v[i][1] = in ? hi_f(xu[i].x) : 0.0f;
    v[i][2] = in ? lo_f(xu[i].y) : 0.0f;
    v[i][3] = in ? hi_f(xu[i].y) : 0.0f;
    s += v[i][0] + v[i][1] + v[i][2] + v[i][3];
  }
  const float mean = wave_sum(s) / C;
  float q = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    if (4 * (lane + 64 * i) < C)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        float d = v[i][e] - mean;
        q += d * d;
      }
  }
  const float rstd = 1.0f / sqrtf(wave_sum(q) / C + eps);
  bf16_t* yr = y + (size_t)row * C;
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    int c = 4 * (lane + 64 * i);
    if (c < C) {
      float o0 = (v[i][0] - mean) * rstd * wv[i].x + bv[i].x;
      float o1 = (v[i][1] - mean) * rstd * wv[i].y + bv[i].y;
      float o2 = (v[i][2] - mean) * rstd * wv[i].z + bv[i].z;
      float o3 = (v[i][3] - mean) * rstd * wv[i].w + bv[i].w;
      *reinterpret_cast<uint2*>(yr + c) = make_uint2(pack2(o0, o1), pack2(o2, o3));
    }
  }
  if (lane == 0) {
    mean_out[row] = mean;
    rstd_out[row] = rstd;
  }
}

// dx = rstd * (g - mean(g) - xhat * mean(g * xhat)), g = dy * w; the result is
// added to the residual-stream gradient read from dres_in and written to
// dres_out (the two may be the same buffer: each row is read before it is
// written, by the same wave). Per-block sums of dy*xhat and dy.
template <int MAXCH>
__global__ __launch_bounds__(256) void ln_bwd_kernel(const bf16_t* __restrict__ dy, const bf16_t* __restrict__ x,
                                                     const float* __restrict__ mean_in,
                                                     const float* __restrict__ rstd_in, const float* __restrict__ w,
                                                     const bf16_t* dres_in, bf16_t* dres_out, int has_res,
                                                     float* __restrict__ part, int rows, int C) {
  __shared__ float red[4][MAXCH * 4 * 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float aw[MAXCH][4], ab[MAXCH][4], ar[MAXCH][4], wr[MAXCH][4];
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    // chunks past C read an in-range address; their values are never used
    const int c = min(4 * (lane + 64 * i), C - 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) aw[i][e] = ab[i][e] = ar[i][e] = 0.0f;
    const float4 wv = *reinterpret_cast<const float4*>(w + c);
    wr[i][0] = wv.x; wr[i][1] = wv.y; wr[i][2] = wv.z; wr[i][3] = wv.w;
  }
  // Rows are software-pipelined: the next row's inputs (x, dy, the residual
  // gradient, mean, rstd) are loaded while the current row is reduced and
  // written, so each row costs one memory round trip, not two.
  uint2 xu[MAXCH], du[MAXCH], ru[MAXCH];
  float mean = 0.0f, rstd = 0.0f;
  auto load_row = [&](int row, uint2 (&xl)[MAXCH], uint2 (&dl)[MAXCH], uint2 (&rl)[MAXCH], float& ml, float& sl) {
    ml = mean_in[row];
    sl = rstd_in[row];
    const bf16_t* xr = x + (size_t)row * C;
    const bf16_t* dr = dy + (size_t)row * C;
    const bf16_t* rr = dres_in + (size_t)row * C;
    // all loads issued at once (no branch per chunk): chunks past C read the
    // row's last chunk and are never used
#pragma unroll
    for (int i = 0; i < MAXCH; ++i) {
      const int c = min(4 * (lane + 64 * i), C - 4);
      xl[i] = *reinterpret_cast<const uint2*>(xr + c);
      dl[i] = *reinterpret_cast<const uint2*>(dr + c);
      rl[i] = has_res ? *reinterpret_cast<const uint2*>(rr + c) : make_uint2(0, 0);
    }
  };
  const int stride = gridDim.x * 4;
  int row = blockIdx.x * 4 + wave;
  if (row < rows) load_row(row, xu, du, ru, mean, rstd);
  for (; row < rows; row += stride) {
    uint2 xn[MAXCH], dn[MAXCH], rn[MAXCH];
    float mean_n = 0.0f, rstd_n = 0.0f;
    if (row + stride < rows) load_row(row + stride, xn, dn, rn, mean_n, rstd_n);
    float xh[MAXCH][4], gg[MAXCH][4];
    float s1 = 0.0f, s2 = 0.0f;
#pragma unroll
    for (int i = 0; i < MAXCH; ++i) {
      int c = 4 * (lane + 64 * i);
      if (c < C) {
        float xv[4] = {lo_f(xu[i].x), hi_f(xu[i].x), lo_f(xu[i].y), hi_f(xu[i].y)};
        float dv[4] = {lo_f(du[i].x), hi_f(du[i].x), lo_f(du[i].y), hi_f(du[i].y)};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          xh[i][e] = (xv[e] - mean) * rstd;
          gg[i][e] = dv[e] * wr[i][e];
          s1 += gg[i][e];
          s2 += gg[i][e] * xh[i][e];
          aw[i][e] += dv[e] * xh[i][e];
          ab[i][e] += dv[e];
        }
      }
    }
    const float gm = wave_sum(s1) / C, gxm = wave_sum(s2) / C;
    bf16_t* rr = dres_out + (size_t)row * C;
#pragma unroll
    for (int i = 0; i < MAXCH; ++i) {
      int c = 4 * (lane + 64 * i);
      if (c < C) {
        float o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = rstd * (gg[i][e] - gm - xh[i][e] * gxm);
        if (has_res) {
          o[0] += lo_f(ru[i].x); o[1] += hi_f(ru[i].x); o[2] += lo_f(ru[i].y); o[3] += hi_f(ru[i].y);
        }
        const uint2 ou = make_uint2(pack2(o[0], o[1]), pack2(o[2], o[3]));
        *reinterpret_cast<uint2*>(rr + c) = ou;
        // the stored (rounded) values, so the sum matches what consumers read
        ar[i][0] += lo_f(ou.x); ar[i][1] += hi_f(ou.x); ar[i][2] += lo_f(ou.y); ar[i][3] += hi_f(ou.y);
      }
    }
#pragma unroll
    for (int i = 0; i < MAXCH; ++i) {
      xu[i] = xn[i];
      du[i] = dn[i];
      ru[i] = rn[i];
    }
    mean = mean_n;
    rstd = rstd_n;
  }
  // combine the four waves' partial sums in a fixed order; the block's row of
  // partials is [dw | db | column sum of the residual gradient], 3*C floats
  for (int pass = 0; pass < 3; ++pass) {
#pragma unroll
    for (int i = 0; i < MAXCH; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        red[wave][(i * 64 + lane) * 4 + e] = pass == 0 ? aw[i][e] : (pass == 1 ? ab[i][e] : ar[i][e]);
    __syncthreads();
    float* dst = part + (size_t)blockIdx.x * 3 * C + pass * C;
    for (int c = threadIdx.x; c < C; c += 256) {
      // channel c lives at chunk i = (c/4)/64, lane (c/4)%64, element c%4
      int cq = c >> 2, i = cq >> 6, l = cq & 63, e = c & 3;
      int k = (i * 64 + l) * 4 + e;
      dst[c] = red[0][k] + red[1][k] + red[2][k] + red[3][k];
    }
    __syncthreads();
  }
}

// the residual addition alone: out = bf16(res + x), 4 elements per thread
__global__ void residual_add_kernel(const bf16_t* __restrict__ res, const bf16_t* __restrict__ x,
                                    bf16_t* __restrict__ out, long n) {
  const long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= n) return;
  *reinterpret_cast<uint2*>(out + i) =
      add_rows(*reinterpret_cast<const uint2*>(res + i), *reinterpret_cast<const uint2*>(x + i));
}

template <int MAXCH>
hipError_t fwd_t(const bf16_t* x, const bf16_t* res, bf16_t* xsum, const float* w, const float* b, bf16_t* y,
                 float* mean, float* rstd, int rows, int C, float eps, hipStream_t s) {
  if (res)
    hipLaunchKernelGGL((ln_fwd_kernel<MAXCH, true>), dim3((rows + 3) / 4), dim3(256), 0, s, x, res, xsum, w, b, y,
                       mean, rstd, rows, C, eps);
  else
    hipLaunchKernelGGL((ln_fwd_kernel<MAXCH, false>), dim3((rows + 3) / 4), dim3(256), 0, s, x, nullptr, nullptr, w,
                       b, y, mean, rstd, rows, C, eps);
  return hipGetLastError();
}

template <int MAXCH>
hipError_t bwd_t(const bf16_t* dy, const bf16_t* x, const float* mean, const float* rstd, const float* w,
                 const bf16_t* dres_in, bf16_t* dres_out, int has_res, float* part, int rows, int C, hipStream_t s) {
  hipLaunchKernelGGL(ln_bwd_kernel<MAXCH>, dim3(layernorm_bwd_blocks(rows)), dim3(256), 0, s, dy, x, mean, rstd, w,
                     dres_in, dres_out, has_res, part, rows, C);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_add_layernorm_fwd(const bf16_t* x, const bf16_t* res, bf16_t* xsum, const float* w, const float* b,
                                    bf16_t* y, float* mean, float* rstd, int rows, int C, float eps, hipStream_t s) {
  if (C % 4 || (res && !xsum)) return hipErrorInvalidValue;
  if (C <= 256) return fwd_t<1>(x, res, xsum, w, b, y, mean, rstd, rows, C, eps, s);
  if (C <= 512) return fwd_t<2>(x, res, xsum, w, b, y, mean, rstd, rows, C, eps, s);
  if (C <= 768) return fwd_t<3>(x, res, xsum, w, b, y, mean, rstd, rows, C, eps, s);
  if (C <= 1024) return fwd_t<4>(x, res, xsum, w, b, y, mean, rstd, rows, C, eps, s);
  if (C <= 2048) return fwd_t<8>(x, res, xsum, w, b, y, mean, rstd, rows, C, eps, s);
  return hipErrorInvalidValue;
}

hipError_t launch_layernorm_fwd(const bf16_t* x, const float* w, const float* b, bf16_t* y, float* mean,
                                float* rstd, int rows, int C, float eps, hipStream_t s) {
  return launch_add_layernorm_fwd(x, nullptr, nullptr, w, b, y, mean, rstd, rows, C, eps, s);
}

hipError_t launch_residual_add(const bf16_t* res, const bf16_t* x, bf16_t* out, long n, hipStream_t s) {
  if (n % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(residual_add_kernel, dim3((unsigned)((n / 4 + 255) / 256)), dim3(256), 0, s, res, x, out, n);
  return hipGetLastError();
}

// At least 4 rows per wave, 4 waves per block, each block writing one row of
// partial sums; at most 768 blocks, three per CU, which is what the
// backward's registers (two rows' inputs in flight per wave) let stay
// resident at once
int layernorm_bwd_blocks(int rows) {
  int n = (rows + 15) / 16;
  return n < 768 ? (n < 1 ? 1 : n) : 768;
}

hipError_t launch_layernorm_bwd(const bf16_t* dy, const bf16_t* x, const float* mean, const float* rstd,
                                const float* w, const bf16_t* dres_in, bf16_t* dres_out, int has_res, float* part,
                                int rows, int C, hipStream_t s) {
  if (C % 4) return hipErrorInvalidValue;
  if (C <= 256) return bwd_t<1>(dy, x, mean, rstd, w, dres_in, dres_out, has_res, part, rows, C, s);
  if (C <= 512) return bwd_t<2>(dy, x, mean, rstd, w, dres_in, dres_out, has_res, part, rows, C, s);
  if (C <= 768) return bwd_t<3>(dy, x, mean, rstd, w, dres_in, dres_out, has_res, part, rows, C, s);
  if (C <= 1024) return bwd_t<4>(dy, x, mean, rstd, w, dres_in, dres_out, has_res, part, rows, C, s);
  if (C <= 2048) return bwd_t<8>(dy, x, mean, rstd, w, dres_in, dres_out, has_res, part, rows, C, s);
  return hipErrorInvalidValue;
}
