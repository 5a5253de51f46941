// Memory-bound kernels of the training step: embedding forward/backward, the
// fused softmax cross-entropy over the real vocabulary, column sums for bias
// gradients, slice reductions, the global gradient norm, and the fused AdamW
// update that also refreshes the bf16 weight copy.
#include "common.h"
#include "kernels.h"

namespace {

// ------------------------------------------------------------ reductions

__global__ void reduce_slices_kernel(const float* __restrict__ src, int nslices, long n, float* __restrict__ dst,
                                     int accumulate) {
  long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= n) return;
  float4 acc = accumulate ? *reinterpret_cast<const float4*>(dst + i) : make_float4(0, 0, 0, 0);
  // up to 16 slices' loads in flight before their sums
#pragma unroll 16
  for (int s = 0; s < nslices; ++s) {
    float4 v = *reinterpret_cast<const float4*>(src + (size_t)s * n + i);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  *reinterpret_cast<float4*>(dst + i) = acc;
}

// dst[i] (bf16) = scale * sum_s src[s*n + i], four elements per thread
__global__ void reduce_slices_bf16_kernel(const float* __restrict__ src, int nslices, long n, float scale,
                                          bf16_t* __restrict__ dst) {
  long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= n) return;
  float4 acc = make_float4(0, 0, 0, 0);
#pragma unroll 16
  for (int s = 0; s < nslices; ++s) {
    float4 v = *reinterpret_cast<const float4*>(src + (size_t)s * n + i);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  *reinterpret_cast<uint2*>(dst + i) =
      make_uint2(pack2(acc.x * scale, acc.y * scale), pack2(acc.z * scale, acc.w * scale));
}

// Two independent reductions in one launch; blockIdx.y picks the segment.
__global__ void reduce_slices2_kernel(const float* __restrict__ src, int nslices, long n, float* __restrict__ dst,
                                      const float* __restrict__ src2, int nslices2, long n2,
                                      float* __restrict__ dst2, int accumulate) {
  const bool second = blockIdx.y == 1;
  const float* sp = second ? src2 : src;
  const int ns = second ? nslices2 : nslices;
  const long nn = second ? n2 : n;
  float* dp = second ? dst2 : dst;
  long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= nn) return;
  float4 acc = accumulate ? *reinterpret_cast<const float4*>(dp + i) : make_float4(0, 0, 0, 0);
#pragma unroll 16
  for (int k = 0; k < ns; ++k) {
    float4 v = *reinterpret_cast<const float4*>(sp + (size_t)k * nn + i);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  *reinterpret_cast<float4*>(dp + i) = acc;
}

// 16 waves per block, 64 columns per block: wave w sums slices w, w+16, ...
// sixteen loads at a time, then the waves are combined in order.
DEV void reduce_parts_block(const float* __restrict__ part, int S, long stride, int n, int nd, float* __restrict__ d0,
                            float* __restrict__ d1, float* __restrict__ d2, int accumulate) {
  __shared__ float red[16][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = blockIdx.x * 64 + lane;
  const bool ok = col < n * nd;
  float a = 0.0f;
  if (ok) {
    // 16 loads in flight per wave (slices s, s+16, ..., s+240), then summed
    // in slice order
    int s = w;
    for (; s + 240 < S; s += 256) {
      float v[16];
#pragma unroll
      for (int k = 0; k < 16; ++k) v[k] = part[(size_t)(s + 16 * k) * stride + col];
#pragma unroll
      for (int k = 0; k < 16; ++k) a += v[k];
    }
    for (; s < S; s += 16) a += part[(size_t)s * stride + col];
  }
  red[w][lane] = a;
  __syncthreads();
  if (w == 0 && ok) {
    float t = 0.0f;
#pragma unroll
    for (int i = 0; i < 16; ++i) t += red[i][lane];
    const int j = col / n, c = col % n;
    float* d = j == 0 ? d0 : (j == 1 ? d1 : d2);
    if (d) d[c] = (accumulate ? d[c] : 0.0f) + t;
  }
}

__global__ __launch_bounds__(1024) void reduce_parts_kernel(const float* __restrict__ part, int S, long stride,
                                                            int n, int nd, float* __restrict__ d0,
                                                            float* __restrict__ d1, float* __restrict__ d2,
                                                            int accumulate) {
  reduce_parts_block(part, S, stride, n, nd, d0, d1, d2, accumulate);
}

// The same reduction for several partial-sum arrays of one shape at once:
// blockIdx.y picks the array and its destinations.
__global__ __launch_bounds__(1024) void reduce_parts_multi_kernel(ReducePartsJobs J, int S, long stride, int n, int nd,
                                                                  int accumulate) {
  const int j = blockIdx.y;
  reduce_parts_block(J.part[j], S, stride, n, nd, J.d[j][0], J.d[j][1], J.d[j][2], accumulate);
}

template <int NT>
DEV float block_sum(float v, float* sh) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) sh[w] = v;
  __syncthreads();
  float t = 0.0f;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) t += sh[i];
  return t;
}

template <int NT>
DEV float block_max(float v, float* sh) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) sh[w] = v;
  __syncthreads();
  float t = -INFINITY;
#pragma unroll
  for (int i = 0; i < NT / 64; ++i) t = fmaxf(t, sh[i]);
  return t;
}

// one block of 1024 threads, each with up to 16 loads in flight at a time
__global__ __launch_bounds__(1024) void mean_kernel(const float* __restrict__ x, int n, float inv,
                                                    float* __restrict__ out, uint32_t* __restrict__ flag) {
  __shared__ float sh[16];
  float s = 0.0f;
  int i = threadIdx.x;
  for (; i + 15 * 1024 < n; i += 16 * 1024) {
    float v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) v[k] = x[i + 1024 * k];
#pragma unroll
    for (int k = 0; k < 16; ++k) s += v[k];
  }
  for (; i < n; i += 1024) s += x[i];
  s = block_sum<1024>(s, sh);
  if (threadIdx.x == 0) {
    out[0] = s * inv;
    if (flag) {
      // the kernels that set the flag ran before this one on the stream
      reinterpret_cast<uint32_t*>(out)[1] = *flag;
      *flag = 0u;
    }
  }
}

// ------------------------------------------------------------ embedding

__global__ void embed_fwd_kernel(const int32_t* __restrict__ ids, const float* __restrict__ wte,
                                 const float* __restrict__ wpe, bf16_t* __restrict__ x, int BT, int T, int C, int V,
                                 uint32_t* __restrict__ bad) {
  long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= (long)BT * C) return;
  const int row = i / C, c = i % C, t = row % T;
  int id = ids[row];
  if ((unsigned)id >= (unsigned)V) {
    // contract violation: reported, and row 0 read in its place
    if (bad && c == 0) atomicOr(bad, ID_BAD_INPUT);
    id = 0;
  }
  float4 a = *reinterpret_cast<const float4*>(wte + (size_t)id * C + c);
  float4 p = *reinterpret_cast<const float4*>(wpe + (size_t)t * C + c);
  *reinterpret_cast<uint2*>(x + i) = make_uint2(pack2(a.x + p.x, a.y + p.y), pack2(a.z + p.z, a.w + p.w));
}

// token table: scatter-add of each position's gradient into its id's row.
// A workgroup takes EMB_P consecutive positions and one EMB_C-column slice of
// the row (two columns per lane: at C = 768, 16,384 positions make 384
// workgroups); it sorts the positions by (id, position) in LDS, and each wave
// walks 64 of the sorted positions, summing runs of equal ids in registers
// and adding each run once with fp32 atomics. Frequent ids (the token
// distribution is Zipf-like) then cost one atomic per workgroup instead of
// one per occurrence.
constexpr int EMB_P = 256, EMB_C = 128;
constexpr float LOG2E_F = 1.4426950408889634f;
__global__ __launch_bounds__(256) void embed_bwd_wte_kernel(const int32_t* __restrict__ ids,
                                                            const bf16_t* __restrict__ dx, float* __restrict__ dwte,
                                                            int BT, int C, int V) {
  __shared__ unsigned long long key[EMB_P];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int p0 = blockIdx.x * EMB_P;
  const int c = blockIdx.y * EMB_C + 2 * lane;
  {
    // positions past the end and ids outside [0, V) (a contract violation,
    // reported by the forward pass) take the key that sorts last and is skipped
    const int p = p0 + tid;
    const int id = p < BT ? ids[p] : -1;
    key[tid] = (unsigned)id < (unsigned)V ? ((unsigned long long)(uint32_t)id << 32) | (uint32_t)p : ~0ull;
  }
  __syncthreads();
  // bitonic sort of the EMB_P keys, one per thread
  for (int k = 2; k <= EMB_P; k <<= 1)
    for (int j = k >> 1; j > 0; j >>= 1) {
      const int x = tid ^ j;
      if (x > tid) {
        const unsigned long long a = key[tid], b = key[x];
        const bool up = (tid & k) == 0;
        if ((a > b) == up) {
          key[tid] = b;
          key[x] = a;
        }
      }
      __syncthreads();
    }
  const bool col_ok = c < C;
  float2 acc = make_float2(0.f, 0.f);
  constexpr int BATCH = 8;
  for (int k0 = 0; k0 < 64; k0 += BATCH) {
    unsigned long long kk[BATCH];
    uint32_t u[BATCH];
#pragma unroll
    for (int q = 0; q < BATCH; ++q) {
      kk[q] = key[64 * w + k0 + q];
      u[q] = 0;
      if (kk[q] != ~0ull && col_ok) {
        const uint32_t pos = (uint32_t)kk[q];
        u[q] = *reinterpret_cast<const uint32_t*>(dx + (size_t)pos * C + c);
      }
    }
#pragma unroll
    for (int q = 0; q < BATCH; ++q) {
      if (kk[q] == ~0ull) continue;
      acc.x += lo_f(u[q]); acc.y += hi_f(u[q]);
      const int kn = k0 + q + 1;
      const unsigned long long nxt = kn < 64 ? key[64 * w + kn] : ~0ull;
      const uint32_t id = (uint32_t)(kk[q] >> 32);
      if ((uint32_t)(nxt >> 32) != id || nxt == ~0ull) {
        if (col_ok) {
          float* d = dwte + (size_t)id * C + c;
          atomicAdd(d + 0, acc.x);
          atomicAdd(d + 1, acc.y);
        }
        acc = make_float2(0.f, 0.f);
      }
    }
  }
}

// position table: dwpe[t] = sum over the batch, in batch order; rows t >= T
// get no gradient
__global__ void embed_bwd_wpe_kernel(const bf16_t* __restrict__ dx, float* __restrict__ dwpe, int B, int T, int Tmax,
                                     int C, int accumulate) {
  long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= (long)Tmax * C) return;
  const int t = i / C;
  float4 acc = accumulate ? *reinterpret_cast<const float4*>(dwpe + i) : make_float4(0, 0, 0, 0);
  if (t < T) {
    for (int b = 0; b < B; ++b) {
      uint2 u = *reinterpret_cast<const uint2*>(dx + (size_t)b * T * C + i);
      acc.x += lo_f(u.x); acc.y += hi_f(u.x); acc.z += lo_f(u.y); acc.w += hi_f(u.y);
    }
  }
  *reinterpret_cast<float4*>(dwpe + i) = acc;
}

// ------------------------------------------------------------ cross-entropy

// One workgroup per row; the row (Vp bf16) is held in registers as 16-byte
// chunks, so it is read once and written once. Workgroups are small enough
// (a few hundred threads) that several rows are in flight per CU, so one
// row's loads overlap another's stores. Each thread first finds its own
// maximum and its sum of exponentials relative to it; the pairs are then
// combined across the workgroup in one pass: M = max m_i, S = sum s_i
// exp(m_i - M).
template <int NT, int MAXCH, bool GRAD>
__global__ __launch_bounds__(NT) void cross_entropy_kernel(bf16_t* __restrict__ logits,
                                                           const int32_t* __restrict__ targets,
                                                           float* __restrict__ losses, int V, int Vp,
                                                           float grad_scale, int T, int mask_from,
                                                           uint32_t* __restrict__ bad) {
  constexpr int NW = NT / 64;
  __shared__ float shm[NW], shs[NW];
  const int row = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  bf16_t* lr = logits + (size_t)row * Vp;
  // logits row `row` belongs to position pos: the rows are those of the
  // positions t >= mask_from of every sequence of T, in order
  const int nl = T - mask_from;
  const int pos = (row / nl) * T + mask_from + row % nl;
  if (mask_from > 0) {
    // the positions without loss (B * mask_from of them, listed sequence by
    // sequence) get a zero loss, spread over the workgroups
    const int nmask = (int)(gridDim.x / nl) * mask_from;
    for (int k = row + (int)gridDim.x * tid; k < nmask; k += (int)gridDim.x * NT)
      losses[(k / mask_from) * T + k % mask_from] = 0.0f;
  }
  int tgt = targets[pos];
  if ((unsigned)tgt >= (unsigned)V) {
    // contract violation: reported, and column 0 taken in its place
    if (bad && tid == 0) atomicOr(bad, ID_BAD_TARGET);
    tgt = 0;
  }
  // the target's logit, read before the row is overwritten (by every thread,
  // one broadcast address, so the load needs no branch; thread 0 uses it)
  const bf16_t xt_raw = lr[tgt];
  const int nch = Vp / 8;
  // Every thread issues all its row loads at once: chunks past the row end
  // read its last chunk (an in-range address) and are excluded below by the
  // column test (their columns would be >= Vp >= V), so no load waits behind
  // a per-chunk branch.
  uint4 v[MAXCH];
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const int c = min(tid + NT * i, nch - 1);
    v[i] = ld_stream(reinterpret_cast<const uint4*>(lr + c * 8));
  }
  // element j of chunk c counts if j < V (the padding columns carry no
  // probability)
  auto elem = [&](const uint4& q, int e) {
    const uint32_t wd = e < 2 ? q.x : e < 4 ? q.y : e < 6 ? q.z : q.w;
    return (e & 1) ? hi_f(wd) : lo_f(wd);
  };
  // Only the chunk that holds column V-1 mixes real and padding columns:
  // whole chunks below it skip the per-element test, those past it count
  // nothing.
  float m = -INFINITY;
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const int c = tid + NT * i;
    if (c * 8 + 8 <= V) {
#pragma unroll
      for (int e = 0; e < 8; ++e) m = fmaxf(m, elem(v[i], e));
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (c * 8 + e < V) m = fmaxf(m, elem(v[i], e));
    }
  }
  // the packed row is all that stays live between passes (otherwise the
  // compiler keeps every unpacked fp32 value in registers)
  auto opaque = [&]() {
#pragma unroll
    for (int i = 0; i < MAXCH; ++i) asm volatile("" : "+v"(v[i].x), "+v"(v[i].y), "+v"(v[i].z), "+v"(v[i].w));
  };
  opaque();
  // exp(x - m) = 2^(x log2(e) - m log2(e)): one fma and one exponential
  const float ml = m == -INFINITY ? 0.0f : m * LOG2E_F;
  float se = 0.0f;
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const int c = tid + NT * i;
    if (c * 8 + 8 <= V) {
#pragma unroll
      for (int e = 0; e < 8; ++e) se += __builtin_amdgcn_exp2f(fmaf(elem(v[i], e), LOG2E_F, -ml));
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (c * 8 + e < V) se += __builtin_amdgcn_exp2f(fmaf(elem(v[i], e), LOG2E_F, -ml));
    }
  }
  opaque();
  // combine (m, se) over the wave, then over the waves
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float m2 = __shfl_xor(m, o, WAVE), s2 = __shfl_xor(se, o, WAVE);
    const float mn = fmaxf(m, m2);
    se = (m == -INFINITY ? 0.0f : se * __expf(m - mn)) + (m2 == -INFINITY ? 0.0f : s2 * __expf(m2 - mn));
    m = mn;
  }
  if (lane == 0) {
    shm[w] = m;
    shs[w] = se;
  }
  __syncthreads();
  float mx = shm[0];
#pragma unroll
  for (int k = 1; k < NW; ++k) mx = fmaxf(mx, shm[k]);
  float sum = 0.0f;
#pragma unroll
  for (int k = 0; k < NW; ++k) sum += shm[k] == -INFINITY ? 0.0f : shs[k] * __expf(shm[k] - mx);
  // dlogits = (softmax - onehot(target)) * grad_scale: 2^(x log2(e) - mx
  // log2(e)) times grad_scale / sum, the target's column less grad_scale
  const float mxl = mx * LOG2E_F, k = grad_scale / sum;
#pragma unroll
  for (int i = 0; i < MAXCH; ++i) {
    const int c = tid + NT * i;
    if (GRAD && c < nch) {
      float d[8];
      if (c * 8 + 8 <= V) {
#pragma unroll
        for (int e = 0; e < 8; ++e) d[e] = __builtin_amdgcn_exp2f(fmaf(elem(v[i], e), LOG2E_F, -mxl)) * k;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          d[e] = c * 8 + e < V ? __builtin_amdgcn_exp2f(fmaf(elem(v[i], e), LOG2E_F, -mxl)) * k : 0.0f;
      }
      if (c == (tgt >> 3)) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (e == (tgt & 7)) d[e] -= grad_scale;
      }
      st_stream(reinterpret_cast<uint4*>(lr + c * 8),
                make_uint4(pack2(d[0], d[1]), pack2(d[2], d[3]), pack2(d[4], d[5]), pack2(d[6], d[7])));
    }
  }
  if (tid == 0) losses[pos] = mx + logf(sum) - bf2f(xt_raw);
}

// Combine the per-slice softmax statistics of each row (written by the head
// GEMM's statistics epilogue): one wave per row, each lane merging every 64th
// slice (max, sum of exponentials) pair, then the lanes merged in a fixed
// butterfly order.
DEV void merge_ms(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  s = (m == -INFINITY ? 0.0f : s * __expf(m - mn)) + (m2 == -INFINITY ? 0.0f : s2 * __expf(m2 - mn));
  m = mn;
}

__global__ __launch_bounds__(256) void ce_combine_kernel(const float2* __restrict__ stats, int nparts,
                                                         const float* __restrict__ tlogit,
                                                         const int32_t* __restrict__ targets, int V,
                                                         float* __restrict__ lse, float* __restrict__ losses, int rows,
                                                         uint32_t* __restrict__ bad) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= rows) return;
  float m = -INFINITY, sum = 0.0f;
  for (int k = lane; k < nparts; k += 64) {
    const float2 p = stats[(size_t)row * nparts + k];
    merge_ms(m, sum, p.x, p.y);
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    const float m2 = __shfl_xor(m, o, WAVE), s2 = __shfl_xor(sum, o, WAVE);
    merge_ms(m, sum, m2, s2);
  }
  if (lane == 0) {
    const float l = m + logf(sum);
    lse[row] = l;
    losses[row] = l - tlogit[row];
    if ((unsigned)targets[row] >= (unsigned)V && bad) atomicOr(bad, ID_BAD_TARGET);
  }
}

// ------------------------------------------------------------ casts

__global__ void cast_bf16_kernel(const float* __restrict__ src, bf16_t* __restrict__ dst, long n) {
  long i = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= n) return;
  float4 v = *reinterpret_cast<const float4*>(src + i);
  *reinterpret_cast<uint2*>(dst + i) = make_uint2(pack2(v.x, v.y), pack2(v.z, v.w));
}

// ------------------------------------------------------------ optimizer

constexpr int SUMSQ_BLOCKS = 1024;

__global__ __launch_bounds__(256) void sumsq_kernel(const float* __restrict__ g, long n, float* __restrict__ parts) {
  __shared__ float sh[4];
  float s = 0.0f;
  for (long i = ((long)blockIdx.x * 256 + threadIdx.x) * 4; i < n; i += (long)gridDim.x * 256 * 4) {
    float4 v = *reinterpret_cast<const float4*>(g + i);
    s += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  s = block_sum<256>(s, sh);
  if (threadIdx.x == 0) parts[blockIdx.x] = s;
}

__global__ __launch_bounds__(256) void clip_coef_kernel(const float* __restrict__ parts, int nparts, float clip,
                                                        float* __restrict__ norm_coef) {
  __shared__ float sh[4];
  float s = 0.0f;
  for (int i = threadIdx.x; i < nparts; i += 256) s += parts[i];
  s = block_sum<256>(s, sh);
  if (threadIdx.x == 0) {
    float norm = sqrtf(s);
    norm_coef[0] = norm;
    norm_coef[1] = norm > clip ? clip / norm : 1.0f;
  }
}

// Segments (parameter kinds) are walked in order, uniformly across the grid,
// so each one's bounds and decay flag are scalars; within a segment every
// thread updates 4-element chunks in a grid-stride loop, two chunks in
// flight at a time. Segment ends are multiples of 4 (checked at launch).
__global__ __launch_bounds__(256) void adamw_kernel(AdamArgs a) {
  const float coef = a.norm_coef[1];
  const long stride = (long)gridDim.x * 256 * 4;
  // Every rounding of the update is written out (no implicit contraction):
  // the compiler could otherwise fuse the multiply-adds differently in the
  // inlined copies below, and an element's bits would depend on which copy,
  // grid size or segment split handles it.
  auto update = [&](long i, float wd) {
#pragma clang fp contract(off)
    float4 p = ld_stream(reinterpret_cast<const float4*>(a.p + i));
    float4 g = ld_stream(reinterpret_cast<const float4*>(a.g + i));
    float4 m = ld_stream(reinterpret_cast<const float4*>(a.m + i));
    float4 v = ld_stream(reinterpret_cast<const float4*>(a.v + i));
    float pv[4] = {p.x, p.y, p.z, p.w}, gv[4] = {g.x, g.y, g.z, g.w};
    float mv[4] = {m.x, m.y, m.z, m.w}, vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float gg = gv[e] * coef;
      mv[e] = fmaf(a.beta1, mv[e], (1.0f - a.beta1) * gg);
      vv[e] = fmaf(a.beta2, vv[e], ((1.0f - a.beta2) * gg) * gg);
      const float mhat = mv[e] / a.bc1, vhat = vv[e] / a.bc2;
      const float upd = fmaf(wd, pv[e], mhat / (sqrtf(vhat) + a.eps));
      pv[e] = fmaf(-a.lr, upd, pv[e]);
    }
    st_stream(reinterpret_cast<float4*>(a.p + i), make_float4(pv[0], pv[1], pv[2], pv[3]));
    st_stream(reinterpret_cast<float4*>(a.m + i), make_float4(mv[0], mv[1], mv[2], mv[3]));
    st_stream(reinterpret_cast<float4*>(a.v + i), make_float4(vv[0], vv[1], vv[2], vv[3]));
    *reinterpret_cast<uint2*>(a.p_bf16 + i) = make_uint2(pack2(pv[0], pv[1]), pack2(pv[2], pv[3]));
  };
  long lo = 0;
  for (int sg = 0; sg < a.seg.count; ++sg) {
    const long hi = a.seg.end[sg];
    const float wd = a.seg.decay[sg] ? a.weight_decay : 0.0f;
    long i = lo + ((long)blockIdx.x * 256 + threadIdx.x) * 4;
    for (; i + stride < hi; i += 2 * stride) {
      update(i, wd);
      update(i + stride, wd);
    }
    if (i < hi) update(i, wd);
    lo = hi;
  }
}

// ------------------------------------------------------------ seeded init

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011): ten rounds of two
// 32x32->64-bit products whose high halves are XORed with the other counter
// words and the key; the key is bumped by the Weyl constants between rounds.
DEV uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
  constexpr uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u, W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += W0;
      k1 += W1;
    }
    const uint32_t hi0 = __umulhi(M0, c.x), lo0 = M0 * c.x;
    const uint32_t hi1 = __umulhi(M1, c.z), lo1 = M1 * c.z;
    c = make_uint4(hi1 ^ c.y ^ k0, lo1, hi0 ^ c.w ^ k1, lo0);
  }
  return c;
}

// standard normal of flat element i: Box-Muller of the first two words, fp64
DEV double normal_at(long i, uint32_t k0, uint32_t k1) {
  const uint4 x = philox4x32_10(make_uint4((uint32_t)i, (uint32_t)((unsigned long)i >> 32), 0u, 0u), k0, k1);
  const double u1 = ((double)x.x + 0.5) * 0x1p-32, u2 = ((double)x.y + 0.5) * 0x1p-32;
  return sqrt(-2.0 * log(u1)) * cos(2.0 * M_PI * u2);
}

// 4 elements per thread, grid-stride; the segment of a 4-element chunk is
// found by a walk over the (at most 16) segment ends, which are multiples of 4
__global__ __launch_bounds__(256) void init_params_kernel(InitArgs a) {
  const long stride = (long)gridDim.x * 256 * 4;
  for (long i = ((long)blockIdx.x * 256 + threadIdx.x) * 4; i < a.n; i += stride) {
    int k = 0;
    while (k + 1 < a.count && i >= a.end[k]) ++k;
    float v[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const long j = i + e;
      if (j >= a.zero_lo && j < a.zero_hi) v[e] = 0.0f;
      else if (a.std[k] > 0.0) v[e] = (float)(normal_at(j, a.key0, a.key1) * a.std[k]);
      else v[e] = a.fill[k];
    }
    *reinterpret_cast<float4*>(a.p + i) = make_float4(v[0], v[1], v[2], v[3]);
    *reinterpret_cast<float4*>(a.m + i) = make_float4(0.f, 0.f, 0.f, 0.f);
    *reinterpret_cast<float4*>(a.v + i) = make_float4(0.f, 0.f, 0.f, 0.f);
    *reinterpret_cast<uint2*>(a.p_bf16 + i) = make_uint2(pack2(v[0], v[1]), pack2(v[2], v[3]));
  }
}

inline unsigned blocks_for(long n4, int nt) { return (unsigned)((n4 + nt - 1) / nt); }

}  // namespace

hipError_t launch_reduce_slices(const float* src, int nslices, long n, float* dst, int accumulate, hipStream_t s) {
  if (n % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(reduce_slices_kernel, dim3(blocks_for(n / 4, 256)), dim3(256), 0, s, src, nslices, n, dst,
                     accumulate);
  return hipGetLastError();
}

hipError_t launch_reduce_slices_bf16(const float* src, int nslices, long n, float scale, bf16_t* dst,
                                     hipStream_t s) {
  if (n % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(reduce_slices_bf16_kernel, dim3(blocks_for(n / 4, 256)), dim3(256), 0, s, src, nslices, n, scale,
                     dst);
  return hipGetLastError();
}

hipError_t launch_reduce_slices2(const float* src, int nslices, long n, float* dst, const float* src2,
                                 int nslices2, long n2, float* dst2, int accumulate, hipStream_t s) {
  if (n % 4 || n2 % 4) return hipErrorInvalidValue;
  const long nmax = n > n2 ? n : n2;
  hipLaunchKernelGGL(reduce_slices2_kernel, dim3(blocks_for(nmax / 4, 256), 2), dim3(256), 0, s, src, nslices, n, dst,
                     src2, nslices2, n2, dst2, accumulate);
  return hipGetLastError();
}

hipError_t launch_reduce_parts_multi(const ReducePartsJobs& J, int S, long stride, int n, int nd, int accumulate,
                                     hipStream_t s) {
  if (nd < 1 || nd > 3 || J.count < 1 || J.count > REDUCE_JOBS) return hipErrorInvalidValue;
  hipLaunchKernelGGL(reduce_parts_multi_kernel, dim3((unsigned)((n * nd + 63) / 64), (unsigned)J.count), dim3(1024), 0,
                     s, J, S, stride, n, nd, accumulate);
  return hipGetLastError();
}

hipError_t launch_reduce_parts(const float* part, int S, long stride, int n, int nd, float* d0, float* d1,
                               float* d2, int accumulate, hipStream_t s) {
  if (nd < 1 || nd > 3) return hipErrorInvalidValue;
  hipLaunchKernelGGL(reduce_parts_kernel, dim3((unsigned)((n * nd + 63) / 64)), dim3(1024), 0, s, part, S, stride, n,
                     nd, d0, d1, d2, accumulate);
  return hipGetLastError();
}

hipError_t launch_mean(const float* x, int n, float* out, hipStream_t s, uint32_t* flag) {
  hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(1024), 0, s, x, n, 1.0f / (float)n, out, flag);
  return hipGetLastError();
}

hipError_t launch_sum_scaled(const float* x, int n, float scale, float* out, hipStream_t s) {
  hipLaunchKernelGGL(mean_kernel, dim3(1), dim3(1024), 0, s, x, n, scale, out, nullptr);
  return hipGetLastError();
}

hipError_t launch_embed_fwd(const int32_t* ids, const float* wte, const float* wpe, bf16_t* x, int B, int T, int C,
                            int V, uint32_t* bad, hipStream_t s) {
  if (C % 4) return hipErrorInvalidValue;
  long n4 = (long)B * T * C / 4;
  hipLaunchKernelGGL(embed_fwd_kernel, dim3(blocks_for(n4, 256)), dim3(256), 0, s, ids, wte, wpe, x, B * T, T, C, V,
                     bad);
  return hipGetLastError();
}

hipError_t launch_embed_bwd(const int32_t* ids, const bf16_t* dx, float* dwte, int B, int T, int C, int V,
                            hipStream_t s) {
  if (C % 4) return hipErrorInvalidValue;
  const int BT = B * T;
  dim3 grid((BT + EMB_P - 1) / EMB_P, (C + EMB_C - 1) / EMB_C);
  hipLaunchKernelGGL(embed_bwd_wte_kernel, grid, dim3(256), 0, s, ids, dx, dwte, BT, C, V);
  return hipGetLastError();
}

hipError_t launch_embed_bwd_pos(const bf16_t* dx, float* dwpe, int B, int T, int Tmax, int C, int accumulate,
                                hipStream_t s) {
  long n4 = (long)Tmax * C / 4;
  hipLaunchKernelGGL(embed_bwd_wpe_kernel, dim3(blocks_for(n4, 256)), dim3(256), 0, s, dx, dwpe, B, T, Tmax, C,
                     accumulate);
  return hipGetLastError();
}

template <int NT, int MAXCH>
void ce_launch(bf16_t* logits, const int32_t* targets, float* losses, int rows, int V, int Vp, float grad_scale,
               int write_grad, int T, int mask_from, uint32_t* bad, hipStream_t s) {
  if (write_grad)
    hipLaunchKernelGGL((cross_entropy_kernel<NT, MAXCH, true>), dim3(rows), dim3(NT), 0, s, logits, targets, losses, V,
                       Vp, grad_scale, T, mask_from, bad);
  else
    hipLaunchKernelGGL((cross_entropy_kernel<NT, MAXCH, false>), dim3(rows), dim3(NT), 0, s, logits, targets, losses,
                       V, Vp, grad_scale, T, mask_from, bad);
}

hipError_t launch_cross_entropy_masked(bf16_t* logits, const int32_t* targets, float* losses, int rows, int V, int Vp,
                                       float grad_scale, int write_grad, int T, int mask_from, hipStream_t s,
                                       uint32_t* bad) {
  if (Vp % 8 || V < 1 || T < 1 || mask_from < 0 || mask_from >= T || rows % (T - mask_from))
    return hipErrorInvalidValue;
  const int nch = Vp / 8;
  if (nch <= 256 * 2)
    ce_launch<256, 2>(logits, targets, losses, rows, V, Vp, grad_scale, write_grad, T, mask_from, bad, s);
  else if (nch <= 512 * 13)
    ce_launch<512, 13>(logits, targets, losses, rows, V, Vp, grad_scale, write_grad, T, mask_from, bad, s);
  else if (nch <= 1024 * 8)
    ce_launch<1024, 8>(logits, targets, losses, rows, V, Vp, grad_scale, write_grad, T, mask_from, bad, s);
  else if (nch <= 1024 * 19)
    ce_launch<1024, 19>(logits, targets, losses, rows, V, Vp, grad_scale, write_grad, T, mask_from, bad, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_cross_entropy(bf16_t* logits, const int32_t* targets, float* losses, int rows, int V, int Vp,
                                float grad_scale, int write_grad, uint32_t* bad, hipStream_t s) {
  return launch_cross_entropy_masked(logits, targets, losses, rows, V, Vp, grad_scale, write_grad, 1, 0, s, bad);
}

hipError_t launch_cast_bf16(const float* src, bf16_t* dst, long n, hipStream_t s) {
  if (n % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(cast_bf16_kernel, dim3(blocks_for(n / 4, 256)), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

int sumsq_parts() { return SUMSQ_BLOCKS; }

hipError_t launch_sumsq(const float* g, long n, float* parts, hipStream_t s) {
  if (n % 4) return hipErrorInvalidValue;
  hipLaunchKernelGGL(sumsq_kernel, dim3(SUMSQ_BLOCKS), dim3(256), 0, s, g, n, parts);
  return hipGetLastError();
}

hipError_t launch_clip_coef(const float* parts, int nparts, float clip, float* norm_coef, hipStream_t s) {
  hipLaunchKernelGGL(clip_coef_kernel, dim3(1), dim3(256), 0, s, parts, nparts, clip, norm_coef);
  return hipGetLastError();
}

hipError_t launch_adamw(const AdamArgs& a, hipStream_t s) {
  if (a.n % 4) return hipErrorInvalidValue;
  for (int k = 0; k < a.seg.count; ++k)
    if (a.seg.end[k] % 4) return hipErrorInvalidValue;
  long n4 = a.n / 4;
  unsigned blocks = blocks_for(n4, 256);
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(adamw_kernel, dim3(blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_init_params(const InitArgs& a, hipStream_t s) {
  if (a.n % 4 || a.count < 1 || a.count > 16 || a.end[a.count - 1] != a.n) return hipErrorInvalidValue;
  for (int k = 0; k < a.count; ++k)
    if (a.end[k] % 4) return hipErrorInvalidValue;
  unsigned blocks = blocks_for(a.n / 4, 256);
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(init_params_kernel, dim3(blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_ce_combine(const float* stats, int nparts, const float* tlogit, const int32_t* targets, int V,
                             float* lse, float* losses, int rows, uint32_t* bad, hipStream_t s) {
  if (nparts < 1 || rows < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(ce_combine_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s,
                     reinterpret_cast<const float2*>(stats), nparts, tlogit, targets, V, lse, losses, rows, bad);
  return hipGetLastError();
}
