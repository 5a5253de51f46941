// Device-side helpers shared by the gfx950 kernels: bf16 storage, vector
// types, MFMA operand types and wavefront reductions.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;   // bf16 in memory: raw bits

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

#define DEV __device__ __forceinline__

constexpr int WAVE = 64;

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float floatx2 __attribute__((ext_vector_type(2)));

// fp32 -> bf16, round to nearest even (NaN stays NaN): gfx950 converts in
// hardware (v_cvt_pk_bf16_f32, one instruction for a pair).
DEV bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }
DEV float bf2f(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// two bf16 packed in a 32-bit word (low half = first element)
DEV uint32_t pack2(float a, float b) {
  floatx2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}
DEV float lo_f(uint32_t w) { return __uint_as_float(w << 16); }
DEV float hi_f(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

DEV bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Streaming (non-temporal) 16-byte loads and stores, for data that a kernel
// touches once and nothing reads again soon (gigabytes that would only churn
// the L2 and the 256 MB Infinity Cache): the optimizer's parameters, moments
// and gradients, the logits that the cross-entropy overwrites with dlogits.
// (The sum of squares over the gradients reads them with ordinary loads: part
// of them is still cached from the weight-gradient launch that wrote them.)
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
DEV uint4 ld_stream(const uint4* p) {
  const u32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  return make_uint4(t.x, t.y, t.z, t.w);
}
DEV float4 ld_stream(const float4* p) {
  const f32x4_t t = __builtin_nontemporal_load(reinterpret_cast<const f32x4_t*>(p));
  return make_float4(t.x, t.y, t.z, t.w);
}
DEV void st_stream(uint4* p, uint4 v) {
  const u32x4_t t = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(t, reinterpret_cast<u32x4_t*>(p));
}
DEV void st_stream(float4* p, float4 v) {
  const f32x4_t t = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(t, reinterpret_cast<f32x4_t*>(p));
}

DEV float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}
DEV float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, WAVE));
  return v;
}

DEV floatx16 mfma32(bf16x8 a, bf16x8 b, floatx16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Transpose two 4-byte words holding (r0c0,r0c1) and (r1c0,r1c1) into
// (r0c0,r1c0) and (r0c1,r1c1).
DEV uint32_t lo_pair(uint32_t r0, uint32_t r1) { return (r0 & 0xffffu) | (r1 << 16); }
DEV uint32_t hi_pair(uint32_t r0, uint32_t r1) { return (r0 >> 16) | (r1 & 0xffff0000u); }

// GELU, tanh form: 0.5 u (1 + tanh(y)) with y = sqrt(2/pi) (u + 0.044715 u^3).
// Evaluated as u * sigmoid(2y) (the same function, since 0.5 (1 + tanh(y)) =
// 1 / (1 + exp(-2y))): exp(-2y) = 2^z with z = -2 y log2(e) = u (G1 + G3 u^2),
// one hardware base-2 exponential (v_exp_f32) and one hardware reciprocal
// (v_rcp_f32), both within 1 ulp. An IEEE division here would cost ten
// instructions more per element of a GEMM epilogue. Large |u| saturate
// cleanly: 2^z overflows to inf (reciprocal 0) or underflows to 0.
constexpr float GELU_G1 = -2.0f * 0.7978845608028654f * 1.4426950408889634f;
constexpr float GELU_G3 = GELU_G1 * 0.044715f;
DEV float gelu_sigmoid2y(float u, float u2) {
  const float e = __builtin_amdgcn_exp2f(u * fmaf(GELU_G3, u2, GELU_G1));
  return __builtin_amdgcn_rcpf(1.0f + e);
}
DEV float gelu_tanh(float u) { return u * gelu_sigmoid2y(u, u * u); }
// d/du = s + u s (1 - s) 2 sqrt(2/pi) (1 + 3*0.044715 u^2) with s = sigmoid(2y),
// evaluated as s (1 + q), q = u (1 - s) (D0 + D2 u^2)
DEV float gelu_tanh_grad(float u) {
  constexpr float D0 = 2.0f * 0.7978845608028654f, D2 = D0 * 3.0f * 0.044715f;
  const float u2 = u * u;
  const float s = gelu_sigmoid2y(u, u2);
  const float q = (u * (1.0f - s)) * fmaf(D2, u2, D0);
  return fmaf(s, q, s);
}

// SwiGLU of one (gate g, up u) pair, silu(g) u with silu(g) = g sigmoid(g),
// and its gradients given the output gradient d: dg = d u s (1 + g (1 - s)),
// du = d g s with s = sigmoid(g) = 1 / (1 + e^-g), the division correctly
// rounded. Shared by the separate SwiGLU kernels and the GEMM epilogues that
// fuse them, so the two arrangements compute the same bits.
DEV float sigmoid_f(float x) { return 1.0f / (1.0f + __expf(-x)); }
DEV float swiglu1(float g, float u) { return g * sigmoid_f(g) * u; }
DEV void swiglu1_bwd(float d, float g, float u, float& dg, float& du) {
  const float s = sigmoid_f(g);
  dg = d * u * s * (1.0f + g * (1.0f - s));
  du = d * g * s;
}
