// LDS helpers shared by the GEMM and attention kernels: direct HBM->LDS loads
// through raw buffer descriptors, a barrier without a memory fence, and the
// transposed 16-bit LDS read of gfx950.
#pragma once

#include "common.h"

#define LDS_AS __attribute__((address_space(3)))
typedef LDS_AS void lds_void_t;
typedef LDS_AS char lds_char_t;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef LDS_AS v4i16 lds_v4i16_t;
typedef unsigned int v4u32 __attribute__((ext_vector_type(4)));
typedef LDS_AS v4u32 lds_v4u32_t;
typedef int v4i32 __attribute__((ext_vector_type(4)));

// Raw buffer descriptor over [base, base+bytes): stride 0, range checked, so
// loads past the end return zero.
DEV v4i32 make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  v4i32 r;
  r.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r.y = __builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
  r.z = __builtin_amdgcn_readfirstlane((int)bytes);
  r.w = 0x00020000;
  return r;
}

// 16 bytes per lane from the buffer at byte offset voff into LDS at
// lds_base + 16*lane. Issued as inline assembly: kernels track these loads
// themselves (wait_vmcnt before the barrier that publishes a stage); the
// compiler's own conservative wait before every LDS read would serialise the
// pipelines.
DEV void dma16(v4i32 rsrc, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds_base)), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}

DEV uint32_t lds_addr(const lds_char_t* p) { return (uint32_t)reinterpret_cast<uintptr_t>(p); }

// vmcnt-only wait (expcnt and lgkmcnt left at their maxima)
template <int N>
DEV void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// workgroup barrier without the memory fence of __syncthreads (which would
// wait for the prefetches still in flight)
DEV void block_barrier() { asm volatile("s_barrier" ::: "memory"); }

DEV bf16x8 lds_read16(const lds_char_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const lds_v4u32_t*>(p));
}

// ds_read_b64_tr_b16: within each group of 16 lanes, lane t receives element
// t%4 of the 8-byte chunks addressed by lanes t/4 + 4j, j = 0..3. So if lane s
// of the group addresses row r0 + s/4 at columns c0 + 4*(s%4)..+3 of a
// row-major 16-bit tile, lane t receives column c0 + t at rows r0..r0+3.
DEV uint2 lds_read_tr(const lds_char_t* p) {
  return __builtin_bit_cast(uint2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t*)p));
}
