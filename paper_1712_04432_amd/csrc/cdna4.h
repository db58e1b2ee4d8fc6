// gfx950 building blocks shared by the streaming kernels: raw buffer descriptors,
// buffer loads that write LDS directly, barriers with explicit memory-counter waits,
// and the hardware bf16 pack.
#pragma once

#include "common.h"

namespace imbd {

constexpr int BUF_DW3 = 0x00020000;  // raw buffer resource word 3 (gfx9 family): 32-bit format

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

__device__ __forceinline__ i32x4 buf_rsrc(const void *base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  i32x4 r;
  r[0] = (int)(uint32_t)b;
  r[1] = (int)((uint32_t)(b >> 32) & 0xffffu);  // stride 0
  r[2] = (int)bytes;                             // offsets at or past this read as zero
  r[3] = BUF_DW3;
  return r;
}

// One wave writes 64 x 16 bytes to LDS at lds_base + 16*lane from byte offsets voff of
// the buffer; an offset at or past the descriptor's range writes zeros. Issued from
// inline assembly so that the compiler does not drain the loads at every LDS read: the
// caller waits for them explicitly (vmcnt) before the barrier that publishes the slab.
// m0 holds the LDS base of the write. It is an operand of the statement ("{m0}"), so the
// compiler itself writes m0 and knows what it holds: it never keeps a value of its own
// there across the load. The s_nop covers the wait state between a write of m0 and an
// LDS-writing load.
__device__ __forceinline__ void dma16(const i32x4 &rsrc, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(voff), "s"(rsrc), "{m0}"(lds_base)
               : "memory");
}

// The 4-byte form: 64 x 4 bytes to LDS at lds_base + 4*lane (for rows whose pitch is a
// multiple of 4 bytes only; four of these stand in for one 16-byte load).
__device__ __forceinline__ void dma4(const i32x4 &rsrc, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_nop 0\n\tbuffer_load_dword %0, %1, 0 offen lds"
               :
               : "v"(voff), "s"(rsrc), "{m0}"(lds_base)
               : "memory");
}

template <int VM>
__device__ __forceinline__ void vm_barrier() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" : : "n"(VM) : "memory");
}
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" : : : "memory"); }

// Two floats to packed bf16, round to nearest even (the gfx950 conversion instruction).
__device__ __forceinline__ uint32_t cvt_pk_bf16(float x, float y) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){x, y}, bf16x2_t));
}

}  // namespace imbd
