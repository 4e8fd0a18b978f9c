// LDS helpers shared by the attention kernels (forward and backward): loads from global
// memory straight into LDS, and the two LDS read forms the MFMA operands use.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace tsp {

typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char lds_char;

__device__ __forceinline__ void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// 16 bytes per lane from global memory straight into LDS at lds + 16 * lane: the
// buffer form, with the address = resource base (scalar) + soff (scalar) + voff (lane);
// M0 holds the wave's LDS destination.
//
// Issued from inline assembly on purpose.  The compiler cannot tell which LDS bytes an
// LDS-destination load writes, so after one it puts a full vmcnt(0) wait in front of
// the next LDS read it cannot prove disjoint, which would stall every step of a
// pipelined loop on the load of the NEXT tile.  Hidden in asm, the load is ordered only
// by the kernel's own waits: a kernel using it reads a slot only after a vmcnt(0) wait
// that follows the slot's loads and a barrier (or an LDS counter that every loading
// wavefront raises after that wait), and refills a slot only after a barrier (or a
// counter that every reader raises after its last read) that follows its last read.  The compiler's own waits stay correct because loads
// complete in issue order.  Kernels using this helper use M0 nowhere else (a reserved
// register the compiler does not track through asm).
typedef u32x4 rsrc_t;
__device__ __forceinline__ void dma16(const rsrc_t& rsrc, uint32_t voff, uint32_t soff,
                                      lds_char* lds) {
  const uint32_t m0 = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
               :: "v"(voff), "s"(rsrc), "s"(soff), "s"(m0) : "memory", "m0");
}

// Raw buffer resource over [base, base + 4 GiB) (stride 0, no format conversion): base
// address (48 bits), number of records, and the data-format word of a raw resource.
__device__ __forceinline__ rsrc_t make_rsrc(const void* base) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  return rsrc_t{(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a),
                (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32) & 0xffffu),
                0xffffffffu, 0x00020000u};
}

__device__ __forceinline__ u32x4 lds_read16(const lds_char* p) {
  return *reinterpret_cast<const __attribute__((address_space(3))) u32x4*>(p);
}

// gfx950 LDS transpose read (ds_read_b64_tr_b16): in each 16-lane group, source lane s
// points at row kbase + s / 4, columns base + 4 (s % 4), and lane t receives column
// base + t of rows kbase .. kbase + 3 (four bf16, row order).
__device__ __forceinline__ u32x2 lds_read_tr(const lds_char* p) {
  return __builtin_bit_cast(
      u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)p));
}

}  // namespace tsp
