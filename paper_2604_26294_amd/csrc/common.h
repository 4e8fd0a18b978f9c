// Device-side building blocks for the gfx950 kernels of libtsp.
//
// MFMA v_mfma_f32_32x32x16_bf16, per lane l of a 64-wide wavefront (h = l / 32):
//   A operand: 8 bf16 of row i = l % 32 at contraction slots 8h .. 8h+7
//   B operand: 8 bf16 of column j = l % 32 at the same contraction slots
//   C/D      : 16 fp32, element 4g + r holds C[8g + 4h + r][l % 32]  (g, r in 0..3)
// Only the pairing of A and B slots matters for the contraction, so a kernel may
// feed any fixed permutation of its 16 contraction indices to both operands.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tsp {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kXcds = 8;  // MI355X: 8 accelerator complex dies, 32 CUs and one L2 each

__device__ __forceinline__ f32x16 mfma32(const u32x4& a, const u32x4& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Two fp32 -> one dword of two bf16 (round to nearest even; low half = first).
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  bf16x2_t v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint16_t to_bf16_bits(float x) {
  return __builtin_bit_cast(uint16_t, (__bf16)x);
}

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t bits16) {
  return __builtin_bit_cast(float, bits16 << 16);
}

// 16-byte global load / store helpers.
__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, const u32x4& v) { *reinterpret_cast<u32x4*>(p) = v; }

// LDS tiles are arrays of rows made of 16-byte chunks; the chunk index is XORed with
// the low 3 bits of the row so that 8 consecutive rows read at the same logical chunk
// hit 8 different bank groups.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ (row & 7); }

// XCD-aware work order.  Workgroups are dispatched round-robin over the XCDs
// (workgroup b runs on XCD b % 8).  This maps dispatch index b to a work index so
// that each XCD receives one contiguous range of work indices, which keeps tiles
// that share operands in the same L2.  A bijection on [0, total).
__device__ __forceinline__ int xcd_work_index(int b, int total) {
  const int q = total / kXcds, rem = total % kXcds;
  const int x = b % kXcds, local = b / kXcds;
  return x * q + (x < rem ? x : rem) + local;
}

}  // namespace tsp
