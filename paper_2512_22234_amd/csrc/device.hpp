// Device-side building blocks for the gfx950 (CDNA4) kernels.
//
// MFMA conventions used throughout (v_mfma_f32_32x32x16_bf16, wave64):
//   A operand: lane l holds A[m = l%32][k-slot (l/32, e)], e = 0..7
//   B operand: lane l holds B[k-slot (l/32, e)][n = l%32]
//   C/D      : lane l holds C[m = 8*i + 4*(l/32) + j][n = l%32] at index 4*i+j
// The k-slots of A and B are paired by (lane group, element), so any fixed
// order of the 16 contraction indices over the slots gives the same sum.
// When a product's B operand is taken straight from a previous accumulator
// (P or dS), the 16 contraction indices of chunk c land in slot (g, e) as
//   index = 16*c + keyof(8*g + e),  keyof(u) = u with bits 2 and 3 swapped,
// and the matching A operand is read from tiles stored in that order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "tiles.hpp"

namespace bd {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;
constexpr int KBLK_INVALID = 0x3fffffff;  // block index of a key past the end of its half
constexpr int QBLK_INVALID = -1;          // block index of a query past the end of its half

// Storage position of index k inside an aligned group of 16 (self-inverse).
__host__ __device__ inline int perm16(int k) {
  return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1);
}

__device__ inline f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ inline bf16x8 zero_bf16x8() {
  u32x4 z = {0u, 0u, 0u, 0u};
  return __builtin_bit_cast(bf16x8, z);
}

__device__ inline u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ inline void st16(void* p, const u32x4& v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ inline bf16x8 lds_bf16x8(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }

// Eight consecutive accumulator values as a bf16 MFMA operand (round to nearest even).
__device__ inline bf16x8 pack8(const f32x16& acc, int base) {
  bf16x8 r;
#pragma unroll
  for (int e = 0; e < 8; ++e) r[e] = (bf16)acc[base + e];
  return r;
}

// Store four consecutive bf16 values (8 bytes).
__device__ inline void st_bf16x4(bf16* p, float a, float b, float c, float d) {
  bf16x4 v;
  v[0] = (bf16)a;
  v[1] = (bf16)b;
  v[2] = (bf16)c;
  v[3] = (bf16)d;
  *reinterpret_cast<bf16x4*>(p) = v;
}

// Workgroup -> head mapping that keeps all query heads of one KV group on the
// same XCD (workgroups are dispatched round-robin over the 8 XCDs), so K/V of a
// group are shared through that XCD's L2.  pos in [0, nbh); falls back to the
// identity when the counts do not divide evenly.
__device__ inline int xcd_head_remap(int pos, int nbh, int G) {
  const int ngroups = nbh / G;
  if ((nbh & 7) != 0 || (ngroups & 7) != 0) return pos;
  const int x = pos & 7, s = pos >> 3;
  const int group = x + 8 * (s / G);
  return group * G + (s % G);
}

}  // namespace bd
