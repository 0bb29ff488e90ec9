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
// and the matching A operand is read in that order by lds_read_tr.
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

__device__ inline f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// MFMA A/B operand for a contraction over the ROW index of a row-major LDS
// tile X[row][col] (row stride `stride` elements): returns, for this lane, the
// 8 values X[row0 + keyof(8*g + e)][col0 + l%32], e = 0..7, g = lane/32 -- the
// operand layout described above with rows as contraction indices.
//
// ds_read_b64_tr_b16 works on groups of 16 lanes: lane i of a group receives
// element i%4 of the 8-byte chunks addressed by lanes 4r + i/4 of its group,
// r = 0..3.  So lane 4r + c of a group points at row (base + r), columns
// [4c, 4c+4) of its 16-column slice, and two reads cover rows keyof(0..3) and
// keyof(4..7) of the lane's half-wave.
__device__ inline bf16x8 lds_read_tr(const bf16* tile, int stride, int row0, int col0, int lane) {
  const int h = lane >> 4, j = lane & 15;
  const int row = row0 + 4 * (h >> 1) + (j >> 2);
  const int col = col0 + 16 * (h & 1) + 4 * (j & 3);
  const bf16* p0 = tile + row * stride + col;
  const bf16* p1 = p0 + 8 * stride;
  const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p0));
  const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p1));
  typedef short s16x8 __attribute__((ext_vector_type(8)));
  const s16x8 v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return __builtin_bit_cast(bf16x8, v);
}

__device__ inline bf16x8 zero_bf16x8() {
  u32x4 z = {0u, 0u, 0u, 0u};
  return __builtin_bit_cast(bf16x8, z);
}

__device__ inline u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

// 16 bytes of row min(row, nrows-1) of a row-major bf16 array.  Rows past the
// end of a half are always masked out of the softmax (their P is exactly 0),
// so they only need to hold finite data; clamping keeps the load
// unconditional and its result unused until the LDS store, so the compiler's
// count of outstanding loads stays exact and the load latency overlaps the
// compute of the current tile.
__device__ inline u32x4 ld16_rows(const bf16* base, int row, int nrows, int row_elems, int col) {
  const int r = row < nrows ? row : nrows - 1;
  return ld16(base + (size_t)r * row_elems + col);
}

// Keeps the compiler from moving memory operations or scheduling instructions
// across this point.  Placed between a tile's compute and the LDS stores of
// the prefetched next tile, so the prefetch's global-load latency stays hidden
// behind the compute instead of being waited for up front.
__device__ inline void compute_fence() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_sched_barrier(0);
}

// Wait until every global load this wave issued has landed (s_waitcnt vmcnt(0)).
__device__ inline void wait_global_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Block-index window [lo, hi] of keys visible from one query (block bq, or
// QBLK_INVALID past the end of its half) in the quadrant (qh, kh); an empty
// window has lo > hi.  Keys past the end carry KBLK_INVALID and never fall in.
struct BlockWindow {
  int lo, hi;
  __device__ bool has(int b) const { return b >= lo && b <= hi; }
};
__device__ inline BlockWindow key_window(int qh, int kh, int bq) {
  if (bq < 0) return {1, 0};
  if (qh == HALF_NOISY) return kh == HALF_NOISY ? BlockWindow{bq, bq} : BlockWindow{0, bq - 1};
  return kh == HALF_CLEAN ? BlockWindow{0, bq} : BlockWindow{1, 0};
}
// The same rule seen from one key (block bk): window of visible query blocks.
__device__ inline BlockWindow query_window(int qh, int kh, int bk) {
  if (qh == HALF_NOISY) return kh == HALF_NOISY ? BlockWindow{bk, bk} : BlockWindow{bk + 1, 0x7fffffff};
  return kh == HALF_CLEAN ? BlockWindow{bk, 0x7fffffff} : BlockWindow{1, 0};
}
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
