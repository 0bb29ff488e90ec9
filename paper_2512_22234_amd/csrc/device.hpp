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

#include <type_traits>

#include "tiles.hpp"

namespace bd {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// A compile-time flag passed as an argument (selects code variants of a lambda).
template <bool B>
using Flag = std::integral_constant<bool, B>;

constexpr float LOG2E = 1.4426950408889634f;
constexpr float LN2 = 0.6931471805599453f;

__device__ inline bf16x8 zero_bf16x8() {
  u32x4 z = {0u, 0u, 0u, 0u};
  return __builtin_bit_cast(bf16x8, z);
}

__device__ inline f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// LDS tiles are row-major [rows][D] with no padding; the 16-byte chunks of a
// row are permuted by an XOR with chunk_swizzle<D>(row).  With 64 four-byte
// banks, the mask makes both access patterns below conflict-free for every
// group of 16 lanes: 16-byte row slices of 16 consecutive rows at one column
// (row-major MFMA operands), and 8-byte pieces of 4 consecutive rows x 32
// bytes (the transposing read).  Padding can only fix one of the two.
template <int D> __host__ __device__ inline int chunk_swizzle(int r);
template <> __host__ __device__ inline int chunk_swizzle<128>(int r) {
  return ((r & 3) << 1) | ((r >> 2) & 1) | (r & 8);
}
template <> __host__ __device__ inline int chunk_swizzle<64>(int r) {
  return (((r >> 1) & 3) << 1) | ((r >> 3) & 1);
}
// 64-byte rows (GEMM k-chunks of 32): four rows share a 256-byte bank cycle,
// so 16 consecutive rows at one 16-byte column land on 16 distinct bank
// groups when the chunk moves with row / 4.
template <> __host__ __device__ inline int chunk_swizzle<32>(int r) { return (r >> 2) & 3; }
// Element index of (row, col) in a swizzled tile; col % 8 stays in place.
template <int D> __host__ __device__ inline int tile_idx(int row, int col) {
  return row * D + ((((col >> 3) ^ chunk_swizzle<D>(row)) << 3) | (col & 7));
}

// MFMA A/B operand for a contraction over the ROW index of a swizzled LDS
// tile X[row][col]: returns, for this lane, the 8 values
// X[row0 + keyof(8*g + e)][col0 + l%32], e = 0..7, g = lane/32 -- the operand
// layout described above with rows as contraction indices.
//
// ds_read_b64_tr_b16 works on groups of 16 lanes: lane i of a group receives
// element i%4 of the 8-byte chunks addressed by lanes 4r + i/4 of its group,
// r = 0..3.  So lane 4r + c of a group points at row (base + r), columns
// [4c, 4c+4) of its 16-column slice, and two reads cover rows keyof(0..3) and
// keyof(4..7) of the lane's half-wave.
template <int D>
__device__ inline bf16x8 lds_read_tr(const bf16* tile, int row0, int col0, int lane) {
  const int h = lane >> 4, j = lane & 15;
  const int row = row0 + 4 * (h >> 1) + (j >> 2);
  const int col = col0 + 16 * (h & 1) + 4 * (j & 3);
  const bf16* p0 = tile + tile_idx<D>(row, col);
  const bf16* p1 = tile + tile_idx<D>(row + 8, col);
  const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p0));
  const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p1));
  typedef short s16x8 __attribute__((ext_vector_type(8)));
  const s16x8 v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// Per-lane byte offsets that turn every MFMA-operand read of a swizzled tile
// into one XOR with a compile-time constant plus an immediate offset.  With
// F = chunk_swizzle(row) depending only on row % 16, the chunk of a row-slice
// read is (2s + g) ^ F, whose byte offset 32*(s ^ F/2) + 16*(g ^ F%2) equals
// (32*F/2 + 16*(g ^ F%2)) ^ 32*s; likewise the feature block db of a
// transposing read only flips bits 6-7.  Tile offsets must be multiples of
// 256 bytes so that adding them leaves bits 0-7 alone.
template <int D>
struct LdsOperands {
  uint32_t row_rel;          // row-slice reads: row 32*rb + lane%32, columns 16*s + 8*(lane/32)
  uint32_t tr_rel0, tr_rel1;  // transposing reads (rows keyof(0..3) and keyof(4..7) of a chunk)
  __device__ explicit LdsOperands(int lane) {
    const int l32 = lane & 31, g = lane >> 5;
    const int F = chunk_swizzle<D>(l32);
    row_rel = (uint32_t)(l32 * 2 * D + 16 * (g ^ (F & 1)) + 32 * (F >> 1));
    const int h = lane >> 4, j = lane & 15;
    const int x = 2 * (h & 1) + ((j >> 1) & 1);
    const int r0 = 4 * (h >> 1) + (j >> 2);
    const int f0 = chunk_swizzle<D>(r0), f1 = chunk_swizzle<D>(r0 + 8);
    constexpr int HI = (D / 8 - 1) & ~3;
    tr_rel0 = (uint32_t)(r0 * 2 * D + 16 * (f0 & HI) + 16 * (x ^ (f0 & 3)) + 8 * (j & 1));
    tr_rel1 = (uint32_t)((r0 + 8) * 2 * D + 16 * (f1 & HI) + 16 * (x ^ (f1 & 3)) + 8 * (j & 1));
  }
};

// Transposing operand reads in linear k order, for products whose other
// operand is also read from LDS: lane (l32, g) gets X[row0 + 8g + e][col0 + l32],
// e = 0..7 -- the slot order of a row-slice read (k = 8g + e), so a
// transposed tile can meet a row-major one in one MFMA.  Same conflict-free
// pattern as LdsOperands' reads (four consecutive rows of 32 bytes per group
// of 16 lanes).  Tile offsets must be multiples of 256 bytes.
template <int D>
struct LdsLinearTr {
  uint32_t rel0, rel1;  // byte offsets of rows 8g + (lane%16)/4 and 8g + 4 + (lane%16)/4
  __device__ explicit LdsLinearTr(int lane) {
    const int h = lane >> 4, j = lane & 15;
    const int x = 2 * (h & 1) + ((j >> 1) & 1);
    const int r0 = 8 * (h >> 1) + (j >> 2);
    const int f0 = chunk_swizzle<D>(r0), f1 = chunk_swizzle<D>(r0 + 4);
    constexpr int HI = (D / 8 - 1) & ~3;
    rel0 = (uint32_t)(r0 * 2 * D + 16 * (f0 & HI) + 16 * (x ^ (f0 & 3)) + 8 * (j & 1));
    rel1 = (uint32_t)((r0 + 4) * 2 * D + 16 * (f1 & HI) + 16 * (x ^ (f1 & 3)) + 8 * (j & 1));
  }
};

// Row-slice operand (same values as lds_row8<D>(tile, 32*rb + lane%32, 16*s + 8*(lane/32)))
// from a tile starting at byte offset `base - row_rel` of lds.
template <int D>
__device__ inline bf16x8 lds_rows(const char* lds, uint32_t base, int s, int rb) {
  return *reinterpret_cast<const bf16x8*>(lds + ((base ^ (uint32_t)(32 * s)) + (uint32_t)(rb * 64 * D)));
}
// Transposing operand (same values as lds_read_tr<D>(tile, 16*c, 32*db, lane)); b0/b1 = tile offset + tr_rel0/1.
template <int D>
__device__ inline bf16x8 lds_tr(const char* lds, uint32_t b0, uint32_t b1, int c, int db) {
  const uint32_t o = (uint32_t)(c * 32 * D);
  const s16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(lds + ((b0 ^ (uint32_t)(64 * db)) + o)));
  const s16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(lds + ((b1 ^ (uint32_t)(64 * db)) + o)));
  typedef short s16x8 __attribute__((ext_vector_type(8)));
  const s16x8 v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  return __builtin_bit_cast(bf16x8, v);
}

// Buffer resource over `bytes` bytes at base (raw buffer, no stride): loads
// at offsets at or past `bytes` return zero instead of faulting.
__device__ inline __amdgpu_buffer_rsrc_t make_buffer(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)bytes, 0x00020000);
}

// Asynchronous copy of a tile of NR rows x D bf16 from a row-major array into
// a swizzled LDS tile with buffer_load ... lds (16 bytes per lane; the LDS
// address of lane i is M0 + 16*i).  Each wave instruction fills 1 KiB of the
// tile contiguously; lane i fetches the global chunk that belongs at LDS chunk
// p (the XOR swizzle is its own inverse).  The per-lane byte offsets do not
// depend on which tile is copied, so a copy costs one scalar buffer
// descriptor per tile.  Rows past the end of the array read as zero; rows
// past the end of a half read the other half's rows: the kernels mask both out.
//
// Buffer (MUBUF) rather than global (FLAT-encoded) loads: the compiler
// treats a FLAT load into LDS as touching both counters, and while one is in
// flight it turns every LDS-read wait into a full drain (lgkmcnt(0)), which
// would serialise the operand reads of the whole step behind the prefetch.
// Completion is tracked by the wave's vmcnt (wait_global_loads) and must be
// followed by a workgroup barrier before other waves read the tile.
template <int D, int NR, int NT>
struct TileCopy {
  static constexpr int CPR = D / 8;
  static constexpr int NW = NT / 64;
  static constexpr int NI = NR * CPR / NT;
  static_assert(NI * NT == NR * CPR, "tile must split evenly over the workgroup");
  uint32_t boff[NI];  // byte offset of the source chunk from the tile's first row
  int wave;           // wave index, uniform
  __device__ explicit TileCopy(int tid) {
    wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lane = tid & 63;
#pragma unroll
    for (int u = 0; u < NI; ++u) {
      const int p = (u * NW + wave) * 64 + lane;
      const int row = p / CPR;
      boff[u] = (uint32_t)(2 * (row * D + (((p % CPR) ^ chunk_swizzle<D>(row)) << 3)));
    }
  }
  // Buffer over rows [row0, nrows) of the row-major array arr[nrows][D].  It
  // starts at row0 (the range check covers the per-lane offset only), so rows
  // at or past nrows read as zero.
  __device__ static __amdgpu_buffer_rsrc_t rows(const bf16* arr, int nrows, int row0) {
    return make_buffer(arr + (size_t)row0 * D, (uint32_t)((nrows - row0) * D * 2));
  }
  // Instruction u of the copy of the tile at the start of rsrc into dst.
  __device__ void issue_one(__amdgpu_buffer_rsrc_t rsrc, char* dst, int u) const {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rsrc, (__attribute__((address_space(3))) void*)(dst + (u * NW + wave) * 1024), 16, (int)boff[u], 0, 0, 0);
  }
  // Copy the NR rows starting at `first` (of which `left` lie inside the
  // array; the rest read as zero) into the tile at dst.
  __device__ void issue_rows(const bf16* first, int left, char* dst) const {
    const __amdgpu_buffer_rsrc_t rsrc = make_buffer(first, (uint32_t)(left * D * 2));
#pragma unroll
    for (int u = 0; u < NI; ++u) issue_one(rsrc, dst, u);
  }
  // Copy rows [row0, row0 + NR) of arr[nrows][D] into the tile at dst.
  __device__ void issue(const bf16* arr, int nrows, int row0, char* dst) const {
    const __amdgpu_buffer_rsrc_t rsrc = rows(arr, nrows, row0);
#pragma unroll
    for (int u = 0; u < NI; ++u) issue_one(rsrc, dst, u);
  }
};

// Asynchronous copy of 64 consecutive floats arr[row0 .. row0+63] (those at or
// past nrows read as zero) into LDS dst[0..63]: one instruction of one wave.
__device__ inline void async_load_row_floats(const float* arr, int nrows, int row0, float* dst, int lane) {
  const __amdgpu_buffer_rsrc_t rsrc = make_buffer(arr + row0, (uint32_t)((nrows - row0) * 4));
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, (__attribute__((address_space(3))) void*)dst, 4, 4 * lane, 0, 0, 0);
}

// Scheduling request for the current basic block of NM MFMAs that each take
// RPM LDS operand reads and share NV copy instructions: the reads run AHEAD
// MFMAs ahead of their use and the copies are spread evenly between the
// MFMAs.  Place it after the block's last instruction.
template <int NM, int AHEAD, int RPM, int NV>
__device__ inline void pipeline_reads_and_copies() {
  static_assert(AHEAD >= 1 && AHEAD <= NM && (NV == 0 || NM >= NV), "schedule shape");
  __builtin_amdgcn_sched_group_barrier(0x100, AHEAD * RPM, 0);  // DS read
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
    if (i + AHEAD < NM) __builtin_amdgcn_sched_group_barrier(0x100, RPM, 0);
    if (NV > 0 && i % (NM / (NV > 0 ? NV : 1)) == 0 && i / (NM / (NV > 0 ? NV : 1)) < NV)
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // VMEM read (tile copy)
  }
}

// Scheduling request for the current basic block: LDS operand reads run
// AHEAD MFMAs ahead of their use.  The first AHEAD * RPM reads (plus FIRST
// more, e.g. operands shared by all MFMAs) go first, then each MFMA is
// followed by the RPM reads of the operand AHEAD MFMAs later.
template <int NM, int AHEAD, int RPM, int FIRST = 0>
__device__ inline void pipeline_lds_reads() {
  static_assert(AHEAD >= 1 && AHEAD <= NM, "read distance");
  __builtin_amdgcn_sched_group_barrier(0x100, AHEAD * RPM + FIRST, 0);  // DS read
#pragma unroll
  for (int i = 0; i < NM; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
    if (i + AHEAD < NM) __builtin_amdgcn_sched_group_barrier(0x100, RPM, 0);
  }
}

__device__ inline u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }

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
// Wait until all but the N most recent global loads of this wave have landed
// (loads complete in issue order for this counter).
template <int N>
__device__ inline void wait_global_loads_but() {
  static_assert(N >= 0 && N < 64, "vmcnt immediate");
  // vmcnt is split over bits 3:0 and 15:14 of the immediate
  __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

// Workgroup barrier that drains this wave's LDS operations (lgkmcnt(0)) but
// not its global loads.  __syncthreads() would also wait for every global
// load in flight (vmcnt(0)), including tile copies issued for steps well
// ahead; a kernel that uses this barrier waits for the copies it needs with
// wait_global_loads_but<N>() first.  The signal fences keep the compiler from
// moving memory operations across it.
__device__ inline void barrier_lds_only() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt at their maxima (no wait)
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

__device__ inline void st16(void* p, const u32x4& v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ inline bf16x8 lds_bf16x8(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }
// 8 consecutive elements (one 16-byte chunk) of a swizzled tile; col % 8 == 0.
template <int D>
__device__ inline bf16x8 lds_row8(const bf16* tile, int row, int col) {
  return lds_bf16x8(tile + tile_idx<D>(row, col));
}

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

// Combine a per-lane value over the two half-waves (lanes l and l + 32 hold
// the two halves of one row's keys or features) with v_permlane32_swap.
__device__ inline float halves_max(float x) {
  const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(sw[0]), __uint_as_float(sw[1]));
}
__device__ inline float halves_sum(float x) {
  const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(sw[0]) + __uint_as_float(sw[1]);
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
