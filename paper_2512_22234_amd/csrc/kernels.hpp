// Kernel argument blocks and launchers shared between the C-ABI layer and the
// kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

namespace bd {

struct Shape {
  int B, L, S, Hq, Hkv, D;
  int G;        // Hq / Hkv
  float scale;  // softmax scale (already resolved)
};

// Forward tiles: BM queries per workgroup (4 waves x 32), BN keys per step.
constexpr int FWD_BM = 128, FWD_BN = 64;
// dQ tiles: same shape as the forward.
constexpr int DQ_BM = 128, DQ_BN = 64;
// dK/dV tiles: BN keys per workgroup (4 key groups x 32), BM queries per step.
constexpr int DKV_BN = 128, DKV_BM = 32;

hipError_t launch_cast_f32_to_bf16(const float* x, void* y, size_t n, hipStream_t st);
hipError_t launch_cast_bf16_to_f32(const void* x, float* y, size_t n, hipStream_t st);

hipError_t launch_fwd(const Shape& s, const void* Q, const void* K, const void* V,
                      void* O, float* LSE, hipStream_t st);

// Backward, in launch order:
//   dq:   dQ, and per query row the float32 pair (lse2, delta) =
//         (LSE * log2(e), rowsum(dO * O)) interleaved in rs[2 * row], rs[2 * row + 1]
//         (B*Hq*2L rows); also zeroes the dK/dV pairing counters `pair`.
//   dkdv: dK and dV.  Each clean key tile's walk runs as two halves; the half
//         that finishes first leaves float32 sums in `part` (dkdv_partial_floats
//         elements), the other adds them to its own.
hipError_t launch_bwd_dq(const Shape& s, const void* Q, const void* K, const void* V, const void* dO,
                         const void* O, const float* LSE, float* rs, int* pair, void* dQ, hipStream_t st);
hipError_t launch_bwd_dkdv(const Shape& s, const void* Q, const void* K, const void* V,
                           const void* dO, const float* rs, void* dK, void* dV, float* part, int* pair,
                           hipStream_t st);

// float32 sums of one half of the clean key tiles' walks: dK and dV.
inline size_t dkdv_partial_floats(int B, int Hkv, int L, int D) {
  return (size_t)2 * B * Hkv * L * D;
}
// Pairing counters: per (clean key tile, batch x KV head, key group of 32) an
// arrival count and a ready flag.
inline size_t dkdv_pair_ints(int B, int Hkv, int L) {
  return (size_t)2 * 4 * B * Hkv * ((L + DKV_BN - 1) / DKV_BN);
}

}  // namespace bd
