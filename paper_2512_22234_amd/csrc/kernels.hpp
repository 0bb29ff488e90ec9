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

// Per query row the float32 pair (lse2, delta) = (LSE * log2(e), rowsum(dO * O)),
// interleaved: rs[2 * row], rs[2 * row + 1]; B*Hq*2L rows.
hipError_t launch_bwd_pre(const Shape& s, const void* O, const void* dO, const float* LSE, float* rs,
                          hipStream_t st);
// dK/dV kernel: noisy key tiles straight to dK/dV, clean key tiles as two
// float32 partial sums in part (dkdv_partial_floats elements), which the
// combine kernel then adds into dK/dV.
hipError_t launch_bwd_dkdv(const Shape& s, const void* Q, const void* K, const void* V,
                           const void* dO, const float* rs, void* dK, void* dV, float* part, hipStream_t st);
hipError_t launch_bwd_dkdv_combine(const Shape& s, const float* part, void* dK, void* dV, hipStream_t st);
hipError_t launch_bwd_dq(const Shape& s, const void* Q, const void* K, const void* V,
                         const void* dO, const float* rs, void* dQ, hipStream_t st);

// float32 partial sums of the clean half of dK and dV: 2 halves x 2 tensors.
inline size_t dkdv_partial_floats(int B, int Hkv, int L, int D) {
  return (size_t)4 * B * Hkv * L * D;
}

}  // namespace bd
