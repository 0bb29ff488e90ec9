// Kernel argument blocks and launchers shared between the C-ABI layer and the
// kernel translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>

namespace bd {

struct Shape {
  int B, L, S, Hq, Hkv, D;
  int G;        // Hq / Hkv
  int Lp;       // half length padded to a multiple of KEY_PAD in transposed copies
  float scale;  // softmax scale (already resolved)
};

// Transposed K/V copies keep each half padded to a multiple of this many keys
// (zero filled), so key-tile loads from them never need bounds checks.
constexpr int KEY_PAD = 128;

// Forward tiles: BM queries per workgroup (4 waves x 32), BN keys per step.
constexpr int FWD_BM = 128, FWD_BN = 64;
// dQ tiles: same shape as the forward.
constexpr int DQ_BM = 128, DQ_BN = 64;
// dK/dV tiles: BN keys per workgroup (4 waves x 32), BM queries per step.
constexpr int DKV_BN = 128, DKV_BM = 64;

// X [n][2L][D] (bf16) -> Xt [n][D][2*Lp] with keys of each half stored in
// perm16 order and zero padding up to Lp.
hipError_t launch_transpose_keys(const void* X, void* Xt, int n, int L, int Lp, int D, hipStream_t st);
hipError_t launch_cast_f32_to_bf16(const float* x, void* y, size_t n, hipStream_t st);
hipError_t launch_cast_bf16_to_f32(const void* x, float* y, size_t n, hipStream_t st);

hipError_t launch_fwd(const Shape& s, const void* Q, const void* K, const void* Vt,
                      void* O, float* LSE, hipStream_t st);

hipError_t launch_bwd_pre(const Shape& s, const void* O, const void* dO, float* delta, hipStream_t st);
hipError_t launch_bwd_dkdv(const Shape& s, const void* Q, const void* K, const void* V,
                           const void* dO, const float* LSE, const float* delta,
                           void* dK, void* dV, hipStream_t st);
hipError_t launch_bwd_dq(const Shape& s, const void* Q, const void* K, const void* Kt,
                         const void* V, const void* dO, const float* LSE, const float* delta,
                         void* dQ, hipStream_t st);

}  // namespace bd
