// Layout helpers: key-major -> feature-major transposed copies of K and V
// (keys in perm16 order, halves zero-padded), and fp32 <-> bf16 conversion for
// callers that hand the library float32 tensors.
#include "device.hpp"
#include "kernels.hpp"

namespace bd {
namespace {

// One workgroup moves a 64-key x 64-feature block of X [n][2L][D] into
// Xt [n][D][2*Lp]: keys of half h go to columns h*Lp + perm16(key); keys in
// [L, Lp) are written as zeros.
__global__ __launch_bounds__(256) void transpose_keys_kernel(const uint16_t* __restrict__ X,
                                                             uint16_t* __restrict__ Xt, int L, int Lp,
                                                             int D) {
  __shared__ uint16_t tile[64][64 + 2];
  const int tiles_per_half = Lp / 64;
  const int h = blockIdx.x / tiles_per_half;
  const int kt = blockIdx.x - h * tiles_per_half;
  const int d0 = blockIdx.y * 64;
  const size_t n = blockIdx.z;
  const int tid = threadIdx.x;
  const uint16_t* xp = X + n * (size_t)(2 * L) * D;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int c = tid + 256 * u;
    const int key = c / 8, f8 = c % 8;
    const int kl = kt * 64 + key;
    u32x4 v = {0u, 0u, 0u, 0u};
    if (kl < L) v = ld16(xp + (size_t)(h * L + kl) * D + d0 + f8 * 8);
#pragma unroll
    for (int e = 0; e < 8; ++e) tile[key][f8 * 8 + e] = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
  }
  __syncthreads();
  uint16_t* out = Xt + (n * D + d0) * (size_t)(2 * Lp) + h * Lp + kt * 64;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int c = tid + 256 * u;
    const int d = c / 8, p8 = c % 8;
    u32x4 v;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const uint32_t lo = tile[perm16(p8 * 8 + 2 * e)][d];
      const uint32_t hi = tile[perm16(p8 * 8 + 2 * e + 1)][d];
      v[e] = lo | (hi << 16);
    }
    st16(out + (size_t)d * (2 * Lp) + p8 * 8, v);
  }
}

__global__ __launch_bounds__(256) void cast_f32_bf16_kernel(const float* __restrict__ x, bf16* __restrict__ y,
                                                            size_t n) {
  const size_t stride = (size_t)gridDim.x * 256;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) y[i] = (bf16)x[i];
}

__global__ __launch_bounds__(256) void cast_bf16_f32_kernel(const bf16* __restrict__ x, float* __restrict__ y,
                                                            size_t n) {
  const size_t stride = (size_t)gridDim.x * 256;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) y[i] = (float)x[i];
}

unsigned cast_grid(size_t n) {
  size_t blocks = (n + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  if (blocks == 0) blocks = 1;
  return (unsigned)blocks;
}

}  // namespace

hipError_t launch_transpose_keys(const void* X, void* Xt, int n, int L, int Lp, int D, hipStream_t st) {
  const dim3 grid(2 * (Lp / 64), D / 64, n);
  hipLaunchKernelGGL(transpose_keys_kernel, grid, dim3(256), 0, st, static_cast<const uint16_t*>(X),
                     static_cast<uint16_t*>(Xt), L, Lp, D);
  return hipGetLastError();
}

hipError_t launch_cast_f32_to_bf16(const float* x, void* y, size_t n, hipStream_t st) {
  hipLaunchKernelGGL(cast_f32_bf16_kernel, dim3(cast_grid(n)), dim3(256), 0, st, x, static_cast<bf16*>(y), n);
  return hipGetLastError();
}

hipError_t launch_cast_bf16_to_f32(const void* x, float* y, size_t n, hipStream_t st) {
  hipLaunchKernelGGL(cast_bf16_f32_kernel, dim3(cast_grid(n)), dim3(256), 0, st, static_cast<const bf16*>(x), y, n);
  return hipGetLastError();
}

}  // namespace bd
