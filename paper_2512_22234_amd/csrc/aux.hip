// fp32 <-> bf16 conversion for callers that hand the library float32 tensors.
#include "device.hpp"
#include "kernels.hpp"

namespace bd {
namespace {

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

hipError_t launch_cast_f32_to_bf16(const float* x, void* y, size_t n, hipStream_t st, LaunchEvents ev) {
  hipExtLaunchKernelGGL(cast_f32_bf16_kernel, dim3(cast_grid(n)), dim3(256), 0, st, ev.start, ev.stop, 0, x,
                        static_cast<bf16*>(y), n);
  return hipGetLastError();
}

hipError_t launch_cast_bf16_to_f32(const void* x, float* y, size_t n, hipStream_t st, LaunchEvents ev) {
  hipExtLaunchKernelGGL(cast_bf16_f32_kernel, dim3(cast_grid(n)), dim3(256), 0, st, ev.start, ev.stop, 0,
                        static_cast<const bf16*>(x), y, n);
  return hipGetLastError();
}

}  // namespace bd
