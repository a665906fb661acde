// Conversions of the init-time V/O truncation (Appendix A.4): float32 -> bf16 (the cast of the
// float32 weights to the model's bf16, one thread per 8 values and a scalar tail), and the
// float32 <-> float64 copies around the double-precision decomposition; all round to nearest
// even.
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace unstep {
namespace {

constexpr int kThreads = 256;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kThreads) void cast_bf16_kernel(const float* x, uint16_t* y, int64_t n) {
  const int64_t i = (int64_t(blockIdx.x) * kThreads + threadIdx.x) * 8;
  if (i + 8 <= n) {
    const f32x4_t a = *reinterpret_cast<const f32x4_t*>(x + i);
    const f32x4_t b = *reinterpret_cast<const f32x4_t*>(x + i + 4);
    bf16x8_t r;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      r[e] = (__bf16)a[e];
      r[4 + e] = (__bf16)b[e];
    }
    *reinterpret_cast<bf16x8_t*>(y + i) = r;
  } else {
    for (int64_t j = i; j < n; ++j) y[j] = __builtin_bit_cast(uint16_t, (__bf16)x[j]);
  }
}

__global__ __launch_bounds__(kThreads) void widen_kernel(const float* x, double* y, int64_t n) {
  const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (i < n) y[i] = double(x[i]);
}

__global__ __launch_bounds__(kThreads) void narrow_kernel(const double* x, float* y, int64_t n) {
  const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (i < n) y[i] = float(x[i]);
}

}  // namespace

hipError_t launch_widen_f64(const float* x, double* y, int64_t n, hipStream_t stream) {
  hipLaunchKernelGGL(widen_kernel, dim3(unsigned((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, stream, x, y, n);
  return hipGetLastError();
}

hipError_t launch_narrow_f32(const double* x, float* y, int64_t n, hipStream_t stream) {
  hipLaunchKernelGGL(narrow_kernel, dim3(unsigned((n + kThreads - 1) / kThreads)), dim3(kThreads), 0, stream, x, y, n);
  return hipGetLastError();
}

hipError_t launch_cast_bf16(const float* x, uint16_t* y, int64_t n, hipStream_t stream) {
  const int64_t threads = (n + 7) / 8;
  hipLaunchKernelGGL(cast_bf16_kernel, dim3(unsigned((threads + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                     stream, x, y, n);
  return hipGetLastError();
}

}  // namespace unstep
