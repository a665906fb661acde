// Clean-cache renoise and emit updates around one DiT evaluation (paper Section 3.4,
// Equations 1 and 3): out = a x + b y on bf16 latents, with (a, b) = (1 - sigma, sigma) for
// the renoise x_tilde = (1 - sigma) x + sigma eps and (1, -sigma) for the emit
// x_next = x_tilde - sigma v.  Bandwidth-bound: one thread per 16 bytes (8 values) of each
// input.  Arithmetic in float64 with contraction off (each product and the sum rounded to
// float64), then rounded to binary32 and to bf16, both nearest-even; the binary32 value is
// kept opaque so that the two roundings are not folded into one.
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace unstep {
namespace {

constexpr int kThreads = 256;

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ double lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ double hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float affine(double x, double y, double a, double b) {
#pragma clang fp contract(off)
  const double ax = a * x;
  const double by = b * y;
  float r = (float)(ax + by);
  asm volatile("" : "+v"(r));
  return r;
}

__global__ __launch_bounds__(kThreads) void flow_update_kernel(const uint16_t* x, const uint16_t* y, uint16_t* out,
                                                               int64_t n, double a, double b) {
  const int64_t i = (int64_t(blockIdx.x) * kThreads + threadIdx.x) * 8;
  if (i + 8 <= n) {
    const u32x4_t xv = *reinterpret_cast<const u32x4_t*>(x + i);
    const u32x4_t yv = *reinterpret_cast<const u32x4_t*>(y + i);
    u32x4_t o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      bf16x2_t p;
      p[0] = (__bf16)affine(lo(xv[e]), lo(yv[e]), a, b);
      p[1] = (__bf16)affine(hi(xv[e]), hi(yv[e]), a, b);
      o[e] = __builtin_bit_cast(uint32_t, p);
    }
    *reinterpret_cast<u32x4_t*>(out + i) = o;
  } else {
    for (int64_t j = i; j < n; ++j) {
      const double xv = __uint_as_float(uint32_t(x[j]) << 16), yv = __uint_as_float(uint32_t(y[j]) << 16);
      const __bf16 r = (__bf16)affine(xv, yv, a, b);
      out[j] = __builtin_bit_cast(uint16_t, r);
    }
  }
}

}  // namespace

hipError_t launch_flow_update(const uint16_t* x, const uint16_t* y, uint16_t* out, int64_t n, double a, double b,
                              hipStream_t stream) {
  const int64_t threads = (n + 7) / 8;
  hipLaunchKernelGGL(flow_update_kernel, dim3(unsigned((threads + kThreads - 1) / kThreads)), dim3(kThreads), 0,
                     stream, x, y, out, n, a, b);
  return hipGetLastError();
}

}  // namespace unstep
