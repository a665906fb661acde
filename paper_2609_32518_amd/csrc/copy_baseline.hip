// Bandwidth reference of the fused RoPE + append pass: a plain copy of three buffers into
// three others in one launch, with the pass's access pattern (one thread per 16 bytes of each
// buffer, 256 threads per work-group, non-temporal stores).  The append pass moves the same
// rows plus the rotary tables and does its arithmetic on the way; timing both over the same
// sizes says how close the pass gets to what a copy of its bytes reaches in one launch.
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace unstep {
namespace {

constexpr int kThreads = 256;

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__global__ __launch_bounds__(kThreads) void copy3_kernel(const u32x4_t* a, const u32x4_t* b, const u32x4_t* c,
                                                          u32x4_t* x, u32x4_t* y, u32x4_t* z, int64_t n16) {
  const int64_t i = int64_t(blockIdx.x) * kThreads + threadIdx.x;
  if (i >= n16) return;
  const u32x4_t va = a[i], vb = b[i], vc = c[i];
  __builtin_nontemporal_store(va, x + i);
  __builtin_nontemporal_store(vb, y + i);
  __builtin_nontemporal_store(vc, z + i);
}

}  // namespace

hipError_t launch_copy3(const void* a, const void* b, const void* c, void* x, void* y, void* z, int64_t n16,
                        hipStream_t stream) {
  if (n16 <= 0) return hipSuccess;
  hipLaunchKernelGGL(copy3_kernel, dim3(unsigned((n16 + kThreads - 1) / kThreads)), dim3(kThreads), 0, stream,
                     static_cast<const u32x4_t*>(a), static_cast<const u32x4_t*>(b), static_cast<const u32x4_t*>(c),
                     static_cast<u32x4_t*>(x), static_cast<u32x4_t*>(y), static_cast<u32x4_t*>(z), n16);
  return hipGetLastError();
}

}  // namespace unstep
