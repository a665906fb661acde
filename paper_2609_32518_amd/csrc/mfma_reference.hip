// Compute reference of the attention and projection kernels: the rate at which this chip's MFMA
// units run v_mfma_f32_32x32x16_bf16 on bf16 data like the method's, with nothing else to do.
// The chip is power-limited: its clock, and so its MFMA rate, depends on how much the operand
// bits toggle, so a loop on constant operands overstates what a kernel on random data can
// reach.  Launched in the shape of those kernels (one work-group of 8 waves per compute unit,
// the same number of work-groups, one or two multiplying waves per SIMD), timing it beside them
// says how much of their time is the MFMA work itself.
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace unstep {
namespace {

constexpr int kThreads = 512;                 // 8 waves, two per SIMD
constexpr int kSets = 8;                      // operand register sets per wave
constexpr int kBlock = 32;                    // MFMAs between work-group barriers

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// One block of 32 MFMAs on 8 accumulators, operand sets rotated by `s` (a compile-time value).
template <int s>
__device__ __forceinline__ void block(f32x16_t (&acc)[8], const bf16x8_t (&a)[kSets], const bf16x8_t (&b)[kSets]) {
#pragma unroll
  for (int j = 0; j < kBlock; ++j)
    acc[j & 7] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(j + s) & 7], b[((j >> 3) + s) & 7], acc[j & 7], 0, 0, 0);
}

// Wave w multiplies when w < 4 * waves_per_simd (waves w and w + 4 share a SIMD).  Each lane loads
// its 16 operand vectors (256 bytes) once; `blocks` blocks of 32 MFMAs follow, a barrier after
// each (every wave takes part in the barriers); the lane-0 sums of the accumulators are written
// to sum[8 g + w] so that no MFMA can be dropped.
__global__ __launch_bounds__(kThreads, 1) void mfma_reference_kernel(const u32x4_t* src, float* sum, int32_t waves_per_simd,
                                                                      int32_t blocks) {
  __shared__ float lds[32 * 1024];          // 128 KB, as the attention kernel's ring: one work-group per CU
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const bool mult = wave < 4 * waves_per_simd;
  const int64_t base = (int64_t(blockIdx.x) * kThreads + threadIdx.x) * (2 * kSets);
  bf16x8_t a[kSets], b[kSets];
#pragma unroll
  for (int i = 0; i < kSets; ++i) {
    a[i] = __builtin_bit_cast(bf16x8_t, src[base + i]);
    b[i] = __builtin_bit_cast(bf16x8_t, src[base + kSets + i]);
  }
  f32x16_t acc[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) acc[i] = f32x16_t{};
  int32_t left = blocks;
  for (; left >= kSets; left -= kSets) {
    if (mult) block<0>(acc, a, b);
    __syncthreads();
    if (mult) block<1>(acc, a, b);
    __syncthreads();
    if (mult) block<2>(acc, a, b);
    __syncthreads();
    if (mult) block<3>(acc, a, b);
    __syncthreads();
    if (mult) block<4>(acc, a, b);
    __syncthreads();
    if (mult) block<5>(acc, a, b);
    __syncthreads();
    if (mult) block<6>(acc, a, b);
    __syncthreads();
    if (mult) block<7>(acc, a, b);
    __syncthreads();
  }
  // the remaining 0..7 blocks
  if (left > 0) { if (mult) block<0>(acc, a, b); __syncthreads(); }
  if (left > 1) { if (mult) block<1>(acc, a, b); __syncthreads(); }
  if (left > 2) { if (mult) block<2>(acc, a, b); __syncthreads(); }
  if (left > 3) { if (mult) block<3>(acc, a, b); __syncthreads(); }
  if (left > 4) { if (mult) block<4>(acc, a, b); __syncthreads(); }
  if (left > 5) { if (mult) block<5>(acc, a, b); __syncthreads(); }
  if (left > 6) { if (mult) block<6>(acc, a, b); __syncthreads(); }
  float t = 0.f;
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) t += acc[i][e];
  if ((threadIdx.x & 63) == 0) lds[wave] = t;
  __syncthreads();
  if (threadIdx.x < 8) sum[int64_t(blockIdx.x) * 8 + threadIdx.x] = lds[threadIdx.x];
}

}  // namespace

hipError_t launch_mfma_reference(const void* src, float* sum, int32_t groups, int32_t waves_per_simd,
                                 int32_t mfmas, hipStream_t stream) {
  hipLaunchKernelGGL(mfma_reference_kernel, dim3(unsigned(groups)), dim3(kThreads), 0, stream,
                     static_cast<const u32x4_t*>(src), sum, waves_per_simd, mfmas / kBlock);
  return hipGetLastError();
}

}  // namespace unstep
