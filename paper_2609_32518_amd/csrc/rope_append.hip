// Fused rotary embedding of the chunk's queries and keys plus the K/V cache write
// (paper Section 3.1 and Appendix A.5): one bandwidth-bound pass over q, k, v.
//
// Each thread owns 16 bytes (8 bf16 = 4 coordinate pairs) of one (token, head) row of
// q, k and v.  It loads them with the token's cos/sin for those 4 pairs, rotates q and
// k in fp32 and writes q_rot, the rotated key and the value into the cache row of its
// token: the chunk frame's slot (sink slot f, or ring slot S + (f - S) mod R) times T
// plus the token's index in the frame.  Consecutive threads cover consecutive 16-byte
// pieces of a row, then consecutive heads, then consecutive tokens, so the q/k/v reads
// and the q_rot writes stream contiguously and each cache row is written whole.
//
// Rounding: each product and the sum/difference is a separate binary32 operation
// rounded to nearest-even (floating-point contraction is disabled in this function),
// and the result is rounded to bf16 nearest-even by v_cvt_pk_bf16_f32.
//
// The three outputs are written with non-temporal stores: the pass streams ~90 MB per
// full-frame chunk and nothing re-reads the written lines from this CU's caches, so
// streaming them out keeps the L2 for the inputs (~5.2 TB/s instead of ~4.6 TB/s).
#include <hip/hip_runtime.h>

#include "kernels.hpp"
#include "seg_table.hpp"

namespace unstep {
namespace {

constexpr int kThreads = 256;
constexpr int kPieces = kHeadDim / 8;   // 16-byte pieces per head row

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t rotate_pair(uint32_t w, float c, float s) {
#pragma clang fp contract(off)
  const float xe = __uint_as_float(w << 16);
  const float xo = __uint_as_float(w & 0xffff0000u);
  const float a = xe * c;
  const float b = xo * s;
  const float d = xe * s;
  const float e = xo * c;
  const float ye = a - b;
  const float yo = d + e;
  bf16x2_t r;
  r[0] = (__bf16)ye;
  r[1] = (__bf16)yo;
  return __builtin_bit_cast(uint32_t, r);
}

__device__ __forceinline__ u32x4_t rotate8(u32x4_t x, f32x4_t c, f32x4_t s) {
  return u32x4_t{rotate_pair(x.x, c.x, s.x), rotate_pair(x.y, c.y, s.y), rotate_pair(x.z, c.z, s.z),
                 rotate_pair(x.w, c.w, s.w)};
}

// kWithQ: also rotate the queries into q_rot (false: keys and values only, e.g. cache
// prefill), as a separate instantiation so that neither carries the other's branch.
template <bool kWithQ>
__global__ __launch_bounds__(kThreads) void rope_append_kernel(RopeAppendArgs a) {
  const int32_t units = a.T * a.H * kPieces;           // per (batch, frame)
  const int32_t u = blockIdx.x * kThreads + threadIdx.x;
  if (u >= units) return;
  const int32_t piece = u % kPieces;
  const int32_t r = u / kPieces;
  const int32_t h = r % a.H;
  const int32_t t = r / a.H;
  const int32_t fi = blockIdx.y;                         // frame within the chunk
  const int32_t b = blockIdx.z;
  const int32_t f = a.f0 + fi;
  const int32_t slot = frame_slot(f, a.S, a.R);
  const int64_t n = int64_t(fi) * a.T + t;
  const int64_t N = int64_t(a.C) * a.T;

  const int64_t src = (int64_t(b) * N + n) * a.tok_stride + int64_t(h) * a.head_stride + piece * 8;
  const u32x4_t kx = *reinterpret_cast<const u32x4_t*>(a.k + src);
  const u32x4_t vx = *reinterpret_cast<const u32x4_t*>(a.v + src);
  const f32x4_t cs = *reinterpret_cast<const f32x4_t*>(a.cos_t + n * (kHeadDim / 2) + piece * 4);
  const f32x4_t sn = *reinterpret_cast<const f32x4_t*>(a.sin_t + n * (kHeadDim / 2) + piece * 4);
  u32x4_t qx;
  if (kWithQ) qx = *reinterpret_cast<const u32x4_t*>(a.q + src);

  const int64_t dst = ((int64_t(b) * a.H + h) * a.slots + int64_t(slot) * a.T + t) * kHeadDim + piece * 8;
  __builtin_nontemporal_store(rotate8(kx, cs, sn), reinterpret_cast<u32x4_t*>(a.k_cache + dst));
  __builtin_nontemporal_store(vx, reinterpret_cast<u32x4_t*>(a.v_cache + dst));
  if (kWithQ) {
    const int64_t qd = ((int64_t(b) * N + n) * a.H + h) * kHeadDim + piece * 8;
    __builtin_nontemporal_store(rotate8(qx, cs, sn), reinterpret_cast<u32x4_t*>(a.q_rot + qd));
  }
}

// ---- variant with RMS normalisation of q and k (Appendix A.5: the model normalises each
// query and new key over the token's H*128 channels, with learned per-channel weights,
// before splitting it into heads and rotating).
//
// One wave per token: lane l owns the 16-byte pieces l, l + 64, ... of the token's H*16
// pieces (so each load instruction reads 1 KB of consecutive channels).  The statistic
// sum_i x_i^2 is accumulated in fp64 (each bf16 square is exact) and reduced over the wave;
// r = 1 / sqrt(ss / (H*128) + eps) in fp64; each channel becomes bf16(f32((x r) w)) and
// enters the same rotation as above.  V is copied unchanged.
// pieces per lane: 3 covers up to 12 heads (the model's 1536 channels), 8 up to kNormMaxHeads
constexpr int kNormPiecesSmall = 3;
constexpr int kNormPiecesLarge = kNormMaxHeads * kPieces / 64;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

template <int kPer>
__device__ __forceinline__ double sum_sq(const u32x4_t (&x)[kPer], int n) {
  double s = 0.0;
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    if (i >= n) break;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const double lo = bf16_lo(x[i][e]), hi = bf16_hi(x[i][e]);
      s += lo * lo;
      s += hi * hi;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  return s;
}

// bf16(f32((x r) w)) for the 8 channels of one piece.  The binary32 value is kept opaque
// to the optimiser: folded into one double-to-bf16 conversion, a binary32 result that is
// exactly halfway between two bf16 values would round as the unrounded double instead of
// to even.
__device__ __forceinline__ u32x4_t normalise8(u32x4_t x, u32x4_t w, double r) {
  u32x4_t y;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float lo = (float)(((double)bf16_lo(x[e]) * r) * (double)bf16_lo(w[e]));
    float hi = (float)(((double)bf16_hi(x[e]) * r) * (double)bf16_hi(w[e]));
    asm volatile("" : "+v"(lo), "+v"(hi));
    bf16x2_t p;
    p[0] = (__bf16)lo;
    p[1] = (__bf16)hi;
    y[e] = __builtin_bit_cast(uint32_t, p);
  }
  return y;
}

template <bool kWithQ, int kPer>
__global__ __launch_bounds__(kThreads) void rope_norm_append_kernel(RopeAppendArgs a) {
  const int32_t N = a.C * a.T;
  const int32_t n = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);   // token of the chunk
  if (n >= N) return;                                                     // whole wave
  const int lane = threadIdx.x & 63;
  const int b = blockIdx.y;
  const int32_t fi = n / a.T, t = n - fi * a.T;
  const int32_t f = a.f0 + fi;
  const int32_t slot = frame_slot(f, a.S, a.R);
  const int32_t pieces = a.H * kPieces;
  const int np = (pieces - lane + 63) / 64;                               // this lane's pieces

  u32x4_t kx[kPer], vx[kPer], qx[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    if (i >= np) break;
    const int32_t p = lane + 64 * i;
    const int64_t src = (int64_t(b) * N + n) * a.tok_stride + int64_t(p / kPieces) * a.head_stride + (p % kPieces) * 8;
    kx[i] = *reinterpret_cast<const u32x4_t*>(a.k + src);
    vx[i] = *reinterpret_cast<const u32x4_t*>(a.v + src);
    if (kWithQ) qx[i] = *reinterpret_cast<const u32x4_t*>(a.q + src);
  }
  const double inv_c = 1.0 / double(a.H * kHeadDim);
  const double rk = 1.0 / sqrt(sum_sq(kx, np) * inv_c + a.eps);
  double rq = 0.0;
  if (kWithQ) rq = 1.0 / sqrt(sum_sq(qx, np) * inv_c + a.eps);

#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    if (i >= np) break;
    const int32_t p = lane + 64 * i;
    const int32_t h = p / kPieces, piece = p % kPieces;
    const f32x4_t cs = *reinterpret_cast<const f32x4_t*>(a.cos_t + int64_t(n) * (kHeadDim / 2) + piece * 4);
    const f32x4_t sn = *reinterpret_cast<const f32x4_t*>(a.sin_t + int64_t(n) * (kHeadDim / 2) + piece * 4);
    const u32x4_t wk = *reinterpret_cast<const u32x4_t*>(a.wk + p * 8);
    const int64_t dst = ((int64_t(b) * a.H + h) * a.slots + int64_t(slot) * a.T + t) * kHeadDim + piece * 8;
    __builtin_nontemporal_store(rotate8(normalise8(kx[i], wk, rk), cs, sn),
                                reinterpret_cast<u32x4_t*>(a.k_cache + dst));
    __builtin_nontemporal_store(vx[i], reinterpret_cast<u32x4_t*>(a.v_cache + dst));
    if (kWithQ) {
      const u32x4_t wq = *reinterpret_cast<const u32x4_t*>(a.wq + p * 8);
      const int64_t qd = (int64_t(b) * N + n) * int64_t(pieces) * 8 + p * 8;
      __builtin_nontemporal_store(rotate8(normalise8(qx[i], wq, rq), cs, sn),
                                  reinterpret_cast<u32x4_t*>(a.q_rot + qd));
    }
  }
}

}  // namespace

hipError_t launch_rope_append(const RopeAppendArgs& a, hipStream_t stream) {
  if (a.wk) {
    const int32_t N = a.C * a.T;
    dim3 grid(unsigned((N + kThreads / 64 - 1) / (kThreads / 64)), unsigned(a.B));
    const bool small = a.H * kPieces <= 64 * kNormPiecesSmall;
    if (a.q && small)
      hipLaunchKernelGGL((rope_norm_append_kernel<true, kNormPiecesSmall>), grid, dim3(kThreads), 0, stream, a);
    else if (a.q)
      hipLaunchKernelGGL((rope_norm_append_kernel<true, kNormPiecesLarge>), grid, dim3(kThreads), 0, stream, a);
    else if (small)
      hipLaunchKernelGGL((rope_norm_append_kernel<false, kNormPiecesSmall>), grid, dim3(kThreads), 0, stream, a);
    else
      hipLaunchKernelGGL((rope_norm_append_kernel<false, kNormPiecesLarge>), grid, dim3(kThreads), 0, stream, a);
    return hipGetLastError();
  }
  const int64_t units = int64_t(a.T) * a.H * kPieces;
  dim3 grid(unsigned((units + kThreads - 1) / kThreads), unsigned(a.C), unsigned(a.B));
  if (a.q)
    hipLaunchKernelGGL(rope_append_kernel<true>, grid, dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(rope_append_kernel<false>, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace unstep
