// The projection after attention, y = x W^T + b (paper Section 3.5 and Appendix A.4: the
// truncated V/O weights stay dense, so this is a plain bf16 GEMM of the attention output with
// the output weight), as hand-written MFMA kernels for gfx950.
//
// x bf16 [M, K], W bf16 [N, K] (the nn.Linear layout), bias bf16 [N] or none, y bf16 [M, N];
// float32 accumulation, the bias added in float32, one rounding to bf16 (nearest even).  Both
// kernels use v_mfma_f32_32x32x16_bf16 with W rows on the MFMA's M side and x rows on its N
// side, so each lane finishes with one row of y and runs of 4 consecutive columns (8-byte
// stores).  Both operands are k-contiguous in memory and in LDS: a 64-wide k step of a tile is
// rows of 128 bytes whose eight 16-byte chunks are XOR-swizzled by (row >> 1) & 7, so that the
// fragment reads (32 rows at one chunk) hit distinct banks.  Rows past M or N read the last row
// and are not stored.
//
// linear_kernel (any K, N multiple of 8): 4 waves, a 128 x 128 tile of y^T, two work-groups per
// compute unit, wave w owning a 64 x 64 quarter as 2 x 2 blocks.  The k steps are double
// buffered: the global loads of step s + 1 are in flight in registers while step s is
// multiplied, then written to the other LDS buffer before the step's one barrier.  Chunks past
// K read as zeros.
//
// linear_kernel_big (K a multiple of 64, the model's case): below.
#include <hip/hip_runtime.h>

#include "kernels.hpp"

namespace unstep {
namespace {

constexpr int kThreads = 256;
constexpr int kBM = 128;                 // x rows (columns of y^T) per work-group
constexpr int kBN = 128;                 // W rows (columns of y) per work-group
constexpr int kBK = 64;                  // k per step
constexpr int kRowBytes = kBK * 2;       // one tile row in LDS
constexpr int kTileBytes = kBN * kRowBytes;
constexpr int kChunks = kRowBytes / 16;  // 16-byte chunks per tile row
constexpr int kLoads = kTileBytes / 16 / kThreads;   // chunks per thread per operand per step
constexpr int kXcds = 8;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) u32x4_t lds_u32x4_t;

__device__ __forceinline__ int swz(int row) { return (row >> 1) & 7; }

struct LinearArgs {
  const uint16_t* x;
  const uint16_t* w;
  const uint16_t* bias;
  uint16_t* y;
  int32_t M, N, K;
  int32_t tiles_m, tiles_n;
};

// Global loads of one k step: thread t fetches chunks t + 256 j (j < kLoads) of the W tile and
// of the x tile (chunk c = row c / 8, 16-byte piece c % 8).  Returns zeros past K.
__device__ __forceinline__ void load_step(const LinearArgs& a, int32_t n0, int32_t m0, int32_t k0, int tid,
                                          u32x4_t (&wr)[kLoads], u32x4_t (&xr)[kLoads]) {
#pragma unroll
  for (int j = 0; j < kLoads; ++j) {
    const int c = tid + kThreads * j;
    const int row = c / kChunks, piece = c % kChunks;
    const int32_t k = k0 + piece * 8;
    const bool in_k = k < a.K;
    const int32_t nr = min(n0 + row, a.N - 1), mr = min(m0 + row, a.M - 1);
    const u32x4_t zero = {0u, 0u, 0u, 0u};
    wr[j] = in_k ? *reinterpret_cast<const u32x4_t*>(a.w + int64_t(nr) * a.K + k) : zero;
    xr[j] = in_k ? *reinterpret_cast<const u32x4_t*>(a.x + int64_t(mr) * a.K + k) : zero;
  }
}

__device__ __forceinline__ void store_step(uint8_t* lw, uint8_t* lx, int tid, const u32x4_t (&wr)[kLoads],
                                           const u32x4_t (&xr)[kLoads]) {
#pragma unroll
  for (int j = 0; j < kLoads; ++j) {
    const int c = tid + kThreads * j;
    const int row = c / kChunks, piece = c % kChunks;
    const int off = row * kRowBytes + ((piece ^ swz(row)) * 16);
    *reinterpret_cast<lds_u32x4_t*>(reinterpret_cast<uintptr_t>(lw + off)) = wr[j];
    *reinterpret_cast<lds_u32x4_t*>(reinterpret_cast<uintptr_t>(lx + off)) = xr[j];
  }
}

__global__ __launch_bounds__(kThreads, 2) void linear_kernel(LinearArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2][2][kTileBytes];   // [buffer][W, x]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave >> 1, wm = wave & 1;
  const int col = lane & 31, half = lane >> 5;

  // XCD-aware numbering: hardware work-group i runs on XCD i % 8; each XCD gets a contiguous
  // range of tiles, n fastest, so the work-groups of an XCD share x row blocks in its L2
  const int32_t G = gridDim.x;
  const int32_t xcd = blockIdx.x % kXcds;
  const int32_t g = xcd * (G / kXcds) + min(xcd, G % kXcds) + blockIdx.x / kXcds;
  const int32_t tn = g % a.tiles_n, tm = g / a.tiles_n;
  const int32_t n0 = tn * kBN, m0 = tm * kBM;

  // fragment read offsets within a tile: row wn*64 + nb*32 + col (W) or wm*64 + mb*32 + col (x),
  // chunk 2 kk + half; rows 32 apart share the swizzle, so nb / mb is an immediate offset
  int w_off[4], x_off[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    const int rw = wn * 64 + col, rx = wm * 64 + col;
    w_off[kk] = rw * kRowBytes + (((2 * kk + half) ^ swz(rw)) * 16);
    x_off[kk] = rx * kRowBytes + (((2 * kk + half) ^ swz(rx)) * 16);
  }

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{};

  const int32_t steps = (a.K + kBK - 1) / kBK;
  u32x4_t wr[kLoads], xr[kLoads];
  load_step(a, n0, m0, 0, tid, wr, xr);
  store_step(lds[0][0], lds[0][1], tid, wr, xr);
  __syncthreads();
  for (int32_t s = 0; s < steps; ++s) {
    const int buf = s & 1;
    if (s + 1 < steps) load_step(a, n0, m0, (s + 1) * kBK, tid, wr, xr);
    const uint8_t* lw = lds[buf][0];
    const uint8_t* lx = lds[buf][1];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      bf16x8_t fw[2], fx[2];
#pragma unroll
      for (int b = 0; b < 2; ++b) {
        fw[b] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const lds_u32x4_t*>(
                                                 reinterpret_cast<uintptr_t>(lw + w_off[kk] + b * 32 * kRowBytes)));
        fx[b] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const lds_u32x4_t*>(
                                                 reinterpret_cast<uintptr_t>(lx + x_off[kk] + b * 32 * kRowBytes)));
      }
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb)
          acc[nb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[nb], fx[mb], acc[nb][mb], 0, 0, 0);
    }
    // the other buffer was last read in step s - 1, which every wave finished before the
    // barrier that ended it; the barrier below publishes the new contents for step s + 1
    if (s + 1 < steps) store_step(lds[buf ^ 1][0], lds[buf ^ 1][1], tid, wr, xr);
    __syncthreads();
  }

  // epilogue: lane holds y[m][n .. n + 3] for m = m0 + wm*64 + mb*32 + col and the four runs
  // n = n0 + wn*64 + nb*32 + 8 g + 4 half, g = 0..3
  typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
    const int32_t m = m0 + wm * 64 + mb * 32 + col;
    if (m >= a.M) continue;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int32_t n = n0 + wn * 64 + nb * 32 + 8 * gq + 4 * half;
        if (n >= a.N) continue;      // N is a multiple of 8: a run of 4 is all in or all out
        bf16x4_t r;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float v = acc[nb][mb][4 * gq + e];
          if (a.bias) v += __uint_as_float(uint32_t(a.bias[n + e]) << 16);
          r[e] = (__bf16)v;
        }
        *reinterpret_cast<bf16x4_t*>(a.y + int64_t(m) * a.N + n) = r;
      }
  }
}

// ---- K a multiple of 64: direct-to-LDS staging, a three-stage ring, larger tiles ----------------
//
// Work-group: 8 waves, a 128 (n) x 256 (m) tile of y^T.  Waves 0-3 (one per SIMD) multiply: wave
// w owns 64 n (w / 2) x 128 m (w % 2) as 2 x 4 blocks, so a 16-wide k step reads 6 fragments for
// 8 MFMAs.  Waves 4-7 only load: a stage is the 64-wide k step of both tiles (W 128 rows + x 256
// rows of 128 bytes, 48 KB), brought straight from global memory into LDS by
// global_load_lds_dwordx4 (each loader 12 loads of 1 KB = 8 rows): lane l lands in row l / 8,
// physical chunk l % 8, so it fetches logical chunk (l % 8) ^ swz(row).  Loaders issue stage
// s + 2 while stage s is multiplied and wait for stage s + 1 before the barrier that ends the
// step, which also frees stage s's ring slot; issuing a direct-to-LDS load stalls the issuing
// wave, so keeping the loads off the multiplying waves keeps their MFMA stream going.  After the
// k loop the multiplying waves add the bias (loaded before the loop) and write the rounded tile
// into the then free ring, and all 8 waves store it in 16-byte pieces that cover whole row runs
// (each lane's own results are 8-byte pieces of 32 different rows, which stored directly made
// every store instruction touch 32 partial cache lines).
constexpr int kBigBM = 256;
constexpr int kBigStages = 3;
constexpr int kWBytes = kBN * kRowBytes;                  // 16 KB
constexpr int kXBytes = kBigBM * kRowBytes;               // 32 KB
constexpr int kStageBytes = kWBytes + kXBytes;            // 48 KB
constexpr int kLoadsPerWave = kStageBytes / 1024 / 4;     // 12
static_assert(kLoadsPerWave == 12, "vmcnt immediates assume 12 loads per wave per stage");

typedef __attribute__((address_space(1))) void global_void_t;

__device__ __forceinline__ void big_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Load j (0..11) of loader `wave` (0..3) for the stage at k0 into LDS stage address `stage`:
// loads 0-3 are W rows 32 wave + 8 j .. + 7, loads 4-11 x rows 64 wave + 8 (j - 4) .. + 7.
__device__ __forceinline__ void big_load(const LinearArgs& a, uint32_t stage, int wave, int lane, int j, int32_t n0,
                                         int32_t m0, int32_t k0) {
  const bool is_w = j < 4;
  const int row = is_w ? 32 * wave + 8 * j + (lane >> 3) : 64 * wave + 8 * (j - 4) + (lane >> 3);
  const int chunk = (lane & 7) ^ swz(row);
  // rows past N or M read the last row (finite values; those outputs are not stored)
  const int32_t r = is_w ? min(n0 + row, a.N - 1) - n0 : min(m0 + row, a.M - 1) - m0;
  const uint16_t* base = is_w ? a.w + int64_t(n0) * a.K : a.x + int64_t(m0) * a.K;
  const uint32_t off = uint32_t(r) * uint32_t(a.K) * 2u + uint32_t(k0) * 2u + uint32_t(chunk) * 16u;
  const uint32_t m0addr = stage + (is_w ? 0 : kWBytes) + (is_w ? 32 * wave + 8 * j : 64 * wave + 8 * (j - 4)) * kRowBytes;
  // `base` is computed by the scalar unit: an SGPR written by a VALU instruction would need 5 wait
  // states before this load, which the compiler does not insert ahead of inline assembly
  asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "{m0}"(m0addr) : "memory");
}

__device__ __forceinline__ void wait_loads(bool next_in_flight) {
  if (next_in_flight)
    asm volatile("s_waitcnt vmcnt(12)" ::: "memory");
  else
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// Fragment i of the 16-wide k step kk of the stage at LDS offset cur: i < 2 the W block nb = i,
// else the x block mb = i - 2 (blocks are 32 rows = 4096 bytes apart).
__device__ __forceinline__ bf16x8_t frag(const uint32_t (&w_off)[4], const uint32_t (&x_off)[4], uint32_t cur, int kk,
                                         int i) {
  const uint32_t addr = i < 2 ? w_off[kk] + cur + i * 32 * kRowBytes : x_off[kk] + cur + (i - 2) * 32 * kRowBytes;
  return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const lds_u32x4_t*>(uintptr_t(addr)));
}

constexpr int kPCThreads = 512;
// output staging after the k loop: the 256 x 128 bf16 tile in LDS rows of 272 bytes (16-byte
// aligned; consecutive rows start 4 banks apart, so the multiplying waves' 8-byte writes of 32
// rows at one column conflict at most 2-way)
constexpr int kYPitch = 272;
static_assert(kBigBM * kYPitch <= kBigStages * kStageBytes, "the y tile must fit the LDS ring");

// The multiplying waves of linear_kernel_big: the k loop over the LDS ring, then the tile, bias
// added in float32 and rounded once, written to LDS rows of kYPitch bytes.
__device__ __forceinline__ void multiply(const LinearArgs& a, uint32_t lds0, int lw, int lane, int32_t n0,
                                         int32_t m0, int32_t steps) {
  const int wn = lw >> 1, wm = lw & 1;
  const int col = lane & 31, half = lane >> 5;

  // this lane's bias values, loaded before the loop so that their latency is hidden: columns
  // n0 + wn*64 + nb*32 + 8 gq + 4 half + e (N is a multiple of 8: a run of 4 is all in or all out)
  typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
  u32x2_t bq[2][4];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb)
#pragma unroll
    for (int gq = 0; gq < 4; ++gq) {
      const int32_t n = n0 + wn * 64 + nb * 32 + 8 * gq + 4 * half;
      bq[nb][gq] = (a.bias && n < a.N) ? *reinterpret_cast<const u32x2_t*>(a.bias + n) : u32x2_t{0u, 0u};
    }

  // fragment offsets within a stage: W row wn*64 + nb*32 + col, x row wm*128 + mb*32 + col, chunk
  // 2 kk + half; rows 32 apart share the swizzle (nb, mb are immediate offsets)
  uint32_t w_off[4], x_off[4];
#pragma unroll
  for (int kk = 0; kk < 4; ++kk) {
    const int rw = wn * 64 + col, rx = wm * 128 + col;
    w_off[kk] = lds0 + rw * kRowBytes + (((2 * kk + half) ^ swz(rw)) * 16);
    x_off[kk] = lds0 + kWBytes + rx * kRowBytes + (((2 * kk + half) ^ swz(rx)) * 16);
  }

  f32x16_t acc[2][4];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16_t{};

  big_barrier();                               // stage 0 has landed
  for (int32_t s = 0; s < steps; ++s) {
    const uint32_t cur = uint32_t((s % kBigStages) * kStageBytes);
    // fragments of a 16-wide k step kk: [0, 1] = W blocks nb, [2..5] = x blocks mb; the reads of
    // step kk + 1 are issued between the MFMAs of step kk (one after each of the first six), so
    // only the first step of a stage waits for LDS; the schedule is pinned
    bf16x8_t fr[2][6];
#pragma unroll
    for (int i = 0; i < 6; ++i) fr[0][i] = frag(w_off, x_off, cur, 0, i);
    __builtin_amdgcn_sched_group_barrier(0x100, 6, 0);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int nb = i >> 2, mb = i & 3;
        acc[nb][mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fr[kk & 1][nb], fr[kk & 1][2 + mb], acc[nb][mb], 0, 0, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if (kk < 3 && i < 6) {
          fr[(kk + 1) & 1][i] = frag(w_off, x_off, cur, kk + 1, i);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
      }
    big_barrier();                             // stage s read; stage s + 1 has landed
  }

  // lane holds y[m][n .. n + 3] for tile row wm*128 + mb*32 + col and tile columns
  // wn*64 + nb*32 + 8 gq + 4 half; rows past M or N hold finite values and are not stored
  typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) {
    const int r = wm * 128 + mb * 32 + col;
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int cn = wn * 64 + nb * 32 + 8 * gq + 4 * half;
        bf16x4_t v;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const uint32_t b2 = bq[nb][gq][e >> 1];
          const float bias = __uint_as_float((e & 1) ? (b2 & 0xffff0000u) : (b2 << 16));
          v[e] = (__bf16)(acc[nb][mb][4 * gq + e] + bias);
        }
        *reinterpret_cast<__attribute__((address_space(3))) bf16x4_t*>(uintptr_t(lds0 + uint32_t(r * kYPitch + cn * 2))) = v;
      }
  }
}


__global__ __launch_bounds__(kPCThreads, 1) void linear_kernel_big(LinearArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds[kBigStages * kStageBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const bool loader = wave >= 4;
  const int lw = wave & 3;                     // loader index or multiplier index

  const int32_t G = gridDim.x;
  const int32_t xcd = blockIdx.x % kXcds;
  const int32_t g = xcd * (G / kXcds) + min(xcd, G % kXcds) + blockIdx.x / kXcds;
  const int32_t tn = g % a.tiles_n, tm = g / a.tiles_n;
  const int32_t n0 = tn * kBN, m0 = tm * kBigBM;
  const uint32_t lds0 = uint32_t(uintptr_t((__attribute__((address_space(3))) void*)lds));
  const int32_t steps = a.K / kBK;

  if (loader) {
#pragma unroll
    for (int j = 0; j < kLoadsPerWave; ++j) big_load(a, lds0, lw, lane, j, n0, m0, 0);
    if (steps > 1)
#pragma unroll
      for (int j = 0; j < kLoadsPerWave; ++j) big_load(a, lds0 + kStageBytes, lw, lane, j, n0, m0, kBK);
    wait_loads(steps > 1);                     // stage 0
    big_barrier();
    for (int32_t s = 0; s < steps; ++s) {
      const bool more = s + 2 < steps;
      if (more) {
        const uint32_t nxt = lds0 + uint32_t(((s + 2) % kBigStages) * kStageBytes);
#pragma unroll
        for (int j = 0; j < kLoadsPerWave; ++j) big_load(a, nxt, lw, lane, j, n0, m0, (s + 2) * kBK);
      }
      if (s + 1 < steps) wait_loads(more);     // stage s + 1 (stage s + 2 may still be in flight)
      big_barrier();
    }
  } else {
    multiply(a, lds0, lw, lane, n0, m0, steps);
  }
  big_barrier();                               // the y tile is in LDS (the ring is free)

  // all 8 waves store the tile: thread t moves 16-byte piece t % 16 (columns n0 + 8 (t % 16) ..
  // + 7) of tile rows t / 16 + 32 i, so that a wave writes four whole 256-byte row runs
  const int c = tid & 15;
  const int32_t n = n0 + 8 * c;
#pragma unroll
  for (int i = 0; i < kBigBM / 32; ++i) {
    const int r = (tid >> 4) + 32 * i;
    const int32_t m = m0 + r;
    const u32x4_t v = *reinterpret_cast<const lds_u32x4_t*>(uintptr_t(lds0 + uint32_t(r * kYPitch + c * 16)));
    if (m < a.M && n < a.N) *reinterpret_cast<u32x4_t*>(a.y + int64_t(m) * a.N + n) = v;
  }
}

}  // namespace

hipError_t launch_linear(const uint16_t* x, const uint16_t* w, const uint16_t* bias, uint16_t* y, int32_t M,
                         int32_t N, int32_t K, hipStream_t stream) {
  // K a multiple of 64 (the model's 1536) with 256-row x tiles addressable by 32-bit offsets:
  // the direct-to-LDS kernel; anything else: the register-staged one
  if (K % kBK == 0 && int64_t(kBigBM) * K * 2 < (int64_t(1) << 31)) {
    LinearArgs a{x, w, bias, y, M, N, K, (M + kBigBM - 1) / kBigBM, (N + kBN - 1) / kBN};
    const int64_t tiles = int64_t(a.tiles_m) * a.tiles_n;
    hipLaunchKernelGGL(linear_kernel_big, dim3(unsigned(tiles)), dim3(kPCThreads), 0, stream, a);
    return hipGetLastError();
  }
  LinearArgs a{x, w, bias, y, M, N, K, (M + kBM - 1) / kBM, (N + kBN - 1) / kBN};
  const int64_t tiles = int64_t(a.tiles_m) * a.tiles_n;
  hipLaunchKernelGGL(linear_kernel, dim3(unsigned(tiles)), dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace unstep
