// Windowed block-causal attention of a chunk's queries over the retained cache rows
// (paper Sections 3.1 and 3.3; Appendix A.3).  Every query of the chunk attends to
// every retained key (sinks, window, the chunk itself); the retained keys are up to
// UNSTEP_MAX_SEGMENTS runs of consecutive cache rows, so a ring that wraps is read in
// place: the tile loader maps each logical key index to its physical row.
//
// Work-group: 4 waves x 32 queries = 128 queries of one (batch, head), optionally one
// of `splits` contiguous key ranges.  Per 64-key tile:
//   S^T = K_tile * Q^T   (v_mfma_f32_32x32x16_bf16; keys on the M side, queries on N),
// so each lane owns one query column and 32 of the tile's keys (the partner lane
// l^32 owns the other 32): row max and row sum are in-lane plus one exchange.
//   O^T += V^T * P^T     (same MFMA; P^T comes straight from the S^T registers)
// The MFMA contracts over 16 "k" slots per lane pair; the keys behind those slots are
// permuted to match where the S^T accumulator left them, and V^T is read from LDS with
// the same permutation.  Softmax runs in fp32 with base-2 exponentials of
// (s - max) * scale * log2(e); the running output is rescaled when the max grows.
//
// With splits > 1 each work-group writes its normalised partial output and its
// (max, sum) to the workspace and attn_combine merges them by log-sum-exp.
#include <hip/hip_runtime.h>

#include <climits>

#include "kernels.hpp"

namespace unstep {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kQPerWave = 32;
constexpr int kBlockQ = kWaves * kQPerWave;   // 128 queries per work-group
constexpr int kBlockK = 64;                   // keys per tile
constexpr int kKStride = kHeadDim + 8;        // LDS row of K (bf16), padded
constexpr int kVStride = kBlockK + 4;         // LDS row of V^T (bf16), padded
constexpr float kLog2e = 1.4426950408889634f;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

struct Smem {
  uint16_t k[kBlockK * kKStride];
  uint16_t vt[kHeadDim * kVStride];
};

__device__ __forceinline__ int32_t key_row(const AttnArgs& a, int32_t key) {
  int32_t l0 = a.seg_l0[0], r0 = a.seg_row0[0];
#pragma unroll
  for (int s = 1; s < UNSTEP_MAX_SEGMENTS; ++s)
    if (key >= a.seg_l0[s]) { l0 = a.seg_l0[s]; r0 = a.seg_row0[s]; }
  return r0 + (key - l0);
}

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8_t, u); }

__global__ __launch_bounds__(kThreads, 2) void window_attn_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(16))) Smem sm;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int half = lane >> 5;
  const int col = lane & 31;

  const int32_t h = blockIdx.y;
  const int32_t b = blockIdx.z / a.splits;
  const int32_t split = blockIdx.z % a.splits;
  const int32_t qi = blockIdx.x * kBlockQ + wave * kQPerWave + col;
  const int32_t qc = qi < a.N ? qi : a.N - 1;

  // key range of this split, in whole tiles
  const int32_t tiles = (a.n_keys + kBlockK - 1) / kBlockK;
  const int32_t tiles_per = (tiles + a.splits - 1) / a.splits;
  const int32_t k_begin = split * tiles_per * kBlockK;
  const int32_t k_end = min(a.n_keys, (split + 1) * tiles_per * kBlockK);

  // Q^T fragments: for d-step s, this lane holds q[qc][16 s + 8 half .. +8]
  bf16x8_t qf[8];
  {
    const uint16_t* qp = a.q + ((int64_t(b) * a.N + qc) * a.H + h) * kHeadDim + 8 * half;
#pragma unroll
    for (int s = 0; s < 8; ++s) qf[s] = as_bf16x8(*reinterpret_cast<const uint4*>(qp + 16 * s));
  }

  const int64_t bh = (int64_t(b) * a.H + h) * a.slots;
  const uint16_t* kbase = a.k_cache + bh * kHeadDim;
  const uint16_t* vbase = a.v_cache + bh * kHeadDim;
  const float c2 = a.scale * kLog2e;

  f32x16_t o[4];
#pragma unroll
  for (int d = 0; d < 4; ++d)
#pragma unroll
    for (int i = 0; i < 16; ++i) o[d][i] = 0.f;
  float m_run = -INFINITY;
  float l_run = 0.f;

  for (int32_t kt0 = k_begin; kt0 < k_end; kt0 += kBlockK) {
    __syncthreads();
    // ---- stage K (row-major) and V^T into LDS
#pragma unroll
    for (int j = 0; j < (kBlockK * kHeadDim / 8) / kThreads; ++j) {
      const int chunk = tid + kThreads * j;
      const int row = chunk >> 4;
      const int piece = chunk & 15;
      const int32_t key = kt0 + row;
      uint4 kx = make_uint4(0, 0, 0, 0), vx = make_uint4(0, 0, 0, 0);
      if (key < k_end) {
        const int64_t off = int64_t(key_row(a, key)) * kHeadDim + piece * 8;
        kx = *reinterpret_cast<const uint4*>(kbase + off);
        vx = *reinterpret_cast<const uint4*>(vbase + off);
      }
      *reinterpret_cast<uint4*>(&sm.k[row * kKStride + piece * 8]) = kx;
      const uint32_t w[4] = {vx.x, vx.y, vx.z, vx.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        sm.vt[(piece * 8 + 2 * e) * kVStride + row] = uint16_t(w[e] & 0xffffu);
        sm.vt[(piece * 8 + 2 * e + 1) * kVStride + row] = uint16_t(w[e] >> 16);
      }
    }
    __syncthreads();

    // ---- S^T = K * Q^T for two 32-key blocks
    f32x16_t s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int i = 0; i < 16; ++i) s[kb][i] = 0.f;
#pragma unroll
      for (int st = 0; st < 8; ++st) {
        const bf16x8_t kf = as_bf16x8(
            *reinterpret_cast<const uint4*>(&sm.k[(kb * 32 + col) * kKStride + 16 * st + 8 * half]));
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[st], s[kb], 0, 0, 0);
      }
    }

    // ---- mask keys past the range (last tile only)
    if (kt0 + kBlockK > k_end) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int32_t key = kt0 + kb * 32 + 8 * (i >> 2) + 4 * half + (i & 3);
          if (key >= k_end) s[kb][i] = -INFINITY;
        }
    }

    // ---- online softmax (this lane: one query, 32 keys; partner lane: the other 32)
    float mx = s[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[kb][i]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx);
    const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * c2);
    const float moff = m_new * c2;
    float psum = 0.f;
    bf16x8_t pf[4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[kb][i], c2, -moff));
        psum += p;
        pf[kb * 2 + (i >> 3)][i & 7] = (__bf16)p;
      }
    l_run = l_run * alpha + psum;
    m_run = m_new;
#pragma unroll
    for (int d = 0; d < 4; ++d)
#pragma unroll
      for (int i = 0; i < 16; ++i) o[d][i] *= alpha;

    // ---- O^T += V^T * P^T, four 16-key steps
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        const uint16_t* vp = &sm.vt[(d * 32 + col) * kVStride + 16 * t + 4 * half];
        const uint2 lo = *reinterpret_cast<const uint2*>(vp);
        const uint2 hi = *reinterpret_cast<const uint2*>(vp + 8);
        const bf16x8_t vf = as_bf16x8(make_uint4(lo.x, lo.y, hi.x, hi.y));
        o[d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[t], o[d], 0, 0, 0);
      }
    }
  }

  // ---- epilogue
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (a.splits == 1) {
    if (qi < a.N) {
      const float inv = 1.f / l_tot;
      uint16_t* op = a.out + ((int64_t(b) * a.N + qi) * a.H + h) * kHeadDim + 4 * half;
#pragma unroll
      for (int d = 0; d < 4; ++d)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
          bf16x4_t r;
#pragma unroll
          for (int e = 0; e < 4; ++e) r[e] = (__bf16)(o[d][4 * g + e] * inv);
          *reinterpret_cast<bf16x4_t*>(op + d * 32 + 8 * g) = r;
        }
      if (a.lse && half == 0) a.lse[(int64_t(b) * a.H + h) * a.N + qi] = m_run * a.scale + logf(l_tot);
    }
  } else {
    if (qi < a.N) {
      const int64_t row = ((int64_t(split) * a.B + b) * a.H + h) * a.N + qi;
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      float* op = a.part_o + row * kHeadDim + 4 * half;
#pragma unroll
      for (int d = 0; d < 4; ++d)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float4 r = make_float4(o[d][4 * g] * inv, o[d][4 * g + 1] * inv, o[d][4 * g + 2] * inv,
                                 o[d][4 * g + 3] * inv);
          *reinterpret_cast<float4*>(op + d * 32 + 8 * g) = r;
        }
      if (half == 0) {
        a.part_ml[row * 2] = m_run;
        a.part_ml[row * 2 + 1] = l_tot;
      }
    }
  }
}

// Merge the splits' partial results: out = sum_s w_s o_s / sum_s w_s with
// w_s = l_s * 2^((m_s - M) * scale * log2e), M = max_s m_s.  One thread per 4 outputs.
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnArgs a) {
  const int64_t rows = int64_t(a.B) * a.H * a.N;
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  if (idx >= rows * (kHeadDim / 4)) return;
  const int64_t row = idx / (kHeadDim / 4);        // (b, h, n)
  const int part = int(idx % (kHeadDim / 4));
  const float c2 = a.scale * kLog2e;
  float M = -INFINITY;
  for (int s = 0; s < a.splits; ++s) {
    const float l = a.part_ml[(s * rows + row) * 2 + 1];
    if (l > 0.f) M = fmaxf(M, a.part_ml[(s * rows + row) * 2]);
  }
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float wsum = 0.f;
  for (int s = 0; s < a.splits; ++s) {
    const float m = a.part_ml[(s * rows + row) * 2];
    const float l = a.part_ml[(s * rows + row) * 2 + 1];
    if (!(l > 0.f)) continue;
    const float w = l * __builtin_amdgcn_exp2f((m - M) * c2);
    const float4 v = *reinterpret_cast<const float4*>(a.part_o + (s * rows + row) * kHeadDim + part * 4);
    acc.x += w * v.x; acc.y += w * v.y; acc.z += w * v.z; acc.w += w * v.w;
    wsum += w;
  }
  const float inv = 1.f / wsum;
  const int64_t n = row % a.N;
  const int64_t bh = row / a.N;
  const int64_t hh = bh % a.H, bb = bh / a.H;
  typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
  bf16x4_t r;
  r[0] = (__bf16)(acc.x * inv);
  r[1] = (__bf16)(acc.y * inv);
  r[2] = (__bf16)(acc.z * inv);
  r[3] = (__bf16)(acc.w * inv);
  *reinterpret_cast<bf16x4_t*>(a.out + ((bb * a.N + n) * a.H + hh) * kHeadDim + part * 4) = r;
  if (a.lse && part == 0) a.lse[row] = M * a.scale + logf(wsum);
}

}  // namespace

int32_t attn_choose_splits(int32_t B, int32_t H, int32_t N, int32_t n_keys) {
  // Estimated time of s splits: rounds of resident work-groups (256 compute units x 2)
  // times the key tiles each work-group walks, plus the combine's traffic (partials
  // written and read back, fp32) at a sustained 5 TB/s.  A split keeps >= 4 tiles.
  constexpr int64_t kSlots = 256 * 2;
  constexpr double kTileUs = 2.0;             // one 128-query x 64-key tile per work-group
  constexpr double kBytesPerUs = 5.0e6;
  const int64_t groups = int64_t(B) * H * ((N + kBlockQ - 1) / kBlockQ);
  const int32_t tiles = (n_keys + kBlockK - 1) / kBlockK;
  auto cost = [&](int32_t s) {
    const int64_t rounds = (groups * s + kSlots - 1) / kSlots;
    const double walk = double(rounds) * double((tiles + s - 1) / s) * kTileUs;
    const double comb = s > 1 ? double(s) * B * H * N * (kHeadDim + 2) * 4.0 * 2.0 / kBytesPerUs : 0.0;
    return walk + comb;
  };
  int32_t best = 1;
  double best_cost = cost(1);
  for (int32_t s = 2; s <= 8 && tiles / s >= 4; ++s) {
    const double c = cost(s);
    if (c < best_cost) {
      best = s;
      best_cost = c;
    }
  }
  return best;
}

size_t attn_workspace_bytes(int32_t B, int32_t H, int32_t N, int32_t splits) {
  if (splits <= 1) return 0;
  const size_t rows = size_t(splits) * B * H * N;
  return rows * kHeadDim * sizeof(float) + rows * 2 * sizeof(float);
}

hipError_t launch_window_attn(const AttnArgs& a, hipStream_t stream) {
  dim3 grid(unsigned((a.N + kBlockQ - 1) / kBlockQ), unsigned(a.H), unsigned(a.B * a.splits));
  hipLaunchKernelGGL(window_attn_kernel, grid, dim3(kThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.splits == 1) return e;
  const int64_t work = int64_t(a.B) * a.H * a.N * (kHeadDim / 4);
  hipLaunchKernelGGL(attn_combine_kernel, dim3(unsigned((work + 255) / 256)), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace unstep
