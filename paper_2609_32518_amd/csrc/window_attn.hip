// Windowed block-causal attention of a chunk's queries over the retained cache rows
// (paper Sections 3.1 and 3.3; Appendix A.3).  Every query of the chunk attends to
// every retained key (sinks, window, the chunk itself); the retained keys are up to
// UNSTEP_MAX_SEGMENTS runs of consecutive cache rows, so a ring that wraps is read in
// place: the tile loader maps each logical key index to its physical row.
//
// Work-group: 4 waves x 32 queries = one 128-query tile (two work-groups per compute
// unit, so two waves per SIMD from independent work-groups overlap one's MFMAs with the
// other's softmax).  Per 64-key tile, per wave:
//   S^T = K_tile * Q^T   (v_mfma_f32_32x32x16_bf16, keys on the M side, queries on N):
//       each lane owns one query column and 32 of the tile's keys, the partner lane
//       l^32 the other 32, so row max and row sum are in-lane plus one exchange.
//   O^T += V^T * P^T     (same MFMA): P^T comes straight from the S^T registers; the
//       MFMA's 16 contraction slots per lane pair are mapped to the keys where the S^T
//       accumulator left them, and the matching V^T fragments are read from the
//       row-major V tile with the transposing LDS read ds_read_b64_tr_b16.
// K and V tiles are double-buffered in LDS; the next tile's global loads are issued
// before the current tile's MFMAs and written to the other buffer after them (one
// barrier per tile).
// Softmax: fp32, base-2 exponentials of (s - m) * scale * log2(e) with a fixed per-row
// offset m (the max of the range's first tile), so the loop never rescales the output;
// if a row's sum exceeds 2^64 the work-group redoes its range with the exact row max
// (see window_attn_kernel).  Row sums accumulate the bf16-rounded probabilities that
// enter the PV product (v_dot2_f32_bf16).
//
// Schedule: the (query tile, key tile) units of the launch are cut into `groups` equal
// contiguous ranges, one per work-group (a balanced split keeps all compute units busy
// when the query tiles alone would leave some idle).  A query tile whose key range falls
// to several work-groups gets a normalised partial output and its (offset, row sum) from
// each, and attn_combine merges them by log-sum-exp.  Work-groups are numbered so that
// neighbouring ranges (same head, neighbouring query tiles) land on the same XCD and share
// its L2 while they stream the same keys.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>

#include "kernels.hpp"

namespace unstep {
namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kBlockK = 64;                   // keys per tile
#ifndef UNSTEP_ATTN_QB
#define UNSTEP_ATTN_QB 1
#endif
constexpr int kQB = UNSTEP_ATTN_QB;           // 32-query blocks per wave
constexpr int kQPerWave = 32 * kQB;
constexpr int kBlockQ = kWaves * kQPerWave;   // queries per work-group
constexpr int kGroupsPerCU = kQB == 1 ? 2 : 1;
constexpr int kRowBytes = kHeadDim * 2;       // one K or V row (bf16)
constexpr int kTileBytes = kBlockK * kRowBytes;
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kXcds = 8;

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) i16x4_t lds_i16x4_t;
typedef __attribute__((address_space(3))) u32x4_t lds_u32x4_t;
typedef __attribute__((address_space(1))) void global_void_t;
typedef __attribute__((address_space(3))) void lds_void_t;

// LDS: two buffers of one K tile and one V tile, rows of 256 bytes without padding, each
// its own array so that loads into one buffer are seen not to alias reads of the other.
// The sixteen 16-byte slots of row r are XOR-swizzled with swz(r), so that both read
// patterns are bank-conflict free: the b128 K reads (16 lanes = 16 consecutive rows at
// one logical slot) and the transposing V reads (per half-wave 4 consecutive rows x
// 4 consecutive slots).
struct Buffers {
  uint8_t* k;
  uint8_t* v;
};

__device__ __forceinline__ int swz(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }

// Physical cache row of a logical key index: up to four runs of consecutive rows, the
// first starting at logical index 0.
struct SegTable {
  int32_t l1, l2, l3;          // logical start of runs 1..3 (INT32_MAX when absent)
  int32_t r0, r1, r2, r3;      // physical row of each run's first key
  __device__ __forceinline__ int32_t row(int32_t key) const {
    int32_t r = r0 + key;
    r = key >= l1 ? r1 + (key - l1) : r;
    r = key >= l2 ? r2 + (key - l2) : r;
    r = key >= l3 ? r3 + (key - l3) : r;
    return r;
  }
  // Logical start of the run after the one holding key (INT32_MAX for the last run).
  __device__ __forceinline__ int32_t run_end(int32_t key) const {
    return key < l1 ? l1 : key < l2 ? l2 : key < l3 ? l3 : INT32_MAX;
  }
};

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t u) { return __builtin_bit_cast(bf16x8_t, u); }

// Transposing LDS read: within each 16-lane group, lane i receives element (i & 3) of
// the 4 x b16 rows addressed by lanes 4e + (i >> 2), e = 0..3.
__device__ __forceinline__ u32x2_t lds_read_tr(const uint8_t* p) {
  const i16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(p));
  return __builtin_bit_cast(u32x2_t, v);
}

// Everything one work-group needs while it walks its key range.
struct Walk {
  const uint8_t* kbase;        // this (batch, head)'s K rows
  const uint8_t* vbase;
  SegTable seg;
  int32_t k_begin, k_end;      // logical key range
  int wave, lane, col, half;
  int lrow;                    // loader: tile row of this lane in its first load (+4 i)
  int lpiece[4];               // loader: byte offset of this lane's logical 16-byte piece
  int koff[8];                 // K fragment byte offsets for d-steps 0..7 (row = col)
  int voff[2][4];              // V^T fragment byte offsets for (upper 8 keys, d block)
  float c2;                    // scale * log2(e)
};

// Direct-to-LDS load of one 64-key tile of K and V into buffer `buf`.  Wave w loads tile
// rows 16 w .. 16 w + 15 in four 1 KB instructions; lane l of instruction i lands in
// row 16 w + 4 i + (l >> 4), physical slot l & 15, and so fetches logical piece
// (l & 15) ^ swz(row).  Keys past the range read the range's last key (finite values;
// their scores are masked to -inf).
__device__ __forceinline__ void load_tile(Buffers bf, const Walk& w, int32_t kt0) {
  int32_t rows[4];
  const int32_t run_end = w.seg.run_end(kt0);
  if (kt0 + kBlockK <= min(run_end, w.k_end)) {      // whole tile inside one run
    const int32_t base = w.seg.row(kt0);
#pragma unroll
    for (int i = 0; i < 4; ++i) rows[i] = base + w.lrow + 4 * i;
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i) rows[i] = w.seg.row(min(kt0 + w.lrow + 4 * i, w.k_end - 1));
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t off = uint32_t(rows[i]) * kRowBytes + w.lpiece[i];
    uint8_t* kd = bf.k + (16 * w.wave + 4 * i) * kRowBytes;
    uint8_t* vd = bf.v + (16 * w.wave + 4 * i) * kRowBytes;
    __builtin_amdgcn_global_load_lds((global_void_t*)(w.kbase + off), (lds_void_t*)kd, 16, 0, 0);
    __builtin_amdgcn_global_load_lds((global_void_t*)(w.vbase + off), (lds_void_t*)vd, 16, 0, 0);
  }
}

// S^T for both 32-key blocks of the tile in LDS: the sixteen K fragments are read first
// (one LDS round trip), then the MFMAs consume them in order.
__device__ __forceinline__ void qk_tile(f32x16_t (&s0)[kQB], f32x16_t (&s1)[kQB], const uint8_t* kt,
                                        const bf16x8_t (&qf)[kQB][8], const Walk& w) {
  const f32x16_t zero = {};
  bf16x8_t kf[2][8];
#pragma unroll
  for (int st = 0; st < 8; ++st) {
    kf[0][st] = as_bf16x8(*(const lds_u32x4_t*)(kt + w.koff[st]));
    kf[1][st] = as_bf16x8(*(const lds_u32x4_t*)(kt + 32 * kRowBytes + w.koff[st]));
  }
#pragma unroll
  for (int st = 0; st < 8; ++st)
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
      s0[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[0][st], qf[qb][st], st == 0 ? zero : s0[qb], 0, 0, 0);
      s1[qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[1][st], qf[qb][st], st == 0 ? zero : s1[qb], 0, 0, 0);
    }
}

__device__ __forceinline__ void mask_block(f32x16_t (&s)[kQB], int32_t key0, int32_t k_end, int half) {
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (key0 + 8 * (i >> 2) + 4 * half + (i & 3) >= k_end) s[qb][i] = -INFINITY;
}

// Probabilities (bf16) of key block kb and their row sums, then O^T += V^T * P^T over
// the block's two 16-key steps.
__device__ __forceinline__ void pv_block(f32x16_t (&o)[kQB][4], float (&l)[kQB], const f32x16_t (&s)[kQB],
                                         const uint8_t* vt, int kb, const float (&m_off)[kQB], const Walk& w) {
  const bf16x2_t ones = {(__bf16)1.f, (__bf16)1.f};
  bf16x8_t pf[kQB][2];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    const float moff = m_off[qb] * w.c2;
    float acc = l[qb];
#pragma unroll
    for (int i = 0; i < 16; i += 2) {
      bf16x2_t p2;
      p2[0] = (__bf16)__builtin_amdgcn_exp2f(fmaf(s[qb][i], w.c2, -moff));
      p2[1] = (__bf16)__builtin_amdgcn_exp2f(fmaf(s[qb][i + 1], w.c2, -moff));
      acc = __builtin_amdgcn_fdot2_f32_bf16(p2, ones, acc, false);
      pf[qb][i >> 3][i & 7] = p2[0];
      pf[qb][i >> 3][(i & 7) + 1] = p2[1];
    }
    l[qb] = acc;
  }
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    const uint8_t* vr = vt + (32 * kb + 16 * sub) * kRowBytes;
#pragma unroll
    for (int d = 0; d < 4; ++d) {
      const u32x2_t lo = lds_read_tr(vr + w.voff[0][d]);
      const u32x2_t hi = lds_read_tr(vr + w.voff[1][d]);
      const bf16x8_t vf = as_bf16x8(u32x4_t{lo.x, lo.y, hi.x, hi.y});
#pragma unroll
      for (int qb = 0; qb < kQB; ++qb)
        o[qb][d] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[qb][sub], o[qb][d], 0, 0, 0);
    }
  }
}

// One tile from buffer `cur`: S^T, masking of keys past the range, then P and O^T.
__device__ __forceinline__ void attend_tile(Buffers cur, const Walk& w, int32_t kt0, const bf16x8_t (&qf)[kQB][8],
                                            const float (&m_off)[kQB], f32x16_t (&o)[kQB][4], float (&l)[kQB]) {
  f32x16_t s0[kQB], s1[kQB];
  qk_tile(s0, s1, cur.k, qf, w);
  if (kt0 + kBlockK > w.k_end) {
    mask_block(s0, kt0, w.k_end, w.half);
    mask_block(s1, kt0 + 32, w.k_end, w.half);
  }
  pv_block(o, l, s0, cur.v, 0, m_off, w);
  pv_block(o, l, s1, cur.v, 1, m_off, w);
}

// Row max of the scores of the tile in `cur` (the range's first tile): the exponent offsets
// of pass 0.
__device__ __forceinline__ void first_tile_offsets(Buffers cur, const Walk& w, int32_t kt0,
                                                   const bf16x8_t (&qf)[kQB][8], float (&m_off)[kQB]) {
  f32x16_t s0[kQB], s1[kQB];
  qk_tile(s0, s1, cur.k, qf, w);
  if (kt0 + kBlockK > w.k_end) {
    mask_block(s0, kt0, w.k_end, w.half);
    mask_block(s1, kt0 + 32, w.k_end, w.half);
  }
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    float m = s0[qb][0];
#pragma unroll
    for (int i = 0; i < 16; ++i) m = fmaxf(fmaxf(m, s0[qb][i]), s1[qb][i]);
    m_off[qb] = fmaxf(m, __shfl_xor(m, 32));
  }
}

// Walk the key range once with fixed per-row exponent offsets m_off (raw score units).
// kFromFirstTile: set m_off from the first tile's row max (pass 0); otherwise m_off is
// given (the exact row max).  Accumulates O^T (o) and the row sums (l) from zero.
// Tiles alternate between buffers b0 and b1; while one is read, the next tile is loaded
// into the other.
template <bool kFromFirstTile>
__device__ __forceinline__ void attend(Buffers b0, Buffers b1, const Walk& w, const bf16x8_t (&qf)[kQB][8],
                                       float (&m_off)[kQB], f32x16_t (&o)[kQB][4], float (&l)[kQB]) {
  const f32x16_t zero = {};
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    l[qb] = 0.f;
#pragma unroll
    for (int d = 0; d < 4; ++d) o[qb][d] = zero;
  }
  if (w.k_begin < w.k_end) load_tile(b0, w, w.k_begin);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (kFromFirstTile && w.k_begin < w.k_end) first_tile_offsets(b0, w, w.k_begin, qf, m_off);

  int32_t kt0 = w.k_begin;
  for (; kt0 + kBlockK < w.k_end; kt0 += 2 * kBlockK) {
    load_tile(b1, w, kt0 + kBlockK);
    attend_tile(b0, w, kt0, qf, m_off, o, l);
    __builtin_amdgcn_s_waitcnt(0);     // this wave's loads of the next tile have landed
    __syncthreads();                   // ... and everyone's; buffer b0 is free
    const int32_t kt1 = kt0 + kBlockK;
    if (kt1 + kBlockK < w.k_end) load_tile(b0, w, kt1 + kBlockK);
    attend_tile(b1, w, kt1, qf, m_off, o, l);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  }
  if (kt0 < w.k_end) {                 // odd tile count: the last tile, in b0
    attend_tile(b0, w, kt0, qf, m_off, o, l);
    __syncthreads();
  }
}

// Exact row max of the scores over the key range (QK only), for the overflow fallback.
__device__ __forceinline__ void exact_row_max(Buffers b0, const Walk& w, const bf16x8_t (&qf)[kQB][8],
                                              float (&m_off)[kQB]) {
  float mx[kQB];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) mx[qb] = -INFINITY;
  for (int32_t kt0 = w.k_begin; kt0 < w.k_end; kt0 += kBlockK) {
    __syncthreads();
    load_tile(b0, w, kt0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    f32x16_t s0[kQB], s1[kQB];
    qk_tile(s0, s1, b0.k, qf, w);
    mask_block(s0, kt0, w.k_end, w.half);
    mask_block(s1, kt0 + 32, w.k_end, w.half);
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx[qb] = fmaxf(mx[qb], fmaxf(s0[qb][i], s1[qb][i]));
  }
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) m_off[qb] = fmaxf(mx[qb], __shfl_xor(mx[qb], 32));
  __syncthreads();
}

// Unit bookkeeping of the balanced schedule: unit u = (query tile t, key tile k) =
// t * Tk + k; work-group g owns units [start(g), start(g + 1)), start(g) = floor(g U / G).
struct Schedule {
  int64_t U, G;
  int32_t Tk;
  __device__ __forceinline__ int64_t start(int64_t g) const { return g * U / G; }
  __device__ __forceinline__ int64_t owner(int64_t u) const { return ((u + 1) * G - 1) / U; }
};

__device__ __forceinline__ Schedule make_schedule(const AttnArgs& a, int32_t* qtiles_out) {
  const int32_t qtiles = (a.N + kBlockQ - 1) / kBlockQ;
  *qtiles_out = qtiles;
  Schedule sc;
  sc.Tk = (a.n_keys + kBlockK - 1) / kBlockK;
  sc.U = int64_t(a.B) * a.H * qtiles * sc.Tk;
  sc.G = a.groups;
  return sc;
}

__global__ __launch_bounds__(kThreads, kGroupsPerCU) void window_attn_kernel(AttnArgs a) {
  __shared__ __attribute__((aligned(1024))) uint8_t lds_k0[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_v0[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_k1[kTileBytes];
  __shared__ __attribute__((aligned(1024))) uint8_t lds_v1[kTileBytes];
  const Buffers b0{lds_k0, lds_v0}, b1{lds_k1, lds_v1};

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int half = lane >> 5;
  const int col = lane & 31;
  const int32_t N = a.N, H = a.H;

  // XCD-aware numbering: hardware work-group i runs on XCD i % 8; give each XCD a
  // contiguous range of logical work-groups, hence of neighbouring query tiles.
  const int32_t G = gridDim.x;
  const int32_t xcd = blockIdx.x % kXcds;
  const int32_t g = xcd * (G / kXcds) + min(xcd, G % kXcds) + blockIdx.x / kXcds;

  int32_t qtiles;
  const Schedule sc = make_schedule(a, &qtiles);

  Walk w;
  w.seg.l1 = a.seg_l0[1];
  w.seg.l2 = a.seg_l0[2];
  w.seg.l3 = a.seg_l0[3];
  w.seg.r0 = a.seg_row0[0];
  w.seg.r1 = a.seg_row0[1];
  w.seg.r2 = a.seg_row0[2];
  w.seg.r3 = a.seg_row0[3];
  w.wave = wave;
  w.lane = lane;
  w.col = col;
  w.half = half;
  w.c2 = a.scale * kLog2e;
  // loader: row 16 wave + 4 i + (lane >> 4); swz of that row = ((lane >> 4) << 2) | i
  w.lrow = 16 * wave + (lane >> 4);
#pragma unroll
  for (int i = 0; i < 4; ++i) w.lpiece[i] = ((lane & 15) ^ (((lane >> 4) << 2) | i)) * 16;
  // K fragment for d-step st: row col (+32 kb), logical slot 2 st + half
#pragma unroll
  for (int st = 0; st < 8; ++st) w.koff[st] = col * kRowBytes + ((2 * st + half) ^ swz(col)) * 16;
  // V^T fragment (transposing read): lane (g = lane >> 4, e = (lane & 15) >> 2, q = lane & 3)
  // addresses row 8 up + 4 half + e, d columns 32 d + 16 (g & 1) + 4 q .. +3
  {
    const int e = (lane & 15) >> 2, q = lane & 3, g16 = lane >> 4;
#pragma unroll
    for (int up = 0; up < 2; ++up)
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        const int row = 8 * up + 4 * half + e;
        const int piece = 4 * d + 2 * (g16 & 1) + (q >> 1);
        w.voff[up][d] = row * kRowBytes + (piece ^ swz(row)) * 16 + (q & 1) * 8;
      }
  }

  // Segments (query tile, key-tile range) of this work-group's unit range, walked from
  // the last to the first: every work-group then starts at the first key tile of a query
  // tile, so work-groups stream the same keys at about the same time (shared L2).
  const int64_t u_begin = sc.start(g);
  for (int64_t u_hi = sc.start(int64_t(g) + 1); u_hi > u_begin;) {
    // segment: query tile t, key tiles [k0, k1)
    const int64_t t = (u_hi - 1) / sc.Tk;
    const int64_t u_lo = max<int64_t>(u_begin, t * sc.Tk);
    const int32_t k0 = int32_t(u_lo - t * sc.Tk);
    const int32_t k1 = int32_t(u_hi - t * sc.Tk);
    const int slot = u_lo == u_begin ? 0 : 1;
    const bool full = k0 == 0 && k1 == sc.Tk;
    u_hi = u_lo;

    const int32_t qt = int32_t(t % qtiles);
    const int32_t bh_idx = int32_t(t / qtiles);      // b * H + h
    const int32_t h = bh_idx % H;
    const int32_t b = bh_idx / H;
    const int64_t bh = int64_t(bh_idx) * a.slots * kHeadDim;
    w.kbase = reinterpret_cast<const uint8_t*>(a.k_cache + bh);
    w.vbase = reinterpret_cast<const uint8_t*>(a.v_cache + bh);
    w.k_begin = k0 * kBlockK;
    w.k_end = min(a.n_keys, k1 * kBlockK);

    // Q^T fragments: for query block qb and d-step s, q[query][16 s + 8 half .. +8]
    const int32_t q0 = qt * kBlockQ + wave * kQPerWave;
    bf16x8_t qf[kQB][8];
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
      const int32_t qi = q0 + qb * 32 + col;
      const int32_t qc = qi < N ? qi : N - 1;
      const uint16_t* qp = a.q + ((int64_t(b) * N + qc) * H + h) * kHeadDim + 8 * half;
#pragma unroll
      for (int s = 0; s < 8; ++s) qf[qb][s] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(qp + 16 * s));
    }

    // Pass 0: each row's exponent offset is the max of the range's first key tile, so
    // later probabilities may exceed 1.  If a row's sum exceeds 2^64 (its scores grew by
    // more than 64 / (scale log2 e) after the first tile), the work-group redoes the
    // segment with the exact row max, where no probability exceeds 1.
    f32x16_t o[kQB][4];
    float m_off[kQB];
    float l_run[kQB];
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) m_off[qb] = 0.f;
    attend<true>(b0, b1, w, qf, m_off, o, l_run);
    bool overflow = false;
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) overflow = overflow || !(l_run[qb] <= 0x1p64f);
    if (__syncthreads_or(overflow)) {
      exact_row_max(b0, w, qf, m_off);
      attend<false>(b0, b1, w, qf, m_off, o, l_run);
    }

    // ---- segment epilogue: the final output, or a partial for the combine pass
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) {
      const int32_t r = wave * kQPerWave + qb * 32 + col;       // row within the query tile
      const int32_t qi = qt * kBlockQ + r;
      const float l_tot = l_run[qb] + __shfl_xor(l_run[qb], 32);
      if (qi >= N) continue;
      if (full) {
        const float inv = 1.f / l_tot;
        uint16_t* op = a.out + ((int64_t(b) * N + qi) * H + h) * kHeadDim + 4 * half;
#pragma unroll
        for (int d = 0; d < 4; ++d)
#pragma unroll
          for (int gg = 0; gg < 4; ++gg) {
            typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
            bf16x4_t rr;
#pragma unroll
            for (int e = 0; e < 4; ++e) rr[e] = (__bf16)(o[qb][d][4 * gg + e] * inv);
            *reinterpret_cast<bf16x4_t*>(op + d * 32 + 8 * gg) = rr;
          }
        if (a.lse && half == 0) a.lse[(int64_t(b) * H + h) * N + qi] = m_off[qb] * a.scale + logf(l_tot);
      } else {
        const int64_t prow = (int64_t(g) * 2 + slot) * kBlockQ + r;
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        float* op = a.part_o + prow * kHeadDim + 4 * half;
#pragma unroll
        for (int d = 0; d < 4; ++d)
#pragma unroll
          for (int gg = 0; gg < 4; ++gg) {
            const float4 rr = make_float4(o[qb][d][4 * gg] * inv, o[qb][d][4 * gg + 1] * inv,
                                          o[qb][d][4 * gg + 2] * inv, o[qb][d][4 * gg + 3] * inv);
            *reinterpret_cast<float4*>(op + d * 32 + 8 * gg) = rr;
          }
        if (half == 0) {
          a.part_ml[prow * 2] = l_tot > 0.f ? m_off[qb] : -INFINITY;
          a.part_ml[prow * 2 + 1] = l_tot;
        }
      }
    }
  }
}

// Finish every query tile whose key range was shared by several work-groups: merge their
// partials by log-sum-exp, out = sum_p w_p o_p / sum_p w_p with w_p = l_p 2^((m_p - M) c2),
// M = max_p m_p.  Thread = (query tile, row, 4 output columns).
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnArgs a) {
  int32_t qtiles;
  const Schedule sc = make_schedule(a, &qtiles);
  const int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x;
  const int64_t t = idx / (kBlockQ * (kHeadDim / 4));
  if (t >= int64_t(a.B) * a.H * qtiles) return;
  const int32_t r = int32_t((idx / (kHeadDim / 4)) % kBlockQ);
  const int32_t part = int32_t(idx % (kHeadDim / 4));
  const int32_t qt = int32_t(t % qtiles);
  const int32_t qi = qt * kBlockQ + r;
  if (qi >= a.N) return;
  const int64_t ua = t * sc.Tk;
  const int64_t ga = sc.owner(ua), gb = sc.owner(ua + sc.Tk - 1);
  if (ga == gb) return;                               // written directly by its work-group
  const float c2 = a.scale * kLog2e;
  float M = -INFINITY;
  for (int64_t g = ga; g <= gb; ++g) {
    const int64_t prow = (g * 2 + (sc.start(g) >= ua ? 0 : 1)) * kBlockQ + r;
    if (a.part_ml[prow * 2 + 1] > 0.f) M = fmaxf(M, a.part_ml[prow * 2]);
  }
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float wsum = 0.f;
  for (int64_t g = ga; g <= gb; ++g) {
    const int64_t prow = (g * 2 + (sc.start(g) >= ua ? 0 : 1)) * kBlockQ + r;
    const float m = a.part_ml[prow * 2];
    const float l = a.part_ml[prow * 2 + 1];
    if (!(l > 0.f)) continue;
    const float wgt = l * __builtin_amdgcn_exp2f((m - M) * c2);
    const float4 v = *reinterpret_cast<const float4*>(a.part_o + prow * kHeadDim + part * 4);
    acc.x += wgt * v.x;
    acc.y += wgt * v.y;
    acc.z += wgt * v.z;
    acc.w += wgt * v.w;
    wsum += wgt;
  }
  const float inv = 1.f / wsum;
  const int32_t bh_idx = int32_t(t / qtiles);
  const int32_t h = bh_idx % a.H, b = bh_idx / a.H;
  typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
  bf16x4_t o;
  o[0] = (__bf16)(acc.x * inv);
  o[1] = (__bf16)(acc.y * inv);
  o[2] = (__bf16)(acc.z * inv);
  o[3] = (__bf16)(acc.w * inv);
  *reinterpret_cast<bf16x4_t*>(a.out + ((int64_t(b) * a.N + qi) * a.H + h) * kHeadDim + part * 4) = o;
  if (a.lse && part == 0) a.lse[(int64_t(b) * a.H + h) * a.N + qi] = M * a.scale + logf(wsum);
}

}  // namespace

AttnPlan attn_plan(int32_t B, int32_t H, int32_t N, int32_t n_keys) {
  // Plain: one work-group per query tile over its whole key range.  Balanced: 2 work-groups
  // per compute unit (256 CUs) share all (query tile, key tile) units equally, and query
  // tiles cut between work-groups are merged by attn_combine.  Estimated times (us): a
  // work-group's 128-query x 64-key tile ~1.85 with two per CU; partials (fp32, written
  // and read back) at ~5 TB/s plus ~5 us for the extra launch.
  constexpr int64_t kSlots = 256 * kGroupsPerCU;
  constexpr double kTileUs = 1.85;
  const int64_t qtiles = int64_t(B) * H * ((N + kBlockQ - 1) / kBlockQ);
  const int64_t tk = (n_keys + kBlockK - 1) / kBlockK;
  const int64_t units = qtiles * tk;
  AttnPlan plain{int32_t(qtiles), 0, int32_t(qtiles), 0};
  const int64_t g = std::min<int64_t>(kSlots, units / 4);
  if (g <= qtiles) return plain;
  const double t_plain = double((qtiles + kSlots - 1) / kSlots) * double(tk) * kTileUs;
  const size_t ws = attn_workspace_bytes(int32_t(g));
  const double t_bal = double((units + g - 1) / g) * kTileUs + double(ws) * 2.0 / 5.0e6 + 5.0;
  if (t_bal >= t_plain) return plain;
  return AttnPlan{int32_t(g), ws, int32_t(qtiles), size_t(g) * 2 * kBlockQ * kHeadDim};
}

size_t attn_workspace_bytes(int32_t groups) {
  const size_t rows = size_t(groups) * 2 * kBlockQ;
  return rows * kHeadDim * sizeof(float) + rows * 2 * sizeof(float);
}

hipError_t launch_window_attn(const AttnArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(window_attn_kernel, dim3(unsigned(a.groups)), dim3(kThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.part_o == nullptr) return e;
  const int64_t qtiles = int64_t(a.B) * a.H * ((a.N + kBlockQ - 1) / kBlockQ);
  const int64_t work = qtiles * kBlockQ * (kHeadDim / 4);
  hipLaunchKernelGGL(attn_combine_kernel, dim3(unsigned((work + 255) / 256)), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace unstep
