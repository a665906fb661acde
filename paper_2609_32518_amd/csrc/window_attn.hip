// Windowed block-causal attention of a chunk's queries over the retained cache rows
// (paper Sections 3.1 and 3.3; Appendix A.3).  Every query of the chunk attends to
// every retained key (sinks, window, the chunk itself); the retained keys are up to
// UNSTEP_MAX_SEGMENTS runs of consecutive cache rows, so a ring that wraps is read in
// place: the tile loader maps each logical key index to its physical row.
//
// Work-group: 8 waves x 32 queries = one 256-query tile, one work-group per compute unit.
// Waves 0-3 (group A) and 4-7 (group B) share the four SIMDs, one wave of each group per
// SIMD, and run half a key tile apart: the work-group alternates two phases separated by
// barriers, and in each phase one wave of a SIMD issues MFMAs while the other computes
// the softmax of its previous tile.  Per 64-key tile t, per wave:
//   M phase: O^T += V^T(t-1) * P^T(t-1) and S^T(t) = K(t) * Q^T   (32 MFMAs)
//   V phase: P(t) = exp2((S(t) - m) * scale * log2(e)) in bf16, row sums   (VALU), and
//            this wave's share of the loads of a later stage
// Both products use v_mfma_f32_32x32x16_bf16 with keys (S^T) or head dimensions (O^T) on
// the M side and the wave's 32 queries on N: each lane owns one query column and half of
// the 32 rows, the partner lane l^32 the other half, so row max and row sum are in-lane
// plus one exchange.  P^T comes straight from the S^T registers: the MFMA's 16 contraction
// slots per lane pair are mapped to the keys where the S^T accumulator left them, and the
// matching V^T fragments are read from the row-major V tile with the transposing LDS read
// ds_read_b64_tr_b16.
// LDS: a ring of four stages; stage t holds K tile t and V tile t-1 (the operands of the
// M phase of tile t) and is loaded straight from global memory into LDS (inline-assembly
// global_load_lds, counted by hand) three tiles ahead, each wave fetching one eighth of it
// during its V phase, when the wave's issue slots are not needed for MFMAs.  Fragment
// reads in the M phase run four MFMAs ahead of their use (pinned schedule).
// Softmax: fp32, base-2 exponentials with a fixed per-row offset m (the max of the range's
// first tile), so the loop never rescales the output; if a row's sum exceeds 2^64 the
// work-group redoes its range with the exact row max.  Row sums add the fp32
// probabilities with plain fp32 adds: the packed dot-product instructions would wait for
// the other wave's MFMAs to drain.
//
// Waves whose 32 queries all lie past the chunk's end (in the ragged last query tile) run the
// loads and barriers of the walk only.
//
// Schedule: the (query tile, key tile) units of the launch are cut into `groups` equal
// contiguous ranges, one per work-group: either one work-group per query tile (its whole key
// range), or about one per compute unit when the query tiles alone would leave too many idle
// (attn_plan weighs the two with costs measured on the chip); in the second case every query
// tile is cut into k equal parts when a whole number k >= 2 per tile nearly fills the chip.  A query tile whose key range
// falls to several work-groups gets a normalised partial output and its (offset, row sum)
// from each, and attn_combine merges them by log-sum-exp.  Work-groups are numbered so that
// neighbouring ranges (same head, neighbouring query tiles) land on the same XCD and share
// its L2 while they stream the same keys.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cfloat>
#include <climits>
#include <mutex>

#include "kernels.hpp"
#include "seg_table.hpp"

namespace unstep {
namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kBlockK = kAttnBlockK;          // keys per tile
constexpr int kBlockQ = kAttnBlockQ;          // queries per work-group (8 waves x 32)
static_assert(kBlockQ == kWaves * 32, "one 32-query block per wave");
constexpr int kStages = 4;                    // LDS ring
constexpr int kAhead = kStages - 1;           // stages in flight ahead of the one in use
constexpr int kDmaPerStage = 4;               // direct-to-LDS loads per wave per stage
constexpr int kRowBytes = kHeadDim * 2;       // one K or V row (bf16)
constexpr int kTileBytes = kBlockK * kRowBytes;
// output staging of a finished query tile in the ring: 272-byte rows (16-byte aligned;
// consecutive rows 4 banks apart, so 8-byte writes of 32 rows at one offset conflict 2-way)
constexpr int kOutPitch = kRowBytes + 16;
static_assert(kBlockQ * kOutPitch <= 2 * kStages * kTileBytes, "the output tile must fit the ring");
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

// LDS rows are 256 bytes without padding; the sixteen 16-byte slots of row r are
// XOR-swizzled with swz(r), so that both read patterns are bank-conflict free: the b128 K
// reads (16 lanes = 16 consecutive rows at one logical slot) and the transposing V reads
// (per half-wave 4 consecutive rows x 4 consecutive slots).
__device__ __forceinline__ int swz(int row) { return ((row & 3) << 2) | ((row >> 2) & 3); }

__device__ __forceinline__ bf16x8_t as_bf16x8(u32x4_t u) { return __builtin_bit_cast(bf16x8_t, u); }

// Transposing LDS read: within each 16-lane group, lane i receives element (i & 3) of
// the 4 x b16 rows addressed by lanes 4e + (i >> 2), e = 0..3.
__device__ __forceinline__ u32x2_t lds_read_tr(uint32_t addr) {
  const i16x4_t v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4_t*)(uintptr_t)(addr));
  return __builtin_bit_cast(u32x2_t, v);
}

// Workgroup barrier that also keeps the compiler from moving memory accesses across it
// (LDS reads of a stage must not be hoisted above the barrier that publishes it).
// The LDS reads issued before it have returned (their stage may be refilled right after).
__device__ __forceinline__ void barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Wait until at most n (0, 1 or 2) stages of this wave's direct-to-LDS loads are in flight.
// The loads are issued as inline assembly (below), so the counter waits are too: the
// compiler neither sees these loads nor may drop or relax the waits.
__device__ __forceinline__ void wait_stages_in_flight(int n) {
  static_assert(kDmaPerStage == 4, "vmcnt immediates assume four loads per stage");
  if (n <= 0)
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  else if (n == 1)
    asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
  else
    asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
}

// Per-wave state of one walk over a key range.
struct Walk {
  const uint8_t* kbase;        // this (batch, head)'s K rows
  const uint8_t* vbase;
  SegTable seg;
  int32_t k_begin, k_end;      // logical key range
  int32_t n;                   // tiles in the range
  int half;
  int lrow;                    // loader: tile row of this lane in its first load (+4 in the second)
  RowCursor kc, vc;            // loader cursors of walks over several runs (K tiles, V tiles)
  int lpiece[2];               // loader: byte offset of this lane's logical 16-byte piece
  uint32_t loff[2];            // loader: (lrow + 4 i) rows + lpiece[i], the lane's offset in a tile
  uint32_t lds_k, lds_v;       // LDS address of ring slot 0's K tile and V tile (uniform)
  uint32_t koff[8];            // LDS address of the K fragment for d-step 0..7 in slot 0
  uint32_t voff[2][4];         // LDS address of the V^T fragment (upper 8 keys, d block) in slot 0
  float c2;                    // scale * log2(e)
};

// Direct-to-LDS load of 8 rows (this wave's share) of the 64-key tile starting at logical
// key kt0 into the tile at LDS address dst: lane l of instruction i lands in row lrow + 4 i,
// lrow = 8 wave + (l >> 4), physical slot l & 15, and so fetches logical piece
// (l & 15) ^ swz(row).  The rows come from tile_rows (the walk's segment table and its
// cursor for this operand); keys past the range read the range's last key (finite values;
// their scores are masked to -inf).  The scalar work of the lookup shares the V-phase wave's
// issue slots with its softmax, which is why a range inside one run takes the lookup-free path
// and other walks keep a cursor per operand.
// Written as inline assembly: M0 holds the wave's LDS destination, the lane's 16 bytes land
// at M0 + 16 l.  The scalar base must come from the scalar unit: an SGPR that a VALU instruction
// wrote (v_readfirstlane) needs 5 wait states before a vector-memory read of it, which the
// compiler does not insert ahead of inline assembly.
template <bool kOneRun>
__device__ __forceinline__ void load_rows(uint32_t dst, const uint8_t* base, const Walk& w, RowCursor& cur, int wave,
                                          int32_t kt0) {
  if (kOneRun && kt0 + kBlockK <= w.k_end) {
    // a whole tile inside the single run: its first row is uniform and goes into the scalar
    // base, each lane keeping its constant offset, so the loads need no vector address
    // arithmetic (tile_rows' per-lane clamp to the range's last key cannot bind here)
    const uint8_t* tb = base + int64_t(run0_tile_row0(w.seg, kt0)) * kRowBytes;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const uint32_t off = w.loff[i];
      const uint32_t m0 = dst + (8 * wave + 4 * i) * kRowBytes;
      asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(tb), "{m0}"(m0) : "memory");
    }
    return;
  }
  int32_t rows[2];
  tile_rows<kOneRun, kBlockK, 2, 4>(w.seg, w.k_end, cur, kt0, w.lrow, rows);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const uint32_t off = uint32_t(rows[i]) * kRowBytes + w.lpiece[i];
    const uint32_t m0 = dst + (8 * wave + 4 * i) * kRowBytes;
    asm volatile("global_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "{m0}"(m0) : "memory");
  }
}

// Stage t into ring slot `slot`: K tile t and V tile t - 1.  The first and last stages hold
// only one of them; the other half is filled with a duplicate tile so that every stage
// costs each wave the same number of loads (the in-flight accounting counts loads).
template <bool kOneRun>
__device__ __forceinline__ void load_stage(int slot, Walk& w, int wave, int32_t t) {
  const int32_t tk = min(t, w.n - 1), tv = max(t - 1, 0);
  load_rows<kOneRun>(w.lds_k + slot * kTileBytes, w.kbase, w, w.kc, wave, w.k_begin + tk * kBlockK);
  load_rows<kOneRun>(w.lds_v + slot * kTileBytes, w.vbase, w, w.vc, wave, w.k_begin + tv * kBlockK);
}

// Register state of one wave.
struct Acc {
  f32x16_t o[4];               // O^T: head dims 32 d .. 32 d + 31 x the wave's 32 queries
  f32x16_t s[2];               // S^T of the current tile: keys 32 kb .. 32 kb + 31
  bf16x8_t p[2][2];            // P^T of the previous tile: (key block, 16-key step)
  float l;                     // row sum (this lane's half of the keys)
  float m_off;                 // exponent offset (raw score units)
  float mx;                    // running row max (max-only walk)
};

// The 32 MFMA jobs of an M phase.  Job code c: 0..15 the PV product of the previous tile
// (key block c / 8, 16-key step (c / 4) % 2, head-dim block c % 4), 16..31 the QK product
// of this tile (key block (c - 16) / 8, d-step (c - 16) % 8).  Issue position j runs PV
// and QK jobs alternately, which spreads the LDS reads (two per PV job, one per QK job)
// evenly over the phase.
__device__ __forceinline__ constexpr int job_id(int j) { return (j & 1) ? 16 + (j >> 1) : (j >> 1); }
__device__ __forceinline__ constexpr int job_reads(int j) { return job_id(j) < 16 ? 2 : 1; }

__device__ __forceinline__ bf16x8_t fetch_job(int jj, int slot, const Walk& w) {
  const int j = job_id(jj);
  if (j < 16) {
    const uint32_t rel = slot * kTileBytes + (32 * (j >> 3) + 16 * ((j >> 2) & 1)) * kRowBytes;
    const u32x2_t lo = lds_read_tr(w.voff[0][j & 3] + rel);
    const u32x2_t hi = lds_read_tr(w.voff[1][j & 3] + rel);
    return as_bf16x8(u32x4_t{lo.x, lo.y, hi.x, hi.y});
  }
  const int kb = (j - 16) >> 3, st = (j - 16) & 7;
  return as_bf16x8(*(const lds_u32x4_t*)(uintptr_t)(w.koff[st] + slot * kTileBytes + 32 * kb * kRowBytes));
}

__device__ __forceinline__ void run_job(Acc& a, int jj, bf16x8_t f, const bf16x8_t (&qf)[8]) {
  const int j = job_id(jj);
  if (j < 16) {
    a.o[j & 3] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f, a.p[j >> 3][(j >> 2) & 1], a.o[j & 3], 0, 0, 0);
  } else {
    const int kb = (j - 16) >> 3, st = (j - 16) & 7;
    const f32x16_t zero = {};
    a.s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f, qf[st], st == 0 ? zero : a.s[kb], 0, 0, 0);
  }
}

constexpr int kFetchAhead = 4;               // fragments in flight ahead of the MFMA that uses them

// M phase of tile t from the stage in ring slot `slot`: PV of tile t - 1 and QK of tile t
// as one straight-line sequence whose fragment reads run kFetchAhead MFMAs ahead (the
// schedule is pinned so that the reads are not serialised behind the MFMAs).
template <int J>
struct MJob {
  // MFMA J, then the reads of fragment J + kFetchAhead, each pinned in this order
  static __device__ __forceinline__ void run(Acc& a, bf16x8_t (&f)[32], int slot, const bf16x8_t (&qf)[8],
                                             const Walk& w) {
    if constexpr (J + kFetchAhead < 32) f[J + kFetchAhead] = fetch_job(J + kFetchAhead, slot, w);
    run_job(a, J, f[J], qf);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if constexpr (J + kFetchAhead < 32) __builtin_amdgcn_sched_group_barrier(0x100, job_reads(J + kFetchAhead), 0);
    if constexpr (J + 1 < 32) MJob<J + 1>::run(a, f, slot, qf, w);
  }
};

// Every M phase runs all 32 jobs, so the loop has a single path for the accumulators: in
// the first tile's phase P is still zero (the PV product adds nothing), and in the phase
// after the last tile the QK product of the duplicate K tile is not used.
__device__ __forceinline__ void m_phase(Acc& a, int slot, const bf16x8_t (&qf)[8], const Walk& w) {
  bf16x8_t f[32];
#pragma unroll
  for (int j = 0; j < kFetchAhead; ++j) f[j] = fetch_job(j, slot, w);
  __builtin_amdgcn_sched_group_barrier(0x100, 3 * kFetchAhead / 2, 0);
  MJob<0>::run(a, f, slot, qf, w);
}


// V phase of tile t: mask keys past the range (last tile), the exponent offsets (first
// tile of pass 0), then P and its row sums (kMode 2: only the row max), with this wave's
// share of the loads of stage t + 3 issued before and after the arithmetic.
template <int kMode, int kLoadSlot, bool kOneRun>
__device__ __forceinline__ void v_phase(Acc& a, int32_t t, Walk& w, int wave) {
  // this wave's share of stage t + 3 (K tile t + 3, V tile t + 2) into the slot that held
  // stage t - 1
  const bool load = t + kAhead <= w.n;
  if (load) load_rows<kOneRun>(w.lds_k + kLoadSlot * kTileBytes, w.kbase, w, w.kc, wave, w.k_begin + min(t + kAhead, w.n - 1) * kBlockK);
  const int32_t kt0 = w.k_begin + t * kBlockK;
  if (kt0 + kBlockK > w.k_end) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i)
        if (kt0 + 32 * kb + 8 * (i >> 2) + 4 * w.half + (i & 3) >= w.k_end) a.s[kb][i] = -INFINITY;
  }
  if (kMode == 2) {
#pragma unroll
    for (int i = 0; i < 16; ++i) a.mx = fmaxf(a.mx, fmaxf(a.s[0][i], a.s[1][i]));
    if (load) load_rows<kOneRun>(w.lds_v + kLoadSlot * kTileBytes, w.vbase, w, w.vc, wave, w.k_begin + (t + kAhead - 1) * kBlockK);
    return;
  }
  if (kMode == 0 && t == 0) {
    float m = a.s[0][0];
#pragma unroll
    for (int i = 0; i < 16; ++i) m = fmaxf(fmaxf(m, a.s[0][i]), a.s[1][i]);
    a.m_off = fmaxf(m, __shfl_xor(m, 32));
  }
  const float moff = a.m_off * w.c2;
  float acc0 = 0.f, acc1 = 0.f;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int i = 0; i < 16; i += 2) {
      const float e0 = __builtin_amdgcn_exp2f(fmaf(a.s[kb][i], w.c2, -moff));
      const float e1 = __builtin_amdgcn_exp2f(fmaf(a.s[kb][i + 1], w.c2, -moff));
      acc0 += e0;
      acc1 += e1;
      a.p[kb][i >> 3][i & 7] = (__bf16)e0;
      a.p[kb][i >> 3][(i & 7) + 1] = (__bf16)e1;
    }
  a.l += acc0 + acc1;
  if (load) load_rows<kOneRun>(w.lds_v + kLoadSlot * kTileBytes, w.vbase, w, w.vc, wave, w.k_begin + (t + kAhead - 1) * kBlockK);
}

// Tile t of the walk, with stage t in ring slot kSlot: the M phase of tile t, the stage
// accounting, then the V phase of tile t (which loads this wave's share of stage t + 3).
// Every wave runs the same sequence; group B entered the walk one barrier later than
// group A, so its phases fall one phase later.  A wave waits for its share of stage t + 1
// (loaded in its V phase of tile t - 2, or before the loop) at the end of its M phase,
// when only stage t + 2 may still be in flight: group A's wait precedes the barrier that
// ends global phase 2t, group B's the one that ends 2t + 1, so stage t + 1 is complete
// for everyone when phase 2t + 2 (group A's M phase of tile t + 1) starts.  The slot
// refilled with stage t + 3 (group A in phase 2t + 1, group B in 2t + 2) last held stage
// t - 1, read by group B in global phase 2t - 1.
template <int kMode, int kSlot, bool kOneRun, bool kIdle>
__device__ __forceinline__ void step(Acc& a, Walk& w, const bf16x8_t (&qf)[8], int wave, int32_t t) {
  if (t > w.n) return;
  constexpr int kLoadSlot = (kSlot + kAhead) % kStages;
  if (!kIdle) m_phase(a, kSlot, qf, w);
  if (t + 1 <= w.n) wait_stages_in_flight(min(kAhead - 2, w.n - t - 1));
  barrier();
  if (kIdle) {
    // a wave with no query of the tile: only its share of the loads, in the same order
    if (t < w.n && t + kAhead <= w.n) {
      load_rows<kOneRun>(w.lds_k + kLoadSlot * kTileBytes, w.kbase, w, w.kc, wave,
                         w.k_begin + min(t + kAhead, w.n - 1) * kBlockK);
      load_rows<kOneRun>(w.lds_v + kLoadSlot * kTileBytes, w.vbase, w, w.vc, wave,
                         w.k_begin + (t + kAhead - 1) * kBlockK);
    }
  } else if (t < w.n) {
    v_phase<kMode, kLoadSlot, kOneRun>(a, t, w, wave);
  }
  barrier();
}

// One walk over the key range.  kMode 0: exponent offsets from the first tile (pass 0);
// 1: offsets given in a.m_off; 2: exact row max only (a.mx).  Accumulates O^T and the row
// sums from zero (modes 0 and 1).
template <int kMode, bool kOneRun, bool kIdle>
__device__ __forceinline__ void walk(Acc& a, Walk& w, const bf16x8_t (&qf)[8], int wave, int group) {
  const f32x16_t zero = {};
#pragma unroll
  for (int d = 0; d < 4; ++d) a.o[d] = zero;
  a.l = 0.f;
  a.mx = -INFINITY;
  const bf16x8_t pz = {};
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int sub = 0; sub < 2; ++sub) a.p[kb][sub] = pz;
  // everything earlier (Q loads, previous stores) has drained: the in-flight accounting
  // below counts only this walk's stage loads
  __builtin_amdgcn_s_waitcnt(0);
  barrier();                                   // the ring is free
  if (!kOneRun) {                              // loader cursors at the range's first key
    cursor_at(w.seg, w.k_end, w.k_begin, w.kc);
    w.vc = w.kc;
  }
#pragma unroll
  for (int t = 0; t < kAhead; ++t)
    if (t <= w.n) load_stage<kOneRun>(t, w, wave, t);
  wait_stages_in_flight(min(kAhead - 1, w.n));
  barrier();                                   // stage 0 is complete: global phase 0
  if (group == 1) barrier();                   // group B idles in phase 0
  for (int32_t t0 = 0; t0 <= w.n; t0 += kStages) {
    step<kMode, 0, kOneRun, kIdle>(a, w, qf, wave, t0);
    step<kMode, 1, kOneRun, kIdle>(a, w, qf, wave, t0 + 1);
    step<kMode, 2, kOneRun, kIdle>(a, w, qf, wave, t0 + 2);
    step<kMode, 3, kOneRun, kIdle>(a, w, qf, wave, t0 + 3);
  }
  if (group == 0) barrier();                   // group A idles in the last phase
}

__device__ __forceinline__ Schedule make_schedule(const AttnArgs& a, int32_t* qtiles_out) {
  const int32_t qtiles = (a.N + kBlockQ - 1) / kBlockQ;
  *qtiles_out = qtiles;
  Schedule sc;
  sc.Tk = (a.n_keys + kBlockK - 1) / kBlockK;
  sc.U = int64_t(a.B) * a.H * qtiles * sc.Tk;
  sc.G = a.groups;
  return sc;
}

__global__ __launch_bounds__(kThreads) void window_attn_kernel(AttnArgs a) {
  // K ring (kStages tiles), then V ring: fragment reads address a slot by an immediate
  // offset from a per-lane base register (all offsets within a ring stay below 64 KB)
  __shared__ __attribute__((aligned(1024))) uint8_t lds[2 * kStages * kTileBytes];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int group = wave >> 2;
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
  w.half = half;
  w.c2 = a.scale * kLog2e;
  w.lds_k = uint32_t(uintptr_t((lds_void_t*)lds));
  w.lds_v = w.lds_k + kStages * kTileBytes;
  // loader: row 8 wave + 4 i + (lane >> 4); swz of that row = ((lane >> 4) << 2) | ((2 wave + i) & 3)
  w.lrow = 8 * wave + (lane >> 4);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    w.lpiece[i] = ((lane & 15) ^ (((lane >> 4) << 2) | ((2 * wave + i) & 3))) * 16;
    w.loff[i] = uint32_t((w.lrow + 4 * i) * kRowBytes + w.lpiece[i]);
  }
  // K fragment for d-step st: row col (+32 kb), logical slot 2 st + half
#pragma unroll
  for (int st = 0; st < 8; ++st) w.koff[st] = w.lds_k + col * kRowBytes + ((2 * st + half) ^ swz(col)) * 16;
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
        w.voff[up][d] = w.lds_v + row * kRowBytes + (piece ^ swz(row)) * 16 + (q & 1) * 8;
      }
  }

  // Segments (query tile, key-tile range) of this work-group's unit range, walked from
  // the last to the first: every work-group then starts at the first key tile of a query
  // tile, so work-groups stream the same keys at about the same time (shared L2).
  const int64_t u_begin = sc.start(g);
  for (int64_t u_hi = sc.start(int64_t(g) + 1); u_hi > u_begin;) {
    const Segment sg = take_segment(sc, u_begin, u_hi);
    const int64_t t = sg.t;
    const int32_t k0 = sg.k0, k1 = sg.k1;
    const int slot = sg.slot;
    const bool full = sg.full;

    const int32_t qt = int32_t(t % qtiles);
    const int32_t bh_idx = int32_t(t / qtiles);      // b * H + h
    const int32_t h = bh_idx % H;
    const int32_t b = bh_idx / H;
    const int64_t bh = int64_t(bh_idx) * a.slots * kHeadDim;
    w.kbase = reinterpret_cast<const uint8_t*>(a.k_cache + bh);
    w.vbase = reinterpret_cast<const uint8_t*>(a.v_cache + bh);
    w.k_begin = k0 * kBlockK;
    w.k_end = min(a.n_keys, k1 * kBlockK);
    w.n = (w.k_end - w.k_begin + kBlockK - 1) / kBlockK;

    // Q^T fragments: for d-step s, q[query][16 s + 8 half .. +8]
    const int32_t r = wave * 32 + col;                 // row within the query tile
    const int32_t qi = qt * kBlockQ + r;
    bf16x8_t qf[8];
    {
      const int32_t qc = qi < N ? qi : N - 1;
      const uint16_t* qp = a.q + ((int64_t(b) * N + qc) * H + h) * kHeadDim + 8 * half;
#pragma unroll
      for (int s = 0; s < 8; ++s) qf[s] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(qp + 16 * s));
    }

    // Pass 0: each row's exponent offset is the max of the range's first key tile, so
    // later probabilities may exceed 1.  If a row's sum exceeds 2^64 (its scores grew by
    // more than 64 / (scale log2 e) after the first tile), the work-group redoes the
    // segment with the exact row max, where no probability exceeds 1.
    Acc acc;
    acc.m_off = 0.f;
    // a range inside the first run of the segment table takes the loader's branch-free path
    // a wave whose 32 queries all lie past the chunk's end (the last, ragged query tile) runs
    // the walk's loads and barriers only
    const bool idle = qt * kBlockQ + wave * 32 >= N;
    if (w.k_end <= w.seg.l1) {
      if (idle)
        walk<0, true, true>(acc, w, qf, wave, group);
      else
        walk<0, true, false>(acc, w, qf, wave, group);
      if (__syncthreads_or(!(acc.l <= 0x1p64f))) {
        if (idle) {
          walk<2, true, true>(acc, w, qf, wave, group);
          walk<1, true, true>(acc, w, qf, wave, group);
        } else {
          walk<2, true, false>(acc, w, qf, wave, group);
          acc.m_off = fmaxf(acc.mx, __shfl_xor(acc.mx, 32));
          walk<1, true, false>(acc, w, qf, wave, group);
        }
      }
    } else {
      if (idle)
        walk<0, false, true>(acc, w, qf, wave, group);
      else
        walk<0, false, false>(acc, w, qf, wave, group);
      if (__syncthreads_or(!(acc.l <= 0x1p64f))) {
        if (idle) {
          walk<2, false, true>(acc, w, qf, wave, group);
          walk<1, false, true>(acc, w, qf, wave, group);
        } else {
          walk<2, false, false>(acc, w, qf, wave, group);
          acc.m_off = fmaxf(acc.mx, __shfl_xor(acc.mx, 32));
          walk<1, false, false>(acc, w, qf, wave, group);
        }
      }
    }

    // ---- segment epilogue: the final output, or a partial for the combine pass
    const float l_tot = acc.l + __shfl_xor(acc.l, 32);
    if (full) {
      // The tile's rows go out through the ring, free once every wave has left the walk: each
      // lane holds 8-byte pieces of its query's row, which stored directly would make every
      // store instruction touch 32 rows; from LDS a wave stores four whole 256-byte rows.
      // Rows past the chunk's end are staged but not stored.
      typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
      typedef __attribute__((address_space(3))) bf16x4_t lds_bf16x4_t;
      __builtin_amdgcn_s_waitcnt(0);
      barrier();                                 // every wave has finished with the ring
      const float inv = 1.f / l_tot;
      const uint32_t orow = w.lds_k + uint32_t(r * kOutPitch + 8 * half);
#pragma unroll
      for (int d = 0; d < 4; ++d)
#pragma unroll
        for (int gg = 0; gg < 4; ++gg) {
          bf16x4_t rr;
#pragma unroll
          for (int e = 0; e < 4; ++e) rr[e] = (__bf16)(acc.o[d][4 * gg + e] * inv);
          *reinterpret_cast<lds_bf16x4_t*>(uintptr_t(orow + (d * 32 + 8 * gg) * 2)) = rr;
        }
      barrier();                                 // the tile is in LDS
      const int pc = threadIdx.x & 15;           // 16-byte piece: dims 8 pc .. 8 pc + 7
#pragma unroll
      for (int i = 0; i < kBlockQ / (kThreads / 16); ++i) {
        const int rs = int(threadIdx.x >> 4) + (kThreads / 16) * i;
        const int32_t qs = qt * kBlockQ + rs;
        const u32x4_t v = *reinterpret_cast<const lds_u32x4_t*>(uintptr_t(w.lds_k + uint32_t(rs * kOutPitch + pc * 16)));
        if (qs < N) *reinterpret_cast<u32x4_t*>(a.out + ((int64_t(b) * N + qs) * H + h) * kHeadDim + 8 * pc) = v;
      }
      if (qi < N && a.lse && half == 0) a.lse[(int64_t(b) * H + h) * N + qi] = acc.m_off * a.scale + logf(l_tot);
    } else if (qi < N) {
      const int64_t prow = (int64_t(g) * 2 + slot) * kBlockQ + r;
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      float* op = a.part_o + prow * kHeadDim + 4 * half;
#pragma unroll
      for (int d = 0; d < 4; ++d)
#pragma unroll
        for (int gg = 0; gg < 4; ++gg) {
          const float4 rr = make_float4(acc.o[d][4 * gg] * inv, acc.o[d][4 * gg + 1] * inv,
                                        acc.o[d][4 * gg + 2] * inv, acc.o[d][4 * gg + 3] * inv);
          *reinterpret_cast<float4*>(op + d * 32 + 8 * gg) = rr;
        }
      if (half == 0) {
        a.part_ml[prow * 2] = l_tot > 0.f ? acc.m_off : -INFINITY;
        a.part_ml[prow * 2 + 1] = l_tot;
      }
    }
  }
}

// Finish every query tile whose key range was shared by several work-groups: merge their
// partials by log-sum-exp in one pass, keeping a running offset M: each partial (m, l, o)
// rescales the sums by 2^((M_old - M) c2) when it raises M and adds w = l 2^((m - M) c2),
// out = sum w o / sum w.  Work-group = (query tile, 32 rows), thread = (4 rows, 4 output
// columns): the schedule arithmetic (64-bit divisions) is work-group uniform and runs on the
// scalar unit, and each thread keeps the loads of 4 rows in flight.
constexpr int kCombineRowsPerThread = 4;
constexpr int kCombineRows = 8 * kCombineRowsPerThread;   // rows per work-group

__global__ __launch_bounds__(256) void attn_combine_kernel(AttnArgs a) {
  int32_t qtiles;
  const Schedule sc = make_schedule(a, &qtiles);
  constexpr int kGroupsPerTile = kBlockQ / kCombineRows;
  const int64_t t = blockIdx.x / kGroupsPerTile;                       // (b, h, query tile)
  const int32_t qt = int32_t(t % qtiles);
  const int32_t r0 = int32_t(blockIdx.x % kGroupsPerTile) * kCombineRows + int32_t(threadIdx.x >> 5);
  const int32_t part = threadIdx.x & 31;
  const int64_t ua = t * sc.Tk;
  const int64_t ga = sc.owner(ua), gb = sc.owner(ua + sc.Tk - 1);
  if (ga == gb) return;                                              // written directly by its work-group
  const float c2 = a.scale * kLog2e;
  float M[kCombineRowsPerThread], W[kCombineRowsPerThread];
  float4 acc[kCombineRowsPerThread];
#pragma unroll
  for (int j = 0; j < kCombineRowsPerThread; ++j) {
    M[j] = -FLT_MAX;
    W[j] = 0.f;
    acc[j] = make_float4(0.f, 0.f, 0.f, 0.f);
  }
  for (int64_t g = ga; g <= gb; ++g) {
    const int64_t base = (g * 2 + (sc.start(g) >= ua ? 0 : 1)) * kBlockQ + r0;
    float2 ml[kCombineRowsPerThread];
    float4 v[kCombineRowsPerThread];
#pragma unroll
    for (int j = 0; j < kCombineRowsPerThread; ++j) {
      const int64_t prow = base + 8 * j;
      ml[j] = *reinterpret_cast<const float2*>(a.part_ml + prow * 2);
      v[j] = *reinterpret_cast<const float4*>(a.part_o + prow * kHeadDim + part * 4);
    }
#pragma unroll
    for (int j = 0; j < kCombineRowsPerThread; ++j) {
      const float l = ml[j].y > 0.f ? ml[j].y : 0.f;              // an empty partial adds nothing
      const float m = ml[j].y > 0.f ? ml[j].x : -FLT_MAX;
      const float mn = fmaxf(M[j], m);
      const float s_old = __builtin_amdgcn_exp2f((M[j] - mn) * c2);
      const float w = l * __builtin_amdgcn_exp2f((m - mn) * c2);
      acc[j].x = acc[j].x * s_old + w * v[j].x;
      acc[j].y = acc[j].y * s_old + w * v[j].y;
      acc[j].z = acc[j].z * s_old + w * v[j].z;
      acc[j].w = acc[j].w * s_old + w * v[j].w;
      W[j] = W[j] * s_old + w;
      M[j] = mn;
    }
  }
  const int32_t bh_idx = int32_t(t / qtiles);
  const int32_t h = bh_idx % a.H, b = bh_idx / a.H;
  typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
#pragma unroll
  for (int j = 0; j < kCombineRowsPerThread; ++j) {
    const int32_t qi = qt * kBlockQ + r0 + 8 * j;
    if (qi >= a.N) break;
    const float inv = 1.f / W[j];
    bf16x4_t o;
    o[0] = (__bf16)(acc[j].x * inv);
    o[1] = (__bf16)(acc[j].y * inv);
    o[2] = (__bf16)(acc[j].z * inv);
    o[3] = (__bf16)(acc[j].w * inv);
    *reinterpret_cast<bf16x4_t*>(a.out + ((int64_t(b) * a.N + qi) * a.H + h) * kHeadDim + part * 4) = o;
    if (a.lse && part == 0) a.lse[(int64_t(b) * a.H + h) * a.N + qi] = M[j] * a.scale + logf(W[j]);
  }
}

}  // namespace

hipError_t launch_window_attn(const AttnArgs& a, hipStream_t stream) {
  hipLaunchKernelGGL(window_attn_kernel, dim3(unsigned(a.groups)), dim3(kThreads), 0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.part_o == nullptr) return e;
  const int64_t qtiles = int64_t(a.B) * a.H * ((a.N + kBlockQ - 1) / kBlockQ);
  hipLaunchKernelGGL(attn_combine_kernel, dim3(unsigned(qtiles * (kBlockQ / kCombineRows))), dim3(256), 0, stream, a);
  return hipGetLastError();
}

// Scratch of the allocation-free entry point (unstep_window_attn_noalloc): room for the
// partials of the largest balanced launch, one copy per device that the library runs on,
// held until the process ends.  Host code never passes the array's name to a kernel (on
// the host it names a stand-in, not device memory): it looks up the device address once per
// device with hipGetSymbolAddress and passes that.
static __device__ __align__(256) uint8_t scratch[kAttnMaxWorkspace];

hipError_t static_attn_scratch(void** ptr, size_t* bytes) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* addr[kMaxDevices] = {};
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  *bytes = kAttnMaxWorkspace;
  return hipSuccess;
}

}  // namespace unstep
