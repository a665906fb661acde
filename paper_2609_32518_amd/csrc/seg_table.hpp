// Address arithmetic shared by the kernels and the host: the cache slot of an appended frame
// (token t of the frame in slot s is cache row s*T + t), the physical cache row of each
// logical key that the attention loader fetches, and the attention work split.  The
// same functions run inside the kernels (inlined) and in host code, so the CPU tests can
// replay a launch's addressing against the oracle's slot map without a GPU.
//
// Retained keys (paper Section 3.3, Appendix A.3): the sinks older than the window, the
// window, the chunk, in that logical order.  They occupy up to UNSTEP_MAX_SEGMENTS runs of
// consecutive cache rows; a ring that has wrapped is read in place by mapping each logical
// key to its row.
#pragma once

#include <climits>
#include <cstdint>

#include "unstep.h"

#if defined(__HIPCC__) || defined(__HIP__)
#define UNSTEP_HD __host__ __device__ __forceinline__
#else
#define UNSTEP_HD inline
#endif

namespace unstep {

// Slot of latent frame f: sink slot f for f < S, else ring slot S + (f - S) mod R.
UNSTEP_HD int32_t frame_slot(int32_t f, int32_t S, int32_t R) { return f < S ? f : S + (f - S) % R; }

UNSTEP_HD int32_t imin(int32_t a, int32_t b) { return a < b ? a : b; }

// Physical row of a logical key index: up to four runs of consecutive rows, the first
// starting at logical index 0.
struct SegTable {
  int32_t l1, l2, l3;          // logical start of runs 1..3 (INT32_MAX when absent)
  int32_t r0, r1, r2, r3;      // physical row of each run's first key
  UNSTEP_HD int32_t row(int32_t key) const {
    // key + the offset of its run (the offsets are uniform across a wave: one add per key)
    int32_t d = r0;
    d = key >= l1 ? r1 - l1 : d;
    d = key >= l2 ? r2 - l2 : d;
    d = key >= l3 ? r3 - l3 : d;
    return key + d;
  }
  // Logical start of the run after the one holding key (INT32_MAX for the last run).
  UNSTEP_HD int32_t run_end(int32_t key) const {
    return key < l1 ? l1 : key < l2 ? l2 : key < l3 ? l3 : INT32_MAX;
  }
  // Logical start of the run holding key.
  UNSTEP_HD int32_t run_start(int32_t key) const {
    return key >= l3 ? l3 : key >= l2 ? l2 : key >= l1 ? l1 : 0;
  }
};

// Loader cursor of a walk over several runs: a tile whose keys [kt0, kt0 + tile) lie in
// [lo, hi) maps key kt0 + r to row kt0 + r + delta.
struct RowCursor {
  int32_t lo, hi, delta;
};

// Cursor at the run holding `key`, cut at the range's end.
UNSTEP_HD void cursor_at(const SegTable& seg, int32_t k_end, int32_t key, RowCursor& c) {
  c.lo = seg.run_start(key);
  c.hi = imin(seg.run_end(key), k_end);
  c.delta = seg.row(key) - key;
}

// Physical rows of tile rows r0, r0 + kStride, ..., r0 + (kN - 1) kStride of the kTile-key tile
// starting at logical key kt0 of a walk over [.., k_end).  Keys past the range map to the
// range's last key (the kernel masks their scores).  kOneRun: the whole range lies in the
// table's first run (a cache that has not wrapped and holds no separate sinks), so rows follow
// keys with no lookup.  Otherwise a tile inside the cursor's run costs two compares, and only a
// tile that crosses a run boundary or the range's end looks rows up per key and moves the
// cursor to the run of the next tile.
// First row of a whole tile inside the table's first run (kt0 + tile <= k_end <= l1): the tile's
// rows are this plus 0 .. tile - 1, so the loader can put it in its scalar base and keep one
// constant offset per lane.
UNSTEP_HD int32_t run0_tile_row0(const SegTable& seg, int32_t kt0) { return kt0 + seg.r0; }

template <bool kOneRun, int kTile, int kN, int kStride>
UNSTEP_HD void tile_rows(const SegTable& seg, int32_t k_end, RowCursor& c, int32_t kt0, int32_t r0,
                         int32_t (&rows)[kN]) {
  if (kOneRun) {
#pragma unroll
    for (int i = 0; i < kN; ++i) rows[i] = imin(kt0 + r0 + kStride * i, k_end - 1) + seg.r0;
  } else if (kt0 >= c.lo && kt0 + kTile <= c.hi) {
    rows[0] = kt0 + c.delta + r0;
#pragma unroll
    for (int i = 1; i < kN; ++i) rows[i] = rows[0] + kStride * i;
  } else {
#pragma unroll
    for (int i = 0; i < kN; ++i) rows[i] = seg.row(imin(kt0 + r0 + kStride * i, k_end - 1));
    cursor_at(seg, k_end, kt0 + kTile, c);
  }
}

// Work split of a launch: unit u = (query tile t, key tile k) = t * Tk + k; work-group g owns
// units [start(g), start(g + 1)), start(g) = floor(g U / G).
struct Schedule {
  int64_t U, G;
  int32_t Tk;
  UNSTEP_HD int64_t start(int64_t g) const { return g * U / G; }
  UNSTEP_HD int64_t owner(int64_t u) const { return ((u + 1) * G - 1) / U; }
};

// One segment of a work-group's unit range: query tile t, key tiles [k0, k1).  `slot` is the
// partial-output slot (0 for the segment at the start of the range, 1 otherwise) and `full`
// says whether the segment covers the query tile's whole key range.
struct Segment {
  int64_t t;
  int32_t k0, k1;
  int slot;
  bool full;
};

// The segment ending at unit u_hi (exclusive) of a range starting at u_begin; moves u_hi to
// the segment's first unit.  A work-group walks its segments from the last to the first.
UNSTEP_HD Segment take_segment(const Schedule& sc, int64_t u_begin, int64_t& u_hi) {
  Segment s;
  s.t = (u_hi - 1) / sc.Tk;
  const int64_t first = s.t * sc.Tk;
  const int64_t u_lo = u_begin > first ? u_begin : first;
  s.k0 = int32_t(u_lo - first);
  s.k1 = int32_t(u_hi - first);
  s.slot = u_lo == u_begin ? 0 : 1;
  s.full = s.k0 == 0 && s.k1 == sc.Tk;
  u_hi = u_lo;
  return s;
}

}  // namespace unstep
