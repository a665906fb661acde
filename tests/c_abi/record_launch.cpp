// Host-only check of the library's launch descriptors, built with AddressSanitizer and
// UndefinedBehaviorSanitizer (no GPU, no HIP runtime).
//
// The library's host sources (api.cpp, attn_plan.cpp, rope_tables.cpp) are linked against
// stand-ins for the kernel launchers that record the descriptors instead of launching, and for
// the three HIP runtime calls the host code makes.  A call script on stdin drives the C ABI;
// for every call the program prints one JSON line: the status, the handle's frame map, and
// for each recorded launch the cache rows the kernels would address, computed with the same
// address arithmetic the kernels use (seg_table.hpp):
//   append: the slot every chunk frame is written to;
//   attention: for every (batch, head, query tile), the row the K loader and the V loader fetch
//   for every retained key, walking each work-group's segments and loader cursors in the
//   kernel's tile order; plus checks that the segments of every query tile cover its keys
//   exactly once, that K and V rows agree, that every row lies inside the cache, and that the
//   merge reads only partials some work-group wrote.
// The Python side (tests/test_descriptors_cpu.py) compares these rows with the oracle's slot
// map and key rows.
//
// Script lines:
//   create B H grid_h grid_w S R
//   append f0 C with_q         (unstep_kv_append)
//   advance f0 C               (unstep_cache_advance)
//   step f0 C W split          (unstep_step; split: pass a large enough workspace)
//   attn f0 C W split          (unstep_window_attn)
//   noalloc f0 C W             (unstep_window_attn_noalloc)
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstring>
#include <sstream>
#include <string>
#include <vector>

#include "kernels.hpp"
#include "seg_table.hpp"
#include "unstep.h"

// ---- HIP runtime stand-ins: the host code calls these three --------------------------------
extern "C" {
const char* hipGetErrorString(hipError_t) { return "recorded launch"; }
hipError_t hipMemcpyAsync(void*, const void*, size_t, hipMemcpyKind, hipStream_t) { return hipErrorNotSupported; }
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }
}

// ---- recording launchers ---------------------------------------------------------------------
namespace unstep {
static std::vector<RopeAppendArgs> g_append;
static std::vector<AttnArgs> g_attn;
static void* const kFakeScratch = reinterpret_cast<void*>(uintptr_t(0x7f0000000000ull));

hipError_t launch_rope_append(const RopeAppendArgs& a, hipStream_t) {
  g_append.push_back(a);
  return hipSuccess;
}
hipError_t launch_window_attn(const AttnArgs& a, hipStream_t) {
  g_attn.push_back(a);
  return hipSuccess;
}
hipError_t launch_flow_update(const uint16_t*, const uint16_t*, uint16_t*, int64_t, double, double, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_mfma_reference(const void*, float*, int32_t, int32_t, int32_t, hipStream_t) { return hipSuccess; }
hipError_t launch_copy3(const void*, const void*, const void*, void*, void*, void*, int64_t, hipStream_t) {
  return hipSuccess;
}
hipError_t static_attn_scratch(void** ptr, size_t* bytes) {
  *ptr = kFakeScratch;
  *bytes = kAttnMaxWorkspace;
  return hipSuccess;
}
}  // namespace unstep

namespace {

using unstep::AttnArgs;
using unstep::RopeAppendArgs;

// fake, 16-byte aligned device addresses (never dereferenced: nothing is launched)
void* fake(int i) { return reinterpret_cast<void*>(uintptr_t(0x100000000ull) * uintptr_t(i + 1)); }

std::string ints(const std::vector<int64_t>& v) {
  std::string s = "[";
  for (size_t i = 0; i < v.size(); ++i) s += (i ? "," : "") + std::to_string(v[i]);
  return s + "]";
}

// The append kernel writes chunk frame i to slot frame_slot(f0 + i): report the slots and
// whether every written row lies inside the cache.
std::string describe_append(const RopeAppendArgs& a) {
  std::vector<int64_t> slots;
  bool in_bounds = true;
  for (int32_t i = 0; i < a.C; ++i) {
    const int32_t s = unstep::frame_slot(a.f0 + i, a.S, a.R);
    slots.push_back(s);
    in_bounds = in_bounds && s >= 0 && int64_t(s + 1) * a.T <= a.slots;
  }
  return "{\"f0\":" + std::to_string(a.f0) + ",\"C\":" + std::to_string(a.C) + ",\"slots\":" + ints(slots) +
         ",\"in_bounds\":" + (in_bounds ? "true" : "false") + ",\"with_q\":" + (a.q ? "true" : "false") + "}";
}

// The tiles one operand's loader fetches over a walk of n tiles, in the kernel's order: the
// three stages before the loop (stage t: K tile min(t, n - 1), V tile max(t - 1, 0)), then in
// the step of tile t < n the stage t + 3 when t + 3 <= n (K tile min(t + 3, n - 1), V tile t + 2).
std::vector<int32_t> tile_sequence(int32_t n, bool is_v) {
  constexpr int kAhead = 3;
  std::vector<int32_t> seq;
  for (int32_t t = 0; t < kAhead; ++t)
    if (t <= n) seq.push_back(is_v ? (t - 1 > 0 ? t - 1 : 0) : (t < n - 1 ? t : n - 1));
  for (int32_t t = 0; t < n; ++t)
    if (t + kAhead <= n) seq.push_back(is_v ? t + kAhead - 1 : (t + kAhead < n - 1 ? t + kAhead : n - 1));
  return seq;
}

std::string describe_attn(const AttnArgs& a) {
  constexpr int kQ = unstep::kAttnBlockQ, kK = unstep::kAttnBlockK;
  unstep::SegTable seg;
  seg.l1 = a.seg_l0[1];
  seg.l2 = a.seg_l0[2];
  seg.l3 = a.seg_l0[3];
  seg.r0 = a.seg_row0[0];
  seg.r1 = a.seg_row0[1];
  seg.r2 = a.seg_row0[2];
  seg.r3 = a.seg_row0[3];
  const int32_t qtiles = (a.N + kQ - 1) / kQ;
  unstep::Schedule sc;
  sc.Tk = (a.n_keys + kK - 1) / kK;
  sc.U = int64_t(a.B) * a.H * qtiles * sc.Tk;
  sc.G = a.groups;
  const int64_t n_tiles = int64_t(a.B) * a.H * qtiles;
  // per query tile: the row of every key from the K and the V loader, and how often each key
  // was covered by a segment
  std::vector<std::vector<int32_t>> krow(n_tiles, std::vector<int32_t>(a.n_keys, -1));
  std::vector<std::vector<int32_t>> vrow(n_tiles, std::vector<int32_t>(a.n_keys, -1));
  std::vector<std::vector<int32_t>> cover(n_tiles, std::vector<int32_t>(a.n_keys, 0));
  std::vector<std::vector<int>> wrote(n_tiles);       // partial slot written by each group, per tile
  std::vector<std::vector<int64_t>> writer(n_tiles);
  bool rows_in_bounds = true, kv_agree = true, tail_ok = true, fast_ok = true;
  int64_t segments = 0;
  for (int64_t g = 0; g < sc.G; ++g) {
    const int64_t u_begin = sc.start(g);
    for (int64_t u_hi = sc.start(g + 1); u_hi > u_begin;) {
      const unstep::Segment s = unstep::take_segment(sc, u_begin, u_hi);
      ++segments;
      const int32_t k_begin = s.k0 * kK;
      const int32_t k_end = a.n_keys < s.k1 * kK ? a.n_keys : s.k1 * kK;
      const int32_t n = (k_end - k_begin + kK - 1) / kK;
      const bool one_run = k_end <= seg.l1;
      for (int32_t key = k_begin; key < k_end; ++key) ++cover[s.t][key];
      if (!s.full) {
        wrote[s.t].push_back(s.slot);
        writer[s.t].push_back(g);
      }
      for (int op = 0; op < 2; ++op) {
        unstep::RowCursor cur;
        unstep::cursor_at(seg, k_end, k_begin, cur);
        for (int32_t tile : tile_sequence(n, op == 1)) {
          const int32_t kt0 = k_begin + tile * kK;
          int32_t rows[kK];
          if (one_run)
            unstep::tile_rows<true, kK, kK, 1>(seg, k_end, cur, kt0, 0, rows);
          else
            unstep::tile_rows<false, kK, kK, 1>(seg, k_end, cur, kt0, 0, rows);
          // the kernel's loader takes a whole tile inside a single run from its first row
          if (one_run && kt0 + kK <= k_end)
            for (int r = 0; r < kK; ++r) fast_ok = fast_ok && rows[r] == unstep::run0_tile_row0(seg, kt0) + r;
          for (int r = 0; r < kK; ++r) {
            const int32_t key = kt0 + r;
            rows_in_bounds = rows_in_bounds && rows[r] >= 0 && rows[r] < a.slots;
            if (key >= k_end) {      // past the range: the range's last key
              tail_ok = tail_ok && rows[r] == seg.row(k_end - 1);
              continue;
            }
            std::vector<int32_t>& dst = op == 0 ? krow[s.t] : vrow[s.t];
            if (dst[key] >= 0 && dst[key] != rows[r]) kv_agree = false;
            dst[key] = rows[r];
          }
        }
      }
    }
  }
  bool covered = true, same_for_all_tiles = true, merge_ok = true;
  for (int64_t t = 0; t < n_tiles; ++t) {
    for (int32_t key = 0; key < a.n_keys; ++key) {
      covered = covered && cover[t][key] == 1;
      kv_agree = kv_agree && krow[t][key] == vrow[t][key];
      same_for_all_tiles = same_for_all_tiles && krow[t][key] == krow[0][key];
    }
    // a query tile cut between work-groups: the merge reads the partial of every group from its
    // first owner to its last, in slot 0 if the group's range starts inside the tile, else 1
    const int64_t ua = t * sc.Tk, ga = sc.owner(ua), gb = sc.owner(ua + sc.Tk - 1);
    if (ga == gb) {
      merge_ok = merge_ok && wrote[t].empty();
      continue;
    }
    if (!a.part_o) merge_ok = false;
    for (int64_t g = ga; g <= gb; ++g) {
      const int want_slot = sc.start(g) >= ua ? 0 : 1;
      bool found = false;
      for (size_t i = 0; i < writer[t].size(); ++i) found = found || (writer[t][i] == g && wrote[t][i] == want_slot);
      merge_ok = merge_ok && found;
    }
  }
  std::vector<int64_t> rows0(krow[0].begin(), krow[0].end());
  std::string out = "{\"n_keys\":" + std::to_string(a.n_keys) + ",\"groups\":" + std::to_string(a.groups) +
                    ",\"split\":" + (a.part_o ? "true" : "false") + ",\"query_tiles\":" + std::to_string(n_tiles) +
                    ",\"segments\":" + std::to_string(segments) + ",\"covered_once\":" + (covered ? "true" : "false") +
                    ",\"k_v_agree\":" + (kv_agree ? "true" : "false") +
                    ",\"same_rows_every_tile\":" + (same_for_all_tiles ? "true" : "false") +
                    ",\"rows_in_bounds\":" + (rows_in_bounds ? "true" : "false") +
                    ",\"tail_rows_ok\":" + (tail_ok ? "true" : "false") +
                    ",\"merge_reads_written\":" + (merge_ok ? "true" : "false") +
                    ",\"single_run_tiles_ok\":" + (fast_ok ? "true" : "false") + ",\"rows\":" + ints(rows0) + "}";
  return out;
}

}  // namespace

int main() {
  unstep_cache* c = nullptr;
  int32_t S = 0, R = 0, H = 1;
  std::string line;
  char buf[4096];
  while (fgets(buf, sizeof buf, stdin)) {
    line = buf;
    std::istringstream in(line);
    std::string op;
    if (!(in >> op)) continue;
    unstep::g_append.clear();
    unstep::g_attn.clear();
    int rc = UNSTEP_OK;
    if (op == "create") {
      int32_t B, gh, gw;
      in >> B >> H >> gh >> gw >> S >> R;
      if (c) unstep_cache_destroy(c);
      c = nullptr;
      rc = unstep_cache_create(&c, B, H, UNSTEP_HEAD_DIM, gh, gw, S, R, fake(0), fake(1));
    } else if (op == "append" || op == "advance") {
      int32_t f0, C, with_q = 0;
      in >> f0 >> C;
      if (op == "append") {
        in >> with_q;
        const int64_t hs = UNSTEP_HEAD_DIM;
        rc = unstep_kv_append(c, f0, C, with_q ? fake(2) : nullptr, fake(3), fake(4), H * hs, hs,
                              (const float*)fake(5), (const float*)fake(6), with_q ? fake(7) : nullptr, nullptr);
      } else {
        rc = unstep_cache_advance(c, f0, C);
      }
    } else if (op == "step" || op == "attn" || op == "noalloc") {
      int32_t f0, C, W, split = 0;
      in >> f0 >> C >> W;
      if (op != "noalloc") in >> split;
      size_t ws = 0;
      if (split && c) unstep_attn_workspace_size(c, f0, C, W, &ws);
      void* wsp = split && ws ? fake(8) : nullptr;
      if (op == "step")
        rc = unstep_step(c, f0, C, W, fake(2), fake(3), fake(4), int64_t(H) * UNSTEP_HEAD_DIM, UNSTEP_HEAD_DIM,
                         (const float*)fake(5),
                         (const float*)fake(6), fake(7), fake(9), nullptr, 0.f, wsp, ws, nullptr);
      else if (op == "attn")
        rc = unstep_window_attn(c, f0, C, W, fake(7), fake(9), nullptr, 0.f, wsp, ws, nullptr);
      else
        rc = unstep_window_attn_noalloc(c, f0, C, W, fake(7), fake(9), nullptr, 0.f, nullptr);
    } else {
      std::fprintf(stderr, "unknown op %s\n", op.c_str());
      return 2;
    }
    std::string js = "{\"op\":\"" + op + "\",\"rc\":" + std::to_string(rc);
    if (c) {
      std::vector<int32_t> fm(size_t(S) + R);
      int32_t newest = -2;
      unstep_cache_frame_map(c, fm.data(), &newest);
      js += ",\"frame_of_slot\":" + ints(std::vector<int64_t>(fm.begin(), fm.end())) + ",\"newest\":" +
            std::to_string(newest);
    }
    js += ",\"append\":[";
    for (size_t i = 0; i < unstep::g_append.size(); ++i) js += (i ? "," : "") + describe_append(unstep::g_append[i]);
    js += "],\"attn\":[";
    for (size_t i = 0; i < unstep::g_attn.size(); ++i) js += (i ? "," : "") + describe_attn(unstep::g_attn[i]);
    js += "]}";
    std::printf("%s\n", js.c_str());
    std::fflush(stdout);
  }
  if (c) unstep_cache_destroy(c);
  return 0;
}
