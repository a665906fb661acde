// Host-held positions of the sink + ring KV cache (paper Section 3.1, Section 3.3,
// Appendix A.3 and A.5).  Pure C++: no HIP calls, so it is exercised on machines
// without a GPU.
//
// Frames f < S live in sink slot f; later frames in ring slot S + (f - S) mod R.
// Token t of the frame in slot s is cache row s*T + t.  The retained keys of a chunk
// [f0, f0 + C) with W prior frames are frames [0, min(S, lo)) then [lo, f0 + C),
// lo = max(0, f0 - W).
#pragma once

#include <cstdint>
#include <string>
#include <utility>
#include <vector>

#include "unstep.h"

namespace unstep {

struct Segments {
  int32_t n = 0;
  int32_t row0[UNSTEP_MAX_SEGMENTS] = {0, 0, 0, 0};
  int32_t len[UNSTEP_MAX_SEGMENTS] = {0, 0, 0, 0};
  int32_t total() const {
    int32_t t = 0;
    for (int i = 0; i < n; ++i) t += len[i];
    return t;
  }
};

// The retained rows of `s` as maximal runs in ascending cache order.  Attention over the
// retained keys does not depend on their order (every query of the chunk sees every retained
// key, paper Section 3.3), so the attention launch walks them in cache order, where a full ring
// and its sinks form one run however the ring has wrapped.
inline Segments cache_order(const Segments& s) {
  Segments o = s;
  for (int i = 1; i < o.n; ++i)
    for (int j = i; j > 0 && o.row0[j - 1] > o.row0[j]; --j) {
      std::swap(o.row0[j - 1], o.row0[j]);
      std::swap(o.len[j - 1], o.len[j]);
    }
  Segments m;
  for (int i = 0; i < o.n; ++i) {
    if (m.n > 0 && m.row0[m.n - 1] + m.len[m.n - 1] == o.row0[i]) {
      m.len[m.n - 1] += o.len[i];
    } else {
      m.row0[m.n] = o.row0[i];
      m.len[m.n] = o.len[i];
      ++m.n;
    }
  }
  return m;
}

class CacheIndex {
 public:
  CacheIndex() = default;
  CacheIndex(int32_t T, int32_t S, int32_t R) : T_(T), S_(S), R_(R), frame_of_slot_(S + R, -1) {}

  int32_t T() const { return T_; }
  int32_t S() const { return S_; }
  int32_t R() const { return R_; }
  int32_t newest() const { return newest_; }
  const std::vector<int32_t>& frame_of_slot() const { return frame_of_slot_; }

  int32_t slot(int32_t f) const { return f < S_ ? f : S_ + (f - S_) % R_; }
  bool resident(int32_t f) const { return f >= 0 && frame_of_slot_[slot(f)] == f; }

  // Frames of [lo, hi) that live in the ring (frame >= S), counted without visiting them.
  int64_t ring_count(int64_t lo, int64_t hi) const {
    const int64_t first = lo > S_ ? lo : S_;
    return hi > first ? hi - first : 0;
  }

  // Validation of an append of frames [f0, f0 + C); UNSTEP_OK or a status + message.  The
  // sizes are checked arithmetically before any loop over frames, so a huge request costs
  // nothing and allocates nothing.
  int check_append(int32_t f0, int32_t C, std::string* why) const {
    if (C < 1) return fail(UNSTEP_E_SHAPE, "empty chunk (n_frames < 1)", why);
    if (f0 < 0) return fail(UNSTEP_E_RANGE, "negative start frame", why);
    if (ring_count(f0, int64_t(f0) + C) > R_)
      return fail(UNSTEP_E_RANGE, "chunk has more ring frames than the ring holds", why);
    if (int64_t(f0) + C - 1 > INT32_MAX - 1) return fail(UNSTEP_E_RANGE, "frame index overflow", why);
    if (f0 > newest_ + 1) return fail(UNSTEP_E_STATE, "gap: chunk starts after newest stored frame + 1", why);
    for (int32_t f = f0; f < f0 + C; ++f)
      if (f <= newest_ && !resident(f))
        return fail(UNSTEP_E_STATE, "re-appended frame " + std::to_string(f) + " was evicted", why);
    return UNSTEP_OK;
  }

  // Apply a validated append.
  void commit_append(int32_t f0, int32_t C) {
    for (int32_t f = f0; f < f0 + C; ++f) frame_of_slot_[slot(f)] = f;
    if (f0 + C - 1 > newest_) newest_ = f0 + C - 1;
  }

  // Retained frames in logical order (sinks, window, chunk), validated.
  int retained(int32_t f0, int32_t C, int32_t W, std::vector<int32_t>* frames, std::string* why) const {
    if (C < 1) return fail(UNSTEP_E_SHAPE, "empty chunk (n_frames < 1)", why);
    if (f0 < 0 || W < 0) return fail(UNSTEP_E_RANGE, "negative start frame or window", why);
    if (int64_t(f0) + C - 1 > INT32_MAX - 1) return fail(UNSTEP_E_RANGE, "frame index overflow", why);
    const int32_t lo = f0 - W > 0 ? f0 - W : 0;
    const int32_t n_sink = S_ < lo ? S_ : lo;
    // the sinks lie below S; the window and the chunk may not need more ring slots than exist
    if (ring_count(lo, int64_t(f0) + C) > R_)
      return fail(UNSTEP_E_RANGE, "window plus chunk has more ring frames than the ring holds", why);
    frames->clear();
    for (int32_t f = 0; f < n_sink; ++f) frames->push_back(f);
    for (int32_t f = lo; f < f0 + C; ++f) frames->push_back(f);
    for (int32_t f : *frames)
      if (!resident(f)) return fail(UNSTEP_E_STATE, "frame " + std::to_string(f) + " is not in the cache", why);
    return UNSTEP_OK;
  }

  // Number of retained frames from the window formula alone (no residency check; the ring
  // must hold the window and the chunk, so the count is at most S + R).
  int retained_count(int32_t f0, int32_t C, int32_t W, int32_t* count, std::string* why) const {
    if (C < 1) return fail(UNSTEP_E_SHAPE, "empty chunk (n_frames < 1)", why);
    if (f0 < 0 || W < 0) return fail(UNSTEP_E_RANGE, "negative start frame or window", why);
    if (int64_t(f0) + C - 1 > INT32_MAX - 1) return fail(UNSTEP_E_RANGE, "frame index overflow", why);
    const int32_t lo = f0 - W > 0 ? f0 - W : 0;
    if (ring_count(lo, int64_t(f0) + C) > R_)
      return fail(UNSTEP_E_RANGE, "window plus chunk has more ring frames than the ring holds", why);
    *count = (S_ < lo ? S_ : lo) + (f0 + C - lo);
    return UNSTEP_OK;
  }

  // Retained keys as maximal runs of consecutive cache rows, in logical order.
  int segments(int32_t f0, int32_t C, int32_t W, Segments* out, std::string* why) const {
    std::vector<int32_t> frames;
    int rc = retained(f0, C, W, &frames, why);
    if (rc != UNSTEP_OK) return rc;
    Segments s;
    for (int32_t f : frames) {
      const int32_t r0 = slot(f) * T_;
      if (s.n > 0 && s.row0[s.n - 1] + s.len[s.n - 1] == r0) {
        s.len[s.n - 1] += T_;
      } else {
        if (s.n == UNSTEP_MAX_SEGMENTS) return fail(UNSTEP_E_RANGE, "too many key segments", why);
        s.row0[s.n] = r0;
        s.len[s.n] = T_;
        ++s.n;
      }
    }
    *out = s;
    return UNSTEP_OK;
  }

 private:
  static int fail(int code, const std::string& msg, std::string* why) {
    if (why) *why = msg;
    return code;
  }

  int32_t T_ = 0, S_ = 0, R_ = 1;
  int32_t newest_ = -1;
  std::vector<int32_t> frame_of_slot_;
};

}  // namespace unstep
