// C ABI of the windowed-attention chunk step (declared in include/unstep.h).
//
// Every entry point validates its arguments and the host-held cache state first and
// only then enqueues kernels, so a failing call leaves no trace on the GPU or in the
// handle.  Nothing here reads device memory or synchronises, except
// unstep_rope_tables, which waits for its table upload.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <string>
#include <vector>

#include "cache_index.hpp"
#include "kernels.hpp"
#include "rope_tables.hpp"
#include "status.hpp"
#include "unstep.h"

struct unstep_cache {
  unstep::CacheIndex idx;
  int32_t B, H, D, grid_h, grid_w;
  int32_t slots;
  uint16_t* k;
  uint16_t* v;
};

namespace {

using unstep::aligned16;
using unstep::fail;
using unstep::fail_msg;
using unstep::ok;

int check_table_args(const char* where, int32_t f0, int32_t F, int32_t gh, int32_t gw, int32_t D,
                     double theta, const void* c, const void* s) {
  if (!c || !s) return fail(UNSTEP_E_NULL, "%s: cos_out/sin_out is NULL", where);
  if (D != UNSTEP_HEAD_DIM) return fail(UNSTEP_E_SHAPE, "%s: head_dim %d unsupported (need 128)", where, D);
  if (F < 1 || gh < 1 || gw < 1) return fail(UNSTEP_E_SHAPE, "%s: n_frames, grid_h, grid_w must be >= 1", where);
  if (int64_t(F) * gh * gw > (int64_t(1) << 31) / 64)
    return fail(UNSTEP_E_SHAPE, "%s: table too large", where);
  if (f0 < 0 || int64_t(f0) + F > INT32_MAX) return fail(UNSTEP_E_RANGE, "%s: bad start_frame", where);
  if (!(theta > 1.0) || !std::isfinite(theta)) return fail(UNSTEP_E_RANGE, "%s: theta must be > 1", where);
  return UNSTEP_OK;
}

struct AppendPlan {
  unstep::RopeAppendArgs args;
};

// Validation of an append on index `idx` (which may be a scratch copy).
int plan_append(const unstep_cache* c, const unstep::CacheIndex& idx, int32_t f0, int32_t C,
                const void* q, const void* k, const void* v, int64_t tok_stride, int64_t head_stride,
                const float* cos_t, const float* sin_t, void* q_rot, AppendPlan* plan, const char* where) {
  if (!c) return fail(UNSTEP_E_NULL, "%s: cache handle is NULL", where);
  if (!k || !v || !cos_t || !sin_t) return fail(UNSTEP_E_NULL, "%s: k, v, cos_t or sin_t is NULL", where);
  if (q && !q_rot) return fail(UNSTEP_E_NULL, "%s: q given but q_rot is NULL", where);
  std::string why;
  int rc = idx.check_append(f0, C, &why);
  if (rc != UNSTEP_OK) return fail_msg(rc, where, why);
  if (head_stride < UNSTEP_HEAD_DIM || tok_stride < int64_t(c->H) * head_stride)
    return fail(UNSTEP_E_SHAPE, "%s: strides (tok %lld, head %lld) overlap for %d heads of 128", where,
                (long long)tok_stride, (long long)head_stride, c->H);
  if ((tok_stride % 8) || (head_stride % 8))
    return fail(UNSTEP_E_ALIGN, "%s: strides must be multiples of 8 elements", where);
  if (!aligned16(k) || !aligned16(v) || !aligned16(cos_t) || !aligned16(sin_t) || (q && !aligned16(q)) ||
      (q_rot && !aligned16(q_rot)))
    return fail(UNSTEP_E_ALIGN, "%s: pointers must be 16-byte aligned", where);
  unstep::RopeAppendArgs& a = plan->args;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.tok_stride = tok_stride;
  a.head_stride = head_stride;
  a.cos_t = cos_t;
  a.sin_t = sin_t;
  a.q_rot = q ? static_cast<uint16_t*>(q_rot) : nullptr;
  a.k_cache = c->k;
  a.v_cache = c->v;
  a.B = c->B;
  a.H = c->H;
  a.T = idx.T();
  a.C = C;
  a.slots = c->slots;
  a.f0 = f0;
  a.S = idx.S();
  a.R = idx.R();
  a.wq = nullptr;
  a.wk = nullptr;
  a.eps = 0.0;
  return UNSTEP_OK;
}

int plan_attn(const unstep_cache* c, const unstep::CacheIndex& idx, int32_t f0, int32_t C, int32_t W,
              const void* q_rot, void* out, float* lse, float scale, void* workspace, size_t ws_bytes,
              unstep::AttnArgs* a, const char* where) {
  if (!c) return fail(UNSTEP_E_NULL, "%s: cache handle is NULL", where);
  if (!q_rot || !out) return fail(UNSTEP_E_NULL, "%s: q_rot or out is NULL", where);
  unstep::Segments logical;
  std::string why;
  int rc = idx.segments(f0, C, W, &logical, &why);
  if (rc != UNSTEP_OK) return fail_msg(rc, where, why);
  const unstep::Segments seg = unstep::cache_order(logical);
  if (!aligned16(q_rot) || !aligned16(out) || (lse && (reinterpret_cast<uintptr_t>(lse) & 3u)) ||
      (workspace && !aligned16(workspace)))
    return fail(UNSTEP_E_ALIGN, "%s: pointers must be 16-byte aligned", where);
  const int32_t N = C * idx.T();
  // one 512-thread work-group per 256-query tile: the launch's work-item count must fit 32 bits
  if (int64_t(c->B) * c->H * ((int64_t(N) + 255) / 256) * 512 > int64_t(UINT32_MAX))
    return fail(UNSTEP_E_SHAPE, "%s: too many query tiles (batch x heads x chunk tokens / 256 >= 2^23)", where);
  a->q = static_cast<const uint16_t*>(q_rot);
  a->k_cache = c->k;
  a->v_cache = c->v;
  a->out = static_cast<uint16_t*>(out);
  a->lse = lse;
  a->B = c->B;
  a->N = N;
  a->H = c->H;
  a->slots = c->slots;
  a->n_keys = seg.total();
  a->n_seg = seg.n;
  int32_t l = 0;
  for (int i = 0; i < UNSTEP_MAX_SEGMENTS; ++i) {
    if (i < seg.n) {
      a->seg_l0[i] = l;
      a->seg_row0[i] = seg.row0[i];
      l += seg.len[i];
    } else {
      a->seg_l0[i] = INT32_MAX;
      a->seg_row0[i] = 0;
    }
  }
  a->seg_l0[UNSTEP_MAX_SEGMENTS] = INT32_MAX;
  a->scale = scale > 0.f ? scale : 1.0f / std::sqrt(float(UNSTEP_HEAD_DIM));
  const unstep::AttnPlan plan = unstep::attn_plan(c->B, c->H, N, a->n_keys);
  if (plan.workspace > 0 && workspace && ws_bytes >= plan.workspace) {
    a->groups = plan.groups;
    a->part_o = static_cast<float*>(workspace);
    a->part_ml = static_cast<float*>(workspace) + plan.part_o_floats;
  } else {
    // one work-group per query tile over the whole key range: no scratch needed
    a->groups = plan.plain_groups;
    a->part_o = nullptr;
    a->part_ml = nullptr;
  }
  return UNSTEP_OK;
}

}  // namespace

extern "C" {

int unstep_version(void) { return 100; }

const char* unstep_last_error(void) { return unstep::g_err; }

int unstep_cache_create(unstep_cache** out, int32_t batch, int32_t n_heads, int32_t head_dim, int32_t grid_h,
                        int32_t grid_w, int32_t sink_frames, int32_t ring_frames, void* k_cache, void* v_cache) {
  return unstep::guarded("unstep_cache_create", [&]() -> int {
    if (!out || !k_cache || !v_cache) return fail(UNSTEP_E_NULL, "unstep_cache_create: NULL argument");
    if (head_dim != UNSTEP_HEAD_DIM)
      return fail(UNSTEP_E_SHAPE, "unstep_cache_create: head_dim %d unsupported (need 128)", head_dim);
    if (batch < 1 || n_heads < 1 || grid_h < 1 || grid_w < 1 || sink_frames < 0 || ring_frames < 1)
      return fail(UNSTEP_E_SHAPE, "unstep_cache_create: sizes must be >= 1 (sink_frames >= 0)");
    const int64_t T = int64_t(grid_h) * grid_w;
    const int64_t slots = (int64_t(sink_frames) + ring_frames) * T;
    // kernels address one (batch, head)'s rows with 32-bit byte offsets (rows x 256 B), and the
    // append pass numbers the 16-byte pieces of one frame's tokens x heads in 32 bits
    if (slots * UNSTEP_HEAD_DIM * 2 > INT32_MAX || int64_t(batch) * n_heads > 65535 || T > INT32_MAX / 64 ||
        T * n_heads * (UNSTEP_HEAD_DIM * 2 / 16) > INT32_MAX)
      return fail(UNSTEP_E_SHAPE, "unstep_cache_create: cache too large");
    if (!aligned16(k_cache) || !aligned16(v_cache))
      return fail(UNSTEP_E_ALIGN, "unstep_cache_create: cache buffers must be 16-byte aligned");
    unstep_cache* c = new (std::nothrow) unstep_cache{unstep::CacheIndex(int32_t(T), sink_frames, ring_frames),
                                                      batch, n_heads, head_dim, grid_h, grid_w, int32_t(slots),
                                                      static_cast<uint16_t*>(k_cache),
                                                      static_cast<uint16_t*>(v_cache)};
    if (!c) return fail(UNSTEP_E_HOST, "unstep_cache_create: out of host memory");
    *out = c;
    return ok();
  });
}

int unstep_cache_destroy(unstep_cache* c) {
  delete c;
  return ok();
}

int unstep_cache_frame_map(const unstep_cache* c, int32_t* frame_of_slot, int32_t* newest) {
  return unstep::guarded("unstep_cache_frame_map", [&]() -> int {
    if (!c || !frame_of_slot) return fail(UNSTEP_E_NULL, "unstep_cache_frame_map: NULL argument");
    const auto& m = c->idx.frame_of_slot();
    for (size_t i = 0; i < m.size(); ++i) frame_of_slot[i] = m[i];
    if (newest) *newest = c->idx.newest();
    return ok();
  });
}

int unstep_cache_advance(unstep_cache* c, int32_t start_frame, int32_t n_frames) {
  return unstep::guarded("unstep_cache_advance", [&]() -> int {
    if (!c) return fail(UNSTEP_E_NULL, "unstep_cache_advance: cache handle is NULL");
    std::string why;
    int rc = c->idx.check_append(start_frame, n_frames, &why);
    if (rc != UNSTEP_OK) return fail_msg(rc, "unstep_cache_advance", why);
    c->idx.commit_append(start_frame, n_frames);
    return ok();
  });
}

int unstep_window_segments(const unstep_cache* c, int32_t start_frame, int32_t n_frames, int32_t window_frames,
                           int32_t* seg_row0, int32_t* seg_len, int32_t* n_seg) {
  return unstep::guarded("unstep_window_segments", [&]() -> int {
    if (!c || !seg_row0 || !seg_len || !n_seg) return fail(UNSTEP_E_NULL, "unstep_window_segments: NULL argument");
    unstep::Segments s;
    std::string why;
    int rc = c->idx.segments(start_frame, n_frames, window_frames, &s, &why);
    if (rc != UNSTEP_OK) return fail_msg(rc, "unstep_window_segments", why);
    for (int i = 0; i < s.n; ++i) {
      seg_row0[i] = s.row0[i];
      seg_len[i] = s.len[i];
    }
    *n_seg = s.n;
    return ok();
  });
}

int unstep_rope_tables_host(int32_t start_frame, int32_t n_frames, int32_t grid_h, int32_t grid_w, int32_t head_dim,
                            double theta, float* cos_out, float* sin_out) {
  return unstep::guarded("unstep_rope_tables_host", [&]() -> int {
    int rc = check_table_args("unstep_rope_tables_host", start_frame, n_frames, grid_h, grid_w, head_dim, theta,
                              cos_out, sin_out);
    if (rc != UNSTEP_OK) return rc;
    unstep::build_rope_tables(start_frame, n_frames, grid_h, grid_w, head_dim, theta, cos_out, sin_out);
    return ok();
  });
}

int unstep_rope_tables(int32_t start_frame, int32_t n_frames, int32_t grid_h, int32_t grid_w, int32_t head_dim,
                       double theta, float* cos_out, float* sin_out, void* hip_stream) {
  return unstep::guarded("unstep_rope_tables", [&]() -> int {
    int rc = check_table_args("unstep_rope_tables", start_frame, n_frames, grid_h, grid_w, head_dim, theta, cos_out,
                              sin_out);
    if (rc != UNSTEP_OK) return rc;
    if (!aligned16(cos_out) || !aligned16(sin_out))
      return fail(UNSTEP_E_ALIGN, "unstep_rope_tables: pointers must be 16-byte aligned");
    const size_t n = size_t(n_frames) * grid_h * grid_w * (head_dim / 2);
    std::vector<float> hc(n), hs(n);
    unstep::build_rope_tables(start_frame, n_frames, grid_h, grid_w, head_dim, theta, hc.data(), hs.data());
    hipStream_t st = static_cast<hipStream_t>(hip_stream);
    hipError_t e = hipMemcpyAsync(cos_out, hc.data(), n * sizeof(float), hipMemcpyHostToDevice, st);
    if (e == hipSuccess) e = hipMemcpyAsync(sin_out, hs.data(), n * sizeof(float), hipMemcpyHostToDevice, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return fail(UNSTEP_E_HIP, "unstep_rope_tables: %s", hipGetErrorString(e));
    return ok();
  });
}

int unstep_kv_append(unstep_cache* c, int32_t start_frame, int32_t n_frames, const void* q, const void* k,
                     const void* v, int64_t tok_stride, int64_t head_stride, const float* cos_t,
                     const float* sin_t, void* q_rot, void* hip_stream) {
  return unstep::guarded("unstep_kv_append", [&]() -> int {
    if (!c) return fail(UNSTEP_E_NULL, "unstep_kv_append: cache handle is NULL");
    AppendPlan p;
    int rc = plan_append(c, c->idx, start_frame, n_frames, q, k, v, tok_stride, head_stride, cos_t, sin_t, q_rot,
                         &p, "unstep_kv_append");
    if (rc != UNSTEP_OK) return rc;
    hipError_t e = unstep::launch_rope_append(p.args, static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return fail(UNSTEP_E_HIP, "unstep_kv_append: %s", hipGetErrorString(e));
    c->idx.commit_append(start_frame, n_frames);
    return ok();
  });
}

int unstep_kv_append_qknorm(unstep_cache* c, int32_t start_frame, int32_t n_frames, const void* q, const void* k,
                            const void* v, int64_t tok_stride, int64_t head_stride, const float* cos_t,
                            const float* sin_t, const void* q_norm_weight, const void* k_norm_weight,
                            double norm_eps, void* q_rot, void* hip_stream) {
  return unstep::guarded("unstep_kv_append_qknorm", [&]() -> int {
    const char* where = "unstep_kv_append_qknorm";
    if (!c) return fail(UNSTEP_E_NULL, "%s: cache handle is NULL", where);
    if (!k_norm_weight || (q && !q_norm_weight))
      return fail(UNSTEP_E_NULL, "%s: k_norm_weight (and q_norm_weight when q is given) is NULL", where);
    if (c->H > unstep::kNormMaxHeads)
      return fail(UNSTEP_E_SHAPE, "%s: %d heads; the normalising pass handles at most %d", where, c->H,
                  unstep::kNormMaxHeads);
    if (!(norm_eps >= 0.0) || !std::isfinite(norm_eps))
      return fail(UNSTEP_E_RANGE, "%s: norm_eps must be finite and >= 0", where);
    AppendPlan p;
    int rc = plan_append(c, c->idx, start_frame, n_frames, q, k, v, tok_stride, head_stride, cos_t, sin_t, q_rot,
                         &p, where);
    if (rc != UNSTEP_OK) return rc;
    if (!aligned16(k_norm_weight) || (q && !aligned16(q_norm_weight)))
      return fail(UNSTEP_E_ALIGN, "%s: norm weights must be 16-byte aligned", where);
    p.args.wq = q ? static_cast<const uint16_t*>(q_norm_weight) : nullptr;
    p.args.wk = static_cast<const uint16_t*>(k_norm_weight);
    p.args.eps = norm_eps;
    hipError_t e = unstep::launch_rope_append(p.args, static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return fail(UNSTEP_E_HIP, "%s: %s", where, hipGetErrorString(e));
    c->idx.commit_append(start_frame, n_frames);
    return ok();
  });
}

int unstep_attn_workspace_size(const unstep_cache* c, int32_t start_frame, int32_t n_frames, int32_t window_frames,
                               size_t* bytes) {
  return unstep::guarded("unstep_attn_workspace_size", [&]() -> int {
    if (!c || !bytes) return fail(UNSTEP_E_NULL, "unstep_attn_workspace_size: NULL argument");
    int32_t frames = 0;
    std::string why;
    int rc = c->idx.retained_count(start_frame, n_frames, window_frames, &frames, &why);
    if (rc != UNSTEP_OK) return fail_msg(rc, "unstep_attn_workspace_size", why);
    const int32_t N = n_frames * c->idx.T();
    *bytes = unstep::attn_plan(c->B, c->H, N, frames * c->idx.T()).workspace;
    return ok();
  });
}

int unstep_window_attn(const unstep_cache* c, int32_t start_frame, int32_t n_frames, int32_t window_frames,
                       const void* q_rot, void* out, float* lse, float softmax_scale, void* workspace,
                       size_t workspace_bytes, void* hip_stream) {
  return unstep::guarded("unstep_window_attn", [&]() -> int {
    if (!c) return fail(UNSTEP_E_NULL, "unstep_window_attn: cache handle is NULL");
    unstep::AttnArgs a;
    int rc = plan_attn(c, c->idx, start_frame, n_frames, window_frames, q_rot, out, lse, softmax_scale, workspace,
                       workspace_bytes, &a, "unstep_window_attn");
    if (rc != UNSTEP_OK) return rc;
    hipError_t e = unstep::launch_window_attn(a, static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return fail(UNSTEP_E_HIP, "unstep_window_attn: %s", hipGetErrorString(e));
    return ok();
  });
}

int unstep_window_attn_noalloc(const unstep_cache* c, int32_t start_frame, int32_t n_frames, int32_t window_frames,
                               const void* q_rot, void* out, float* lse, float softmax_scale, void* hip_stream) {
  return unstep::guarded("unstep_window_attn_noalloc", [&]() -> int {
    const char* where = "unstep_window_attn_noalloc";
    if (!c) return fail(UNSTEP_E_NULL, "%s: cache handle is NULL", where);
    unstep::AttnArgs a;
    int rc = plan_attn(c, c->idx, start_frame, n_frames, window_frames, q_rot, out, lse, softmax_scale, nullptr, 0,
                       &a, where);
    if (rc != UNSTEP_OK) return rc;
    const unstep::AttnPlan plan = unstep::attn_plan(a.B, a.H, a.N, a.n_keys);
    if (plan.workspace > 0) {
      // the split-key partials go to the library's static scratch of the current device
      if (plan.workspace > unstep::kAttnMaxWorkspace)
        return fail(UNSTEP_E_SHAPE, "%s: the split needs %zu bytes of scratch, more than the static %zu", where,
                    plan.workspace, unstep::kAttnMaxWorkspace);
      void* scratch = nullptr;
      size_t bytes = 0;
      hipError_t e = unstep::static_attn_scratch(&scratch, &bytes);
      if (e != hipSuccess) return fail(UNSTEP_E_HIP, "%s: scratch lookup: %s", where, hipGetErrorString(e));
      a.groups = plan.groups;
      a.part_o = static_cast<float*>(scratch);
      a.part_ml = static_cast<float*>(scratch) + plan.part_o_floats;
    }
    hipError_t e = unstep::launch_window_attn(a, static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return fail(UNSTEP_E_HIP, "%s: %s", where, hipGetErrorString(e));
    return ok();
  });
}

int unstep_step(unstep_cache* c, int32_t start_frame, int32_t n_frames, int32_t window_frames, const void* q,
                const void* k, const void* v, int64_t tok_stride, int64_t head_stride, const float* cos_t,
                const float* sin_t, void* q_rot, void* out, float* lse, float softmax_scale, void* workspace,
                size_t workspace_bytes, void* hip_stream) {
  return unstep::guarded("unstep_step", [&]() -> int {
    if (!c) return fail(UNSTEP_E_NULL, "unstep_step: cache handle is NULL");
    if (!q) return fail(UNSTEP_E_NULL, "unstep_step: q is NULL");
    AppendPlan p;
    int rc = plan_append(c, c->idx, start_frame, n_frames, q, k, v, tok_stride, head_stride, cos_t, sin_t, q_rot, &p,
                         "unstep_step");
    if (rc != UNSTEP_OK) return rc;
    unstep::CacheIndex after = c->idx;      // the attention half is checked on the post-append state
    after.commit_append(start_frame, n_frames);
    unstep::AttnArgs a;
    rc = plan_attn(c, after, start_frame, n_frames, window_frames, q_rot, out, lse, softmax_scale, workspace,
                   workspace_bytes, &a, "unstep_step");
    if (rc != UNSTEP_OK) return rc;
    hipStream_t st = static_cast<hipStream_t>(hip_stream);
    hipError_t e = unstep::launch_rope_append(p.args, st);
    if (e != hipSuccess) return fail(UNSTEP_E_HIP, "unstep_step (append): %s", hipGetErrorString(e));
    c->idx = after;
    e = unstep::launch_window_attn(a, st);
    if (e != hipSuccess) return fail(UNSTEP_E_HIP, "unstep_step (attention): %s", hipGetErrorString(e));
    return ok();
  });
}

int unstep_shift_schedule(int32_t n_steps, double shift, double* sigma_out, double* t_out) {
  return unstep::guarded("unstep_shift_schedule", [&]() -> int {
    if (!sigma_out || !t_out) return fail(UNSTEP_E_NULL, "unstep_shift_schedule: output is NULL");
    if (n_steps < 1) return fail(UNSTEP_E_SHAPE, "unstep_shift_schedule: n_steps must be >= 1");
    if (!(shift > 0.0) || !std::isfinite(shift)) return fail(UNSTEP_E_RANGE, "unstep_shift_schedule: shift must be > 0");
    for (int32_t i = 0; i < n_steps; ++i) {
      const double u = 1000.0 * double(n_steps - i) / double(n_steps);
      const double sigma = shift * u / (1000.0 + (shift - 1.0) * u);
      sigma_out[i] = sigma;
      t_out[i] = 1000.0 * sigma;
    }
    return ok();
  });
}

int unstep_sampler_calls(int32_t variant, int32_t n_chunks, int32_t chunk_frames, double clean_sigma,
                         int32_t capacity, int32_t* n_calls, int32_t* chunk, int32_t* start_frame,
                         int32_t* schedule_index, double* sigma, double* t_label) {
  return unstep::guarded("unstep_sampler_calls", [&]() -> int {
    if (!n_calls) return fail(UNSTEP_E_NULL, "unstep_sampler_calls: n_calls is NULL");
    *n_calls = 0;
    if (variant < UNSTEP_SAMPLER_SELF_FORCING || variant > UNSTEP_SAMPLER_UNSTEP_ONE_STEP)
      return fail(UNSTEP_E_RANGE, "unstep_sampler_calls: unknown variant %d", variant);
    if (n_chunks < 0 || chunk_frames < 1)
      return fail(UNSTEP_E_SHAPE, "unstep_sampler_calls: n_chunks must be >= 0 and chunk_frames >= 1");
    if (int64_t(n_chunks) * chunk_frames > INT32_MAX)
      return fail(UNSTEP_E_RANGE, "unstep_sampler_calls: frame indices overflow int32");
    if (std::isnan(clean_sigma) || clean_sigma > 1.0)
      return fail(UNSTEP_E_RANGE, "unstep_sampler_calls: clean_sigma must be at most 1 (negative: the default)");
    const double sc = clean_sigma >= 0.0 ? clean_sigma : variant == UNSTEP_SAMPLER_SELF_FORCING ? 0.0 : 0.02;
    // steps of chunk c: the four-step table for the first chunk (and every chunk of Self
    // Forcing); later chunks index 0, then index 2 and 3 alternating (odd chunks 2) for the
    // two-step variant or nothing more for the one-step variant; then the clean call
    auto steps = [&](int32_t c, int32_t* idx) -> int {
      if (c == 0 || variant == UNSTEP_SAMPLER_SELF_FORCING) {
        for (int i = 0; i < 4; ++i) idx[i] = i;
        return 4;
      }
      idx[0] = 0;
      if (variant == UNSTEP_SAMPLER_UNSTEP_ONE_STEP) return 1;
      idx[1] = (c & 1) ? 2 : 3;
      return 2;
    };
    int64_t total = 0;
    int32_t idx[4];
    for (int32_t c = 0; c < n_chunks; ++c) total += steps(c, idx) + 1;
    if (total > INT32_MAX) return fail(UNSTEP_E_RANGE, "unstep_sampler_calls: too many calls");
    *n_calls = int32_t(total);
    if (total > capacity)
      return fail(UNSTEP_E_RANGE, "unstep_sampler_calls: %lld calls do not fit capacity %d", (long long)total, capacity);
    if (total == 0) return ok();
    if (!chunk || !start_frame || !schedule_index || !sigma || !t_label)
      return fail(UNSTEP_E_NULL, "unstep_sampler_calls: output array is NULL");
    double tab_sigma[4], tab_t[4];
    unstep_shift_schedule(4, 5.0, tab_sigma, tab_t);
    int32_t k = 0;
    for (int32_t c = 0; c < n_chunks; ++c) {
      const int n = steps(c, idx);
      for (int i = 0; i <= n; ++i, ++k) {
        chunk[k] = c;
        start_frame[k] = c * chunk_frames;
        schedule_index[k] = i < n ? idx[i] : UNSTEP_SCHEDULE_CLEAN;
        sigma[k] = i < n ? tab_sigma[idx[i]] : sc;
        t_label[k] = i < n ? tab_t[idx[i]] : 0.0;
      }
    }
    return ok();
  });
}

namespace {
int flow_update(const char* where, const void* x, const void* y, void* out, int64_t n, double sigma, double a,
                double b, void* hip_stream) {
  if (!x || !y || !out) return fail(UNSTEP_E_NULL, "%s: NULL tensor", where);
  if (n < 0) return fail(UNSTEP_E_SHAPE, "%s: negative element count", where);
  if (!(sigma >= 0.0 && sigma <= 1.0)) return fail(UNSTEP_E_RANGE, "%s: sigma must lie in [0, 1]", where);
  if (!aligned16(x) || !aligned16(y) || !aligned16(out)) return fail(UNSTEP_E_ALIGN, "%s: pointers must be 16-byte aligned", where);
  if (n == 0) return ok();
  hipError_t e = unstep::launch_flow_update(static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(y),
                                            static_cast<uint16_t*>(out), n, a, b, static_cast<hipStream_t>(hip_stream));
  if (e != hipSuccess) return fail(UNSTEP_E_HIP, "%s: %s", where, hipGetErrorString(e));
  return ok();
}
}  // namespace

int unstep_copy3(const void* a, const void* b, const void* c, void* x, void* y, void* z, int64_t bytes,
                 void* hip_stream) {
  return unstep::guarded("unstep_copy3", [&]() -> int {
    if (!a || !b || !c || !x || !y || !z) return fail(UNSTEP_E_NULL, "unstep_copy3: NULL buffer");
    if (bytes < 0 || bytes % 16) return fail(UNSTEP_E_SHAPE, "unstep_copy3: bytes must be a multiple of 16");
    if (!aligned16(a) || !aligned16(b) || !aligned16(c) || !aligned16(x) || !aligned16(y) || !aligned16(z))
      return fail(UNSTEP_E_ALIGN, "unstep_copy3: pointers must be 16-byte aligned");
    hipError_t e = unstep::launch_copy3(a, b, c, x, y, z, bytes / 16, static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return fail(UNSTEP_E_HIP, "unstep_copy3: %s", hipGetErrorString(e));
    return ok();
  });
}

int unstep_mfma_reference(const void* src, float* sum, int32_t groups, int32_t waves_per_simd, int32_t mfmas,
                          void* hip_stream) {
  return unstep::guarded("unstep_mfma_reference", [&]() -> int {
    const char* where = "unstep_mfma_reference";
    if (!src || !sum) return fail(UNSTEP_E_NULL, "%s: src and sum are required", where);
    if (groups < 1 || groups > 65536) return fail(UNSTEP_E_SHAPE, "%s: groups must be in [1, 65536]", where);
    if (waves_per_simd != 1 && waves_per_simd != 2) return fail(UNSTEP_E_SHAPE, "%s: waves_per_simd must be 1 or 2", where);
    if (mfmas < 32 || mfmas % 32) return fail(UNSTEP_E_SHAPE, "%s: mfmas must be a positive multiple of 32", where);
    if (!aligned16(src) || !aligned16(sum)) return fail(UNSTEP_E_ALIGN, "%s: pointers must be 16-byte aligned", where);
    hipError_t e = unstep::launch_mfma_reference(src, sum, groups, waves_per_simd, mfmas,
                                                 static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return fail(UNSTEP_E_HIP, "%s: %s", where, hipGetErrorString(e));
    return ok();
  });
}

int unstep_renoise(const void* x, const void* eps, double sigma, void* x_tilde, int64_t n, void* hip_stream) {
  return unstep::guarded("unstep_renoise", [&]() -> int {
    return flow_update("unstep_renoise", x, eps, x_tilde, n, sigma, 1.0 - sigma, sigma, hip_stream);
  });
}

int unstep_emit(const void* x_tilde, const void* v, double sigma, void* x_next, int64_t n, void* hip_stream) {
  return unstep::guarded("unstep_emit", [&]() -> int {
    return flow_update("unstep_emit", x_tilde, v, x_next, n, sigma, 1.0, -sigma, hip_stream);
  });
}

}  // extern "C"
