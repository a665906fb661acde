// Launch descriptors of the step's HIP kernels (gfx950).  Filled and validated by the
// C ABI layer; the launchers only compute the grid and enqueue.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "unstep.h"

namespace unstep {

constexpr int kHeadDim = UNSTEP_HEAD_DIM;

// Fused rotary embedding of q and k plus the K/V cache write of one chunk.
struct RopeAppendArgs {
  const uint16_t* q;       // bf16 [B, N, H, 128] at (tok_stride, head_stride); may be null
  const uint16_t* k;
  const uint16_t* v;
  int64_t tok_stride;      // elements between consecutive tokens
  int64_t head_stride;     // elements between consecutive heads
  const float* cos_t;      // [N, 64]
  const float* sin_t;
  uint16_t* q_rot;         // bf16 [B, N, H, 128] contiguous; null iff q is null
  uint16_t* k_cache;       // bf16 [B, H, slots, 128]
  uint16_t* v_cache;
  int32_t B, H, T, C;      // batch, heads, tokens per frame, chunk frames
  int32_t slots;           // cache rows per (batch, head)
  int32_t f0, S, R;        // start frame, sink frames, ring frames
  // optional RMS normalisation of q and k over each token's H*128 channels before the
  // rotation: per-channel bf16 weights (wk non-null switches it on; wq non-null iff q is)
  const uint16_t* wq;
  const uint16_t* wk;
  double eps;
};

// Largest head count of the normalising variant (one wave holds a token's channels).
constexpr int kNormMaxHeads = 32;

hipError_t launch_rope_append(const RopeAppendArgs& a, hipStream_t stream);

// Attention tiling: 256 queries per work-group (8 waves x 32), 64 keys per tile, and at most
// one work-group per compute unit (256 on MI355X) in the balanced schedule.
constexpr int kAttnBlockQ = 256;
constexpr int kAttnBlockK = 64;
constexpr int kAttnMaxGroups = 256;

// Attention of a chunk's queries over the retained cache rows.
struct AttnArgs {
  const uint16_t* q;       // bf16 [B, N, H, 128] contiguous (rotated queries)
  const uint16_t* k_cache; // bf16 [B, H, slots, 128]
  const uint16_t* v_cache;
  uint16_t* out;           // bf16 [B, N, H, 128]
  float* lse;              // [B, H, N] or null
  float* part_o;           // balanced schedule: partial outputs [groups, 2, 256, 128] fp32
  float* part_ml;          // ... and their (exponent offset, row sum) [groups, 2, 256, 2]; null
                           // when groups equals the number of query tiles (no partials)
  int32_t B, N, H, slots;
  int32_t n_keys;          // retained keys
  int32_t n_seg;           // key segments (logical order)
  int32_t seg_l0[UNSTEP_MAX_SEGMENTS + 1];   // logical start of each segment (INT32_MAX unused)
  int32_t seg_row0[UNSTEP_MAX_SEGMENTS];     // physical row of each segment's first key
  int32_t groups;          // work-groups sharing the (query tile, key tile) units equally
  float scale;             // softmax scale
};

// Work-groups and scratch bytes for an attention launch of this shape: either one
// work-group per query tile (no scratch) or a balanced split over all compute units.
struct AttnPlan {
  int32_t groups;          // balanced work-groups (== plain_groups when not worth it)
  size_t workspace;        // scratch bytes the balanced schedule needs (0 for plain)
  int32_t plain_groups;    // one work-group per query tile
  size_t part_o_floats;    // offset of the (offset, sum) array in the scratch, in floats
};
// out = a x + b y on n bf16 values (renoise / emit of the clean-cache pass); n may be any
// count, pointers 16-byte aligned.
hipError_t launch_flow_update(const uint16_t* x, const uint16_t* y, uint16_t* out, int64_t n, double a, double b,
                              hipStream_t stream);

// The MFMA rate reference: `groups` work-groups of 8 waves, `waves_per_simd` (1 or 2) of each
// SIMD's two waves running `mfmas` (a multiple of 32) bf16 MFMAs on operands from src (groups *
// 512 lanes * 256 bytes); sum: groups * 8 floats.
hipError_t launch_mfma_reference(const void* src, float* sum, int32_t groups, int32_t waves_per_simd,
                                 int32_t mfmas, hipStream_t stream);
// x = a, y = b, z = c on n16 pieces of 16 bytes each, one launch (the bandwidth reference of
// the append pass); all pointers 16-byte aligned.
hipError_t launch_copy3(const void* a, const void* b, const void* c, void* x, void* y, void* z, int64_t n16,
                        hipStream_t stream);

// y = x W^T + b: x bf16 [M, K], W bf16 [N, K], bias bf16 [N] or null, y bf16 [M, N], all
// contiguous; K and N multiples of 8.
hipError_t launch_linear(const uint16_t* x, const uint16_t* w, const uint16_t* bias, uint16_t* y, int32_t M,
                         int32_t N, int32_t K, hipStream_t stream);

// y = bf16(x) on n values, round to nearest even; x and y 16-byte aligned.
hipError_t launch_cast_bf16(const float* x, uint16_t* y, int64_t n, hipStream_t stream);
// y = double(x), and y = float(x) rounded to nearest even, on n values.
hipError_t launch_widen_f64(const float* x, double* y, int64_t n, hipStream_t stream);
hipError_t launch_narrow_f32(const double* x, float* y, int64_t n, hipStream_t stream);

AttnPlan attn_plan(int32_t B, int32_t H, int32_t N, int32_t n_keys);

// Scratch of a balanced launch: two partial-output slots of 256 rows x 128 fp32 per
// work-group, then their (exponent offset, row sum) pairs.
constexpr size_t attn_workspace_bytes(int32_t groups) {
  return size_t(groups) * 2 * kAttnBlockQ * (kHeadDim + 2) * sizeof(float);
}
// The most any launch needs (kAttnMaxGroups work-groups).
constexpr size_t kAttnMaxWorkspace = attn_workspace_bytes(kAttnMaxGroups);

hipError_t launch_window_attn(const AttnArgs& a, hipStream_t stream);

// The allocation-free entry point's scratch on the current device: a static device array of
// kAttnMaxWorkspace bytes whose device address is looked up once per device and kept.
hipError_t static_attn_scratch(void** ptr, size_t* bytes);

}  // namespace unstep
