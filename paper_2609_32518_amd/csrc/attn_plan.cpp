// Work split of an attention launch (host arithmetic only, no HIP calls, so the CPU tests
// exercise it): one work-group per 256-query tile over its whole key range, or the launch's
// (query tile, key tile) units shared equally by about one work-group per compute unit, with
// the query tiles cut between work-groups merged afterwards by log-sum-exp.
#include <algorithm>
#include <cstdint>

#include "kernels.hpp"

namespace unstep {

AttnPlan attn_plan(int32_t B, int32_t H, int32_t N, int32_t n_keys) {
  // Costs measured on MI355X (us): a 256-query x 64-key tile takes ~1.66 when a work-group
  // walks one query tile's whole range and ~1.82 per unit in the balanced schedule (two
  // segments per work-group, fp32 partials written, and all compute units drawing power,
  // which lowers the clock of the power-limited chip); the merge reads the partials at
  // ~4.5 TB/s plus ~2 us.
  constexpr int64_t kSlots = kAttnMaxGroups;
  constexpr double kTileUsPlain = 1.66, kTileUsBalanced = 1.82;
  const int64_t qtiles = int64_t(B) * H * ((N + kAttnBlockQ - 1) / kAttnBlockQ);
  const int64_t tk = (n_keys + kAttnBlockK - 1) / kAttnBlockK;
  const int64_t units = qtiles * tk;
  AttnPlan plain{int32_t(qtiles), 0, int32_t(qtiles), 0};
  const int64_t g = std::min<int64_t>(kSlots, units / 4);
  if (g <= qtiles) return plain;
  const double t_plain = double((qtiles + kSlots - 1) / kSlots) * double(tk) * kTileUsPlain;
  const size_t ws = attn_workspace_bytes(int32_t(g));
  const double t_bal = double((units + g - 1) / g) * kTileUsBalanced + double(ws) / 4.5e6 + 2.0;
  if (t_bal >= t_plain) return plain;
  // When a whole number of work-groups per query tile nearly fills the chip, split every query
  // tile into that many equal parts: each work-group then walks one segment (one pipeline
  // fill, one partial written and merged) instead of the ends of two.  Every work-group keeps
  // at least 4 units, so none is empty: the merge reads the partial of every work-group between
  // a tile's first and last owner.
  const int64_t per = kSlots / qtiles;
  const int64_t g_aligned = qtiles * per;
  const int64_t groups = (per >= 2 && g_aligned * 10 >= kSlots * 9 && g_aligned <= units / 4) ? g_aligned : g;
  const size_t ws_g = attn_workspace_bytes(int32_t(groups));
  return AttnPlan{int32_t(groups), ws_g, int32_t(qtiles), size_t(groups) * 2 * kAttnBlockQ * kHeadDim};
}

}  // namespace unstep
