// Per-chunk rotary cos/sin tables, built on the host (paper Appendix A.5: fp32
// coefficients per token and coordinate pair, shared by all heads, cached per start
// latent frame and grid size and reused by every layer and denoising call).
//
// Pair j of a head of width D: the first d_t/2 pairs rotate with the token's absolute
// latent frame index, the next d_h/2 with its grid row, the last d_w/2 with its grid
// column, d_h = d_w = 2*(D/6), d_t = D - d_h - d_w.  Ladder step k on an axis of d_a
// dims has frequency w_k = 1 / theta^(2k/d_a).  The angle p*w_k, pow, cos and sin are
// double-precision C-library evaluations, rounded once to float.  Only the distinct
// (axis position, pair) angles are evaluated; token rows are gathered from them.
#include "rope_tables.hpp"

#include <cmath>
#include <vector>

namespace unstep {

void build_rope_tables(int32_t start_frame, int32_t n_frames, int32_t grid_h, int32_t grid_w,
                       int32_t head_dim, double theta, float* cos_out, float* sin_out) {
  const int32_t d_h = 2 * (head_dim / 6);
  const int32_t d_w = d_h;
  const int32_t d_t = head_dim - d_h - d_w;
  const int32_t n_pairs = head_dim / 2;
  const int32_t axis_pairs[3] = {d_t / 2, d_h / 2, d_w / 2};
  const int32_t axis_dims[3] = {d_t, d_h, d_w};
  const int32_t axis_len[3] = {n_frames, grid_h, grid_w};
  const int32_t axis_origin[3] = {start_frame, 0, 0};

  // per axis: [position][ladder step] -> (cos, sin)
  std::vector<float> ac[3], as[3];
  for (int a = 0; a < 3; ++a) {
    ac[a].resize(size_t(axis_len[a]) * axis_pairs[a]);
    as[a].resize(ac[a].size());
    for (int32_t k = 0; k < axis_pairs[a]; ++k) {
      const double w = 1.0 / std::pow(theta, (2.0 * k) / double(axis_dims[a]));
      for (int32_t i = 0; i < axis_len[a]; ++i) {
        const double ang = double(axis_origin[a] + i) * w;
        ac[a][size_t(i) * axis_pairs[a] + k] = float(std::cos(ang));
        as[a][size_t(i) * axis_pairs[a] + k] = float(std::sin(ang));
      }
    }
  }

  const int64_t T = int64_t(grid_h) * grid_w;
  for (int32_t fi = 0; fi < n_frames; ++fi)
    for (int32_t r = 0; r < grid_h; ++r)
      for (int32_t c = 0; c < grid_w; ++c) {
        const int64_t n = fi * T + int64_t(r) * grid_w + c;
        float* co = cos_out + n * n_pairs;
        float* so = sin_out + n * n_pairs;
        const int32_t pos[3] = {fi, r, c};
        int32_t j = 0;
        for (int a = 0; a < 3; ++a)
          for (int32_t k = 0; k < axis_pairs[a]; ++k, ++j) {
            co[j] = ac[a][size_t(pos[a]) * axis_pairs[a] + k];
            so[j] = as[a][size_t(pos[a]) * axis_pairs[a] + k];
          }
      }
}

}  // namespace unstep
