#pragma once

#include <cstdint>

namespace unstep {

// cos_out, sin_out: host float [n_frames*grid_h*grid_w, head_dim/2].  Arguments are
// validated by the caller.
void build_rope_tables(int32_t start_frame, int32_t n_frames, int32_t grid_h, int32_t grid_w,
                       int32_t head_dim, double theta, float* cos_out, float* sin_out);

}  // namespace unstep
