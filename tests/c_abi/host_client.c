/* A C99 consumer of the library's C ABI (include/unstep.h), built and run by
 * tests/test_c_abi.py on a machine without a GPU: it calls only the entry points that touch
 * no device memory and checks their results against closed forms and the paper's counts.
 * Exit status 0 on success; the failing check is printed otherwise. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "unstep.h"

static int failures = 0;
#define CHECK(cond)                                                      \
  do {                                                                   \
    if (!(cond)) {                                                       \
      fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                        \
    }                                                                    \
  } while (0)

int main(void) {
  CHECK(unstep_version() == 100);

  /* rotary tables of the chunk at frame 6 (3 frames, 4x6 grid): every (cos, sin) pair lies on
   * the unit circle to float rounding, and temporal pair 0 of frame 6 turns by exactly 6 rad */
  enum { F = 3, GH = 4, GW = 6, N = F * GH * GW, P = UNSTEP_HEAD_DIM / 2 };
  static float c[N * P], s[N * P];
  CHECK(unstep_rope_tables_host(6, F, GH, GW, UNSTEP_HEAD_DIM, 10000.0, c, s) == UNSTEP_OK);
  for (int i = 0; i < N * P; ++i) CHECK(fabs((double)c[i] * c[i] + (double)s[i] * s[i] - 1.0) < 1e-6);
  CHECK(c[0] == (float)cos(6.0) && s[0] == (float)sin(6.0));
  CHECK(unstep_rope_tables_host(0, 1, 1, 1, 64, 10000.0, c, s) == UNSTEP_E_SHAPE);
  CHECK(strlen(unstep_last_error()) > 0);

  /* the paper's default window at 30x52: 3 sink frames + a ring of 6, chunks of 3; the chunk
   * at frame 9 sees frames 0-2 (sinks), 6-8 (window) and 9-11 (the chunk): 14,040 keys in the
   * slots 0-2, 6-8 (frames 9-11 wrapped in) and 3-5 */
  static uint8_t fake[64] __attribute__((aligned(16)));
  unstep_cache* h = NULL;
  CHECK(unstep_cache_create(&h, 1, 12, UNSTEP_HEAD_DIM, 30, 52, 3, 6, fake, fake + 16) == UNSTEP_OK);
  for (int f0 = 0; f0 < 12; f0 += 3) CHECK(unstep_cache_advance(h, f0, 3) == UNSTEP_OK);
  int32_t row0[UNSTEP_MAX_SEGMENTS], len[UNSTEP_MAX_SEGMENTS], n_seg = 0, total = 0;
  CHECK(unstep_window_segments(h, 9, 3, 3, row0, len, &n_seg) == UNSTEP_OK);
  for (int i = 0; i < n_seg; ++i) total += len[i];
  CHECK(total == 14040);
  CHECK(n_seg == 3 && row0[0] == 0 && row0[1] == 6 * 1560 && row0[2] == 3 * 1560);
  int32_t fm[9], newest = -2;
  CHECK(unstep_cache_frame_map(h, fm, &newest) == UNSTEP_OK);
  CHECK(newest == 11 && fm[0] == 0 && fm[3] == 9 && fm[8] == 8);
  /* frame 12 was never stored, frames 3-5 were evicted */
  CHECK(unstep_window_segments(h, 12, 3, 3, row0, len, &n_seg) == UNSTEP_E_STATE);
  CHECK(unstep_window_segments(h, 9, 3, 6, row0, len, &n_seg) == UNSTEP_E_RANGE);
  CHECK(unstep_cache_advance(h, 13, 3) == UNSTEP_E_STATE);          /* a gap */
  CHECK(unstep_cache_destroy(h) == UNSTEP_OK);
  CHECK(unstep_cache_destroy(NULL) == UNSTEP_OK);

  /* DiT forwards of a 5 s clip (7 chunks): 35 for Self Forcing, 23 for UnStep two-step; a
   * zero-capacity call reports the count (with E_RANGE, as nothing fits), then the calls */
  int32_t count = -1;
  CHECK(unstep_sampler_calls(UNSTEP_SAMPLER_SELF_FORCING, 7, 3, 0.0, 0, &count, NULL, NULL, NULL, NULL, NULL) ==
        UNSTEP_E_RANGE);
  CHECK(count == 35);
  CHECK(unstep_sampler_calls(UNSTEP_SAMPLER_UNSTEP, 7, 3, 0.02, 0, &count, NULL, NULL, NULL, NULL, NULL) ==
        UNSTEP_E_RANGE);
  CHECK(count == 23);
  int32_t chunk[23], start[23], index[23];
  double sigma[23], t_label[23];
  CHECK(unstep_sampler_calls(UNSTEP_SAMPLER_UNSTEP, 7, 3, 0.02, 23, &count, chunk, start, index, sigma, t_label) ==
        UNSTEP_OK);
  /* chunk 0 runs the four-step table then its clean call at sigma 0.02; chunk 6 starts at frame 18 */
  CHECK(chunk[0] == 0 && index[0] == 0 && sigma[0] == 1.0 && index[3] == 3 && sigma[3] == 0.625);
  CHECK(index[4] == UNSTEP_SCHEDULE_CLEAN && sigma[4] == 0.02);
  CHECK(chunk[22] == 6 && start[22] == 18 && index[22] == UNSTEP_SCHEDULE_CLEAN);

  if (failures == 0) printf("c abi host client: ok\n");
  return failures == 0 ? 0 : 1;
}
