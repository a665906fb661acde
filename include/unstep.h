/*
 * unstep.h -- C ABI of the windowed-attention chunk step of a causal video DiT
 * (UnStep, arXiv 2609.32518), for one AMD MI355X (gfx950).
 *
 * One self-attention step for a chunk of C latent frames (Section 3.1, Section 3.3,
 * Appendix A.3 and A.5 of the paper):
 *   1. rotate the chunk's queries and keys with cached fp32 cos/sin tables (3D RoPE);
 *   2. write the rotated keys and the values into a sink + ring-buffer KV cache whose
 *      positions are held on the host;
 *   3. run softmax attention of the chunk's queries over the retained keys: the sink
 *      frames older than the window, the W frames before the chunk, and the chunk.
 *
 * Conventions shared by every entry point:
 *   - bf16 tensors are passed as `const void*` / `void*` holding IEEE bfloat16 values;
 *     fp32 tensors as `float*`.  Device pointers are caller-owned (this library never
 *     allocates, frees or reads device memory on the step path) and must be 16-byte
 *     aligned; head_dim (the innermost axis) has stride 1.
 *   - Token order inside a chunk is frame-major, then grid row, then grid column:
 *     token n = (i*grid_h + r)*grid_w + c for chunk frame i, row r, column c.
 *   - N = n_frames * T, T = grid_h * grid_w tokens per latent frame.
 *   - Functions taking `hip_stream` enqueue their kernels on that stream (a
 *     hipStream_t; NULL = the default stream) and return without synchronising,
 *     except unstep_rope_tables, which waits for its upload (it runs once per
 *     (start frame, grid), off the step path).
 *   - Every function returns UNSTEP_OK or a negative unstep_status and never aborts;
 *     unstep_last_error() then describes the failure.  All argument and state checks
 *     happen before any work is enqueued; a failed call changes no state.
 *   - A cache handle is not thread-safe; distinct handles are independent.  Calls on one
 *     handle must also run in order on the device (one stream, or events between streams):
 *     each reads the cache rows the previous ones wrote.  An attention workspace must not be
 *     in use by another call that may run at the same time.
 *   - Only head_dim == 128 is supported (the model's 12 heads of width 128, App. A.5).
 */
#ifndef UNSTEP_H
#define UNSTEP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  UNSTEP_OK = 0,
  UNSTEP_E_NULL = -1,   /* a required pointer is NULL                                   */
  UNSTEP_E_SHAPE = -2,  /* unsupported or inconsistent sizes (head_dim != 128, empty...) */
  UNSTEP_E_RANGE = -3,  /* frame index / window / chunk outside what the cache can hold  */
  UNSTEP_E_STATE = -4,  /* cache state forbids the call (gap, evicted or missing frame)  */
  UNSTEP_E_HIP = -5,    /* the HIP runtime reported an error (message from HIP)          */
  UNSTEP_E_ALIGN = -6,  /* a pointer is not 16-byte aligned or a stride not a multiple of 8 */
  UNSTEP_E_HOST = -7    /* a host-side failure, e.g. out of host memory (no state changed)  */
} unstep_status;

#define UNSTEP_HEAD_DIM 128
#define UNSTEP_MAX_SEGMENTS 4

/* Library version, major*10000 + minor*100 + patch. */
int unstep_version(void);

/* Message describing the last failed call on this thread ("" if none).  The string is
 * owned by the library and valid until the next call on the same thread. */
const char* unstep_last_error(void);

/* ---------------------------------------------------------------------------------
 * KV cache handle: host-held positions (Section 3.1 and Appendix A.5: the positions
 * depend only on token counts, so they live on the CPU and no call reads the GPU).
 *
 * Slots: S sink slots hold frames 0..S-1; R ring slots hold every later frame f at
 * slot S + (f - S) mod R (the sink + sliding-window cache of Section 3.3 / App. A.3,
 * evicting whole latent frames).  Token t of the frame in slot s is cache row s*T + t.
 * ------------------------------------------------------------------------------- */
typedef struct unstep_cache unstep_cache;

/* Create a handle over caller-owned device buffers k_cache, v_cache, each bf16
 * [batch, n_heads, (sink_frames + ring_frames) * grid_h * grid_w, head_dim], which the
 * caller keeps alive until unstep_cache_destroy.  The handle starts empty (no frame
 * stored).  Touches no device memory.  Errors: E_NULL (out, k_cache, v_cache),
 * E_SHAPE (head_dim != 128, batch/n_heads/grid < 1, sink_frames < 0, ring_frames < 1,
 * more than 2^31 bytes per (batch, head) cache, i.e. (S + R) * T > 8388607 rows,
 * batch * n_heads > 65535, or T * n_heads > 134217727 tokens x heads per frame),
 * E_ALIGN. */
int unstep_cache_create(unstep_cache** out, int32_t batch, int32_t n_heads, int32_t head_dim,
                        int32_t grid_h, int32_t grid_w, int32_t sink_frames, int32_t ring_frames,
                        void* k_cache, void* v_cache);

/* Free the host state (never the device buffers).  NULL is accepted. */
int unstep_cache_destroy(unstep_cache* c);

/* Host copy of the index state: frame_of_slot[S + R] receives the latent frame stored
 * in each slot (-1 = never written); *newest (optional) the newest frame stored
 * (-1 = none).  Errors: E_NULL. */
int unstep_cache_frame_map(const unstep_cache* c, int32_t* frame_of_slot, int32_t* newest);

/* Record frames [start_frame, start_frame + n_frames) as stored without touching device
 * memory, exactly as unstep_kv_append would update the positions (same checks).  For
 * callers that fill the K/V buffers by other means, e.g. restoring a snapshot (the K/V
 * buffers plus the frame map are the whole cache state).  Errors: as the index checks
 * of unstep_kv_append (E_NULL, E_SHAPE, E_RANGE, E_STATE). */
int unstep_cache_advance(unstep_cache* c, int32_t start_frame, int32_t n_frames);

/* Retained keys of the chunk [start_frame, start_frame + n_frames) with a window of
 * window_frames prior frames: frames [0, min(S, lo)) then [lo, start_frame + n_frames),
 * lo = max(0, start_frame - window_frames), in that order (the sinks, the window, the
 * chunk; Section 3.3).  Written as maximal runs of consecutive cache rows:
 * seg_row0[i], seg_len[i] for i < *n_seg (at most UNSTEP_MAX_SEGMENTS).
 * Errors: E_NULL, E_SHAPE (n_frames < 1), E_RANGE (negative frame or window; more
 * ring frames retained than the ring holds), E_STATE (a retained frame is not in the
 * cache: never appended or evicted). */
int unstep_window_segments(const unstep_cache* c, int32_t start_frame, int32_t n_frames,
                           int32_t window_frames, int32_t* seg_row0, int32_t* seg_len,
                           int32_t* n_seg);

/* ---------------------------------------------------------------------------------
 * Rotary tables (Appendix A.5: fp32 cos/sin per token and coordinate pair, shared by
 * all heads, cached per (start latent frame, grid size)).
 *
 * Pair j = 0..head_dim/2-1 belongs to the temporal axis for j < d_t/2, to the grid
 * row axis for the next d_h/2 pairs and to the column axis for the last d_w/2, with
 * d_h = d_w = 2*(head_dim/6) and d_t = head_dim - d_h - d_w (22/21/21 pairs at 128).
 * Pair j with ladder step k on an axis of d_a dims turns by angle p * w,
 * w = 1 / pow(theta, 2k/d_a), p = the token's absolute frame index, grid row or grid
 * column.  Angle, pow, cos and sin are evaluated in double precision with the C
 * library and rounded once to float.
 * ------------------------------------------------------------------------------- */

/* Host variant: writes cos_out, sin_out (host float [N, head_dim/2]).  Touches no GPU.
 * Errors: E_NULL, E_SHAPE (head_dim not 128, sizes < 1), E_RANGE (start_frame < 0,
 * theta <= 1). */
int unstep_rope_tables_host(int32_t start_frame, int32_t n_frames, int32_t grid_h, int32_t grid_w,
                            int32_t head_dim, double theta, float* cos_out, float* sin_out);

/* Device variant: the same tables written to device buffers cos_out, sin_out (float
 * [N, head_dim/2]) through hip_stream; returns after the upload completed.
 * Errors: as the host variant, plus E_ALIGN and E_HIP. */
int unstep_rope_tables(int32_t start_frame, int32_t n_frames, int32_t grid_h, int32_t grid_w,
                       int32_t head_dim, double theta, float* cos_out, float* sin_out,
                       void* hip_stream);

/* ---------------------------------------------------------------------------------
 * Fused RoPE + KV append (Section 3.1 and Appendix A.5; one bandwidth-bound pass).
 *
 * For every chunk token n, head h, pair j (x_e = x[2j], x_o = x[2j+1], c/s the table
 * entries of token n, pair j):  y_e = x_e*c - x_o*s,  y_o = x_e*s + x_o*c, each
 * product and the sum/difference an IEEE fp32 operation rounded to nearest-even (no
 * fused multiply-add), the result rounded to bf16 nearest-even.
 *   q_rot[b, n, h, :] = rotate(q[b, n, h, :])             (skipped if q == NULL)
 *   K-cache row of token n = rotate(k[b, n, h, :]);  V-cache row of token n = v (bits)
 * q, k, v: bf16 [batch, N, n_heads, 128] at element strides tok_stride (between tokens)
 * and head_stride (between heads); batch stride N*tok_stride.  q_rot: bf16 contiguous
 * [batch, N, n_heads, 128].  cos_t, sin_t: device float [N, 64] from unstep_rope_tables
 * for the same start frame and grid.
 *
 * Index update (host): the chunk may start at most one frame after the newest stored
 * frame; re-appending stored frames overwrites them in place without advancing the
 * positions (repeated denoising calls, App. A.5); new frames evict the ring slot's
 * previous frame.  Errors: E_NULL (c, k, v, cos_t, sin_t; q_rot when q != NULL),
 * E_SHAPE (n_frames < 1, strides too small), E_ALIGN, E_RANGE (start_frame < 0; more
 * ring frames than the ring holds), E_STATE (gap after the newest frame; a re-appended
 * frame was evicted), E_HIP.  On error nothing is enqueued and the state is unchanged. */
int unstep_kv_append(unstep_cache* c, int32_t start_frame, int32_t n_frames,
                     const void* q, const void* k, const void* v,
                     int64_t tok_stride, int64_t head_stride,
                     const float* cos_t, const float* sin_t,
                     void* q_rot, void* hip_stream);

/* The same pass with the RMS normalisation that precedes RoPE in the paper's model
 * (Appendix A.5: each query and new key is RMS-normalised over the token's
 * n_heads*128 channels, then split into heads and rotated).  For every token, separately
 * for q and k, with C = n_heads*128 and w the per-channel weight:
 *   ss = sum_i x_i^2                  (fp64; each bf16 square is exact)
 *   r  = 1 / sqrt(ss / C + norm_eps)  (fp64)
 *   x'_j = bf16(fp32((x_j * r) * w_j)) (fp64 products, nearest-even roundings)
 * and x' replaces x in the rotation above; V is stored unchanged.  q_norm_weight,
 * k_norm_weight: device bf16 [n_heads*128], 16-byte aligned (q_norm_weight is ignored
 * when q == NULL).  norm_eps: the model's epsilon (1e-6 is the reading taken for the
 * paper's model; the paper does not state it).  Strides as above.  Errors: those of
 * unstep_kv_append, plus E_NULL (k_norm_weight; q_norm_weight when q != NULL), E_SHAPE
 * (n_heads > 32), E_RANGE (norm_eps negative or not finite), E_ALIGN (weights). */
int unstep_kv_append_qknorm(unstep_cache* c, int32_t start_frame, int32_t n_frames,
                            const void* q, const void* k, const void* v,
                            int64_t tok_stride, int64_t head_stride,
                            const float* cos_t, const float* sin_t,
                            const void* q_norm_weight, const void* k_norm_weight,
                            double norm_eps, void* q_rot, void* hip_stream);

/* ---------------------------------------------------------------------------------
 * Windowed block-causal attention (Sections 3.1 and 3.3; Appendix A.3).
 *
 * out[b, n, h, :] = sum_m softmax_m(scale * <q_rot[b, n, h, :], K_m>) V_m over the
 * retained keys m of unstep_window_segments (every query of the chunk sees every
 * retained key, the chunk's own included).  bf16 MFMA products, fp32 accumulation and
 * fp32 online softmax; out is bf16 [batch, N, n_heads, 128] contiguous.  lse
 * (optional, NULL to skip): float [batch, n_heads, N], the natural-log
 * log-sum-exp of the scaled scores.  softmax_scale <= 0 selects 1/sqrt(128).
 *
 * workspace (optional): device scratch for splitting the key range over several
 * work-groups; unstep_attn_workspace_size gives the bytes used for this call.  With
 * workspace == NULL or workspace_bytes smaller than that, the call runs unsplit (same
 * results up to fp32 summation order, possibly slower).  The size depends only on the
 * shapes (batch, heads, chunk tokens, retained key count), not on what is stored, so it
 * can be queried before the chunk is appended.
 * Errors: those of unstep_window_segments, plus E_NULL (q_rot, out), E_SHAPE (batch * heads *
 * ceil(N / 256) >= 2^23 query tiles), E_ALIGN, E_HIP;
 * unstep_attn_workspace_size: E_NULL, E_SHAPE, E_RANGE (argument checks only). */
int unstep_attn_workspace_size(const unstep_cache* c, int32_t start_frame, int32_t n_frames,
                               int32_t window_frames, size_t* bytes);

int unstep_window_attn(const unstep_cache* c, int32_t start_frame, int32_t n_frames,
                       int32_t window_frames, const void* q_rot, void* out, float* lse,
                       float softmax_scale, void* workspace, size_t workspace_bytes,
                       void* hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, serving
 * loops, harnesses that forbid hipMalloc): unstep_window_attn with the split-key scratch taken
 * from a static device array inside the library instead of a workspace argument.  The array
 * holds the partials of the largest split the library plans (256 work-groups: 68,157,440
 * bytes); each device the library runs on gets its own copy, which it holds until the process
 * ends.  The first call on a device looks up the array's device address (hipGetSymbolAddress);
 * no call allocates or frees device memory, enqueues a memset or synchronises.  The array of
 * the current device is used, so hip_stream must belong to the current device.  Every call on
 * a device shares that device's array: calls that may overlap on one device (different streams
 * without ordering between them) race on it and must not be issued; calls on one stream, or
 * ordered by events, are safe.  Nothing in it needs to start at zero: each launch writes every
 * partial it reads.  Results equal those of unstep_window_attn given a workspace of at least
 * unstep_attn_workspace_size bytes, bit for bit.  Errors: those of unstep_window_attn, plus
 * E_SHAPE if a split ever needed more than the static array holds, E_HIP if the address lookup
 * fails. */
int unstep_window_attn_noalloc(const unstep_cache* c, int32_t start_frame, int32_t n_frames,
                               int32_t window_frames, const void* q_rot, void* out, float* lse,
                               float softmax_scale, void* hip_stream);

/* ---------------------------------------------------------------------------------
 * One whole chunk step: unstep_kv_append followed by unstep_window_attn on the same
 * stream (q must not be NULL).  All checks of both halves run before anything is
 * enqueued.  Errors: the union of both. */
int unstep_step(unstep_cache* c, int32_t start_frame, int32_t n_frames, int32_t window_frames,
                const void* q, const void* k, const void* v, int64_t tok_stride, int64_t head_stride,
                const float* cos_t, const float* sin_t, void* q_rot, void* out, float* lse,
                float softmax_scale, void* workspace, size_t workspace_bytes, void* hip_stream);

/* ---------------------------------------------------------------------------------
 * Sampler schedule and clean-cache updates (Section 3.4, Equations 1 and 3, and the
 * appendix's shift-five schedule; a later row than the attention step).
 * ------------------------------------------------------------------------------- */

/* Host: the n-step shifted schedule in double precision.  u_i = 1000 (n - i) / n,
 * sigma_i = shift u_i / (1000 + (shift - 1) u_i), t_i = 1000 sigma_i, for i < n_steps
 * (the paper's 4 steps with shift 5 give sigma = 1, 15/16, 5/6, 5/8).  sigma_out, t_out:
 * host double [n_steps].  Errors: E_NULL, E_SHAPE (n_steps < 1), E_RANGE (shift <= 0). */
int unstep_shift_schedule(int32_t n_steps, double shift, double* sigma_out, double* t_out);

/* Equation 1: x_tilde = (1 - sigma) x + sigma eps on n bf16 values (device, 16-byte
 * aligned; x_tilde may alias x).  eps is the caller's N(0, I) draw.  Equation 3:
 * x_next = x_tilde - sigma v.  Arithmetic: each product and the sum/difference in double
 * precision (no fused multiply-add), then rounded to float and to bf16, both
 * nearest-even; sigma = 0 makes both identities (the original clean pass), the clean pass
 * here uses sigma = 0.02.  Errors: E_NULL, E_SHAPE (n < 0), E_RANGE (sigma outside [0, 1]
 * or NaN), E_ALIGN, E_HIP. */
int unstep_renoise(const void* x, const void* eps, double sigma, void* x_tilde, int64_t n, void* hip_stream);
int unstep_emit(const void* x_tilde, const void* v, double sigma, void* x_next, int64_t n, void* hip_stream);

/* ---------------------------------------------------------------------------------
 * DiT call sequence of a clip (Section 3.2, Section 3.4 and Appendix A.2).  A clip is
 * generated in chunks of chunk_frames latent frames; every DiT evaluation of a chunk is one
 * call at noise level sigma and label t: renoise (Equation 1), the DiT with one
 * unstep_step per attention layer, emit (Equation 3).  Steps index the four-step
 * shift-five table (sigma = 1, 15/16, 5/6, 5/8):
 *   UNSTEP_SAMPLER_SELF_FORCING     every chunk 0, 1, 2, 3
 *   UNSTEP_SAMPLER_UNSTEP           chunk 0: 0, 1, 2, 3; later chunks 0 then 2 (odd chunks)
 *                                   or 3 (even chunks), alternating
 *   UNSTEP_SAMPLER_UNSTEP_ONE_STEP  chunk 0: 0, 1, 2, 3; later chunks 0
 * and every chunk ends with one clean-cache call, schedule index UNSTEP_SCHEDULE_CLEAN,
 * t = 0, sigma = clean_sigma (negative selects the variant's own: 0 for Self Forcing, where
 * renoise and emit are identities, 0.02 for UnStep).
 * ------------------------------------------------------------------------------- */
typedef enum {
  UNSTEP_SAMPLER_SELF_FORCING = 0,
  UNSTEP_SAMPLER_UNSTEP = 1,
  UNSTEP_SAMPLER_UNSTEP_ONE_STEP = 2
} unstep_sampler;

#define UNSTEP_SCHEDULE_CLEAN (-1)

/* Host: writes the calls of a clip of n_chunks chunks in order into the caller's arrays
 * of `capacity` entries (chunk index, start frame = chunk * chunk_frames, schedule index,
 * sigma, t) and their count into *n_calls.  *n_calls is set even when the arrays are too
 * small (then E_RANGE and nothing written), so capacity 0 with NULL arrays asks for the
 * count.  Errors: E_NULL (n_calls; an array when calls are written), E_SHAPE
 * (n_chunks < 0, chunk_frames < 1), E_RANGE (unknown variant, clean_sigma above 1 or NaN,
 * frame indices past int32, capacity below the count). */
int unstep_sampler_calls(int32_t variant, int32_t n_chunks, int32_t chunk_frames, double clean_sigma,
                         int32_t capacity, int32_t* n_calls, int32_t* chunk, int32_t* start_frame,
                         int32_t* schedule_index, double* sigma, double* t_label);

/* ---------------------------------------------------------------------------------
 * V/O truncated SVD and the projection after attention (Section 3.5 and Appendix A.4:
 * the value and output weights of layers 8-29 are replaced, once at initialisation, by
 * their rank r = round(0.92 * 1536) = 1413 reconstruction W_r = U_r S_r V_r^T, kept dense
 * in W's shape, so the projection's cost is unchanged).
 * ------------------------------------------------------------------------------- */

/* Init-time: W_r of w (device float32, row-major [rows, cols]) at the given rank, computed
 * in float64 (the leading singular subspace from rocSOLVER's eigendecomposition of the
 * smaller Gram matrix, W_r = W V_r V_r^T, with rocBLAS GEMMs; the paper uses float32, whose
 * rocSOLVER SVD is far less accurate than float32 rounding) and written,
 * rounded to nearest even, to w_r (device float32 [rows, cols]) and/or w_r_bf16 (device
 * bf16, the float32 value rounded again: the paper's cast of the float32 weights); sigma_out (optional host float [min(rows, cols)]) receives the singular
 * values in decreasing order.  w is not modified; w_r may alias w.  Allocates scratch device
 * memory and returns after the work on hip_stream finished.  Errors: E_NULL (w, or both
 * outputs), E_SHAPE (rows or cols < 1, more than 2^28 values), E_RANGE (rank outside
 * [0, min(rows, cols)]), E_ALIGN, E_HIP (including an SVD that did not converge). */
int unstep_svd_truncate(const float* w, int32_t rows, int32_t cols, int32_t rank, float* w_r, void* w_r_bf16,
                        float* sigma_out, void* hip_stream);

/* y = x W^T + b: x bf16 [M, K] (e.g. the attention output [tokens, heads * 128]), w bf16
 * [N, K] (the nn.Linear layout [out, in]), bias bf16 [N] or NULL, y bf16 [M, N]; all
 * row-major and contiguous, on the device.  float32 accumulation and bias add, one rounding to
 * bf16 (nearest even).  One launch of the library's MFMA kernel on hip_stream: no scratch, no
 * allocation, no synchronisation.  Errors: E_NULL (x, w, y), E_SHAPE (sizes < 1, K or N not a
 * multiple of 8, more than 2^31 128 x 128 output tiles), E_ALIGN, E_HIP. */
int unstep_linear(const void* x, const void* w, const void* bias, void* y, int32_t M, int32_t N, int32_t K,
                  void* hip_stream);

/* ---------------------------------------------------------------------------------
 * Measurement reference (not part of the method).
 * ------------------------------------------------------------------------------- */

/* x = a, y = b, z = c for three device buffers of `bytes` bytes each, in one launch with the
 * access pattern of the fused RoPE + append pass (one thread per 16 bytes of each buffer,
 * non-temporal stores): what a plain copy of that pass's bytes reaches, for comparing the
 * pass's bandwidth against.  bytes must be a multiple of 16; pointers 16-byte aligned; the
 * outputs must not overlap the inputs.  Errors: E_NULL, E_SHAPE (bytes < 0 or not a multiple
 * of 16), E_ALIGN, E_HIP. */
int unstep_copy3(const void* a, const void* b, const void* c, void* x, void* y, void* z, int64_t bytes,
                 void* hip_stream);

/* The rate at which this chip's MFMA units run v_mfma_f32_32x32x16_bf16 on bf16 data like the
 * method's, with no other work: `groups` work-groups of 8 waves (one per compute unit, as the
 * attention and projection kernels launch), of which `waves_per_simd` (1: waves 0-3, 2: all 8)
 * per SIMD multiply.  Each multiplying wave runs `mfmas` MFMAs on eight independent
 * accumulators, its operands cycling through eight register sets loaded once from src, with a
 * work-group barrier after every 32.  The chip is power-limited and its clock depends on how
 * much the operand bits toggle: filled with random values of the method's magnitude, src makes
 * the time of this launch the MFMA work alone of a kernel of that shape on such data.
 * src: bf16 (any 16-bit pattern), device, groups * 512 * 256 bytes, lane l of work-group g
 * reading bytes (512 g + l) * 256 .. + 255; sum: fp32, device, groups * 8 values, written with
 * each wave's lane-0 sum of its accumulators (a checksum that keeps every MFMA).  mfmas: a
 * positive multiple of 32.  Errors: E_NULL, E_SHAPE (groups outside [1, 65536], waves_per_simd
 * not 1 or 2, mfmas), E_ALIGN, E_HIP. */
int unstep_mfma_reference(const void* src, float* sum, int32_t groups, int32_t waves_per_simd, int32_t mfmas,
                          void* hip_stream);

#ifdef __cplusplus
}
#endif

#endif /* UNSTEP_H */
