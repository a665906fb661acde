// V/O truncated SVD at wrapper initialisation and the dense projection after attention
// (paper Section 3.5 and Appendix A.4).
//
// unstep_svd_truncate: W (float32, row-major rows x cols) is handed to rocSOLVER as the
// column-major cols x rows matrix B = W^T; B = U S V^T gives W = V S U^T, so the rank-r
// reconstruction of B, written column-major, is W_r row-major.  B_r = (U_r S_r) V_r^T is one
// rocBLAS GEMM.  The leading singular subspace comes from the eigendecomposition of the smaller
// Gram matrix (B^T B or B B^T): W_r = W V_r V_r^T = U_r U_r^T W is the same matrix as
// U_r S_r V_r^T.  The paper works in float32; here the Gram matrix, its eigendecomposition and
// the reconstruction run in float64 (rocSOLVER's float32 SVD of a 1536 x 1536 weight with a
// clustered spectrum was off by ~2.6e-4 sigma_max in its singular values, about a hundred
// times float32 rounding, and its float64 SVD took ~5 s per matrix), and the result is
// rounded to float32 and, optionally, to bf16 (the paper's cast).
// Init-time only: it allocates scratch and synchronises the stream.
//
// unstep_linear: y = x W^T + b in bf16 with float32 accumulation, run by the hand-written MFMA
// kernel of linear.hip (one launch, no scratch, no synchronisation).
#include <hip/hip_runtime.h>
#include <rocblas/rocblas.h>
#include <rocsolver/rocsolver.h>

#include <algorithm>
#include <cmath>
#include <map>
#include <mutex>
#include <tuple>
#include <utility>
#include <vector>

#include "kernels.hpp"
#include "status.hpp"
#include "unstep.h"

using unstep::aligned16;
using unstep::fail;
using unstep::ok;

namespace {

std::mutex g_mu;

int hip_fail(const char* where, hipError_t e) { return fail(UNSTEP_E_HIP, "%s: %s", where, hipGetErrorString(e)); }

// ---- rocBLAS handle per device (rocSOLVER runs on it)
rocblas_handle blas_handle(int dev) {
  static std::map<int, rocblas_handle> handles;
  std::lock_guard<std::mutex> lk(g_mu);
  auto it = handles.find(dev);
  if (it != handles.end()) return it->second;
  rocblas_handle h = nullptr;
  if (rocblas_create_handle(&h) != rocblas_status_success) return nullptr;
  handles[dev] = h;
  return h;
}

template <typename T>
struct DeviceBuffer {
  T* p = nullptr;
  ~DeviceBuffer() {
    if (p) (void)hipFree(p);
  }
  hipError_t alloc(size_t n) { return hipMalloc(reinterpret_cast<void**>(&p), n * sizeof(T)); }
};

}  // namespace

extern "C" {

int unstep_svd_truncate(const float* w, int32_t rows, int32_t cols, int32_t rank, float* w_r, void* w_r_bf16,
                        float* sigma_out, void* hip_stream) {
  return unstep::guarded("unstep_svd_truncate", [&]() -> int {
    const char* where = "unstep_svd_truncate";
    if (!w || (!w_r && !w_r_bf16)) return fail(UNSTEP_E_NULL, "%s: w and one of w_r, w_r_bf16 required", where);
    if (rows < 1 || cols < 1) return fail(UNSTEP_E_SHAPE, "%s: rows and cols must be >= 1", where);
    if (int64_t(rows) * cols > (int64_t(1) << 28)) return fail(UNSTEP_E_SHAPE, "%s: matrix too large", where);
    const int32_t k = rows < cols ? rows : cols;
    if (rank < 0 || rank > k) return fail(UNSTEP_E_RANGE, "%s: rank %d outside [0, %d]", where, rank, k);
    if (!aligned16(w) || (w_r && !aligned16(w_r)) || (w_r_bf16 && !aligned16(w_r_bf16)))
      return fail(UNSTEP_E_ALIGN, "%s: pointers must be 16-byte aligned", where);
    hipStream_t st = static_cast<hipStream_t>(hip_stream);
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(where, e);
    rocblas_handle h = blas_handle(dev);
    if (!h) return fail(UNSTEP_E_HIP, "%s: rocblas_create_handle failed", where);
    std::lock_guard<std::mutex> lk(g_mu);               // the handle's stream is shared state
    if (rocblas_set_stream(h, st) != rocblas_status_success) return fail(UNSTEP_E_HIP, "%s: rocblas_set_stream", where);

    // column-major B = W^T: mb = cols rows, nb = rows columns, ld = cols
    const int32_t mb = cols, nb = rows;
    const size_t n = size_t(rows) * cols;
    const bool right = nb <= mb;                         // Gram of the smaller side: B^T B or B B^T
    DeviceBuffer<double> b, g, d, ework, t1, c64;
    DeviceBuffer<float> out;
    DeviceBuffer<rocblas_int> info;
    if ((e = b.alloc(n)) != hipSuccess || (e = g.alloc(size_t(k) * k)) != hipSuccess || (e = d.alloc(k)) != hipSuccess ||
        (e = ework.alloc(k)) != hipSuccess || (e = t1.alloc(size_t(k) * (right ? mb : nb))) != hipSuccess ||
        (e = c64.alloc(n)) != hipSuccess || (e = info.alloc(1)) != hipSuccess || (!w_r && (e = out.alloc(n)) != hipSuccess))
      return hip_fail(where, e);
    float* c = w_r ? w_r : out.p;
    if ((e = unstep::launch_widen_f64(w, b.p, int64_t(n), st)) != hipSuccess) return hip_fail(where, e);
    const double one = 1.0, zero = 0.0;
    // G = B^T B (k = nb) or B B^T (k = mb), then its eigenvectors in ascending eigenvalue order:
    // the last r columns span the leading right (resp. left) singular subspace of B
    if (rocblas_dsyrk(h, rocblas_fill_upper, right ? rocblas_operation_transpose : rocblas_operation_none, k,
                      right ? mb : nb, &one, b.p, mb, &zero, g.p, k) != rocblas_status_success)
      return fail(UNSTEP_E_HIP, "%s: rocblas_dsyrk failed", where);
    if (rocsolver_dsyevd(h, rocblas_evect_original, rocblas_fill_upper, k, g.p, k, d.p, ework.p, info.p) !=
        rocblas_status_success)
      return fail(UNSTEP_E_HIP, "%s: rocsolver_dsyevd failed", where);
    if (rank == 0) {
      if ((e = hipMemsetAsync(c, 0, n * sizeof(float), st)) != hipSuccess) return hip_fail(where, e);
    } else {
      const double* lead = g.p + size_t(k - rank) * k;   // the r leading singular vectors, ld k
      bool good;
      if (right)   // B_r = (B V_r) V_r^T
        good = rocblas_dgemm(h, rocblas_operation_none, rocblas_operation_none, mb, rank, nb, &one, b.p, mb, lead, k,
                             &zero, t1.p, mb) == rocblas_status_success &&
               rocblas_dgemm(h, rocblas_operation_none, rocblas_operation_transpose, mb, nb, rank, &one, t1.p, mb, lead,
                             k, &zero, c64.p, mb) == rocblas_status_success;
      else         // B_r = U_r (U_r^T B)
        good = rocblas_dgemm(h, rocblas_operation_transpose, rocblas_operation_none, rank, nb, mb, &one, lead, k, b.p,
                             mb, &zero, t1.p, rank) == rocblas_status_success &&
               rocblas_dgemm(h, rocblas_operation_none, rocblas_operation_none, mb, nb, rank, &one, lead, k, t1.p, rank,
                             &zero, c64.p, mb) == rocblas_status_success;
      if (!good) return fail(UNSTEP_E_HIP, "%s: rocBLAS reconstruction failed", where);
      if ((e = unstep::launch_narrow_f32(c64.p, c, int64_t(n), st)) != hipSuccess) return hip_fail(where, e);
    }
    if (w_r_bf16 && (e = unstep::launch_cast_bf16(c, static_cast<uint16_t*>(w_r_bf16), int64_t(n), st)) != hipSuccess)
      return hip_fail(where, e);
    rocblas_int info_h = 0;
    std::vector<double> d_h(sigma_out ? k : 0);
    if ((e = hipMemcpyAsync(&info_h, info.p, sizeof info_h, hipMemcpyDeviceToHost, st)) != hipSuccess)
      return hip_fail(where, e);
    if (sigma_out && (e = hipMemcpyAsync(d_h.data(), d.p, k * sizeof(double), hipMemcpyDeviceToHost, st)) != hipSuccess)
      return hip_fail(where, e);
    if ((e = hipStreamSynchronize(st)) != hipSuccess) return hip_fail(where, e);
    if (info_h != 0) return fail(UNSTEP_E_HIP, "%s: the eigensolver did not converge (info %d)", where, info_h);
    // singular values: square roots of the Gram eigenvalues, largest first
    for (int32_t i = 0; i < int32_t(d_h.size()); ++i) sigma_out[i] = float(std::sqrt(std::max(d_h[k - 1 - i], 0.0)));
    return ok();
  });
}

int unstep_linear(const void* x, const void* w, const void* bias, void* y, int32_t M, int32_t N, int32_t K,
                  void* hip_stream) {
  return unstep::guarded("unstep_linear", [&]() -> int {
    const char* where = "unstep_linear";
    if (!x || !w || !y) return fail(UNSTEP_E_NULL, "%s: x, w and y are required", where);
    if (M < 1 || N < 1 || K < 1) return fail(UNSTEP_E_SHAPE, "%s: M, N, K must be >= 1", where);
    if (K % 8 || N % 8) return fail(UNSTEP_E_SHAPE, "%s: K and N must be multiples of 8", where);
    if ((int64_t(M) + 127) / 128 * ((int64_t(N) + 127) / 128) > INT32_MAX)
      return fail(UNSTEP_E_SHAPE, "%s: too many 128 x 128 output tiles for one launch", where);
    if (!aligned16(x) || !aligned16(w) || !aligned16(y) || (bias && !aligned16(bias)))
      return fail(UNSTEP_E_ALIGN, "%s: pointers must be 16-byte aligned", where);
    hipError_t e = unstep::launch_linear(static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w),
                                         static_cast<const uint16_t*>(bias), static_cast<uint16_t*>(y), M, N, K,
                                         static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return hip_fail(where, e);
    return ok();
  });
}

}  // extern "C"
