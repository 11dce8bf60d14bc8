// rocBLAS handle per device and the bf16 product wrapper (see blas.h).
#include "blas.h"

#include <mutex>

namespace moe {
namespace {

constexpr int kMaxDev = 64;
struct Dev {
  std::mutex mu;
  rocblas_handle h = nullptr;
};
Dev& dev_slot(int dev) {
  static Dev d[kMaxDev];
  return d[dev];
}

}  // namespace

BlasLease::BlasLease(hipStream_t s, void* ws) {
  int dev = 0;
  if ((err_ = hipGetDevice(&dev)) != hipSuccess) return;
  if (dev < 0 || dev >= kMaxDev) {
    err_ = hipErrorInvalidDevice;
    return;
  }
  Dev& D = dev_slot(dev);
  D.mu.lock();
  mu_ = &D.mu;
  if (D.h == nullptr) {
    rocblas_handle h = nullptr;
    if ((err_ = blas_status(rocblas_create_handle(&h))) != hipSuccess) return;
    if ((err_ = blas_status(rocblas_set_atomics_mode(h, rocblas_atomics_not_allowed))) !=
        hipSuccess) {
      rocblas_destroy_handle(h);
      return;
    }
    D.h = h;
  }
  h_ = D.h;
  if ((err_ = blas_status(rocblas_set_stream(h_, s))) != hipSuccess) return;
  err_ = blas_status(rocblas_set_workspace(h_, ws, kBlasWs));
}

BlasLease::~BlasLease() {
  if (mu_) static_cast<std::mutex*>(mu_)->unlock();
}

hipError_t gemm_bf16(rocblas_handle h, bool ta, bool tb, int m, int n, int k, const void* A,
                     int lda, int64_t stride_a, const void* B, int ldb, int64_t stride_b,
                     float beta, void* C, bool c_bf16, int ldc, int64_t stride_c, int batch) {
  const float alpha = 1.0f;
  const rocblas_datatype ct = c_bf16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
  const rocblas_operation oa = ta ? rocblas_operation_transpose : rocblas_operation_none;
  const rocblas_operation ob = tb ? rocblas_operation_transpose : rocblas_operation_none;
  if (batch <= 1)
    return blas_status(rocblas_gemm_ex(h, oa, ob, m, n, k, &alpha, A, rocblas_datatype_bf16_r, lda,
                                       B, rocblas_datatype_bf16_r, ldb, &beta, C, ct, ldc, C, ct,
                                       ldc, rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0,
                                       0));
  return blas_status(rocblas_gemm_strided_batched_ex(
      h, oa, ob, m, n, k, &alpha, A, rocblas_datatype_bf16_r, lda, stride_a, B,
      rocblas_datatype_bf16_r, ldb, stride_b, &beta, C, ct, ldc, stride_c, C, ct, ldc, stride_c,
      batch, rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0, 0));
}

}  // namespace moe
