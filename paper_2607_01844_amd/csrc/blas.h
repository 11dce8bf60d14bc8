// Plain dense products through rocBLAS (bf16 operands, fp32 accumulation),
// shared by the vocabulary loss and the router backward.  Internal header.
#pragma once

#include <rocblas/rocblas.h>

#include "common.h"

namespace moe {

constexpr size_t kBlasWs = size_t{32} << 20;  // rocBLAS workspace slice of the caller's (bytes)

// The device's rocBLAS handle, bound to one call's stream and workspace
// slice.  One handle per device, created on first use (atomics off, so
// every product is summed in a fixed order and results repeat bit for bit)
// and kept until the process ends; the handle is not reentrant, so the
// lease holds the device's lock until it goes out of scope.
class BlasLease {
 public:
  BlasLease(hipStream_t s, void* ws);
  ~BlasLease();
  BlasLease(const BlasLease&) = delete;
  BlasLease& operator=(const BlasLease&) = delete;
  hipError_t status() const { return err_; }
  rocblas_handle handle() const { return h_; }

 private:
  void* mu_ = nullptr;
  rocblas_handle h_ = nullptr;
  hipError_t err_ = hipSuccess;
};

inline hipError_t blas_status(rocblas_status st) {
  return st == rocblas_status_success ? hipSuccess : hipErrorUnknown;
}

// C (fp32 or bf16, column-major m x n, ldc) = op(A) op(B) + beta C with
// bf16 A, B and fp32 accumulation; `batch` products at the given element
// strides when batch > 1.
hipError_t gemm_bf16(rocblas_handle h, bool ta, bool tb, int m, int n, int k, const void* A,
                     int lda, int64_t stride_a, const void* B, int ldb, int64_t stride_b,
                     float beta, void* C, bool c_bf16, int ldc, int64_t stride_c, int batch = 1);

}  // namespace moe
