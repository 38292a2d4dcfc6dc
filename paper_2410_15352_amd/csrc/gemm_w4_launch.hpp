// Host entry into the persistent four-wave GEMM (kernels_w4.hip, a separate
// translation unit compiled with the machine scheduler off, see gemm_w4.hpp).
#pragma once
#include <hip/hip_runtime.h>

#include "gemm_w4.hpp"

namespace compact {

// True when the persistent kernel handles this problem (see the requirements
// in gemm_w4.hpp); `ldc_cols` lists each segment's (ldc, cols).
bool gemm_w4_eligible(int64_t M, int64_t K, int64_t lda, int64_t ldb, int64_t rows_b, int64_t ldc0,
                      int64_t cols0, int64_t ldc1, int64_t cols1);

// Launches C = A B^T on `stream`, one workgroup per CU (at most one per tile).
hipError_t gemm_w4_launch(const W4Gemm& g, hipStream_t stream);

}  // namespace compact
