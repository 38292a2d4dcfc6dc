// Host entries into the kernels of kernels_w4.hip, a separate translation
// unit compiled with the machine scheduler off (their K steps are written in
// issue order): the persistent four-wave GEMM (gemm_w4.hpp), the split-K
// G^ kernel (gemm_ghat.hpp) and the decompression (gemm_dec.hpp).
#pragma once
#include <hip/hip_runtime.h>

#include "gemm_dec.hpp"
#include "gemm_ghat.hpp"
#include "gemm_w4.hpp"

namespace compact {

// True when the persistent kernel handles this problem (see the requirements
// in gemm_w4.hpp): each output segment's (ldc, cols); b_tiled: B is the
// K-tiled operand this library stages (needed when K % 8 != 0).
bool gemm_w4_eligible(int64_t M, int64_t K, int64_t lda, int64_t ldb, int64_t rows_b, int64_t ldc0,
                      int64_t cols0, int64_t ldc1, int64_t cols1, bool b_tiled);

// Which pass a launch serves (each has its own kernel instantiation).
enum class W4Use { kForward, kDx };

// Launches C = A B^T on `stream`, one workgroup per CU (at most one per tile).
hipError_t gemm_w4_launch(const W4Gemm& g, W4Use use, hipStream_t stream);

// G^ partials: one workgroup per (split, layer, column tile, row tile).
hipError_t ghat_w4_launch(const GhatW4Params& p, hipStream_t stream);

// True when the decompression kernel takes a layer of this shape and layout.
bool dec_w4_eligible(int64_t n, int64_t m, int64_t r, int64_t ldw, int64_t ldn, int64_t ldpt, bool w_f32);

// W <- W - coef P N for every layer of the batch: one workgroup per 128 x 128
// tile of W (begin[] holds each layer's first workgroup).
hipError_t dec_w4_launch(const DecW4Batch& d, bool w_f32, hipStream_t stream);

}  // namespace compact
