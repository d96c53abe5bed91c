// Skinny products (gemm_skinny.hip) and the split reduction they share with
// the GEMM engine (gemm.hip).
#pragma once

#include "gemm_core.h"
#include "internal.h"

namespace mdnn {

// Whether D = op(A) op(B) may run on the skinny kernels: K <= 4 (any
// layout), N <= 4 with A K-contiguous (NN / NT, B staged in 64 KB of LDS;
// N <= 16 when M <= 2048), or TN with N <= 16.  Never while a tile override is set (those force the
// MFMA kernels).  skinny_takes: whether it does, given the workspace.
bool skinny_applies(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K);
bool skinny_takes(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K, const void* ws, size_t ws_bytes);
// Workspace the TN skinny kernel can use for its K split (0: none).
size_t skinny_ws_bytes(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K);
mdnn_status_t gemm_skinny(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                          const void* B, int64_t ldb, mdnn_dtype_t ab_type, mdnn_dtype_t d_type, const Epilogue& ep,
                          void* ws, size_t ws_bytes, hipStream_t st);

// D = epilogue(sum over `splits` fp32 partials [splits][M][N] in ws), summed
// in a fixed order; mask_t / out_t: element types of the mask and of D.
mdnn_status_t reduce_splits_epilogue(const void* ws, int splits, int64_t M, int64_t N, const Epilogue& ep,
                                     mdnn_dtype_t mask_t, mdnn_dtype_t out_t, hipStream_t st);

}  // namespace mdnn
