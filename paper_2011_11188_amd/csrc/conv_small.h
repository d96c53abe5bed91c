// Direct kernels for convolutions whose reduction is tiny (conv_small.hip).
#pragma once

#include "gemm_core.h"
#include "internal.h"

namespace mdnn {

// Validates a convolution shape (sizes, output not empty, ranges) into g.
mdnn_status_t check_conv_shape(const mdnn_conv_shape_t* s, ConvGeom& g);

// Forward with K = r*s*c_in <= 64 and c_out <= 256: any storage type, any
// epilogue (bias, ReLU, output type).
bool conv_small_fwd_ok(const ConvGeom& g);
mdnn_status_t conv_small_fwd(const ConvGeom& g, const void* x, const void* w, const Epilogue& ep, mdnn_dtype_t io,
                             mdnn_dtype_t out, hipStream_t st);

// Filter gradient with r*s*c_in <= 64 and c_out * r*s*c_in <= 1024: number
// of pixel blocks (the partials it writes:
// blocks * c_out * r*s*c_in floats), or 0 when the shape does not qualify.
int64_t conv_small_filter_blocks(const ConvGeom& g, mdnn_dtype_t io);
// dw = sum over pixel blocks of the partials in ws (fixed order; the sum
// goes into `defer` when one is given).
mdnn_status_t conv_small_filter(const ConvGeom& g, const void* x, const void* dy, float* dw, void* ws,
                                mdnn_dtype_t io, hipStream_t st, ReduceBatch* defer = nullptr);

}  // namespace mdnn
