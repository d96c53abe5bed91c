// Convolutions on the pipelined MFMA mainloop (gemm_lds.h).  Each entry
// returns MDNN_SUCCESS with *done = false, having launched nothing, when the
// shape or the pointers do not meet that kernel's preconditions; the caller
// then runs the general implicit-GEMM kernel.
#pragma once

#include "gemm_core.h"
#include "internal.h"

namespace mdnn {

// Forward: y = epilogue(im2col(x) . w^T), M = n*ho*wo, N = c_out, K = r*s*c_in.
// Needs c_in % 32 == 0 (one tap per K step when c_in % 64 == 0, else two
// 32-channel half blocks per step with K padded), 16-byte aligned x and w,
// x (and, for c_in % 64 != 0, w) below 2^31 bytes.
mdnn_status_t conv_pipe_fwd(const ConvGeom& g, const void* x, const void* w, const Epilogue& ep,
                            mdnn_dtype_t io, mdnn_dtype_t out, hipStream_t st, bool* done);

// Backward data: dx = epilogue(im2col'(dy) . w'), M = n*h*w, N = c_in,
// K = r*s*c_out (mirrored taps).  Needs c_out % 64 == 0, c_in % 8 == 0,
// 16-byte aligned dy and w, dy below 2^31 bytes.
mdnn_status_t conv_pipe_bwd_data(const ConvGeom& g, const void* dy, const void* w, const Epilogue& ep,
                                 mdnn_dtype_t io, mdnn_dtype_t out, hipStream_t st, bool* done);

// Split plan of the pipelined backward-filter GEMM (M = c_out,
// N = r*s*c_in, K = n*ho*wo), or splits == 0 when the shape is not eligible:
// a size-preserving convolution with c_in, c_out multiples of 8, K a
// multiple of 64, x below 2^31 bytes.  A function of the shape only.
SplitPlan conv_pipe_filter_plan(const ConvGeom& g);

// Backward filter into fp32 dw[c_out][r*s*c_in]; split partials go to `ws`
// (conv_pipe_filter_plan(g).splits * M * N floats when splits > 1), their
// sum into `defer` when one is given.
mdnn_status_t conv_pipe_bwd_filter(const ConvGeom& g, const void* x, const void* dy, float* dw, void* ws,
                                   mdnn_dtype_t io, hipStream_t st, bool* done, ReduceBatch* defer = nullptr);

}  // namespace mdnn
