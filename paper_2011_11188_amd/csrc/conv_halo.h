// 3x3 convolutions of 64 input channels (stride 1, zero padding 1, output
// the size of the input) whose input tile, with its one-pixel border, is
// staged in LDS once and read by all nine taps from there.
#pragma once

#include "gemm_core.h"
#include "internal.h"

namespace mdnn {

// Forward y = conv(x, w) (bwd false; src = x) or backward data
// dx = conv(dy, w flipped, channel axes swapped) (bwd true; src = dy) with
// the epilogue `ep` (bias, ReLU, mask, 16-bit or fp32 output) when the shape
// qualifies: 16-bit data, 3x3 filter, padding 1, 64 channels in the
// convolved tensor, output channels a multiple of 64, 16-byte aligned
// operands, and whole image rows (or whole images) of 256 output pixels per
// workgroup.  *done stays false when the shape does not qualify (the caller
// takes another kernel).
mdnn_status_t conv_halo(const ConvGeom& g, bool bwd, const void* src, const void* w, const Epilogue& ep,
                        mdnn_dtype_t io, mdnn_dtype_t out, hipStream_t st, bool* done);

}  // namespace mdnn
