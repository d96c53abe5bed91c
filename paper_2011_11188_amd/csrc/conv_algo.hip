// Forward convolution with a selectable algorithm (section 2.1: the
// convolution algorithm behind one operation is interchangeable, chosen per
// layer).  Three algorithms compute the same y:
//   implicit GEMM  (mdnn_conv2d_fwd): im2col is never stored, the GEMM
//                  loaders gather its rows from x;
//   im2col + GEMM  the im2col matrix [n*Ho*Wo][r*s*c_in] is written to the
//                  workspace once, then one plain GEMM (NT against the
//                  filter stored [c_out][r*s*c_in]) with the bias / ReLU
//                  epilogue;
//   Winograd F(2x2,3x3) (mdnn_conv2d_fwd_winograd): fewer multiplications,
//                  two more operand roundings (outside the 1e-4 bar).
// The automatic choice is a fixed table of per-shape measurements on MI355X
// restricted to the two algorithms that meet the implicit GEMM's accuracy,
// and to what fits the caller's workspace.
#include "gemm_launch.h"
#include "internal.h"

namespace mdnn {

mdnn_status_t check_conv_shape(const mdnn_conv_shape_t* s, ConvGeom& g);

namespace {

// col[m][kk] = x[n, i + tr - pad, j + ts - pad, ch], zero outside the image,
// for m = (n, i, j) over the output grid and kk = (tr, ts, ch).  Each thread
// copies V consecutive channels of one tap of one output pixel (16 bytes when
// the channel count allows it).
template <class S, int V>
__global__ void __launch_bounds__(256)
im2col_kernel(ConvGeom g, const S* __restrict__ x, S* __restrict__ col, int64_t total) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= total) return;
  const int32_t cb_n = g.c / V, taps = g.r * g.s;
  const int32_t cb = (int32_t)(idx % cb_n);
  const int64_t t = idx / cb_n;
  const int32_t tap = (int32_t)(t % taps);
  const int64_t m = t / taps;
  const int32_t j = (int32_t)(m % g.wo);
  const int64_t q = m / g.wo;
  const int32_t i = (int32_t)(q % g.ho), n = (int32_t)(q / g.ho);
  const int32_t tr = tap / g.s, ts = tap - tr * g.s;
  const int32_t hi = i + tr - g.pad, wi = j + ts - g.pad;
  const int64_t K = (int64_t)taps * g.c;
  S* dst = col + m * K + (int64_t)tap * g.c + (int64_t)cb * V;
  const bool in = hi >= 0 && hi < g.h && wi >= 0 && wi < g.w;
  const S* src = x + (((int64_t)n * g.h + hi) * g.w + wi) * g.c + (int64_t)cb * V;
  if constexpr (V * sizeof(S) == 16) {
    *(uint4*)dst = in ? *(const uint4*)src : make_uint4(0, 0, 0, 0);
  } else {
#pragma unroll
    for (int e = 0; e < V; ++e) dst[e] = in ? src[e] : (S)0;
  }
}

template <class S>
mdnn_status_t launch_im2col(const ConvGeom& g, const void* x, void* col, hipStream_t st) {
  constexpr int VV = 16 / (int)sizeof(S);
  const bool vec = g.c % VV == 0 && aligned(x, 16) && aligned(col, 16);
  const int64_t M = (int64_t)g.n * g.ho * g.wo, taps = (int64_t)g.r * g.s;
  const int64_t total = M * taps * (vec ? g.c / VV : g.c);
  const int64_t blocks = ceil_div(total, 256);
  if (blocks > 0x7fffffffLL) return fail(MDNN_ERR_SHAPE, "im2col: problem too large for the launch grid");
  if (vec)
    hipLaunchKernelGGL((im2col_kernel<S, VV>), dim3((unsigned)blocks), dim3(256), 0, st, g, (const S*)x, (S*)col,
                       total);
  else
    hipLaunchKernelGGL((im2col_kernel<S, 1>), dim3((unsigned)blocks), dim3(256), 0, st, g, (const S*)x, (S*)col,
                       total);
  return check_launch("im2col_kernel");
}

size_t im2col_bytes(const ConvGeom& g, mdnn_dtype_t io) {
  const size_t M = (size_t)g.n * g.ho * g.wo, K = (size_t)g.r * g.s * g.c;
  return (M * K * dtype_size(io) + 255) & ~(size_t)255;
}

// The automatic choice.  Forward timings on MI355X at the workloads' batch
// sizes (microseconds; implicit GEMM / im2col + GEMM / Winograd):
//   5x5,   1 ->  32 at 28x28, n 256 (bf16, bias+ReLU):  27.0 /  67.8 /   -
//   5x5,  32 ->  64 at 14x14, n 256 (bf16, bias+ReLU):  17.4 /  50.5 /   -
//   3x3,  64 ->  64 at 32x32, n 128 (fp16):             20.2 /  74.5 / 88.2
//   3x3, 128 -> 128 at 16x16, n 128 (fp16):             15.6 /  47.4 / 57.4
//   3x3, 256 -> 256 at  8x8,  n 128 (fp16):             22.1 /  36.0 / 37.5
// The stored im2col matrix is r*s times the input, written once and read
// back by the GEMM: at these sizes that traffic costs more than the implicit
// GEMM's per-tap gathers through L2, so every entry is the implicit GEMM.
// im2col + GEMM is picked only where it measured faster and its workspace
// is given; every shape not in the table runs the implicit GEMM (no
// workspace, no extra HBM pass).
struct Choice {
  int32_t h, w, c_in, c_out, r, s, pad;
  mdnn_conv_algo_t algo;
};
constexpr Choice kChoices[] = {
    {28, 28, 1, 32, 5, 5, 2, MDNN_CONV_IMPLICIT_GEMM},
    {14, 14, 32, 64, 5, 5, 2, MDNN_CONV_IMPLICIT_GEMM},
    {32, 32, 64, 64, 3, 3, 1, MDNN_CONV_IMPLICIT_GEMM},
    {16, 16, 128, 128, 3, 3, 1, MDNN_CONV_IMPLICIT_GEMM},
    {8, 8, 256, 256, 3, 3, 1, MDNN_CONV_IMPLICIT_GEMM},
};

}  // namespace
}  // namespace mdnn

using namespace mdnn;

extern "C" size_t mdnn_conv2d_fwd_algo_workspace(const mdnn_conv_shape_t* shape, mdnn_dtype_t io_type,
                                                 mdnn_conv_algo_t algo) {
  ConvGeom g;
  if (check_conv_shape(shape, g) != MDNN_SUCCESS || !dtype_ok(io_type)) return 0;
  switch (algo) {
    case MDNN_CONV_IM2COL_GEMM: return im2col_bytes(g, io_type);
    case MDNN_CONV_WINOGRAD: return mdnn_conv2d_fwd_winograd_workspace(shape, io_type);
    default: return 0;
  }
}

extern "C" mdnn_conv_algo_t mdnn_conv2d_fwd_choose(const mdnn_conv_shape_t* shape, mdnn_dtype_t io_type,
                                                   size_t ws_bytes) {
  ConvGeom g;
  if (check_conv_shape(shape, g) != MDNN_SUCCESS || !dtype_ok(io_type)) return MDNN_CONV_IMPLICIT_GEMM;
  for (const Choice& c : kChoices) {
    if (c.h == g.h && c.w == g.w && c.c_in == g.c && c.c_out == g.k && c.r == g.r && c.s == g.s &&
        c.pad == g.pad) {
      if (c.algo == MDNN_CONV_IM2COL_GEMM && ws_bytes < im2col_bytes(g, io_type)) break;
      return c.algo;
    }
  }
  return MDNN_CONV_IMPLICIT_GEMM;
}

extern "C" mdnn_status_t mdnn_conv2d_fwd_algo(const mdnn_conv_shape_t* shape, const void* x, const void* w,
                                              mdnn_dtype_t io_type, const float* bias, mdnn_act_t act, void* y,
                                              mdnn_dtype_t y_type, mdnn_conv_algo_t algo, void* workspace,
                                              size_t ws_bytes, mdnn_stream_t stream) {
  if (algo == MDNN_CONV_AUTO) algo = mdnn_conv2d_fwd_choose(shape, io_type, ws_bytes);
  switch (algo) {
    case MDNN_CONV_IMPLICIT_GEMM:
      return mdnn_conv2d_fwd(shape, x, w, io_type, bias, act, y, y_type, stream);
    case MDNN_CONV_WINOGRAD:
      return mdnn_conv2d_fwd_winograd(shape, x, w, io_type, bias, act, y, y_type, workspace, ws_bytes, stream);
    case MDNN_CONV_IM2COL_GEMM:
      break;
    default:
      return fail(MDNN_ERR_DTYPE, "conv fwd: unknown algorithm %d", (int)algo);
  }
  ConvGeom g;
  MDNN_TRY(check_conv_shape(shape, g));
  if (!dtype_ok(io_type) || !dtype_ok(y_type) || (y_type != MDNN_F32 && y_type != io_type))
    return fail(MDNN_ERR_DTYPE, "conv fwd (im2col): y_type must be fp32 or io_type");
  if (act != MDNN_ACT_NONE && act != MDNN_ACT_RELU) return fail(MDNN_ERR_DTYPE, "conv fwd (im2col): unknown act");
  if (g.n == 0) return MDNN_SUCCESS;
  if (!x || !w || !y) return fail(MDNN_ERR_NULL, "conv fwd (im2col): x, w and y are required");
  const size_t es = dtype_size(io_type);
  if (!aligned(x, es) || !aligned(w, es) || !aligned(y, dtype_size(y_type)) || (bias && !aligned(bias, 4)))
    return fail(MDNN_ERR_MISALIGNED, "conv fwd (im2col): misaligned base pointer");
  const size_t need = im2col_bytes(g, io_type);
  if (!workspace || ws_bytes < need || !aligned(workspace, 256))
    return fail(MDNN_ERR_WORKSPACE, "conv fwd (im2col): needs %zu bytes of 256-byte aligned workspace", need);
  clear_error();
  hipStream_t st = as_stream(stream);
  switch (io_type) {
    case MDNN_F32: MDNN_TRY(launch_im2col<float>(g, x, workspace, st)); break;
    default: MDNN_TRY(launch_im2col<uint16_t>(g, x, workspace, st)); break;
  }
  const int64_t M = (int64_t)g.n * g.ho * g.wo, K = (int64_t)g.r * g.s * g.c;
  // y[M][c_out] = col[M][K] * w[c_out][K]^T  (+ bias, ReLU) on the GEMM engine
  return gemm_mixed_ws(MDNN_NT, M, g.k, K, 1.0f, workspace, K, w, K, io_type, 0.0f, nullptr, 0, y, g.k, y_type,
                       bias, act, nullptr, 0, nullptr, 0, stream);
}
