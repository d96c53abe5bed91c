// Winograd minimal filtering F(2x2, 3x3) for 3x3 forward convolutions: the
// alternative convolution algorithm of section 2.1 (the algorithm is chosen
// per layer), following Lavin and Gray's fast algorithm for small filters.
//
//   U[xi][k][c] = (G g_kc G^T)[xi]                 filter transform
//   V[xi][t][c] = (B^T d_tc B)[xi]                 input transform (t: 2x2 output tile,
//                                                  d: its 4x4 input window)
//   M[xi][t][k] = sum_c V[xi][t][c] U[xi][k][c]    16 products, one batched MFMA launch
//   y(tile t)[k] = A^T M_tk A (+ bias, ReLU)       output transform
//
// The transforms run in fp32 and are rounded once to the storage type (U, V)
// for the matrix cores; M stays fp32.  For 16-bit inputs the input transform
// is exact in fp32 (sums of at most four inputs); the filter transform sums
// at most nine taps scaled by 1/4.  Relative to the implicit GEMM this trades
// 2.25x fewer multiply-adds for three extra passes over HBM (V and M are four
// times the size of the input and output).
#include "conv_small.h"
#include "gemm_launch.h"

namespace mdnn {
namespace {

size_t seg(size_t b) { return (b + 255) & ~(size_t)255; }

// base[off] if ok, else 0; the load is unconditional (clamped address), so a
// thread's sixteen window loads are in flight together.
template <class T>
__device__ __forceinline__ float ldz(const typename T::storage* base, int64_t off, bool ok) {
  const float v = to_f<T>(base[ok ? off : 0]);
  return ok ? v : 0.0f;
}

// One thread per (k, c): 9 taps (stride C in KRSC) -> 16 transformed values.
template <class T>
__global__ void __launch_bounds__(256)
wino_filter_kernel(const typename T::storage* __restrict__ w, typename T::storage* __restrict__ U, int K, int C) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)K * C) return;
  const int64_t k = idx / C, c = idx - k * C;
  float g[3][3];
#pragma unroll
  for (int r = 0; r < 3; ++r)
#pragma unroll
    for (int s = 0; s < 3; ++s) g[r][s] = to_f<T>(w[((k * 3 + r) * 3 + s) * C + c]);
  float t[4][3];  // G g
#pragma unroll
  for (int s = 0; s < 3; ++s) {
    t[0][s] = g[0][s];
    t[1][s] = 0.5f * (g[0][s] + g[1][s] + g[2][s]);
    t[2][s] = 0.5f * (g[0][s] - g[1][s] + g[2][s]);
    t[3][s] = g[2][s];
  }
  const int64_t KC = (int64_t)K * C;
#pragma unroll
  for (int a = 0; a < 4; ++a) {  // (G g) G^T
    const float u[4] = {t[a][0], 0.5f * (t[a][0] + t[a][1] + t[a][2]), 0.5f * (t[a][0] - t[a][1] + t[a][2]), t[a][2]};
#pragma unroll
    for (int b = 0; b < 4; ++b) U[(a * 4 + b) * KC + idx] = from_f<T>(u[b]);
  }
}

// One thread per (tile t, channel c): the 4x4 window (zero outside the
// image) -> 16 transformed values.
template <class T>
__global__ void __launch_bounds__(256)
wino_input_kernel(const typename T::storage* __restrict__ x, typename T::storage* __restrict__ V, ConvGeom g, int th,
                  int tw, int64_t tiles) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t TC = tiles * g.c;
  if (idx >= TC) return;
  const int64_t t = idx / g.c;
  const int c = (int)(idx - t * g.c);
  const int64_t n = t / ((int64_t)th * tw);
  const int rem = (int)(t - n * th * tw);
  const int i = rem / tw, j = rem - i * tw;
  const int y0 = 2 * i - g.pad, x0 = 2 * j - g.pad;
  float d[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int yy = y0 + a, xx = x0 + b;
      const bool ok = yy >= 0 && yy < g.h && xx >= 0 && xx < g.w;
      d[a][b] = ldz<T>(x, ((n * g.h + yy) * g.w + xx) * g.c + c, ok);
    }
  float s[4][4];  // B^T d
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    s[0][b] = d[0][b] - d[2][b];
    s[1][b] = d[1][b] + d[2][b];
    s[2][b] = d[2][b] - d[1][b];
    s[3][b] = d[1][b] - d[3][b];
  }
#pragma unroll
  for (int a = 0; a < 4; ++a) {  // (B^T d) B
    const float v[4] = {s[a][0] - s[a][2], s[a][1] + s[a][2], s[a][2] - s[a][1], s[a][1] - s[a][3]};
#pragma unroll
    for (int b = 0; b < 4; ++b) V[(a * 4 + b) * TC + idx] = from_f<T>(v[b]);
  }
}

// One thread per (tile t, output channel k): 16 products -> the 2x2 outputs.
template <class OutT>
__global__ void __launch_bounds__(256)
wino_output_kernel(const float* __restrict__ Mp, typename OutT::storage* __restrict__ y, const float* __restrict__ bias,
                   int act, ConvGeom g, int th, int tw, int64_t tiles) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t TK = tiles * g.k;
  if (idx >= TK) return;
  const int64_t t = idx / g.k;
  const int k = (int)(idx - t * g.k);
  const int64_t n = t / ((int64_t)th * tw);
  const int rem = (int)(t - n * th * tw);
  const int i = rem / tw, j = rem - i * tw;
  float m[4][4];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < 4; ++b) m[a][b] = Mp[(a * 4 + b) * TK + idx];
  float s[2][4];  // A^T m
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    s[0][b] = m[0][b] + m[1][b] + m[2][b];
    s[1][b] = m[1][b] - m[2][b] - m[3][b];
  }
  const float bk = bias ? bias[k] : 0.0f;
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    const float yq[2] = {s[p][0] + s[p][1] + s[p][2], s[p][1] - s[p][2] - s[p][3]};  // (A^T m) A
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int oy = 2 * i + p, ox = 2 * j + q;
      if (oy < g.ho && ox < g.wo) {
        float v = yq[q] + bk;
        if (act == MDNN_ACT_RELU) v = relu_f(v);
        y[((n * g.ho + oy) * g.wo + ox) * g.k + k] = from_f<OutT>(v);
      }
    }
  }
}

struct WinoPlan {
  int th, tw;
  int64_t tiles;
  size_t u_off, v_off, m_off, total;
};

WinoPlan wino_plan(const ConvGeom& g, size_t es) {
  WinoPlan p;
  p.th = (g.ho + 1) / 2;
  p.tw = (g.wo + 1) / 2;
  p.tiles = (int64_t)g.n * p.th * p.tw;
  p.u_off = 0;
  p.v_off = seg((size_t)16 * g.k * g.c * es);
  p.m_off = p.v_off + seg((size_t)16 * p.tiles * g.c * es);
  p.total = p.m_off + seg((size_t)16 * p.tiles * g.k * sizeof(float));
  return p;
}

template <class T>
mdnn_status_t wino_run(const ConvGeom& g, const void* x, const void* w, const float* bias, mdnn_act_t act, void* y,
                       mdnn_dtype_t y_type, char* ws, const WinoPlan& p, hipStream_t st) {
  typedef typename T::storage S;
  S* U = (S*)(ws + p.u_off);
  S* V = (S*)(ws + p.v_off);
  float* Mp = (float*)(ws + p.m_off);
  const int64_t KC = (int64_t)g.k * g.c, TC = p.tiles * g.c, TK = p.tiles * g.k;
  if (ceil_div(TC, 256) > 0x7fffffffLL || ceil_div(TK, 256) > 0x7fffffffLL || ceil_div(p.tiles, 64) > 0x7fffffffLL)
    return fail(MDNN_ERR_SHAPE, "winograd: problem too large for the launch grid");
  hipLaunchKernelGGL((wino_filter_kernel<T>), dim3((unsigned)ceil_div(KC, 256)), dim3(256), 0, st, (const S*)w, U, g.k,
                     g.c);
  hipLaunchKernelGGL((wino_input_kernel<T>), dim3((unsigned)ceil_div(TC, 256)), dim3(256), 0, st, (const S*)x, V, g,
                     p.th, p.tw, p.tiles);
  MDNN_TRY(check_launch("winograd transforms"));
  // M[xi] (tiles x K) = V[xi] (tiles x C) U[xi]^T, xi = grid z
  const bool vec = g.c % 8 == 0;
  SrcMatK<uint16_t> a{(const uint16_t*)V, g.c, p.tiles, g.c, vec};
  a.bs = TC;
  SrcMatK<uint16_t> b{(const uint16_t*)U, g.c, g.k, g.c, vec};
  b.bs = KC;
  Epilogue ep{};
  ep.alpha = 1.0f;
  ep.D = Mp;
  ep.ldd = g.k;
  ep.act = MDNN_ACT_NONE;
  ep.vec4 = g.k % 4 == 0;
  ep.bstride_d = TK;
  if (g.k <= 64) {
    const dim3 grid((unsigned)(ceil_div(p.tiles, 64) * ceil_div(g.k, 64)), 1, 16);
    hipLaunchKernelGGL((gemm_mfma_kernel<T, F32, SrcMatK<uint16_t>, SrcMatK<uint16_t>, 64, 64, 1, 2>), grid, dim3(128),
                       0, st, a, b, p.tiles, (int64_t)g.k, (int64_t)g.c, ep);
  } else {
    const dim3 grid((unsigned)(ceil_div(p.tiles, 128) * ceil_div(g.k, 128)), 1, 16);
    hipLaunchKernelGGL((gemm_mfma_kernel<T, F32, SrcMatK<uint16_t>, SrcMatK<uint16_t>, 128, 128, 2, 2>), grid,
                       dim3(256), 0, st, a, b, p.tiles, (int64_t)g.k, (int64_t)g.c, ep);
  }
  MDNN_TRY(check_launch("winograd products"));
  const dim3 og((unsigned)ceil_div(TK, 256));
  if (y_type == MDNN_F32)
    hipLaunchKernelGGL((wino_output_kernel<F32>), og, dim3(256), 0, st, (const float*)Mp, (float*)y, bias, (int)act, g,
                       p.th, p.tw, p.tiles);
  else
    hipLaunchKernelGGL((wino_output_kernel<T>), og, dim3(256), 0, st, (const float*)Mp, (S*)y, bias, (int)act, g, p.th,
                       p.tw, p.tiles);
  return check_launch("winograd output transform");
}

}  // namespace
}  // namespace mdnn

using namespace mdnn;

extern "C" size_t mdnn_conv2d_fwd_winograd_workspace(const mdnn_conv_shape_t* shape, mdnn_dtype_t io_type) {
  ConvGeom g;
  if (check_conv_shape(shape, g) != MDNN_SUCCESS || g.r != 3 || g.s != 3 ||
      (io_type != MDNN_F16 && io_type != MDNN_BF16))
    return 0;
  clear_error();
  return wino_plan(g, dtype_size(io_type)).total;
}

extern "C" mdnn_status_t mdnn_conv2d_fwd_winograd(const mdnn_conv_shape_t* shape, const void* x, const void* w,
                                                  mdnn_dtype_t io_type, const float* bias, mdnn_act_t act, void* y,
                                                  mdnn_dtype_t y_type, void* workspace, size_t ws_bytes,
                                                  mdnn_stream_t stream) {
  ConvGeom g;
  MDNN_TRY(check_conv_shape(shape, g));
  if (g.r != 3 || g.s != 3) return fail(MDNN_ERR_SHAPE, "winograd: F(2x2,3x3) needs a 3x3 filter");
  if (io_type != MDNN_F16 && io_type != MDNN_BF16)
    return fail(MDNN_ERR_DTYPE, "winograd: io_type must be fp16 or bf16");
  if (y_type != MDNN_F32 && y_type != io_type) return fail(MDNN_ERR_DTYPE, "winograd: y_type must be fp32 or io_type");
  if (act != MDNN_ACT_NONE && act != MDNN_ACT_RELU) return fail(MDNN_ERR_DTYPE, "winograd: unknown act");
  if (g.n == 0) return MDNN_SUCCESS;
  if (!x || !w || !y) return fail(MDNN_ERR_NULL, "winograd: x, w and y are required");
  const size_t es = dtype_size(io_type);
  if (!aligned(x, es) || !aligned(w, es) || !aligned(y, dtype_size(y_type)) || (bias && !aligned(bias, 4)))
    return fail(MDNN_ERR_MISALIGNED, "winograd: misaligned base pointer");
  const WinoPlan p = wino_plan(g, es);
  if (!workspace || ws_bytes < p.total || !aligned(workspace, 256))
    return fail(MDNN_ERR_WORKSPACE, "winograd: needs %zu bytes of 256-byte aligned workspace", p.total);
  clear_error();
  hipStream_t st = as_stream(stream);
  if (io_type == MDNN_F16) return wino_run<F16>(g, x, w, bias, act, y, y_type, (char*)workspace, p, st);
  return wino_run<BF16>(g, x, w, bias, act, y, y_type, (char*)workspace, p, st);
}
