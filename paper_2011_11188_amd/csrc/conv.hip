// 2-D convolution entry points: implicit GEMM on the shared MFMA engine.
//   fwd:        M = n*Ho*Wo, N = c_out, K = r*s*c_in   (A = im2col(x), B = w as [c_out][K])
//   bwd_data:   M = n*h*w,   N = c_in,  K = r*s*c_out  (A = im2col of dy with flipped taps, B = w)
//   bwd_filter: M = c_out,   N = r*s*c_in, K = n*Ho*Wo (A = dy^T, B = shifted x), split over K
// No im2col buffer is materialised: the operand sources compute addresses.
#include <mutex>

#include "conv_halo.h"
#include "conv_pipe.h"
#include "conv_small.h"
#include "gemm_launch.h"

namespace mdnn {

mdnn_status_t check_conv_shape(const mdnn_conv_shape_t* s, ConvGeom& g) {
  if (!s) return fail(MDNN_ERR_NULL, "conv: shape is NULL");
  if (s->n < 0 || s->h < 1 || s->w < 1 || s->c_in < 1 || s->c_out < 1 || s->r < 1 || s->s < 1 ||
      s->pad < 0)
    return fail(MDNN_ERR_SHAPE, "conv: sizes must be positive (n >= 0, pad >= 0)");
  const int64_t ho = s->h + 2 * s->pad - s->r + 1, wo = s->w + 2 * s->pad - s->s + 1;
  if (ho < 1 || wo < 1) return fail(MDNN_ERR_SHAPE, "conv: empty output");
  const int64_t lim = 0x7fffffffLL;
  if (s->h > lim || s->w > lim || s->c_in > lim || s->c_out > lim || s->r > 64 || s->s > 64 ||
      s->pad > 64 || s->n > lim)
    return fail(MDNN_ERR_SHAPE, "conv: size out of range");
  g = ConvGeom{(int32_t)s->n, (int32_t)s->h, (int32_t)s->w, (int32_t)s->c_in, (int32_t)s->c_out,
               (int32_t)s->r, (int32_t)s->s, (int32_t)s->pad, (int32_t)ho, (int32_t)wo};
  return MDNN_SUCCESS;
}

// The pipelined kernels run unless a general tile is forced (tests of the
// general path).
static bool pipe_allowed() {
  const int o = gemm_tile_override();
  return !(o >= TILE_256x256 && o <= TILE_64x64);
}
// the halo kernel for the 3x3 layers it takes unless a kernel family is
// forced (forcing the pipelined kernels runs the implicit GEMM there too)
static bool halo_allowed() { return gemm_tile_override() == TILE_AUTO; }

static Epilogue plain_epilogue(void* D, int64_t ldd, mdnn_dtype_t d_type) {
  Epilogue ep{};
  ep.alpha = 1.0f;
  ep.beta = 0.0f;
  ep.D = D;
  ep.ldd = ldd;
  ep.act = MDNN_ACT_NONE;
  ep.vec4 = (ldd % 4 == 0) && aligned(D, 4 * dtype_size(d_type));
  return ep;
}

template <class T, class OutT, class SrcA, class SrcB>
static mdnn_status_t conv_run(const SrcA& a, const SrcB& b, int64_t M, int64_t N, int64_t K,
                              const Epilogue& ep, int splits, hipStream_t st) {
  if constexpr (sizeof(typename T::storage) == 4)
    return run_gemm32(a, b, M, N, K, ep, splits, st);
  else
    return run_gemm16<T, OutT>(a, b, M, N, K, ep, splits, st);
}

template <class T>
static mdnn_status_t fwd_impl(const ConvGeom& g, const void* x, const void* w, const Epilogue& ep,
                              mdnn_dtype_t y_type, hipStream_t st) {
  typedef typename T::storage S;
  const int64_t M = (int64_t)g.n * g.ho * g.wo, N = g.k, K = (int64_t)g.r * g.s * g.c;
  const bool vx = aligned(x, 16) && g.c % 8 == 0;
  const bool vw = aligned(w, 16) && K % 8 == 0;
  SrcConvFwdA<S> a{(const S*)x, g, M, K, vx};
  SrcMatK<S> b{(const S*)w, K, N, K, vw};
  if (y_type == MDNN_F32) return conv_run<T, F32>(a, b, M, N, K, ep, 1, st);
  return conv_run<T, T>(a, b, M, N, K, ep, 1, st);
}

template <class T>
static mdnn_status_t bwd_data_impl(const ConvGeom& g, const void* dy, const void* w,
                                   const Epilogue& ep, mdnn_dtype_t dx_type, hipStream_t st) {
  typedef typename T::storage S;
  const int64_t M = (int64_t)g.n * g.h * g.w, N = g.c, K = (int64_t)g.r * g.s * g.k;
  const bool vdy = aligned(dy, 16) && g.k % 8 == 0;
  const bool vw = aligned(w, 16) && g.c % 8 == 0;
  SrcConvBwdA<S> a{(const S*)dy, g, M, K, vdy};
  SrcConvBwdB<S> b{(const S*)w, g, N, K, vw};
  if (dx_type == MDNN_F32) return conv_run<T, F32>(a, b, M, N, K, ep, 1, st);
  return conv_run<T, T>(a, b, M, N, K, ep, 1, st);
}

// Split-K plan of the backward-filter GEMM; a function of the shape only.
static constexpr size_t FILTER_WS_MAX = 64ull << 20;
static SplitPlan filter_plan(const ConvGeom& g) {
  const int64_t M = g.k, N = (int64_t)g.r * g.s * g.c, K = (int64_t)g.n * g.ho * g.wo;
  const int64_t tiles = ceil_div(M, 128) * ceil_div(N, 128);
  return plan_splits(M, N, K, tiles, FILTER_WS_MAX);
}

template <class T>
static mdnn_status_t bwd_filter_impl(const ConvGeom& g, const void* x, const void* dy, float* dw,
                                     void* ws, hipStream_t st, ReduceBatch* defer) {
  typedef typename T::storage S;
  const int64_t M = g.k, N = (int64_t)g.r * g.s * g.c, K = (int64_t)g.n * g.ho * g.wo;
  const bool vdy = aligned(dy, 16) && g.k % 8 == 0;
  const bool vx = aligned(x, 16) && g.c % 8 == 0;
  SrcMatMN<S> a{(const S*)dy, g.k, M, K, vdy};
  SrcConvFiltB<S> b{(const S*)x, g, N, K, vx};
  SplitPlan p = filter_plan(g);
  Epilogue ep = plain_epilogue(dw, N, MDNN_F32);
  if (p.splits > 1) {
    ep.partial = (float*)ws;
    ep.k_per_split = p.k_per_split;
  }
  MDNN_TRY((conv_run<T, F32>(a, b, M, N, K, ep, p.splits, st)));
  if (p.splits > 1) return reduce_splits((const float*)ws, p.splits, M, N, dw, st, defer);
  return MDNN_SUCCESS;
}

}  // namespace mdnn

using namespace mdnn;

extern "C" mdnn_status_t mdnn_conv2d_fwd(const mdnn_conv_shape_t* shape, const void* x,
                                         const void* w, mdnn_dtype_t io_type, const float* bias,
                                         mdnn_act_t act, void* y, mdnn_dtype_t y_type,
                                         mdnn_stream_t stream) {
  ConvGeom g;
  MDNN_TRY(check_conv_shape(shape, g));
  if (!dtype_ok(io_type) || !dtype_ok(y_type) || (y_type != MDNN_F32 && y_type != io_type))
    return fail(MDNN_ERR_DTYPE, "conv fwd: y_type must be fp32 or io_type");
  if (act != MDNN_ACT_NONE && act != MDNN_ACT_RELU) return fail(MDNN_ERR_DTYPE, "conv fwd: unknown act");
  if (g.n == 0) return MDNN_SUCCESS;
  if (!x || !w || !y) return fail(MDNN_ERR_NULL, "conv fwd: x, w and y are required");
  const size_t es = dtype_size(io_type);
  if (!aligned(x, es) || !aligned(w, es) || !aligned(y, dtype_size(y_type)) || (bias && !aligned(bias, 4)))
    return fail(MDNN_ERR_MISALIGNED, "conv fwd: misaligned base pointer");
  Epilogue ep = plain_epilogue(y, g.k, y_type);
  ep.bias = bias;
  ep.act = act;
  clear_error();
  hipStream_t st = as_stream(stream);
  if (pipe_allowed()) {
    if (conv_small_fwd_ok(g)) return conv_small_fwd(g, x, w, ep, io_type, y_type, st);
    bool done = false;
    if (halo_allowed()) MDNN_TRY(conv_halo(g, false, x, w, ep, io_type, y_type, st, &done));
    if (done) return MDNN_SUCCESS;
    MDNN_TRY(conv_pipe_fwd(g, x, w, ep, io_type, y_type, st, &done));
    if (done) return MDNN_SUCCESS;
  }
  switch (io_type) {
    case MDNN_F16: return fwd_impl<F16>(g, x, w, ep, y_type, st);
    case MDNN_BF16: return fwd_impl<BF16>(g, x, w, ep, y_type, st);
    default: return fwd_impl<F32>(g, x, w, ep, y_type, st);
  }
}

extern "C" mdnn_status_t mdnn_conv2d_bwd_data(const mdnn_conv_shape_t* shape, const void* dy,
                                              const void* w, mdnn_dtype_t io_type,
                                              const void* mask_src, void* dx,
                                              mdnn_dtype_t dx_type, mdnn_stream_t stream) {
  ConvGeom g;
  MDNN_TRY(check_conv_shape(shape, g));
  if (!dtype_ok(io_type) || !dtype_ok(dx_type) || (dx_type != MDNN_F32 && dx_type != io_type))
    return fail(MDNN_ERR_DTYPE, "conv bwd_data: dx_type must be fp32 or io_type");
  if (g.n == 0) return MDNN_SUCCESS;
  if (!dy || !w || !dx) return fail(MDNN_ERR_NULL, "conv bwd_data: dy, w and dx are required");
  const size_t es = dtype_size(io_type);
  if (!aligned(dy, es) || !aligned(w, es) || !aligned(dx, dtype_size(dx_type)) ||
      (mask_src && !aligned(mask_src, es)))
    return fail(MDNN_ERR_MISALIGNED, "conv bwd_data: misaligned base pointer");
  Epilogue ep = plain_epilogue(dx, g.c, dx_type);
  ep.mask = mask_src;
  ep.ldm = g.c;
  ep.vec4_m = mask_src && (g.c % 4 == 0) && aligned(mask_src, 4 * es);
  clear_error();
  hipStream_t st = as_stream(stream);
  if (pipe_allowed()) {
    bool done = false;
    if (halo_allowed()) MDNN_TRY(conv_halo(g, true, dy, w, ep, io_type, dx_type, st, &done));
    if (done) return MDNN_SUCCESS;
    MDNN_TRY(conv_pipe_bwd_data(g, dy, w, ep, io_type, dx_type, st, &done));
    if (done) return MDNN_SUCCESS;
  }
  switch (io_type) {
    case MDNN_F16: return bwd_data_impl<F16>(g, dy, w, ep, dx_type, st);
    case MDNN_BF16: return bwd_data_impl<BF16>(g, dy, w, ep, dx_type, st);
    default: return bwd_data_impl<F32>(g, dy, w, ep, dx_type, st);
  }
}

// Workspace: split-K partials of dw (room for the pipelined kernel's plan and
// the general kernel's, whichever runs), then (256-byte aligned) the partial
// column sums of db.
static size_t filter_ws_split_bytes(const ConvGeom& g) {
  const size_t mn = (size_t)g.k * ((size_t)g.r * g.s * g.c) * sizeof(float);
  const SplitPlan p = filter_plan(g), q = conv_pipe_filter_plan(g);
  size_t splits = p.splits > 1 ? (size_t)p.splits : 0;
  if (q.splits > 1 && (size_t)q.splits > splits) splits = (size_t)q.splits;
  // the vector-ALU kernels' block count (at least the matrix-core kernel's)
  const int64_t sb = conv_small_filter_blocks(g, MDNN_F32);
  if (sb > 0 && (size_t)sb > splits) splits = (size_t)sb;
  return (splits * mn + 255) & ~(size_t)255;
}


extern "C" size_t mdnn_conv2d_bwd_filter_workspace(const mdnn_conv_shape_t* shape,
                                                   mdnn_dtype_t io_type) {
  ConvGeom g;
  if (check_conv_shape(shape, g) != MDNN_SUCCESS || !dtype_ok(io_type)) return 0;
  return filter_ws_split_bytes(g) + column_sums_ws_bytes((int64_t)g.n * g.ho * g.wo, g.k);
}

// Workspace of mdnn_conv2d_bwd_filter_noalloc: one fixed array per GPU, held
// until the process ends.  Host code never passes the array's name to a
// kernel or a copy (in host code it is not a device address): it uses the
// address hipGetSymbolAddress returns for the current device, looked up on
// the entry point's first call on that device.
constexpr size_t kNoAllocScratchBytes = (size_t)48 << 20;
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

mdnn_status_t scratch_of_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(MDNN_ERR_LAUNCH, "bwd_filter_noalloc: hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(MDNN_ERR_LAUNCH, "bwd_filter_noalloc: device %d out of range", dev);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(MDNN_ERR_LAUNCH, "bwd_filter_noalloc: hipGetSymbolAddress: %s", hipGetErrorString(e));
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return MDNN_SUCCESS;
}
}  // namespace

extern "C" size_t mdnn_conv2d_bwd_filter_noalloc_max_workspace(void) { return kNoAllocScratchBytes; }

extern "C" mdnn_status_t mdnn_conv2d_bwd_filter_noalloc(const mdnn_conv_shape_t* shape, const void* x,
                                                        const void* dy, mdnn_dtype_t io_type, float* dw,
                                                        float* db, mdnn_stream_t stream) {
  ConvGeom g;
  MDNN_TRY(check_conv_shape(shape, g));
  if (!dtype_ok(io_type)) return fail(MDNN_ERR_DTYPE, "conv bwd_filter_noalloc: unknown io_type");
  const size_t need = mdnn_conv2d_bwd_filter_workspace(shape, io_type);
  if (need > kNoAllocScratchBytes)
    return fail(MDNN_ERR_WORKSPACE,
                "conv bwd_filter_noalloc: this shape needs %zu bytes of workspace, above the fixed %zu; "
                "use mdnn_conv2d_bwd_filter with a caller workspace",
                need, kNoAllocScratchBytes);
  void* ws = nullptr;
  if (need > 0) MDNN_TRY(scratch_of_current_device(&ws));
  return mdnn_conv2d_bwd_filter(shape, x, dy, io_type, dw, db, ws, need, stream);
}

mdnn_status_t mdnn::conv2d_bwd_filter_deferred(const mdnn_conv_shape_t* shape, const void* x, const void* dy,
                                               mdnn_dtype_t io_type, float* dw, float* db, void* workspace,
                                               size_t ws_bytes, hipStream_t st, ReduceBatch* defer) {
  ConvGeom g;
  MDNN_TRY(check_conv_shape(shape, g));
  if (!dtype_ok(io_type)) return fail(MDNN_ERR_DTYPE, "conv bwd_filter: unknown io_type");
  if (!dw) return fail(MDNN_ERR_NULL, "conv bwd_filter: dw is required");
  if (g.n > 0 && (!x || !dy)) return fail(MDNN_ERR_NULL, "conv bwd_filter: x and dy are required");
  const size_t es = dtype_size(io_type);
  if ((x && !aligned(x, es)) || (dy && !aligned(dy, es)) || !aligned(dw, 4) || (db && !aligned(db, 4)))
    return fail(MDNN_ERR_MISALIGNED, "conv bwd_filter: misaligned base pointer");
  const size_t need = mdnn_conv2d_bwd_filter_workspace(shape, io_type);
  if (need > 0 && (!workspace || ws_bytes < need || !aligned(workspace, 256)))
    return fail(MDNN_ERR_WORKSPACE, "conv bwd_filter: needs %zu bytes of 256-byte aligned workspace",
                need);
  clear_error();
  if (g.n == 0) {
    // empty batch: zero gradients
    MDNN_TRY(fill_zero(dw, (size_t)g.k * g.r * g.s * g.c * 4, st));
    return db ? fill_zero(db, (size_t)g.k * 4, st) : MDNN_SUCCESS;
  }
  bool done = false;
  if (pipe_allowed() && conv_small_filter_blocks(g, io_type) > 0) {
    MDNN_TRY(conv_small_filter(g, x, dy, dw, workspace, io_type, st, defer));
    done = true;
  }
  if (!done && pipe_allowed())
    MDNN_TRY(conv_pipe_bwd_filter(g, x, dy, dw, workspace, io_type, st, &done, defer));
  if (!done) {
    switch (io_type) {
      case MDNN_F16: MDNN_TRY(bwd_filter_impl<F16>(g, x, dy, dw, workspace, st, defer)); break;
      case MDNN_BF16: MDNN_TRY(bwd_filter_impl<BF16>(g, x, dy, dw, workspace, st, defer)); break;
      default: MDNN_TRY(bwd_filter_impl<F32>(g, x, dy, dw, workspace, st, defer)); break;
    }
  }
  if (db) {
    const size_t off = filter_ws_split_bytes(g);
    const size_t cs = column_sums_ws_bytes((int64_t)g.n * g.ho * g.wo, g.k);
    return column_sums(dy, nullptr, io_type, (int64_t)g.n * g.ho * g.wo, g.k, db,
                       cs ? (char*)workspace + off : nullptr, cs, st, defer);
  }
  return MDNN_SUCCESS;
}

extern "C" mdnn_status_t mdnn_conv2d_bwd_filter(const mdnn_conv_shape_t* shape, const void* x,
                                                const void* dy, mdnn_dtype_t io_type, float* dw,
                                                float* db, void* workspace, size_t ws_bytes,
                                                mdnn_stream_t stream) {
  // the weight and bias sums' second passes in one launch
  hipStream_t st = as_stream(stream);
  ReduceBatch batch{};
  MDNN_TRY(conv2d_bwd_filter_deferred(shape, x, dy, io_type, dw, db, workspace, ws_bytes, st, &batch));
  return reduce_batch_launch(batch, st);
}
