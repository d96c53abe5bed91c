// Implicit-GEMM convolutions (section 2.1's convolution layers, stride 1,
// zero padding) on the pipelined mainloop of gemm_lds.h.  The im2col
// operands are gathered straight into LDS by the convolution loaders; no
// im2col buffer exists.
//
// Tiles:
//   forward / backward data: 256 x 64 when N <= 64 (8 waves of 64 x 32);
//   else 128 x 128 (8 waves of 64 x 32), or 64 x 128 (4 waves of 32 x 64)
//   when 128 x 128 tiles would leave CUs idle (3x3, 256 -> 256 at 8x8,
//   batch 128: 128 tiles; forward 21.1 -> 16.3 us, backward data 23.0 ->
//   18.8 us); 2 stages.
//   backward filter: 64 x 128 (8 waves of 32 x 32) when M <= 64, else
//   64 x 64 (4 waves of 32 x 32); 3 stages and a split over K (output
//   pixels) sized to about 256 (M <= 64) or 512 workgroups, reduced in split
//   order (deterministic).  Against the former 64 x 256 / 128 x 128 tiles on
//   the ResNet-style layers (including the reduction): 38.9 -> 32.7,
//   40.2 -> 26.1, 33.6 -> 26.5 us.
#include "conv_pipe.h"

#include <numeric>
#include "gemm_launch.h"

namespace mdnn {

namespace {

typedef lds::Tile<256, 64, 4, 2, 4> TileTall;
typedef lds::Tile<128, 128, 2, 4, 4> TileSquare;
typedef lds::Tile<64, 128, 2, 2, 4> TileFlat;
// backward filter
typedef lds::Tile<64, 128, 2, 4, 2> TileFiltN;
typedef lds::Tile<64, 64, 2, 2, 4> TileFiltS;

// 128 x 128 tiles fill fewer than 256 workgroups: the 64 x 128 tile instead
bool flat_tiles(int64_t M, int64_t N) { return ceil_div(M, 128) * ceil_div(N, 128) < 256; }
constexpr int FILTER_STAGES = 3;
constexpr size_t FILTER_WS_MAX = 64ull << 20;
constexpr int64_t BUF_MAX = 0x7fffffffLL;  // range-checked buffers: offsets below 2^31

uint32_t magic_of(uint32_t d) { return d == 1 ? 0u : (uint32_t)(((1ull << 32) + d - 1) / d); }

template <class T, class OutT, class TL, class LB>
mdnn_status_t run_rows(const lds::ConvRowsArgs& a, const typename LB::Args& b, int64_t M, int64_t N, int64_t K,
                       const Epilogue& ep, hipStream_t st) {
  return run_pipe<T, OutT, TL, 2, lds::ConvRowsLoader<TL::BM, TL::LA>, LB>(a, b, M, N, K, ep, 1, st);
}

// fwd (B = filter as a K-contiguous matrix) or bwd_data (B = TapWeightLoader)
template <class T, class OutT, bool BWD>
mdnn_status_t rows_dispatch(const lds::ConvRowsArgs& a, const void* w, int32_t ldw, const ConvGeom& g, int64_t M,
                            int64_t N, int64_t K, const Epilogue& ep, hipStream_t st) {
  if constexpr (!BWD) {
    const lds::MatArgs b{w, ldw, N};
    if (N <= 64) return run_rows<T, OutT, TileTall, lds::MatLoader<true, 64, TileTall::LB>>(a, b, M, N, K, ep, st);
    if (flat_tiles(M, N))
      return run_rows<T, OutT, TileFlat, lds::MatLoader<true, 128, TileFlat::LB>>(a, b, M, N, K, ep, st);
    return run_rows<T, OutT, TileSquare, lds::MatLoader<true, 128, TileSquare::LB>>(a, b, M, N, K, ep, st);
  } else {
    const lds::TapWeightArgs b{w, g.k, g.r * g.s, g.c};
    if (N <= 64) return run_rows<T, OutT, TileTall, lds::TapWeightLoader<64, TileTall::LB>>(a, b, M, N, K, ep, st);
    if (flat_tiles(M, N))
      return run_rows<T, OutT, TileFlat, lds::TapWeightLoader<128, TileFlat::LB>>(a, b, M, N, K, ep, st);
    return run_rows<T, OutT, TileSquare, lds::TapWeightLoader<128, TileSquare::LB>>(a, b, M, N, K, ep, st);
  }
}

template <bool BWD>
mdnn_status_t rows_typed(const lds::ConvRowsArgs& a, const void* w, int32_t ldw, const ConvGeom& g, int64_t M,
                         int64_t N, int64_t K, const Epilogue& ep, mdnn_dtype_t io, mdnn_dtype_t out,
                         hipStream_t st) {
  if (io == MDNN_F16)
    return out == MDNN_F32 ? rows_dispatch<F16, F32, BWD>(a, w, ldw, g, M, N, K, ep, st)
                           : rows_dispatch<F16, F16, BWD>(a, w, ldw, g, M, N, K, ep, st);
  return out == MDNN_F32 ? rows_dispatch<BF16, F32, BWD>(a, w, ldw, g, M, N, K, ep, st)
                         : rows_dispatch<BF16, BF16, BWD>(a, w, ldw, g, M, N, K, ep, st);
}

}  // namespace

// Forward with c_in % 32 == 0 (not 64): K padded to whole steps of two
// 32-channel half blocks, the filter read range-checked.
template <class T, class OutT>
mdnn_status_t rows32_dispatch(const lds::ConvRowsArgs& a, const lds::MatRCArgs& b, int64_t M, int64_t N, int64_t Kp,
                              const Epilogue& ep, hipStream_t st) {
  if (N <= 64)
    return run_pipe<T, OutT, TileTall, 2, lds::ConvRows32Loader<256, TileTall::LA>,
                    lds::MatLoaderRC<64, TileTall::LB>>(a, b, M, N, Kp, ep, 1, st);
  return run_pipe<T, OutT, TileSquare, 2, lds::ConvRows32Loader<128, TileSquare::LA>,
                  lds::MatLoaderRC<128, TileSquare::LB>>(a, b, M, N, Kp, ep, 1, st);
}

mdnn_status_t conv_pipe_fwd32(const ConvGeom& g, const void* x, const void* w, const Epilogue& ep, mdnn_dtype_t io,
                              mdnn_dtype_t out, hipStream_t st, bool* done) {
  const int64_t M = (int64_t)g.n * g.ho * g.wo, N = g.k, K = (int64_t)g.r * g.s * g.c;
  const int64_t x_bytes = (int64_t)g.n * g.h * g.w * g.c * 2, w_bytes = N * K * 2;
  if (x_bytes > BUF_MAX || w_bytes > BUF_MAX || M > BUF_MAX) return MDNN_SUCCESS;
  const int64_t Kp = ceil_div(K, (int64_t)lds::BK) * lds::BK;
  lds::ConvRowsArgs a{x, (uint32_t)x_bytes, g.h, g.w, g.c, g.ho, g.wo, g.s, g.pad, 0, M};
  a.r = g.r;
  const lds::MatRCArgs b{w, (uint32_t)w_bytes, K, N};
  if (io == MDNN_F16)
    MDNN_TRY((out == MDNN_F32 ? rows32_dispatch<F16, F32>(a, b, M, N, Kp, ep, st)
                              : rows32_dispatch<F16, F16>(a, b, M, N, Kp, ep, st)));
  else
    MDNN_TRY((out == MDNN_F32 ? rows32_dispatch<BF16, F32>(a, b, M, N, Kp, ep, st)
                              : rows32_dispatch<BF16, BF16>(a, b, M, N, Kp, ep, st)));
  *done = true;
  return MDNN_SUCCESS;
}

mdnn_status_t conv_pipe_fwd(const ConvGeom& g, const void* x, const void* w, const Epilogue& ep,
                            mdnn_dtype_t io, mdnn_dtype_t out, hipStream_t st, bool* done) {
  *done = false;
  const int64_t M = (int64_t)g.n * g.ho * g.wo, N = g.k, K = (int64_t)g.r * g.s * g.c;
  const int64_t x_bytes = (int64_t)g.n * g.h * g.w * g.c * 2;
  if (io == MDNN_F32 || !aligned(x, 16) || !aligned(w, 16)) return MDNN_SUCCESS;
  if (g.c % 64 != 0) return g.c % 32 == 0 ? conv_pipe_fwd32(g, x, w, ep, io, out, st, done) : MDNN_SUCCESS;
  if (x_bytes > BUF_MAX || M > BUF_MAX || N * K * 2 >= ((int64_t)1 << 32)) return MDNN_SUCCESS;
  const lds::ConvRowsArgs a{x, (uint32_t)x_bytes, g.h, g.w, g.c, g.ho, g.wo, g.s, g.pad, 0, M};
  MDNN_TRY(rows_typed<false>(a, w, (int32_t)K, g, M, N, K, ep, io, out, st));
  *done = true;
  return MDNN_SUCCESS;
}

mdnn_status_t conv_pipe_bwd_data(const ConvGeom& g, const void* dy, const void* w, const Epilogue& ep,
                                 mdnn_dtype_t io, mdnn_dtype_t out, hipStream_t st, bool* done) {
  *done = false;
  const int64_t M = (int64_t)g.n * g.h * g.w, N = g.c, K = (int64_t)g.r * g.s * g.k;
  const int64_t dy_bytes = (int64_t)g.n * g.ho * g.wo * g.k * 2;
  if (io == MDNN_F32 || g.k % 64 != 0 || g.c % 8 != 0 || !aligned(dy, 16) || !aligned(w, 16)) return MDNN_SUCCESS;
  const int64_t ldw = (int64_t)g.r * g.s * g.c;  // filter elements between consecutive c_out
  if (dy_bytes > BUF_MAX || M > BUF_MAX || (64 * ldw + N) * 2 >= ((int64_t)1 << 32)) return MDNN_SUCCESS;
  // rows over the h x w input grid, gathered from the ho x wo grid of dy
  const lds::ConvRowsArgs a{dy, (uint32_t)dy_bytes, g.ho, g.wo, g.k, g.h, g.w, g.s, g.pad, 1, M};
  MDNN_TRY(rows_typed<true>(a, w, 0, g, M, N, K, ep, io, out, st));
  *done = true;
  return MDNN_SUCCESS;
}

SplitPlan conv_pipe_filter_plan(const ConvGeom& g) {
  SplitPlan p{0, 0};
  const int64_t M = g.k, N = (int64_t)g.r * g.s * g.c, K = (int64_t)g.n * g.ho * g.wo;
  const int64_t x_bytes = (int64_t)g.n * g.h * g.w * g.c * 2;
  if (g.ho != g.h || g.wo != g.w || g.c % 8 != 0 || g.k % 8 != 0 || K % lds::BK != 0 || K == 0) return p;
  if (x_bytes > BUF_MAX || K * (g.w - 1) >= ((int64_t)1 << 32) || (K / g.w) * (g.h - 1) >= ((int64_t)1 << 32))
    return p;
  if (N > BUF_MAX / 4 || M * N > BUF_MAX / 4) return p;
  // aim at about 256 (64 x 128 tiles, 8 waves) or 512 (64 x 64 tiles, 4
  // waves) workgroups; each split keeps at least 4 K steps and the partials
  // stay within the cap
  const bool narrow = M <= 64;
  const int64_t tiles = narrow ? ceil_div(N, TileFiltN::BN) : ceil_div(M, 64) * ceil_div(N, 64);
  const int64_t steps = K / lds::BK;
  int64_t s = ceil_div(narrow ? 256 : 512, tiles);
  if (s > steps / 4) s = steps / 4;
  while (s > 1 && (size_t)s * M * N * 4 > FILTER_WS_MAX) --s;
  if (s < 1) s = 1;
  // with few tiles, tiles x splits a multiple of 8 lets the kernel keep the
  // tiles of one split on one XCD (its slice of x and dy then comes through
  // that L2 once)
  const int64_t q = 8 / std::gcd(tiles, (int64_t)8);
  if (tiles <= SPLIT_XCD_MAX_TILES && s >= q) s -= s % q;
  const int64_t kps = ceil_div(steps, s) * lds::BK;
  p.splits = (int)ceil_div(K, kps);
  p.k_per_split = kps;
  return p;
}

namespace {

template <class T, class TL>
mdnn_status_t filter_run(const ConvGeom& g, const void* x, const void* dy, float* dw, void* ws, const SplitPlan& p,
                         hipStream_t st, ReduceBatch* defer) {
  const int64_t M = g.k, N = (int64_t)g.r * g.s * g.c, K = (int64_t)g.n * g.ho * g.wo;
  const lds::MatArgs a{dy, g.k, g.k};
  const lds::ConvColsArgs b{x, (uint32_t)((int64_t)g.n * g.h * g.w * g.c * 2), g.h, g.w, g.c, g.s, g.pad,
                            magic_of((uint32_t)g.w), magic_of((uint32_t)g.h), N};
  Epilogue ep{};
  ep.alpha = 1.0f;
  ep.D = dw;
  ep.ldd = N;
  ep.act = MDNN_ACT_NONE;
  ep.vec4 = (N % 4 == 0) && aligned(dw, 16);
  ep.k_per_split = K;
  if (p.splits > 1) {
    ep.partial = (float*)ws;
    ep.k_per_split = p.k_per_split;
  }
  MDNN_TRY((run_pipe<T, F32, TL, FILTER_STAGES, lds::MatLoader<false, TL::BM, TL::LA>,
                     lds::ConvColsLoader<TL::BN, TL::LB>>(a, b, M, N, K, ep, p.splits, st)));
  if (p.splits > 1) return reduce_splits((const float*)ws, p.splits, M, N, dw, st, defer);
  return MDNN_SUCCESS;
}

}  // namespace

mdnn_status_t conv_pipe_bwd_filter(const ConvGeom& g, const void* x, const void* dy, float* dw, void* ws,
                                   mdnn_dtype_t io, hipStream_t st, bool* done, ReduceBatch* defer) {
  *done = false;
  const SplitPlan p = conv_pipe_filter_plan(g);
  if (io == MDNN_F32 || p.splits == 0 || !aligned(x, 16) || !aligned(dy, 16)) return MDNN_SUCCESS;
  if (p.splits > 1 && (!ws || !aligned(ws, 16))) return MDNN_SUCCESS;
  if (g.k <= 64)
    MDNN_TRY((io == MDNN_F16 ? filter_run<F16, TileFiltN>(g, x, dy, dw, ws, p, st, defer)
                             : filter_run<BF16, TileFiltN>(g, x, dy, dw, ws, p, st, defer)));
  else
    MDNN_TRY((io == MDNN_F16 ? filter_run<F16, TileFiltS>(g, x, dy, dw, ws, p, st, defer)
                             : filter_run<BF16, TileFiltS>(g, x, dy, dw, ws, p, st, defer)));
  *done = true;
  return MDNN_SUCCESS;
}

}  // namespace mdnn
