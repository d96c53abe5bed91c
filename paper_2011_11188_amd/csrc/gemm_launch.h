// Launch helpers of the GEMM engine, shared by the GEMM and convolution
// entry points.  Tile selection is a fixed table keyed on the problem size.
#pragma once

#include "gemm_core.h"
#include "gemm_lds.h"
#include "internal.h"

namespace mdnn {

// fp32 path: 64x64 tiles, 4x4 outputs per thread, K step 16, operands staged
// through LDS element by element (vector FMA; config-sized fp32 problems are
// small and latency-bound).  KG groups of 256 threads split the tile's K range
// among themselves and combine their sums through LDS in group order (fixed,
// so deterministic): a grid of only a few tiles over a long K then keeps KG
// times as many waves busy.
// src.elem(mn, k) when ok, else 0, as an unconditional load from a clamped
// address (base()[0] is an element of the operand) and a select: guarded loads
// in divergent branches are each waited for before the branch joins, so a
// branch-free fetch keeps all of a thread's loads in flight together.
template <class Src>
__device__ __forceinline__ float fetch_sel(const Src& src, int64_t mn, int64_t k, bool ok) {
  const int64_t o = ok ? src.off(mn, k) : -1;
  const float v = (float)src.base()[o >= 0 ? o : 0];
  return o >= 0 ? v : 0.0f;
}

template <class SrcA, class SrcB, int KG>
__global__ void __launch_bounds__(256 * KG)
gemm_f32_kernel(SrcA a, SrcB b, int64_t M, int64_t N, int64_t K, Epilogue ep) {
  constexpr int STAGE = 2 * 16 * 68;  // As + Bs of one group
  constexpr int RED = (KG - 1) * 64 * 64;
  __shared__ float smem[KG * STAGE > RED ? KG * STAGE : RED];
  const int grp = threadIdx.x >> 8, tid = threadIdx.x & 255;
  float(*As)[68] = (float(*)[68])(smem + grp * STAGE);
  float(*Bs)[68] = (float(*)[68])(smem + grp * STAGE + 16 * 68);
  const int tx = tid & 15, ty = tid >> 4;
  const int64_t m0 = (int64_t)blockIdx.x * 64, n0 = (int64_t)blockIdx.y * 64;
  int64_t kbeg = 0, kend = K;
  if (ep.partial) {
    kbeg = (int64_t)blockIdx.z * ep.k_per_split;
    kend = kbeg + ep.k_per_split < K ? kbeg + ep.k_per_split : K;
  }
  // this group's share of [kbeg, kend), whole K steps; every group runs the
  // same number of steps (the barriers are block-wide)
  const int64_t steps = ceil_div(kend - kbeg, 16), per = ceil_div(steps, KG);
  const int64_t gbeg = kbeg + grp * per * 16;
  const int64_t gend = gbeg + per * 16 < kend ? gbeg + per * 16 : kend;
  // staging: thread tid owns elements tid + 256 q (q < 4) of each 64 x 16
  // operand slab; the next step's elements are loaded into registers while
  // the current step computes (one memory latency per step, overlapped)
  int sr[2][4], sk[2][4];  // (row, k) of each owned element, per operand
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int idx = tid + q * 256;
    sr[0][q] = SrcA::KC ? idx >> 4 : idx & 63;
    sk[0][q] = SrcA::KC ? idx & 15 : idx >> 6;
    sr[1][q] = SrcB::KC ? idx >> 4 : idx & 63;
    sk[1][q] = SrcB::KC ? idx & 15 : idx >> 6;
  }
  float ra[4], rb[4];
  auto fetch = [&](int64_t k0) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      ra[q] = fetch_sel(a, m0 + sr[0][q], k0 + sk[0][q], k0 + sk[0][q] < gend);
      rb[q] = fetch_sel(b, n0 + sr[1][q], k0 + sk[1][q], k0 + sk[1][q] < gend);
    }
  };
  float acc[4][4] = {};
  if (per > 0) fetch(gbeg);
  for (int64_t it = 0; it < per; ++it) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      As[sk[0][q]][sr[0][q]] = ra[q];
      Bs[sk[1][q]][sr[1][q]] = rb[q];
    }
    __syncthreads();
    if (it + 1 < per) fetch(gbeg + (it + 1) * 16);
#pragma unroll
    for (int kk = 0; kk < 16; ++kk) {
      float av[4], bv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) { av[i] = As[kk][ty * 4 + i]; bv[i] = Bs[kk][tx * 4 + i]; }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
    }
    __syncthreads();
  }
  if (KG > 1) {
    // groups 1.. hand their sums to group 0, which adds them in group order
    if (grp > 0) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) smem[(grp - 1) * 4096 + (ty * 4 + i) * 64 + tx * 4 + j] = acc[i][j];
    }
    __syncthreads();
    if (grp > 0) return;
    for (int g = 1; g < KG; ++g)
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] += smem[(g - 1) * 4096 + (ty * 4 + i) * 64 + tx * 4 + j];
  }
  const int64_t n = n0 + tx * 4;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int64_t m = m0 + ty * 4 + i;
    if (ep.partial) {
      if (m < M) {
        float* p = ep.partial + ((int64_t)blockIdx.z * M + m) * N + n;
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (n + j < N) p[j] = acc[i][j];
      }
    } else {
      epilogue_store4<F32, F32>(ep, M, N, m, n, (float4_t){acc[i][0], acc[i][1], acc[i][2], acc[i][3]});
    }
  }
}

// Tile configurations of the MFMA kernels.  TILE_LDS_PIPE / TILE_LDS_PIPE128
// force the 256 x 256 / 128 x 128 direct-to-LDS pipelined mainloop
// (gemm_lds.h) for plain matrices that meet its preconditions; TILE_AUTO
// picks the tile by problem size.
enum TileCfg {
  TILE_AUTO = 0,
  TILE_256x256 = 1,
  TILE_128x128 = 2,
  TILE_64x64 = 3,
  TILE_LDS_PIPE = 4,
  TILE_LDS_PIPE128 = 5
};

int gemm_tile_override();

inline TileCfg choose_tile(int64_t M, int64_t N, int splits) {
  int o = gemm_tile_override();
  if (o >= TILE_256x256 && o <= TILE_64x64) return (TileCfg)o;
  if (o >= TILE_LDS_PIPE) return TILE_256x256;  // this path has no pipelined kernel
  if (M <= 64 || N <= 64) return TILE_64x64;  // a wider tile would be mostly padding
  const int64_t t256 = ceil_div(M, 256) * ceil_div(N, 256) * splits;
  if (t256 >= 256 && M > 128 && N > 128) return TILE_256x256;
  const int64_t t128 = ceil_div(M, 128) * ceil_div(N, 128) * splits;
  if (t128 >= 160) return TILE_128x128;
  return TILE_64x64;
}

template <class T, class OutT, class SrcA, class SrcB, int BM, int BN, int WM, int WN>
inline void launch_mfma(const SrcA& a, const SrcB& b, int64_t M, int64_t N, int64_t K,
                        const Epilogue& ep, int splits, hipStream_t stream) {
  dim3 grid((unsigned)(ceil_div(M, BM) * ceil_div(N, BN)), (unsigned)splits, 1);
  hipLaunchKernelGGL((gemm_mfma_kernel<T, OutT, SrcA, SrcB, BM, BN, WM, WN>), grid,
                     dim3(WM * WN * 64), 0, stream, a, b, M, N, K, ep);
}

// D (or split partials) = op(A) op(B) with the epilogue; T is F16 or BF16.
template <class T, class OutT, class SrcA, class SrcB>
inline mdnn_status_t run_gemm16(const SrcA& a, const SrcB& b, int64_t M, int64_t N, int64_t K,
                                const Epilogue& ep, int splits, hipStream_t stream) {
  if (ceil_div(M, 64) * ceil_div(N, 64) > 0x7fffffffLL || splits > 65535)
    return fail(MDNN_ERR_SHAPE, "gemm: problem too large for the launch grid");
  switch (choose_tile(M, N, splits)) {
    case TILE_256x256: launch_mfma<T, OutT, SrcA, SrcB, 256, 256, 2, 4>(a, b, M, N, K, ep, splits, stream); break;
    case TILE_128x128: launch_mfma<T, OutT, SrcA, SrcB, 128, 128, 2, 2>(a, b, M, N, K, ep, splits, stream); break;
    default:           launch_mfma<T, OutT, SrcA, SrcB, 64, 64, 1, 2>(a, b, M, N, K, ep, splits, stream); break;
  }
  return check_launch("gemm_mfma_kernel");
}

// Plain-matrix operand of the pipelined kernel: `kc` = K-contiguous.
struct LdsOperand {
  const void* p;
  int64_t ld, MN;
  bool kc;
};

// Whether the pipelined kernel can run this problem (see gemm_lds.h): the
// 256 x 256 tile when it gives at least one tile per CU, else 128 x 128 or
// 64 x 64 tiles (run_gemm_lds) when 128 x 128 tiles number at least 32.
inline bool lds_pipe_eligible(const LdsOperand& a, const LdsOperand& b, int64_t M, int64_t N,
                              int64_t K, int64_t k_per_split, int splits) {
  const int o = gemm_tile_override();
  if (o >= TILE_256x256 && o <= TILE_64x64) return false;
  if (K <= 0 || K % lds::BK != 0 || k_per_split % lds::BK != 0) return false;
  if (o < TILE_LDS_PIPE && ceil_div(M, 128) * ceil_div(N, 128) * splits < 32) return false;
  for (const LdsOperand* op : {&a, &b}) {
    if (!aligned(op->p, 16) || op->ld % 8 != 0) return false;
    const int64_t reach = op->kc ? (op->MN - 1) * op->ld + K : (int64_t)lds::BK * op->ld + op->MN;
    if (reach * 2 >= (int64_t)1 << 32) return false;
    if (!op->kc && (op->MN % 8 != 0 || op->MN < 8)) return false;
  }
  return true;
}

template <class T, class OutT, class TL, bool A_KC, bool B_KC, int NS = 2>
inline void launch_gemm_lds(const LdsOperand& a, const LdsOperand& b, int64_t M, int64_t N, int64_t K,
                            const Epilogue& ep, int splits, hipStream_t stream) {
  dim3 grid((unsigned)(ceil_div(M, TL::BM) * ceil_div(N, TL::BN)), (unsigned)splits, 1);
  lds::MatArgs oa{a.p, a.ld, a.MN}, ob{b.p, b.ld, b.MN};
  hipLaunchKernelGGL((lds::gemm_lds_kernel<T, OutT, TL, NS, lds::MatLoader<A_KC, TL::BM, TL::LA>,
                                           lds::MatLoader<B_KC, TL::BN, TL::LB>>),
                     grid, dim3(TL::NT), 0, stream, oa, ob, M, N, K, ep);
}

// Narrow products: a 256 x 64 (64 x 256) tile when N (M) is at most 64, so
// that a square tile's columns (rows) are not mostly padding.
typedef lds::Tile<256, 64, 4, 2, 4> TileNarrowN;
typedef lds::Tile<64, 256, 2, 4, 2> TileNarrowM;
// 128 x 128 with three LDS stages (96 KB): one workgroup of four waves per
// CU, so two tiles are in flight behind the MFMAs (against eight waves of
// 64 x 32 with four stages: TN 1024 x 4096 x 4096 41.7 -> 38.3 us,
// NN 2048 x 2048 x 4096 39.2 -> 35.8 us)
typedef lds::Tile<128, 128, 2, 2, 1> Tile128Deep;
// Grids of fewer than 128 tiles of 128 x 128 (e.g. 1024 x 1024): 64 x 64
// tiles with four waves of 32 x 32 put four times as many workgroups on the
// chip (1024^3: 11.2 -> 7.2 us; splitting each tile's K among more waves of
// one workgroup measured no faster, the time being the load latency, the
// epilogue and the launch rather than the K loop).
typedef lds::Tile<64, 64, 2, 2, 4> Tile64;

template <class T, class OutT, bool A_KC, bool B_KC>
inline mdnn_status_t run_gemm_lds(const LdsOperand& a, const LdsOperand& b, int64_t M, int64_t N,
                                  int64_t K, const Epilogue& ep, int splits, hipStream_t stream) {
  const int o = gemm_tile_override();
  if (o == TILE_AUTO && N <= 64 && M > 64)
    launch_gemm_lds<T, OutT, TileNarrowN, A_KC, B_KC>(a, b, M, N, K, ep, splits, stream);
  else if (o == TILE_AUTO && M <= 64 && N > 64)
    launch_gemm_lds<T, OutT, TileNarrowM, A_KC, B_KC>(a, b, M, N, K, ep, splits, stream);
  else if (o == TILE_LDS_PIPE ||
           (o != TILE_LDS_PIPE128 && N > 128 && M > 128 && ceil_div(M, 256) * ceil_div(N, 256) * splits >= 256))
    launch_gemm_lds<T, OutT, lds::Tile256, A_KC, B_KC>(a, b, M, N, K, ep, splits, stream);
  else if (o == TILE_AUTO && ceil_div(M, 128) * ceil_div(N, 128) * splits < 128 &&
           ceil_div(M, 64) * ceil_div(N, 64) * splits >= 128) {
    // a 64 x 64 x 64 step is a few hundred cycles of MFMAs, far less than a
    // load's latency: keep two (three, over a long K) steps' loads in flight
    // (1024 x 1024 x 4096: 30.1 -> 15.9-18.2 us; 1024^3: 7.8-8.2 -> 7.1-7.8 us)
    if ((splits > 1 ? ep.k_per_split : K) >= 2048)
      launch_gemm_lds<T, OutT, Tile64, A_KC, B_KC, 4>(a, b, M, N, K, ep, splits, stream);
    else
      launch_gemm_lds<T, OutT, Tile64, A_KC, B_KC, 3>(a, b, M, N, K, ep, splits, stream);
  }
  else if (ceil_div(M, 128) * ceil_div(N, 128) * splits <= 256)
    // at most one workgroup per CU: the LDS a second one would use holds
    // another stage instead
    launch_gemm_lds<T, OutT, Tile128Deep, A_KC, B_KC, 3>(a, b, M, N, K, ep, splits, stream);
  else
    launch_gemm_lds<T, OutT, lds::Tile128, A_KC, B_KC>(a, b, M, N, K, ep, splits, stream);
  return check_launch("gemm_lds_kernel");
}

// Pipelined kernel with explicit tile and loaders (the convolutions).
template <class T, class OutT, class TL, int NS, class LA, class LB>
inline mdnn_status_t run_pipe(const typename LA::Args& a, const typename LB::Args& b, int64_t M, int64_t N,
                              int64_t K, const Epilogue& ep, int splits, hipStream_t stream) {
  const int64_t tiles = ceil_div(M, TL::BM) * ceil_div(N, TL::BN);
  if (tiles > 0x7fffffffLL || splits > 65535)
    return fail(MDNN_ERR_SHAPE, "gemm: problem too large for the launch grid");
  dim3 grid((unsigned)tiles, (unsigned)splits, 1);
  hipLaunchKernelGGL((lds::gemm_lds_kernel<T, OutT, TL, NS, LA, LB>), grid, dim3(TL::NT), 0, stream, a, b, M, N,
                     K, ep);
  return check_launch("gemm_lds_kernel");
}

template <class SrcA, class SrcB>
inline mdnn_status_t run_gemm32(const SrcA& a, const SrcB& b, int64_t M, int64_t N, int64_t K,
                                const Epilogue& ep, int splits, hipStream_t stream) {
  if (ceil_div(M, 64) > 0x7fffffffLL || ceil_div(N, 64) > 65535 || splits > 65535)
    return fail(MDNN_ERR_SHAPE, "gemm: problem too large for the fp32 launch grid");
  dim3 grid((unsigned)ceil_div(M, 64), (unsigned)ceil_div(N, 64), (unsigned)splits);
  // few workgroups over a long K: four K groups per tile
  const int64_t blocks = (int64_t)grid.x * grid.y * grid.z;
  const int64_t k_each = splits > 1 ? ep.k_per_split : K;
  if (blocks < 128 && k_each >= 256)
    hipLaunchKernelGGL((gemm_f32_kernel<SrcA, SrcB, 4>), grid, dim3(1024), 0, stream, a, b, M, N, K, ep);
  else
    hipLaunchKernelGGL((gemm_f32_kernel<SrcA, SrcB, 1>), grid, dim3(256), 0, stream, a, b, M, N, K, ep);
  return check_launch("gemm_f32_kernel");
}

// Number of K splits so that the grid fills the chip, each split a multiple
// of the K step, and the partials stay within `max_ws` bytes.
inline SplitPlan plan_splits(int64_t M, int64_t N, int64_t K, int64_t tiles, size_t max_ws) {
  SplitPlan p{1, K};
  const int64_t target = 512;
  if (tiles >= target || K <= 2 * GEMM_BK) return p;
  int64_t s = ceil_div(target, tiles);
  int64_t max_s = K / (2 * GEMM_BK);
  if (s > max_s) s = max_s;
  while (s > 1 && (size_t)s * M * N * 4 > max_ws) --s;
  if (s < 1) s = 1;
  int64_t kps = ceil_div(ceil_div(K, s), GEMM_BK) * GEMM_BK;
  p.splits = (int)ceil_div(K, kps);
  p.k_per_split = kps;
  return p;
}

}  // namespace mdnn
