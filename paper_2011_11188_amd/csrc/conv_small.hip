// Convolutions with a tiny reduction (section 2.1's convolution layers; the
// first layer of an image network, e.g. one input channel and a 5x5 filter):
// the GEMM engine would spend almost all of a tile on padding, so these run
// as direct kernels on the vector ALUs, fp32 accumulation.
//
//   forward (K = r*s*c_in <= 64): with c_out <= 32 a thread owns one output
//     pixel (its im2col row gathered once into LDS, the filter staged once per
//     256 pixels, all channels from broadcast filter reads); wider outputs:
//     a block stages the im2col rows of 64 output pixels and the whole filter
//     in LDS, and each thread produces four consecutive output channels of
//     one pixel.  Both end in the shared epilogue.
//   backward filter (c_out * r*s*c_in <= 1024 outputs, r*s*c_in <= 64): each
//     block accumulates every filter element over its chunk of output pixels
//     into fp32 partials, which the split reduction then sums in a fixed
//     order (deterministic).
#include "conv_small.h"

namespace mdnn {
namespace {

constexpr int TP = 64;  // output pixels per staging round

// Offset in x of the im2col element (pixel m of the output grid, column
// kk = (r*s_ + s)*c + ch), or -1 in the zero padding.
__device__ __forceinline__ int64_t patch_off(const ConvGeom& g, int64_t m64, int kk) {
  const int m = (int)m64;  // the direct kernels run only while n*ho*wo < 2^31: 32-bit divisions
  const int hw = g.ho * g.wo;
  const int n = m / hw;
  const int rem = m - n * hw;
  const int i = rem / g.wo, j = rem - i * g.wo;
  const int tap = kk / g.c, ch = kk - tap * g.c;
  const int r = tap / g.s, s = tap - r * g.s;
  const int y = i + r - g.pad, xx = j + s - g.pad;
  if (y < 0 || y >= g.h || xx < 0 || xx >= g.w) return -1;
  return (((int64_t)n * g.h + y) * g.w + xx) * g.c + ch;
}

// Stage `count` table entries into LDS: entry e comes from src[off(e)] (0
// where off(e) < 0) and goes to lds[dst(e)].  Each thread issues eight loads
// before it stores any (the address is clamped to src[0] instead of
// branching around the load), so a round of staging costs one memory latency
// rather than one per element.
template <class T, class Off, class Dst>
__device__ __forceinline__ void stage(const typename T::storage* __restrict__ src, int count, Off off, Dst dst,
                                      float* lds) {
  for (int base = 0; base < count; base += 8 * 256) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = base + u * 256 + (int)threadIdx.x;
      const int64_t o = e < count ? off(e) : -1;
      const float x = to_f<T>(src[o >= 0 ? o : 0]);
      v[u] = o >= 0 ? x : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = base + u * 256 + (int)threadIdx.x;
      if (e < count) lds[dst(e)] = v[u];
    }
  }
}

// Row stride of an LDS table with `cols` columns: odd, so that a column walk
// by consecutive lanes spreads over the banks.
__host__ __device__ constexpr int odd_stride(int cols) { return cols | 1; }

// Output channels padded to a multiple of four, so that four consecutive
// channels are one 16-byte LDS read.
__host__ __device__ constexpr int quad_pad(int n) { return (n + 3) & ~3; }

template <class T, class OutT>
__global__ void __launch_bounds__(256)
conv_small_fwd_kernel(const typename T::storage* __restrict__ x, const typename T::storage* __restrict__ w,
                      ConvGeom g, int64_t M, Epilogue ep) {
  extern __shared__ float smem[];
  const int K = g.r * g.s * g.c, N = g.k, KS = odd_stride(K), NP = quad_pad(N);
  float* xs = smem;            // [TP][KS] im2col rows
  float* wt = smem + TP * KS;  // [K][NP] filter, transposed (zero beyond N)
  const int tid = threadIdx.x;
  stage<T>(w, K * NP, [=](int e) -> int64_t { const int kk = e / NP, n = e - kk * NP; return n < N ? (int64_t)n * K + kk : -1; },
           [](int e) { return e; }, wt);
  const int64_t m0 = (int64_t)blockIdx.x * TP;
  stage<T>(
      x, TP * K, [=](int e) -> int64_t { const int p = e / K; return m0 + p < M ? patch_off(g, m0 + p, e - p * K) : -1; },
      [=](int e) { return (e / K) * KS + e % K; }, xs);
  __syncthreads();
  // thread task: pixel p, output channels n4 .. n4+3 (one 16-byte read of the
  // filter and one broadcast read of the patch per four FMAs)
  const int groups = NP / 4;
  for (int q = tid; q < TP * groups; q += 256) {
    const int p = q / groups, n4 = (q - p * groups) * 4;
    float4_t acc = {0.f, 0.f, 0.f, 0.f};
    const float* xr = xs + p * KS;
    for (int kk = 0; kk < K; ++kk) {
      const float a = xr[kk];
      const float4 b = *(const float4*)(wt + kk * NP + n4);
      acc[0] = fmaf(a, b.x, acc[0]);
      acc[1] = fmaf(a, b.y, acc[1]);
      acc[2] = fmaf(a, b.z, acc[2]);
      acc[3] = fmaf(a, b.w, acc[3]);
    }
    epilogue_store4<T, OutT>(ep, M, N, m0 + p, n4, acc);
  }
}

// Narrow outputs (c_out <= 32): one output pixel per thread.  The thread
// decomposes its pixel once and gathers its own im2col row (taps walked with
// counters, eight loads in flight) into LDS, the block stages the filter
// once for 256 pixels, and the thread then produces all c_out channels from
// its row and broadcast reads of the filter.
constexpr int PX = 256;         // output pixels per block (one per thread)
constexpr int PX_QUADS = 8;     // c_out <= 32

template <class T, class OutT>
__global__ void __launch_bounds__(256)
conv_small_fwd_px_kernel(const typename T::storage* __restrict__ x, const typename T::storage* __restrict__ w,
                         ConvGeom g, int64_t M, Epilogue ep) {
  extern __shared__ float smem[];
  const int K = g.r * g.s * g.c, N = g.k, KS = odd_stride(K), NP = quad_pad(N), nq = NP / 4;
  float* xs = smem;            // [PX][KS] im2col rows
  float* wt = smem + PX * KS;  // [K][NP] filter, transposed (zero beyond N)
  const int tid = threadIdx.x;
  stage<T>(w, K * NP, [=](int e) -> int64_t { const int kk = e / NP, n = e - kk * NP; return n < N ? (int64_t)n * K + kk : -1; },
           [](int e) { return e; }, wt);
  const int64_t m = (int64_t)blockIdx.x * PX + tid;
  float* row = xs + tid * KS;
  if (m < M) {
    const int mi = (int)m, hw = g.ho * g.wo;  // pixel counts below 2^31 on this path
    const int n = mi / hw, rem = mi - n * hw, i = rem / g.wo, j = rem - i * g.wo;
    const typename T::storage* xn = x + (int64_t)n * g.h * g.w * g.c;
    int tr = 0, ts = 0, ch = 0;  // tap row, tap column, channel of element kk
    for (int kb = 0; kb < K; kb += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int y = i + tr - g.pad, xx = j + ts - g.pad;
        const bool ok = kb + u < K && (unsigned)y < (unsigned)g.h && (unsigned)xx < (unsigned)g.w;
        const float val = to_f<T>(xn[ok ? ((int64_t)y * g.w + xx) * g.c + ch : 0]);
        v[u] = ok ? val : 0.0f;
        if (++ch == g.c) {
          ch = 0;
          if (++ts == g.s) {
            ts = 0;
            ++tr;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (kb + u < K) row[kb + u] = v[u];
    }
  }
  __syncthreads();
  if (m >= M) return;
  float4_t acc[PX_QUADS];
#pragma unroll
  for (int q = 0; q < PX_QUADS; ++q) acc[q] = (float4_t){0.f, 0.f, 0.f, 0.f};
  for (int kk = 0; kk < K; ++kk) {
    const float a = row[kk];
    const float* wk = wt + kk * NP;
#pragma unroll
    for (int q = 0; q < PX_QUADS; ++q) {
      if (q < nq) {
        const float4 b = *(const float4*)(wk + 4 * q);
        acc[q][0] = fmaf(a, b.x, acc[q][0]);
        acc[q][1] = fmaf(a, b.y, acc[q][1]);
        acc[q][2] = fmaf(a, b.z, acc[q][2]);
        acc[q][3] = fmaf(a, b.w, acc[q][3]);
      }
    }
  }
  const bool full = full_tile_epilogue(ep, 4 * nq <= N, N);
#pragma unroll
  for (int q = 0; q < PX_QUADS; ++q) {
    if (q < nq) {
      if (full)
        epilogue_store4<T, OutT, true>(ep, M, N, m, 4 * q, acc[q]);
      else
        epilogue_store4<T, OutT>(ep, M, N, m, 4 * q, acc[q]);
    }
  }
}

// partial[b][k][kk] over the pixels of block b (pixels_per_block of them).
// Thread task: output channels k4 .. k4+3 of filter column kk; per pixel one
// 16-byte read of the output gradient row and one read of the patch.
template <class T>
__global__ void __launch_bounds__(256)
conv_small_filter_kernel(const typename T::storage* __restrict__ x, const typename T::storage* __restrict__ dy,
                         ConvGeom g, int64_t P, int64_t pixels_per_block, float* __restrict__ partial) {
  extern __shared__ float smem[];
  const int K = g.r * g.s * g.c, N = g.k, MN = N * K, KS = odd_stride(K), NP = quad_pad(N);
  float* xs = smem;            // [TP][KS] im2col rows
  float* ds = smem + TP * KS;  // [TP][NP] output gradient rows (zero beyond N)
  const int tid = threadIdx.x;
  const int G4 = NP / 4, tasks = G4 * K;  // <= 256 + K: at most two per thread
  float4_t acc[2] = {{0.f, 0.f, 0.f, 0.f}, {0.f, 0.f, 0.f, 0.f}};
  const int64_t p_beg = (int64_t)blockIdx.x * pixels_per_block;
  const int64_t p_end = p_beg + pixels_per_block < P ? p_beg + pixels_per_block : P;
  for (int64_t p0 = p_beg; p0 < p_end; p0 += TP) {
    __syncthreads();
    stage<T>(
        x, TP * K,
        [=](int e) -> int64_t { const int p = e / K; return p0 + p < p_end ? patch_off(g, p0 + p, e - p * K) : -1; },
        [=](int e) { return (e / K) * KS + e % K; }, xs);
    stage<T>(
        dy, TP * NP,
        [=](int e) -> int64_t { const int p = e / NP, k = e - p * NP; return (p0 + p < p_end && k < N) ? (p0 + p) * N + k : -1; },
        [](int e) { return e; }, ds);
    __syncthreads();
#pragma unroll
    for (int o = 0; o < 2; ++o) {
      const int t = tid + o * 256;
      if (t < tasks) {
        const int kk = t / G4, k4 = (t - kk * G4) * 4;
        float4_t s = acc[o];
        for (int p = 0; p < TP; ++p) {
          const float a = xs[p * KS + kk];
          const float4 d = *(const float4*)(ds + p * NP + k4);
          s[0] = fmaf(d.x, a, s[0]);
          s[1] = fmaf(d.y, a, s[1]);
          s[2] = fmaf(d.z, a, s[2]);
          s[3] = fmaf(d.w, a, s[3]);
        }
        acc[o] = s;
      }
    }
  }
#pragma unroll
  for (int o = 0; o < 2; ++o) {
    const int t = tid + o * 256;
    if (t < tasks) {
      const int kk = t / G4, k4 = (t - kk * G4) * 4;
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (k4 + e < N) partial[(int64_t)blockIdx.x * MN + (int64_t)(k4 + e) * K + kk] = acc[o][e];
    }
  }
}

// Filter gradient, one output pixel per thread for the staging: the thread
// gathers its pixel's im2col row and output-gradient row into LDS (pixel
// decomposed once, taps walked with counters, eight loads in flight), then
// each thread accumulates four filter elements over the block's PX pixels.
// partial[b][k][kk] as conv_small_filter_kernel, PX pixels per block.
template <class T>
__global__ void __launch_bounds__(256)
conv_small_filter_px_kernel(const typename T::storage* __restrict__ x, const typename T::storage* __restrict__ dy,
                            ConvGeom g, int64_t P, float* __restrict__ partial) {
  extern __shared__ float smem[];
  const int K = g.r * g.s * g.c, N = g.k, MN = N * K, KS = odd_stride(K), NP = quad_pad(N);
  float* xs = smem;            // [PX][KS] im2col rows
  float* ds = smem + PX * KS;  // [PX][NP] output gradient rows (zero beyond N)
  const int tid = threadIdx.x;
  const int64_t pix = (int64_t)blockIdx.x * PX + tid;
  float* xrow = xs + tid * KS;
  float* drow = ds + tid * NP;
  if (pix < P) {
    const int mi = (int)pix, hw = g.ho * g.wo;  // pixel counts below 2^31 on this path
    const int n = mi / hw, rem = mi - n * hw, i = rem / g.wo, j = rem - i * g.wo;
    const typename T::storage* xn = x + (int64_t)n * g.h * g.w * g.c;
    int tr = 0, ts = 0, ch = 0;
    for (int kb = 0; kb < K; kb += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int y = i + tr - g.pad, xx = j + ts - g.pad;
        const bool ok = kb + u < K && (unsigned)y < (unsigned)g.h && (unsigned)xx < (unsigned)g.w;
        const float val = to_f<T>(xn[ok ? ((int64_t)y * g.w + xx) * g.c + ch : 0]);
        v[u] = ok ? val : 0.0f;
        if (++ch == g.c) {
          ch = 0;
          if (++ts == g.s) {
            ts = 0;
            ++tr;
          }
        }
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (kb + u < K) xrow[kb + u] = v[u];
    }
    const typename T::storage* drp = dy + pix * N;
    for (int kb = 0; kb < NP; kb += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const bool ok = kb + u < N;
        const float val = to_f<T>(drp[ok ? kb + u : 0]);
        v[u] = ok ? val : 0.0f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (kb + u < NP) drow[kb + u] = v[u];
    }
  } else {
    for (int kk = 0; kk < K; ++kk) xrow[kk] = 0.0f;
    for (int k = 0; k < NP; ++k) drow[k] = 0.0f;
  }
  __syncthreads();
  const int G4 = NP / 4, tasks = G4 * K;
  for (int t = tid; t < tasks; t += 256) {
    const int kk = t / G4, k4 = (t - kk * G4) * 4;
    float4_t s = {0.f, 0.f, 0.f, 0.f};
    for (int p = 0; p < PX; ++p) {
      const float a = xs[p * KS + kk];
      const float4 d = *(const float4*)(ds + p * NP + k4);
      s[0] = fmaf(d.x, a, s[0]);
      s[1] = fmaf(d.y, a, s[1]);
      s[2] = fmaf(d.z, a, s[2]);
      s[3] = fmaf(d.w, a, s[3]);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (k4 + e < N) partial[(int64_t)blockIdx.x * MN + (int64_t)(k4 + e) * K + kk] = s[e];
  }
}

// ---------------------------------------------------------------------------
// 16-bit data with K = r*s*c_in <= 32: the whole reduction of a forward
// output is one 32-deep MFMA step, and the filter gradient is a product of
// depth n*ho*wo with a 32 x 32 (or smaller) result; both run on the matrix
// cores.  Fragments are gathered straight from global memory (x is small
// and stays in the caches): lane l owns row l % 16 of a 16 x 32 operand
// fragment and the eight consecutive reduction indices 8 (l / 16) .. + 7,
// zero past the reduction, in the padding or past the last pixel.
// ---------------------------------------------------------------------------

// Eight consecutive im2col entries (pixel m, columns kk0 .. kk0 + 7) of a
// stride-1 convolution, as packed 16-bit bits.
template <class T>
__device__ __forceinline__ uint4 im2col8(const typename T::storage* __restrict__ x, const ConvGeom& g, int m,
                                         bool m_ok, int kk0, int K) {
  uint16_t v[8];
  const int hw = g.ho * g.wo;
  const int n = m / hw, rem = m - n * hw, i = rem / g.wo, j = rem - i * g.wo;
  int tap = kk0 / g.c, ch = kk0 - tap * g.c;
  int tr = tap / g.s, ts = tap - tr * g.s;
  const typename T::storage* xn = x + (int64_t)n * g.h * g.w * g.c;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int y = i + tr - g.pad, xx = j + ts - g.pad;
    const bool ok = m_ok && kk0 + e < K && (unsigned)y < (unsigned)g.h && (unsigned)xx < (unsigned)g.w;
    const uint16_t val = xn[ok ? ((int64_t)y * g.w + xx) * g.c + ch : 0];
    v[e] = ok ? val : (uint16_t)0;
    if (++ch == g.c) {
      ch = 0;
      if (++ts == g.s) {
        ts = 0;
        ++tr;
      }
    }
  }
  return pack8(v);
}

// y[m][n] = epi(sum_kk im2col[m][kk] w[n][kk]): a wave loads the filter's
// fragments once (all output channels, up to 64, 16 per MFMA), then handles
// MF_Q blocks of 16 output pixels with every block's gathers in flight
// together before any of its products.
constexpr int MF_NB = 4;
constexpr int MF_Q = 4;
template <class T, class OutT>
__global__ void __launch_bounds__(256)
conv_small_fwd_mfma_kernel(const typename T::storage* __restrict__ x, const typename T::storage* __restrict__ w,
                           ConvGeom g, int64_t M, Epilogue ep) {
  const int lane = threadIdx.x & 63;
  const int K = g.r * g.s * g.c, N = g.k, nb_n = (N + 15) / 16;
  const int64_t pb0 = ((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6)) * MF_Q;
  if (pb0 * 16 >= M) return;
  const int kk0 = 8 * (lane >> 4);
  uint4 wf[MF_NB];
#pragma unroll
  for (int nb = 0; nb < MF_NB; ++nb) {
    const int n = nb * 16 + (lane & 15);
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const bool ok = nb < nb_n && n < N && kk0 + e < K;
      const uint16_t val = w[ok ? (int64_t)n * K + kk0 + e : 0];
      v[e] = ok ? val : (uint16_t)0;
    }
    wf[nb] = pack8(v);
  }
  uint4 a[MF_Q];
#pragma unroll
  for (int q = 0; q < MF_Q; ++q) {
    const int64_t m = (pb0 + q) * 16 + (lane & 15);
    a[q] = im2col8<T>(x, g, (int)(m < M ? m : 0), m < M, kk0, K);
  }
  const int64_t nrow = 4 * (lane >> 4);
#pragma unroll
  for (int q = 0; q < MF_Q; ++q) {
    const int64_t mrow = (pb0 + q) * 16 + (lane & 15);
#pragma unroll
    for (int nb = 0; nb < MF_NB; ++nb) {
      if (nb < nb_n) {
        const float4_t acc = Mfma<T>::run(wf[nb], a[q], (float4_t){0.f, 0.f, 0.f, 0.f});
        epilogue_store4<T, OutT>(ep, M, N, mrow, nb * 16 + nrow, acc);
      }
    }
  }
}

// partial[b][k][kk] = sum over block b's pixels of dy[p][k] * im2col[p][kk]
// (c_out <= 32, K <= 32): each wave takes every fourth pair of 32-pixel steps
// of the block's range (both steps' fragments gathered before their
// products), and the four waves' sums are added in wave order in LDS.
constexpr int MF_FILTER_PAIRS = 2;  // pairs of 32-pixel steps per wave
constexpr int64_t MF_FILTER_PIXELS = 4 * MF_FILTER_PAIRS * 64;

// A = dy^T (rows k) and B^T = im2col^T (rows kk) fragments of the 32-pixel
// step whose lane pixels start at p0.
template <class T>
__device__ __forceinline__ void filter_frags(const typename T::storage* __restrict__ x,
                                             const typename T::storage* __restrict__ dy, const ConvGeom& g,
                                             int64_t P, int64_t p0, int lane, int K, uint4 (&af)[2], uint4 (&bf)[2]) {
  const int N = g.k;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb) {
    const int k = mb * 16 + (lane & 15);
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const bool ok = k < N && p0 + e < P;
      const uint16_t val = dy[ok ? (p0 + e) * N + k : 0];
      v[e] = ok ? val : (uint16_t)0;
    }
    af[mb] = pack8(v);
  }
#pragma unroll
  for (int tb = 0; tb < 2; ++tb) {
    const int kk = tb * 16 + (lane & 15);
    const int tap = kk / g.c, ch = kk - tap * g.c, tr = tap / g.s, ts = tap - tr * g.s;
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int64_t p = p0 + e;
      bool ok = kk < K && p < P;
      int64_t off = 0;
      if (ok) {
        const int pi = (int)p, hw = g.ho * g.wo;
        const int n = pi / hw, rem = pi - n * hw, i = rem / g.wo, j = rem - i * g.wo;
        const int y = i + tr - g.pad, xx = j + ts - g.pad;
        ok = (unsigned)y < (unsigned)g.h && (unsigned)xx < (unsigned)g.w;
        off = (((int64_t)n * g.h + y) * g.w + xx) * g.c + ch;
      }
      const uint16_t val = x[ok ? off : 0];
      v[e] = ok ? val : (uint16_t)0;
    }
    bf[tb] = pack8(v);
  }
}

template <class T>
__global__ void __launch_bounds__(256)
conv_small_filter_mfma_kernel(const typename T::storage* __restrict__ x, const typename T::storage* __restrict__ dy,
                              ConvGeom g, int64_t P, float* __restrict__ partial) {
  __shared__ float red[3][4][64][4];  // waves 1..3: [wave][fragment][lane][4]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int K = g.r * g.s * g.c, N = g.k;
  float4_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = (float4_t){0.f, 0.f, 0.f, 0.f};
  const int pk0 = 8 * (lane >> 4);  // this lane's 8 pixels within a 32-pixel step
  for (int pr = 0; pr < MF_FILTER_PAIRS; ++pr) {
    const int64_t s0 = (int64_t)blockIdx.x * MF_FILTER_PIXELS + (int64_t)(pr * 4 + wave) * 64;
    if (s0 >= P) break;
    uint4 af[2][2], bf[2][2];
#pragma unroll
    for (int h = 0; h < 2; ++h) filter_frags<T>(x, dy, g, P, s0 + h * 32 + pk0, lane, K, af[h], bf[h]);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int tb = 0; tb < 2; ++tb)
#pragma unroll
        for (int mb = 0; mb < 2; ++mb) acc[mb][tb] = Mfma<T>::run(bf[h][tb], af[h][mb], acc[mb][tb]);
  }
  // acc[mb][tb][e] = D[k = mb*16 + lane%16][kk = tb*16 + 4*(lane/16) + e]
  if (wave > 0) {
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int tb = 0; tb < 2; ++tb)
        *(float4_t*)red[wave - 1][mb * 2 + tb][lane] = acc[mb][tb];
  }
  __syncthreads();
  if (wave > 0) return;
  const int MN = N * K;
#pragma unroll
  for (int mb = 0; mb < 2; ++mb)
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      float4_t s = acc[mb][tb];
      for (int wv = 0; wv < 3; ++wv) s += *(const float4_t*)red[wv][mb * 2 + tb][lane];
      const int k = mb * 16 + (lane & 15), kk = tb * 16 + 4 * (lane >> 4);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (k < N && kk + e < K) partial[(int64_t)blockIdx.x * MN + (int64_t)k * K + kk + e] = s[e];
    }
}

bool mfma_small(const ConvGeom& g, mdnn_dtype_t io) { return io != MDNN_F32 && g.r * g.s * g.c <= 32; }

constexpr int64_t FILTER_PIXELS = 128;  // pixels per block of the filter gradient (enough blocks to hide the staging latency)
constexpr size_t LDS_LIMIT = 65536;      // dynamic LDS bytes per block

size_t fwd_lds(const ConvGeom& g) {
  const int K = g.r * g.s * g.c;
  return ((size_t)TP * odd_stride(K) + (size_t)K * quad_pad(g.k)) * sizeof(float);
}
size_t fwd_px_lds(const ConvGeom& g) {
  const int K = g.r * g.s * g.c;
  return ((size_t)PX * odd_stride(K) + (size_t)K * quad_pad(g.k)) * sizeof(float);
}
bool fwd_px_ok(const ConvGeom& g) { return quad_pad(g.k) <= 4 * PX_QUADS && fwd_px_lds(g) <= LDS_LIMIT; }
size_t filter_lds(const ConvGeom& g) {
  return (size_t)TP * (odd_stride(g.r * g.s * g.c) + quad_pad(g.k)) * sizeof(float);
}
size_t filter_px_lds(const ConvGeom& g) {
  return (size_t)PX * (odd_stride(g.r * g.s * g.c) + quad_pad(g.k)) * sizeof(float);
}
bool filter_px_ok(const ConvGeom& g) { return filter_px_lds(g) <= LDS_LIMIT; }

}  // namespace

static bool pixels_fit(const ConvGeom& g) { return (int64_t)g.n * g.ho * g.wo < ((int64_t)1 << 31); }

bool conv_small_fwd_ok(const ConvGeom& g) {
  return g.r * g.s * g.c <= 64 && g.k <= 256 && fwd_lds(g) <= LDS_LIMIT && pixels_fit(g);
}

template <class T, class OutT>
static void small_fwd_launch(const ConvGeom& g, const void* x, const void* w, const Epilogue& ep, int64_t M,
                             bool px, hipStream_t st) {
  typedef typename T::storage S;
  if (px)
    hipLaunchKernelGGL((conv_small_fwd_px_kernel<T, OutT>), dim3((unsigned)ceil_div(M, PX)), dim3(256),
                       fwd_px_lds(g), st, (const S*)x, (const S*)w, g, M, ep);
  else
    hipLaunchKernelGGL((conv_small_fwd_kernel<T, OutT>), dim3((unsigned)ceil_div(M, TP)), dim3(256), fwd_lds(g),
                       st, (const S*)x, (const S*)w, g, M, ep);
}

template <class T, class OutT>
static void small_fwd_mfma_launch(const ConvGeom& g, const void* x, const void* w, const Epilogue& ep, int64_t M,
                                  hipStream_t st) {
  typedef typename T::storage S;
  hipLaunchKernelGGL((conv_small_fwd_mfma_kernel<T, OutT>), dim3((unsigned)ceil_div(M, 64 * MF_Q)), dim3(256), 0, st,
                     (const S*)x, (const S*)w, g, M, ep);
}

mdnn_status_t conv_small_fwd(const ConvGeom& g, const void* x, const void* w, const Epilogue& ep, mdnn_dtype_t io,
                             mdnn_dtype_t out, hipStream_t st) {
  const int64_t M = (int64_t)g.n * g.ho * g.wo;
  if (M == 0) return MDNN_SUCCESS;
  if (ceil_div(M, TP) > 0x7fffffffLL) return fail(MDNN_ERR_SHAPE, "conv: too many output pixels");
  if (mfma_small(g, io) && g.k <= 16 * MF_NB) {
    // one 32-deep matrix-core step per 16 pixels x 16 channels
    if (io == MDNN_F16) {
      if (out == MDNN_F32) small_fwd_mfma_launch<F16, F32>(g, x, w, ep, M, st);
      else small_fwd_mfma_launch<F16, F16>(g, x, w, ep, M, st);
    } else {
      if (out == MDNN_F32) small_fwd_mfma_launch<BF16, F32>(g, x, w, ep, M, st);
      else small_fwd_mfma_launch<BF16, BF16>(g, x, w, ep, M, st);
    }
    return check_launch("conv_small_fwd_mfma_kernel");
  }
  // one pixel per thread when c_out fits its registers
  const bool px = fwd_px_ok(g);
  if (io == MDNN_F16) {
    if (out == MDNN_F32) small_fwd_launch<F16, F32>(g, x, w, ep, M, px, st);
    else small_fwd_launch<F16, F16>(g, x, w, ep, M, px, st);
  } else if (io == MDNN_BF16) {
    if (out == MDNN_F32) small_fwd_launch<BF16, F32>(g, x, w, ep, M, px, st);
    else small_fwd_launch<BF16, BF16>(g, x, w, ep, M, px, st);
  } else {
    small_fwd_launch<F32, F32>(g, x, w, ep, M, px, st);
  }
  return check_launch("conv_small_fwd_kernel");
}

// the matrix-core filter gradient: 16-bit data, K <= 32, c_out <= 32
static bool filter_mfma_ok(const ConvGeom& g, mdnn_dtype_t io) { return mfma_small(g, io) && g.k <= 32; }

int64_t conv_small_filter_blocks(const ConvGeom& g, mdnn_dtype_t io) {
  const int K = g.r * g.s * g.c;
  if (K > 64 || g.k > 256 || (int64_t)g.k * K > 1024 || filter_lds(g) > LDS_LIMIT || !pixels_fit(g)) return 0;
  const int64_t P = (int64_t)g.n * g.ho * g.wo;
  if (filter_mfma_ok(g, io)) return ceil_div(P, MF_FILTER_PIXELS);
  return ceil_div(P, filter_px_ok(g) ? (int64_t)PX : FILTER_PIXELS);
}

// one pixel per thread when the block's rows fit in LDS (the block count
// conv_small_filter_blocks gives matches the kernel chosen here)
template <class T>
static void small_filter_launch(const ConvGeom& g, const void* x, const void* dy, int64_t P, int64_t blocks,
                                float* part, hipStream_t st) {
  typedef typename T::storage S;
  if (filter_px_ok(g))
    hipLaunchKernelGGL((conv_small_filter_px_kernel<T>), dim3((unsigned)blocks), dim3(256), filter_px_lds(g), st,
                       (const S*)x, (const S*)dy, g, P, part);
  else
    hipLaunchKernelGGL((conv_small_filter_kernel<T>), dim3((unsigned)blocks), dim3(256), filter_lds(g), st,
                       (const S*)x, (const S*)dy, g, P, FILTER_PIXELS, part);
}

mdnn_status_t conv_small_filter(const ConvGeom& g, const void* x, const void* dy, float* dw, void* ws,
                                mdnn_dtype_t io, hipStream_t st, ReduceBatch* defer) {
  const int64_t blocks = conv_small_filter_blocks(g, io);
  const int64_t P = (int64_t)g.n * g.ho * g.wo;
  if (blocks <= 0 || blocks > 0x7fffffffLL) return fail(MDNN_ERR_SHAPE, "conv: filter gradient shape");
  float* part = (float*)ws;
  if (filter_mfma_ok(g, io)) {
    if (io == MDNN_F16)
      hipLaunchKernelGGL(conv_small_filter_mfma_kernel<F16>, dim3((unsigned)blocks), dim3(256), 0, st,
                         (const uint16_t*)x, (const uint16_t*)dy, g, P, part);
    else
      hipLaunchKernelGGL(conv_small_filter_mfma_kernel<BF16>, dim3((unsigned)blocks), dim3(256), 0, st,
                         (const uint16_t*)x, (const uint16_t*)dy, g, P, part);
    MDNN_TRY(check_launch("conv_small_filter_mfma_kernel"));
    return reduce_splits(part, (int)blocks, g.k, (int64_t)g.r * g.s * g.c, dw, st, defer);
  }
  if (io == MDNN_F16) small_filter_launch<F16>(g, x, dy, P, blocks, part, st);
  else if (io == MDNN_BF16) small_filter_launch<BF16>(g, x, dy, P, blocks, part, st);
  else small_filter_launch<F32>(g, x, dy, P, blocks, part, st);
  MDNN_TRY(check_launch("conv_small_filter_kernel"));
  return reduce_splits(part, (int)blocks, g.k, (int64_t)g.r * g.s * g.c, dw, st, defer);
}

}  // namespace mdnn
