// Skinny products: section 3.2's D = C + A*B where one dimension is tiny -- a
// regression head (N = 1), the weight gradient of a narrow head (TN with
// N <= 16) and the back-propagation through a regression head (K <= 4).  An
// MFMA tile would be almost all padding and the product is bound by streaming
// the large operand, so these kernels read it once with wide loads on the
// vector ALUs, accumulate in fp32 and reduce in a fixed order (deterministic).
//
//   rows  (A K-contiguous, N <= 4, or N <= 16 on at most 2048 rows): B is
//         staged in LDS as [N][K]; one wave (or four, when rows are few) per
//         output row, 8 consecutive k per lane, butterfly sum per column.
//   cols  (TN, N <= 16): a lane owns MB consecutive m, the block's four waves
//         take every fourth k of the block's K range and are combined in wave
//         order; with a workspace K is split across blocks into fp32 partials
//         that the split reduction sums before the epilogue.
//   depth (K <= 4, any layout): one thread per eight consecutive outputs of
//         a row (write-bound: the outer-product shape of back-propagating
//         through a regression head).
#include "gemm_skinny.h"

namespace mdnn {

int gemm_tile_override();

namespace {

template <class T> constexpr mdnn_dtype_t code_of();
template <> constexpr mdnn_dtype_t code_of<F32>() { return MDNN_F32; }
template <> constexpr mdnn_dtype_t code_of<F16>() { return MDNN_F16; }
template <> constexpr mdnn_dtype_t code_of<BF16>() { return MDNN_BF16; }

constexpr int NMAX = 16;          // widest "skinny" N
constexpr int KMAX_DEPTH = 4;     // deepest product of the depth kernel
constexpr size_t ROWS_LDS = 65536;
constexpr int64_t ROWS_WIDE_MAX_M = 2048;  // 4 < N <= 16: few rows only

template <class T>
__device__ __forceinline__ float ldf(const typename T::storage* p) { return to_f<T>(*p); }

// base[off] if ok, else 0, without a branch around the load: the address is
// clamped to base[0] (an element of the operand) and the value selected, so
// several guarded loads can be in flight at once (a load inside a divergent
// branch is waited for before the branch joins).
template <class T>
__device__ __forceinline__ float ldz(const typename T::storage* base, int64_t off, bool ok) {
  const float v = to_f<T>(base[ok ? off : 0]);
  return ok ? v : 0.0f;
}

// Eight consecutive elements as floats (p aligned to 16 bytes).
template <class T>
__device__ __forceinline__ void load8(const typename T::storage* p, float (&o)[8]) {
  if constexpr (sizeof(typename T::storage) == 4) {
    const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
    o[0] = a.x, o[1] = a.y, o[2] = a.z, o[3] = a.w, o[4] = b.x, o[5] = b.y, o[6] = b.z, o[7] = b.w;
  } else {
    const uint4 q = *(const uint4*)p;
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = to_f<T>((uint16_t)(w[e >> 1] >> ((e & 1) * 16)));
  }
}

__device__ __forceinline__ float wave_sum64(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Epilogue of up to NMAX outputs of row m held in acc (lane-uniform values).
template <class T, class OutT>
__device__ __forceinline__ void store_row(const Epilogue& ep, int64_t M, int N, int64_t m, const float (&acc)[NMAX]) {
#pragma unroll
  for (int q = 0; q < NMAX / 4; ++q)
    if (q * 4 < N) epilogue_store4<T, OutT>(ep, M, N, m, q * 4, (float4_t){acc[4 * q], acc[4 * q + 1], acc[4 * q + 2], acc[4 * q + 3]});
}

// ---------------------------------------------------------------------------
// rows: D[m][n] = sum_k A[m][k] B(k, n); B(k, n) = B[k*ldb + n] (NN) or
// B[n*ldb + k] (NT).  WPR waves share a row (few rows: more waves busy), each
// taking every WPR-th chunk of 512 k; their sums are added in wave order.
// ---------------------------------------------------------------------------
template <class T, int N_>
__device__ __forceinline__ void rows_chunk(const float (&a)[8], const float* Bs, int Kp, int N, int k0,
                                           float (&acc)[NMAX]) {
#pragma unroll
  for (int n = 0; n < NMAX; ++n) {
    if (n < N) {
      const float4 b0 = *(const float4*)(Bs + n * Kp + k0), b1 = *(const float4*)(Bs + n * Kp + k0 + 4);
      float s = acc[n];
      s = fmaf(a[0], b0.x, s), s = fmaf(a[1], b0.y, s), s = fmaf(a[2], b0.z, s), s = fmaf(a[3], b0.w, s);
      s = fmaf(a[4], b1.x, s), s = fmaf(a[5], b1.y, s), s = fmaf(a[6], b1.z, s), s = fmaf(a[7], b1.w, s);
      acc[n] = s;
    }
  }
}

template <class T, class OutT, bool B_NK, int WPR>
__global__ void __launch_bounds__(256)
skinny_rows_kernel(const typename T::storage* __restrict__ A, int64_t lda, const typename T::storage* __restrict__ B,
                   int64_t ldb, int64_t M, int N, int K, int Kp, bool vec, bool vec_b, Epilogue ep) {
  extern __shared__ float Bs[];  // [N][Kp], zero beyond K
  __shared__ float part[4][NMAX];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (vec_b) {
    // B's K x N (NN, ldb = N) or N x K (NT, ldb = K) elements are one
    // 16-byte aligned run: eight per load, all of a thread's loads in flight
    // (Kp = K here, a multiple of 8)
    constexpr int VB = 16 / sizeof(typename T::storage);
    const int nv = N * K / VB;
    for (int base = 0; base < nv; base += 4 * 256) {
      float v[4][VB];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = base + u * 256 + tid;
        const int ic = i < nv ? i : 0;
        if constexpr (VB == 8) {
          load8<T>(B + (int64_t)ic * 8, v[u]);
        } else {
          const float4 q = *(const float4*)(B + (int64_t)ic * 4);
          v[u][0] = q.x, v[u][1] = q.y, v[u][2] = q.z, v[u][3] = q.w;
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = base + u * 256 + tid;
        if (i < nv)
#pragma unroll
          for (int e = 0; e < VB; ++e) {
            const int f = i * VB + e;  // flat index into B's run
            const int k = B_NK ? f % K : f / N, n = B_NK ? f / K : f % N;
            Bs[n * Kp + k] = v[u][e];
          }
      }
    }
  }
  // eight loads per thread in flight, then their stores
  for (int base = 0; base < N * Kp && !vec_b; base += 8 * 256) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int idx = base + u * 256 + tid;
      const int n = idx / Kp, k = idx - n * Kp;
      v[u] = ldz<T>(B, B_NK ? (int64_t)n * ldb + k : (int64_t)k * ldb + n, idx < N * Kp && k < K);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int idx = base + u * 256 + tid;
      if (idx < N * Kp) Bs[idx] = v[u];
    }
  }
  __syncthreads();
  constexpr int RPB = 4 / WPR;  // rows per block and round
  const int sub = wave % WPR;
  const int64_t rounds = ceil_div(M, (int64_t)gridDim.x * RPB);
  for (int64_t r = 0; r < rounds; ++r) {
    const int64_t m = (r * gridDim.x + blockIdx.x) * RPB + wave / WPR;
    float acc[NMAX];
#pragma unroll
    for (int n = 0; n < NMAX; ++n) acc[n] = 0.0f;
    if (m < M) {
      const typename T::storage* a_row = A + m * lda;
      const int stride = 512 * WPR;  // k distance between this wave's chunks
      int base = sub * 512;
      if (vec) {
        // four chunks in flight, no per-lane guards while all four fit
        for (; base + 3 * stride + 512 <= K; base += 4 * stride) {
          float a[4][8];
#pragma unroll
          for (int u = 0; u < 4; ++u) load8<T>(a_row + base + u * stride + lane * 8, a[u]);
#pragma unroll
          for (int u = 0; u < 4; ++u) rows_chunk<T, 0>(a[u], Bs, Kp, N, base + u * stride + lane * 8, acc);
        }
      }
      for (; base < K; base += stride) {
        const int k0 = base + lane * 8;
        float a[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) a[e] = ldz<T>(a_row, k0 + e, k0 + e < K);
        if (k0 < K) rows_chunk<T, 0>(a, Bs, Kp, N, k0, acc);
      }
#pragma unroll
      for (int n = 0; n < NMAX; ++n)
        if (n < N) acc[n] = wave_sum64(acc[n]);
    }
    if (WPR > 1) {
      if (lane == 0 && m < M) {
#pragma unroll
        for (int n = 0; n < NMAX; ++n) part[wave][n] = acc[n];
      }
      __syncthreads();
      if (sub == 0 && lane == 0 && m < M) {
#pragma unroll
        for (int w = 1; w < WPR; ++w)
#pragma unroll
          for (int n = 0; n < NMAX; ++n) acc[n] += part[wave + w][n];
        store_row<T, OutT>(ep, M, N, m, acc);
      }
      __syncthreads();
    } else if (lane == 0 && m < M) {
      store_row<T, OutT>(ep, M, N, m, acc);
    }
  }
}

// ---------------------------------------------------------------------------
// cols: D[m][n] = sum_k A[k][m] B[k][n] (TN), lane owns MB consecutive m.
// ---------------------------------------------------------------------------
template <class T, class OutT, int MB, int NB>
__global__ void __launch_bounds__(256)
skinny_cols_kernel(const typename T::storage* __restrict__ A, int64_t lda, const typename T::storage* __restrict__ B,
                   int64_t ldb, int64_t M, int N, int64_t K, int64_t k_per_split, bool vec, Epilogue ep) {
  __shared__ float red[3][64 * MB * NB];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t m0 = ((int64_t)blockIdx.x * 64 + lane) * MB;
  const int64_t kbeg = (int64_t)blockIdx.y * k_per_split;
  const int64_t kend = kbeg + k_per_split < K ? kbeg + k_per_split : K;
  float acc[MB][NB];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int n = 0; n < NB; ++n) acc[i][n] = 0.0f;
  const bool full = vec && m0 + MB <= M;
  // wave w takes k = kbeg + w, +4, +8, ...; four of its k in flight at once
  for (int64_t kb = kbeg + wave; kb < kend; kb += 16) {
    float a[4][MB];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t k = kb + 4 * u;
      const bool kin = k < kend;
      bool done = false;
      if constexpr (MB == 8) {
        if (full) {
          // the whole row of eight in one vector load; a k beyond the range
          // re-reads row kbeg (in range) and is multiplied by b = 0 below
          load8<T>(A + (kin ? k : kbeg) * lda + m0, a[u]);
          done = true;
        }
      }
      if (!done) {
#pragma unroll
        for (int i = 0; i < MB; ++i) a[u][i] = ldz<T>(A, k * lda + m0 + i, kin && m0 + i < M);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int64_t k = kb + 4 * u;
      const bool kin = k < kend;
      float b[NB];
#pragma unroll
      for (int n = 0; n < NB; ++n) b[n] = ldz<T>(B, k * ldb + n, kin && n < N);
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int n = 0; n < NB; ++n) acc[i][n] = fmaf(a[u][i], b[n], acc[i][n]);
    }
  }
  // waves 1..3 hand their sums to wave 0, which adds them in wave order
  if (wave > 0) {
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int n = 0; n < NB; ++n) red[wave - 1][(i * NB + n) * 64 + lane] = acc[i][n];
  }
  __syncthreads();
  if (wave > 0) return;
#pragma unroll
  for (int w = 0; w < 3; ++w)
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int n = 0; n < NB; ++n) acc[i][n] += red[w][(i * NB + n) * 64 + lane];
#pragma unroll
  for (int i = 0; i < MB; ++i) {
    const int64_t m = m0 + i;
    if (m >= M) break;
    if (ep.partial) {
      float* p = ep.partial + ((int64_t)blockIdx.y * M + m) * N;
#pragma unroll
      for (int n = 0; n < NB; ++n)
        if (n < N) p[n] = acc[i][n];
    } else {
#pragma unroll
      for (int q = 0; q < (NB + 3) / 4; ++q) {
        float4_t v;
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = q * 4 + e < NB ? acc[i][q * 4 + e] : 0.0f;
        if (q * 4 < N) epilogue_store4<T, OutT>(ep, M, N, m, q * 4, v);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// depth: K <= KT (1 or 4), any layout; eight consecutive n per thread.
// ---------------------------------------------------------------------------
template <class T, class OutT, int KT>
__global__ void __launch_bounds__(256)
skinny_depth_kernel(mdnn_layout_t layout, const typename T::storage* __restrict__ A, int64_t lda,
                    const typename T::storage* __restrict__ B, int64_t ldb, int64_t M, int64_t N, int K,
                    Epilogue ep) {
  // x: eight consecutive n per thread (B held in registers, K <= KT); y:
  // rows, grid-stride, so each thread reuses its B over several rows
  const int64_t n = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
  if (n >= N) return;
  // this thread's eight columns inside N with vector access (rows m < M by the loop)
  const bool full = full_tile_epilogue(ep, n + 8 <= N, N);
  float b[8][KT];
#pragma unroll
  for (int e = 0; e < 8; ++e)
#pragma unroll
    for (int k = 0; k < KT; ++k)
      b[e][k] = ldz<T>(B, layout == MDNN_NT ? (n + e) * ldb + k : (int64_t)k * ldb + n + e, k < K && n + e < N);
  // a ReLU mask with nothing else after the product (back-propagation into a
  // hidden layer): four of this thread's rows with their mask runs loaded
  // before any is stored, the mask applied before the epilogue (alpha * 0 is
  // still 0).  A row at a time, each mask load waited for behind the previous
  // row's stores, had left the 4096 x 4096 outer product at 3 TB/s.
  if (full && ep.mask && ep.beta == 0.0f && !ep.bias && ep.act == MDNN_ACT_NONE && (ep.ldm & 7) == 0 &&
      ((uintptr_t)ep.mask & 15) == 0) {
    constexpr int RB = 4;
    Epilogue e2 = ep;
    e2.mask = nullptr;
    const typename T::storage* mk = (const typename T::storage*)ep.mask;
    for (int64_t m0 = blockIdx.y; m0 < M; m0 += RB * (int64_t)gridDim.y) {
      float a[RB][KT], mv[RB][8];
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        const int64_t m = m0 + r * (int64_t)gridDim.y, mm = m < M ? m : m0;
#pragma unroll
        for (int k = 0; k < KT; ++k)
          a[r][k] = ldz<T>(A, layout == MDNN_TN ? (int64_t)k * lda + mm : mm * lda + k, k < K);
        load8<T>(mk + mm * ep.ldm + n, mv[r]);
      }
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        const int64_t m = m0 + r * (int64_t)gridDim.y;
        if (m >= M) break;
        float4_t lo = {0.f, 0.f, 0.f, 0.f}, hi = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int k = 0; k < KT; ++k) {
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            lo[e] = fmaf(a[r][k], b[e][k], lo[e]);
            hi[e] = fmaf(a[r][k], b[4 + e][k], hi[e]);
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (!(mv[r][e] > 0.0f)) lo[e] = 0.0f;
          if (!(mv[r][4 + e] > 0.0f)) hi[e] = 0.0f;
        }
        epilogue_store4<T, OutT, true>(e2, M, N, m, n, lo);
        epilogue_store4<T, OutT, true>(e2, M, N, m, n + 4, hi);
      }
    }
    return;
  }
  for (int64_t m = blockIdx.y; m < M; m += gridDim.y) {
    float a[KT];
#pragma unroll
    for (int k = 0; k < KT; ++k) a[k] = ldz<T>(A, layout == MDNN_TN ? (int64_t)k * lda + m : m * lda + k, k < K);
    float4_t lo = {0.f, 0.f, 0.f, 0.f}, hi = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int k = 0; k < KT; ++k) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        lo[e] = fmaf(a[k], b[e][k], lo[e]);
        hi[e] = fmaf(a[k], b[4 + e][k], hi[e]);
      }
    }
    if (full) {
      epilogue_store4<T, OutT, true>(ep, M, N, m, n, lo);
      epilogue_store4<T, OutT, true>(ep, M, N, m, n + 4, hi);
    } else {
      epilogue_store4<T, OutT>(ep, M, N, m, n, lo);
      if (n + 4 < N) epilogue_store4<T, OutT>(ep, M, N, m, n + 4, hi);
    }
  }
}

// Split of the cols kernel's K range over ~512 workgroups (whole groups of
// sixteen k: four waves with four k each in flight); splits = 1 when the
// grid is already full.
SplitPlan cols_plan(int64_t M, int64_t K, int mb) {
  SplitPlan p{1, K};
  const int64_t xb = ceil_div(M, 64 * mb);
  if (xb >= 256 || K < 32) return p;
  int64_t kps = ceil_div(ceil_div(K, ceil_div(512, xb)), 16) * 16;
  p.splits = (int)ceil_div(K, kps);
  p.k_per_split = kps;
  if (p.splits < 2 || p.splits > 65535) p = SplitPlan{1, K};
  return p;
}

int cols_mb(int64_t N) { return N <= 4 ? 8 : 2; }

// ---------------------------------------------------------------------------
// rows with N = 1, 16-bit, both operands k-contiguous and 16-byte aligned (a
// one-output head's forward product): D[m] = sum_k A[m][k] B[k], one wave per
// row; each lane loads its 16-byte runs of A and of B together (no staging
// of B through LDS), a row's runs eight at a time.
// ---------------------------------------------------------------------------
template <class T>
__device__ __forceinline__ void dot8(const uint4& a, const uint4& b, float& acc) {
  const uint32_t aw[4] = {a.x, a.y, a.z, a.w}, bw[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
  for (int e = 0; e < 8; ++e)
    acc = fmaf(to_f<T>((uint16_t)(aw[e >> 1] >> ((e & 1) * 16))), to_f<T>((uint16_t)(bw[e >> 1] >> ((e & 1) * 16))),
               acc);
}

template <class T, class OutT>
__global__ void __launch_bounds__(256)
skinny_rows1_kernel(const uint16_t* __restrict__ A, int64_t lda, const uint16_t* __restrict__ B, int64_t M, int K,
                    Epilogue ep) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t m = (int64_t)blockIdx.x * 4 + wave;
  if (m >= M) return;  // whole waves; the kernel has no barrier
  const uint16_t* a_row = A + m * lda;
  float acc = 0.0f;
  int base = 0;
  for (; base + 8 * 512 <= K; base += 8 * 512) {
    uint4 va[8], vb[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      va[u] = *(const uint4*)(a_row + base + u * 512 + lane * 8);
      vb[u] = *(const uint4*)(B + base + u * 512 + lane * 8);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) dot8<T>(va[u], vb[u], acc);
  }
  for (; base + 512 <= K; base += 512)
    dot8<T>(*(const uint4*)(a_row + base + lane * 8), *(const uint4*)(B + base + lane * 8), acc);
  if (base < K) {
    const int k0 = base + lane * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (k0 + e < K) acc = fmaf(to_f<T>(a_row[k0 + e]), to_f<T>(B[k0 + e]), acc);
  }
  acc = wave_sum64(acc);
  if (lane == 0) {
    float r[NMAX] = {};
    r[0] = acc;
    store_row<T, OutT>(ep, M, 1, m, r);
  }
}

// ---------------------------------------------------------------------------
// cols with N = 1 (the weight gradient of a one-output head), 16-bit A with
// M % 512 == 0: D[m] = sum_k A[k][m] B[k] is a column sum of A's rows
// weighted by B.  Chunks of COLS1_ROWS k; a block reduces one chunk x 512 m,
// each wave reading whole 1 KB runs of its rows (wave w: k = w, w + 4, ...;
// eight m per lane), the four waves combined in a fixed order, into
// partial[chunk][m] for the split reduction's epilogue.
// ---------------------------------------------------------------------------
constexpr int64_t COLS1_ROWS = 64;

template <class T>
__global__ void __launch_bounds__(256)
skinny_cols1_strip_kernel(const uint16_t* __restrict__ A, int64_t lda, const uint16_t* __restrict__ B, int64_t ldb,
                          int64_t M, int64_t K, float* __restrict__ partial) {
  __shared__ float4 red[4][2][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t m0 = (int64_t)blockIdx.x * 512 + lane * 8;
  const int64_t k0 = (int64_t)blockIdx.y * COLS1_ROWS;
  const int64_t nk = K - k0 < COLS1_ROWS ? K - k0 : COLS1_ROWS;
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  auto fma8 = [&](const uint4& v, float b) {
    const uint32_t vw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] = fmaf(to_f<T>((uint16_t)(vw[e >> 1] >> ((e & 1) * 16))), b, s[e]);
  };
  const uint16_t* base = A + (k0 + w) * lda + m0;
  if (nk == COLS1_ROWS) {
    // a whole chunk: all of this lane's rows (and their weights) are loaded
    // before any is added
    constexpr int RPW = COLS1_ROWS / 4;
    uint4 v[RPW];
    float bw[RPW];
#pragma unroll
    for (int u = 0; u < RPW; ++u) {
      v[u] = *(const uint4*)(base + (int64_t)(4 * u) * lda);
      bw[u] = to_f<T>(B[(k0 + w + 4 * u) * ldb]);
    }
#pragma unroll
    for (int u = 0; u < RPW; ++u) fma8(v[u], bw[u]);
  } else {
    for (int64_t r = w; r < nk; r += 4) fma8(*(const uint4*)(base + (r - w) * lda), to_f<T>(B[(k0 + r) * ldb]));
  }
  red[w][0][lane] = make_float4(s[0], s[1], s[2], s[3]);
  red[w][1][lane] = make_float4(s[4], s[5], s[6], s[7]);
  __syncthreads();
  // thread t: m = 2t and 2t + 1 of the block's 512 (lane t / 4's values)
  const int l = threadIdx.x >> 2, h = (threadIdx.x >> 1) & 1, q = threadIdx.x & 1;
  float2 t = make_float2(0.f, 0.f);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float4 v = red[k][h][l];
    t.x += q ? v.z : v.x;
    t.y += q ? v.w : v.y;
  }
  *(float2*)(partial + blockIdx.y * M + (int64_t)blockIdx.x * 512 + 2 * threadIdx.x) = t;
}

template <class T, class OutT>
mdnn_status_t launch_cols(const void* A, int64_t lda, const void* B, int64_t ldb, int64_t M, int64_t N, int64_t K,
                          const Epilogue& ep_in, void* ws, size_t ws_bytes, hipStream_t st) {
  typedef typename T::storage S;
  if constexpr (sizeof(S) == 2) {
    const int64_t chunks = ceil_div(K, COLS1_ROWS);
    if (N == 1 && M % 512 == 0 && K >= 512 && chunks <= 65535 && M / 512 <= 0x7fffffffLL && aligned(A, 16) &&
        lda % 8 == 0 && ws && aligned(ws, 16) && ws_bytes >= (size_t)chunks * M * sizeof(float)) {
      hipLaunchKernelGGL(skinny_cols1_strip_kernel<T>, dim3((unsigned)(M / 512), (unsigned)chunks), dim3(256), 0, st,
                         (const uint16_t*)A, lda, (const uint16_t*)B, ldb, M, K, (float*)ws);
      MDNN_TRY(check_launch("skinny_cols1_strip_kernel"));
      return reduce_splits_epilogue(ws, (int)chunks, M, N, ep_in, code_of<T>(), code_of<OutT>(), st);
    }
  }
  const int mb = cols_mb(N);
  const SplitPlan plan = cols_plan(M, K, mb);
  Epilogue ep = ep_in;
  int splits = 1;
  int64_t kps = K;
  if (plan.splits > 1 && ws && aligned(ws, 16) && ws_bytes >= (size_t)plan.splits * M * N * sizeof(float)) {
    splits = plan.splits;
    kps = plan.k_per_split;
    ep.partial = (float*)ws;
  } else {
    ep.partial = nullptr;
  }
  const int64_t xb = ceil_div(M, 64 * mb);
  if (xb > 0x7fffffffLL) return fail(MDNN_ERR_SHAPE, "gemm: problem too large for the launch grid");
  const size_t es = sizeof(S);
  const bool vec = aligned(A, es * mb) && (lda % mb) == 0;
  const dim3 grid((unsigned)xb, (unsigned)splits);
  if (mb == 8)
    hipLaunchKernelGGL((skinny_cols_kernel<T, OutT, 8, 4>), grid, dim3(256), 0, st, (const S*)A, lda, (const S*)B, ldb,
                       M, (int)N, K, kps, vec, ep);
  else
    hipLaunchKernelGGL((skinny_cols_kernel<T, OutT, 2, NMAX>), grid, dim3(256), 0, st, (const S*)A, lda, (const S*)B,
                       ldb, M, (int)N, K, kps, vec, ep);
  MDNN_TRY(check_launch("skinny_cols_kernel"));
  if (splits == 1) return MDNN_SUCCESS;
  return reduce_splits_epilogue(ws, splits, M, N, ep_in, code_of<T>(), code_of<OutT>(), st);
}

template <class T, class OutT>
mdnn_status_t launch_skinny(mdnn_layout_t layout, const void* A, int64_t lda, const void* B, int64_t ldb, int64_t M,
                            int64_t N, int64_t K, const Epilogue& ep, void* ws, size_t ws_bytes, hipStream_t st) {
  typedef typename T::storage S;
  if (K <= KMAX_DEPTH) {
    const int64_t bx = ceil_div(ceil_div(N, 8), 256);
    if (bx > 0x7fffffffLL) return fail(MDNN_ERR_SHAPE, "gemm: problem too large for the launch grid");
    // about 2048 blocks in all, each over several rows
    int64_t by = ceil_div(2048, bx);
    if (by > M) by = M;
    if (by > 65535) by = 65535;
    const dim3 grid((unsigned)bx, (unsigned)by);
    if (K == 1)
      hipLaunchKernelGGL((skinny_depth_kernel<T, OutT, 1>), grid, dim3(256), 0, st, layout, (const S*)A, lda,
                         (const S*)B, ldb, M, N, (int)K, ep);
    else
      hipLaunchKernelGGL((skinny_depth_kernel<T, OutT, 4>), grid, dim3(256), 0, st, layout, (const S*)A, lda,
                         (const S*)B, ldb, M, N, (int)K, ep);
    return check_launch("skinny_depth_kernel");
  }
  if (layout == MDNN_TN) return launch_cols<T, OutT>(A, lda, B, ldb, M, N, K, ep, ws, ws_bytes, st);
  if constexpr (sizeof(S) == 2) {
    // B's one column (NN, ldb = 1) or one row (NT) is k-contiguous
    if (N == 1 && K >= 512 && aligned(A, 16) && lda % 8 == 0 && aligned(B, 16) && (layout == MDNN_NT || ldb == 1) &&
        ceil_div(M, 4) <= 0x7fffffffLL) {
      hipLaunchKernelGGL((skinny_rows1_kernel<T, OutT>), dim3((unsigned)ceil_div(M, 4)), dim3(256), 0, st,
                         (const uint16_t*)A, lda, (const uint16_t*)B, M, (int)K, ep);
      return check_launch("skinny_rows1_kernel");
    }
  }
  const int kp = (int)ceil_div(K, 8) * 8;
  const size_t lds = (size_t)N * kp * sizeof(float);
  const bool vec = K % 8 == 0 && lda % 8 == 0 && aligned(A, 16);
  // B one contiguous run: NN with ldb = N, NT with ldb = K
  const bool vec_b = K % 8 == 0 && aligned(B, 16) && ldb == (layout == MDNN_NT ? K : N);
  // fewer than 2048 rows: four waves per row (each a quarter of the chunks)
  const bool share = M < 2048 && K >= 1024;
  int64_t blocks = share ? M : ceil_div(M, 4);
  if (blocks > 1024) blocks = 1024;
#define MDNN_ROWS(NK, WPR)                                                                                          \
  hipLaunchKernelGGL((skinny_rows_kernel<T, OutT, NK, WPR>), dim3((unsigned)blocks), dim3(256), lds, st, (const S*)A, \
                     lda, (const S*)B, ldb, M, (int)N, (int)K, kp, vec, vec_b, ep)
  if (layout == MDNN_NT) {
    if (share) MDNN_ROWS(true, 4); else MDNN_ROWS(true, 1);
  } else {
    if (share) MDNN_ROWS(false, 4); else MDNN_ROWS(false, 1);
  }
#undef MDNN_ROWS
  return check_launch("skinny_rows_kernel");
}

}  // namespace

// Measured against the MFMA kernels (with their workspace split): the depth
// kernel wins for K <= 4 (K = 10 is a tie; a K <= 16 instantiation took
// 12.5 us against 11.8 for 256 x 1024 x 10), the rows kernel for N <= 4 and,
// with B staged by 16-byte loads, for N <= 16 on few rows (256 x 10 x 1024:
// 13.2 us in one launch against 9.8 + 4.4 for the split MFMA product and its
// reduction), the cols kernel for N <= 16 when it can split K over a
// workspace or the grid is already wide.
bool skinny_applies(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K) {
  if (gemm_tile_override() != 0 || M <= 0 || N <= 0 || K <= 0) return false;
  if (K <= KMAX_DEPTH) return true;
  if (layout == MDNN_TN) return N <= NMAX;
  return N <= NMAX && K <= 0x7fffffff - 8 && (size_t)N * ceil_div(K, 8) * 8 * sizeof(float) <= ROWS_LDS &&
         (N <= 4 || M <= ROWS_WIDE_MAX_M);
}

size_t skinny_ws_bytes(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K) {
  if (!skinny_applies(layout, M, N, K) || K <= KMAX_DEPTH || layout != MDNN_TN) return 0;
  const SplitPlan p = cols_plan(M, K, cols_mb(N));
  return p.splits > 1 ? (size_t)p.splits * M * N * sizeof(float) : 0;
}

bool skinny_takes(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K, const void* ws, size_t ws_bytes) {
  if (!skinny_applies(layout, M, N, K)) return false;
  if (layout != MDNN_TN || K <= KMAX_DEPTH) return true;
  // the cols kernel alone runs ceil(M / (64 MB)) workgroups: without its K
  // split it only pays off on a wide grid
  const int mb = cols_mb(N);
  const SplitPlan p = cols_plan(M, K, mb);
  if (p.splits == 1) return true;
  return ws && aligned(ws, 16) && ws_bytes >= (size_t)p.splits * M * N * sizeof(float);
}

mdnn_status_t gemm_skinny(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                          const void* B, int64_t ldb, mdnn_dtype_t ab_type, mdnn_dtype_t d_type, const Epilogue& ep,
                          void* ws, size_t ws_bytes, hipStream_t st) {
  if (ab_type == MDNN_F32) return launch_skinny<F32, F32>(layout, A, lda, B, ldb, M, N, K, ep, ws, ws_bytes, st);
  if (ab_type == MDNN_F16) {
    if (d_type == MDNN_F32) return launch_skinny<F16, F32>(layout, A, lda, B, ldb, M, N, K, ep, ws, ws_bytes, st);
    return launch_skinny<F16, F16>(layout, A, lda, B, ldb, M, N, K, ep, ws, ws_bytes, st);
  }
  if (d_type == MDNN_F32) return launch_skinny<BF16, F32>(layout, A, lda, B, ldb, M, N, K, ep, ws, ws_bytes, st);
  return launch_skinny<BF16, BF16>(layout, A, lda, B, ldb, M, N, K, ep, ws, ws_bytes, st);
}

}  // namespace mdnn
