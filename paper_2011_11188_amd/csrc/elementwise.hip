// Memory-bound kernels of the SGD step: precision conversion, the stand-alone
// bias+activation epilogue, 2x2 max pooling, the two losses and the SGD /
// momentum update with dynamic loss scaling.  All reductions are taken in a
// fixed order, so results are bitwise reproducible.
#include "gemm_core.h"
#include "internal.h"

namespace mdnn {

static inline unsigned grid_for(int64_t work, int per_block) {
  int64_t b = ceil_div(work, per_block);
  if (b < 1) b = 1;
  if (b > 0x7fffffffLL) b = 0x7fffffffLL;
  return (unsigned)b;
}

// Grid of a grid-stride streaming kernel (256 threads, `work` items): one
// item per thread up to 2^20 blocks.  On MI355X the HBM-bound passes run
// ~9% faster with every item in flight than with 8192 blocks looping (54.5M
// fp32 SGD parameters: 244 -> 223 us; a 218 MB copy: 5.6 -> 6.1 TB/s).
static inline unsigned stream_grid(int64_t work) {
  const unsigned g = grid_for(work, 256);
  return g > (1u << 20) ? (1u << 20) : g;
}

// ---------------------------------------------------------------------------
// zero fill (used instead of memset nodes so callers can capture graphs)
// ---------------------------------------------------------------------------
__global__ void fill_zero_kernel(uint32_t* __restrict__ p, int64_t n_words) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_words;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = 0u;
}

mdnn_status_t fill_zero(void* p, size_t bytes, hipStream_t st) {
  if (bytes == 0) return MDNN_SUCCESS;
  if (bytes % 4 || !aligned(p, 4)) return fail(MDNN_ERR_MISALIGNED, "fill_zero: needs 4-byte units");
  int64_t words = (int64_t)(bytes / 4);
  const unsigned g = stream_grid(words);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(g), dim3(256), 0, st, (uint32_t*)p, words);
  return check_launch("fill_zero_kernel");
}

// ---------------------------------------------------------------------------
// cast
// ---------------------------------------------------------------------------
// Four consecutive elements in one vector access (p aligned to four elements).
template <class T>
__device__ __forceinline__ void load_quad(const typename T::storage* p, float (&v)[4]) {
  if constexpr (sizeof(typename T::storage) == 4) {
    const float4 q = *(const float4*)p;
    v[0] = q.x, v[1] = q.y, v[2] = q.z, v[3] = q.w;
  } else {
    const uint2 q = *(const uint2*)p;
    v[0] = to_f<T>((uint16_t)(q.x & 0xffffu)), v[1] = to_f<T>((uint16_t)(q.x >> 16));
    v[2] = to_f<T>((uint16_t)(q.y & 0xffffu)), v[3] = to_f<T>((uint16_t)(q.y >> 16));
  }
}
template <class T>
__device__ __forceinline__ void store_quad(typename T::storage* p, const float (&v)[4]) {
  if constexpr (sizeof(typename T::storage) == 4) {
    *(float4*)p = make_float4(v[0], v[1], v[2], v[3]);
  } else {
    uint2 q;
    q.x = (uint32_t)from_f<T>(v[0]) | ((uint32_t)from_f<T>(v[1]) << 16);
    q.y = (uint32_t)from_f<T>(v[2]) | ((uint32_t)from_f<T>(v[3]) << 16);
    *(uint2*)p = q;
  }
}

template <class Src, class Dst, bool VEC>
__global__ void cast_kernel(const typename Src::storage* __restrict__ src,
                            typename Dst::storage* __restrict__ dst, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  if (VEC) {  // 4 elements per thread in one vector load and store, n % 4 == 0, 4-element aligned
    for (int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4; i < n; i += stride * 4) {
      float v[4];
      load_quad<Src>(src + i, v);
      store_quad<Dst>(dst + i, v);
    }
  } else {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
      dst[i] = from_f<Dst>(to_f<Src>(src[i]));
  }
}

// fp32 -> 16-bit cast that also sets *nonfinite when a stored value is Inf
// or NaN (an all-ones exponent: finite inputs beyond the type's range count)
template <class Dst, bool VEC>
__global__ void cast_checked_kernel(const float* __restrict__ src, typename Dst::storage* __restrict__ dst, int64_t n,
                                    int32_t* __restrict__ nonfinite) {
  constexpr uint16_t EXP = Dst::id == MDNN_F16 ? 0x7c00u : 0x7f80u;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  bool bad = false;
  if (VEC) {
    for (int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4; i < n; i += stride * 4) {
      float v[4];
      load_quad<F32>(src + i, v);
      store_quad<Dst>(dst + i, v);
#pragma unroll
      for (int e = 0; e < 4; ++e) bad |= (from_f<Dst>(v[e]) & EXP) == EXP;
    }
  } else {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
      const uint16_t h = from_f<Dst>(src[i]);
      dst[i] = h;
      bad |= (h & EXP) == EXP;
    }
  }
  if (bad) atomicOr(nonfinite, 1);
}

mdnn_status_t cast_f32_checked(int64_t n, const float* src, void* dst, mdnn_dtype_t d, int32_t* nonfinite,
                               hipStream_t st) {
  if (n == 0) return MDNN_SUCCESS;
  if (d != MDNN_F16 && d != MDNN_BF16) return fail(MDNN_ERR_DTYPE, "cast: the checked cast writes 16-bit values");
  const bool vec = n % 4 == 0 && aligned(src, 16) && aligned(dst, 8);
  const unsigned g = stream_grid(ceil_div(n, vec ? 4 : 1));
  if (d == MDNN_F16) {
    if (vec)
      hipLaunchKernelGGL((cast_checked_kernel<F16, true>), dim3(g), dim3(256), 0, st, src, (uint16_t*)dst, n, nonfinite);
    else
      hipLaunchKernelGGL((cast_checked_kernel<F16, false>), dim3(g), dim3(256), 0, st, src, (uint16_t*)dst, n,
                         nonfinite);
  } else {
    if (vec)
      hipLaunchKernelGGL((cast_checked_kernel<BF16, true>), dim3(g), dim3(256), 0, st, src, (uint16_t*)dst, n,
                         nonfinite);
    else
      hipLaunchKernelGGL((cast_checked_kernel<BF16, false>), dim3(g), dim3(256), 0, st, src, (uint16_t*)dst, n,
                         nonfinite);
  }
  return check_launch("cast_checked_kernel");
}

template <class Src, class Dst>
static void cast_launch(const void* src, void* dst, int64_t n, bool vec, hipStream_t st) {
  const unsigned g = stream_grid(ceil_div(n, vec ? 4 : 1));
  if (vec)
    hipLaunchKernelGGL((cast_kernel<Src, Dst, true>), dim3(g), dim3(256), 0, st,
                       (const typename Src::storage*)src, (typename Dst::storage*)dst, n);
  else
    hipLaunchKernelGGL((cast_kernel<Src, Dst, false>), dim3(g), dim3(256), 0, st,
                       (const typename Src::storage*)src, (typename Dst::storage*)dst, n);
}

mdnn_status_t cast_any(int64_t n, const void* src, mdnn_dtype_t s, void* dst, mdnn_dtype_t d,
                       hipStream_t st) {
  if (n == 0) return MDNN_SUCCESS;
  const bool vec = n % 4 == 0 && aligned(src, 4 * dtype_size(s)) && aligned(dst, 4 * dtype_size(d));
#define MDNN_CAST_CASE(S_, D_, SI, DI) \
  if (s == SI && d == DI) { cast_launch<S_, D_>(src, dst, n, vec, st); return check_launch("cast_kernel"); }
  MDNN_CAST_CASE(F32, F16, MDNN_F32, MDNN_F16)
  MDNN_CAST_CASE(F32, BF16, MDNN_F32, MDNN_BF16)
  MDNN_CAST_CASE(F16, F32, MDNN_F16, MDNN_F32)
  MDNN_CAST_CASE(BF16, F32, MDNN_BF16, MDNN_F32)
  MDNN_CAST_CASE(F32, F32, MDNN_F32, MDNN_F32)
  MDNN_CAST_CASE(F16, F16, MDNN_F16, MDNN_F16)
  MDNN_CAST_CASE(BF16, BF16, MDNN_BF16, MDNN_BF16)
  MDNN_CAST_CASE(F16, BF16, MDNN_F16, MDNN_BF16)
  MDNN_CAST_CASE(BF16, F16, MDNN_BF16, MDNN_F16)
#undef MDNN_CAST_CASE
  return fail(MDNN_ERR_DTYPE, "cast: unsupported pair");
}

// ---------------------------------------------------------------------------
// bias + activation
// ---------------------------------------------------------------------------
template <class OutT>
__global__ void bias_act_fwd_kernel(const float* __restrict__ x, const float* __restrict__ bias,
                                    int act, typename OutT::storage* __restrict__ y, int64_t rows,
                                    int64_t cols) {
  const int64_t n = rows * cols;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    float v = x[i];
    if (bias) v += bias[i % cols];
    if (act == MDNN_ACT_RELU) v = relu_f(v);
    y[i] = from_f<OutT>(v);
  }
}

template <class T>
__global__ void relu_mask_kernel(const typename T::storage* __restrict__ dy,
                                 const typename T::storage* __restrict__ y,
                                 typename T::storage* __restrict__ dz, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    typename T::storage v = dy[i];
    dz[i] = (y == nullptr || to_f<T>(y[i]) > 0.0f) ? v : (typename T::storage)0;
  }
}

// ---------------------------------------------------------------------------
// 2x2 / stride 2 max pooling, NHWC
// ---------------------------------------------------------------------------
template <class T>
__global__ void maxpool2_fwd_kernel(const typename T::storage* __restrict__ x,
                                    typename T::storage* __restrict__ y,
                                    uint8_t* __restrict__ arg, int64_t n, int32_t h, int32_t w,
                                    int32_t c) {
  const int32_t ho = h / 2, wo = w / 2;
  const int64_t total = n * ho * wo * c;
  for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total;
       o += (int64_t)gridDim.x * blockDim.x) {
    const int32_t ch = (int32_t)(o % c);
    int64_t t = o / c;
    const int32_t j = (int32_t)(t % wo);
    t /= wo;
    const int32_t i = (int32_t)(t % ho);
    const int64_t b = t / ho;
    const typename T::storage* p = x + ((b * h + 2 * i) * w + 2 * j) * c + ch;
    typename T::storage cand[4] = {p[0], p[c], p[(int64_t)w * c], p[(int64_t)w * c + c]};
    typename T::storage best = cand[0];
    float bv = to_f<T>(best);
    int bi = 0;
#pragma unroll
    for (int k = 1; k < 4; ++k) {
      float v = to_f<T>(cand[k]);
      if (v > bv) { bv = v; best = cand[k]; bi = k; }
    }
    y[o] = best;
    if (arg) arg[o] = (uint8_t)bi;
  }
}

template <class T>
__global__ void maxpool2_bwd_kernel(const typename T::storage* __restrict__ dy,
                                    const uint8_t* __restrict__ arg,
                                    typename T::storage* __restrict__ dx, int64_t n, int32_t h,
                                    int32_t w, int32_t c) {
  const int32_t ho = h / 2, wo = w / 2;
  const int64_t total = n * h * w * c;
  for (int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int32_t ch = (int32_t)(e % c);
    int64_t t = e / c;
    const int32_t xw = (int32_t)(t % w);
    t /= w;
    const int32_t xh = (int32_t)(t % h);
    const int64_t b = t / h;
    const int32_t i = xh >> 1, j = xw >> 1;
    typename T::storage v = 0;
    if (i < ho && j < wo) {
      const int64_t o = ((b * ho + i) * wo + j) * c + ch;
      if (arg[o] == (uint8_t)(((xh & 1) << 1) | (xw & 1))) v = dy[o];
    }
    dx[e] = v;
  }
}

// 16-bit storage, even h and w, c % 8 == 0: a thread owns eight channels of
// one pooled position (16-byte loads and stores), 32-bit index arithmetic
// (the caller checks the sizes).  Same window order and tie rule as above.
__global__ void maxpool2_fwd_vec_kernel(const uint16_t* __restrict__ x, uint16_t* __restrict__ y,
                                        uint8_t* __restrict__ arg, int32_t units, int32_t wo, int32_t c8,
                                        int32_t c, bool bf16) {
  const int32_t u = (int32_t)(blockIdx.x * blockDim.x + threadIdx.x);
  if (u >= units) return;
  const int32_t cg = u % c8, t = u / c8;
  const int32_t j = t % wo, r = t / wo;  // r = b * ho + i: input rows 2r, 2r + 1
  const int64_t wc = (int64_t)2 * wo * c;
  const uint16_t* p = x + (int64_t)2 * r * wc + (int64_t)2 * j * c + cg * 8;
  uint4 cand[4] = {*(const uint4*)p, *(const uint4*)(p + c), *(const uint4*)(p + wc), *(const uint4*)(p + wc + c)};
  const uint16_t* cv[4] = {(const uint16_t*)&cand[0], (const uint16_t*)&cand[1], (const uint16_t*)&cand[2],
                           (const uint16_t*)&cand[3]};
  uint16_t out[8];
  uint8_t am[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    uint16_t best = cv[0][e];
    float bv = bf16 ? bf16_to_f32(best) : f16_to_f32(best);
    int bi = 0;
#pragma unroll
    for (int k = 1; k < 4; ++k) {
      const float v = bf16 ? bf16_to_f32(cv[k][e]) : f16_to_f32(cv[k][e]);
      if (v > bv) { bv = v; best = cv[k][e]; bi = k; }
    }
    out[e] = best;
    am[e] = (uint8_t)bi;
  }
  const int64_t o = ((int64_t)r * wo + j) * c + cg * 8;
  *(uint4*)(y + o) = *(const uint4*)out;
  if (arg) *(uint2*)(arg + o) = *(const uint2*)am;
}

__global__ void maxpool2_bwd_vec_kernel(const uint16_t* __restrict__ dy, const uint8_t* __restrict__ arg,
                                        uint16_t* __restrict__ dx, int32_t units, int32_t wo, int32_t c8,
                                        int32_t c) {
  const int32_t u = (int32_t)(blockIdx.x * blockDim.x + threadIdx.x);
  if (u >= units) return;
  const int32_t cg = u % c8, t = u / c8;
  const int32_t j = t % wo, r = t / wo;
  const int64_t o = ((int64_t)r * wo + j) * c + cg * 8;
  const uint4 g = *(const uint4*)(dy + o);
  const uint2 a = *(const uint2*)(arg + o);
  const uint16_t* gv = (const uint16_t*)&g;
  const uint8_t* av = (const uint8_t*)&a;
  const int64_t wc = (int64_t)2 * wo * c;
  uint16_t* q = dx + (int64_t)2 * r * wc + (int64_t)2 * j * c + cg * 8;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = av[e] == k ? gv[e] : (uint16_t)0;
    *(uint4*)(q + (k >> 1) * wc + (k & 1) * c) = *(const uint4*)v;
  }
}

static bool pool_vec_ok(int64_t n, int64_t h, int64_t w, int64_t c, mdnn_dtype_t t) {
  return t != MDNN_F32 && h % 2 == 0 && w % 2 == 0 && c % 8 == 0 && n * h * w * c < ((int64_t)1 << 31);
}

// ---------------------------------------------------------------------------
// losses: one block; waves own rows in a fixed order, block sum in a fixed order
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

constexpr int LOSS_THREADS = 1024;

template <class OutT>
__global__ void __launch_bounds__(LOSS_THREADS)
softmax_xent_kernel(int64_t B, int64_t C, const float* __restrict__ z, int64_t ldl,
                    const int32_t* __restrict__ labels, const float* __restrict__ scale_p,
                    float* __restrict__ loss_out, typename OutT::storage* __restrict__ dz,
                    int64_t ldd) {
  __shared__ float wsum[LOSS_THREADS / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nw = LOSS_THREADS / 64;
  const float S = scale_p ? *scale_p : 1.0f;
  const float inv_b = 1.0f / (float)B;
  float acc = 0.0f;  // lane 0: this wave's rows, in order
  for (int64_t r = wave; r < B; r += nw) {
    const float* zr = z + r * ldl;
    float m = -INFINITY;
    for (int64_t j = lane; j < C; j += 64) m = fmaxf(m, zr[j]);
    m = wave_max(m);
    float se = 0.0f;
    for (int64_t j = lane; j < C; j += 64) se += expf(zr[j] - m);
    se = wave_sum(se);
    const float lse = m + logf(se);
    const int32_t lab = labels[r];
    const bool ok = lab >= 0 && lab < C;
    for (int64_t j = lane; j < C; j += 64) {
      const float p = expf(zr[j] - lse);
      float g = S * (p - (j == lab ? 1.0f : 0.0f)) * inv_b;
      if (!ok) g = NAN;
      dz[r * ldd + j] = from_f<OutT>(g);
    }
    if (lane == 0) acc += ok ? (lse - zr[lab]) : NAN;
  }
  if (lane == 0) wsum[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.0f;
    for (int k = 0; k < nw; ++k) t += wsum[k];
    *loss_out = t * inv_b;
  }
}

// Few classes (C <= 32): one thread per row, so all rows run at once (a
// wave per row would leave most lanes idle and walk the rows 16 at a time).
// Thread t sums the losses of rows t, t + 1024, ... in order; the block then
// adds the 1024 partial sums in a fixed tree order.
constexpr int SMALL_C = 32;
constexpr size_t XENT_DB_LDS = 48 * 1024;  // the stored dz rows kept for the bias gradient

// db (nullable, B <= LOSS_THREADS): also the column sums of the stored dz
// (the classifier's bias gradient), kept as float in dynamic LDS [B][C], in
// row order within 32 row segments and then segment order; nonfinite
// (nullable) is set when one of them is Inf or NaN.
template <class OutT>
__global__ void __launch_bounds__(LOSS_THREADS)
softmax_xent_rows_kernel(int64_t B, int64_t C, const float* __restrict__ z, int64_t ldl,
                         const int32_t* __restrict__ labels, const float* __restrict__ scale_p,
                         float* __restrict__ loss_out, typename OutT::storage* __restrict__ dz, int64_t ldd,
                         float* __restrict__ db, int32_t* __restrict__ nonfinite) {
  __shared__ float red[LOSS_THREADS];
  __shared__ float seg_sum[SMALL_C][33];
  extern __shared__ float dzs[];
  const float S = scale_p ? *scale_p : 1.0f;
  const float inv_b = 1.0f / (float)B;
  float acc = 0.0f;
  for (int64_t r = threadIdx.x; r < B; r += LOSS_THREADS) {
    const float* zr = z + r * ldl;
    float v[SMALL_C];
    float m = -INFINITY;
#pragma unroll
    for (int j = 0; j < SMALL_C; ++j) {
      v[j] = j < C ? zr[j] : -INFINITY;
      m = fmaxf(m, v[j]);
    }
    float se = 0.0f;
#pragma unroll
    for (int j = 0; j < SMALL_C; ++j)
      if (j < C) se += expf(v[j] - m);
    const float lse = m + logf(se);
    const int32_t lab = labels[r];
    const bool ok = lab >= 0 && lab < C;
#pragma unroll
    for (int j = 0; j < SMALL_C; ++j) {
      if (j < C) {
        float g = S * (expf(v[j] - lse) - (j == lab ? 1.0f : 0.0f)) * inv_b;
        if (!ok) g = NAN;
        const typename OutT::storage q = from_f<OutT>(g);
        dz[r * ldd + j] = q;
        if (db) dzs[r * C + j] = to_f<OutT>(q);
      }
    }
    acc += ok ? (lse - zr[lab]) : NAN;
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = LOSS_THREADS / 2; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) *loss_out = red[0] * inv_b;
  if (!db) return;
  // column j, segment t of ceil(B / 32) rows: thread 32 j + t
  const int j = threadIdx.x >> 5, t = threadIdx.x & 31;
  const int64_t seg = (B + 31) / 32;
  if (j < C) {
    float cs = 0.0f;
    const int64_t r1 = (t + 1) * seg < B ? (t + 1) * seg : B;
    // eight reads in flight, added in row order
    for (int64_t r = t * seg; r < r1; r += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = dzs[(r + u < r1 ? r + u : r) * C + j];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (r + u < r1) cs += v[u];
    }
    seg_sum[j][t] = cs;
  }
  __syncthreads();
  if ((int)threadIdx.x < C) {
    float v[32];
#pragma unroll
    for (int u = 0; u < 32; ++u) v[u] = seg_sum[threadIdx.x][u];
    float tot = 0.0f;
#pragma unroll
    for (int u = 0; u < 32; ++u) tot += v[u];
    db[threadIdx.x] = tot;
    if (nonfinite && !isfinite(tot)) atomicOr(nonfinite, 1);
  }
}

template <class OutT>
__global__ void __launch_bounds__(LOSS_THREADS)
mse_kernel(int64_t n, int64_t B, const float* __restrict__ y, const float* __restrict__ t,
           const float* __restrict__ scale_p, float* __restrict__ loss_out,
           typename OutT::storage* __restrict__ dy) {
  __shared__ float red[LOSS_THREADS];
  const float S = scale_p ? *scale_p : 1.0f;
  const float c = 2.0f * S / (float)B;
  float acc = 0.0f;
  for (int64_t i = threadIdx.x; i < n; i += LOSS_THREADS) {
    const float d = y[i] - t[i];
    acc = fmaf(d, d, acc);
    dy[i] = from_f<OutT>(c * d);
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int s = LOSS_THREADS / 2; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) *loss_out = red[0] / (float)B;
}

// ---------------------------------------------------------------------------
// SGD / momentum with dynamic loss scaling
//   check:    scaler->reserved |= any(!isfinite(g))          (reserved starts at 0)
//   update:   skipped when reserved != 0
//   finalize: scale / good_steps / overflow state machine; reserved = 0
// ---------------------------------------------------------------------------
__global__ void finite_check_kernel(const float* __restrict__ g, int64_t n,
                                    mdnn_scaler_t* __restrict__ sc) {
  int bad = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t n4 = n / 4;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    float4 v = ((const float4*)g)[i];
    bad |= (int)!isfinite(v.x) | (int)!isfinite(v.y) | (int)!isfinite(v.z) | (int)!isfinite(v.w);
  }
  for (int64_t i = n4 * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    bad |= !isfinite(g[i]);
  bad = __syncthreads_or(bad);
  if (bad && threadIdx.x == 0) atomicOr(&sc->reserved, 1);
}

// finite_check_kernel over a few ranges of g: block row y covers range y
__global__ void finite_check_ranges_kernel(const float* __restrict__ g, CheckRanges r,
                                           mdnn_scaler_t* __restrict__ sc) {
  const float* p = g + r.off[blockIdx.y];
  const int64_t n = r.len[blockIdx.y];
  int bad = 0;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) bad |= !isfinite(p[i]);
  bad = __syncthreads_or(bad);
  if (bad && threadIdx.x == 0) atomicOr(&sc->reserved, 1);
}

// sgd_kernel over a few ranges of the flat parameter vector: block row y
// covers range y (the same arithmetic per element)
template <class LpT, bool MOM, bool SCALE>
__global__ void sgd_ranges_kernel(CheckRanges r, float* __restrict__ w, const float* __restrict__ g,
                                  float* __restrict__ v, typename LpT::storage* __restrict__ wlp, float lr,
                                  float mu, const mdnn_scaler_t* __restrict__ sc, bool vec) {
  float S = 1.0f;
  if (SCALE) {
    if (sc->reserved) return;  // overflow: skip the whole update
    S = sc->scale;
  }
  const int64_t off = r.off[blockIdx.y], n = r.len[blockIdx.y];
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  int64_t done = 0;
  if (vec && off % 4 == 0) {
    // four elements per thread with 16-byte accesses (the buffers are
    // 16-byte aligned at element 0), the same arithmetic per element
    typedef float f4v __attribute__((ext_vector_type(4)));
    typedef uint32_t u2v __attribute__((ext_vector_type(2)));
    const int64_t n4 = n / 4;
    for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n4; q += stride) {
      const int64_t k = off + 4 * q;
      const f4v gi = __builtin_nontemporal_load((const f4v*)(g + k));
      const f4v wi = __builtin_nontemporal_load((const f4v*)(w + k));
      float ga[4] = {gi[0], gi[1], gi[2], gi[3]}, wa[4] = {wi[0], wi[1], wi[2], wi[3]};
      if (SCALE) {
#pragma unroll
        for (int e = 0; e < 4; ++e) ga[e] = ga[e] / S;
      }
      if (MOM) {
        const f4v vi = __builtin_nontemporal_load((const f4v*)(v + k));
        float va[4] = {vi[0], vi[1], vi[2], vi[3]};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          va[e] = fmaf(mu, va[e], ga[e]);
          wa[e] = fmaf(-lr, va[e], wa[e]);
        }
        __builtin_nontemporal_store((f4v){va[0], va[1], va[2], va[3]}, (f4v*)(v + k));
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) wa[e] = fmaf(-lr, ga[e], wa[e]);
      }
      __builtin_nontemporal_store((f4v){wa[0], wa[1], wa[2], wa[3]}, (f4v*)(w + k));
      if (wlp) {
        if constexpr (sizeof(typename LpT::storage) == 4) {
          __builtin_nontemporal_store((f4v){wa[0], wa[1], wa[2], wa[3]}, (f4v*)(wlp + k));
        } else {
          u2v u;
          u[0] = (uint32_t)from_f<LpT>(wa[0]) | ((uint32_t)from_f<LpT>(wa[1]) << 16);
          u[1] = (uint32_t)from_f<LpT>(wa[2]) | ((uint32_t)from_f<LpT>(wa[3]) << 16);
          __builtin_nontemporal_store(u, (u2v*)(wlp + k));
        }
      }
    }
    done = n4 * 4;
  }
  for (int64_t i = done + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    const int64_t k = off + i;
    float gi = g[k];
    if (SCALE) gi = gi / S;
    float wi = w[k];
    if (MOM) {
      const float vi = fmaf(mu, v[k], gi);
      v[k] = vi;
      wi = fmaf(-lr, vi, wi);
    } else {
      wi = fmaf(-lr, gi, wi);
    }
    w[k] = wi;
    if (wlp) wlp[k] = from_f<LpT>(wi);
  }
}

template <class LpT, bool MOM, bool SCALE>
__global__ void sgd_kernel(int64_t n, float* __restrict__ w, const float* __restrict__ g,
                           float* __restrict__ v, typename LpT::storage* __restrict__ wlp, float lr,
                           float mu, const mdnn_scaler_t* __restrict__ sc) {
  float S = 1.0f;
  if (SCALE) {
    if (sc->reserved) return;  // overflow: skip the whole update
    S = sc->scale;
  }
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    float gi = g[i];
    if (SCALE) gi = gi / S;
    float wi = w[i];
    if (MOM) {
      const float vi = fmaf(mu, v[i], gi);
      v[i] = vi;
      wi = fmaf(-lr, vi, wi);
    } else {
      wi = fmaf(-lr, gi, wi);
    }
    w[i] = wi;
    if (wlp) wlp[i] = from_f<LpT>(wi);
  }
}

// Asynchronous variant (section 3.1): the step -lr*v (or -lr*g) is added to
// the shared weights with hardware fp32 atomics, so concurrent updates from
// other streams are never lost; reads of w by other work may see any mix of
// old and new values (Hogwild!-style inconsistent reads).
template <bool MOM, bool SCALE>
__global__ void sgd_async_kernel(int64_t n, float* w, const float* __restrict__ g, float* __restrict__ v,
                                 float lr, float mu, const mdnn_scaler_t* __restrict__ sc) {
  float S = 1.0f;
  if (SCALE) {
    if (sc->reserved) return;  // overflow: this worker's update is skipped
    S = sc->scale;
  }
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
    float gi = g[i];
    if (SCALE) gi = gi / S;
    if (MOM) {
      const float vi = fmaf(mu, v[i], gi);
      v[i] = vi;
      gi = vi;
    }
    unsafeAtomicAdd(&w[i], -lr * gi);
  }
}

__global__ void scaler_finalize_kernel(mdnn_scaler_t* sc) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  if (sc->reserved) {
    float s = sc->scale * sc->backoff;
    sc->scale = s < sc->min_scale ? sc->min_scale : s;
    sc->good_steps = 0;
    sc->overflow = 1;
  } else {
    sc->overflow = 0;
    sc->good_steps += 1;
    if (sc->good_steps >= sc->growth_interval) {
      sc->scale = sc->scale * sc->growth;
      sc->good_steps = 0;
    }
  }
  sc->reserved = 0;
}

// Four consecutive parameters per thread with 16-byte loads and stores (w,
// g, v 16-byte aligned; the working copy 4-element aligned); the same
// arithmetic per element as sgd_kernel.  The n % 4 tail is done by thread 0.
template <class LpT, bool MOM, bool SCALE>
__global__ void sgd_vec_kernel(int64_t n, float* __restrict__ w, const float* __restrict__ g,
                               float* __restrict__ v, typename LpT::storage* __restrict__ wlp, float lr,
                               float mu, const mdnn_scaler_t* __restrict__ sc) {
  float S = 1.0f;
  if (SCALE) {
    if (sc->reserved) return;  // overflow: skip the whole update
    S = sc->scale;
  }
  const int64_t n4 = n / 4;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  // every element is read and written once per step: non-temporal loads and
  // stores (a 54.5M-parameter update streamed from HBM: 224.8 -> 205.4 us in
  // isolation, the caches left to the products)
  typedef float f4v __attribute__((ext_vector_type(4)));
  typedef uint32_t u2v __attribute__((ext_vector_type(2)));
  for (int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; q < n4; q += stride) {
    const f4v gi = __builtin_nontemporal_load((const f4v*)g + q);
    const f4v wi = __builtin_nontemporal_load((const f4v*)w + q);
    float ga[4] = {gi[0], gi[1], gi[2], gi[3]}, wa[4] = {wi[0], wi[1], wi[2], wi[3]};
    if (SCALE) {
#pragma unroll
      for (int e = 0; e < 4; ++e) ga[e] = ga[e] / S;
    }
    if (MOM) {
      const f4v vi = __builtin_nontemporal_load((const f4v*)v + q);
      float va[4] = {vi[0], vi[1], vi[2], vi[3]};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        va[e] = fmaf(mu, va[e], ga[e]);
        wa[e] = fmaf(-lr, va[e], wa[e]);
      }
      __builtin_nontemporal_store((f4v){va[0], va[1], va[2], va[3]}, (f4v*)v + q);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) wa[e] = fmaf(-lr, ga[e], wa[e]);
    }
    __builtin_nontemporal_store((f4v){wa[0], wa[1], wa[2], wa[3]}, (f4v*)w + q);
    if (wlp) {
      if constexpr (sizeof(typename LpT::storage) == 4) {
        __builtin_nontemporal_store((f4v){wa[0], wa[1], wa[2], wa[3]}, (f4v*)wlp + q);
      } else {
        u2v u;
        u[0] = (uint32_t)from_f<LpT>(wa[0]) | ((uint32_t)from_f<LpT>(wa[1]) << 16);
        u[1] = (uint32_t)from_f<LpT>(wa[2]) | ((uint32_t)from_f<LpT>(wa[3]) << 16);
        __builtin_nontemporal_store(u, (u2v*)wlp + q);
      }
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    for (int64_t i = n4 * 4; i < n; ++i) {
      float gi = g[i];
      if (SCALE) gi = gi / S;
      float wi = w[i];
      if (MOM) {
        const float vi = fmaf(mu, v[i], gi);
        v[i] = vi;
        wi = fmaf(-lr, vi, wi);
      } else {
        wi = fmaf(-lr, gi, wi);
      }
      w[i] = wi;
      if (wlp) wlp[i] = from_f<LpT>(wi);
    }
  }
}

// scaler->reserved |= any non-finite g[0..n): 16-byte vectors when g allows,
// else the element-wise ranged pass over one range
static mdnn_status_t finite_check_all(const float* g32, int64_t n, mdnn_scaler_t* scaler, hipStream_t st) {
  if (aligned(g32, 16)) {
    const unsigned g = stream_grid(ceil_div(n, 4));
    hipLaunchKernelGGL(finite_check_kernel, dim3(g), dim3(256), 0, st, g32, n, scaler);
    return check_launch("finite_check_kernel");
  }
  CheckRanges r{};
  r.n = 1;
  r.off[0] = 0;
  r.len[0] = n;
  return finite_check_ranges(g32, r, scaler, st);
}

template <class LpT, bool MOM, bool SCALE>
static void sgd_launch_t(int64_t n, float* w, const float* g, float* v, void* wlp, float lr, float mu,
                         const mdnn_scaler_t* sc, hipStream_t st) {
  typedef typename LpT::storage L;
  // 16-byte vectors when every buffer allows them, else one element per thread
  const bool vec = aligned(w, 16) && aligned(g, 16) && (!v || aligned(v, 16)) && (!wlp || aligned(wlp, 4 * sizeof(L)));
  const unsigned grid = stream_grid(vec ? ceil_div(n, 4) : n);
  if (vec)
    hipLaunchKernelGGL((sgd_vec_kernel<LpT, MOM, SCALE>), dim3(grid), dim3(256), 0, st, n, w, g, v, (L*)wlp, lr, mu,
                       sc);
  else
    hipLaunchKernelGGL((sgd_kernel<LpT, MOM, SCALE>), dim3(grid), dim3(256), 0, st, n, w, g, v, (L*)wlp, lr, mu, sc);
}

template <class LpT>
static void sgd_launch(int64_t n, float* w, const float* g, float* v, void* wlp, float lr, float mu,
                       const mdnn_scaler_t* sc, hipStream_t st) {
  if (v && sc) sgd_launch_t<LpT, true, true>(n, w, g, v, wlp, lr, mu, sc, st);
  else if (v) sgd_launch_t<LpT, true, false>(n, w, g, v, wlp, lr, mu, sc, st);
  else if (sc) sgd_launch_t<LpT, false, true>(n, w, g, v, wlp, lr, mu, sc, st);
  else sgd_launch_t<LpT, false, false>(n, w, g, v, wlp, lr, mu, sc, st);
}

}  // namespace mdnn

using namespace mdnn;

extern "C" mdnn_status_t mdnn_cast(int64_t n, const void* src, mdnn_dtype_t src_type, void* dst,
                                   mdnn_dtype_t dst_type, mdnn_stream_t stream) {
  if (n < 0) return fail(MDNN_ERR_SHAPE, "cast: n < 0");
  if (!dtype_ok(src_type) || !dtype_ok(dst_type)) return fail(MDNN_ERR_DTYPE, "cast: unknown dtype");
  if (n == 0) return MDNN_SUCCESS;
  if (!src || !dst) return fail(MDNN_ERR_NULL, "cast: NULL buffer");
  if (!aligned(src, dtype_size(src_type)) || !aligned(dst, dtype_size(dst_type)))
    return fail(MDNN_ERR_MISALIGNED, "cast: misaligned buffer");
  clear_error();
  return cast_any(n, src, src_type, dst, dst_type, as_stream(stream));
}

extern "C" mdnn_status_t mdnn_bias_act_fwd(int64_t rows, int64_t cols, const float* x,
                                           const float* bias, mdnn_act_t act, void* y,
                                           mdnn_dtype_t y_type, mdnn_stream_t stream) {
  if (rows < 0 || cols < 0) return fail(MDNN_ERR_SHAPE, "bias_act_fwd: negative size");
  if (!dtype_ok(y_type)) return fail(MDNN_ERR_DTYPE, "bias_act_fwd: unknown dtype");
  if (act != MDNN_ACT_NONE && act != MDNN_ACT_RELU) return fail(MDNN_ERR_DTYPE, "bias_act_fwd: unknown act");
  if (rows == 0 || cols == 0) return MDNN_SUCCESS;
  if (!x || !y) return fail(MDNN_ERR_NULL, "bias_act_fwd: NULL buffer");
  if (!aligned(x, 4) || !aligned(y, dtype_size(y_type)) || (bias && !aligned(bias, 4)))
    return fail(MDNN_ERR_MISALIGNED, "bias_act_fwd: misaligned buffer");
  clear_error();
  hipStream_t st = as_stream(stream);
  const unsigned g = stream_grid(rows * cols);
  switch (y_type) {
    case MDNN_F32: hipLaunchKernelGGL(bias_act_fwd_kernel<F32>, dim3(g), dim3(256), 0, st, x, bias, (int)act, (float*)y, rows, cols); break;
    case MDNN_F16: hipLaunchKernelGGL(bias_act_fwd_kernel<F16>, dim3(g), dim3(256), 0, st, x, bias, (int)act, (uint16_t*)y, rows, cols); break;
    default: hipLaunchKernelGGL(bias_act_fwd_kernel<BF16>, dim3(g), dim3(256), 0, st, x, bias, (int)act, (uint16_t*)y, rows, cols); break;
  }
  return check_launch("bias_act_fwd_kernel");
}

template <class T>
static mdnn_status_t bias_act_bwd_t(int64_t rows, int64_t cols, const void* dy, const void* y,
                                    void* dz, float* db, void* ws, size_t ws_bytes, hipStream_t st) {
  typedef typename T::storage S;
  if (db) MDNN_TRY(column_sums(dy, y, T::id, rows, cols, db, ws, ws_bytes, st));
  if (dz) {
    const unsigned g = stream_grid(rows * cols);
    hipLaunchKernelGGL(relu_mask_kernel<T>, dim3(g), dim3(256), 0, st, (const S*)dy, (const S*)y, (S*)dz,
                       rows * cols);
    MDNN_TRY(check_launch("relu_mask_kernel"));
  }
  return MDNN_SUCCESS;
}

extern "C" size_t mdnn_bias_act_bwd_workspace(int64_t rows, int64_t cols) {
  if (rows < 0 || cols < 0) return 0;
  return column_sums_ws_bytes(rows, cols);
}

extern "C" mdnn_status_t mdnn_bias_act_bwd(int64_t rows, int64_t cols, const void* dy,
                                           const void* y, mdnn_act_t act, void* dz, float* db,
                                           mdnn_dtype_t dtype, void* workspace, size_t ws_bytes,
                                           mdnn_stream_t stream) {
  if (rows < 0 || cols < 0) return fail(MDNN_ERR_SHAPE, "bias_act_bwd: negative size");
  if (!dtype_ok(dtype)) return fail(MDNN_ERR_DTYPE, "bias_act_bwd: unknown dtype");
  if (act != MDNN_ACT_NONE && act != MDNN_ACT_RELU) return fail(MDNN_ERR_DTYPE, "bias_act_bwd: unknown act");
  if (cols == 0) return MDNN_SUCCESS;
  if (db && rows == 0) {
    clear_error();
    return fill_zero(db, (size_t)cols * 4, as_stream(stream));
  }
  if (rows == 0) return MDNN_SUCCESS;
  if (!dy) return fail(MDNN_ERR_NULL, "bias_act_bwd: dy is NULL");
  if (act == MDNN_ACT_RELU && !y) return fail(MDNN_ERR_NULL, "bias_act_bwd: ReLU needs y");
  const size_t es = dtype_size(dtype);
  if (!aligned(dy, es) || (y && !aligned(y, es)) || (dz && !aligned(dz, es)) || (db && !aligned(db, 4)) ||
      (workspace && !aligned(workspace, 16)))
    return fail(MDNN_ERR_MISALIGNED, "bias_act_bwd: misaligned buffer");
  const void* ym = act == MDNN_ACT_RELU ? y : nullptr;
  if (dz == dy && act == MDNN_ACT_NONE) dz = nullptr;  // nothing to write
  clear_error();
  hipStream_t st = as_stream(stream);
  switch (dtype) {
    case MDNN_F32: return bias_act_bwd_t<F32>(rows, cols, dy, ym, dz, db, workspace, ws_bytes, st);
    case MDNN_F16: return bias_act_bwd_t<F16>(rows, cols, dy, ym, dz, db, workspace, ws_bytes, st);
    default: return bias_act_bwd_t<BF16>(rows, cols, dy, ym, dz, db, workspace, ws_bytes, st);
  }
}

extern "C" mdnn_status_t mdnn_maxpool2_fwd(int64_t n, int64_t h, int64_t w, int64_t c,
                                           const void* x, void* y, uint8_t* argmax,
                                           mdnn_dtype_t dtype, mdnn_stream_t stream) {
  if (n < 0 || h < 0 || w < 0 || c < 0 || h > 0x7fffffff || w > 0x7fffffff || c > 0x7fffffff)
    return fail(MDNN_ERR_SHAPE, "maxpool2_fwd: bad size");
  if (!dtype_ok(dtype)) return fail(MDNN_ERR_DTYPE, "maxpool2_fwd: unknown dtype");
  const int64_t total = n * (h / 2) * (w / 2) * c;
  if (total == 0) return MDNN_SUCCESS;
  if (!x || !y) return fail(MDNN_ERR_NULL, "maxpool2_fwd: NULL buffer");
  const size_t es = dtype_size(dtype);
  if (!aligned(x, es) || !aligned(y, es)) return fail(MDNN_ERR_MISALIGNED, "maxpool2_fwd: misaligned");
  clear_error();
  hipStream_t st = as_stream(stream);
  if (pool_vec_ok(n, h, w, c, dtype) && aligned(x, 16) && aligned(y, 16) && (!argmax || aligned(argmax, 8))) {
    const int64_t units = total / 8;
    hipLaunchKernelGGL(maxpool2_fwd_vec_kernel, dim3((unsigned)ceil_div(units, 256)), dim3(256), 0, st,
                       (const uint16_t*)x, (uint16_t*)y, argmax, (int32_t)units, (int32_t)(w / 2), (int32_t)(c / 8),
                       (int32_t)c, dtype == MDNN_BF16);
    return check_launch("maxpool2_fwd_vec_kernel");
  }
  unsigned g = grid_for(total, 256);
  if (g > 16384) g = 16384;
  switch (dtype) {
    case MDNN_F32: hipLaunchKernelGGL(maxpool2_fwd_kernel<F32>, dim3(g), dim3(256), 0, st, (const float*)x, (float*)y, argmax, n, (int32_t)h, (int32_t)w, (int32_t)c); break;
    case MDNN_F16: hipLaunchKernelGGL(maxpool2_fwd_kernel<F16>, dim3(g), dim3(256), 0, st, (const uint16_t*)x, (uint16_t*)y, argmax, n, (int32_t)h, (int32_t)w, (int32_t)c); break;
    default: hipLaunchKernelGGL(maxpool2_fwd_kernel<BF16>, dim3(g), dim3(256), 0, st, (const uint16_t*)x, (uint16_t*)y, argmax, n, (int32_t)h, (int32_t)w, (int32_t)c); break;
  }
  return check_launch("maxpool2_fwd_kernel");
}

extern "C" mdnn_status_t mdnn_maxpool2_bwd(int64_t n, int64_t h, int64_t w, int64_t c,
                                           const void* dy, const uint8_t* argmax, void* dx,
                                           mdnn_dtype_t dtype, mdnn_stream_t stream) {
  if (n < 0 || h < 0 || w < 0 || c < 0 || h > 0x7fffffff || w > 0x7fffffff || c > 0x7fffffff)
    return fail(MDNN_ERR_SHAPE, "maxpool2_bwd: bad size");
  if (!dtype_ok(dtype)) return fail(MDNN_ERR_DTYPE, "maxpool2_bwd: unknown dtype");
  const int64_t total = n * h * w * c;
  if (total == 0) return MDNN_SUCCESS;
  if (!dx) return fail(MDNN_ERR_NULL, "maxpool2_bwd: dx is NULL");
  if ((n * (h / 2) * (w / 2) * c) > 0 && (!dy || !argmax))
    return fail(MDNN_ERR_NULL, "maxpool2_bwd: dy and argmax are required");
  const size_t es = dtype_size(dtype);
  if ((dy && !aligned(dy, es)) || !aligned(dx, es)) return fail(MDNN_ERR_MISALIGNED, "maxpool2_bwd: misaligned");
  clear_error();
  hipStream_t st = as_stream(stream);
  if (pool_vec_ok(n, h, w, c, dtype) && aligned(dy, 16) && aligned(dx, 16) && aligned(argmax, 8)) {
    const int64_t units = n * (h / 2) * (w / 2) * (c / 8);
    hipLaunchKernelGGL(maxpool2_bwd_vec_kernel, dim3((unsigned)ceil_div(units, 256)), dim3(256), 0, st,
                       (const uint16_t*)dy, argmax, (uint16_t*)dx, (int32_t)units, (int32_t)(w / 2), (int32_t)(c / 8),
                       (int32_t)c);
    return check_launch("maxpool2_bwd_vec_kernel");
  }
  unsigned g = grid_for(total, 256);
  if (g > 16384) g = 16384;
  switch (dtype) {
    case MDNN_F32: hipLaunchKernelGGL(maxpool2_bwd_kernel<F32>, dim3(g), dim3(256), 0, st, (const float*)dy, argmax, (float*)dx, n, (int32_t)h, (int32_t)w, (int32_t)c); break;
    case MDNN_F16: hipLaunchKernelGGL(maxpool2_bwd_kernel<F16>, dim3(g), dim3(256), 0, st, (const uint16_t*)dy, argmax, (uint16_t*)dx, n, (int32_t)h, (int32_t)w, (int32_t)c); break;
    default: hipLaunchKernelGGL(maxpool2_bwd_kernel<BF16>, dim3(g), dim3(256), 0, st, (const uint16_t*)dy, argmax, (uint16_t*)dx, n, (int32_t)h, (int32_t)w, (int32_t)c); break;
  }
  return check_launch("maxpool2_bwd_kernel");
}

namespace mdnn {
namespace {
mdnn_status_t launch_xent_rows(int64_t B, int64_t C, const float* logits, int64_t ldl, const int32_t* labels,
                               const float* loss_scale, float* loss_out, void* dlogits, int64_t ldd,
                               mdnn_dtype_t t, float* db, int32_t* nonfinite, hipStream_t st) {
  const size_t lds = db ? (size_t)B * C * sizeof(float) : 0;
  switch (t) {
    case MDNN_F32: hipLaunchKernelGGL(softmax_xent_rows_kernel<F32>, dim3(1), dim3(LOSS_THREADS), lds, st, B, C, logits, ldl, labels, loss_scale, loss_out, (float*)dlogits, ldd, db, nonfinite); break;
    case MDNN_F16: hipLaunchKernelGGL(softmax_xent_rows_kernel<F16>, dim3(1), dim3(LOSS_THREADS), lds, st, B, C, logits, ldl, labels, loss_scale, loss_out, (uint16_t*)dlogits, ldd, db, nonfinite); break;
    default: hipLaunchKernelGGL(softmax_xent_rows_kernel<BF16>, dim3(1), dim3(LOSS_THREADS), lds, st, B, C, logits, ldl, labels, loss_scale, loss_out, (uint16_t*)dlogits, ldd, db, nonfinite); break;
  }
  return check_launch("softmax_xent_rows_kernel");
}
}  // namespace

bool softmax_xent_db_ok(int64_t B, int64_t C) {
  return B >= 1 && B <= LOSS_THREADS && C >= 1 && C <= SMALL_C && (size_t)B * C * sizeof(float) <= XENT_DB_LDS;
}

mdnn_status_t softmax_xent_db(int64_t B, int64_t C, const float* logits, int64_t ldl, const int32_t* labels,
                              const float* loss_scale, float* loss_out, void* dlogits, int64_t ldd, mdnn_dtype_t t,
                              float* db, int32_t* nonfinite, hipStream_t st) {
  if (!softmax_xent_db_ok(B, C)) return fail(MDNN_ERR_SHAPE, "softmax_xent_db: shape outside the fused kernel");
  return launch_xent_rows(B, C, logits, ldl, labels, loss_scale, loss_out, dlogits, ldd, t, db, nonfinite, st);
}
}  // namespace mdnn

extern "C" mdnn_status_t mdnn_softmax_xent(int64_t B, int64_t C, const float* logits, int64_t ldl,
                                           const int32_t* labels, const float* loss_scale,
                                           float* loss_out, void* dlogits, int64_t ldd,
                                           mdnn_dtype_t dlogits_type, mdnn_stream_t stream) {
  if (B < 1 || C < 1 || C > 1024) return fail(MDNN_ERR_SHAPE, "softmax_xent: need B >= 1, 1 <= C <= 1024");
  if (ldl < C || ldd < C) return fail(MDNN_ERR_LAYOUT, "softmax_xent: row stride < C");
  if (!dtype_ok(dlogits_type)) return fail(MDNN_ERR_DTYPE, "softmax_xent: unknown dtype");
  if (!logits || !labels || !loss_out || !dlogits) return fail(MDNN_ERR_NULL, "softmax_xent: NULL buffer");
  if (!aligned(logits, 4) || !aligned(labels, 4) || !aligned(loss_out, 4) ||
      !aligned(dlogits, dtype_size(dlogits_type)) || (loss_scale && !aligned(loss_scale, 4)))
    return fail(MDNN_ERR_MISALIGNED, "softmax_xent: misaligned buffer");
  clear_error();
  hipStream_t st = as_stream(stream);
  if (C <= SMALL_C) return launch_xent_rows(B, C, logits, ldl, labels, loss_scale, loss_out, dlogits, ldd,
                                            dlogits_type, nullptr, nullptr, st);
  switch (dlogits_type) {
    case MDNN_F32: hipLaunchKernelGGL(softmax_xent_kernel<F32>, dim3(1), dim3(LOSS_THREADS), 0, st, B, C, logits, ldl, labels, loss_scale, loss_out, (float*)dlogits, ldd); break;
    case MDNN_F16: hipLaunchKernelGGL(softmax_xent_kernel<F16>, dim3(1), dim3(LOSS_THREADS), 0, st, B, C, logits, ldl, labels, loss_scale, loss_out, (uint16_t*)dlogits, ldd); break;
    default: hipLaunchKernelGGL(softmax_xent_kernel<BF16>, dim3(1), dim3(LOSS_THREADS), 0, st, B, C, logits, ldl, labels, loss_scale, loss_out, (uint16_t*)dlogits, ldd); break;
  }
  return check_launch("softmax_xent_kernel");
}

extern "C" mdnn_status_t mdnn_mse_loss(int64_t B, int64_t O, const float* y, const float* t,
                                       const float* loss_scale, float* loss_out, void* dy,
                                       mdnn_dtype_t dy_type, mdnn_stream_t stream) {
  if (B < 1 || O < 1) return fail(MDNN_ERR_SHAPE, "mse_loss: need B, O >= 1");
  if (!dtype_ok(dy_type)) return fail(MDNN_ERR_DTYPE, "mse_loss: unknown dtype");
  if (!y || !t || !loss_out || !dy) return fail(MDNN_ERR_NULL, "mse_loss: NULL buffer");
  if (!aligned(y, 4) || !aligned(t, 4) || !aligned(loss_out, 4) || !aligned(dy, dtype_size(dy_type)) ||
      (loss_scale && !aligned(loss_scale, 4)))
    return fail(MDNN_ERR_MISALIGNED, "mse_loss: misaligned buffer");
  clear_error();
  hipStream_t st = as_stream(stream);
  const int64_t n = B * O;
  switch (dy_type) {
    case MDNN_F32: hipLaunchKernelGGL(mse_kernel<F32>, dim3(1), dim3(LOSS_THREADS), 0, st, n, B, y, t, loss_scale, loss_out, (float*)dy); break;
    case MDNN_F16: hipLaunchKernelGGL(mse_kernel<F16>, dim3(1), dim3(LOSS_THREADS), 0, st, n, B, y, t, loss_scale, loss_out, (uint16_t*)dy); break;
    default: hipLaunchKernelGGL(mse_kernel<BF16>, dim3(1), dim3(LOSS_THREADS), 0, st, n, B, y, t, loss_scale, loss_out, (uint16_t*)dy); break;
  }
  return check_launch("mse_kernel");
}

extern "C" mdnn_status_t mdnn_sgd_update_async(int64_t n, float* w32, const float* g32, float* v32,
                                               float lr, float momentum, mdnn_scaler_t* scaler,
                                               mdnn_stream_t stream) {
  if (n < 0) return fail(MDNN_ERR_SHAPE, "sgd_update_async: n < 0");
  if (n > 0 && (!w32 || !g32)) return fail(MDNN_ERR_NULL, "sgd_update_async: w32 and g32 are required");
  if ((w32 && !aligned(w32, 4)) || (g32 && !aligned(g32, 4)) || (v32 && !aligned(v32, 4)) ||
      (scaler && !aligned(scaler, 4)))
    return fail(MDNN_ERR_MISALIGNED, "sgd_update_async: misaligned pointer");
  clear_error();
  hipStream_t st = as_stream(stream);
  if (scaler && n > 0) MDNN_TRY(finite_check_all(g32, n, scaler, st));
  if (n > 0) {
    const unsigned g = stream_grid(n);
    const bool mom = v32 != nullptr, sc = scaler != nullptr;
    if (mom && sc)
      hipLaunchKernelGGL((sgd_async_kernel<true, true>), dim3(g), dim3(256), 0, st, n, w32, g32, v32, lr, momentum, scaler);
    else if (mom)
      hipLaunchKernelGGL((sgd_async_kernel<true, false>), dim3(g), dim3(256), 0, st, n, w32, g32, v32, lr, momentum, scaler);
    else if (sc)
      hipLaunchKernelGGL((sgd_async_kernel<false, true>), dim3(g), dim3(256), 0, st, n, w32, g32, v32, lr, momentum, scaler);
    else
      hipLaunchKernelGGL((sgd_async_kernel<false, false>), dim3(g), dim3(256), 0, st, n, w32, g32, v32, lr, momentum, scaler);
    MDNN_TRY(check_launch("sgd_async_kernel"));
  }
  if (scaler) {
    hipLaunchKernelGGL(scaler_finalize_kernel, dim3(1), dim3(64), 0, st, scaler);
    MDNN_TRY(check_launch("scaler_finalize_kernel"));
  }
  return MDNN_SUCCESS;
}

static mdnn_status_t sgd_update_impl(int64_t n, float* w32, const float* g32, float* v32, void* w_lp,
                                     mdnn_dtype_t lp_type, float lr, float momentum, mdnn_scaler_t* scaler,
                                     mdnn_stream_t stream, bool check);

extern "C" mdnn_status_t mdnn_sgd_update(int64_t n, float* w32, const float* g32, float* v32,
                                         void* w_lp, mdnn_dtype_t lp_type, float lr,
                                         float momentum, mdnn_scaler_t* scaler,
                                         mdnn_stream_t stream) {
  return sgd_update_impl(n, w32, g32, v32, w_lp, lp_type, lr, momentum, scaler, stream, true);
}

mdnn_status_t mdnn::sgd_update_prechecked(int64_t n, float* w32, const float* g32, float* v32, void* w_lp,
                                          mdnn_dtype_t lp_type, float lr, float momentum, mdnn_scaler_t* scaler,
                                          mdnn_stream_t stream) {
  return sgd_update_impl(n, w32, g32, v32, w_lp, lp_type, lr, momentum, scaler, stream, false);
}

mdnn_status_t mdnn::finite_check_ranges(const float* g, const CheckRanges& r, mdnn_scaler_t* scaler,
                                        hipStream_t st) {
  if (r.n <= 0) return MDNN_SUCCESS;
  if (r.n > kMaxCheckRanges) return fail(MDNN_ERR_SHAPE, "finite check: too many ranges");
  int64_t longest = 0;
  for (int i = 0; i < r.n; ++i) longest = r.len[i] > longest ? r.len[i] : longest;
  if (longest == 0) return MDNN_SUCCESS;
  unsigned gx = grid_for(longest, 256);
  if (gx > 256) gx = 256;
  hipLaunchKernelGGL(finite_check_ranges_kernel, dim3(gx, (unsigned)r.n), dim3(256), 0, st, g, r, scaler);
  return check_launch("finite_check_ranges_kernel");
}

template <class LpT>
static void sgd_ranges_launch(const CheckRanges& r, unsigned gx, float* w, const float* g, float* v, void* wlp,
                              float lr, float mu, const mdnn_scaler_t* sc, hipStream_t st) {
  typedef typename LpT::storage L;
  const dim3 grid(gx, (unsigned)r.n);
  const bool vec = aligned(w, 16) && aligned(g, 16) && (!v || aligned(v, 16)) && (!wlp || aligned(wlp, 4 * sizeof(L)));
  if (v && sc)
    hipLaunchKernelGGL((sgd_ranges_kernel<LpT, true, true>), grid, dim3(256), 0, st, r, w, g, v, (L*)wlp, lr, mu, sc,
                       vec);
  else if (v)
    hipLaunchKernelGGL((sgd_ranges_kernel<LpT, true, false>), grid, dim3(256), 0, st, r, w, g, v, (L*)wlp, lr, mu,
                       sc, vec);
  else if (sc)
    hipLaunchKernelGGL((sgd_ranges_kernel<LpT, false, true>), grid, dim3(256), 0, st, r, w, g, v, (L*)wlp, lr, mu,
                       sc, vec);
  else
    hipLaunchKernelGGL((sgd_ranges_kernel<LpT, false, false>), grid, dim3(256), 0, st, r, w, g, v, (L*)wlp, lr, mu,
                       sc, vec);
}

mdnn_status_t mdnn::sgd_update_ranges_prechecked(const CheckRanges& r, float* w32, const float* g32, float* v32,
                                                 void* w_lp, mdnn_dtype_t lp_type, float lr, float momentum,
                                                 mdnn_scaler_t* scaler, hipStream_t st) {
  if (r.n < 0 || r.n > kMaxCheckRanges) return fail(MDNN_ERR_SHAPE, "sgd_update: too many ranges");
  int64_t longest = 0;
  for (int i = 0; i < r.n; ++i) longest = r.len[i] > longest ? r.len[i] : longest;
  if (longest > 0) {
    const unsigned gx = stream_grid(ceil_div(longest, (int64_t)4));
    float* v = momentum != 0.0f ? v32 : nullptr;
    switch (lp_type) {
      case MDNN_F32: sgd_ranges_launch<F32>(r, gx, w32, g32, v, w_lp, lr, momentum, scaler, st); break;
      case MDNN_F16: sgd_ranges_launch<F16>(r, gx, w32, g32, v, w_lp, lr, momentum, scaler, st); break;
      default: sgd_ranges_launch<BF16>(r, gx, w32, g32, v, w_lp, lr, momentum, scaler, st); break;
    }
    MDNN_TRY(check_launch("sgd_ranges_kernel"));
  }
  if (scaler) {
    hipLaunchKernelGGL(scaler_finalize_kernel, dim3(1), dim3(64), 0, st, scaler);
    MDNN_TRY(check_launch("scaler_finalize_kernel"));
  }
  return MDNN_SUCCESS;
}

static mdnn_status_t sgd_update_impl(int64_t n, float* w32, const float* g32, float* v32, void* w_lp,
                                     mdnn_dtype_t lp_type, float lr, float momentum, mdnn_scaler_t* scaler,
                                     mdnn_stream_t stream, bool check) {
  if (n < 0) return fail(MDNN_ERR_SHAPE, "sgd_update: n < 0");
  if (!dtype_ok(lp_type)) return fail(MDNN_ERR_DTYPE, "sgd_update: unknown lp_type");
  if (n > 0 && (!w32 || !g32)) return fail(MDNN_ERR_NULL, "sgd_update: w32 and g32 are required");
  if ((w32 && !aligned(w32, 4)) || (g32 && !aligned(g32, 4)) || (v32 && !aligned(v32, 4)) ||
      (w_lp && !aligned(w_lp, dtype_size(lp_type))) || (scaler && !aligned(scaler, 4)))
    return fail(MDNN_ERR_MISALIGNED, "sgd_update: a pointer is not aligned to its element size");
  clear_error();
  hipStream_t st = as_stream(stream);
  if (check && scaler && n > 0) MDNN_TRY(finite_check_all(g32, n, scaler, st));
  if (n > 0) {
    switch (lp_type) {
      case MDNN_F32: sgd_launch<F32>(n, w32, g32, v32, w_lp, lr, momentum, scaler, st); break;
      case MDNN_F16: sgd_launch<F16>(n, w32, g32, v32, w_lp, lr, momentum, scaler, st); break;
      default: sgd_launch<BF16>(n, w32, g32, v32, w_lp, lr, momentum, scaler, st); break;
    }
    MDNN_TRY(check_launch("sgd_kernel"));
  }
  if (scaler) {
    hipLaunchKernelGGL(scaler_finalize_kernel, dim3(1), dim3(64), 0, st, scaler);
    MDNN_TRY(check_launch("scaler_finalize_kernel"));
  }
  return MDNN_SUCCESS;
}
