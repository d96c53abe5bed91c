// mdnn_gemm_mixed: validation and dispatch of the GEMM engine; fixed-order
// reductions shared with the other entry points.
#include <atomic>

#include "gemm_launch.h"

namespace mdnn {

static std::atomic<int> g_tile_override{0};
int gemm_tile_override() { return g_tile_override.load(std::memory_order_relaxed); }

// ---------------------------------------------------------------------------
// fixed-order reductions
// ---------------------------------------------------------------------------
__global__ void reduce_splits_kernel(const float* __restrict__ part, int splits, int64_t n,
                                     float* __restrict__ out) {
  int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= n) return;
  if (i + 4 <= n && (n & 3) == 0) {
    float4 s = *(const float4*)(part + i);
    for (int k = 1; k < splits; ++k) {
      float4 v = *(const float4*)(part + (int64_t)k * n + i);
      s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
    }
    *(float4*)(out + i) = s;
  } else {
    for (int64_t e = i; e < i + 4 && e < n; ++e) {
      float s = part[e];
      for (int k = 1; k < splits; ++k) s += part[(int64_t)k * n + e];
      out[e] = s;
    }
  }
}

mdnn_status_t reduce_splits(const float* partial, int splits, int64_t rows, int64_t cols,
                            float* out, hipStream_t stream) {
  const int64_t n = rows * cols;
  if (n == 0) return MDNN_SUCCESS;
  const int64_t blocks = ceil_div(ceil_div(n, 4), 256);
  hipLaunchKernelGGL(reduce_splits_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, partial,
                     splits, n, out);
  return check_launch("reduce_splits_kernel");
}

// Column sums: a block owns 32 columns; 8 row lanes stride over the rows in
// order and are combined in a fixed order through LDS.
template <class T>
__global__ void __launch_bounds__(256)
column_sums_kernel(const typename T::storage* __restrict__ x, int64_t rows, int64_t cols,
                   float* __restrict__ out) {
  __shared__ float part[8][33];
  const int cx = threadIdx.x & 31, ry = threadIdx.x >> 5;
  const int64_t col = (int64_t)blockIdx.x * 32 + cx;
  float s = 0.0f;
  if (col < cols)
    for (int64_t r = ry; r < rows; r += 8) s += to_f<T>(x[r * cols + col]);
  part[ry][cx] = s;
  __syncthreads();
  if (ry == 0 && col < cols) {
    float t = part[0][cx];
#pragma unroll
    for (int k = 1; k < 8; ++k) t += part[k][cx];
    out[col] = t;
  }
}

mdnn_status_t column_sums(const void* x, mdnn_dtype_t t, int64_t rows, int64_t cols, float* out,
                          hipStream_t stream) {
  if (cols == 0) return MDNN_SUCCESS;
  dim3 grid((unsigned)ceil_div(cols, 32));
  switch (t) {
    case MDNN_F32:
      hipLaunchKernelGGL(column_sums_kernel<F32>, grid, dim3(256), 0, stream, (const float*)x, rows, cols, out);
      break;
    case MDNN_F16:
      hipLaunchKernelGGL(column_sums_kernel<F16>, grid, dim3(256), 0, stream, (const uint16_t*)x, rows, cols, out);
      break;
    default:
      hipLaunchKernelGGL(column_sums_kernel<BF16>, grid, dim3(256), 0, stream, (const uint16_t*)x, rows, cols, out);
      break;
  }
  return check_launch("column_sums_kernel");
}

// ---------------------------------------------------------------------------
// mdnn_gemm_mixed
// ---------------------------------------------------------------------------
template <class T, class OutT>
static mdnn_status_t gemm_dispatch16(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K,
                                     const void* A, int64_t lda, bool va, const void* B,
                                     int64_t ldb, bool vb, const Epilogue& ep, hipStream_t st) {
  const uint16_t* a = (const uint16_t*)A;
  const uint16_t* b = (const uint16_t*)B;
  switch (layout) {
    case MDNN_NN:
      return run_gemm16<T, OutT>(SrcMatK<uint16_t>{a, lda, M, K, va},
                                 SrcMatMN<uint16_t>{b, ldb, N, K, vb}, M, N, K, ep, 1, st);
    case MDNN_NT:
      return run_gemm16<T, OutT>(SrcMatK<uint16_t>{a, lda, M, K, va},
                                 SrcMatK<uint16_t>{b, ldb, N, K, vb}, M, N, K, ep, 1, st);
    default:
      return run_gemm16<T, OutT>(SrcMatMN<uint16_t>{a, lda, M, K, va},
                                 SrcMatMN<uint16_t>{b, ldb, N, K, vb}, M, N, K, ep, 1, st);
  }
}

static mdnn_status_t gemm_dispatch32(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K,
                                     const void* A, int64_t lda, const void* B, int64_t ldb,
                                     const Epilogue& ep, hipStream_t st) {
  const float* a = (const float*)A;
  const float* b = (const float*)B;
  switch (layout) {
    case MDNN_NN:
      return run_gemm32(SrcMatK<float>{a, lda, M, K, false}, SrcMatMN<float>{b, ldb, N, K, false},
                        M, N, K, ep, 1, st);
    case MDNN_NT:
      return run_gemm32(SrcMatK<float>{a, lda, M, K, false}, SrcMatK<float>{b, ldb, N, K, false},
                        M, N, K, ep, 1, st);
    default:
      return run_gemm32(SrcMatMN<float>{a, lda, M, K, false}, SrcMatMN<float>{b, ldb, N, K, false},
                        M, N, K, ep, 1, st);
  }
}

}  // namespace mdnn

using namespace mdnn;

extern "C" mdnn_status_t mdnn_gemm_mixed(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K,
                                         float alpha, const void* A, int64_t lda, const void* B,
                                         int64_t ldb, mdnn_dtype_t ab_type, float beta,
                                         const void* C, int64_t ldc, void* D, int64_t ldd,
                                         mdnn_dtype_t d_type, const float* bias, mdnn_act_t act,
                                         const void* mask_src, int64_t ldm, mdnn_stream_t stream) {
  if (layout != MDNN_NN && layout != MDNN_NT && layout != MDNN_TN)
    return fail(MDNN_ERR_LAYOUT, "gemm: unknown layout %d", (int)layout);
  if (M < 0 || N < 0 || K < 0) return fail(MDNN_ERR_SHAPE, "gemm: negative size");
  if (!dtype_ok(ab_type) || !dtype_ok(d_type)) return fail(MDNN_ERR_DTYPE, "gemm: unknown dtype");
  if (d_type != MDNN_F32 && d_type != ab_type)
    return fail(MDNN_ERR_DTYPE, "gemm: d_type must be fp32 or equal to ab_type");
  if (act != MDNN_ACT_NONE && act != MDNN_ACT_RELU) return fail(MDNN_ERR_DTYPE, "gemm: unknown act");
  if (M == 0 || N == 0) return MDNN_SUCCESS;
  if (!D) return fail(MDNN_ERR_NULL, "gemm: D is NULL");
  if (K > 0 && (!A || !B)) return fail(MDNN_ERR_NULL, "gemm: A or B is NULL");
  if (beta != 0.0f && !C) return fail(MDNN_ERR_NULL, "gemm: beta != 0 but C is NULL");
  // leading dimensions (row-major storage)
  const int64_t a_w = (layout == MDNN_TN) ? M : K;   // stored width of A
  const int64_t b_w = (layout == MDNN_NT) ? K : N;   // stored width of B
  if (K > 0 && (lda < a_w || lda < 1)) return fail(MDNN_ERR_LAYOUT, "gemm: lda %lld < %lld", (long long)lda, (long long)a_w);
  if (K > 0 && (ldb < b_w || ldb < 1)) return fail(MDNN_ERR_LAYOUT, "gemm: ldb %lld < %lld", (long long)ldb, (long long)b_w);
  if (ldd < N) return fail(MDNN_ERR_LAYOUT, "gemm: ldd < N");
  if (beta != 0.0f && ldc < N) return fail(MDNN_ERR_LAYOUT, "gemm: ldc < N");
  if (mask_src && ldm < N) return fail(MDNN_ERR_LAYOUT, "gemm: ldm < N");
  const size_t es = dtype_size(ab_type), ds = dtype_size(d_type);
  if ((A && !aligned(A, es)) || (B && !aligned(B, es)) || !aligned(D, ds) || (C && !aligned(C, ds)) ||
      (mask_src && !aligned(mask_src, es)) || (bias && !aligned(bias, 4)))
    return fail(MDNN_ERR_MISALIGNED, "gemm: a base pointer is not aligned to its element size");
  if (ab_type == MDNN_F32 && d_type != MDNN_F32)
    return fail(MDNN_ERR_DTYPE, "gemm: fp32 operands need an fp32 output");

  Epilogue ep{};
  ep.alpha = alpha;
  ep.beta = beta;
  ep.C = C;
  ep.ldc = ldc;
  ep.D = D;
  ep.ldd = ldd;
  ep.bias = bias;
  ep.mask = mask_src;
  ep.ldm = ldm;
  ep.act = act;
  ep.vec4 = (ldd % 4 == 0) && aligned(D, 4 * ds);
  ep.partial = nullptr;
  ep.k_per_split = K;
  hipStream_t st = as_stream(stream);
  clear_error();

  if (ab_type == MDNN_F32) return gemm_dispatch32(layout, M, N, K, A, lda, B, ldb, ep, st);
  const bool va = aligned(A, 16) && lda % 8 == 0;
  const bool vb = aligned(B, 16) && ldb % 8 == 0;
  if (ab_type == MDNN_F16) {
    if (d_type == MDNN_F32) return gemm_dispatch16<F16, F32>(layout, M, N, K, A, lda, va, B, ldb, vb, ep, st);
    return gemm_dispatch16<F16, F16>(layout, M, N, K, A, lda, va, B, ldb, vb, ep, st);
  }
  if (d_type == MDNN_F32) return gemm_dispatch16<BF16, F32>(layout, M, N, K, A, lda, va, B, ldb, vb, ep, st);
  return gemm_dispatch16<BF16, BF16>(layout, M, N, K, A, lda, va, B, ldb, vb, ep, st);
}

extern "C" int mdnn_set_gemm_tile(int code) {
  if (code < 0 || code > 3) return -1;
  g_tile_override.store(code, std::memory_order_relaxed);
  return 0;
}
