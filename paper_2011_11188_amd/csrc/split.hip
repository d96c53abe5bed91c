// fp32 matrix products on the fp16 matrix cores: section 3.2's Eq. (1).
//
// An fp32 matrix X at a power-of-two scale s is split into fp16 matrices
//   X1 = RNE16(X / s),  X2 = RNE16((X / s - X1) * 2^11),
// so that X ~ s*X1 + s*2^-11*X2 to about 22 significant bits (X / s - X1 is
// exact in fp32, and scaling by powers of two is exact).  A product of two
// split matrices keeps three fp16 products,
//   A B ~ a b [ A1 B1 + 2^-11 (A1 B2 + A2 B1) ],
// which run on the MFMA GEMM engine as two launches: the two correction
// products as one GEMM over the concatenated depth [A1 | A2] x [B2 ; B1]
// (fp32 result, with beta*C folded in), then the leading product whose
// epilogue adds that result.  Both accumulate in fp32.
#include <cmath>

#include "common.h"
#include "internal.h"

namespace mdnn {
namespace {

constexpr float SHIFT_UP = 2048.0f;  // 2^11 = s / s2

// rows x cols fp32 (leading dimension ldx) -> hi / lo fp16.  inv_scale = 1/s
// (a power of two, so x * inv_scale is exact for normal results), or 1 /
// *scale_dev when the scale was chosen on the device.
__global__ void __launch_bounds__(256)
split_f16_kernel(int64_t rows, int64_t cols, const float* __restrict__ x, int64_t ldx, float inv_scale,
                 const float* __restrict__ scale_dev, uint16_t* __restrict__ hi, int64_t ldh,
                 uint16_t* __restrict__ lo, int64_t ldl) {
  if (scale_dev) inv_scale = 1.0f / *scale_dev;  // exact: a power of two in [2^-126, 2^113]
  const int64_t row = blockIdx.y;
  for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < cols; c += (int64_t)gridDim.x * 256) {
    const float v = x[row * ldx + c] * inv_scale;
    const uint16_t h = f32_to_f16(v);
    const float r = v - f16_to_f32(h);  // exact: v and h agree in their leading 11 bits
    hi[row * ldh + c] = h;
    lo[row * ldl + c] = f32_to_f16(r * SHIFT_UP);
  }
}

// Automatic scale (the paper does not say how to pick a1): the power of two
// s = 2^(floor(log2 max|x|) - 14), which puts max|x| / s in [2^14, 2^15),
// inside fp16's range with its leading bits in the normal range; s = 1 when
// max|x| is 0, Inf or NaN; s >= 2^-126.  Pass 1: max |x| as fp32 bit
// patterns (ordered like the magnitudes; NaN above Inf), one atomic max per
// block into a word that starts at 0.
__global__ void __launch_bounds__(256)
absmax_bits_kernel(int64_t rows, int64_t cols, const float* __restrict__ x, int64_t ldx, uint32_t* bits) {
  const int64_t row = blockIdx.y;
  uint32_t m = 0;
  for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < cols; c += (int64_t)gridDim.x * 256) {
    const uint32_t u = __float_as_uint(x[row * ldx + c]) & 0x7fffffffu;
    m = u > m ? u : m;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint32_t o = (uint32_t)__shfl_xor((int)m, off);
    m = o > m ? o : m;
  }
  __shared__ uint32_t wmax[4];
  if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w) m = wmax[w] > m ? wmax[w] : m;
    m = wmax[0] > m ? wmax[0] : m;
    if (m) atomicMax(bits, m);
  }
}

__device__ float auto_scale(uint32_t bits) {
  if (bits == 0 || bits >= 0x7f800000u) return 1.0f;
  int e = ilogbf(__uint_as_float(bits)) - 14;  // floor(log2 max|x|) - 14
  if (e < -126) e = -126;
  return ldexpf(1.0f, e);
}

// Pass 2: words[0] and words[1] hold the bit maxima of A and B (or are
// unused when a fixed scale > 0 is given); they become the scales s_a, s_b,
// and words[2] = s_a * s_b.
__global__ void scales_kernel(uint32_t* words, float a_fixed, float b_fixed) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const float sa = a_fixed > 0.0f ? a_fixed : auto_scale(words[0]);
  const float sb = b_fixed > 0.0f ? b_fixed : auto_scale(words[1]);
  float* f = (float*)words;
  f[0] = sa;
  f[1] = sb;
  f[2] = sa * sb;
}

// the automatic scale of one matrix, in place (word 0 only)
__global__ void scale_one_kernel(uint32_t* word) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  *(float*)word = auto_scale(*word);
}

bool power_of_two(float s) {
  if (!(s > 0.0f) || !std::isfinite(s)) return false;
  int e;
  return std::frexp(s, &e) == 0.5f && e > -125 && e < 126;
}

size_t seg(size_t bytes) { return (bytes + 255) & ~(size_t)255; }

// scale_dev: device scale (chosen on the device) or null (host `scale`)
mdnn_status_t launch_split(int64_t rows, int64_t cols, const float* x, int64_t ldx, float scale,
                           const float* scale_dev, void* hi, int64_t ldh, void* lo, int64_t ldl, hipStream_t st) {
  if (rows == 0 || cols == 0) return MDNN_SUCCESS;
  if (rows > 65535) {
    // the grid's y extent holds the row; split tall matrices into bands
    for (int64_t r0 = 0; r0 < rows; r0 += 65535) {
      const int64_t nr = rows - r0 < 65535 ? rows - r0 : 65535;
      MDNN_TRY(launch_split(nr, cols, x + r0 * ldx, ldx, scale, scale_dev, (uint16_t*)hi + r0 * ldh, ldh,
                            (uint16_t*)lo + r0 * ldl, ldl, st));
    }
    return MDNN_SUCCESS;
  }
  int64_t bx = ceil_div(cols, 256);
  if (bx > 1024) bx = 1024;
  hipLaunchKernelGGL(split_f16_kernel, dim3((unsigned)bx, (unsigned)rows), dim3(256), 0, st, rows, cols, x, ldx,
                     scale_dev ? 1.0f : 1.0f / scale, scale_dev, (uint16_t*)hi, ldh, (uint16_t*)lo, ldl);
  return check_launch("split_f16_kernel");
}

// atomic max of |x|'s bit patterns into *bits (pass 1 of the automatic scale)
mdnn_status_t launch_absmax(int64_t rows, int64_t cols, const float* x, int64_t ldx, uint32_t* bits,
                            hipStream_t st) {
  if (rows == 0 || cols == 0) return MDNN_SUCCESS;
  for (int64_t r0 = 0; r0 < rows; r0 += 65535) {
    const int64_t nr = rows - r0 < 65535 ? rows - r0 : 65535;
    int64_t bx = ceil_div(cols, 256);
    if (bx > 64) bx = 64;
    hipLaunchKernelGGL(absmax_bits_kernel, dim3((unsigned)bx, (unsigned)nr), dim3(256), 0, st, nr, cols,
                       x + r0 * ldx, ldx, bits);
    MDNN_TRY(check_launch("absmax_bits_kernel"));
  }
  return MDNN_SUCCESS;
}

}  // namespace
}  // namespace mdnn

using namespace mdnn;

extern "C" mdnn_status_t mdnn_split_f16(int64_t rows, int64_t cols, const float* x, int64_t ldx, float scale,
                                        float* scale_out, void* hi, int64_t ldh, void* lo, int64_t ldl,
                                        mdnn_stream_t stream) {
  if (rows < 0 || cols < 0) return fail(MDNN_ERR_SHAPE, "split: negative size");
  const bool automatic = scale == 0.0f;
  if (!automatic && !power_of_two(scale))
    return fail(MDNN_ERR_SHAPE, "split: scale must be a positive power of two, or 0 (chosen on the device)");
  if (automatic && !scale_out) return fail(MDNN_ERR_NULL, "split: scale 0 needs scale_out");
  if (scale_out && !aligned(scale_out, 4)) return fail(MDNN_ERR_MISALIGNED, "split: scale_out is misaligned");
  if ((rows == 0 || cols == 0) && !automatic) return MDNN_SUCCESS;
  if ((rows > 0 && cols > 0) && (!x || !hi || !lo)) return fail(MDNN_ERR_NULL, "split: x, hi and lo are required");
  if (rows > 0 && cols > 0 && (ldx < cols || ldh < cols || ldl < cols))
    return fail(MDNN_ERR_LAYOUT, "split: leading dimension < cols");
  if ((x && !aligned(x, 4)) || (hi && !aligned(hi, 2)) || (lo && !aligned(lo, 2)))
    return fail(MDNN_ERR_MISALIGNED, "split: misaligned base pointer");
  clear_error();
  hipStream_t st = as_stream(stream);
  if (!automatic) return launch_split(rows, cols, x, ldx, scale, nullptr, hi, ldh, lo, ldl, st);
  uint32_t* w = (uint32_t*)scale_out;
  MDNN_TRY(fill_zero(w, 4, st));
  MDNN_TRY(launch_absmax(rows, cols, x, ldx, w, st));
  hipLaunchKernelGGL(scale_one_kernel, dim3(1), dim3(64), 0, st, w);
  MDNN_TRY(check_launch("scale_one_kernel"));
  return launch_split(rows, cols, x, ldx, 1.0f, scale_out, hi, ldh, lo, ldl, st);
}

// Workspace: [A1 | A2] (2 M K fp16), [B2 ; B1] (2 K N fp16), the fp32
// correction product (M N), and three scale words (s_a, s_b, s_a s_b), each
// 256-byte aligned.
extern "C" size_t mdnn_gemm_split3_workspace(int64_t M, int64_t N, int64_t K) {
  if (M < 0 || N < 0 || K < 0) return 0;
  return seg((size_t)2 * M * K * 2) + seg((size_t)2 * K * N * 2) + seg((size_t)M * N * 4) + 256;
}

extern "C" mdnn_status_t mdnn_gemm_split3(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K, float alpha,
                                          const float* A, int64_t lda, float a_scale, const float* B, int64_t ldb,
                                          float b_scale, float beta, const float* C, int64_t ldc, float* D,
                                          int64_t ldd, void* workspace, size_t ws_bytes, mdnn_stream_t stream) {
  if (layout != MDNN_NN && layout != MDNN_NT && layout != MDNN_TN)
    return fail(MDNN_ERR_LAYOUT, "gemm_split3: unknown layout %d", (int)layout);
  if (M < 0 || N < 0 || K < 0) return fail(MDNN_ERR_SHAPE, "gemm_split3: negative size");
  if ((a_scale != 0.0f && !power_of_two(a_scale)) || (b_scale != 0.0f && !power_of_two(b_scale)))
    return fail(MDNN_ERR_SHAPE, "gemm_split3: scales must be positive powers of two, or 0 (chosen on the device)");
  if (M == 0 || N == 0) return MDNN_SUCCESS;
  if (!D) return fail(MDNN_ERR_NULL, "gemm_split3: D is NULL");
  if (K > 0 && (!A || !B)) return fail(MDNN_ERR_NULL, "gemm_split3: A or B is NULL");
  if (beta != 0.0f && !C) return fail(MDNN_ERR_NULL, "gemm_split3: beta != 0 but C is NULL");
  const int64_t a_w = layout == MDNN_TN ? M : K, b_w = layout == MDNN_NT ? K : N;
  if (K > 0 && (lda < a_w || lda < 1)) return fail(MDNN_ERR_LAYOUT, "gemm_split3: lda < %lld", (long long)a_w);
  if (K > 0 && (ldb < b_w || ldb < 1)) return fail(MDNN_ERR_LAYOUT, "gemm_split3: ldb < %lld", (long long)b_w);
  if (ldd < N) return fail(MDNN_ERR_LAYOUT, "gemm_split3: ldd < N");
  if (beta != 0.0f && ldc < N) return fail(MDNN_ERR_LAYOUT, "gemm_split3: ldc < N");
  if ((A && !aligned(A, 4)) || (B && !aligned(B, 4)) || !aligned(D, 4) || (C && !aligned(C, 4)))
    return fail(MDNN_ERR_MISALIGNED, "gemm_split3: a base pointer is not 4-byte aligned");
  const size_t need = mdnn_gemm_split3_workspace(M, N, K);
  if (!workspace || ws_bytes < need || !aligned(workspace, 256))
    return fail(MDNN_ERR_WORKSPACE, "gemm_split3: needs %zu bytes of 256-byte aligned workspace", need);
  clear_error();
  hipStream_t st = as_stream(stream);
  char* ws = (char*)workspace;
  uint16_t* ah = (uint16_t*)ws;                                           // [A1 | A2]
  uint16_t* bh = (uint16_t*)(ws + seg((size_t)2 * M * K * 2));            // [B2 ; B1]
  float* dlo = (float*)(ws + seg((size_t)2 * M * K * 2) + seg((size_t)2 * K * N * 2));
  // scales chosen on the device (a_scale or b_scale 0): the split kernels
  // read theirs and the products' epilogues multiply alpha by s_a s_b
  const bool automatic = a_scale == 0.0f || b_scale == 0.0f;
  float* scl = (float*)(ws + seg((size_t)2 * M * K * 2) + seg((size_t)2 * K * N * 2) + seg((size_t)M * N * 4));
  const float* sa_dev = nullptr;
  const float* sb_dev = nullptr;
  const float* ab_dev = nullptr;
  if (automatic) {
    uint32_t* w = (uint32_t*)scl;
    MDNN_TRY(fill_zero(w, 16, st));
    if (a_scale == 0.0f) {
      if (layout == MDNN_TN)
        MDNN_TRY(launch_absmax(K, M, A, lda, w, st));
      else
        MDNN_TRY(launch_absmax(M, K, A, lda, w, st));
    }
    if (b_scale == 0.0f) {
      if (layout == MDNN_NT)
        MDNN_TRY(launch_absmax(N, K, B, ldb, w + 1, st));
      else
        MDNN_TRY(launch_absmax(K, N, B, ldb, w + 1, st));
    }
    hipLaunchKernelGGL(scales_kernel, dim3(1), dim3(64), 0, st, w, a_scale, b_scale);
    MDNN_TRY(check_launch("scales_kernel"));
    sa_dev = scl;
    sb_dev = scl + 1;
    ab_dev = scl + 2;
  }
  // concatenated operands: K-contiguous ones side by side along the row,
  // MN-contiguous ones stacked by rows
  int64_t ld_ah, ld_bh;
  const uint16_t *a1, *b1;
  if (layout == MDNN_TN) {  // A stored [K][M]
    ld_ah = M;
    MDNN_TRY(launch_split(K, M, A, lda, a_scale, sa_dev, ah, M, ah + K * M, M, st));
  } else {  // A stored [M][K]
    ld_ah = 2 * K;
    MDNN_TRY(launch_split(M, K, A, lda, a_scale, sa_dev, ah, 2 * K, ah + K, 2 * K, st));
  }
  a1 = ah;
  if (layout == MDNN_NT) {  // B stored [N][K]: [B2 | B1]
    ld_bh = 2 * K;
    MDNN_TRY(launch_split(N, K, B, ldb, b_scale, sb_dev, bh + K, 2 * K, bh, 2 * K, st));
    b1 = bh + K;
  } else {  // B stored [K][N]: [B2 ; B1]
    ld_bh = N;
    MDNN_TRY(launch_split(K, N, B, ldb, b_scale, sb_dev, bh + K * N, N, bh, N, st));
    b1 = bh + K * N;
  }
  const float ab = automatic ? alpha : alpha * a_scale * b_scale;
  // corrections: alpha a b 2^-11 (A1 B2 + A2 B1) + beta C
  MDNN_TRY(gemm_mixed_ws(layout, M, N, 2 * K, ab / SHIFT_UP, ah, ld_ah, bh, ld_bh, MDNN_F16, beta, C, ldc, dlo, N,
                         MDNN_F32, nullptr, MDNN_ACT_NONE, nullptr, 0, nullptr, 0, stream, nullptr, ab_dev));
  // leading product plus the corrections
  return gemm_mixed_ws(layout, M, N, K, ab, a1, ld_ah, b1, ld_bh, MDNN_F16, 1.0f, dlo, N, D, ldd, MDNN_F32, nullptr,
                       MDNN_ACT_NONE, nullptr, 0, nullptr, 0, stream, nullptr, ab_dev);
}
