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
// (a power of two, so x * inv_scale is exact for normal results).
__global__ void __launch_bounds__(256)
split_f16_kernel(int64_t rows, int64_t cols, const float* __restrict__ x, int64_t ldx, float inv_scale,
                 uint16_t* __restrict__ hi, int64_t ldh, uint16_t* __restrict__ lo, int64_t ldl) {
  const int64_t row = blockIdx.y;
  for (int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x; c < cols; c += (int64_t)gridDim.x * 256) {
    const float v = x[row * ldx + c] * inv_scale;
    const uint16_t h = f32_to_f16(v);
    const float r = v - f16_to_f32(h);  // exact: v and h agree in their leading 11 bits
    hi[row * ldh + c] = h;
    lo[row * ldl + c] = f32_to_f16(r * SHIFT_UP);
  }
}

bool power_of_two(float s) {
  if (!(s > 0.0f) || !std::isfinite(s)) return false;
  int e;
  return std::frexp(s, &e) == 0.5f && e > -125 && e < 126;
}

size_t seg(size_t bytes) { return (bytes + 255) & ~(size_t)255; }

mdnn_status_t launch_split(int64_t rows, int64_t cols, const float* x, int64_t ldx, float scale, void* hi,
                           int64_t ldh, void* lo, int64_t ldl, hipStream_t st) {
  if (rows == 0 || cols == 0) return MDNN_SUCCESS;
  if (rows > 65535) {
    // the grid's y extent holds the row; split tall matrices into bands
    for (int64_t r0 = 0; r0 < rows; r0 += 65535) {
      const int64_t nr = rows - r0 < 65535 ? rows - r0 : 65535;
      MDNN_TRY(launch_split(nr, cols, x + r0 * ldx, ldx, scale, (uint16_t*)hi + r0 * ldh, ldh,
                            (uint16_t*)lo + r0 * ldl, ldl, st));
    }
    return MDNN_SUCCESS;
  }
  int64_t bx = ceil_div(cols, 256);
  if (bx > 1024) bx = 1024;
  hipLaunchKernelGGL(split_f16_kernel, dim3((unsigned)bx, (unsigned)rows), dim3(256), 0, st, rows, cols, x, ldx,
                     1.0f / scale, (uint16_t*)hi, ldh, (uint16_t*)lo, ldl);
  return check_launch("split_f16_kernel");
}

}  // namespace
}  // namespace mdnn

using namespace mdnn;

extern "C" mdnn_status_t mdnn_split_f16(int64_t rows, int64_t cols, const float* x, int64_t ldx, float scale,
                                        void* hi, int64_t ldh, void* lo, int64_t ldl, mdnn_stream_t stream) {
  if (rows < 0 || cols < 0) return fail(MDNN_ERR_SHAPE, "split: negative size");
  if (!power_of_two(scale)) return fail(MDNN_ERR_SHAPE, "split: scale must be a positive power of two");
  if (rows == 0 || cols == 0) return MDNN_SUCCESS;
  if (!x || !hi || !lo) return fail(MDNN_ERR_NULL, "split: x, hi and lo are required");
  if (ldx < cols || ldh < cols || ldl < cols) return fail(MDNN_ERR_LAYOUT, "split: leading dimension < cols");
  if (!aligned(x, 4) || !aligned(hi, 2) || !aligned(lo, 2))
    return fail(MDNN_ERR_MISALIGNED, "split: misaligned base pointer");
  clear_error();
  return launch_split(rows, cols, x, ldx, scale, hi, ldh, lo, ldl, as_stream(stream));
}

// Workspace: [A1 | A2] (2 M K fp16), [B2 ; B1] (2 K N fp16), the fp32
// correction product (M N), each 256-byte aligned.
extern "C" size_t mdnn_gemm_split3_workspace(int64_t M, int64_t N, int64_t K) {
  if (M < 0 || N < 0 || K < 0) return 0;
  return seg((size_t)2 * M * K * 2) + seg((size_t)2 * K * N * 2) + seg((size_t)M * N * 4);
}

extern "C" mdnn_status_t mdnn_gemm_split3(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K, float alpha,
                                          const float* A, int64_t lda, float a_scale, const float* B, int64_t ldb,
                                          float b_scale, float beta, const float* C, int64_t ldc, float* D,
                                          int64_t ldd, void* workspace, size_t ws_bytes, mdnn_stream_t stream) {
  if (layout != MDNN_NN && layout != MDNN_NT && layout != MDNN_TN)
    return fail(MDNN_ERR_LAYOUT, "gemm_split3: unknown layout %d", (int)layout);
  if (M < 0 || N < 0 || K < 0) return fail(MDNN_ERR_SHAPE, "gemm_split3: negative size");
  if (!power_of_two(a_scale) || !power_of_two(b_scale))
    return fail(MDNN_ERR_SHAPE, "gemm_split3: scales must be positive powers of two");
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
  // concatenated operands: K-contiguous ones side by side along the row,
  // MN-contiguous ones stacked by rows
  int64_t ld_ah, ld_bh;
  const uint16_t *a1, *b1;
  if (layout == MDNN_TN) {  // A stored [K][M]
    ld_ah = M;
    MDNN_TRY(launch_split(K, M, A, lda, a_scale, ah, M, ah + K * M, M, st));
  } else {  // A stored [M][K]
    ld_ah = 2 * K;
    MDNN_TRY(launch_split(M, K, A, lda, a_scale, ah, 2 * K, ah + K, 2 * K, st));
  }
  a1 = ah;
  if (layout == MDNN_NT) {  // B stored [N][K]: [B2 | B1]
    ld_bh = 2 * K;
    MDNN_TRY(launch_split(N, K, B, ldb, b_scale, bh + K, 2 * K, bh, 2 * K, st));
    b1 = bh + K;
  } else {  // B stored [K][N]: [B2 ; B1]
    ld_bh = N;
    MDNN_TRY(launch_split(K, N, B, ldb, b_scale, bh + K * N, N, bh, N, st));
    b1 = bh + K * N;
  }
  const float ab = alpha * a_scale * b_scale;
  // corrections: alpha a b 2^-11 (A1 B2 + A2 B1) + beta C
  MDNN_TRY(mdnn_gemm_mixed(layout, M, N, 2 * K, ab / SHIFT_UP, ah, ld_ah, bh, ld_bh, MDNN_F16, beta, C, ldc, dlo, N,
                           MDNN_F32, nullptr, MDNN_ACT_NONE, nullptr, 0, stream));
  // leading product plus the corrections
  return mdnn_gemm_mixed(layout, M, N, K, ab, a1, ld_ah, b1, ld_bh, MDNN_F16, 1.0f, dlo, N, D, ldd, MDNN_F32,
                         nullptr, MDNN_ACT_NONE, nullptr, 0, stream);
}
