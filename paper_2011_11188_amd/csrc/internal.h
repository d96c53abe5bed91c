// Host-side internals of libmdnn: error reporting, argument checks and the
// launchers shared between translation units.
#pragma once

#include <hip/hip_runtime.h>
#include <stdarg.h>
#include <stdint.h>
#include <stdio.h>

#include "../../include/mdnn.h"

namespace mdnn {

mdnn_status_t fail(mdnn_status_t st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();
mdnn_status_t check_launch(const char* what);

inline size_t dtype_size(mdnn_dtype_t t) { return t == MDNN_F32 ? 4 : 2; }
inline bool dtype_ok(int t) { return t == MDNN_F32 || t == MDNN_F16 || t == MDNN_BF16; }
inline bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }
inline hipStream_t as_stream(mdnn_stream_t s) { return (hipStream_t)s; }

#define MDNN_TRY(expr)                          \
  do {                                          \
    mdnn_status_t st__ = (expr);                \
    if (st__ != MDNN_SUCCESS) return st__;      \
  } while (0)

// Split-K GEMM used by the convolution backward-filter path: partial sums
// are reduced by reduce_splits() in split order.
struct SplitPlan {
  int splits;
  int64_t k_per_split;
};

// Second passes of several split reductions, gathered for one launch.
// reduce_splits() and column_sums() given a batch append their second pass
// to it (when it is the many-splits reduction; other second passes launch
// at once) instead of launching it: the same sums in the same order, done
// when the caller launches the batch with reduce_batch_launch(), which must
// come after the partials are written and before their memory is reused.
// A full batch is launched by the call that would overflow it; a batch of
// one runs as that reduction's own launch.
constexpr int kMaxReduceBatch = 8;
struct ReduceBatch {
  int n;
  const float* part[kMaxReduceBatch];
  float* out[kMaxReduceBatch];
  int64_t elems[kMaxReduceBatch];
  int splits[kMaxReduceBatch];
  int opb[kMaxReduceBatch];  // outputs per block: 16 or 64
  int64_t first_block[kMaxReduceBatch + 1];
};
mdnn_status_t reduce_batch_launch(ReduceBatch& b, hipStream_t stream);

// Sum `splits` fp32 [rows, cols] partial matrices in split order into
// out[rows, cols] (fp32).
mdnn_status_t reduce_splits(const float* partial, int splits, int64_t rows, int64_t cols,
                            float* out, hipStream_t stream, ReduceBatch* defer = nullptr);
// mdnn_conv2d_bwd_filter with the second passes of its weight and bias
// sums appended to `defer` (the entry point launches them at once; a caller
// that keeps each layer's workspace apart can launch several layers' sums
// together).
mdnn_status_t conv2d_bwd_filter_deferred(const mdnn_conv_shape_t* shape, const void* x, const void* dy,
                                         mdnn_dtype_t io_type, float* dw, float* db, void* workspace,
                                         size_t ws_bytes, hipStream_t stream, ReduceBatch* defer);
// Zero `bytes` (a multiple of 4) with a fill kernel (no memset nodes, so the
// caller may capture the stream into a graph).
mdnn_status_t fill_zero(void* p, size_t bytes, hipStream_t stream);
// Element-wise conversion between any two storage types (RNE when narrowing).
mdnn_status_t cast_any(int64_t n, const void* src, mdnn_dtype_t s, void* dst, mdnn_dtype_t d,
                       hipStream_t stream);
// fp32 -> F16 / BF16 as cast_any, also setting *nonfinite (atomic OR) when a
// stored value is Inf or NaN.
mdnn_status_t cast_f32_checked(int64_t n, const float* src, void* dst, mdnn_dtype_t d, int32_t* nonfinite,
                               hipStream_t stream);
// Deterministic column sums of a [rows, cols] matrix x of type t (entries
// where y <= 0 skipped when y != NULL) into fp32 out[cols].  Uses a two-pass
// reduction when a workspace of column_sums_ws_bytes(rows, cols) bytes is
// given, a single (slower) pass otherwise.
size_t column_sums_ws_bytes(int64_t rows, int64_t cols);
mdnn_status_t column_sums(const void* x, const void* y, mdnn_dtype_t t, int64_t rows, int64_t cols,
                          float* out, void* ws, size_t ws_bytes, hipStream_t stream,
                          ReduceBatch* defer = nullptr);
// The two passes apart, for a caller that finishes several matrices' sums in
// one launch: pass 1 writes partial[column_sums_chunks(rows, cols, t)][cols]
// (fp32, 8-byte aligned; 16-bit rows whose width is a multiple of 512 are
// read in 64-row chunks of whole 1 KB runs and need 16-byte aligned x, other
// shapes take column_sums' 256-row chunks); pass 2 sums each entry's
// partials in a fixed order and, when nonfinite is given, ORs 1 into it for
// every non-finite sum (the loss scaler's overflow test of the sums it
// stores).  Deterministic, but not bitwise the same as column_sums where
// the chunks differ.
int64_t column_sums_chunks(int64_t rows, int64_t cols, mdnn_dtype_t t);

// mdnn_softmax_xent (C <= 32) that also writes db[C], the column sums of the
// stored dlogits (the classifier layer's bias gradient), in one launch;
// nonfinite (nullable) is set when a sum is Inf or NaN.  Shapes:
// softmax_xent_db_ok (B <= 1024 and B * C floats within the kernel's LDS).
bool softmax_xent_db_ok(int64_t B, int64_t C);
mdnn_status_t softmax_xent_db(int64_t B, int64_t C, const float* logits, int64_t ldl, const int32_t* labels,
                              const float* loss_scale, float* loss_out, void* dlogits, int64_t ldd, mdnn_dtype_t t,
                              float* db, int32_t* nonfinite, hipStream_t st);
mdnn_status_t column_sums_partial(const void* x, mdnn_dtype_t t, int64_t rows, int64_t cols, float* partial,
                                  hipStream_t stream);
constexpr int kMaxColsumBatch = 32;
struct ColsumBatch {
  int32_t n;
  const float* part[kMaxColsumBatch];
  float* out[kMaxColsumBatch];
  int64_t chunks[kMaxColsumBatch], cols[kMaxColsumBatch];
};
mdnn_status_t column_sums_final(const ColsumBatch& b, int32_t* nonfinite, hipStream_t stream);
// Pass 1 for several matrices of one height in one launch, each a 16-bit
// matrix of a multiple of 512 columns (16-byte aligned rows, 8-byte aligned
// partials: column_sums_strip_ok); the partials are those column_sums_partial
// writes.
struct StripBatch {
  int32_t n;
  const uint16_t* x[kMaxColsumBatch];
  float* partial[kMaxColsumBatch];
  int64_t cols[kMaxColsumBatch];
};
bool column_sums_strip_ok(const void* x, mdnn_dtype_t t, int64_t cols, const float* partial);
mdnn_status_t column_sums_partial_batch(const StripBatch& b, mdnn_dtype_t t, int64_t rows, hipStream_t stream);

// mdnn_gemm_mixed with an optional workspace (NULL / too small: same as
// mdnn_gemm_mixed).  With one, fp32 problems whose grid would be a handful of
// tiles over a long K split K across workgroups and reduce the fp32
// partials in split order (deterministic) before the epilogue.
size_t gemm_ws_bytes(mdnn_dtype_t ab_type, int64_t M, int64_t N, int64_t K);
mdnn_status_t gemm_mixed_ws(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K, float alpha, const void* A,
                            int64_t lda, const void* B, int64_t ldb, mdnn_dtype_t ab_type, float beta,
                            const void* C, int64_t ldc, void* D, int64_t ldd, mdnn_dtype_t d_type,
                            const float* bias, mdnn_act_t act, const void* mask_src, int64_t ldm, void* ws,
                            size_t ws_bytes, mdnn_stream_t stream, int32_t* nonfinite = nullptr,
                            const float* alpha_dev = nullptr);

// K splits of a 16-bit product given a large enough workspace (1: none).
int gemm_lp_splits(int64_t M, int64_t N, int64_t K);
// Whether mdnn_gemm_tn_update takes this problem (16-bit operands, M and N
// multiples of 256, the pipelined kernel's operand alignment, 16-byte
// aligned w32 / v32, 8-byte aligned w_lp, ldw a multiple of 4).
bool gemm_tn_update_ok(mdnn_dtype_t ab_type, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                       const void* B, int64_t ldb, const float* w32, const float* v32, const void* w_lp,
                       int64_t ldw);

// Loss-scaled updates whose gradients were checked where they were produced:
// gemm_mixed_ws with `nonfinite` = &scaler->reserved covers every fp32 value
// it stores (all of its kernel paths store through the same epilogue); the
// ranges no such producer wrote are checked here, one block row per range.
constexpr int kMaxCheckRanges = 32;
struct CheckRanges {
  int32_t n;
  int64_t off[kMaxCheckRanges], len[kMaxCheckRanges];
};
mdnn_status_t finite_check_ranges(const float* g, const CheckRanges& r, mdnn_scaler_t* scaler, hipStream_t st);
// mdnn_sgd_update without its finite check of g32 (the caller has set
// scaler->reserved for every non-finite gradient already).
mdnn_status_t sgd_update_prechecked(int64_t n, float* w32, const float* g32, float* v32, void* w_lp,
                                    mdnn_dtype_t lp_type, float lr, float momentum, mdnn_scaler_t* scaler,
                                    mdnn_stream_t stream);
// The same update over the listed ranges of the flat vectors only (one
// launch), then the scaler's state update.
mdnn_status_t sgd_update_ranges_prechecked(const CheckRanges& r, float* w32, const float* g32, float* v32,
                                           void* w_lp, mdnn_dtype_t lp_type, float lr, float momentum,
                                           mdnn_scaler_t* scaler, hipStream_t st);

}  // namespace mdnn
