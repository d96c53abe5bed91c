/*
 * mdnn.h -- C ABI of the MI355X (gfx950) hot path of a MagmaDNN-style
 * minibatch SGD step: mixed-precision dense contractions (fully connected
 * GEMMs and implicit-GEMM 2-D convolutions in forward, backward-data and
 * backward-weight form), their fused epilogues, loss, optimizer and
 * precision-conversion kernels.
 *
 * Paper: Archibald et al., "Integrating Deep Learning in Domain Sciences at
 * Exascale".  The operations follow its statement of the problem:
 *   - tensors, a compute graph of ops and backpropagation (section 2.1);
 *   - memory handling hidden from the model code (section 2.1, MemoryManager):
 *     here every buffer is owned by the caller;
 *   - convolution algorithms are swappable (section 2.1): convolution has its
 *     own entry points, separate from the GEMM;
 *   - the mixed-precision multiply-accumulate D = C + A*B with fp16 (or bf16)
 *     A, B and fp32 C, D (section 3.2);
 *   - minibatch SGD (section 3.1).
 *
 * Conventions shared by every entry point
 *   - All tensors are row-major.  Activations are [rows, features]; images are
 *     NHWC; fully connected weights are W[in, out]; convolution filters are
 *     [Cout][R][S][Cin] ("KRSC").  Convolutions have stride 1 and zero padding.
 *   - Every pointer argument is a DEVICE pointer (memory the caller allocated,
 *     e.g. through PyTorch) unless the comment says "host".  The library never
 *     allocates, frees or retains device memory; the only library-owned memory
 *     is the host-side net handle of the train-step API.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream).  Every call
 *     only enqueues work on that stream and returns without synchronising.
 *   - Every call validates its arguments on the host first and returns a
 *     status; nothing aborts.  On a non-success status nothing was launched
 *     (except MDNN_ERR_LAUNCH, which reports a failed launch), and
 *     mdnn_last_error() returns a message naming the problem.
 *   - Conditions that live in device data are data, not errors: a non-finite
 *     gradient sets the loss scaler's overflow flag; a label outside [0, C)
 *     makes that row's loss and gradient NaN.
 *   - Low-precision stores round to nearest even, keep fp16 subnormals,
 *     overflow to +-inf and keep NaN.
 *   - Functions are reentrant; calls that overlap in time on different
 *     streams must not write the same buffers.
 */
#ifndef MDNN_H
#define MDNN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  MDNN_SUCCESS = 0,
  MDNN_ERR_NULL = 1,        /* a required pointer is NULL                         */
  MDNN_ERR_SHAPE = 2,       /* a size is negative / inconsistent / too large       */
  MDNN_ERR_LAYOUT = 3,      /* unknown layout, leading dimension below the width   */
  MDNN_ERR_DTYPE = 4,       /* unsupported combination of element types            */
  MDNN_ERR_MISALIGNED = 5,  /* a base pointer is not aligned to its element size   */
  MDNN_ERR_WORKSPACE = 6,   /* workspace missing or smaller than required          */
  MDNN_ERR_LAUNCH = 7,      /* the HIP runtime reported an error                    */
  MDNN_ERR_STATE = 8        /* net handle misuse (not bound, wrong kind of layer)   */
} mdnn_status_t;

typedef enum { MDNN_F32 = 0, MDNN_F16 = 1, MDNN_BF16 = 2 } mdnn_dtype_t;

/* Operand storage of D = op(A) op(B), row-major:
 *   NN: A[M,K], B[K,N]   -- forward           Y  = X  W
 *   NT: A[M,K], B[N,K]   -- backward-data     dX = dY W^T
 *   TN: A[K,M], B[K,N]   -- backward-weight   dW = X^T dY                       */
typedef enum { MDNN_NN = 0, MDNN_NT = 1, MDNN_TN = 2 } mdnn_layout_t;

typedef enum { MDNN_ACT_NONE = 0, MDNN_ACT_RELU = 1 } mdnn_act_t;

typedef void* mdnn_stream_t; /* a hipStream_t */

/* Message of the last non-success status returned on this host thread. */
const char* mdnn_last_error(void);
/* Library version string (static). */
const char* mdnn_version(void);

/* ---------------------------------------------------------------------------
 * Mixed-precision GEMM (section 3.2: D = C + A*B, low-precision A and B,
 * fp32 accumulation), generalised to
 *     D = epi(alpha * op(A) op(B) + beta * C)
 *     epi(v) = mask( act( v + bias[n] ) )
 *     mask(v) = (mask_src[m, n] > 0) ? v : 0        (if mask_src != NULL)
 * computed in fp32 and rounded once to d_type.
 *   ab_type: MDNN_F16 or MDNN_BF16 (MFMA path) or MDNN_F32 (fp32 path, then
 *            d_type must be MDNN_F32).
 *   d_type:  MDNN_F32 or ab_type.  C (read only if beta != 0) has d_type.
 *   bias:    NULL or fp32[N].     mask_src: NULL or ab_type [M, ldm] -- the
 *            stored output of the ReLU that produced the backward-data result
 *            (a layer's input), applying the ReLU derivative [y > 0].
 *   lda/ldb/ldc/ldd/ldm are in elements and must be >= the stored row width.
 *   Any M, N, K >= 0 (M or N == 0: no-op; K == 0: D = epi(beta*C)).
 * Deterministic: the same inputs give bitwise-identical D on every call.
 * ------------------------------------------------------------------------- */
mdnn_status_t mdnn_gemm_mixed(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K,
                              float alpha, const void* A, int64_t lda, const void* B,
                              int64_t ldb, mdnn_dtype_t ab_type, float beta, const void* C,
                              int64_t ldc, void* D, int64_t ldd, mdnn_dtype_t d_type,
                              const float* bias, mdnn_act_t act, const void* mask_src,
                              int64_t ldm, mdnn_stream_t stream);

/* The same GEMM with a caller-provided device workspace (section 3.2's
 * product on shapes whose output is only a few tiles, e.g. a batch of 64 to
 * 256 rows against a narrow layer: the few workgroups' serial K loops would
 * leave most CUs idle).  When the workspace holds at least
 * mdnn_gemm_workspace(ab_type, M, N, K) bytes (16-byte aligned), such a
 * problem splits K across workgroups into fp32 partials that one more kernel
 * sums in a fixed order before the epilogue: deterministic, but the fp32
 * summation order differs from mdnn_gemm_mixed's.  A NULL / smaller /
 * misaligned workspace, or a shape that does not need splitting, gives
 * exactly mdnn_gemm_mixed.  mdnn_gemm_workspace returns 0 when no split is
 * planned (and for negative sizes).  The workspace is scratch, overwritten;
 * calls that share one must be ordered on one stream.
 * nonfinite (nullable, device int32): the dynamic loss scaler's overflow
 * test done where the gradients are produced -- every kernel path sets
 * *nonfinite = 1 (atomic OR) if any value it stores into D is Inf or NaN
 * (16-bit D: the stored value, so a finite result that rounds to Inf counts),
 * and never clears it; for mdnn_sgd_update's scaler this is
 * scaler->reserved. */
size_t mdnn_gemm_workspace(mdnn_dtype_t ab_type, int64_t M, int64_t N, int64_t K);
mdnn_status_t mdnn_gemm_mixed_ws(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K,
                                 float alpha, const void* A, int64_t lda, const void* B,
                                 int64_t ldb, mdnn_dtype_t ab_type, float beta, const void* C,
                                 int64_t ldc, void* D, int64_t ldd, mdnn_dtype_t d_type,
                                 const float* bias, mdnn_act_t act, const void* mask_src,
                                 int64_t ldm, void* workspace, size_t ws_bytes,
                                 int32_t* nonfinite, mdnn_stream_t stream);

/* Tuning knob for measurements (process-wide): force the MFMA kernel of the
 * GEMM engine.  0 = automatic (default), 1 = 256x256, 2 = 128x128, 3 = 64x64
 * general kernels (convolutions then also use the general kernels), 4 / 5 =
 * the 256x256 / 128x128 direct-to-LDS pipelined kernel wherever its
 * preconditions hold (K % 64 == 0, 16-byte aligned operands with leading
 * dimensions multiple of 8, MN-contiguous extents multiple of 8), the
 * automatic choice elsewhere (3x3 convolutions then run their implicit-GEMM
 * kernels instead of the LDS-halo kernels).  Returns 0, or -1 for an unknown
 * code.  Results do not depend on the kernel except through the fp32
 * summation order of split-K. */
int mdnn_set_gemm_tile(int code);

/* ---------------------------------------------------------------------------
 * fp32 products on the fp16 matrix cores (section 3.2, Eq. (1)).
 *
 * mdnn_split_f16: the two-term fp16 split of an fp32 matrix at a power-of-two
 * scale s,
 *   hi = RNE16(x / s),   lo = RNE16((x / s - hi) * 2^11),
 * so that x ~ s*hi + s*2^-11*lo to about 22 significant bits (the section's
 * a2 = 2^-11 a1).  x is rows x cols fp32 with leading dimension ldx; hi and lo
 * are fp16 with leading dimensions ldh, ldl (each >= cols).  |x| / s must stay
 * below 65504 (larger values give inf / NaN); values below 2^-14 * s lose bits
 * to fp16 subnormals.
 * The section gives a1 only for well-scaled data.  scale == 0 asks the
 * library to choose it on the device: s = 2^(floor(log2 max|x|) - 14), so
 * that max|x| / s lies in [2^14, 2^15) (s = 1 when max|x| is 0, Inf or NaN;
 * s >= 2^-126); the chosen s is written to the device fp32 scalar scale_out
 * (required then, ignored and may be NULL otherwise).  No host read-back.
 * Errors: MDNN_ERR_SHAPE for negative sizes or a scale that is neither 0 nor
 * a positive power of two, MDNN_ERR_NULL, MDNN_ERR_LAYOUT,
 * MDNN_ERR_MISALIGNED (x, scale_out 4-byte, hi / lo 2-byte aligned).
 */
mdnn_status_t mdnn_split_f16(int64_t rows, int64_t cols, const float* x, int64_t ldx, float scale,
                             float* scale_out, void* hi, int64_t ldh, void* lo, int64_t ldl,
                             mdnn_stream_t stream);

/* D = alpha * op(A) op(B) + beta * C for fp32 A, B, C, D through three fp16
 * MFMA products of the Eq. (1) splits of A (scale a_scale) and B (scale
 * b_scale):  a b [A1 B1 + 2^-11 (A1 B2 + A2 B1)], each accumulated in fp32
 * (the A2 B2 product, 2^-22 below the leading one, is dropped).  Layouts,
 * leading dimensions and the beta == 0 rule as mdnn_gemm_mixed; scales are
 * positive powers of two chosen so that |A| / a_scale and |B| / b_scale stay
 * below 65504 (1 for data of moderate magnitude), or 0: chosen on the device
 * by the rule of mdnn_split_f16 (the products' epilogues then read a_scale *
 * b_scale from the workspace; no host read-back).  The caller provides
 * mdnn_gemm_split3_workspace(M, N, K) bytes of 256-byte aligned device
 * workspace (the split operands, one fp32 M x N product and the scales);
 * C may alias D.
 * Four or more launches on `stream`, no host synchronisation.
 */
size_t mdnn_gemm_split3_workspace(int64_t M, int64_t N, int64_t K);
mdnn_status_t mdnn_gemm_split3(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K, float alpha,
                               const float* A, int64_t lda, float a_scale, const float* B, int64_t ldb,
                               float b_scale, float beta, const float* C, int64_t ldc, float* D,
                               int64_t ldd, void* workspace, size_t ws_bytes, mdnn_stream_t stream);

/* ---------------------------------------------------------------------------
 * 2-D convolution as implicit GEMM (section 2.1: a convolution is an
 * interchangeable algorithm behind one operation).  Stride 1, zero padding
 * `pad`, output Ho = h + 2*pad - r + 1, Wo = w + 2*pad - s + 1 (both >= 1).
 *   x  [n, h, w, c_in]        w  [c_out, r, s, c_in]      y/dy [n, Ho, Wo, c_out]
 *   fwd:        y[n,i,j,k]  = epi( sum_{r,s,c} x[n,i+r-p,j+s-p,c] * w[k,r,s,c] )
 *   bwd_data:   dx[n,h,w,c] = mask( sum_{k,r,s} dy[n,h-r+p,w-s+p,k] * w[k,r,s,c] )
 *   bwd_filter: dw[k,r,s,c] = sum_{n,i,j} dy[n,i,j,k] * x[n,i+r-p,j+s-p,c]
 *               db[k]       = sum_{n,i,j} dy[n,i,j,k]
 * io_type: MDNN_F16, MDNN_BF16 or MDNN_F32 for x, w, dy (and the mask source).
 * Accumulation is fp32; dw and db are fp32; y_type / dx_type is MDNN_F32 or
 * io_type.
 * ------------------------------------------------------------------------- */
typedef struct {
  int64_t n, h, w, c_in, c_out, r, s, pad;
} mdnn_conv_shape_t;

mdnn_status_t mdnn_conv2d_fwd(const mdnn_conv_shape_t* shape, const void* x, const void* w,
                              mdnn_dtype_t io_type, const float* bias, mdnn_act_t act, void* y,
                              mdnn_dtype_t y_type, mdnn_stream_t stream);

/* mask_src: NULL or io_type [n, h, w, c_in] (the stored, post-ReLU input of
 * the layer); where it is <= 0 the result is 0. */
mdnn_status_t mdnn_conv2d_bwd_data(const mdnn_conv_shape_t* shape, const void* dy, const void* w,
                                   mdnn_dtype_t io_type, const void* mask_src, void* dx,
                                   mdnn_dtype_t dx_type, mdnn_stream_t stream);

/* Bytes of device workspace mdnn_conv2d_bwd_filter needs for this shape
 * (fp32 split-K partial sums of dw and partial column sums of db, each
 * reduced in a fixed order); 0 on a bad shape. */
size_t mdnn_conv2d_bwd_filter_workspace(const mdnn_conv_shape_t* shape, mdnn_dtype_t io_type);

/* dw: fp32 [c_out, r, s, c_in] (overwritten).  db: NULL or fp32 [c_out]
 * (overwritten).  workspace: device memory of at least the size above,
 * 256-byte aligned (may be NULL when that size is 0).  Deterministic. */
mdnn_status_t mdnn_conv2d_bwd_filter(const mdnn_conv_shape_t* shape, const void* x, const void* dy,
                                     mdnn_dtype_t io_type, float* dw, float* db, void* workspace,
                                     size_t ws_bytes, mdnn_stream_t stream);

/* mdnn_conv2d_bwd_filter for callers that cannot allocate device memory
 * (code under HIP graph capture, serving loops, harnesses that forbid
 * hipMalloc): the same computation and result, with the workspace taken
 * from one fixed array in device memory per GPU instead of a caller buffer.
 * The array holds mdnn_conv2d_bwd_filter_noalloc_max_workspace() bytes
 * (48 MiB; every GPU the library runs on keeps it until the process ends);
 * a shape whose mdnn_conv2d_bwd_filter_workspace() exceeds that returns
 * MDNN_ERR_WORKSPACE before anything runs.  The call allocates nothing: no
 * hipMalloc, hipFree or allocating library routine.  It runs on the current
 * device's array (stream must belong to the current device).  Every call on
 * one GPU shares that GPU's array and leaves its contents behind: calls that
 * overlap on one GPU (other streams, other host threads) race and must be
 * serialised by the caller.  Nothing in the array needs to start at zero
 * (every partial sum the reduction reads is written first by the same call).
 * Other arguments and errors as mdnn_conv2d_bwd_filter. */
size_t mdnn_conv2d_bwd_filter_noalloc_max_workspace(void);
mdnn_status_t mdnn_conv2d_bwd_filter_noalloc(const mdnn_conv_shape_t* shape, const void* x, const void* dy,
                                             mdnn_dtype_t io_type, float* dw, float* db,
                                             mdnn_stream_t stream);

/* Alternative forward algorithm for 3x3 filters (section 2.1: the
 * convolution algorithm is swappable per layer): Winograd minimal filtering
 * F(2x2, 3x3) (Lavin and Gray).  Same operands, output, bias and activation
 * as mdnn_conv2d_fwd (any padding; r = s = 3), computed as
 *   U = G g G^T per (c_out, c_in), V = B^T d B per 2x2 output tile and c_in
 *   (d: the tile's 4x4 input window), M = 16 products V U^T on the matrix
 *   cores (fp32 accumulation), y = A^T M A + bias, ReLU.
 * U and V are rounded once to io_type, so the result carries one more
 * storage rounding per operand than the implicit GEMM: its error is bounded
 * by about 2u * |A^T| (sum_c |U||V|) |A| (u: io_type's unit roundoff), not by
 * the implicit GEMM's 1e-4.  io_type: fp16 or bf16 (MDNN_ERR_DTYPE for fp32);
 * MDNN_ERR_SHAPE unless r = s = 3.  workspace: at least
 * mdnn_conv2d_fwd_winograd_workspace(shape, io_type) bytes (16 * (c_out*c_in
 * + tiles*c_in) io_type elements + 16 * tiles*c_out floats, tiles =
 * n * ceil(Ho/2) * ceil(Wo/2)), 256-byte aligned, overwritten (0 for an
 * invalid shape or type).  Deterministic. */
size_t mdnn_conv2d_fwd_winograd_workspace(const mdnn_conv_shape_t* shape, mdnn_dtype_t io_type);
mdnn_status_t mdnn_conv2d_fwd_winograd(const mdnn_conv_shape_t* shape, const void* x, const void* w,
                                       mdnn_dtype_t io_type, const float* bias, mdnn_act_t act, void* y,
                                       mdnn_dtype_t y_type, void* workspace, size_t ws_bytes,
                                       mdnn_stream_t stream);

/* Forward convolution with the algorithm chosen per layer (section 2.1: the
 * convolution algorithm behind the operation is interchangeable).  Same
 * operands, output, bias and activation as mdnn_conv2d_fwd.
 *   MDNN_CONV_IMPLICIT_GEMM  mdnn_conv2d_fwd (no workspace);
 *   MDNN_CONV_IM2COL_GEMM    the im2col matrix [n*Ho*Wo][r*s*c_in] (io_type)
 *                            is written to the workspace, then one GEMM
 *                            y = col * w^T with the bias / ReLU epilogue;
 *                            same accuracy as the implicit GEMM;
 *   MDNN_CONV_WINOGRAD       mdnn_conv2d_fwd_winograd (3x3 only; its error
 *                            bound is larger than the implicit GEMM's);
 *   MDNN_CONV_AUTO           mdnn_conv2d_fwd_choose(shape, io_type, ws_bytes).
 * mdnn_conv2d_fwd_choose: the library's per-layer choice, a fixed table of
 * shapes timed on MI355X restricted to the algorithms that keep the implicit
 * GEMM's accuracy (Winograd is never chosen automatically) and to what the
 * given workspace holds; shapes not in the table run the implicit GEMM.
 * mdnn_conv2d_fwd_algo_workspace: bytes of 256-byte aligned workspace an
 * algorithm needs (0 for the implicit GEMM or a bad shape).  Errors as the
 * algorithm's own entry point; MDNN_ERR_WORKSPACE when the workspace is too
 * small; MDNN_ERR_DTYPE for an unknown algorithm. */
typedef enum {
  MDNN_CONV_AUTO = 0,
  MDNN_CONV_IMPLICIT_GEMM = 1,
  MDNN_CONV_IM2COL_GEMM = 2,
  MDNN_CONV_WINOGRAD = 3
} mdnn_conv_algo_t;
mdnn_conv_algo_t mdnn_conv2d_fwd_choose(const mdnn_conv_shape_t* shape, mdnn_dtype_t io_type, size_t ws_bytes);
size_t mdnn_conv2d_fwd_algo_workspace(const mdnn_conv_shape_t* shape, mdnn_dtype_t io_type,
                                      mdnn_conv_algo_t algo);
mdnn_status_t mdnn_conv2d_fwd_algo(const mdnn_conv_shape_t* shape, const void* x, const void* w,
                                   mdnn_dtype_t io_type, const float* bias, mdnn_act_t act, void* y,
                                   mdnn_dtype_t y_type, mdnn_conv_algo_t algo, void* workspace,
                                   size_t ws_bytes, mdnn_stream_t stream);

/* ---------------------------------------------------------------------------
 * Bias + activation epilogue as stand-alone kernels (section 2.1: a layer's
 * activation and its derivative in backpropagation).
 *   fwd: y = act(x + bias[col]) rounded to y_type;  x fp32 [rows, cols];
 *        bias NULL or fp32 [cols].
 *   bwd: dz = dy * [y > 0] (act RELU) or dy (act NONE), stored in `dtype`
 *        (dz may be NULL, may alias dy); db = column sums of dz in fp32
 *        (db may be NULL), summed in a fixed order (deterministic).
 *        dy, y, dz are `dtype` [rows, cols]; y may be NULL when act is NONE.
 *        workspace: NULL, or device memory of mdnn_bias_act_bwd_workspace()
 *        bytes (16-byte aligned) that lets db use a two-pass reduction spread
 *        over the whole GPU; without it db is summed by one pass per column
 *        group (same result, much slower for tall matrices).
 * ------------------------------------------------------------------------- */
mdnn_status_t mdnn_bias_act_fwd(int64_t rows, int64_t cols, const float* x, const float* bias,
                                mdnn_act_t act, void* y, mdnn_dtype_t y_type,
                                mdnn_stream_t stream);
size_t mdnn_bias_act_bwd_workspace(int64_t rows, int64_t cols);
mdnn_status_t mdnn_bias_act_bwd(int64_t rows, int64_t cols, const void* dy, const void* y,
                                mdnn_act_t act, void* dz, float* db, mdnn_dtype_t dtype,
                                void* workspace, size_t ws_bytes, mdnn_stream_t stream);

/* ---------------------------------------------------------------------------
 * 2x2 stride-2 max pooling, NHWC (the LeNet-style workload's pooling layers).
 * Output [n, h/2, w/2, c] (floor).  The window is scanned row-major and the
 * first maximum wins; argmax (NULL allowed in fwd) holds that window index
 * 0..3 per output element.  bwd writes every element of dx [n, h, w, c]:
 * dy at the argmax position, 0 elsewhere.
 * ------------------------------------------------------------------------- */
mdnn_status_t mdnn_maxpool2_fwd(int64_t n, int64_t h, int64_t w, int64_t c, const void* x,
                                void* y, uint8_t* argmax, mdnn_dtype_t dtype,
                                mdnn_stream_t stream);
mdnn_status_t mdnn_maxpool2_bwd(int64_t n, int64_t h, int64_t w, int64_t c, const void* dy,
                                const uint8_t* argmax, void* dx, mdnn_dtype_t dtype,
                                mdnn_stream_t stream);

/* ---------------------------------------------------------------------------
 * Losses, mean over the batch.  S = *loss_scale (device fp32; NULL means 1).
 * softmax_xent: logits fp32 [B, C] (row stride ldl >= C), labels int32 [B];
 *   *loss_out = -(1/B) sum_i log_softmax(z_i)[label_i]   (unscaled, fp32)
 *   dlogits[i, j] = S * (softmax(z_i)_j - [j == label_i]) / B  in dlogits_type,
 *   row stride ldd >= C.  C <= 1024.
 * mse_loss: y, t fp32 [B, O] (contiguous);
 *   *loss_out = (1/B) sum (y - t)^2 ;   dy = S * 2 (y - t) / B  in dy_type.
 * Sums are taken in a fixed order (deterministic).
 * ------------------------------------------------------------------------- */
mdnn_status_t mdnn_softmax_xent(int64_t B, int64_t C, const float* logits, int64_t ldl,
                                const int32_t* labels, const float* loss_scale, float* loss_out,
                                void* dlogits, int64_t ldd, mdnn_dtype_t dlogits_type,
                                mdnn_stream_t stream);
mdnn_status_t mdnn_mse_loss(int64_t B, int64_t O, const float* y, const float* t,
                            const float* loss_scale, float* loss_out, void* dy,
                            mdnn_dtype_t dy_type, mdnn_stream_t stream);

/* ---------------------------------------------------------------------------
 * SGD update (section 3.1) on the flat fp32 master parameters, with optional
 * heavy-ball momentum and dynamic loss scaling, then the low-precision
 * working copy:
 *   if scaler: overflow = any(!isfinite(g));  on overflow the update is skipped
 *              (w, v, w_lp untouched), scale = max(scale*backoff, min_scale),
 *              good_steps = 0;  otherwise g /= scale and, after the update,
 *              ++good_steps == growth_interval -> scale *= growth, good_steps = 0.
 *   v = momentum*v + g; w -= lr*v        (v != NULL)
 *   w -= lr*g                            (v == NULL)
 *   w_lp = RNE(w)                        (w_lp != NULL, lp_type F16/BF16/F32)
 * The scaler lives in device memory; its overflow field is written by the
 * call (1 when the step was skipped).  With a scaler the call enqueues three
 * kernels (finite check, update, scaler state update), otherwise one.
 * Pointers need only their element alignment (fp32: 4 bytes); when w32, g32,
 * v32 are 16-byte aligned and w_lp 4-element aligned the passes use 16-byte
 * vectors, otherwise one element per thread (same arithmetic).
 * Errors: MDNN_ERR_SHAPE (n < 0), MDNN_ERR_DTYPE, MDNN_ERR_NULL (w32 / g32
 * missing with n > 0), MDNN_ERR_MISALIGNED (a pointer below its element
 * alignment), MDNN_ERR_LAUNCH.
 * ------------------------------------------------------------------------- */
typedef struct {
  float scale;
  int32_t good_steps;
  int32_t overflow;
  int32_t growth_interval;
  float growth;
  float backoff;
  float min_scale;
  int32_t reserved;  /* internal pending-overflow flag: initialise to 0; every
                        mdnn_sgd_update call leaves it 0 again */
} mdnn_scaler_t;

mdnn_status_t mdnn_sgd_update(int64_t n, float* w32, const float* g32, float* v32, void* w_lp,
                              mdnn_dtype_t lp_type, float lr, float momentum,
                              mdnn_scaler_t* scaler, mdnn_stream_t stream);

/* Asynchronous variant (section 3.1: asynchronous SGD with lock-free updates
 * of a shared parameter vector): the same check and state machine, but the
 * step -lr*v (or -lr*g) is added to w32 with fp32 atomics, so several streams
 * may update one w32 concurrently without losing updates; no working copy is
 * written.  The order of concurrent updates (hence the rounding of w32) is
 * not deterministic.  v32 and the scaler belong to the caller of this update
 * (one per worker).  Pointers need only 4-byte alignment. */
mdnn_status_t mdnn_sgd_update_async(int64_t n, float* w32, const float* g32, float* v32, float lr,
                                    float momentum, mdnn_scaler_t* scaler, mdnn_stream_t stream);

/* Weight-gradient product with the SGD update applied where it is produced
 * (section 3.1's update of the fp32 master weights, section 3.2's mixed
 * precision): G = A^T B in the TN layout of mdnn_gemm_mixed (A [K][M] with
 * lda >= M, B [K][N] with ldb >= N, ab_type F16 or BF16, fp32 accumulation)
 * is not stored; element (m, n) of G updates w32[m*ldw + n], v32[m*ldw + n]
 * and w_lp[m*ldw + n] exactly as mdnn_sgd_update does with g = G[m][n]
 * (bit for bit: g / scale with a scaler, v = momentum*v + g, w -= lr*v, or
 * w -= lr*g when momentum is 0, w_lp = RNE(w) in ab_type).  scaler
 * (nullable) is only read: when scaler->reserved is set nothing is updated.
 * G itself is not tested for Inf / NaN, so a loss-scaled caller must have
 * set reserved for every non-finite operand value before the call (with
 * finite fp16 operands the fp32 product is finite for any K below 2^96; the
 * train step tests the stored activations and output gradients; bf16
 * operands carry no such bound).  The scaler's state is not advanced (the
 * update of the remaining parameters does that).
 * Shapes: M and N positive multiples of 256, K a positive multiple of 64,
 * M * N at least 32 tiles of 128 x 128; A, B 16-byte aligned with lda, ldb
 * multiples of 8; w32 (and v32) 16-byte aligned, w_lp 8-byte aligned
 * (nullable: no working copy), ldw >= N a multiple of 4; v32 required when
 * momentum != 0.  The product takes the pipelined kernel of mdnn_gemm_mixed
 * (same tiles, no K split), every tile interior.
 * Errors: MDNN_ERR_DTYPE (F32 or unknown ab_type), MDNN_ERR_NULL,
 * MDNN_ERR_SHAPE (sizes, or operands the pipelined kernel does not take),
 * MDNN_ERR_LAYOUT (a leading dimension too small), MDNN_ERR_MISALIGNED,
 * MDNN_ERR_LAUNCH. */
mdnn_status_t mdnn_gemm_tn_update(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                                  const void* B, int64_t ldb, mdnn_dtype_t ab_type, float* w32,
                                  float* v32, void* w_lp, int64_t ldw, float lr, float momentum,
                                  const mdnn_scaler_t* scaler, mdnn_stream_t stream);

/* ---------------------------------------------------------------------------
 * Precision conversion (section 3.2: fp32 data stored as fp16 or bf16).
 * dst[i] = convert(src[i]) for i < n, round to nearest even.
 * ------------------------------------------------------------------------- */
mdnn_status_t mdnn_cast(int64_t n, const void* src, mdnn_dtype_t src_type, void* dst,
                        mdnn_dtype_t dst_type, mdnn_stream_t stream);

/* ---------------------------------------------------------------------------
 * Train step of a fixed layer chain (section 2.1 compute graph, fixed here;
 * section 3.1 minibatch SGD).  One call = forward, loss, backpropagation and
 * update of one minibatch, all enqueued on one stream with no host sync.
 *
 * Layer chain: FC (in=c_in, out=c_out), CONV (input [h, w, c_in], c_out
 * filters r x s, pad; output "same" size required: 2*pad == r-1 == s-1),
 * MAXPOOL2 (input [h, w, c_in], output [h/2, w/2, c_in], h and w even).
 * act applies to FC / CONV.  The last layer must be FC or CONV with act NONE.
 * Storage (section 3.2): activations, working weights and activation
 * gradients in cfg.dtype; accumulation, bias, logits / outputs, weight
 * gradients, master weights and momentum in fp32.
 * Flat parameter packing: per layer in order, weights then bias.
 * ------------------------------------------------------------------------- */
typedef enum { MDNN_LAYER_FC = 0, MDNN_LAYER_CONV = 1, MDNN_LAYER_MAXPOOL2 = 2 } mdnn_layer_kind_t;
typedef enum { MDNN_LOSS_XENT = 0, MDNN_LOSS_MSE = 1 } mdnn_loss_t;

typedef struct {
  int32_t kind;   /* mdnn_layer_kind_t */
  int32_t act;    /* mdnn_act_t        */
  int64_t c_in, h, w, c_out, r, s, pad;
} mdnn_layer_t;

typedef struct {
  int32_t dtype;        /* mdnn_dtype_t storage type                          */
  int32_t loss;         /* mdnn_loss_t                                         */
  float lr;
  float momentum;       /* 0: plain SGD (momentum buffer may be NULL)          */
  int32_t loss_scaling; /* nonzero: dynamic loss scaling via the bound scaler  */
  int32_t n_classes;    /* cross-entropy classes (= last layer's outputs)      */
  int32_t fuse_update;  /* nonzero: FC layers whose weight
                           gradient fits mdnn_gemm_tn_update (in and out
                           multiples of 256, batch a multiple of 64, 16-bit
                           storage; fp16 when the loss is scaled; buffers
                           aligned as that call needs) and is not split
                           over K in the unfused step are updated inside
                           that product, after the whole backward pass: the
                           same results bit for bit, without storing and
                           re-reading their fp32 weight gradients          */
} mdnn_train_cfg_t;

typedef struct mdnn_net mdnn_net_t;

/* Validate the chain and create a host-side handle (host memory only). */
mdnn_status_t mdnn_net_create(const mdnn_layer_t* layers, int32_t n_layers, int64_t batch,
                              const mdnn_train_cfg_t* cfg, mdnn_net_t** net);
/* Host outputs: number of parameters and bytes of workspace to bind. */
mdnn_status_t mdnn_net_sizes(const mdnn_net_t* net, int64_t* n_params, size_t* workspace_bytes);
/* Bind caller-owned device memory: master_w fp32[n_params] (initialised by the
 * caller), grads fp32[n_params], momentum fp32[n_params] (NULL iff momentum
 * is 0; caller zeroes it), lowp_w cfg.dtype[n_params] (NULL for fp32 nets;
 * filled by mdnn_net_sync_lowp), workspace (>= workspace_bytes, 256-byte
 * aligned), scaler (NULL iff loss scaling is off; caller initialises it).
 * The parameter buffers need only their element alignment (4 bytes; lowp_w
 * 2 bytes); each kernel of the step picks its vector or element-wise form
 * from the alignment it is given.  MDNN_ERR_MISALIGNED otherwise, or for a
 * workspace that is not 256-byte aligned. */
mdnn_status_t mdnn_net_bind(mdnn_net_t* net, float* master_w, float* grads, float* momentum,
                            void* lowp_w, void* workspace, size_t workspace_bytes,
                            mdnn_scaler_t* scaler);
/* Recompute the working low-precision weights from the master weights
 * (call once after initialising master_w). */
mdnn_status_t mdnn_net_sync_lowp(mdnn_net_t* net, mdnn_stream_t stream);
/* One SGD step.  x: fp32 [batch, in_features] (NHWC-flattened images);
 * target: int32 labels [batch] (XENT) or fp32 [batch, out] (MSE);
 * loss_out: device fp32 scalar, the unscaled loss of this step's forward pass.
 * With loss scaling the update is skipped when any gradient is Inf or NaN,
 * as in mdnn_sgd_update; the step tests the gradients where it produces
 * them (GEMM epilogues, the bias column sums) plus one pass over the ranges
 * no such producer covers, instead of a second pass over all gradients.
 * grads holds this step's scaled gradients afterwards, except the weight
 * gradients of layers fused by cfg.fuse_update (never stored). */
mdnn_status_t mdnn_train_step(mdnn_net_t* net, const float* x, const void* target,
                              float* loss_out, mdnn_stream_t stream);
/* Asynchronous step (section 3.1): for several nets bound to the same
 * master_w (each with its own grads, momentum, lowp_w, workspace and scaler)
 * stepping concurrently on different streams.  The step first re-derives its
 * working copy from the shared master weights (fp32 nets read them directly),
 * runs forward, loss and backward, then adds its update to the shared
 * weights with mdnn_sgd_update_async.  Reads may see other workers' updates
 * part-applied and gradients may be stale: results are not deterministic,
 * by design.  A net sharing master_w must only use this step. */
mdnn_status_t mdnn_train_step_async(mdnn_net_t* net, const float* x, const void* target,
                                    float* loss_out, mdnn_stream_t stream);
/* Device pointer of stored activation i (0 = the low-precision input, i = output
 * of layer i-1) inside the bound workspace, for inspection; NULL if invalid. */
const void* mdnn_net_activation(const mdnn_net_t* net, int32_t i);
/* Device pointer of one of the two buffers (which = 0 or 1) that hold the
 * output gradients of the backward pass (the low-precision storage type,
 * batch x features of the layer), for inspection; NULL if invalid.  The
 * loss gradient (last layer, L - 1) goes to buffer 0 and each layer's input
 * gradient to the other buffer, so the gradient with respect to the output
 * of layer i is in buffer (L - 1 - i) % 2; after a step the buffers hold
 * those of layers 0 and 1 (the last two written).  With cfg.fuse_update the
 * gradient of a fused layer's output is in a workspace buffer of its own
 * instead (the rule holds for the other layers). */
const void* mdnn_net_output_grad(const mdnn_net_t* net, int32_t which);
void mdnn_net_destroy(mdnn_net_t* net);

/* Recorded steps.  Section 3.1's SGD step for a small network is a few
 * dozen short kernels, so its time is set by launch latency: these calls
 * record one mdnn_train_step (forward, loss, backward, update; the same
 * kernels in the same order) into a HIP graph once, and replay it with a
 * single launch.
 *   mdnn_train_graph_create: records the step of `net` on the buffers x,
 *     target and loss_out exactly as mdnn_train_step would run it; nothing
 *     executes.  The graph keeps those device addresses and the net's bound
 *     memory: they must stay allocated, unmoved, for the graph's lifetime (to
 *     feed new data, write it into the same x / target buffers first).  The
 *     recording happens on a private stream; the caller's streams are not
 *     touched.  *out receives a library-owned handle (a host object plus the
 *     HIP runtime's instantiated graph).  Errors: those of mdnn_train_step
 *     (the step is validated while it is recorded) and MDNN_ERR_LAUNCH if the
 *     runtime refuses the capture; *out is NULL then.
 *   mdnn_graph_launch: enqueues one replay on `stream` (any stream, the
 *     legacy default included); replays on one stream run in order.  The
 *     result equals mdnn_train_step's on the same inputs, bit for bit.
 *   mdnn_graph_destroy: releases the handle (NULL is ignored).  Pending
 *     replays must have finished. */
typedef struct mdnn_graph mdnn_graph_t;
mdnn_status_t mdnn_train_graph_create(mdnn_net_t* net, const float* x, const void* target,
                                      float* loss_out, mdnn_graph_t** out);
mdnn_status_t mdnn_graph_launch(mdnn_graph_t* graph, mdnn_stream_t stream);
void mdnn_graph_destroy(mdnn_graph_t* graph);

#ifdef __cplusplus
}
#endif
#endif /* MDNN_H */
