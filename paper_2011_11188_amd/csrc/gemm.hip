// mdnn_gemm_mixed: validation and dispatch of the GEMM engine; fixed-order
// reductions shared with the other entry points.
#include <atomic>

#include "gemm_launch.h"
#include "gemm_skinny.h"

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

// Few outputs, many splits: a block of 1024 threads sums OPB outputs with
// G = 1024 / OPB split groups.  Thread (g, j) sums splits g, g+G, g+2G, ...
// of output j into four interleaved accumulators (four loads in flight),
// adds them in order, and the G group sums are combined by a fixed tree in
// LDS: a fixed order, so the result is deterministic.  `red` holds 1024
// floats; `blk` is the block's index within its reduction.
template <int OPB>
__device__ __forceinline__ void reduce_wide_block(const float* __restrict__ part, int splits, int64_t n,
                                                  float* __restrict__ out, int64_t blk, float* red) {
  constexpr int G = 1024 / OPB;
  const int j = threadIdx.x % OPB, g = threadIdx.x / OPB;
  const int64_t e = blk * OPB + j;
  float s0 = 0.0f, s1 = 0.0f, s2 = 0.0f, s3 = 0.0f;
  if (e < n) {
    int k = g;
    for (; k + 3 * G < splits; k += 4 * G) {
      s0 += part[(int64_t)k * n + e];
      s1 += part[(int64_t)(k + G) * n + e];
      s2 += part[(int64_t)(k + 2 * G) * n + e];
      s3 += part[(int64_t)(k + 3 * G) * n + e];
    }
    for (; k < splits; k += G) s0 += part[(int64_t)k * n + e];
  }
  red[g * OPB + j] = (s0 + s1) + (s2 + s3);
  __syncthreads();
#pragma unroll
  for (int h = G / 2; h > 0; h >>= 1) {
    if (g < h) red[g * OPB + j] += red[(g + h) * OPB + j];
    __syncthreads();
  }
  if (g == 0 && e < n) out[e] = red[j];
}

template <int OPB>
__global__ void __launch_bounds__(1024)
reduce_splits_wide_kernel(const float* __restrict__ part, int splits, int64_t n, float* __restrict__ out) {
  __shared__ float red[1024];
  reduce_wide_block<OPB>(part, splits, n, out, blockIdx.x, red);
}

// Several wide reductions in one launch: block b works on the reduction s
// with first_block[s] <= b < first_block[s + 1], with that reduction's
// outputs per block -- the same sums, in the same order, as its own launch.
__global__ void __launch_bounds__(1024) reduce_batch_kernel(ReduceBatch b) {
  __shared__ float red[1024];
  int s = 0;
  while (s + 1 < b.n && (int64_t)blockIdx.x >= b.first_block[s + 1]) ++s;
  const int64_t blk = (int64_t)blockIdx.x - b.first_block[s];
  if (b.opb[s] == 16)
    reduce_wide_block<16>(b.part[s], b.splits[s], b.elems[s], b.out[s], blk, red);
  else
    reduce_wide_block<64>(b.part[s], b.splits[s], b.elems[s], b.out[s], blk, red);
}

static mdnn_status_t reduce_wide(const float* partial, int splits, int64_t n, float* out, hipStream_t stream,
                                 ReduceBatch* defer);

mdnn_status_t reduce_batch_launch(ReduceBatch& b, hipStream_t stream) {
  if (b.n == 0) return MDNN_SUCCESS;
  const ReduceBatch todo = b;
  b.n = 0;
  if (todo.n == 1) return reduce_wide(todo.part[0], todo.splits[0], todo.elems[0], todo.out[0], stream, nullptr);
  const int64_t blocks = todo.first_block[todo.n];
  if (blocks > 0x7fffffffLL) return fail(MDNN_ERR_SHAPE, "split reductions: too many blocks");
  hipLaunchKernelGGL(reduce_batch_kernel, dim3((unsigned)blocks), dim3(1024), 0, stream, todo);
  return check_launch("reduce_batch_kernel");
}

static mdnn_status_t reduce_wide(const float* partial, int splits, int64_t n, float* out, hipStream_t stream,
                                 ReduceBatch* defer) {
  // up to 1024 outputs: 16 per block, 64 split groups (a 64-column bias sum
  // over 512 row chunks: 8 partials per thread in 4 blocks, not 32 in one)
  const int opb = n <= 1024 ? 16 : 64;
  if (defer) {
    if (defer->n == kMaxReduceBatch) MDNN_TRY(reduce_batch_launch(*defer, stream));
    const int s = defer->n++;
    if (s == 0) defer->first_block[0] = 0;
    defer->part[s] = partial;
    defer->out[s] = out;
    defer->elems[s] = n;
    defer->splits[s] = splits;
    defer->opb[s] = opb;
    defer->first_block[s + 1] = defer->first_block[s] + ceil_div(n, (int64_t)opb);
    return MDNN_SUCCESS;
  }
  const dim3 grid((unsigned)ceil_div(n, (int64_t)opb));
  if (opb == 16)
    hipLaunchKernelGGL(reduce_splits_wide_kernel<16>, grid, dim3(1024), 0, stream, partial, splits, n, out);
  else
    hipLaunchKernelGGL(reduce_splits_wide_kernel<64>, grid, dim3(1024), 0, stream, partial, splits, n, out);
  return check_launch("reduce_splits_wide_kernel");
}

mdnn_status_t reduce_splits(const float* partial, int splits, int64_t rows, int64_t cols,
                            float* out, hipStream_t stream, ReduceBatch* defer) {
  const int64_t n = rows * cols;
  if (n == 0) return MDNN_SUCCESS;
  if (splits >= 32 && n <= ((int64_t)1 << 18)) return reduce_wide(partial, splits, n, out, stream, defer);
  const int64_t blocks = ceil_div(ceil_div(n, 4), 256);
  hipLaunchKernelGGL(reduce_splits_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, partial,
                     splits, n, out);
  return check_launch("reduce_splits_kernel");
}

// Column sums of a [rows, cols] matrix (optionally masked by [y > 0]), in a
// fixed order so the result is bitwise reproducible.
//
// With a workspace (two passes): pass 1 splits the rows into chunks of
// COLSUM_ROWS; a block reduces one chunk x 64 columns (8 column groups of 8
// read as 16-byte vectors, 32 row lanes, then a fixed-order combine in LDS)
// into partial[chunk][col].  Pass 2 sums the partials of each column with
// the split reduction below (many chunks) or 8 strided lanes per column (few
// chunks), each combined in a fixed order.
// Without a workspace: one block per 32 columns walks all rows (slow for very
// tall matrices; kept for callers that cannot provide memory).
constexpr int64_t COLSUM_ROWS = 256;

template <class T>
__device__ __forceinline__ float masked_val(const typename T::storage* x, const typename T::storage* y,
                                            int64_t i) {
  return (y == nullptr || to_f<T>(y[i]) > 0.0f) ? to_f<T>(x[i]) : 0.0f;
}

template <class T>
__global__ void __launch_bounds__(256)
colsum_partial_kernel(const typename T::storage* __restrict__ x, const typename T::storage* __restrict__ y,
                      int64_t rows, int64_t cols, bool vec, float* __restrict__ partial) {
  __shared__ float red[32][65];
  const int cg = threadIdx.x & 7, rl = threadIdx.x >> 3;
  const int64_t c0 = (int64_t)blockIdx.x * 64 + cg * 8;
  const int64_t r0 = (int64_t)blockIdx.y * COLSUM_ROWS;
  const int64_t r1 = r0 + COLSUM_ROWS < rows ? r0 + COLSUM_ROWS : rows;
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  // adds one row's 8 values (16 bytes of x, and of the mask y) to s
  auto add8 = [&](const uint4& v, const uint4& m) {
    const uint32_t vw[4] = {v.x, v.y, v.z, v.w};
    const uint32_t mw[4] = {m.x, m.y, m.z, m.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint16_t xv = (uint16_t)(vw[e >> 1] >> ((e & 1) * 16));
      const uint16_t yv = (uint16_t)(mw[e >> 1] >> ((e & 1) * 16));
      if (y == nullptr || to_f<T>((typename T::storage)yv) > 0.0f) s[e] += to_f<T>((typename T::storage)xv);
    }
  };
  const uint4 ones = make_uint4(0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu);
  if (vec && sizeof(typename T::storage) == 2 && c0 + 8 <= cols && r1 - r0 == COLSUM_ROWS) {
    // a whole chunk: all of this thread's rows are loaded before any is added
    // (same order of additions as the row loop below)
    constexpr int RPT = COLSUM_ROWS / 32;
    uint4 v[RPT], m[RPT];
#pragma unroll
    for (int u = 0; u < RPT; ++u) v[u] = *(const uint4*)(x + (r0 + rl + 32 * u) * cols + c0);
#pragma unroll
    for (int u = 0; u < RPT; ++u) m[u] = y ? *(const uint4*)(y + (r0 + rl + 32 * u) * cols + c0) : ones;
#pragma unroll
    for (int u = 0; u < RPT; ++u) add8(v[u], m[u]);
  } else if (vec && sizeof(typename T::storage) == 2 && c0 + 8 <= cols) {
    for (int64_t r = r0 + rl; r < r1; r += 32)
      add8(*(const uint4*)(x + r * cols + c0), y ? *(const uint4*)(y + r * cols + c0) : ones);
  } else {
    for (int64_t r = r0 + rl; r < r1; r += 32)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (c0 + e < cols) s[e] += masked_val<T>(x, y, r * cols + c0 + e);
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) red[rl][cg * 8 + e] = s[e];
  __syncthreads();
  if (threadIdx.x < 64) {
    const int64_t c = (int64_t)blockIdx.x * 64 + threadIdx.x;
    float t = red[0][threadIdx.x];
    for (int k = 1; k < 32; ++k) t += red[k][threadIdx.x];
    if (c < cols) partial[(int64_t)blockIdx.y * cols + c] = t;
  }
}

// Pass 1 of the split API for 16-bit rows whose width is a multiple of 512
// (the train step's bias gradients): chunks of COLSUM_STRIP_ROWS rows; a
// block reduces one chunk x 512 columns, each wave reading whole 1 KB runs
// of its rows (wave w: rows w, w + 4, ...; 8 columns per lane), then the
// four waves' sums are combined in a fixed order.
constexpr int64_t COLSUM_STRIP_ROWS = 64;
static bool colsum_strip(mdnn_dtype_t t, int64_t cols) { return t != MDNN_F32 && cols % 512 == 0; }

// block (bx, by): columns bx * 512 .. + 511 of row chunk by
template <class T>
__device__ __forceinline__ void colsum_strip_block(const uint16_t* __restrict__ x, int64_t rows, int64_t cols,
                                                   float* __restrict__ partial, int64_t bx, int64_t by) {
  __shared__ float4 red[4][2][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t c0 = bx * 512 + lane * 8;
  const int64_t r0 = by * COLSUM_STRIP_ROWS;
  const int64_t nr = rows - r0 < COLSUM_STRIP_ROWS ? rows - r0 : COLSUM_STRIP_ROWS;
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  auto add8 = [&](const uint4& v) {
    const uint32_t vw[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] += to_f<T>((uint16_t)(vw[e >> 1] >> ((e & 1) * 16)));
  };
  const uint16_t* base = x + (r0 + w) * cols + c0;
  if (nr == COLSUM_STRIP_ROWS) {
    // a whole chunk: all of this lane's rows are loaded before any is added
    constexpr int RPW = COLSUM_STRIP_ROWS / 4;
    uint4 v[RPW];
#pragma unroll
    for (int u = 0; u < RPW; ++u) v[u] = *(const uint4*)(base + (int64_t)(4 * u) * cols);
#pragma unroll
    for (int u = 0; u < RPW; ++u) add8(v[u]);
  } else {
    for (int64_t r = w; r < nr; r += 4) add8(*(const uint4*)(base + (r - w) * cols));
  }
  red[w][0][lane] = make_float4(s[0], s[1], s[2], s[3]);
  red[w][1][lane] = make_float4(s[4], s[5], s[6], s[7]);
  __syncthreads();
  // thread t: columns 2t and 2t + 1 of the block's 512 (lane t / 4's values)
  const int l = threadIdx.x >> 2, h = (threadIdx.x >> 1) & 1, q = threadIdx.x & 1;
  float2 t = make_float2(0.f, 0.f);
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const float4 v = red[k][h][l];
    t.x += q ? v.z : v.x;
    t.y += q ? v.w : v.y;
  }
  *(float2*)(partial + by * cols + bx * 512 + 2 * threadIdx.x) = t;
}

template <class T>
__global__ void __launch_bounds__(256)
colsum_strip_kernel(const uint16_t* __restrict__ x, int64_t rows, int64_t cols, float* __restrict__ partial) {
  colsum_strip_block<T>(x, rows, cols, partial, blockIdx.x, blockIdx.y);
}

// several matrices of the same height in one launch (grid z = matrix); the
// blocks of each are those of colsum_strip_kernel, so the partials are the same
template <class T>
__global__ void __launch_bounds__(256) colsum_strip_batch_kernel(StripBatch b, int64_t rows) {
  const int i = blockIdx.z;
  if ((int64_t)blockIdx.x * 512 >= b.cols[i]) return;  // the whole block: narrower than the widest
  colsum_strip_block<T>(b.x[i], rows, b.cols[i], b.partial[i], blockIdx.x, blockIdx.y);
}

// sum of partial[k][c] over k = ln, ln + 8, ... < chunks, in that order,
// eight loads in flight at a time
__device__ __forceinline__ float strided_sum8(const float* __restrict__ partial, int64_t chunks, int64_t cols,
                                              int64_t c, int ln) {
  float s = 0.0f;
  int64_t k = ln;
  for (; k + 56 < chunks; k += 64) {
    float v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = partial[(k + 8 * u) * cols + c];
#pragma unroll
    for (int u = 0; u < 8; ++u) s += v[u];
  }
  for (; k < chunks; k += 8) s += partial[k * cols + c];
  return s;
}

__global__ void __launch_bounds__(256)
colsum_final_kernel(const float* __restrict__ partial, int64_t chunks, int64_t cols,
                    float* __restrict__ out) {
  __shared__ float red[8][33];
  const int cx = threadIdx.x & 31, ln = threadIdx.x >> 5;
  const int64_t c = (int64_t)blockIdx.x * 32 + cx;
  float s = 0.0f;
  if (c < cols) s = strided_sum8(partial, chunks, cols, c, ln);
  red[ln][cx] = s;
  __syncthreads();
  if (ln == 0 && c < cols) {
    float t = red[0][cx];
#pragma unroll
    for (int k = 1; k < 8; ++k) t += red[k][cx];
    out[c] = t;
  }
}

// colsum_final_kernel over a batch of matrices (block row y = entry y), with
// the loss scaler's overflow flag on the stored sums.
__global__ void __launch_bounds__(256)
colsum_final_batch_kernel(ColsumBatch b, int32_t* __restrict__ nonfinite) {
  __shared__ float red[8][33];
  const int cx = threadIdx.x & 31, ln = threadIdx.x >> 5;
  const int64_t cols = b.cols[blockIdx.y], chunks = b.chunks[blockIdx.y];
  const float* __restrict__ partial = b.part[blockIdx.y];
  const int64_t c = (int64_t)blockIdx.x * 32 + cx;
  float s = 0.0f;
  if (c < cols) s = strided_sum8(partial, chunks, cols, c, ln);
  red[ln][cx] = s;
  __syncthreads();
  if (ln == 0 && c < cols) {
    float t = red[0][cx];
#pragma unroll
    for (int k = 1; k < 8; ++k) t += red[k][cx];
    b.out[blockIdx.y][c] = t;
    if (nonfinite && !isfinite(t)) atomicOr(nonfinite, 1);
  }
}

template <class T>
__global__ void __launch_bounds__(256)
colsum_single_kernel(const typename T::storage* __restrict__ x, const typename T::storage* __restrict__ y,
                     int64_t rows, int64_t cols, float* __restrict__ out) {
  __shared__ float part[8][33];
  const int cx = threadIdx.x & 31, ry = threadIdx.x >> 5;
  const int64_t col = (int64_t)blockIdx.x * 32 + cx;
  float s = 0.0f;
  if (col < cols) {
    int64_t r = ry;
    // eight of this thread's rows in flight, added in row order (a load per
    // dependent add had left the kernel waiting on memory once per row)
    for (; r + 56 < rows; r += 64) {
      float v[8], keep[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int64_t i = (r + 8 * u) * cols + col;
        v[u] = to_f<T>(x[i]);
        keep[u] = y ? to_f<T>(y[i]) : 1.0f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) s += keep[u] > 0.0f ? v[u] : 0.0f;
    }
    for (; r < rows; r += 8) s += masked_val<T>(x, y, r * cols + col);
  }
  part[ry][cx] = s;
  __syncthreads();
  if (ry == 0 && col < cols) {
    float t = part[0][cx];
#pragma unroll
    for (int k = 1; k < 8; ++k) t += part[k][cx];
    out[col] = t;
  }
}

size_t column_sums_ws_bytes(int64_t rows, int64_t cols) {
  if (rows <= COLSUM_ROWS) return 0;
  return (size_t)ceil_div(rows, COLSUM_ROWS) * (size_t)cols * sizeof(float);
}

template <class T>
static mdnn_status_t colsum_launch(const void* x, const void* y, int64_t rows, int64_t cols, float* out,
                                   void* ws, size_t ws_bytes, hipStream_t st, ReduceBatch* defer) {
  typedef typename T::storage S;
  const size_t need = column_sums_ws_bytes(rows, cols);
  const bool vec = aligned(x, 16) && (!y || aligned(y, 16)) && cols % 8 == 0;
  if (rows <= COLSUM_ROWS) {
    // one chunk: pass 1 alone gives the sums (its 16-byte row reads keep
    // more loads in flight than the single-pass kernel)
    hipLaunchKernelGGL(colsum_partial_kernel<T>, dim3((unsigned)ceil_div(cols, 64), 1u), dim3(256), 0, st,
                       (const S*)x, (const S*)y, rows, cols, vec, out);
  } else if (need > 0 && ws && ws_bytes >= need && aligned(ws, 4)) {
    const int64_t chunks = ceil_div(rows, COLSUM_ROWS);
    hipLaunchKernelGGL(colsum_partial_kernel<T>, dim3((unsigned)ceil_div(cols, 64), (unsigned)chunks), dim3(256),
                       0, st, (const S*)x, (const S*)y, rows, cols, vec, (float*)ws);
    MDNN_TRY(check_launch("column sums (partials)"));
    if (chunks >= 32 && cols <= ((int64_t)1 << 18))
      return reduce_wide((const float*)ws, (int)chunks, cols, out, st, defer);
    hipLaunchKernelGGL(colsum_final_kernel, dim3((unsigned)ceil_div(cols, 32)), dim3(256), 0, st,
                       (const float*)ws, chunks, cols, out);
  } else {
    hipLaunchKernelGGL(colsum_single_kernel<T>, dim3((unsigned)ceil_div(cols, 32)), dim3(256), 0, st,
                       (const S*)x, (const S*)y, rows, cols, out);
  }
  return check_launch("column sums");
}

mdnn_status_t column_sums(const void* x, const void* y, mdnn_dtype_t t, int64_t rows, int64_t cols,
                          float* out, void* ws, size_t ws_bytes, hipStream_t stream, ReduceBatch* defer) {
  if (cols == 0) return MDNN_SUCCESS;
  if (ceil_div(rows, COLSUM_ROWS) > 65535) ws = nullptr;  // grid limit: single pass
  switch (t) {
    case MDNN_F32: return colsum_launch<F32>(x, y, rows, cols, out, ws, ws_bytes, stream, defer);
    case MDNN_F16: return colsum_launch<F16>(x, y, rows, cols, out, ws, ws_bytes, stream, defer);
    default: return colsum_launch<BF16>(x, y, rows, cols, out, ws, ws_bytes, stream, defer);
  }
}

int64_t column_sums_chunks(int64_t rows, int64_t cols, mdnn_dtype_t t) {
  return ceil_div(rows, colsum_strip(t, cols) ? COLSUM_STRIP_ROWS : COLSUM_ROWS);
}

mdnn_status_t column_sums_partial(const void* x, mdnn_dtype_t t, int64_t rows, int64_t cols, float* partial,
                                  hipStream_t st) {
  const int64_t chunks = column_sums_chunks(rows, cols, t);
  if (cols == 0 || chunks == 0) return MDNN_SUCCESS;
  if (chunks > 65535 || ceil_div(cols, 64) > 0x7fffffffLL) return fail(MDNN_ERR_SHAPE, "column sums: too many rows");
  if (colsum_strip(t, cols)) {
    if (!aligned(x, 16) || !aligned(partial, 8))
      return fail(MDNN_ERR_MISALIGNED, "column sums: rows of 512k 16-bit columns need 16-byte alignment");
    const dim3 sgrid((unsigned)(cols / 512), (unsigned)chunks);
    if (t == MDNN_F16)
      hipLaunchKernelGGL(colsum_strip_kernel<F16>, sgrid, dim3(256), 0, st, (const uint16_t*)x, rows, cols, partial);
    else
      hipLaunchKernelGGL(colsum_strip_kernel<BF16>, sgrid, dim3(256), 0, st, (const uint16_t*)x, rows, cols, partial);
    return check_launch("column sums (partials)");
  }
  const dim3 grid((unsigned)ceil_div(cols, 64), (unsigned)chunks);
  const bool vec = aligned(x, 16) && cols % 8 == 0;
  switch (t) {
    case MDNN_F32:
      hipLaunchKernelGGL(colsum_partial_kernel<F32>, grid, dim3(256), 0, st, (const float*)x, nullptr, rows, cols,
                         vec, partial);
      break;
    case MDNN_F16:
      hipLaunchKernelGGL(colsum_partial_kernel<F16>, grid, dim3(256), 0, st, (const uint16_t*)x, nullptr, rows,
                         cols, vec, partial);
      break;
    default:
      hipLaunchKernelGGL(colsum_partial_kernel<BF16>, grid, dim3(256), 0, st, (const uint16_t*)x, nullptr, rows,
                         cols, vec, partial);
  }
  return check_launch("column sums (partials)");
}

bool column_sums_strip_ok(const void* x, mdnn_dtype_t t, int64_t cols, const float* partial) {
  return colsum_strip(t, cols) && aligned(x, 16) && aligned(partial, 8);
}

mdnn_status_t column_sums_partial_batch(const StripBatch& b, mdnn_dtype_t t, int64_t rows, hipStream_t st) {
  if (b.n <= 0) return MDNN_SUCCESS;
  if (b.n > kMaxColsumBatch) return fail(MDNN_ERR_SHAPE, "column sums: batch too large");
  int64_t widest = 0;
  for (int i = 0; i < b.n; ++i) {
    if (!column_sums_strip_ok(b.x[i], t, b.cols[i], b.partial[i]))
      return fail(MDNN_ERR_SHAPE, "column sums: a batched matrix does not take the strip pass");
    widest = b.cols[i] > widest ? b.cols[i] : widest;
  }
  const int64_t chunks = column_sums_chunks(rows, widest, t);
  if (widest == 0 || chunks == 0) return MDNN_SUCCESS;
  if (chunks > 65535) return fail(MDNN_ERR_SHAPE, "column sums: too many rows");
  const dim3 grid((unsigned)(widest / 512), (unsigned)chunks, (unsigned)b.n);
  if (t == MDNN_F16)
    hipLaunchKernelGGL(colsum_strip_batch_kernel<F16>, grid, dim3(256), 0, st, b, rows);
  else
    hipLaunchKernelGGL(colsum_strip_batch_kernel<BF16>, grid, dim3(256), 0, st, b, rows);
  return check_launch("column sums (batched partials)");
}

mdnn_status_t column_sums_final(const ColsumBatch& b, int32_t* nonfinite, hipStream_t st) {
  if (b.n <= 0) return MDNN_SUCCESS;
  if (b.n > kMaxColsumBatch) return fail(MDNN_ERR_SHAPE, "column sums: batch too large");
  int64_t widest = 0;
  for (int i = 0; i < b.n; ++i) widest = b.cols[i] > widest ? b.cols[i] : widest;
  if (widest == 0) return MDNN_SUCCESS;
  if (ceil_div(widest, 32) > 0x7fffffffLL) return fail(MDNN_ERR_SHAPE, "column sums: too many columns");
  hipLaunchKernelGGL(colsum_final_batch_kernel, dim3((unsigned)ceil_div(widest, 32), (unsigned)b.n), dim3(256), 0,
                     st, b, nonfinite);
  return check_launch("column sums (final)");
}

// ---------------------------------------------------------------------------
// fp32 split-K over a workspace
// ---------------------------------------------------------------------------
// A grid of few 64 x 64 tiles over K >= 64 is bound by the latency of its
// serial K loop: split K so that about 256 workgroups run, each over at
// least two K steps.
static SplitPlan f32_split_plan(int64_t M, int64_t N, int64_t K) {
  SplitPlan p{1, K};
  const int64_t tiles = ceil_div(M, 64) * ceil_div(N, 64);
  if (tiles >= 64 || K < 64) return p;
  int64_t kps = ceil_div(ceil_div(K, ceil_div(256, tiles)), 16) * 16;
  if (kps < 32) kps = 32;
  p.splits = (int)ceil_div(K, kps);
  p.k_per_split = kps;
  if (p.splits > 65535) p = SplitPlan{1, K};
  return p;
}

// out = epilogue(sum over splits of partial[s][m][n]).  A block covers 16
// groups of four consecutive outputs of a row; its 16 thread rows sum splits
// g, g+16, g+32, ... of each group, and the 16 row sums are added in row
// order: a fixed order, so the result is deterministic.
template <class MaskT, class OutT>
__global__ void __launch_bounds__(256)
reduce_splits_epilogue_kernel(const float* __restrict__ part, int splits, int64_t M, int64_t N, Epilogue ep) {
  __shared__ float4_t rows[16][16];
  const int ql = threadIdx.x & 15, g = threadIdx.x >> 4;
  const int64_t groups = ceil_div(N, 4);
  const int64_t q = (int64_t)blockIdx.x * 16 + ql;
  const bool valid = q < M * groups;
  const int64_t m = valid ? q / groups : 0, n = valid ? (q - m * groups) * 4 : 0;
  const int64_t MN = M * N;
  const bool vec = (N & 3) == 0;  // rows of 16-byte aligned quads (the workspace is 16-byte aligned)
  float4_t acc = {0.f, 0.f, 0.f, 0.f};
  if (valid) {
    const float* p = part + m * N + n;
    int s = g;
    // four of this thread's splits in flight at a time (same order of additions)
    for (; s + 48 < splits; s += 64) {
      float4_t v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const float* ps = p + (int64_t)(s + 16 * u) * MN;
        if (vec) {
          const float4 t = *(const float4*)ps;
          v[u] = (float4_t){t.x, t.y, t.z, t.w};
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e) v[u][e] = n + e < N ? ps[e] : 0.0f;
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (vec || n + e < N) acc[e] += v[u][e];
    }
    for (; s < splits; s += 16) {
      const float* ps = p + (int64_t)s * MN;
      if (vec) {
        const float4 v = *(const float4*)ps;
        acc[0] += v.x, acc[1] += v.y, acc[2] += v.z, acc[3] += v.w;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (n + e < N) acc[e] += ps[e];
      }
    }
  }
  rows[g][ql] = acc;
  __syncthreads();
  if (g != 0 || !valid) return;
  float4_t tot = rows[0][ql];
  for (int r = 1; r < 16; ++r) tot += rows[r][ql];
  epilogue_store4<MaskT, OutT>(ep, M, N, m, n, tot);
}

// At most 8 splits: one thread per output quad adds the splits in split
// order, four in flight at a time.  The grouped kernel above gives each of
// its groups one split in that case and then adds the groups in order, so
// the sums are the same; this one keeps every thread busy instead of one in
// sixteen (a 256 x 3136 output over 3 splits: 11.6 -> 4.2 us, 256 x 1024
// over 7: 6.1 -> 3.9 us).  With 16 splits its four rounds of loads were
// slower than the grouped kernel's one (1024 x 10: 6.8 against 5.0 us).
constexpr int REDUCE_SEQ_MAX_SPLITS = 8;
template <class MaskT, class OutT>
__global__ void __launch_bounds__(256)
reduce_splits_seq_kernel(const float* __restrict__ part, int splits, int64_t M, int64_t N, Epilogue ep) {
  const int64_t groups = ceil_div(N, 4);
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= M * groups) return;
  const int64_t m = q / groups, n = (q - m * groups) * 4;
  const int64_t MN = M * N;
  const bool vec = (N & 3) == 0;  // rows of 16-byte aligned quads (the workspace is 16-byte aligned)
  const float* p = part + m * N + n;
  float4_t acc = {0.f, 0.f, 0.f, 0.f};
  auto load = [&](int sp) -> float4_t {
    const float* ps = p + (int64_t)sp * MN;
    if (vec) {
      const float4 t = *(const float4*)ps;
      return (float4_t){t.x, t.y, t.z, t.w};
    }
    float4_t v;
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = n + e < N ? ps[e] : 0.0f;
    return v;
  };
  int s = 0;
  for (; s + 4 <= splits; s += 4) {
    float4_t v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) v[u] = load(s + u);
#pragma unroll
    for (int u = 0; u < 4; ++u) acc += v[u];
  }
  for (; s < splits; ++s) acc += load(s);
  epilogue_store4<MaskT, OutT>(ep, M, N, m, n, acc);
}

template <class MaskT, class OutT>
static mdnn_status_t reduce_epilogue(const void* ws, int splits, int64_t M, int64_t N, const Epilogue& ep,
                                     hipStream_t st) {
  const int64_t quads = M * ceil_div(N, 4);
  if (ceil_div(quads, 16) > 0x7fffffffLL) return fail(MDNN_ERR_SHAPE, "gemm: problem too large for the reduction");
  if (splits <= REDUCE_SEQ_MAX_SPLITS) {
    hipLaunchKernelGGL((reduce_splits_seq_kernel<MaskT, OutT>), dim3((unsigned)ceil_div(quads, 256)), dim3(256), 0,
                       st, (const float*)ws, splits, M, N, ep);
    return check_launch("reduce_splits_seq_kernel");
  }
  hipLaunchKernelGGL((reduce_splits_epilogue_kernel<MaskT, OutT>), dim3((unsigned)ceil_div(quads, 16)), dim3(256),
                     0, st, (const float*)ws, splits, M, N, ep);
  return check_launch("reduce_splits_epilogue_kernel");
}

mdnn_status_t reduce_splits_epilogue(const void* ws, int splits, int64_t M, int64_t N, const Epilogue& ep,
                                     mdnn_dtype_t mask_t, mdnn_dtype_t out_t, hipStream_t st) {
  if (mask_t == MDNN_F32) return reduce_epilogue<F32, F32>(ws, splits, M, N, ep, st);
  if (mask_t == MDNN_F16)
    return out_t == MDNN_F32 ? reduce_epilogue<F16, F32>(ws, splits, M, N, ep, st)
                             : reduce_epilogue<F16, F16>(ws, splits, M, N, ep, st);
  return out_t == MDNN_F32 ? reduce_epilogue<BF16, F32>(ws, splits, M, N, ep, st)
                           : reduce_epilogue<BF16, BF16>(ws, splits, M, N, ep, st);
}

// Low-precision problems whose grid of `tile` x `tile` tiles covers fewer
// than half of the CUs, over K >= 256: split K (whole 64-deep steps, at
// least two per split) so that about 256 workgroups run.
static SplitPlan lp_split_plan(int64_t M, int64_t N, int64_t K, int64_t tile) {
  SplitPlan p{1, K};
  const int64_t tiles = ceil_div(M, tile) * ceil_div(N, tile);
  if (tiles >= 128 || K < 256 || gemm_tile_override() != TILE_AUTO) return p;
  int64_t sp = ceil_div(256, tiles);
  if (sp > K / 128) sp = K / 128;
  // the fp32 partials are written and read back once more: keep them within
  // about 8 MiB unless the output is larger than that (then two splits)
  const int64_t cap = ceil_div((int64_t)8 << 20, M * N * 4);
  if (sp > (cap > 2 ? cap : 2)) sp = cap > 2 ? cap : 2;
  if (sp < 2) return p;
  const int64_t kps = ceil_div(ceil_div(K, sp), 64) * 64;
  p.splits = (int)ceil_div(K, kps);
  p.k_per_split = kps;
  if (p.splits < 2) p = SplitPlan{1, K};
  return p;
}

static bool ws_fits(const SplitPlan& p, int64_t M, int64_t N, const void* ws, size_t ws_bytes) {
  return p.splits > 1 && ws && aligned(ws, 16) && ws_bytes >= (size_t)p.splits * M * N * sizeof(float);
}

// ---------------------------------------------------------------------------
// mdnn_gemm_mixed
// ---------------------------------------------------------------------------
template <class T, class OutT>
static mdnn_status_t gemm_dispatch16(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K,
                                     const void* A, int64_t lda, bool va, const void* B,
                                     int64_t ldb, bool vb, const Epilogue& ep_in, void* ws, size_t ws_bytes,
                                     hipStream_t st) {
  const uint16_t* a = (const uint16_t*)A;
  const uint16_t* b = (const uint16_t*)B;
  const LdsOperand la{A, lda, M, layout != MDNN_TN}, lb{B, ldb, N, layout == MDNN_NT};
  // split K over the workspace when the grid is small (partials in fp32,
  // then the epilogue in a fixed-order reduction)
  Epilogue ep = ep_in;
  int splits = 1;
  SplitPlan plan = lp_split_plan(M, N, K, 128);
  bool pipe = ws_fits(plan, M, N, ws, ws_bytes) && lds_pipe_eligible(la, lb, M, N, K, plan.k_per_split, plan.splits);
  if (pipe) {
    splits = plan.splits;
  } else {
    pipe = lds_pipe_eligible(la, lb, M, N, K, K, 1);
    if (!pipe) {
      plan = lp_split_plan(M, N, K, 64);
      if (ws_fits(plan, M, N, ws, ws_bytes)) splits = plan.splits;
    }
  }
  if (splits > 1) {
    ep.partial = (float*)ws;
    ep.k_per_split = plan.k_per_split;
  }
  if (pipe) {
    switch (layout) {
      case MDNN_NN: MDNN_TRY((run_gemm_lds<T, OutT, true, false>(la, lb, M, N, K, ep, splits, st))); break;
      case MDNN_NT: MDNN_TRY((run_gemm_lds<T, OutT, true, true>(la, lb, M, N, K, ep, splits, st))); break;
      default: MDNN_TRY((run_gemm_lds<T, OutT, false, false>(la, lb, M, N, K, ep, splits, st)));
    }
  } else {
    switch (layout) {
      case MDNN_NN:
        MDNN_TRY((run_gemm16<T, OutT>(SrcMatK<uint16_t>{a, lda, M, K, va}, SrcMatMN<uint16_t>{b, ldb, N, K, vb}, M,
                                      N, K, ep, splits, st)));
        break;
      case MDNN_NT:
        MDNN_TRY((run_gemm16<T, OutT>(SrcMatK<uint16_t>{a, lda, M, K, va}, SrcMatK<uint16_t>{b, ldb, N, K, vb}, M,
                                      N, K, ep, splits, st)));
        break;
      default:
        MDNN_TRY((run_gemm16<T, OutT>(SrcMatMN<uint16_t>{a, lda, M, K, va}, SrcMatMN<uint16_t>{b, ldb, N, K, vb},
                                      M, N, K, ep, splits, st)));
    }
  }
  if (splits == 1) return MDNN_SUCCESS;
  return reduce_epilogue<T, OutT>(ws, splits, M, N, ep_in, st);
}

static mdnn_status_t gemm_dispatch32(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K,
                                     const void* A, int64_t lda, const void* B, int64_t ldb,
                                     const Epilogue& ep_in, void* ws, size_t ws_bytes, hipStream_t st) {
  const float* a = (const float*)A;
  const float* b = (const float*)B;
  Epilogue ep = ep_in;
  const SplitPlan plan = f32_split_plan(M, N, K);
  const bool split = ws_fits(plan, M, N, ws, ws_bytes);
  int splits = 1;
  if (split) {
    ep.partial = (float*)ws;
    ep.k_per_split = plan.k_per_split;
    splits = plan.splits;
  }
  switch (layout) {
    case MDNN_NN:
      MDNN_TRY(run_gemm32(SrcMatK<float>{a, lda, M, K, false}, SrcMatMN<float>{b, ldb, N, K, false},
                          M, N, K, ep, splits, st));
      break;
    case MDNN_NT:
      MDNN_TRY(run_gemm32(SrcMatK<float>{a, lda, M, K, false}, SrcMatK<float>{b, ldb, N, K, false},
                          M, N, K, ep, splits, st));
      break;
    default:
      MDNN_TRY(run_gemm32(SrcMatMN<float>{a, lda, M, K, false}, SrcMatMN<float>{b, ldb, N, K, false},
                          M, N, K, ep, splits, st));
  }
  if (!split) return MDNN_SUCCESS;
  return reduce_epilogue<F32, F32>(ws, splits, M, N, ep_in, st);
}

}  // namespace mdnn

using namespace mdnn;

size_t mdnn::gemm_ws_bytes(mdnn_dtype_t ab_type, int64_t M, int64_t N, int64_t K) {
  if (M <= 0 || N <= 0 || K <= 0 || !dtype_ok(ab_type)) return 0;
  int splits = 1;
  if (ab_type == MDNN_F32) {
    splits = f32_split_plan(M, N, K).splits;
  } else {  // either kernel family may run: room for the larger plan
    const int s128 = lp_split_plan(M, N, K, 128).splits, s64 = lp_split_plan(M, N, K, 64).splits;
    splits = s128 > s64 ? s128 : s64;
  }
  const size_t tiles = splits > 1 ? (size_t)splits * M * N * sizeof(float) : 0;
  // the skinny TN kernel's split (the layout is not an argument: room for it)
  const size_t sk = skinny_ws_bytes(MDNN_TN, M, N, K);
  return tiles > sk ? tiles : sk;
}

extern "C" mdnn_status_t mdnn_gemm_mixed(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K,
                                         float alpha, const void* A, int64_t lda, const void* B,
                                         int64_t ldb, mdnn_dtype_t ab_type, float beta,
                                         const void* C, int64_t ldc, void* D, int64_t ldd,
                                         mdnn_dtype_t d_type, const float* bias, mdnn_act_t act,
                                         const void* mask_src, int64_t ldm, mdnn_stream_t stream) {
  return gemm_mixed_ws(layout, M, N, K, alpha, A, lda, B, ldb, ab_type, beta, C, ldc, D, ldd, d_type, bias, act,
                       mask_src, ldm, nullptr, 0, stream);
}

extern "C" size_t mdnn_gemm_workspace(mdnn_dtype_t ab_type, int64_t M, int64_t N, int64_t K) {
  return gemm_ws_bytes(ab_type, M, N, K);
}

extern "C" mdnn_status_t mdnn_gemm_mixed_ws(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K, float alpha,
                                            const void* A, int64_t lda, const void* B, int64_t ldb,
                                            mdnn_dtype_t ab_type, float beta, const void* C, int64_t ldc, void* D,
                                            int64_t ldd, mdnn_dtype_t d_type, const float* bias, mdnn_act_t act,
                                            const void* mask_src, int64_t ldm, void* workspace, size_t ws_bytes,
                                            int32_t* nonfinite, mdnn_stream_t stream) {
  if (nonfinite && !aligned(nonfinite, 4)) return fail(MDNN_ERR_MISALIGNED, "gemm: nonfinite is misaligned");
  return gemm_mixed_ws(layout, M, N, K, alpha, A, lda, B, ldb, ab_type, beta, C, ldc, D, ldd, d_type, bias, act,
                       mask_src, ldm, workspace, ws_bytes, stream, nonfinite);
}

mdnn_status_t mdnn::gemm_mixed_ws(mdnn_layout_t layout, int64_t M, int64_t N, int64_t K, float alpha,
                                  const void* A, int64_t lda, const void* B, int64_t ldb, mdnn_dtype_t ab_type,
                                  float beta, const void* C, int64_t ldc, void* D, int64_t ldd,
                                  mdnn_dtype_t d_type, const float* bias, mdnn_act_t act, const void* mask_src,
                                  int64_t ldm, void* ws, size_t ws_bytes, mdnn_stream_t stream,
                                  int32_t* nonfinite, const float* alpha_dev) {
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
  ep.vec4_c = beta != 0.0f && (ldc % 4 == 0) && aligned(C, 4 * ds);
  ep.vec4_m = mask_src && (ldm % 4 == 0) && aligned(mask_src, 4 * es);
  ep.partial = nullptr;
  ep.k_per_split = K;
  ep.nonfinite = nonfinite;
  ep.alpha_dev = alpha_dev;
  hipStream_t st = as_stream(stream);
  clear_error();

  if (skinny_takes(layout, M, N, K, ws, ws_bytes))
    return gemm_skinny(layout, M, N, K, A, lda, B, ldb, ab_type, d_type, ep, ws, ws_bytes, st);
  if (ab_type == MDNN_F32) return gemm_dispatch32(layout, M, N, K, A, lda, B, ldb, ep, ws, ws_bytes, st);
  const bool va = aligned(A, 16) && lda % 8 == 0;
  const bool vb = aligned(B, 16) && ldb % 8 == 0;
  if (ab_type == MDNN_F16) {
    if (d_type == MDNN_F32)
      return gemm_dispatch16<F16, F32>(layout, M, N, K, A, lda, va, B, ldb, vb, ep, ws, ws_bytes, st);
    return gemm_dispatch16<F16, F16>(layout, M, N, K, A, lda, va, B, ldb, vb, ep, ws, ws_bytes, st);
  }
  if (d_type == MDNN_F32)
    return gemm_dispatch16<BF16, F32>(layout, M, N, K, A, lda, va, B, ldb, vb, ep, ws, ws_bytes, st);
  return gemm_dispatch16<BF16, BF16>(layout, M, N, K, A, lda, va, B, ldb, vb, ep, ws, ws_bytes, st);
}

int mdnn::gemm_lp_splits(int64_t M, int64_t N, int64_t K) { return lp_split_plan(M, N, K, 128).splits; }

bool mdnn::gemm_tn_update_ok(mdnn_dtype_t ab_type, int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                              const void* B, int64_t ldb, const float* w32, const float* v32, const void* w_lp,
                              int64_t ldw) {
  if (ab_type != MDNN_F16 && ab_type != MDNN_BF16) return false;
  // every tile of every pipelined configuration is interior, no K split
  if (M <= 0 || N <= 0 || K <= 0 || M % 256 != 0 || N % 256 != 0) return false;
  if (lda < M || ldb < N || ldw < N || ldw % 4 != 0) return false;
  if (!w32 || !aligned(w32, 16) || (v32 && !aligned(v32, 16)) || (w_lp && !aligned(w_lp, 8))) return false;
  const LdsOperand la{A, lda, M, false}, lb{B, ldb, N, false};
  return lds_pipe_eligible(la, lb, M, N, K, K, 1);
}

extern "C" mdnn_status_t mdnn_gemm_tn_update(int64_t M, int64_t N, int64_t K, const void* A, int64_t lda,
                                             const void* B, int64_t ldb, mdnn_dtype_t ab_type, float* w32,
                                             float* v32, void* w_lp, int64_t ldw, float lr, float momentum,
                                             const mdnn_scaler_t* scaler, mdnn_stream_t stream) {
  if (!dtype_ok(ab_type)) return fail(MDNN_ERR_DTYPE, "gemm_tn_update: unknown dtype");
  if (ab_type == MDNN_F32) return fail(MDNN_ERR_DTYPE, "gemm_tn_update: 16-bit operands only");
  if (!A || !B || !w32) return fail(MDNN_ERR_NULL, "gemm_tn_update: A, B and w32 are required");
  if (momentum != 0.0f && !v32) return fail(MDNN_ERR_NULL, "gemm_tn_update: v32 is required with momentum");
  if (M <= 0 || N <= 0 || K <= 0 || M % 256 != 0 || N % 256 != 0 || K % lds::BK != 0)
    return fail(MDNN_ERR_SHAPE, "gemm_tn_update: M and N must be positive multiples of 256, K of %d", lds::BK);
  if (lda < M || ldb < N || ldw < N) return fail(MDNN_ERR_LAYOUT, "gemm_tn_update: a leading dimension is too small");
  if (!aligned(A, 16) || !aligned(B, 16) || lda % 8 != 0 || ldb % 8 != 0 || !aligned(w32, 16) ||
      (v32 && !aligned(v32, 16)) || (w_lp && !aligned(w_lp, 8)) || ldw % 4 != 0 || (scaler && !aligned(scaler, 4)))
    return fail(MDNN_ERR_MISALIGNED,
                "gemm_tn_update: A, B, w32, v32 need 16-byte alignment (w_lp 8), lda / ldb multiples of 8, ldw of 4");
  if (!gemm_tn_update_ok(ab_type, M, N, K, A, lda, B, ldb, w32, momentum != 0.0f ? v32 : nullptr, w_lp, ldw))
    return fail(MDNN_ERR_SHAPE, "gemm_tn_update: the operands do not fit the pipelined kernel");
  Epilogue ep{};
  ep.alpha = 1.0f;
  ep.D = w32;  // never stored: every tile is interior and takes the update
  ep.ldd = ldw;
  ep.vec4 = 1;
  ep.k_per_split = K;
  ep.upd_w = w32;
  ep.upd_v = momentum != 0.0f ? v32 : nullptr;
  ep.upd_lp = w_lp;
  ep.upd_lr = lr;
  ep.upd_mu = momentum;
  ep.upd_sc = scaler;
  const LdsOperand la{A, lda, M, false}, lb{B, ldb, N, false};
  clear_error();
  hipStream_t st = as_stream(stream);
  if (ab_type == MDNN_F16) return run_gemm_lds<F16, F32, false, false>(la, lb, M, N, K, ep, 1, st);
  return run_gemm_lds<BF16, F32, false, false>(la, lb, M, N, K, ep, 1, st);
}

extern "C" int mdnn_set_gemm_tile(int code) {
  if (code < 0 || code > TILE_LDS_PIPE128) return -1;
  g_tile_override.store(code, std::memory_order_relaxed);
  return 0;
}
