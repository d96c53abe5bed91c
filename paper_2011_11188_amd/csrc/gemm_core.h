// MFMA GEMM engine for gfx950: D = epi(alpha * op(A) op(B) + beta * C).
//
// Section 3.2 of the paper: the matrix unit computes D = C + A*B with
// low-precision A, B and an fp32 accumulator; on CDNA4 that unit is
// v_mfma_f32_16x16x32_{f16,bf16} (16x16 output, 32-deep, fp32 accumulate).
//
// Structure (one workgroup = one BM x BN output tile, WM x WN waves of 64):
//   * operands are described by "sources" that return 16-byte chunks of 8
//     consecutive elements along their contiguous dimension: plain row-major
//     matrices, or implicit-im2col views of NHWC tensors for convolution;
//   * each K step of BK = 64 is staged global -> registers -> LDS, with two
//     LDS buffers so the next tile's global loads are in flight while the
//     current tile feeds the MFMAs (one barrier per K step);
//   * LDS holds both operands K-contiguous, [rows][BK + 8] (the 16-byte row
//     pad spreads the 16-byte fragment reads of 16 rows over all banks);
//     an operand stored MN-contiguous in memory is transposed in registers
//     (4 k x 8 mn blocks) on its way to LDS;
//   * the MFMA is issued with B as its first operand, so each lane ends with
//     4 consecutive columns of one row (a 16-byte fp32 / 8-byte fp16 store);
//   * the epilogue applies alpha, beta*C, bias, ReLU, the ReLU mask of a
//     backward-data product and the rounding to the output type, or writes
//     fp32 split-K partials that a second kernel reduces in a fixed order.
//   * workgroup ids are remapped so that consecutive tiles land on the same
//     XCD (8 XCDs, round-robin dispatch), grouped by GROUP_M tile rows.
#pragma once

#include "common.h"

namespace mdnn {

constexpr int GEMM_BK = 64;
constexpr int GEMM_PAD = 8;                     // elements of row padding in LDS
constexpr int GEMM_LDK = GEMM_BK + GEMM_PAD;    // LDS row pitch (elements)

// ---------------------------------------------------------------------------
// operand sources (16-bit element types; `vec` allows 16-byte loads)
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint4 pack8(const uint16_t v[8]) {
  uint4 r;
  r.x = (uint32_t)v[0] | ((uint32_t)v[1] << 16);
  r.y = (uint32_t)v[2] | ((uint32_t)v[3] << 16);
  r.z = (uint32_t)v[4] | ((uint32_t)v[5] << 16);
  r.w = (uint32_t)v[6] | ((uint32_t)v[7] << 16);
  return r;
}

// Sixteen bytes of zeros in device memory: an out-of-range chunk is loaded
// from here instead of being skipped or selected away, so every chunk load of
// a tile is one unconditional instruction and they all stay in flight (a
// load under a divergent branch, or one whose register another branch writes,
// is waited for before the code can go on).
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
__device__ __attribute__((aligned(16))) const u32x4_t kZeroChunk = {0u, 0u, 0u, 0u};

__device__ __forceinline__ uint4 load_chunk_or_zero(const void* p, bool ok) {
  // loaded through a global-address-space pointer: a generic (flat) load
  // would also count against the LDS wait counter and stall the next LDS
  // read until it lands
  typedef const __attribute__((address_space(1))) u32x4_t GlobalChunk;
  const u32x4_t v = *(GlobalChunk*)(ok ? p : (const void*)&kZeroChunk);
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Every source gives elem(mn, k) (bounds-checked, zero outside; mn is the
// operand's M index for A and N index for B) for any storage type S, the
// same as an offset from base() (off(mn, k), -1 outside or in padding), and, for
// 16-bit storage, chunk(...) = 8 consecutive elements along the contiguous
// dimension packed into 16 bytes: chunk(mn, k) for K-contiguous sources,
// chunk(k, mn) for MN-contiguous ones.

// Row-major matrix whose contiguous dimension is K: elem(mn, k) = p[mn*ld + k].
template <class S>
struct SrcMatK {
  static constexpr bool KC = true;
  const S* p;
  int64_t ld, MN, K;
  bool vec;
  int64_t bs = 0;  // elements between consecutive matrices of a batch (grid z)
  __device__ __forceinline__ S elem(int64_t mn, int64_t k) const {
    return (mn < MN && k < K) ? p[mn * ld + k] : (S)0;
  }
  __device__ __forceinline__ const S* base() const { return p; }
  __device__ __forceinline__ int64_t off(int64_t mn, int64_t k) const { return (mn < MN && k < K) ? mn * ld + k : -1; }
  __device__ __forceinline__ uint4 chunk(int64_t mn, int64_t k) const {
    if (vec && (k + 8 <= K || k >= K)) {
      const bool ok = mn < MN && k + 8 <= K;
      return load_chunk_or_zero(p + (ok ? mn * ld + k : 0), ok);
    }
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = elem(mn, k + e);
    return pack8(v);
  }
};

// Row-major matrix whose contiguous dimension is M (or N): elem(mn, k) = p[k*ld + mn].
template <class S>
struct SrcMatMN {
  static constexpr bool KC = false;
  const S* p;
  int64_t ld, MN, K;
  bool vec;
  int64_t bs = 0;  // elements between consecutive matrices of a batch (grid z)
  __device__ __forceinline__ S elem(int64_t mn, int64_t k) const {
    return (k < K && mn < MN) ? p[k * ld + mn] : (S)0;
  }
  __device__ __forceinline__ const S* base() const { return p; }
  __device__ __forceinline__ int64_t off(int64_t mn, int64_t k) const { return (k < K && mn < MN) ? k * ld + mn : -1; }
  __device__ __forceinline__ uint4 chunk(int64_t k, int64_t mn) const {
    if (vec && (mn + 8 <= MN || mn >= MN)) {
      const bool ok = k < K && mn + 8 <= MN;
      return load_chunk_or_zero(p + (ok ? k * ld + mn : 0), ok);
    }
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = elem(mn + e, k);
    return pack8(v);
  }
};

// Convolution geometry, stride 1, zero padding.
struct ConvGeom {
  int32_t n, h, w, c, k, r, s, pad, ho, wo;
};

// Forward, operand A[m, kk]: m = (n, i, j) over the output, kk = (r, s, c);
// elem = x[n, i + r - pad, j + s - pad, c].  K-contiguous (c fastest).
template <class S>
struct SrcConvFwdA {
  static constexpr bool KC = true;
  const S* x;
  ConvGeom g;
  int64_t MN, K;
  bool vec;  // c % 8 == 0 and 16-byte aligned base
  // offset of (m, kk) in x, or -1 in the zero padding
  __device__ __forceinline__ int64_t offset(int64_t m, int64_t kk) const {
    int32_t c = (int32_t)(kk % g.c);
    int32_t rs = (int32_t)(kk / g.c);
    int32_t s = rs % g.s, r = rs / g.s;
    int32_t j = (int32_t)(m % g.wo);
    int64_t t = m / g.wo;
    int32_t i = (int32_t)(t % g.ho);
    int32_t n = (int32_t)(t / g.ho);
    int32_t hi = i + r - g.pad, wi = j + s - g.pad;
    if (hi < 0 || hi >= g.h || wi < 0 || wi >= g.w) return -1;
    return (((int64_t)n * g.h + hi) * g.w + wi) * g.c + c;
  }
  __device__ __forceinline__ S elem(int64_t m, int64_t kk) const {
    if (m >= MN || kk >= K) return (S)0;
    int64_t o = offset(m, kk);
    return o < 0 ? (S)0 : x[o];
  }
  __device__ __forceinline__ const S* base() const { return x; }
  __device__ __forceinline__ int64_t off(int64_t m, int64_t kk) const {
    return (m < MN && kk < K) ? offset(m, kk) : -1;
  }
  __device__ __forceinline__ uint4 chunk(int64_t m, int64_t kk) const {
    if (vec && (kk + 8 <= K || kk >= K)) {
      const int64_t o = (m < MN && kk + 8 <= K) ? offset(m, kk) : -1;
      return load_chunk_or_zero(x + (o < 0 ? 0 : o), o >= 0);
    }
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = elem(m, kk + e);
    return pack8(v);
  }
};

// Backward-data, operand A[m, kk]: m = (n, h, w) over the input image,
// kk = (r, s, k); elem = dy[n, h - r + pad, w - s + pad, k].  K-contiguous.
template <class S>
struct SrcConvBwdA {
  static constexpr bool KC = true;
  const S* dy;
  ConvGeom g;
  int64_t MN, K;
  bool vec;  // k % 8 == 0
  __device__ __forceinline__ int64_t offset(int64_t m, int64_t kk) const {
    int32_t ch = (int32_t)(kk % g.k);
    int32_t rs = (int32_t)(kk / g.k);
    int32_t s = rs % g.s, r = rs / g.s;
    int32_t wj = (int32_t)(m % g.w);
    int64_t t = m / g.w;
    int32_t hi = (int32_t)(t % g.h);
    int32_t n = (int32_t)(t / g.h);
    int32_t i = hi - r + g.pad, j = wj - s + g.pad;
    if (i < 0 || i >= g.ho || j < 0 || j >= g.wo) return -1;
    return (((int64_t)n * g.ho + i) * g.wo + j) * g.k + ch;
  }
  __device__ __forceinline__ S elem(int64_t m, int64_t kk) const {
    if (m >= MN || kk >= K) return (S)0;
    int64_t o = offset(m, kk);
    return o < 0 ? (S)0 : dy[o];
  }
  __device__ __forceinline__ const S* base() const { return dy; }
  __device__ __forceinline__ int64_t off(int64_t m, int64_t kk) const {
    return (m < MN && kk < K) ? offset(m, kk) : -1;
  }
  __device__ __forceinline__ uint4 chunk(int64_t m, int64_t kk) const {
    if (vec && (kk + 8 <= K || kk >= K)) {
      const int64_t o = (m < MN && kk + 8 <= K) ? offset(m, kk) : -1;
      return load_chunk_or_zero(dy + (o < 0 ? 0 : o), o >= 0);
    }
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = elem(m, kk + e);
    return pack8(v);
  }
};

// Backward-data, operand B[kk, c] with kk = (r, s, k): elem = w[k, r, s, c].
// MN-contiguous along c.
template <class S>
struct SrcConvBwdB {
  static constexpr bool KC = false;
  const S* wt;
  ConvGeom g;
  int64_t MN, K;  // MN = c, K = r*s*k
  bool vec;       // c % 8 == 0
  __device__ __forceinline__ int64_t row(int64_t kk) const {
    int32_t ch = (int32_t)(kk % g.k);
    int32_t rs = (int32_t)(kk / g.k);
    return ((int64_t)ch * g.r * g.s + rs) * g.c;
  }
  __device__ __forceinline__ S elem(int64_t c, int64_t kk) const {
    return (kk < K && c < MN) ? wt[row(kk) + c] : (S)0;
  }
  __device__ __forceinline__ const S* base() const { return wt; }
  __device__ __forceinline__ int64_t off(int64_t c, int64_t kk) const { return (kk < K && c < MN) ? row(kk) + c : -1; }
  __device__ __forceinline__ uint4 chunk(int64_t kk, int64_t c) const {
    if (vec && (c + 8 <= MN || c >= MN)) {
      const bool ok = kk < K && c + 8 <= MN;
      return load_chunk_or_zero(wt + (ok ? row(kk) + c : 0), ok);
    }
    if (kk >= K) return make_uint4(0, 0, 0, 0);
    const S* p = wt + row(kk);
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (c + e < MN) ? p[c + e] : (S)0;
    return pack8(v);
  }
};

// Backward-filter, operand B[kk, nn] with kk = (n, i, j) over the output and
// nn = (r, s, c): elem = x[n, i + r - pad, j + s - pad, c].  MN-contiguous.
template <class S>
struct SrcConvFiltB {
  static constexpr bool KC = false;
  const S* x;
  ConvGeom g;
  int64_t MN, K;  // MN = r*s*c, K = n*ho*wo
  bool vec;       // c % 8 == 0
  __device__ __forceinline__ int64_t offset(int64_t kk, int64_t nn) const {
    int32_t c = (int32_t)(nn % g.c);
    int32_t rs = (int32_t)(nn / g.c);
    int32_t s = rs % g.s, r = rs / g.s;
    int32_t j = (int32_t)(kk % g.wo);
    int64_t t = kk / g.wo;
    int32_t i = (int32_t)(t % g.ho);
    int32_t n = (int32_t)(t / g.ho);
    int32_t hi = i + r - g.pad, wi = j + s - g.pad;
    if (hi < 0 || hi >= g.h || wi < 0 || wi >= g.w) return -1;
    return (((int64_t)n * g.h + hi) * g.w + wi) * g.c + c;
  }
  __device__ __forceinline__ S elem(int64_t nn, int64_t kk) const {
    if (kk >= K || nn >= MN) return (S)0;
    int64_t o = offset(kk, nn);
    return o < 0 ? (S)0 : x[o];
  }
  __device__ __forceinline__ const S* base() const { return x; }
  __device__ __forceinline__ int64_t off(int64_t nn, int64_t kk) const {
    return (kk < K && nn < MN) ? offset(kk, nn) : -1;
  }
  __device__ __forceinline__ uint4 chunk(int64_t kk, int64_t nn) const {
    if (vec && (nn + 8 <= MN || nn >= MN)) {
      const int64_t o = (kk < K && nn + 8 <= MN) ? offset(kk, nn) : -1;
      return load_chunk_or_zero(x + (o < 0 ? 0 : o), o >= 0);
    }
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = elem(nn + e, kk);
    return pack8(v);
  }
};

// ---------------------------------------------------------------------------
// epilogue description
// ---------------------------------------------------------------------------
struct Epilogue {
  float alpha, beta;
  const void* C;       // d_type [M, ldc], read iff beta != 0
  int64_t ldc;
  void* D;             // d_type [M, ldd]  (or fp32 partials when split)
  int64_t ldd;
  const float* bias;   // [N] or null
  const void* mask;    // ab_type [M, ldm] or null
  int64_t ldm;
  int32_t act;
  int32_t vec4;        // 4-wide stores of D allowed (ldd % 4 == 0, D aligned to 4 elements)
  int32_t vec4_c;      // 4-wide loads of C allowed (ldc % 4 == 0, C aligned to 4 elements)
  int32_t vec4_m;      // 4-wide loads of the mask allowed (ldm % 4 == 0, mask aligned to 4 elements)
  float* partial;      // split-K: fp32 [splits][M][N]; null otherwise
  int64_t k_per_split; // multiple of GEMM_BK
  int64_t bstride_d;   // batched products (grid z): elements of D between batch entries
  int32_t* nonfinite;  // set to 1 (atomic OR) when a stored value is Inf or NaN (16-bit D: as stored); or null
  const float* alpha_dev;  // device scalar multiplied into alpha (scales chosen on the device), or null
  // SGD update in place of storing D (the pipelined kernel's TN products
  // with an fp32 gradient, interior tiles only; see update_epilogue in
  // gemm_lds.h): element (m, n) of the product is the gradient of
  // upd_w[m * ldd + n]; null otherwise
  float* upd_w;
  float* upd_v;        // momentum, same indexing, or null (plain SGD)
  void* upd_lp;        // working copy in the operands' 16-bit type, same indexing, or null
  float upd_lr, upd_mu;
  const mdnn_scaler_t* upd_sc;  // loss scaler (skip when reserved, divide by scale), or null
};

// Batched products: grid z selects one matrix of a batch of plain matrices
// (SrcMatK / SrcMatMN with bs != 0); other sources are never batched.
template <class S>
__device__ __forceinline__ void shift_batch(SrcMatK<S>& s, int z) { s.p += (int64_t)z * s.bs; }
template <class S>
__device__ __forceinline__ void shift_batch(SrcMatMN<S>& s, int z) { s.p += (int64_t)z * s.bs; }
template <class Src>
__device__ __forceinline__ void shift_batch(Src&, int) {}

// Four consecutive stored elements as floats, in one vector load (p aligned
// to four elements).
template <class T>
__device__ __forceinline__ void load4(const typename T::storage* p, float (&o)[4]) {
  if constexpr (sizeof(typename T::storage) == 4) {
    const float4 q = *(const float4*)p;
    o[0] = q.x, o[1] = q.y, o[2] = q.z, o[3] = q.w;
  } else {
    const uint2 q = *(const uint2*)p;
    o[0] = to_f<T>((uint16_t)(q.x & 0xffffu));
    o[1] = to_f<T>((uint16_t)(q.x >> 16));
    o[2] = to_f<T>((uint16_t)(q.y & 0xffffu));
    o[3] = to_f<T>((uint16_t)(q.y >> 16));
  }
}

// Whether a tile (every row < M and column < N: `inside`) can take the
// straight-line epilogue (FULL below): 4-aligned rows of D, C and the mask,
// a 16-byte aligned bias.
__device__ __forceinline__ bool full_tile_epilogue(const Epilogue& ep, bool inside, int64_t N) {
  return inside && ep.vec4 && (N & 3) == 0 && (ep.beta == 0.0f || ep.vec4_c) &&
         (!ep.bias || ((uintptr_t)ep.bias & 15) == 0) && (!ep.mask || ep.vec4_m);
}

// FULL: the caller guarantees m < M, n + 4 <= N and 4-element vector access
// to every operand the epilogue touches (vec4, vec4_c when beta != 0, vec4_m
// with a mask, a 16-byte aligned bias), so no per-lane bound is tested and
// the code is straight-line.  mv_in / bias_in (FULL only, nullable): the four
// mask values / bias values, loaded by the caller.
template <class MaskT, class OutT, bool FULL = false>
__device__ __forceinline__ void epilogue_store4(const Epilogue& ep, int64_t M, int64_t N, int64_t m,
                                                int64_t n, float4_t acc, const float* mv_in = nullptr,
                                                const float* bias_in = nullptr) {
  if (!FULL && m >= M) return;
  float v[4] = {acc[0], acc[1], acc[2], acc[3]};
  const bool in4 = FULL || n + 4 <= N;
  const bool full = FULL || (ep.vec4 && in4);
  const float alpha = ep.alpha_dev ? ep.alpha * *ep.alpha_dev : ep.alpha;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    v[e] *= alpha;
  }
  if (ep.beta != 0.0f) {
    const typename OutT::storage* c = (const typename OutT::storage*)ep.C + m * ep.ldc + n;
    if (FULL || (ep.vec4_c && in4)) {
      float cv[4];
      load4<OutT>(c, cv);
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] += ep.beta * cv[e];
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (n + e < N) v[e] += ep.beta * to_f<OutT>(c[e]);
    }
  }
  if (ep.bias) {
    if (FULL && bias_in) {
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] += bias_in[e];
    } else if (FULL || (in4 && ((uintptr_t)(ep.bias + n) & 15) == 0)) {
      const float4 b = *(const float4*)(ep.bias + n);
      v[0] += b.x, v[1] += b.y, v[2] += b.z, v[3] += b.w;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (n + e < N) v[e] += ep.bias[n + e];
    }
  }
  if (ep.act == MDNN_ACT_RELU) {
#pragma unroll
    for (int e = 0; e < 4; ++e) v[e] = relu_f(v[e]);
  }
  if (ep.mask) {
    const typename MaskT::storage* mk = (const typename MaskT::storage*)ep.mask + m * ep.ldm + n;
    if (FULL && mv_in) {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (!(mv_in[e] > 0.0f)) v[e] = 0.0f;
    } else if (FULL || (ep.vec4_m && in4)) {
      float mv[4];
      load4<MaskT>(mk, mv);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (!(mv[e] > 0.0f)) v[e] = 0.0f;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (n + e < N && !(to_f<MaskT>(mk[e]) > 0.0f)) v[e] = 0.0f;
    }
  }
  typename OutT::storage* d = (typename OutT::storage*)ep.D + m * ep.ldd + n;
  if constexpr (sizeof(typename OutT::storage) == 4) {
    // the loss scaler's overflow test, on the values as stored
    if (ep.nonfinite) {
      bool bad = false;
#pragma unroll
      for (int e = 0; e < 4; ++e) bad |= (FULL || n + e < N) && !isfinite(v[e]);
      if (bad) atomicOr(ep.nonfinite, 1);
    }
    if (full) {
      *(float4*)d = make_float4(v[0], v[1], v[2], v[3]);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (n + e < N) d[e] = v[e];
    }
  } else {
    uint16_t h[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) h[e] = from_f<OutT>(v[e]);
    // 16-bit stores: the test is on the stored bits (an all-ones exponent),
    // which also catches finite values that round to Inf
    if (ep.nonfinite) {
      constexpr uint16_t EXP = OutT::id == MDNN_F16 ? 0x7c00u : 0x7f80u;
      bool bad = false;
#pragma unroll
      for (int e = 0; e < 4; ++e) bad |= (FULL || n + e < N) && (h[e] & EXP) == EXP;
      if (bad) atomicOr(ep.nonfinite, 1);
    }
    if (full) {
      uint2 u;
      u.x = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
      u.y = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
      *(uint2*)d = u;
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e)
        if (n + e < N) d[e] = h[e];
    }
  }
}

// The interior epilogue of a wave's FM x FN fragments (16-bit operands; the
// caller has checked full_tile_epilogue): the loads the stores depend on are
// issued before the first store -- the bias quads of the wave's columns once
// (rather than once per fragment) and every ReLU-mask quad of the wave (one
// round trip instead of one per fragment, each of which had waited for its
// load behind the previous fragment's stores).  In the 4096-wide MLP step:
// 3 us per forward product (bias), the mask of a 4096^3 backward data
// product 9.2 -> 6.4 us (its 32 MB read at the end of the tile).
template <class T, class OutT, int FM, int FN>
__device__ __forceinline__ void epilogue_interior(const Epilogue& ep, int64_t M, int64_t N, int64_t mb, int64_t nb,
                                                  const float4_t (&acc)[FM][FN]) {
  typedef typename T::storage S;
  static_assert(sizeof(S) == 2, "16-bit operands and mask");
  float bq[FN][4];
  if (ep.bias) {
#pragma unroll
    for (int j = 0; j < FN; ++j) {
      const float4 b = *(const float4*)(ep.bias + nb + j * 16);
      bq[j][0] = b.x, bq[j][1] = b.y, bq[j][2] = b.z, bq[j][3] = b.w;
    }
  }
  if (ep.mask) {
    uint2 mq[FM][FN];
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        mq[i][j] = *(const uint2*)((const S*)ep.mask + (mb + i * 16) * ep.ldm + nb + j * 16);
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const float mv[4] = {to_f<T>((S)(mq[i][j].x & 0xffffu)), to_f<T>((S)(mq[i][j].x >> 16)),
                             to_f<T>((S)(mq[i][j].y & 0xffffu)), to_f<T>((S)(mq[i][j].y >> 16))};
        epilogue_store4<T, OutT, true>(ep, M, N, mb + i * 16, nb + j * 16, acc[i][j], mv,
                                       ep.bias ? bq[j] : nullptr);
      }
    return;
  }
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
      epilogue_store4<T, OutT, true>(ep, M, N, mb + i * 16, nb + j * 16, acc[i][j], nullptr,
                                     ep.bias ? bq[j] : nullptr);
}

// ---------------------------------------------------------------------------
// the kernel
// ---------------------------------------------------------------------------
template <class T> struct Mfma;
template <> struct Mfma<F16> {
  static __device__ __forceinline__ float4_t run(uint4 a, uint4 b, float4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(half8_t, a),
                                                  __builtin_bit_cast(half8_t, b), c, 0, 0, 0);
  }
};
template <> struct Mfma<BF16> {
  static __device__ __forceinline__ float4_t run(uint4 a, uint4 b, float4_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bhalf8_t, a),
                                                   __builtin_bit_cast(bhalf8_t, b), c, 0, 0, 0);
  }
};

template <int BM, int BN, int WM, int WN>
struct TileShape {
  static constexpr int NT = WM * WN * 64;
  static constexpr int WTM = BM / WM, WTN = BN / WN;  // wave tile
  static constexpr int FM = WTM / 16, FN = WTN / 16;  // 16x16 fragments per wave
  static constexpr int RA = BM * GEMM_BK / 8 / NT;    // 16-byte chunks per thread (A)
  static constexpr int RB = BN * GEMM_BK / 8 / NT;    // (B)
  static constexpr int LDS_ELEMS = (BM + BN) * GEMM_LDK;
  static_assert(BM % (WM * 16) == 0 && BN % (WN * 16) == 0, "wave tile");
  static_assert(RA >= 1 && RB >= 1 && RA * NT * 8 == BM * GEMM_BK && RB * NT * 8 == BN * GEMM_BK,
                "loader split");
  static_assert(BM % 32 == 0 && BN % 32 == 0, "MN-contiguous loader granularity");
};

// Global -> registers for one operand tile of ROWS rows x BK.
// K-contiguous: chunk c = tid + i*NT -> (row = c / 8, k = (c % 8) * 8).
// MN-contiguous: chunk c -> a 4(k) x 8(mn) block: within each group of 64
//   chunks, 16 k-quads x 4 mn-octets; each block = 4 loads of 8 mn values.
template <class Src, int ROWS, int NT, int R>
__device__ __forceinline__ void load_tile(const Src& src, int64_t mn0, int64_t k0, int tid,
                                          uint4 (&reg)[R]) {
  if constexpr (Src::KC) {
#pragma unroll
    for (int i = 0; i < R; ++i) {
      int c = tid + i * NT;
      reg[i] = src.chunk(mn0 + (c >> 3), k0 + (c & 7) * 8);
    }
  } else {
    static_assert(R % 4 == 0 || R < 4, "");
    // R chunks = R/4 blocks of 4 loads (R >= 4), or one block spread over
    // 4/R threads... only R % 4 == 0 is supported.
    static_assert(R % 4 == 0, "MN-contiguous loader needs 4 chunks per thread");
#pragma unroll
    for (int b = 0; b < R / 4; ++b) {
      int blk = tid + b * NT;
      int lane = blk & 63, grp = blk >> 6;
      int k4 = lane & 15, mn8 = grp * 4 + (lane >> 4);
#pragma unroll
      for (int j = 0; j < 4; ++j) reg[b * 4 + j] = src.chunk(k0 + k4 * 4 + j, mn0 + mn8 * 8);
    }
  }
}

// Registers -> LDS ([ROWS][LDK], K-contiguous).
template <bool KC, int ROWS, int NT, int R>
__device__ __forceinline__ void store_tile(uint16_t* lds, int tid, const uint4 (&reg)[R]) {
  if constexpr (KC) {
#pragma unroll
    for (int i = 0; i < R; ++i) {
      int c = tid + i * NT;
      *(uint4*)(lds + (c >> 3) * GEMM_LDK + (c & 7) * 8) = reg[i];
    }
  } else {
#pragma unroll
    for (int b = 0; b < R / 4; ++b) {
      int blk = tid + b * NT;
      int lane = blk & 63, grp = blk >> 6;
      int k4 = lane & 15, mn8 = grp * 4 + (lane >> 4);
      const uint4 r0 = reg[b * 4 + 0], r1 = reg[b * 4 + 1], r2 = reg[b * 4 + 2], r3 = reg[b * 4 + 3];
      const uint32_t a0[4] = {r0.x, r0.y, r0.z, r0.w};
      const uint32_t a1[4] = {r1.x, r1.y, r1.z, r1.w};
      const uint32_t a2[4] = {r2.x, r2.y, r2.z, r2.w};
      const uint32_t a3[4] = {r3.x, r3.y, r3.z, r3.w};
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        // mn = 2d: low halves of k = 0..3 ; mn = 2d+1: high halves
        uint2 lo, hi;
        lo.x = __builtin_amdgcn_perm(a1[d], a0[d], 0x05040100u);
        lo.y = __builtin_amdgcn_perm(a3[d], a2[d], 0x05040100u);
        hi.x = __builtin_amdgcn_perm(a1[d], a0[d], 0x07060302u);
        hi.y = __builtin_amdgcn_perm(a3[d], a2[d], 0x07060302u);
        *(uint2*)(lds + (mn8 * 8 + 2 * d) * GEMM_LDK + k4 * 4) = lo;
        *(uint2*)(lds + (mn8 * 8 + 2 * d + 1) * GEMM_LDK + k4 * 4) = hi;
      }
    }
  }
}

// Tile of output-tile id `bid`: groups of GROUP_M tile rows, column-major
// inside a group (neighbouring ids share operand panels).
__device__ __forceinline__ void tile_of(int64_t bid, int64_t tiles_m, int64_t tiles_n, int& tm, int& tn) {
  constexpr int GROUP_M = 8;
  int64_t group = GROUP_M * tiles_n;
  int64_t gid = bid / group;
  int64_t first = gid * GROUP_M;
  int64_t gsize = tiles_m - first < GROUP_M ? tiles_m - first : GROUP_M;
  int64_t in = bid % group;
  tm = (int)(first + in % gsize);
  tn = (int)(in / gsize);
}

// Workgroups are dispatched round-robin over the 8 XCDs in linear-id order;
// renumbering so that consecutive ids run on one XCD keeps a group's shared
// panels in that XCD's L2.
__device__ __forceinline__ void tile_coords(int64_t tiles_m, int64_t tiles_n, int& tm, int& tn) {
  int64_t nb = (int64_t)gridDim.x;
  int64_t bid = blockIdx.x;
  if (nb % 8 == 0) bid = (bid % 8) * (nb / 8) + bid / 8;  // consecutive ids on one XCD
  tile_of(bid, tiles_m, tiles_n, tm, tn);
}

// Tile and K split of a (tiles, splits) grid.  With few tiles per split
// (at most SPLIT_XCD_MAX_TILES) and a multiple of 8 workgroups, ids are
// renumbered split-major and XCD by XCD: the tiles of one split, which all
// read that split's slice of both operands, then run on one XCD and the
// slice comes through its L2 once instead of through every XCD's.  (A 3x3,
// 64 -> 64 filter gradient over 128 x 32 x 32 pixels, 5 tiles x 48 splits:
// 166 -> 33 MB fetched, 32.2 -> 27.6 us.  With 36 or 144 tiles per split the
// same renumbering was slower, 25.3 -> 26.4 and 25.4 -> 28.0 us, though it
// also cut the fetched bytes 3-4x: those grids are not bound by them.)
constexpr int SPLIT_XCD_MAX_TILES = 16;
__device__ __forceinline__ void split_tile_coords(int64_t tiles_m, int64_t tiles_n, int& tm, int& tn, int& split) {
  const int64_t nt = (int64_t)gridDim.x, total = nt * (int64_t)gridDim.y;
  if (gridDim.y == 1 || nt > SPLIT_XCD_MAX_TILES || total % 8 != 0) {
    split = (int)blockIdx.y;
    tile_coords(tiles_m, tiles_n, tm, tn);
    return;
  }
  int64_t l = (int64_t)blockIdx.x + nt * (int64_t)blockIdx.y;
  l = (l % 8) * (total / 8) + l / 8;
  split = (int)(l / nt);
  tile_of(l % nt, tiles_m, tiles_n, tm, tn);
}

template <class T, class OutT, class SrcA, class SrcB, int BM, int BN, int WM, int WN>
__global__ void __launch_bounds__(WM * WN * 64)
gemm_mfma_kernel(SrcA srcA, SrcB srcB, int64_t M, int64_t N, int64_t K, Epilogue ep) {
  using TS = TileShape<BM, BN, WM, WN>;
  constexpr int NT = TS::NT;
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * TS::LDS_ELEMS];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;

  int tm, tn;
  tile_coords(ceil_div(M, BM), ceil_div(N, BN), tm, tn);
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;
  if (blockIdx.z) {
    shift_batch(srcA, (int)blockIdx.z);
    shift_batch(srcB, (int)blockIdx.z);
    ep.D = (typename OutT::storage*)ep.D + (int64_t)blockIdx.z * ep.bstride_d;
  }

  int64_t kbeg = 0, kend = K;
  if (ep.partial) {
    kbeg = (int64_t)blockIdx.y * ep.k_per_split;
    kend = kbeg + ep.k_per_split < K ? kbeg + ep.k_per_split : K;
  }
  const int nk = (int)ceil_div(kend - kbeg, GEMM_BK);

  float4_t acc[TS::FM][TS::FN];
#pragma unroll
  for (int i = 0; i < TS::FM; ++i)
#pragma unroll
    for (int j = 0; j < TS::FN; ++j) acc[i][j] = (float4_t){0.f, 0.f, 0.f, 0.f};

  uint4 ra[TS::RA], rb[TS::RB];
  if (nk > 0) {
    load_tile<SrcA, BM, NT>(srcA, m0, kbeg, tid, ra);
    load_tile<SrcB, BN, NT>(srcB, n0, kbeg, tid, rb);
    store_tile<SrcA::KC, BM, NT>(smem, tid, ra);
    store_tile<SrcB::KC, BN, NT>(smem + BM * GEMM_LDK, tid, rb);
  }
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) {
      const int64_t kn = kbeg + (int64_t)(kt + 1) * GEMM_BK;
      load_tile<SrcA, BM, NT>(srcA, m0, kn, tid, ra);
      load_tile<SrcB, BN, NT>(srcB, n0, kn, tid, rb);
    }
    const uint16_t* As = smem + cur * TS::LDS_ELEMS;
    const uint16_t* Bs = As + BM * GEMM_LDK;
#pragma unroll
    for (int kk = 0; kk < GEMM_BK / 32; ++kk) {
      uint4 af[TS::FM], bf[TS::FN];
      const int koff = kk * 32 + (lane >> 4) * 8;
#pragma unroll
      for (int i = 0; i < TS::FM; ++i)
        af[i] = *(const uint4*)(As + (wm * TS::WTM + i * 16 + (lane & 15)) * GEMM_LDK + koff);
#pragma unroll
      for (int j = 0; j < TS::FN; ++j)
        bf[j] = *(const uint4*)(Bs + (wn * TS::WTN + j * 16 + (lane & 15)) * GEMM_LDK + koff);
#pragma unroll
      for (int i = 0; i < TS::FM; ++i)
#pragma unroll
        for (int j = 0; j < TS::FN; ++j) acc[i][j] = Mfma<T>::run(bf[j], af[i], acc[i][j]);
    }
    if (more) {
      uint16_t* nxt = smem + (cur ^ 1) * TS::LDS_ELEMS;
      store_tile<SrcA::KC, BM, NT>(nxt, tid, ra);
      store_tile<SrcB::KC, BN, NT>(nxt + BM * GEMM_LDK, tid, rb);
    }
    __syncthreads();
  }

  // lane holds D[m0 + wm*WTM + i*16 + (lane & 15)][n0 + wn*WTN + j*16 + 4*(lane >> 4) + e]
  const int64_t mb = m0 + wm * TS::WTM + (lane & 15);
  const int64_t nb = n0 + wn * TS::WTN + 4 * (lane >> 4);
  if (ep.partial) {
    float* P = ep.partial + (int64_t)blockIdx.y * M * N;
#pragma unroll
    for (int i = 0; i < TS::FM; ++i)
#pragma unroll
      for (int j = 0; j < TS::FN; ++j) {
        const int64_t m = mb + i * 16, n = nb + j * 16;
        if (m >= M) continue;
        float* p = P + m * N + n;
        if ((N & 3) == 0 && n + 4 <= N) {
          *(float4*)p = make_float4(acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (n + e < N) p[e] = acc[i][j][e];
        }
      }
    return;
  }
  if (full_tile_epilogue(ep, m0 + BM <= M && n0 + BN <= N, N)) {
    epilogue_interior<T, OutT, TS::FM, TS::FN>(ep, M, N, mb, nb, acc);
    return;
  }
#pragma unroll
  for (int i = 0; i < TS::FM; ++i)
#pragma unroll
    for (int j = 0; j < TS::FN; ++j)
      epilogue_store4<T, OutT>(ep, M, N, mb + i * 16, nb + j * 16, acc[i][j]);
}

}  // namespace mdnn
