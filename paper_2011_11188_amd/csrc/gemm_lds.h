// Pipelined GEMM mainloop for gfx950: direct global->LDS loads, swizzled LDS
// tiles and transposing LDS reads, for section 3.2's D = C + A*B on the CDNA4
// matrix cores (v_mfma_f32_16x16x32_{f16,bf16}, fp32 accumulation), and for
// the implicit-GEMM convolutions of section 2.1 (im2col never materialised).
//
// A block tile is BM x BN x 64 (Tile<>): WM x WN waves, each owning a
// (BM/WM) x (BN/WN) wave tile of 16 x 16 fragments, accumulators in VGPRs.
// Per K step each operand tile (BM or BN rows of 64 k) is fetched straight
// into LDS with LDS-DMA loads (each lane's 16 bytes land at M0 + 16*lane, so
// the lane -> global address map chooses the LDS layout); two LDS stages let
// the next tile stream in while the MFMAs consume the current one.
//
// Operand loaders decide where each lane's 16 bytes come from:
//   MatLoader        plain matrix; global_load_lds with a scalar base per K
//                    step and loop-invariant per-lane offsets.
//   ConvRowsLoader   im2col rows of a convolution input (forward: x, backward
//                    data: dy with mirrored taps); one K step is 64 channels of
//                    one filter tap, so the tap shift is uniform per step.
//   ConvRows32Loader forward im2col rows when c_in is a multiple of 32 only:
//                    a K step is 32 channels of two taps (per-lane tap state),
//                    with MatLoaderRC reading the filter range-checked.
//   TapWeightLoader  the filter read as [tap, c_out] x [c_in] (backward data).
//   ConvColsLoader   shifted input columns of the backward-filter GEMM
//                    (K = output pixels, N = (tap, c_in)).
// The convolution loaders use buffer_load ... lds with a range-checked buffer
// resource: a padded tap or a row past M gets an offset outside the buffer,
// and the hardware returns zeros for it, so padding costs no branches.
//
// LDS layouts (no padding; XOR swizzles keep the fragment reads free of bank
// conflicts):
//   K-contiguous operand (stored [mn][k]): row r of 128 bytes, logical
//     16-byte chunk c at slot c ^ ((r >> 1) & 7).  Fragments are ds_read_b128
//     of 8 consecutive k.
//   MN-contiguous operand of width W (stored [k][mn]): k-rows of 2W bytes in
//     memory order, logical 32-byte block b at block b ^ g(k), with
//     g(k) = (k & 3) | ((k >> 3 & 1) << 2) for W >= 128 and
//     g(k) = (k >> 1 & 1) | ((k >> 3 & 1) << 1) for W = 64.  Fragments are
//     two ds_read_b64_tr_b16 per 32-deep step: within each 16-lane group,
//     lane j receives element (j mod 4) of the 8-byte rows addressed by lanes
//     j/4, j/4 + 4, j/4 + 8 and j/4 + 12, so lanes addressing k-row
//     kb + i/4, columns c0 + 4*(i mod 4) deliver column c0 + j at 4
//     consecutive k.  Each half-wave then touches 8 distinct 32-byte bank
//     groups.
//
// Preconditions (checked by the host): K % 64 == 0 (per split); 16-byte
// aligned bases; plain operands: leading dimensions multiple of 8, an
// MN-contiguous operand's MN a multiple of 8 and >= 8, per-lane byte offsets
// within one K step below 2^32; convolution loaders: channel counts as the
// loader states, buffers below 2^31 bytes.  Rows / columns past M or N read
// clamped (valid) addresses or zeros and only feed outputs that are never
// stored.
#pragma once

#include <type_traits>

#include "gemm_core.h"

namespace mdnn {
namespace lds {

constexpr int BK = 64;
constexpr uint32_t OOB = 0x80000000u;  // buffer offset past every range-checked buffer

typedef short short4_t __attribute__((ext_vector_type(4)));
typedef int int4_t __attribute__((ext_vector_type(4)));

// OCC_: waves per SIMD the register budget is sized for.
template <int BM_, int BN_, int WM_, int WN_, int OCC_ = 2>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, WM = WM_, WN = WN_, OCC = OCC_;
  static constexpr int NW = WM * WN, NT = NW * 64;
  static constexpr int WTM = BM / WM, WTN = BN / WN;
  static constexpr int FM = WTM / 16, FN = WTN / 16;
  static constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
  static constexpr int LA = A_BYTES / (NT * 16), LB = B_BYTES / (NT * 16);  // loads per thread
  static_assert(LA * NT * 16 == A_BYTES && LB * NT * 16 == B_BYTES, "tile is not whole loads");
  static_assert(WTM % 16 == 0 && WTN % 16 == 0, "wave tile is not whole fragments");
  static_assert(BM >= 64 && BN >= 64, "MN-contiguous layouts need widths >= 64");
};

// Block swizzle of an MN-contiguous tile of width W elements (see above).
template <int W>
__device__ __forceinline__ int mn_swz(int k) {
  if constexpr (W >= 128)
    return (k & 3) | (((k >> 3) & 1) << 2);
  else
    return ((k >> 1) & 1) | (((k >> 3) & 1) << 1);
}

// What load i of this lane fetches for an operand tile of width W: for a
// K-contiguous tile, tile row `r` and k offset `c` (a multiple of 8); for an
// MN-contiguous tile, k-row `r` and mn offset `c` (a multiple of 8).  Load i
// of wave w fills the 1 KB block w * L + i of the tile.
struct LoadPos {
  int r, c;
};
template <bool KC, int W, int L>
__device__ __forceinline__ LoadPos load_pos(int wave, int lane, int i) {
  const int blk = wave * L + i;
  if constexpr (KC) {
    const int r = blk * 8 + (lane >> 3);
    return {r, ((lane & 7) ^ ((r >> 1) & 7)) * 8};
  } else {
    constexpr int LPR = W / 8;     // lanes per k-row (16 bytes each)
    constexpr int KPB = 64 / LPR;  // k-rows per 1 KB block
    const int k = blk * KPB + lane / LPR;
    const int pc = lane % LPR;
    return {k, (((pc >> 1) ^ mn_swz<W>(k)) * 16) + (pc & 1) * 8};
  }
}

__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

// One wave-wide load of 16 bytes per lane into LDS at byte address `lds_addr`
// (wave-uniform): lane l's data lands at lds_addr + 16*l.  Issued as inline
// assembly so that the compiler does not treat it as an LDS store that later
// LDS reads must wait for; completion is waited for explicitly (s_waitcnt
// vmcnt) before the barrier that publishes a stage.  s_nop covers the
// M0 write -> LDS-DMA hazard.
__device__ __forceinline__ void dma_global(const char* kbase, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(kbase), "s"(lds_addr)
               : "memory");
}
// Same through a range-checked buffer resource: offsets at or past the
// resource's size read as zero.
__device__ __forceinline__ void dma_buffer(const int4_t& rsrc, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(voff), "s"(rsrc), "s"(lds_addr)
               : "memory");
}

// Raw buffer resource over [p, p + bytes): stride 0, 32-bit data format
// (the word-3 value of untyped buffer accesses on gfx9-family parts).
__device__ __forceinline__ int4_t make_rsrc(const void* p, uint32_t bytes) {
  const uint64_t a = (uint64_t)p;
  int4_t r;
  r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  r[1] = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xffffu));
  r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
  r[3] = 0x00020000;
  return r;
}

// x / d for x * (d - 1) < 2^32, with magic = ceil(2^32 / d) (d >= 2); d == 1
// is passed as magic 0.
__device__ __forceinline__ uint32_t fast_div(uint32_t x, uint32_t magic) {
  return magic ? __umulhi(x, magic) : x;
}

// ---------------------------------------------------------------- loaders

struct MatArgs {
  const void* p;
  int64_t ld, MN;
};

// Plain matrix: K-contiguous ([mn][k], ld >= K) or MN-contiguous ([k][mn]).
template <bool KC_, int W, int L>
struct MatLoader {
  static constexpr bool KC = KC_;
  typedef MatArgs Args;
  const char* base;  // K step 0 of this split
  int64_t step;      // bytes per K step
  uint32_t off[L];

  __device__ __forceinline__ void init(const MatArgs& a, int64_t mn0, int64_t kbeg, int wave, int lane) {
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const LoadPos q = load_pos<KC, W, L>(wave, lane, i);
      if constexpr (KC) {
        int64_t row = mn0 + q.r;
        if (row >= a.MN) row = a.MN - 1;
        off[i] = (uint32_t)((row * a.ld + q.c) * 2);
      } else {
        int64_t mn = mn0 + q.c;
        if (mn + 8 > a.MN) mn = a.MN - 8;
        off[i] = (uint32_t)(((int64_t)q.r * a.ld + mn) * 2);
      }
    }
    step = (KC ? BK : BK * a.ld) * 2;
    base = (const char*)a.p + (KC ? kbeg : kbeg * a.ld) * 2;
  }
  __device__ __forceinline__ void issue(int t, uint32_t dst) {
    const char* kb = base + (int64_t)t * step;
#pragma unroll
    for (int i = 0; i < L; ++i) dma_global(kb, off[i], dst + (uint32_t)i * 1024u);
  }
  // load i alone (loads of one tile may be issued one at a time, in any order)
  static constexpr bool SPLIT_ISSUE = true;
  __device__ __forceinline__ void issue_one(int t, uint32_t dst, int i) {
    dma_global(base + (int64_t)t * step, off[i], dst + (uint32_t)i * 1024u);
  }
};

// im2col rows: GEMM row m = (n, i, j) over an ho x wo grid, GEMM column
// kk = tap * c + ch with tap = tr * s + ts; the element is
// src[n, i + dh, j + dw, ch] (zero outside hs x ws), where (dh, dw) =
// (tr - pad, ts - pad) for the forward pass and (pad - tr, pad - ts) for
// backward data.  Requires c % 64 == 0, so a K step is 64 channels of one tap.
struct ConvRowsArgs {
  const void* p;
  uint32_t bytes;
  int32_t hs, ws, c;  // source grid and channels
  int32_t ho, wo;     // GEMM row grid
  int32_t s, pad, flip;
  int64_t M;
  int32_t r;          // filter rows (ConvRows32Loader only)
};
template <int W, int L>
struct ConvRowsLoader {
  static constexpr bool KC = true;
  static constexpr bool SPLIT_ISSUE = false;  // the per-step state advances once per tile
  typedef ConvRowsArgs Args;
  int4_t rsrc;
  int32_t hs, ws, c, s, pad, flip, cb_n;
  int32_t cb, ts, tr;  // channel block and tap of the next K step (uniform)
  uint32_t base[L];
  int32_t ii[L], jj[L];

  __device__ __forceinline__ void init(const ConvRowsArgs& a, int64_t mn0, int64_t kbeg, int wave, int lane) {
    rsrc = make_rsrc(a.p, a.bytes);
    hs = a.hs, ws = a.ws, c = a.c, s = a.s, pad = a.pad, flip = a.flip;
    cb_n = a.c / 64;
    const int32_t kt = (int32_t)(kbeg / BK), tap = kt / cb_n;
    cb = kt - tap * cb_n;
    tr = tap / a.s;
    ts = tap - tr * a.s;
    const int32_t hw = a.ho * a.wo;
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const LoadPos q = load_pos<true, W, L>(wave, lane, i);
      const int64_t m = mn0 + q.r;
      if (m < a.M) {
        const int32_t mi = (int32_t)m, n = mi / hw, rem = mi - n * hw, i0 = rem / a.wo, j0 = rem - i0 * a.wo;
        ii[i] = i0;
        jj[i] = j0;
        base[i] = (uint32_t)((((n * a.hs + i0) * a.ws + j0) * a.c + q.c) * 2);
      } else {
        ii[i] = -(1 << 20);  // outside the grid for every tap
        jj[i] = 0;
        base[i] = 0;
      }
    }
  }
  __device__ __forceinline__ void issue(int, uint32_t dst) {
    const int32_t dh = flip ? pad - tr : tr - pad, dw = flip ? pad - ts : ts - pad;
    const uint32_t delta = (uint32_t)(((dh * ws + dw) * c + cb * 64) * 2);
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const bool ok = (uint32_t)(ii[i] + dh) < (uint32_t)hs && (uint32_t)(jj[i] + dw) < (uint32_t)ws;
      dma_buffer(rsrc, ok ? base[i] + delta : OOB, dst + (uint32_t)i * 1024u);
    }
    if (++cb == cb_n) {
      cb = 0;
      if (++ts == s) {
        ts = 0;
        ++tr;
      }
    }
  }
};

// im2col rows for a forward convolution whose input channel count is a
// multiple of 32 but not of 64: a K step is two 32-channel half blocks,
// half block h = tap * (c / 32) + b holding channels 32b .. 32b + 31 of one
// tap, so GEMM column kk = tap * c + ch as in the filter's own layout.  The
// K range is padded to whole steps: a half block past the last tap reads
// zeros (its filter columns are then multiplied by zero).
template <int W, int L>
struct ConvRows32Loader {
  static constexpr bool KC = true;
  static constexpr bool SPLIT_ISSUE = false;  // the per-step state advances once per tile
  typedef ConvRowsArgs Args;
  // A lane's k offset within a step (load_pos) depends on its load index
  // only through the index's parity when L is even (block wave * L + i), so
  // the tap state is kept for P = 2 loads, not L.
  static_assert(L == 1 || L % 2 == 0, "tap state per load parity");
  static constexpr int P = L >= 2 ? 2 : 1;
  int4_t rsrc;
  int32_t hs, ws, c, s, r, pad, cpb;
  uint32_t base[L];
  int32_t ii[L], jj[L];
  int32_t tr[P], ts[P], chb[P], ch[P];

  __device__ __forceinline__ void init(const ConvRowsArgs& a, int64_t mn0, int64_t kbeg, int wave, int lane) {
    rsrc = make_rsrc(a.p, a.bytes);
    hs = a.hs, ws = a.ws, c = a.c, s = a.s, r = a.r, pad = a.pad;
    cpb = a.c / 32;
    const int32_t kt = (int32_t)(kbeg / BK);
    const int32_t hw = a.ho * a.wo;
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const LoadPos q = load_pos<true, W, L>(wave, lane, i);
      if (i < P) {
        const int32_t h = 2 * kt + q.c / 32, tap = h / cpb;
        chb[i] = h - tap * cpb;
        tr[i] = tap / a.s;
        ts[i] = tap - tr[i] * a.s;
        ch[i] = q.c % 32;
      }
      const int64_t m = mn0 + q.r;
      if (m < a.M) {
        const int32_t mi = (int32_t)m, n = mi / hw, rem = mi - n * hw, i0 = rem / a.wo, j0 = rem - i0 * a.wo;
        ii[i] = i0;
        jj[i] = j0;
        base[i] = (uint32_t)(((n * a.hs + i0) * a.ws + j0) * a.c * 2);
      } else {
        ii[i] = -(1 << 20);  // outside the grid for every tap
        jj[i] = 0;
        base[i] = 0;
      }
    }
  }
  __device__ __forceinline__ void issue(int, uint32_t dst) {
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const int p = i % P;
      const int32_t dh = tr[p] - pad, dw = ts[p] - pad;
      const bool ok = tr[p] < r && (uint32_t)(ii[i] + dh) < (uint32_t)hs && (uint32_t)(jj[i] + dw) < (uint32_t)ws;
      const uint32_t off = base[i] + (uint32_t)(((dh * ws + dw) * c + chb[p] * 32 + ch[p]) * 2);
      dma_buffer(rsrc, ok ? off : OOB, dst + (uint32_t)i * 1024u);
    }
    // two half blocks on: at most two tap advances (cpb >= 1)
#pragma unroll
    for (int p = 0; p < P; ++p) {
      chb[p] += 2;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        if (chb[p] >= cpb) {
          chb[p] -= cpb;
          if (++ts[p] == s) {
            ts[p] = 0;
            ++tr[p];
          }
        }
      }
    }
  }
};

// A K-contiguous matrix [MN][ld] read through a range-checked buffer
// resource: columns past the end of the last row (a K range padded to whole
// steps) read as zero instead of past the allocation.
struct MatRCArgs {
  const void* p;
  uint32_t bytes;
  int64_t ld, MN;
};
template <int W, int L>
struct MatLoaderRC {
  static constexpr bool KC = true;
  static constexpr bool SPLIT_ISSUE = false;
  typedef MatRCArgs Args;
  int4_t rsrc;
  uint32_t off[L];

  __device__ __forceinline__ void init(const MatRCArgs& a, int64_t mn0, int64_t kbeg, int wave, int lane) {
    rsrc = make_rsrc(a.p, a.bytes);
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const LoadPos q = load_pos<true, W, L>(wave, lane, i);
      int64_t row = mn0 + q.r;
      if (row >= a.MN) row = a.MN - 1;
      off[i] = (uint32_t)((row * a.ld + kbeg + q.c) * 2);
    }
  }
  __device__ __forceinline__ void issue(int t, uint32_t dst) {
#pragma unroll
    for (int i = 0; i < L; ++i) dma_buffer(rsrc, off[i] + (uint32_t)t * (BK * 2), dst + (uint32_t)i * 1024u);
  }
};

// The filter w[c_out][taps][c_in] as the MN-contiguous B operand of the
// backward-data GEMM: k-row kk = tap * c_out + k, column ch -> w[k][tap][ch].
// Requires c_out % 64 == 0 and c_in % 8 == 0.
struct TapWeightArgs {
  const void* p;
  int32_t c_out, taps, c_in;
};
template <int W, int L>
struct TapWeightLoader {
  static constexpr bool KC = false;
  static constexpr bool SPLIT_ISSUE = false;  // the per-step state advances once per tile
  typedef TapWeightArgs Args;
  const char* p;
  int64_t kstride;  // bytes between consecutive k
  int32_t c_in, kb_n, kb, tap;
  uint32_t off[L];

  __device__ __forceinline__ void init(const TapWeightArgs& a, int64_t mn0, int64_t kbeg, int wave, int lane) {
    p = (const char*)a.p;
    const int64_t ld = (int64_t)a.taps * a.c_in;
    kstride = ld * 2;
    c_in = a.c_in;
    kb_n = a.c_out / 64;
    const int32_t kt = (int32_t)(kbeg / BK);
    tap = kt / kb_n;
    kb = kt - tap * kb_n;
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const LoadPos q = load_pos<false, W, L>(wave, lane, i);
      int64_t mn = mn0 + q.c;
      if (mn + 8 > a.c_in) mn = a.c_in - 8;
      off[i] = (uint32_t)(((int64_t)q.r * ld + mn) * 2);
    }
  }
  __device__ __forceinline__ void issue(int, uint32_t dst) {
    const char* kbase = p + (int64_t)kb * 64 * kstride + (int64_t)tap * c_in * 2;
#pragma unroll
    for (int i = 0; i < L; ++i) dma_global(kbase, off[i], dst + (uint32_t)i * 1024u);
    if (++kb == kb_n) {
      kb = 0;
      ++tap;
    }
  }
};

// Shifted input columns of the backward-filter GEMM for a size-preserving
// convolution (ho == h, wo == w): k-row = output pixel p = (n, i, j), column
// nn = tap * c + ch -> x[n, i + tr - pad, j + ts - pad, ch] (zero outside),
// which is x's element p * c + ((tr - pad) * w + ts - pad) * c + ch.
// Requires c % 8 == 0.
struct ConvColsArgs {
  const void* p;
  uint32_t bytes;
  int32_t h, w, c, s, pad;
  uint32_t magic_w, magic_h;  // ceil(2^32 / w), ceil(2^32 / h); 0 for 1
  int64_t N;
};
template <int W, int L>
struct ConvColsLoader {
  static constexpr bool KC = false;
  static constexpr bool SPLIT_ISSUE = false;  // the per-step state advances once per tile
  typedef ConvColsArgs Args;
  int4_t rsrc;
  int32_t h, w;
  uint32_t magic_w, magic_h, row_bytes, pix0;
  int32_t dh[L], dw[L], coff[L], krow[L];

  __device__ __forceinline__ void init(const ConvColsArgs& a, int64_t mn0, int64_t kbeg, int wave, int lane) {
    rsrc = make_rsrc(a.p, a.bytes);
    h = a.h, w = a.w;
    magic_w = a.magic_w, magic_h = a.magic_h;
    row_bytes = (uint32_t)a.c * 2u;
    pix0 = (uint32_t)kbeg;
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const LoadPos q = load_pos<false, W, L>(wave, lane, i);
      const int64_t nn = mn0 + q.c;
      krow[i] = q.r;
      if (nn < a.N) {
        const int32_t tap = (int32_t)nn / a.c, ch = (int32_t)nn - tap * a.c;
        const int32_t tr = tap / a.s, ts = tap - tr * a.s;
        dh[i] = tr - a.pad;
        dw[i] = ts - a.pad;
        coff[i] = ((dh[i] * a.w + dw[i]) * a.c + ch) * 2;
      } else {
        dh[i] = -(1 << 20);  // outside the grid for every pixel
        dw[i] = 0;
        coff[i] = 0;
      }
    }
  }
  __device__ __forceinline__ void issue(int t, uint32_t dst) {
    const uint32_t p0 = pix0 + (uint32_t)t * BK;
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const uint32_t px = p0 + (uint32_t)krow[i];
      const uint32_t q1 = fast_div(px, magic_w);
      const int32_t j = (int32_t)(px - q1 * (uint32_t)w);
      const uint32_t q2 = fast_div(q1, magic_h);
      const int32_t ii = (int32_t)(q1 - q2 * (uint32_t)h);
      const bool ok = (uint32_t)(ii + dh[i]) < (uint32_t)h && (uint32_t)(j + dw[i]) < (uint32_t)w;
      dma_buffer(rsrc, ok ? px * row_bytes + (uint32_t)coff[i] : OOB, dst + (uint32_t)i * 1024u);
    }
  }
};

// ------------------------------------------------------------- fragments

// Per-lane constants of the fragment reads.  K-contiguous: row-in-group and
// chunk terms; MN-contiguous (transposing reads): the lane's k-row offset and
// its swizzle term.  They are passed through an empty asm once per K step so
// that the compiler recomputes the few address operations inside the loop
// instead of keeping one address per fragment live across it.
struct LaneFrag {
  uint32_t row_off;  // KC: (lane & 15) * 128;  MN: k_lane * 2W + (lane & 3) * 8
  uint32_t swz;      // KC: ((lane & 15) >> 1) & 7;  MN: g(k_lane)
  uint32_t c;        // KC: lane >> 4;  MN: unused
};

template <bool KC, int W>
__device__ __forceinline__ LaneFrag lane_frag(int lane) {
  LaneFrag f;
  if constexpr (KC) {
    f.row_off = (uint32_t)(lane & 15) * 128u;
    f.swz = (uint32_t)(((lane & 15) >> 1) & 7);
    f.c = (uint32_t)(lane >> 4);
  } else {
    const int k = 8 * (lane >> 4) + ((lane & 15) >> 2);
    f.row_off = (uint32_t)k * (2u * W) + (uint32_t)(lane & 3) * 8u;
    f.swz = (uint32_t)mn_swz<W>(k);
    f.c = 0;
  }
  return f;
}

__device__ __forceinline__ void opaque(LaneFrag& f) {
  asm volatile("" : "+v"(f.row_off), "+v"(f.swz), "+v"(f.c));
}

// Fragment of 16 rows (mn) x 32 k starting at tile row `r0` (a multiple of
// 16), k-step `kk` (0 or 1).  K-contiguous: ds_read_b128 of 8 consecutive k.
// MN-contiguous: two transposing reads, k-rows kb + i/4 and kb + 4 + i/4
// (the swizzle term does not depend on k bit 2 or on kk).
template <bool KC, int W>
__device__ __forceinline__ uint4 fragment(const char* tile, int r0, int kk, const LaneFrag& f) {
  if constexpr (KC) {
    // rows r0 + 0..15: ((r >> 1) & 7) == f.swz since r0 is a multiple of 16
    const uint32_t c = (uint32_t)(kk * 4) + f.c;
    return *(const uint4*)(tile + (uint32_t)r0 * 128u + f.row_off + ((c ^ f.swz) << 4));
  } else {
    constexpr uint32_t ROWB = 2u * W;
    const uint32_t b = (uint32_t)(r0 >> 4);
    const char* p0 = tile + (uint32_t)kk * (32u * ROWB) + f.row_off + ((b ^ f.swz) << 5);
    short4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4_t*)p0);
    short4_t hi =
        __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4_t*)(p0 + 4 * ROWB));
    uint4 r;
    r.x = (uint32_t)(uint16_t)lo[0] | ((uint32_t)(uint16_t)lo[1] << 16);
    r.y = (uint32_t)(uint16_t)lo[2] | ((uint32_t)(uint16_t)lo[3] << 16);
    r.z = (uint32_t)(uint16_t)hi[0] | ((uint32_t)(uint16_t)hi[1] << 16);
    r.w = (uint32_t)(uint16_t)hi[2] | ((uint32_t)(uint16_t)hi[3] << 16);
    return r;
  }
}

// Ask the scheduler to spread a phase's LDS fragment reads between its
// MFMAs: one read then two MFMAs while MFMAs last (then the remaining MFMAs),
// or an even spread when there are fewer than two MFMAs per read.
template <int R, int READS, int MFMAS>
__device__ __forceinline__ void spread_reads() {
  if constexpr (R < READS) {
    constexpr int n = (R < MFMAS % READS) ? MFMAS / READS + 1 : MFMAS / READS;
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one DS read
    if constexpr (n > 0) __builtin_amdgcn_sched_group_barrier(0x008, n, 0);  // n MFMAs
    spread_reads<R + 1, READS, MFMAS>();
  }
}
template <int READS, int MFMAS>
__device__ __forceinline__ void interleave_reads_mfma() {
  if constexpr (2 * READS <= MFMAS) {
#pragma unroll
    for (int r = 0; r < READS; ++r) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one DS read
      __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // two MFMAs
    }
    if constexpr (MFMAS > 2 * READS) __builtin_amdgcn_sched_group_barrier(0x008, MFMAS - 2 * READS, 0);
  } else {
    spread_reads<0, READS, MFMAS>();
  }
}

// LDS instructions of fragments F0 .. F1-1 (A's FM fragments, then B's)
template <bool A_KC, bool B_KC, int FM>
constexpr int chunk_reads(int f0, int f1) {
  int r = 0;
  for (int f = f0; f < f1; ++f) r += (f < FM ? (A_KC ? 1 : 2) : (B_KC ? 1 : 2));
  return r;
}

// LDS stages are separate objects so that the compiler can prove a stage
// being filled by LDS-DMA does not alias the stage being read: otherwise it
// waits for every outstanding load before each fragment read, which
// serialises the loads with the MFMAs.
template <int NS>
struct Stages {
  char* a[NS];
  char* b[NS];
};

template <class TL>
struct Frags {
  uint4 a[TL::FM], b[TL::FN];
};

// s_waitcnt with vmcnt <= n (this wave's LDS-DMA loads) and lgkmcnt == 0.
template <int N>
__device__ __forceinline__ void wait_vm_lgkm0() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4));
}
// Wait until the oldest outstanding tile has landed while `ahead` newer
// tiles (at most A) may still be in flight; LPT = LDS-DMA instructions per
// thread per tile.
template <int A, int LPT>
__device__ __forceinline__ void wait_tiles(int ahead) {
  if constexpr (A > 0) {
    if (ahead >= A) {
      wait_vm_lgkm0<A * LPT>();
      return;
    }
    wait_tiles<A - 1, LPT>(ahead);
  } else {
    wait_vm_lgkm0<0>();
  }
}

template <class T, class TL, class LA, class LB, int C>
__device__ __forceinline__ void spread_chunk(int tn, uint32_t dst_a, uint32_t dst_b, const char* sa, const char* sb,
                                             int wm, int wn, const LaneFrag& fa_l, const LaneFrag& fb_l, LA& la, LB& lb,
                                             Frags<TL>& f0, const Frags<TL>& f1, float4_t (&acc)[TL::FM][TL::FN]);

// One K step of the pipeline: tile t in stage S = t % NS (see the kernel).
// f0 holds k-step 0 of tile t on entry and k-step 0 of tile t+1 on exit.
// CHECK = false is the steady state (t + NS < nk): no conditions, so each
// half step is one basic block whose LDS reads interleave with its MFMAs.
template <class T, class TL, int NS, class LA, class LB, int S, bool CHECK>
__device__ __forceinline__ void pipeline_step(int t, int nk, const Stages<NS>& st, int wave, LaneFrag fa_l,
                                              LaneFrag fb_l, int wm, int wn, LA& la, LB& lb, Frags<TL>& f0,
                                              Frags<TL>& f1, float4_t (&acc)[TL::FM][TL::FN]) {
  constexpr int FM = TL::FM, FN = TL::FN;
  constexpr int READS = FM * (LA::KC ? 1 : 2) + FN * (LB::KC ? 1 : 2);
  constexpr int S1 = (S + 1) % NS;
  opaque(fa_l);
  opaque(fb_l);
#pragma unroll
  for (int i = 0; i < FM; ++i) f1.a[i] = fragment<LA::KC, TL::BM>(st.a[S], wm * TL::WTM + i * 16, 1, fa_l);
#pragma unroll
  for (int j = 0; j < FN; ++j) f1.b[j] = fragment<LB::KC, TL::BN>(st.b[S], wn * TL::WTN + j * 16, 1, fb_l);
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::run(f0.b[j], f0.a[i], acc[i][j]);
  interleave_reads_mfma<READS, FM * FN>();
  // this wave's reads of stage S, and its loads of tile t+1
  if constexpr (CHECK) {
    const int newest = t + NS - 1 < nk - 1 ? t + NS - 1 : nk - 1;
    wait_tiles<NS - 2, TL::LA + TL::LB>(newest - (t + 1));
  } else {
    wait_vm_lgkm0<(NS - 2) * (TL::LA + TL::LB)>();
  }
  __syncthreads();
  if constexpr (!CHECK && LA::SPLIT_ISSUE && LB::SPLIT_ISSUE) {
    spread_chunk<T, TL, LA, LB, 0>(t + NS, lds_address(st.a[S]) + (uint32_t)(wave * TL::LA) * 1024u,
                                   lds_address(st.b[S]) + (uint32_t)(wave * TL::LB) * 1024u, st.a[S1], st.b[S1], wm,
                                   wn, fa_l, fb_l, la, lb, f0, f1, acc);
    return;
  }
  if (!CHECK || t + NS < nk) {
    la.issue(t + NS, lds_address(st.a[S]) + (uint32_t)(wave * TL::LA) * 1024u);
    lb.issue(t + NS, lds_address(st.b[S]) + (uint32_t)(wave * TL::LB) * 1024u);
  }
  if (!CHECK || t + 1 < nk) {
#pragma unroll
    for (int i = 0; i < FM; ++i) f0.a[i] = fragment<LA::KC, TL::BM>(st.a[S1], wm * TL::WTM + i * 16, 0, fa_l);
#pragma unroll
    for (int j = 0; j < FN; ++j) f0.b[j] = fragment<LB::KC, TL::BN>(st.b[S1], wn * TL::WTN + j * 16, 0, fb_l);
  }
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::run(f1.b[j], f1.a[i], acc[i][j]);
  interleave_reads_mfma<READS, FM * FN>();
}

// Second half of a steady-state K step with the LDS-DMA loads of tile t+NS
// spread over it: chunk C issues load C (A's loads, then B's), then its
// share of the next tile's fragment reads and of this k-step's MFMAs.
// Issuing all of a step's loads at once right after the barrier stalls the
// issuing waves while the loads queue; spread out, they hide behind MFMAs.
template <class T, class TL, class LA, class LB, int C>
__device__ __forceinline__ void spread_chunk(int tn, uint32_t dst_a, uint32_t dst_b, const char* sa, const char* sb,
                                             int wm, int wn, const LaneFrag& fa_l, const LaneFrag& fb_l, LA& la, LB& lb,
                                             Frags<TL>& f0, const Frags<TL>& f1, float4_t (&acc)[TL::FM][TL::FN]) {
  constexpr int FM = TL::FM, FN = TL::FN, NL = TL::LA + TL::LB;
  if constexpr (C < NL) {
    if constexpr (C < TL::LA)
      la.issue_one(tn, dst_a, C);
    else
      lb.issue_one(tn, dst_b, C - TL::LA);
    __builtin_amdgcn_sched_barrier(0);
    constexpr int NFR = FM + FN, F0 = C * NFR / NL, F1 = (C + 1) * NFR / NL;
    constexpr int MF = FM * FN, M0 = C * MF / NL, M1 = (C + 1) * MF / NL;
    int reads = 0;
#pragma unroll
    for (int f = F0; f < F1; ++f) {
      if (f < FM) {
        f0.a[f] = fragment<LA::KC, TL::BM>(sa, wm * TL::WTM + f * 16, 0, fa_l);
        reads += LA::KC ? 1 : 2;
      } else {
        f0.b[f - FM] = fragment<LB::KC, TL::BN>(sb, wn * TL::WTN + (f - FM) * 16, 0, fb_l);
        reads += LB::KC ? 1 : 2;
      }
    }
    (void)reads;
#pragma unroll
    for (int m = M0; m < M1; ++m) acc[m / FN][m % FN] = Mfma<T>::run(f1.b[m % FN], f1.a[m / FN], acc[m / FN][m % FN]);
    constexpr int R = chunk_reads<LA::KC, LB::KC, FM>(F0, F1);
    if constexpr (R > 0) interleave_reads_mfma<R, M1 - M0>();
    __builtin_amdgcn_sched_barrier(0);
    spread_chunk<T, TL, LA, LB, C + 1>(tn, dst_a, dst_b, sa, sb, wm, wn, fa_l, fb_l, la, lb, f0, f1, acc);
  }
}

// Steps t + J .. t + U - 1 of one unrolled round, U = lcm(NS, 2): the stage
// index J % NS is a compile-time constant.
template <class T, class TL, int NS, class LA, class LB, int J, int U, bool CHECK>
__device__ __forceinline__ void pipeline_round(int t, int nk, const Stages<NS>& st, int wave, LaneFrag fa_l,
                                               LaneFrag fb_l, int wm, int wn, LA& la, LB& lb, Frags<TL>& f0,
                                               Frags<TL>& f1, float4_t (&acc)[TL::FM][TL::FN]) {
  if constexpr (J < U) {
    if (CHECK && t + J >= nk) return;
    pipeline_step<T, TL, NS, LA, LB, J % NS, CHECK>(t + J, nk, st, wave, fa_l, fb_l, wm, wn, la, lb, f0, f1, acc);
    pipeline_round<T, TL, NS, LA, LB, J + 1, U, CHECK>(t, nk, st, wave, fa_l, fb_l, wm, wn, la, lb, f0, f1, acc);
  }
}

// The SGD update of a square tile's weights in place of storing its weight
// gradient (mdnn_gemm_tn_update), with g = alpha * acc per element exactly
// the arithmetic of the SGD kernels (g / scale with a scaler, v = fma(mu, v,
// g) and w = fma(-lr, v, w), or w = fma(-lr, g, w), then the working copy
// rounded from w), so the result is bitwise that of storing the gradient
// and updating from it; a set scaler->reserved (an earlier producer of the
// step saw Inf or NaN) skips it.  The accumulators go through LDS (the A
// stage of the pipeline, A_BYTES = 32 rows x BN fp32) 32 rows at a time, so
// that each wave then reads, updates and writes whole 16-byte-per-lane runs
// of those rows: the weight, momentum and working-copy traffic (18 bytes per
// element) is contiguous, where the accumulator layout would split it into
// 64-byte pieces.  LDS slot s of row r holds float4 s ^ (r & 15) (the 16
// lanes writing one column block hit different banks).
struct UpdateArgs {
  float S, alpha;
  bool mom;
};
template <class TL>
struct UpdateShape {
  static constexpr int S4 = TL::BN / 4;                  // float4 slots per row
  static constexpr int ROWS = TL::A_BYTES / (TL::BN * 4);  // rows per pass
  static constexpr int PER = ROWS * S4 / TL::NT;          // float4 per thread per pass
  static_assert(ROWS == 32 && ROWS * S4 == PER * TL::NT && TL::WTM % ROWS == 0, "update staging shape");
};
typedef float upd_f4v __attribute__((ext_vector_type(4)));

// this thread's weight and momentum quads of pass P
template <class TL, int P>
__device__ __forceinline__ void update_loads(const Epilogue& ep, int64_t m0, int64_t n0, int tid, bool mom,
                                             upd_f4v (&wq)[UpdateShape<TL>::PER],
                                             upd_f4v (&vq)[UpdateShape<TL>::PER]) {
  typedef UpdateShape<TL> U;
#pragma unroll
  for (int k = 0; k < U::PER; ++k) {
    const int idx = tid + k * TL::NT, r = idx / U::S4, s = idx % U::S4;
    const int64_t e = (m0 + P * U::ROWS + r) * ep.ldd + n0 + 4 * s;
    wq[k] = *(const upd_f4v*)(ep.upd_w + e);
    if (mom) vq[k] = *(const upd_f4v*)(ep.upd_v + e);
  }
}

// Pass P: issue its weight and momentum loads, stage its rows, read them
// back in row order (the loads' latency hides behind the staging and the
// barriers), then update.
template <class T, class TL, int P, int FM, int FN>
__device__ __forceinline__ void update_pass(const Epilogue& ep, float4* st, int64_t m0, int64_t n0, int wm, int wn,
                                            int lane, int tid, const float4_t (&acc)[FM][FN], const UpdateArgs& u) {
  typedef uint32_t u2v __attribute__((ext_vector_type(2)));
  typedef UpdateShape<TL> U;
  constexpr int S4 = U::S4, ROWS = U::ROWS, PER = U::PER;
  if constexpr (P * ROWS < TL::BM) {
    upd_f4v wq[PER], vq[PER];
    update_loads<TL, P>(ep, m0, n0, tid, u.mom, wq, vq);
    // the waves whose rows fall in this pass (wave row WMP) stage their two
    // fragment rows I0, I0 + 1
    constexpr int WMP = P * ROWS / TL::WTM, I0 = (P * ROWS - WMP * TL::WTM) / 16;
    if (wm == WMP) {
#pragma unroll
      for (int ii = 0; ii < 2; ++ii)
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int r = ii * 16 + (lane & 15);
          const int s = (wn * TL::WTN + j * 16) / 4 + (lane >> 4);
          st[r * S4 + (s ^ (r & 15))] =
              make_float4(acc[I0 + ii][j][0], acc[I0 + ii][j][1], acc[I0 + ii][j][2], acc[I0 + ii][j][3]);
        }
    }
    __syncthreads();
    float4 gq[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int idx = tid + k * TL::NT, r = idx / S4, s = idx % S4;
      gq[k] = st[r * S4 + (s ^ (r & 15))];
    }
    __syncthreads();  // the next pass may overwrite the stage
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int idx = tid + k * TL::NT, r = idx / S4, s = idx % S4;
      const int64_t e = (m0 + P * ROWS + r) * ep.ldd + n0 + 4 * s;
      const float ga[4] = {gq[k].x, gq[k].y, gq[k].z, gq[k].w};
      float w[4] = {wq[k][0], wq[k][1], wq[k][2], wq[k][3]};
      float v[4] = {0.f, 0.f, 0.f, 0.f};
      if (u.mom) v[0] = vq[k][0], v[1] = vq[k][1], v[2] = vq[k][2], v[3] = vq[k][3];
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        float g = ga[c] * u.alpha;
        if (ep.upd_sc) g = g / u.S;
        if (u.mom) {
          v[c] = fmaf(ep.upd_mu, v[c], g);
          w[c] = fmaf(-ep.upd_lr, v[c], w[c]);
        } else {
          w[c] = fmaf(-ep.upd_lr, g, w[c]);
        }
      }
      *(upd_f4v*)(ep.upd_w + e) = (upd_f4v){w[0], w[1], w[2], w[3]};
      if (u.mom) *(upd_f4v*)(ep.upd_v + e) = (upd_f4v){v[0], v[1], v[2], v[3]};
      if (ep.upd_lp) {
        u2v q;
        q[0] = (uint32_t)from_f<T>(w[0]) | ((uint32_t)from_f<T>(w[1]) << 16);
        q[1] = (uint32_t)from_f<T>(w[2]) | ((uint32_t)from_f<T>(w[3]) << 16);
        *(u2v*)((typename T::storage*)ep.upd_lp + e) = q;
      }
    }
    update_pass<T, TL, P + 1>(ep, st, m0, n0, wm, wn, lane, tid, acc, u);
  }
}

template <class T, class TL, int FM, int FN>
__device__ __forceinline__ void update_epilogue(const Epilogue& ep, char* lds, int64_t m0, int64_t n0, int wm, int wn,
                                                int lane, int tid, const float4_t (&acc)[FM][FN]) {
  if (ep.upd_sc && ep.upd_sc->reserved) return;     // uniform: read by every thread alike
  UpdateArgs u;
  u.S = ep.upd_sc ? ep.upd_sc->scale : 1.0f;
  u.alpha = ep.alpha_dev ? ep.alpha * *ep.alpha_dev : ep.alpha;
  u.mom = ep.upd_v != nullptr;
  __syncthreads();  // the mainloop's last fragment reads are done
  update_pass<T, TL, 0>(ep, (float4*)lds, m0, n0, wm, wn, lane, tid, acc, u);
}

// D = epilogue(op(A) op(B)), or fp32 split partials when ep.partial is set
// (grid.y = split index, each split ep.k_per_split deep).  NS LDS stages
// (2..4) of A_BYTES + B_BYTES each.
template <class T, class OutT, class TL, int NS, class LA, class LB>
__global__ void __launch_bounds__(TL::NT, TL::OCC)
gemm_lds_kernel(typename LA::Args aa, typename LB::Args ba, int64_t M, int64_t N, int64_t K, Epilogue ep) {
  static_assert(NS >= 2 && NS <= 4, "2 to 4 stages");
  static_assert(NS * (TL::A_BYTES + TL::B_BYTES) + 2 * (4 - NS) <= 160 * 1024, "LDS budget");
  __shared__ __attribute__((aligned(1024))) char lds_a0[TL::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char lds_b0[TL::B_BYTES];
  __shared__ __attribute__((aligned(1024))) char lds_a1[TL::A_BYTES];
  __shared__ __attribute__((aligned(1024))) char lds_b1[TL::B_BYTES];
  // stages beyond NS shrink to single unaligned bytes
  __shared__ __attribute__((aligned(NS > 2 ? 1024 : 1))) char lds_a2[NS > 2 ? TL::A_BYTES : 1];
  __shared__ __attribute__((aligned(NS > 2 ? 1024 : 1))) char lds_b2[NS > 2 ? TL::B_BYTES : 1];
  __shared__ __attribute__((aligned(NS > 3 ? 1024 : 1))) char lds_a3[NS > 3 ? TL::A_BYTES : 1];
  __shared__ __attribute__((aligned(NS > 3 ? 1024 : 1))) char lds_b3[NS > 3 ? TL::B_BYTES : 1];
  char* const all_a[4] = {lds_a0, lds_a1, lds_a2, lds_a3};
  char* const all_b[4] = {lds_b0, lds_b1, lds_b2, lds_b3};
  Stages<NS> st;
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    st.a[s] = all_a[s];
    st.b[s] = all_b[s];
  }
  constexpr int FM = TL::FM, FN = TL::FN;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / TL::WN, wn = wave % TL::WN;

  int tm, tn, split;
  split_tile_coords(ceil_div(M, TL::BM), ceil_div(N, TL::BN), tm, tn, split);
  const int64_t m0 = (int64_t)tm * TL::BM, n0 = (int64_t)tn * TL::BN;

  int64_t kbeg = 0, kend = K;
  if (ep.partial) {
    kbeg = (int64_t)split * ep.k_per_split;
    kend = kbeg + ep.k_per_split < K ? kbeg + ep.k_per_split : K;
  }
  const int nk = (int)((kend - kbeg) / BK);

  LA la;
  LB lb;
  la.init(aa, m0, kbeg, wave, lane);
  lb.init(ba, n0, kbeg, wave, lane);
  const uint32_t wa = (uint32_t)(wave * TL::LA) * 1024u, wb = (uint32_t)(wave * TL::LB) * 1024u;

  float4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = (float4_t){0.f, 0.f, 0.f, 0.f};

  // Software pipeline (tile t lives in stage t % NS), per K step:
  //   MFMAs of k-step 0 | LDS reads of k-step 1          (tile t)
  //   wait for this wave's reads and its loads of tile t+1; barrier
  //   issue loads of tile t+NS into the stage tile t leaves free
  //   MFMAs of k-step 1 | LDS reads of k-step 0          (tile t+1)
  // so LDS latency hides behind MFMAs and each tile's global loads have
  // NS-1 K steps to land.  Loaders are issued tiles 0, 1, 2, ... in order.
  Frags<TL> f0, f1;
  const LaneFrag fa_l = lane_frag<LA::KC, TL::BM>(lane), fb_l = lane_frag<LB::KC, TL::BN>(lane);
  if (nk > 0) {
#pragma unroll
    for (int s = 0; s < NS; ++s)
      if (s < nk) {
        la.issue(s, lds_address(st.a[s]) + wa);
        lb.issue(s, lds_address(st.b[s]) + wb);
      }
    wait_tiles<NS - 1, TL::LA + TL::LB>((nk < NS ? nk : NS) - 1);  // tile 0 landed
    __syncthreads();
#pragma unroll
    for (int i = 0; i < FM; ++i) f0.a[i] = fragment<LA::KC, TL::BM>(st.a[0], wm * TL::WTM + i * 16, 0, fa_l);
#pragma unroll
    for (int j = 0; j < FN; ++j) f0.b[j] = fragment<LB::KC, TL::BN>(st.b[0], wn * TL::WTN + j * 16, 0, fb_l);
  }
  constexpr int U = NS % 2 == 0 ? NS : 2 * NS;
  // the unconditional steady state needs a few more live registers; with two
  // MN-contiguous operands (more address terms) the 256 x 256 tile would spill
  constexpr bool STEADY = LA::KC || LB::KC || TL::FM * TL::FN < 32;
  int t = 0;
  if constexpr (STEADY)
    for (; t + U - 1 + NS < nk; t += U)  // every step of the round still issues a tile
      pipeline_round<T, TL, NS, LA, LB, 0, U, false>(t, nk, st, wave, fa_l, fb_l, wm, wn, la, lb, f0, f1, acc);
  for (; t < nk; t += U)
    pipeline_round<T, TL, NS, LA, LB, 0, U, true>(t, nk, st, wave, fa_l, fb_l, wm, wn, la, lb, f0, f1, acc);

  const int64_t mb = m0 + wm * TL::WTM + (lane & 15);
  const int64_t nb = n0 + wn * TL::WTN + 4 * (lane >> 4);
  if (ep.partial) {
    float* P = ep.partial + (int64_t)split * M * N;
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j) {
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
  // interior tiles with 4-aligned rows everywhere take the straight-line store
  // the fused SGD update (plain TN products with an fp32 gradient; every
  // tile interior, which the host has checked)
  constexpr bool UPD = std::is_same<OutT, F32>::value && std::is_same<LA, MatLoader<false, TL::BM, TL::LA>>::value &&
                       std::is_same<LB, MatLoader<false, TL::BN, TL::LB>>::value && TL::BM == TL::BN;
  if constexpr (UPD) {
    if (ep.upd_w) {
      update_epilogue<T, TL>(ep, lds_a0, m0, n0, wm, wn, lane, tid, acc);
      return;
    }
  }
  if (full_tile_epilogue(ep, m0 + TL::BM <= M && n0 + TL::BN <= N, N)) {
    epilogue_interior<T, OutT, FM, FN>(ep, M, N, mb, nb, acc);
    return;
  }
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) epilogue_store4<T, OutT>(ep, M, N, mb + i * 16, nb + j * 16, acc[i][j]);
}

// Plain-GEMM configurations: 256 x 256 tile with 8 waves of 128 x 64, and
// for problems with fewer tiles, 128 x 128 with 4 waves of 64 x 64 (each
// wave reads 8 fragments from LDS per 16 MFMAs where a 64 x 32 wave reads 6
// per 8; two such workgroups share a CU; against 8 waves of 64 x 32 at four
// workgroups per CU: TN 2048 x 4096 x 4096 89.2 -> 69.3 us, NN 4096 x 2048 x
// 1024 23.5 -> 22.6 us).
typedef Tile<256, 256, 2, 4> Tile256;
typedef Tile<128, 128, 2, 2, 2> Tile128;

}  // namespace lds
}  // namespace mdnn
