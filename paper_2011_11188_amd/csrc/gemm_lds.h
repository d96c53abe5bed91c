// Fast GEMM mainloop for gfx950: direct global->LDS loads, swizzled LDS tiles
// and transposing LDS reads (section 3.2's D = C + A*B on the CDNA4 matrix
// cores, v_mfma_f32_16x16x32_{f16,bf16}).
//
// Tile 256 x 256 x 64, 8 waves (2 x 4), wave tile 128 x 64, accumulators in
// VGPRs.  Per K step each operand tile (32 KB) is fetched straight into LDS
// with global_load_lds_dwordx4 (each lane's 16 bytes land at M0 + 16*lane, so
// the lane -> global address map chooses the LDS layout); two LDS stages let
// the next tile stream in while the MFMAs consume the current one.
//
// LDS layouts (no padding; XOR swizzles keep the fragment reads free of bank
// conflicts):
//   K-contiguous operand (stored [mn][k] in memory): row r of 128 bytes,
//     logical 16-byte chunk c at slot c ^ ((r >> 1) & 7).  Fragments are
//     ds_read_b128 of 8 consecutive k.
//   MN-contiguous operand (stored [k][mn]): kept in memory order, k-row of
//     512 bytes, logical 32-byte block b at block b ^ g(k),
//     g(k) = (k & 3) | ((k >> 3 & 1) << 2).  Fragments are two
//     ds_read_b64_tr_b16 per 32-deep step: within each 16-lane group, lane j
//     receives element (j mod 4) of the 8-byte rows addressed by lanes j/4,
//     j/4 + 4, j/4 + 8 and j/4 + 12, so lanes addressing k-row kb + i/4,
//     columns c0 + 4*(i mod 4) deliver column c0 + j at 4 consecutive k.
//
// Preconditions (checked by the host): K % 64 == 0; 16-byte aligned bases and
// leading dimensions that are multiples of 8; an MN-contiguous operand's MN
// a multiple of 8; per-lane byte offsets within one K step below 2^32
// (K-contiguous: MN * ld * 2; MN-contiguous: 64 * ld * 2).  Rows / columns past M or N read clamped (valid) addresses
// and only feed outputs that are never stored.
#pragma once

#include "gemm_core.h"

namespace mdnn {
namespace lds {

constexpr int BM = 256, BN = 256, BK = 64, WM = 2, WN = 4;
constexpr int NT = WM * WN * 64;          // 512 threads
constexpr int WTM = BM / WM, WTN = BN / WN;  // 128 x 64 wave tile
constexpr int FM = WTM / 16, FN = WTN / 16;  // 8 x 4 fragments
constexpr int TILE_BYTES = 256 * 64 * 2;     // one operand tile: 32 KB
constexpr int STAGE_BYTES = 2 * TILE_BYTES;  // A + B
constexpr int LDS_BYTES = 2 * STAGE_BYTES;   // two stages: 128 KB
constexpr int LOADS = TILE_BYTES / (NT * 16);  // 16-byte loads per thread per operand: 4

typedef __attribute__((address_space(3))) void lds_void_t;
typedef short short4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int mn_swz(int k) { return (k & 3) | (((k >> 3) & 1) << 2); }

// Per-lane byte offsets (from the operand's K-step base) of the LOADS
// 16-byte chunks this lane fetches for one operand tile.  They do not change
// along K: each K step only moves the scalar base pointer.
template <bool KC>
__device__ __forceinline__ void plan_loads(int64_t ld, int64_t MN, int64_t mn0, int wave, int lane,
                                           uint32_t (&off)[LOADS]) {
#pragma unroll
  for (int i = 0; i < LOADS; ++i) {
    const int blk = wave * LOADS + i;  // 1 KB block of the tile written by this instruction
    if constexpr (KC) {
      const int r = blk * 8 + (lane >> 3);       // tile row (0..255)
      const int c = (lane & 7) ^ ((r >> 1) & 7);  // logical chunk held in this lane's slot
      int64_t row = mn0 + r;
      if (row >= MN) row = MN - 1;
      off[i] = (uint32_t)((row * ld + c * 8) * 2);
    } else {
      const int k = blk * 2 + (lane >> 5);       // tile k-row (0..63)
      const int pc = lane & 31;                  // physical 16-byte chunk in the 512-byte row
      const int b = (pc >> 1) ^ mn_swz(k);       // logical 32-byte block
      int64_t mn = mn0 + b * 16 + (pc & 1) * 8;
      if (mn + 8 > MN) mn = MN - 8;              // MN % 8 == 0 and MN >= 8
      off[i] = (uint32_t)((k * ld + mn) * 2);
    }
  }
}

// One wave-wide load of 16 bytes per lane from kbase + voff into LDS at byte
// address `lds_addr` (wave-uniform): lane l's data lands at lds_addr + 16*l.
// Issued as inline assembly so that the compiler does not treat it as an LDS
// store that later LDS reads must wait for; completion is waited for
// explicitly (s_waitcnt vmcnt) before the barrier that publishes a stage.
// s_nop covers the M0 write -> LDS-DMA read hazard.
__device__ __forceinline__ void dma16(const char* kbase, uint32_t voff, uint32_t lds_addr) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(kbase), "s"(lds_addr)
               : "memory");
}

__device__ __forceinline__ uint32_t lds_address(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}

template <bool KC>
__device__ __forceinline__ void issue_loads(const char* kbase, const uint32_t (&off)[LOADS],
                                            char* tile, int wave) {
  const uint32_t dst = lds_address(tile) + (uint32_t)(wave * LOADS) * 1024u;
#pragma unroll
  for (int i = 0; i < LOADS; ++i) dma16(kbase, off[i], dst + (uint32_t)i * 1024u);
}

// Per-lane constants of the fragment reads.  K-contiguous: row-in-group and
// chunk terms; MN-contiguous (transposing reads): the lane's k-row offset and
// its swizzle term.  They are passed through an empty asm once per K step so
// that the compiler recomputes the few address operations inside the loop
// instead of keeping one address per fragment live across it.
struct LaneFrag {
  uint32_t row_off;  // KC: (lane & 15) * 128;  MN: k_lane * 512 + (i & 3) * 8
  uint32_t swz;      // KC: ((lane & 15) >> 1) & 7;  MN: mn_swz(k_lane)
  uint32_t c;        // KC: lane >> 4;  MN: unused
};

template <bool KC>
__device__ __forceinline__ LaneFrag lane_frag(int lane) {
  LaneFrag f;
  if constexpr (KC) {
    f.row_off = (uint32_t)(lane & 15) * 128u;
    f.swz = (uint32_t)(((lane & 15) >> 1) & 7);
    f.c = (uint32_t)(lane >> 4);
  } else {
    const int k = 8 * (lane >> 4) + ((lane & 15) >> 2);
    f.row_off = (uint32_t)k * 512u + (uint32_t)(lane & 3) * 8u;
    f.swz = (uint32_t)mn_swz(k);
    f.c = 0;
  }
  return f;
}

__device__ __forceinline__ void opaque(LaneFrag& f) {
  asm volatile("" : "+v"(f.row_off), "+v"(f.swz), "+v"(f.c));
}

// Fragment of 16 rows (mn) x 32 k starting at tile row `r0` (a multiple of
// 16), k-step `kk`.  K-contiguous: ds_read_b128 of 8 consecutive k.
// MN-contiguous: two transposing reads, k-rows kb + i/4 and kb + 4 + i/4
// (the swizzle term does not depend on k bit 2 or on kk).
template <bool KC>
__device__ __forceinline__ uint4 fragment(const char* tile, int r0, int kk, const LaneFrag& f) {
  if constexpr (KC) {
    // rows r0 + 0..15: ((r >> 1) & 7) == f.swz since r0 is a multiple of 16
    const uint32_t c = (uint32_t)(kk * 4) + f.c;
    return *(const uint4*)(tile + (uint32_t)r0 * 128u + f.row_off + ((c ^ f.swz) << 4));
  } else {
    const uint32_t b = (uint32_t)(r0 >> 4);
    const char* p0 = tile + (uint32_t)kk * 16384u + f.row_off + ((b ^ f.swz) << 5);
    short4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4_t*)p0);
    short4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) short4_t*)(p0 + 2048));
    uint4 r;
    r.x = (uint32_t)(uint16_t)lo[0] | ((uint32_t)(uint16_t)lo[1] << 16);
    r.y = (uint32_t)(uint16_t)lo[2] | ((uint32_t)(uint16_t)lo[3] << 16);
    r.z = (uint32_t)(uint16_t)hi[0] | ((uint32_t)(uint16_t)hi[1] << 16);
    r.w = (uint32_t)(uint16_t)hi[2] | ((uint32_t)(uint16_t)hi[3] << 16);
    return r;
  }
}

// Ask the scheduler to spread a phase's LDS fragment reads between its 32
// MFMAs (one read, then two MFMAs), instead of bunching them.
template <bool A_KC, bool B_KC>
__device__ __forceinline__ void interleave_reads_mfma() {
  constexpr int reads = FM * (A_KC ? 1 : 2) + FN * (B_KC ? 1 : 2);
#pragma unroll
  for (int r = 0; r < reads; ++r) {
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // one DS read
    __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);  // two MFMAs
  }
  __builtin_amdgcn_sched_group_barrier(0x008, FM * FN - 2 * reads > 0 ? FM * FN - 2 * reads : 0, 0);
}

struct Operand {
  const uint16_t* p;
  int64_t ld, MN;
};

// The two LDS stages are separate objects so that the compiler can prove a
// stage being filled by global_load_lds does not alias the stage being read:
// otherwise it waits for every outstanding load before each fragment read,
// which serialises the loads with the MFMAs.
struct Stages {
  char* a[2];
  char* b[2];
};

// One K step of the pipeline on stage S (tile t); see the kernel.
template <class T, bool A_KC, bool B_KC, int S>
__device__ __forceinline__ void pipeline_step(int t, int nk, const Stages& st, int wave, LaneFrag fa_l,
                                              LaneFrag fb_l,
                                              int wm, int wn, const uint32_t (&sa)[LOADS],
                                              const uint32_t (&sb)[LOADS], const char* a_k0,
                                              int64_t a_step, const char* b_k0, int64_t b_step,
                                              uint4 (&f0a)[FM], uint4 (&f0b)[FN], uint4 (&f1a)[FM],
                                              uint4 (&f1b)[FN], float4_t (&acc)[FM][FN]) {
  opaque(fa_l);
  opaque(fb_l);
#pragma unroll
  for (int i = 0; i < FM; ++i) f1a[i] = fragment<A_KC>(st.a[S], wm * WTM + i * 16, 1, fa_l);
#pragma unroll
  for (int j = 0; j < FN; ++j) f1b[j] = fragment<B_KC>(st.b[S], wn * WTN + j * 16, 1, fb_l);
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::run(f0b[j], f0a[i], acc[i][j]);
  interleave_reads_mfma<A_KC, B_KC>();
  __builtin_amdgcn_s_waitcnt(0);  // this wave's reads of stage S and loads of tile t+1
  __syncthreads();
  if (t + 2 < nk) {
    issue_loads<A_KC>(a_k0 + (int64_t)(t + 2) * a_step, sa, st.a[S], wave);
    issue_loads<B_KC>(b_k0 + (int64_t)(t + 2) * b_step, sb, st.b[S], wave);
  }
  if (t + 1 < nk) {
#pragma unroll
    for (int i = 0; i < FM; ++i) f0a[i] = fragment<A_KC>(st.a[S ^ 1], wm * WTM + i * 16, 0, fa_l);
#pragma unroll
    for (int j = 0; j < FN; ++j) f0b[j] = fragment<B_KC>(st.b[S ^ 1], wn * WTN + j * 16, 0, fb_l);
  }
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = Mfma<T>::run(f1b[j], f1a[i], acc[i][j]);
  interleave_reads_mfma<A_KC, B_KC>();
}

template <class T, class OutT, bool A_KC, bool B_KC>
__global__ void __launch_bounds__(NT, 1)
gemm_lds_kernel(Operand a, Operand b, int64_t M, int64_t N, int64_t K, Epilogue ep) {
  __shared__ __attribute__((aligned(1024))) char lds_a0[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char lds_b0[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char lds_a1[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char lds_b1[TILE_BYTES];
  const Stages st{{lds_a0, lds_a1}, {lds_b0, lds_b1}};
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;

  int tm, tn;
  tile_coords(ceil_div(M, BM), ceil_div(N, BN), tm, tn);
  const int64_t m0 = (int64_t)tm * BM, n0 = (int64_t)tn * BN;

  int64_t kbeg = 0, kend = K;
  if (ep.partial) {
    kbeg = (int64_t)blockIdx.y * ep.k_per_split;
    kend = kbeg + ep.k_per_split < K ? kbeg + ep.k_per_split : K;
  }
  const int nk = (int)((kend - kbeg) / BK);

  uint32_t sa[LOADS], sb[LOADS];
  plan_loads<A_KC>(a.ld, a.MN, m0, wave, lane, sa);
  plan_loads<B_KC>(b.ld, b.MN, n0, wave, lane, sb);
  // byte offset of K step t: K-contiguous operands advance along the row,
  // MN-contiguous ones by whole rows
  const int64_t a_step = (A_KC ? BK : BK * a.ld) * 2;
  const int64_t b_step = (B_KC ? BK : BK * b.ld) * 2;
  const char* a_k0 = (const char*)a.p + (A_KC ? kbeg : kbeg * a.ld) * 2;
  const char* b_k0 = (const char*)b.p + (B_KC ? kbeg : kbeg * b.ld) * 2;

  float4_t acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = (float4_t){0.f, 0.f, 0.f, 0.f};

  // Software pipeline (tile t lives in stage t & 1), per K step:
  //   MFMAs of k-step 0 | LDS reads of k-step 1          (tile t)
  //   wait for this wave's reads and its loads of tile t+1; barrier
  //   issue loads of tile t+2 into the stage tile t leaves free
  //   MFMAs of k-step 1 | LDS reads of k-step 0          (tile t+1)
  // so LDS latency hides behind MFMAs and each tile's global loads have a
  // whole K step to land.
  uint4 f0a[FM], f0b[FN], f1a[FM], f1b[FN];
  const LaneFrag fa_l = lane_frag<A_KC>(lane), fb_l = lane_frag<B_KC>(lane);
  if (nk > 0) {
    issue_loads<A_KC>(a_k0, sa, lds_a0, wave);
    issue_loads<B_KC>(b_k0, sb, lds_b0, wave);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (nk > 1) {
      issue_loads<A_KC>(a_k0 + a_step, sa, lds_a1, wave);
      issue_loads<B_KC>(b_k0 + b_step, sb, lds_b1, wave);
    }
#pragma unroll
    for (int i = 0; i < FM; ++i) f0a[i] = fragment<A_KC>(lds_a0, wm * WTM + i * 16, 0, fa_l);
#pragma unroll
    for (int j = 0; j < FN; ++j) f0b[j] = fragment<B_KC>(lds_b0, wn * WTN + j * 16, 0, fb_l);
  }
  for (int t = 0; t < nk; t += 2) {
    pipeline_step<T, A_KC, B_KC, 0>(t, nk, st, wave, fa_l, fb_l, wm, wn, sa, sb, a_k0, a_step, b_k0,
                                    b_step, f0a, f0b, f1a, f1b, acc);
    if (t + 1 < nk)
      pipeline_step<T, A_KC, B_KC, 1>(t + 1, nk, st, wave, fa_l, fb_l, wm, wn, sa, sb, a_k0, a_step,
                                      b_k0, b_step, f0a, f0b, f1a, f1b, acc);
  }

  const int64_t mb = m0 + wm * WTM + (lane & 15);
  const int64_t nb = n0 + wn * WTN + 4 * (lane >> 4);
  if (ep.partial) {
    float* P = ep.partial + (int64_t)blockIdx.y * M * N;
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
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
      epilogue_store4<T, OutT>(ep, M, N, mb + i * 16, nb + j * 16, acc[i][j]);
}

}  // namespace lds
}  // namespace mdnn
