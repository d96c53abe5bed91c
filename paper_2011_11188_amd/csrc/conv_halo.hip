// 3x3 convolutions of 64 input channels (section 2.1's convolution layers;
// stride 1, padding 1) with the input tile's halo in LDS: the forward pass,
// and backward data as the convolution of dy with the filter flipped in
// both spatial axes and its channel axes swapped (padding 3 - 1 - 1 = 1).
//
// A workgroup (4 waves) computes 256 consecutive output pixels (whole image
// rows of one image, or whole images) x 64 output channels.  It stages the
// tile's input rows plus the one-pixel border (zeros outside the image) in
// LDS once; each of the three filter rows then stages that row's three taps
// of the filter (64 output x 64 input channels each; the next row's loads
// are issued before this row's products) and runs its 3 taps x 2 steps of
// 32 channels on the matrix cores, the A fragments read from the halo at the
// tap's offset.  Each input pixel comes from L2 into the CU once per tile
// instead of once per tap.
//
// LDS rows (a pixel's 64 channels, or a forward filter row's 64 input
// channels) are 128 bytes; their eight 16-byte chunks are stored at
// chunk ^ (row & 7), so the 16-byte fragment reads of eight consecutive rows
// touch distinct banks.  Backward data reads the filter with output channels
// contiguous (w[k][r][s][c] over c), so its stage keeps rows of output
// channels in the pipelined GEMM's layout for such operands and forms the B
// fragments with its transposing reads (lds::fragment).
//
// Measured against the implicit GEMM's pipelined kernels (fp16, batch 128,
// fp16 output): 64 -> 64 channels at 32x32, forward 16.7 against 18.2 us.
// Not taken: 128 and 256 input channels (two and four staged chunks: 18.8
// vs 15.1 us at 16x16, 32.1 vs 16.2 us at 8x8; the staging is not
// overlapped with the products), 512-pixel tiles (one workgroup per CU:
// 20.5 us at 32x32).
#include "conv_halo.h"

#include "gemm_lds.h"

namespace mdnn {

namespace {

constexpr int HT = 256;                // threads per workgroup (4 waves)
constexpr int TPX = 256;               // output pixels per workgroup (64 per wave)
constexpr int TCO = 64;                // output channels per workgroup
constexpr int HCH = 64;                // input channels
constexpr int HALO_MAX_PX = 400;       // halo cap (50 KB): two workgroups per CU
constexpr int WSTAGE = 3 * TCO * HCH;  // one filter row's taps, elements
constexpr int FILT_PER = WSTAGE / 8 / HT;
static_assert((WSTAGE / 8) % HT == 0, "filter stage splits evenly");

struct HaloArgs {
  const uint16_t* x;  // convolved tensor [n][h][w][64]: x (forward) or dy (backward data)
  const uint16_t* w;  // forward [cout][3][3][64]; backward data [64][3][3][cout]
  int32_t h, w_img, cout;
  int32_t hr;         // image rows per tile (h when a tile holds whole images)
  int32_t halo_px;    // (TPX / (hr * w)) * (hr + 2) * (w + 2)
  int32_t tiles_n;    // cout / TCO
};

__device__ __forceinline__ int swz(int row, int chunk) { return row * HCH + ((chunk ^ (row & 7)) << 3); }

// the tile's input rows, border included, into the halo
__device__ __forceinline__ void stage_halo(const HaloArgs& a, uint16_t* halo, int64_t img0, int y0, int tid) {
  const int hw2 = a.w_img + 2, per_img = (a.hr + 2) * hw2;
  const int items = a.halo_px * 8;
  constexpr int B = 8;  // loads in flight per thread
  for (int base = 0; base < items; base += HT * B) {
    uint4 v[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int it = base + u * HT + tid;
      v[u] = make_uint4(0u, 0u, 0u, 0u);
      if (it < items) {
        const int hp = it >> 3, c8 = it & 7;
        const int il = hp / per_img, rem = hp - il * per_img;
        const int hy = rem / hw2, hx = rem - hy * hw2;
        const int y = y0 + hy - 1, x = hx - 1;
        if (y >= 0 && y < a.h && x >= 0 && x < a.w_img)
          v[u] = *(const uint4*)(a.x + (((img0 + il) * a.h + y) * a.w_img + x) * HCH + c8 * 8);
      }
    }
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int it = base + u * HT + tid;
      if (it < items) *(uint4*)(halo + swz(it >> 3, it & 7)) = v[u];
    }
  }
}

// filter row tr's three taps for output channels n0..n0 + 63.  Forward:
// item (s, nl, c8) is 8 input channels of output channel n0 + nl, stored as
// rows of input channels.  Backward data: item (s, kl, n8) is output
// channels n0 + 8 n8 .. + 7 of input channel kl at the flipped tap
// (2 - tr, 2 - s), stored as rows of output channels in the transposing
// reads' layout (lds::mn_swz).
template <bool BWD>
__device__ __forceinline__ void load_filter(const HaloArgs& a, uint4 (&v)[FILT_PER], int tr, int64_t n0, int tid) {
#pragma unroll
  for (int u = 0; u < FILT_PER; ++u) {
    const int it = u * HT + tid;
    if constexpr (!BWD) {
      const int c8 = it & 7, nl = (it >> 3) % TCO, s = (it >> 3) / TCO;
      v[u] = *(const uint4*)(a.w + ((n0 + nl) * 9 + tr * 3 + s) * HCH + c8 * 8);
    } else {
      const int n8 = it & 7, kl = (it >> 3) % HCH, s = (it >> 3) / HCH;
      v[u] = *(const uint4*)(a.w + ((int64_t)kl * 9 + (2 - tr) * 3 + (2 - s)) * a.cout + n0 + n8 * 8);
    }
  }
}

template <bool BWD>
__device__ __forceinline__ void store_filter(uint16_t* ws, const uint4 (&v)[FILT_PER], int tid) {
#pragma unroll
  for (int u = 0; u < FILT_PER; ++u) {
    const int it = u * HT + tid;
    int off;
    if constexpr (!BWD) {
      const int c8 = it & 7, nl = (it >> 3) % TCO, s = (it >> 3) / TCO;
      off = s * TCO * HCH + swz(nl, c8);
    } else {
      const int n8 = it & 7, kl = (it >> 3) % HCH, s = (it >> 3) / HCH;
      off = s * TCO * HCH + kl * TCO + (((n8 >> 1) ^ lds::mn_swz<TCO>(kl)) * 16) + (n8 & 1) * 8;
    }
    // (component-wise: a whole-vector copy kept the array in scratch memory)
    *(uint4*)(ws + off) = make_uint4(v[u].x, v[u].y, v[u].z, v[u].w);
  }
}

template <class T, class OutT, bool BWD>
__global__ void __launch_bounds__(HT) conv_halo_kernel(HaloArgs a, int64_t M, Epilogue ep) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[HALO_MAX_PX * HCH + WSTAGE];
  uint16_t* halo = lds;
  uint16_t* wst = lds + HALO_MAX_PX * HCH;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int64_t tm = blockIdx.x / a.tiles_n, n0 = (int64_t)(blockIdx.x % a.tiles_n) * TCO;
  const int64_t m0 = tm * TPX;
  const int64_t hw = (int64_t)a.h * a.w_img;
  const int64_t img0 = m0 / hw;
  const int y0 = (int)((m0 - img0 * hw) / a.w_img);
  const int hw2 = a.w_img + 2, tile_img = a.hr * a.w_img;

  // halo pixel of this lane's output pixel in each of the wave's 4 fragments
  int hb[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int q = wave * 64 + i * 16 + (lane & 15);
    const int il = q / tile_img, rem = q - il * tile_img;
    const int yl = rem / a.w_img, xl = rem - yl * a.w_img;
    hb[i] = (il * (a.hr + 2) + yl) * hw2 + xl;
  }
  const int kc = lane >> 4;
  const lds::LaneFrag fb = lds::lane_frag<false, TCO>(lane);  // backward data's transposing reads

  float4_t acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = (float4_t){0.f, 0.f, 0.f, 0.f};

  uint4 wpre[FILT_PER];
  load_filter<BWD>(a, wpre, 0, n0, tid);
#pragma unroll 1
  for (int tr = 0; tr < 3; ++tr) {
    if (tr > 0) __syncthreads();  // every wave is done with the previous filter row
    store_filter<BWD>(wst, wpre, tid);
    if (tr == 0) stage_halo(a, halo, img0, y0, tid);
    __syncthreads();
    // the next filter row's loads run under this row's products (after the
    // last row: a harmless reload of row 0, unconditional so the registers
    // stay registers)
    load_filter<BWD>(a, wpre, tr < 2 ? tr + 1 : 0, n0, tid);
#pragma unroll
    for (int s = 0; s < 3; ++s)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        const int c = kk * 4 + kc;
        uint4 af[4], bf[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) af[i] = *(const uint4*)(halo + swz(hb[i] + tr * hw2 + s, c));
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if constexpr (!BWD)
            bf[j] = *(const uint4*)(wst + s * TCO * HCH + swz(j * 16 + (lane & 15), c));
          else
            bf[j] = lds::fragment<false, TCO>((const char*)(wst + s * TCO * HCH), j * 16, kk, fb);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[i][j] = Mfma<T>::run(bf[j], af[i], acc[i][j]);
      }
  }

  // lane holds D[m0 + wave*64 + i*16 + (lane & 15)][n0 + j*16 + 4*(lane >> 4) + e]
  const int64_t N = a.cout;
  const int64_t mb = m0 + wave * 64 + (lane & 15);
  const int64_t nb = n0 + 4 * (lane >> 4);
  if (full_tile_epilogue(ep, true, N)) {
    epilogue_interior<T, OutT, 4, 4>(ep, M, N, mb, nb, acc);
    return;
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) epilogue_store4<T, OutT>(ep, M, N, mb + i * 16, nb + j * 16, acc[i][j]);
}

// the tile's image rows and halo pixels, or false when the shape does not qualify
bool halo_plan(const ConvGeom& g, bool bwd, int* hr, int* halo_px) {
  const int cin = bwd ? g.k : g.c, cout = bwd ? g.c : g.k;
  if (g.r != 3 || g.s != 3 || g.pad != 1 || g.ho != g.h || g.wo != g.w || g.n <= 0) return false;
  if (cin != HCH || cout % TCO != 0 || g.w > TPX) return false;
  const int64_t hw = (int64_t)g.h * g.w;
  int rows, ipt;
  if (hw >= TPX) {
    if (TPX % g.w != 0 || g.h % (TPX / g.w) != 0) return false;
    rows = TPX / g.w, ipt = 1;
  } else {
    if (TPX % hw != 0 || g.n % (TPX / hw) != 0) return false;
    rows = g.h, ipt = (int)(TPX / hw);
  }
  const int px = ipt * (rows + 2) * (g.w + 2);
  if (px > HALO_MAX_PX) return false;
  // (global offsets are 64-bit; this bounds the grid)
  if ((int64_t)g.n * hw / TPX * (cout / TCO) > 0x7fffffffLL) return false;
  *hr = rows;
  *halo_px = px;
  return true;
}

template <class T, class OutT>
mdnn_status_t halo_launch(const HaloArgs& a, bool bwd, int64_t M, const Epilogue& ep, hipStream_t st) {
  const dim3 grid((unsigned)(M / TPX * a.tiles_n));
  if (bwd)
    hipLaunchKernelGGL((conv_halo_kernel<T, OutT, true>), grid, dim3(HT), 0, st, a, M, ep);
  else
    hipLaunchKernelGGL((conv_halo_kernel<T, OutT, false>), grid, dim3(HT), 0, st, a, M, ep);
  return check_launch("conv_halo_kernel");
}

}  // namespace

mdnn_status_t conv_halo(const ConvGeom& g, bool bwd, const void* src, const void* w, const Epilogue& ep,
                        mdnn_dtype_t io, mdnn_dtype_t out, hipStream_t st, bool* done) {
  *done = false;
  int hr = 0, px = 0;
  if ((io != MDNN_F16 && io != MDNN_BF16) || !halo_plan(g, bwd, &hr, &px)) return MDNN_SUCCESS;
  if (!aligned(src, 16) || !aligned(w, 16)) return MDNN_SUCCESS;
  HaloArgs a{};
  a.x = (const uint16_t*)src;
  a.w = (const uint16_t*)w;
  a.h = g.h;
  a.w_img = g.w;
  a.cout = bwd ? g.c : g.k;
  a.hr = hr;
  a.halo_px = px;
  a.tiles_n = a.cout / TCO;
  const int64_t M = (int64_t)g.n * g.h * g.w;
  if (io == MDNN_F16)
    MDNN_TRY((out == MDNN_F32 ? halo_launch<F16, F32>(a, bwd, M, ep, st)
                              : halo_launch<F16, F16>(a, bwd, M, ep, st)));
  else
    MDNN_TRY((out == MDNN_F32 ? halo_launch<BF16, F32>(a, bwd, M, ep, st)
                              : halo_launch<BF16, BF16>(a, bwd, M, ep, st)));
  *done = true;
  return MDNN_SUCCESS;
}

}  // namespace mdnn
