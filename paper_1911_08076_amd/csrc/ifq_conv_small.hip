// Integrated fixed-point quantized convolution for 8-bit input codes with few
// input channels (c_in <= 4, kh*kw <= 16, c_out <= 64), on gfx950 (MI355X):
// the first layer of a detector, where the generic path gathers every K byte
// with its own index arithmetic and spends far more VALU than the layer's
// HBM traffic costs.
//
// The integer part of Eq. (1) is the implicit GEMM D[co][pixel] =
// sum_k W[co][k] * X[pixel][k] on v_mfma_i32_16x16x64_i8 with K laid out as
// 16 taps x 4 channel bytes: one lane's 16 K bytes of a pixel are four whole
// taps, each a single 32-bit LDS read.
//
//  - A workgroup computes whole output rows [oy0, oy0 + rows) of one image.
//    The input rows they need (with the filter halo) are staged once in LDS
//    as 4-byte pixels (channels past c_in and positions outside the image
//    hold the zero code).
//  - 8-bit codes 0..255 enter the MFMA as x - 128 (XOR 0x80); the epilogue
//    adds back 128 * rowsum(W[co]), exact (the same rule as the generic
//    path). Padded taps and channels carry zero weights.
//  - The +-1 weight fragments of all output channels stay in registers for
//    the whole workgroup; the B fragment of 16 pixels is four LDS reads per
//    lane, and one MFMA per 16 output channels follows.
//  - The epilogue is the generic one (ifq_epilogue.h): thresholds (Eq. 7/8),
//    int32 sums or the dump, codes through an LDS output tile copied out with
//    wide stores.
#include <hip/hip_runtime.h>

#include "ifq_epilogue.h"
#include "ifq_internal.h"

namespace ifq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr int kSmallThreads = 256;
constexpr int kSmallMaxPx = 4096;      // output pixels per workgroup
constexpr int kSmallMaxLds = 64 * 1024;

struct SmallGeom {
  int rows;        // output rows per workgroup
  int tiles;       // workgroups per image
  int rin, win;    // staged input rows and columns
  int out_off;     // LDS offsets: epilogue parameters at 0, output tile,
  int in_off;      // then the staged input
  int lds_bytes;
};

__host__ __device__ inline int small_orow(const ConvLaunch& a, int bm) {
  return a.out_mode == 2 ? bm / 4 : bm;
}

template <int FM>
__global__ __launch_bounds__(kSmallThreads) void conv_small8(ConvLaunch a, SmallGeom sg) {
  constexpr int BM = 16 * FM;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int kg = lane >> 4;     // K bytes 16*kg .. 16*kg+15: taps 4*kg .. 4*kg+3
  const int l16 = lane & 15;

  const int nimg = blockIdx.x / sg.tiles;
  const int oy0 = (blockIdx.x - nimg * sg.tiles) * sg.rows;
  const int rows = a.ho - oy0 < sg.rows ? a.ho - oy0 : sg.rows;
  const int npx = rows * a.wo;
  const int p0 = (nimg * a.ho + oy0) * a.wo;
  const int st = a.stride;
  const int ntaps = a.kh * a.kw;

  // ---- stage the input rows: 4 bytes per pixel, x ^ 0x80, zero code
  // (0x80) outside the image and past c_in ---------------------------------
  uint8_t* tile = lds + sg.in_off;
  const int iy0 = oy0 * st - a.pad;
  const int nin = sg.rin * sg.win;
  for (int e = tid; e < nin; e += kSmallThreads) {
    const int r = e / sg.win;
    const int c = e - r * sg.win;
    const int iy = iy0 + r, ix = c - a.pad;
    uint32_t word = 0x80808080u;
    if ((unsigned)iy < (unsigned)a.h && (unsigned)ix < (unsigned)a.w) {
      const uint8_t* src = a.x + (((int64_t)nimg * a.h + iy) * a.w + ix) * a.cin;
      for (int ch = 0; ch < a.cin; ++ch)
        word ^= (uint32_t)src[ch] << (8 * ch);   // 0x80 ^ x in byte ch
    }
    *reinterpret_cast<uint32_t*>(tile + e * 4) = word;
  }
  stage_epilogue(a, lds, 0, BM);

  // ---- weight fragments (A: rows = output channels), K byte 4*j + c of
  // lane group kg = channel c of tap 4*kg + j -------------------------------
  v4i af[FM];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int co = fm * 16 + l16;
    uint32_t w4[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int tap = 4 * kg + j;
      if (tap < ntaps && co < a.cout_pad)
        for (int c = 0; c < a.cin; ++c)
          w4[j] |= (uint32_t)(uint8_t)a.wgt[(int64_t)co * a.kpad + tap * a.cin + c] << (8 * c);
    }
    af[fm] = v4i{(int)w4[0], (int)w4[1], (int)w4[2], (int)w4[3]};
  }
  // LDS byte offsets of this lane's four taps from a pixel's window corner
  int toff[4];
  bool tval[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int tap = 4 * kg + j;
    tval[j] = tap < ntaps;
    const int ty = tval[j] ? tap / a.kw : 0, tx = tval[j] ? tap - ty * a.kw : 0;
    toff[j] = (ty * sg.win + tx) * 4;
  }
  __syncthreads();

  const int orow = small_orow(a, BM);
  uint8_t* otile = lds + sg.out_off;
  const int nblk = (npx + 15) / 16;
  for (int blk = wave; blk < nblk; blk += kSmallThreads / 64) {
    const int q = blk * 16 + l16;
    const int qc = q < npx ? q : npx - 1;
    const int r = fdiv(qc, a.div_wo);
    const int ox = qc - r * a.wo;
    const uint8_t* win = tile + ((r * st) * sg.win + ox * st) * 4;
    uint32_t b4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
      b4[j] = tval[j] ? *reinterpret_cast<const uint32_t*>(win + toff[j]) : 0x80808080u;
    const v4i bf = v4i{(int)b4[0], (int)b4[1], (int)b4[2], (int)b4[3]};
    v4i acc[FM];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
      acc[fm] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[fm], bf, v4i{0, 0, 0, 0}, 0, 0, 0);
    // lane holds channels 16*g + 4*kg .. +3 of pixel q
    epilogue_lane<FM, 1>(
        a, lds, [&](int g, int, int i) { return acc[g][i]; },
        [&](int g) { return g * 16 + 4 * kg; }, 0, p0,
        [&](int) { return q < npx ? q : -1; }, otile, orow);
  }
  __syncthreads();
  copy_out_tile(a, otile, orow, 0, BM, p0, npx);
}

bool small_geom(const ConvLaunch& a, SmallGeom* g) {
  const int fm = (a.cout + 15) / 16;
  const int bm = 16 * fm;
  const int win = (a.wo - 1) * a.stride + a.kw;
  const int64_t rows_total = (int64_t)a.n * a.ho;
  // enough workgroups for a few per CU, each a whole number of output rows
  int rows = (int)((rows_total + 1023) / 1024);
  if (rows < 1) rows = 1;
  if (rows > a.ho) rows = a.ho;
  for (;; --rows) {
    if (rows < 1) return false;
    const int npx = rows * a.wo;
    const int rin = (rows - 1) * a.stride + a.kh;
    const int epi = epilogue_param_bytes(bm);
    const int out = (npx * small_orow(a, bm) + 15) & ~15;
    const int64_t total = (int64_t)epi + out + (int64_t)rin * win * 4;
    if (npx <= kSmallMaxPx && total <= kSmallMaxLds) {
      g->rows = rows;
      g->tiles = (a.ho + rows - 1) / rows;
      g->rin = rin;
      g->win = win;
      g->out_off = epi;
      g->in_off = epi + out;
      g->lds_bytes = (int)total;
      return true;
    }
  }
}

}  // namespace

bool small8_eligible(const ConvLaunch& a) {
  if (!(a.in_bits == 8 && a.in_layout == IFQ_LAYOUT_I8_NHWC && a.cin >= 1 && a.cin <= 4 &&
        a.kh * a.kw <= 16 && a.cout <= 64 && a.join_kind == IFQ_JOIN_NONE && a.m > 0))
    return false;
  if ((int64_t)a.n * a.h * a.w * a.cin >= ((int64_t)1 << 31)) return false;
  SmallGeom g;
  return small_geom(a, &g);
}

const char* conv_small8_name(const ConvLaunch& a) {
  static const char* names[4] = {"conv_small8<1>", "conv_small8<2>", "conv_small8<3>",
                                 "conv_small8<4>"};
  return names[(a.cout + 15) / 16 - 1];
}

hipError_t launch_conv_small8(const ConvLaunch& a, hipStream_t stream) {
  SmallGeom g;
  if (!small_geom(a, &g)) return hipErrorInvalidValue;
  const dim3 grid(a.n * g.tiles);
  switch ((a.cout + 15) / 16) {
    case 1: hipLaunchKernelGGL((conv_small8<1>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g); break;
    case 2: hipLaunchKernelGGL((conv_small8<2>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g); break;
    case 3: hipLaunchKernelGGL((conv_small8<3>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g); break;
    case 4: hipLaunchKernelGGL((conv_small8<4>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace ifq
