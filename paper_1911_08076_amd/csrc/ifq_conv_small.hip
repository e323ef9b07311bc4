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
//  - 2-bit codes (the detector's case): each lane's four output channels
//    are fixed for the whole workgroup, so their threshold records, signs
//    and 128 * rowsum corrections sit in registers; the compares are packed
//    16-bit (|sum| <= 255 * 64 < 2^15), and a lane's byte (or 4 bytes) of
//    codes goes straight to HBM, the four lanes of a pixel writing adjacent
//    bytes. Other outputs (int32 sums, wider codes) take the generic epilogue
//    of ifq_epilogue.h through an LDS output tile.
#include <hip/hip_runtime.h>

#include "ifq_epilogue.h"
#include "ifq_internal.h"
#include "ifq_mfma_common.h"

namespace ifq {
namespace {

constexpr int kSmallThreads = 256;
constexpr int kSmallMaxPx = 4096;      // output pixels per workgroup
constexpr int kSmallMaxLds = 64 * 1024;

struct SmallGeom {
  int rows;        // output rows per workgroup
  int tiles;       // workgroups per image
  int rin, win;    // staged input rows and columns
  FastDiv div_win; // division by win
  int out_off;     // LDS offsets: epilogue parameters at 0, output tile,
  int in_off;      // the staged input, then the raw input bytes
  int raw_off;
  int vec;         // input 16-byte aligned: rows staged with 16-byte loads
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
  if (sg.vec) {
    // the input rows of the tile are one contiguous byte span of the NHWC
    // tensor: 16-byte loads of it (plus a byte tail) into LDS, then each
    // pixel's channels are picked from there
    const int iy_lo = iy0 > 0 ? iy0 : 0;
    const int iy_hi = iy0 + sg.rin - 1 < a.h - 1 ? iy0 + sg.rin - 1 : a.h - 1;
    int lead = 0;
    uint8_t* raw = lds + sg.raw_off;
    if (iy_lo <= iy_hi) {
      const int64_t gs = (((int64_t)nimg * a.h + iy_lo) * a.w) * a.cin;
      const int64_t ge = (((int64_t)nimg * a.h + iy_hi + 1) * a.w) * a.cin;
      const int64_t gs16 = gs & ~(int64_t)15;
      lead = (int)(gs - gs16);
      const int nb = (int)(ge - gs16);
      const int nfull = nb >> 4;
      const uint4* src = reinterpret_cast<const uint4*>(a.x + gs16);
      constexpr int VB = 4;
      for (int i0 = 0; i0 < nfull; i0 += VB * kSmallThreads) {
        uint4 v[VB];
#pragma unroll
        for (int k = 0; k < VB; ++k) {   // unconditional (clamped) loads, all in flight
          const int i = i0 + k * kSmallThreads + tid;
          v[k] = src[i < nfull ? i : nfull - 1];
        }
#pragma unroll
        for (int k = 0; k < VB; ++k) {
          const int i = i0 + k * kSmallThreads + tid;
          if (i < nfull) reinterpret_cast<uint4*>(raw)[i] = v[k];
        }
      }
      for (int i = nfull * 16 + tid; i < nb; i += kSmallThreads) raw[i] = a.x[gs16 + i];
    }
    __syncthreads();
    for (int e = tid; e < nin; e += kSmallThreads) {
      const int r = fdiv(e, sg.div_win);
      const int iy = iy0 + r, ix = e - r * sg.win - a.pad;
      uint32_t word = 0x80808080u;
      if ((unsigned)iy < (unsigned)a.h && (unsigned)ix < (unsigned)a.w) {
        const uint8_t* px = raw + lead + ((iy - iy_lo) * a.w + ix) * a.cin;
#pragma unroll
        for (int ch = 0; ch < 4; ++ch)
          if (ch < a.cin) word ^= (uint32_t)px[ch] << (8 * ch);   // 0x80 ^ x
      }
      *reinterpret_cast<uint32_t*>(tile + e * 4) = word;
    }
  }
  // otherwise batches of SB pixels per thread: every byte load of a batch is
  // issued before the first is used
  constexpr int SB = 8;
  for (int e0 = 0; !sg.vec && e0 < nin; e0 += SB * kSmallThreads) {
    uint32_t word[SB];
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const int e = e0 + k * kSmallThreads + tid;
      const int r = fdiv(e, sg.div_win);
      const int iy = iy0 + r, ix = e - r * sg.win - a.pad;
      word[k] = 0x80808080u;
      if (e < nin && (unsigned)iy < (unsigned)a.h && (unsigned)ix < (unsigned)a.w) {
        const uint8_t* src = a.x + (((int64_t)nimg * a.h + iy) * a.w + ix) * a.cin;
#pragma unroll
        for (int ch = 0; ch < 4; ++ch)
          if (ch < a.cin) word[k] ^= (uint32_t)src[ch] << (8 * ch);   // 0x80 ^ x
      }
    }
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const int e = e0 + k * kSmallThreads + tid;
      if (e < nin) *reinterpret_cast<uint32_t*>(tile + e * 4) = word[k];
    }
  }
  // 2-bit codes into I8 or packed-U2 NHWC: the register epilogue below
  const bool fast = a.out_mode != 0 && a.rec == 4 && a.join_kind == IFQ_JOIN_NONE &&
                    (a.out_layout == IFQ_LAYOUT_I8_NHWC ||
                     (a.out_layout == IFQ_LAYOUT_U2_NHWC_PACKED && (a.cout & 3) == 0));
  if (!fast) stage_epilogue(a, lds, 0, BM);

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
      if (tap < ntaps && co < a.cout_pad) {
        const int8_t* wr = a.wgt + (int64_t)co * a.kpad + tap * a.cin;
#pragma unroll
        for (int c = 0; c < 4; ++c)
          if (c < a.cin) w4[j] |= (uint32_t)(uint8_t)wr[c] << (8 * c);
      }
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
  // register epilogue state: per row block, the lane's channels
  // 16*fm + 4*kg + i: packed 16-bit thresholds T' (sign folded as in the
  // transposed epilogues: T' = -T - 1 and the codes xor 3 for s = -1), the
  // xor mask and the 128 * rowsum corrections
  uint32_t tw[FM][2][3], txm[FM];
  int corr[FM][4];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    uint32_t t16[4][3];
    txm[fm] = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int co = fm * 16 + 4 * kg + i;
      int4 r = int4{1, 0x7FFF, 0x7FFF, 0x7FFF};
      corr[fm][i] = 0;
      if (fast && co < a.cout) {
        r = *reinterpret_cast<const int4*>(a.thr + (int64_t)co * 4);
        corr[fm][i] = 128 * a.rowsum[co];
      }
      const bool flip = r.x < 0;
      const int tt[3] = {r.y, r.z, r.w};
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        int v = flip ? -tt[k] - 1 : tt[k];
        v = v > 32767 ? 32767 : v < -32768 ? -32768 : v;   // |sum| < 2^15 anyway
        t16[i][k] = (uint32_t)v & 0xFFFFu;
      }
      if (flip) txm[fm] |= 3u << ((i & 1) * 16 + (i >> 1) * 4);
    }
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      tw[fm][0][k] = t16[0][k] | t16[1][k] << 16;
      tw[fm][1][k] = t16[2][k] | t16[3][k] << 16;
    }
  }
  __syncthreads();

  const int orow = small_orow(a, BM);
  uint8_t* otile = lds + sg.out_off;
  const bool pooled = a.pool_k > 0;
  uint8_t* y8 = reinterpret_cast<uint8_t*>(a.y);
  const int nblk = (npx + 15) / 16;
  // UB independent blocks of 16 pixels per iteration, so the LDS reads, the
  // MFMAs and the epilogues of different blocks overlap (one block at a time
  // past 32 output channels, where four would not fit the registers)
  constexpr int UB = FM <= 2 ? 4 : 1;
  constexpr int NW = kSmallThreads / 64;
  for (int blk0 = wave; blk0 < nblk; blk0 += NW * UB) {
    v4i accu[UB][FM];
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int q = (blk0 + NW * u) * 16 + l16;
      const int qc = q < npx ? q : npx - 1;
      const int r = fdiv(qc, a.div_wo);
      const int ox = qc - r * a.wo;
      const uint8_t* win = tile + ((r * st) * sg.win + ox * st) * 4;
      uint32_t b4[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        b4[j] = tval[j] ? *reinterpret_cast<const uint32_t*>(win + toff[j]) : 0x80808080u;
      const v4i bf = v4i{(int)b4[0], (int)b4[1], (int)b4[2], (int)b4[3]};
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
        accu[u][fm] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[fm], bf, v4i{0, 0, 0, 0}, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < UB; ++u) {
      const int q = (blk0 + NW * u) * 16 + l16;
      v4i acc[FM];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) acc[fm] = accu[u][fm];
      // lane holds channels 16*g + 4*kg .. +3 of pixel q
      if (fast) {
        const int64_t p = (int64_t)p0 + q;
#pragma unroll
        for (int fm = 0; fm < FM; ++fm) {
          const int co = fm * 16 + 4 * kg;
          const int v0 = acc[fm][0] + corr[fm][0], v1 = acc[fm][1] + corr[fm][1];
          const int v2 = acc[fm][2] + corr[fm][2], v3 = acc[fm][3] + corr[fm][3];
          if (a.acc_dump && q < npx) {
            int32_t* dp = a.acc_dump + p * a.cout + co;
            const int vv[4] = {v0, v1, v2, v3};
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (co + i < a.cout) dp[i] = vv[i];
          }
          const s16x2 p01 = __builtin_amdgcn_cvt_pk_i16(v0, v1);
          const s16x2 p23 = __builtin_amdgcn_cvt_pk_i16(v2, v3);
          const uint32_t c01 = count3_pk(p01, tw[fm][0][0], tw[fm][0][1], tw[fm][0][2]);
          const uint32_t c23 = count3_pk(p23, tw[fm][1][0], tw[fm][1][1], tw[fm][1][2]);
          // codes of channels i = 0..3: c01 bits 0 and 16, c23 bits 0 and 16
          const uint32_t t = (c01 | (c23 << 4)) ^ txm[fm];
          if (q < npx && co < a.cout && pooled) {
            // into the LDS tile for the pooled copy-out (cout % 16 == 0 for
            // packed codes, % 4 for bytes)
            if (a.out_mode == 2)
              otile[q * orow + (co >> 2)] = (uint8_t)(t | (t >> 14));
            else
              *reinterpret_cast<uint32_t*>(otile + q * orow + co) =
                  (t & 3u) | ((t >> 16) & 3u) << 8 | ((t >> 4) & 3u) << 16 | ((t >> 20) & 3u) << 24;
          } else if (q < npx && co < a.cout) {
            if (a.out_layout == IFQ_LAYOUT_U2_NHWC_PACKED) {
              y8[(p * a.cout + co) >> 2] = (uint8_t)(t | (t >> 14));
            } else {
              const uint32_t b4 = (t & 3u) | ((t >> 16) & 3u) << 8 | ((t >> 4) & 3u) << 16 |
                                  ((t >> 20) & 3u) << 24;
              uint8_t* dst = y8 + p * a.cout + co;
              if (co + 4 <= a.cout && ((p * a.cout + co) & 3) == 0) {
                *reinterpret_cast<uint32_t*>(dst) = b4;
              } else {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                  if (co + i < a.cout) dst[i] = (uint8_t)(b4 >> (8 * i));
              }
            }
          }
        }
      } else {
        epilogue_lane<FM, 1>(
            a, lds, [&](int g, int, int i) { return acc[g][i]; },
            [&](int g) { return g * 16 + 4 * kg; }, 0, p0,
            [&](int) { return q < npx ? q : -1; }, otile, orow);
      }
    }
  }
  if (!fast || pooled) {
    __syncthreads();
    if (pooled)
      pool_out_tile(a, otile, orow, 0, BM, p0, npx);
    else
      copy_out_tile(a, otile, orow, 0, BM, p0, npx);
  }
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
  // a fused pool needs whole rows of pooling windows (or the whole image)
  // per workgroup
  const int rstep = a.pool_k == 0 ? 1 : a.pool_img ? a.ho : a.pool_k;
  rows = (rows + rstep - 1) / rstep * rstep;
  if (rows > a.ho) rows = a.ho / rstep * rstep;
  for (;; rows -= rstep) {
    if (rows < 1) return false;
    const int npx = rows * a.wo;
    const int rin = (rows - 1) * a.stride + a.kh;
    const int epi = epilogue_param_bytes(bm);
    const int out = (npx * small_orow(a, bm) + 15) & ~15;
    const int64_t in = ((int64_t)rin * win * 4 + 15) & ~(int64_t)15;   // raw buffer 16-aligned
    const int64_t rawb = ((int64_t)rin * a.w * a.cin + 16 + 15) & ~(int64_t)15;
    const int64_t total = (int64_t)epi + out + in + rawb;
    if (npx <= kSmallMaxPx && total <= kSmallMaxLds) {
      g->rows = rows;
      g->tiles = (a.ho + rows - 1) / rows;
      g->rin = rin;
      g->win = win;
      g->div_win = make_fastdiv((uint32_t)win);
      g->out_off = epi;
      g->in_off = epi + out;
      g->raw_off = (int)(epi + out + in);
      g->vec = ((uintptr_t)a.x & 15) == 0;
      g->lds_bytes = (int)total;
      return true;
    }
  }
}

// ---------------------------------------------------------------------------
// 2-bit input codes with 16 or 32 input channels (a detector's second and
// third layers): 3x3, stride 1, pad 1, 2-bit output codes with thresholds,
// optionally with the following max-pool fused. The implicit GEMM runs on
// v_mfma_i32_32x32x32_i8 with K in the weight blob's order (tap-major, the
// 16 channels of a group transposed as 4x4, which is the order in which a
// lane unpacks the 16 codes of a packed 32-bit word): K32 step s covers the
// two taps 2s, 2s+1 (c_in 16) or the one tap s (c_in 32), and the half h of
// the lanes takes the 16 K values 32s + 16h .. +15, i.e. one packed 32-bit
// word of the input window per lane and step.
//  - A workgroup computes whole output rows of one image; the input rows they
//    need are staged once in LDS as packed pixels of c_in/4 bytes with a
//    column of zero codes on either side, rows outside the image zero.
//  - The weight fragments of all K steps and output channels stay in
//    registers for the whole workgroup (K <= 288, c_out <= 64).
//  - Epilogue: the packed 16-bit threshold compare from LDS records, codes
//    into the LDS output tile, then the tile (or its pooled form) to HBM.
template <int FM, int CIN>
__global__ __launch_bounds__(kSmallThreads) void conv_small2(ConvLaunch a, SmallGeom sg) {
  constexpr int BM = 32 * FM;
  constexpr int KS = (9 * CIN + 31) / 32;        // K32 steps
  constexpr int BPP = CIN / 4;                   // bytes per packed pixel (4 or 8)
  constexpr int WPP = CIN / 16;                  // 32-bit words per pixel (1 or 2)
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int h = lane >> 5;
  const int l32 = lane & 31;

  const int nimg = blockIdx.x / sg.tiles;
  const int oy0 = (blockIdx.x - nimg * sg.tiles) * sg.rows;
  const int rows = a.ho - oy0 < sg.rows ? a.ho - oy0 : sg.rows;
  const int npx = rows * a.wo;
  const int p0 = (nimg * a.ho + oy0) * a.wo;

  // ---- stage the input rows (1 or 2 words per pixel) ------------------------
  uint32_t* tile = reinterpret_cast<uint32_t*>(lds + sg.in_off);
  const int iy0 = oy0 - 1;
  const int nwords = sg.rin * sg.win * WPP;
  const uint32_t* x32 = reinterpret_cast<const uint32_t*>(a.x);
  constexpr int SB = 8;
  for (int e0 = 0; e0 < nwords; e0 += SB * kSmallThreads) {
    uint32_t v[SB];
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const int e = e0 + k * kSmallThreads + tid;
      const int px = e / WPP, wd = e - px * WPP;
      const int r = fdiv(px, sg.div_win);
      const int iy = iy0 + r, ix = px - r * sg.win - 1;
      v[k] = 0u;
      if (e < nwords && (unsigned)iy < (unsigned)a.h && (unsigned)ix < (unsigned)a.w)
        v[k] = x32[(((int64_t)nimg * a.h + iy) * a.w + ix) * WPP + wd];
    }
#pragma unroll
    for (int k = 0; k < SB; ++k) {
      const int e = e0 + k * kSmallThreads + tid;
      if (e < nwords) tile[e] = v[k];
    }
  }
  // ---- threshold records (stage_thr_pk's layout; channels past c_out get
  // records whose codes are never stored) and weight fragments --------------
  if (tid < BM / 4) {
    uint32_t w[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = 4 * tid + i;
      int4 r = int4{1, 0, 0, 0};
      if (c < a.cout) r = *reinterpret_cast<const int4*>(a.thr + (int64_t)c * 4);
      const bool flip = r.x < 0;
      const int t[3] = {r.y, r.z, r.w};
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        int vv = flip ? -t[k] - 1 : t[k];
        vv = vv > 32767 ? 32767 : vv < -32768 ? -32768 : vv;   // |sum| <= 3 * 288
        w[(i >> 1) * 3 + k] |= ((uint32_t)vv & 0xFFFFu) << (16 * (i & 1));
      }
      if (flip) w[6] |= 3u << ((i & 1) * 16 + (i >> 1) * 4);
    }
    uint4* dst = reinterpret_cast<uint4*>(lds + tid * kPkRecBytes);
    dst[0] = uint4{w[0], w[1], w[2], w[3]};
    dst[1] = uint4{w[4], w[5], w[6], w[7]};
  }
  v4i af[KS][FM];
#pragma unroll
  for (int s = 0; s < KS; ++s)
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int row = fm * 32 + l32;
      const int k0 = 32 * s + 16 * h;
      af[s][fm] = v4i{0, 0, 0, 0};
      if (row < a.cout_pad && k0 < a.kpad)
        af[s][fm] = *reinterpret_cast<const v4i*>(a.wgt + (int64_t)row * a.kpad + k0);
    }
  // LDS byte offset of this lane's word of K step s from a pixel's window corner
  int toff[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int k0 = 32 * s + 16 * h;
    const int tap = k0 / CIN, c0 = k0 - tap * CIN;
    const int ty = tap / 3, tx = tap - ty * 3;
    toff[s] = tap < 9 ? ((ty * sg.win + tx) * BPP + (c0 >> 2)) : -1;
  }
  __syncthreads();

  const int orow = small_orow(a, BM);
  uint8_t* otile = lds + sg.out_off;
  const int nblk = (npx + 31) / 32;
  constexpr int NW = kSmallThreads / 64;
  for (int blk = wave; blk < nblk; blk += NW) {
    const int q = blk * 32 + l32;
    const int qc = q < npx ? q : npx - 1;
    const int r = fdiv(qc, a.div_wo);
    const int ox = qc - r * a.wo;
    const uint8_t* win = lds + sg.in_off + (r * sg.win + ox) * BPP;
    v16i acc[FM];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) acc[fm] = v16i{0};
    uint32_t u[KS];
#pragma unroll
    for (int s = 0; s < KS; ++s)
      u[s] = toff[s] >= 0 ? *reinterpret_cast<const uint32_t*>(win + toff[s]) : 0u;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const v4i bf = unpack2(u[s]);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
        acc[fm] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[s][fm], bf, acc[fm], 0, 0, 0);
    }
    if (a.acc_dump && q < npx) {
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int c = fm * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
          if (c < a.cout) a.acc_dump[(int64_t)(p0 + q) * a.cout + c] = acc[fm][v];
        }
    }
    if (q < npx) epilogue_thr_pk<FM>(a, lds, acc, 0, h, 0, q, otile, orow);
  }
  __syncthreads();
  if (a.pool_k)
    pool_out_tile(a, otile, orow, 0, BM, p0, npx);
  else
    copy_out_tile(a, otile, orow, 0, BM, p0, npx);
}

bool small2_geom(const ConvLaunch& a, SmallGeom* g) {
  const int bm = 32 * ((a.cout + 31) / 32);
  const int win = a.wo + 2;
  const int64_t rows_total = (int64_t)a.n * a.ho;
  int rows = (int)((rows_total + 1023) / 1024);
  if (rows < 1) rows = 1;
  if (rows > a.ho) rows = a.ho;
  const int rstep = a.pool_k == 0 ? 1 : a.pool_img ? a.ho : a.pool_k;
  rows = (rows + rstep - 1) / rstep * rstep;
  if (rows > a.ho) rows = a.ho / rstep * rstep;
  for (;; rows -= rstep) {
    if (rows < 1) return false;
    const int npx = rows * a.wo;
    const int rin = rows + 2;
    const int rec = bm / 4 * kPkRecBytes;
    const int out = (npx * small_orow(a, bm) + 15) & ~15;
    const int64_t in = ((int64_t)rin * win * (a.cin / 4) + 15) & ~(int64_t)15;
    const int64_t total = (int64_t)rec + out + in;
    if (npx <= kSmallMaxPx && total <= kSmallMaxLds) {
      g->rows = rows;
      g->tiles = (a.ho + rows - 1) / rows;
      g->rin = rin;
      g->win = win;
      g->div_win = make_fastdiv((uint32_t)win);
      g->out_off = rec;
      g->in_off = (int)(rec + out);
      g->raw_off = 0;
      g->vec = 0;
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
  if (a.pool_k && !pool_epilogue_ok(a)) return false;
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

bool small2_eligible(const ConvLaunch& a) {
  if (!(a.in_bits == 2 && a.in_layout == IFQ_LAYOUT_U2_NHWC_PACKED &&
        (a.cin == 16 || a.cin == 32) && a.kh == 3 && a.kw == 3 && a.stride == 1 &&
        a.pad == 1 && a.cout <= 64 && a.out_mode == 2 && a.rec == 4 &&
        a.join_kind == IFQ_JOIN_NONE && a.m > 0))
    return false;
  if (((uintptr_t)a.x & 3) != 0) return false;   // staged as 32-bit words
  if (a.pool_k && !pool_epilogue_ok(a)) return false;
  SmallGeom g;
  return small2_geom(a, &g);
}

const char* conv_small2_name(const ConvLaunch& a) {
  const bool two = a.cout > 32;
  if (a.cin == 16) return two ? "conv_small2<2, 16>" : "conv_small2<1, 16>";
  return two ? "conv_small2<2, 32>" : "conv_small2<1, 32>";
}

hipError_t launch_conv_small2(const ConvLaunch& a, hipStream_t stream) {
  SmallGeom g;
  if (!small2_geom(a, &g)) return hipErrorInvalidValue;
  const dim3 grid(a.n * g.tiles);
  const int key = (a.cout > 32 ? 2 : 0) + (a.cin == 32 ? 1 : 0);
  switch (key) {
    case 0: hipLaunchKernelGGL((conv_small2<1, 16>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g); break;
    case 1: hipLaunchKernelGGL((conv_small2<1, 32>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g); break;
    case 2: hipLaunchKernelGGL((conv_small2<2, 16>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g); break;
    case 3: hipLaunchKernelGGL((conv_small2<2, 32>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace ifq
