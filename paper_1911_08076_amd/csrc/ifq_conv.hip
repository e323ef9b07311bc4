// Integrated fixed-point quantized convolution on gfx950 (MI355X).
//
// One kernel computes a quantized substructure of IFQ-Net:
//   a    = W_b (x) X_q            integer part of Eq. (1), as an implicit GEMM
//                                 D[co][pixel] = sum_k W[co][k] * X[pixel][k]
//                                 on v_mfma_i32_16x16x64_i8 (int8 x int8 -> int32)
//   code = #{i : s*a > T_i}       Eq. (7)/(8): integer thresholds folded on the
//                                 host (Sec. 3.2); or the residual join, or the
//                                 int32 sum itself for layers without quantizer
//
// K runs over (tap, channel): k = (r*kw + s)*c_in + c. The A operand (rows =
// output channels) is the packed +-1 weight matrix, the B operand (columns =
// output pixels) is gathered on the fly from the NHWC codes, 16 channels of
// one tap at a time, with zero codes for padded positions. Both tiles go
// through LDS, double-buffered, one barrier per 64-wide K step.
//
// Output channels sit on the MFMA row dimension, so each lane of a 16x16
// accumulator block holds four consecutive output channels of one pixel:
// four codes pack into one 32-bit word (byte per code) or one byte (2-bit)
// without any cross-lane traffic.
//
// 8-bit input codes (0..255) do not fit signed int8. They enter the MFMA as
// x - 128 (XOR 0x80), padded positions as -128 (i.e. x = 0), and the epilogue
// adds back 128 * rowsum(W[co]): sum W*x = sum W*(x-128) + 128 * sum W, exact.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "ifq_internal.h"

namespace ifq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

enum Gather {
  kGatherI8 = 0,     // byte-per-code input, c_in % 16 == 0: 16-byte loads
  kGatherU2 = 1,     // 2-bit packed input, c_in % 16 == 0: 4-byte loads
  kGatherBytes = 2,  // byte-per-code input, any c_in: byte loads
};

constexpr uint32_t kLow2 = 0x03030303u;

// Sixteen zero bytes in device memory: gather loads that fall outside the
// image read them instead of branching around the load.
__device__ uint4 g_zero_chunk;

// XOR swizzle of the four 16-byte chunks of a 64-byte LDS row, so that the
// 16-byte reads of eight consecutive rows hit distinct banks.
__device__ __forceinline__ int swz(int row) { return (row >> 1) & 3; }

// Copies the per-channel epilogue parameters of output channels
// [co0, co0 + bm) into LDS once per workgroup: the threshold records
// (bm * rec int32) or the join coefficients (bm * 3 doubles). The caller
// brackets it with barriers (the LDS is the main loop's, no longer in use).
__device__ __forceinline__ void stage_epilogue(const ConvLaunch& a, uint8_t* lds,
                                               int co0, int bm) {
  if (a.out_mode == 0) return;
  const int tid = threadIdx.x;
  if (a.join_kind == IFQ_JOIN_NONE) {
    const int n = bm * a.rec;
    int32_t* dst = reinterpret_cast<int32_t*>(lds);
    const int32_t* src = a.thr + (int64_t)co0 * a.rec;
    const int lim = (a.cout - co0) * a.rec;
    for (int i = tid; i < n; i += blockDim.x) dst[i] = i < lim ? src[i] : 0;
  } else {
    double* dst = reinterpret_cast<double*>(lds);
    const double* src = a.coef + (int64_t)co0 * 3;
    const int lim = (a.cout - co0) * 3;
    for (int i = tid; i < bm * 3; i += blockDim.x) dst[i] = i < lim ? src[i] : 0.0;
  }
}

// Epilogue modes, decided once per launch (uniform branch) so that each
// inlined copy is straight-line code.
enum EpiMode {
  kEpiI32 = 0,      // int32 sums are the output
  kEpiThr4 = 1,     // codes from {s, T1, T2, T3} records (2-bit output)
  kEpiThr = 2,      // codes from records of any length 2^out_bits
  kEpiJoinConv = 3, // join with an int32 shortcut (1x1 downsample sums)
  kEpiJoinU2 = 4,   // join with a 2-bit packed code shortcut
  kEpiJoinI8 = 5,   // join with a byte-per-code shortcut
};

// The accumulators of a lane are seen as NG groups of four consecutive output
// channels (co_of(g) .. co_of(g)+3) times FN pixel blocks: val(g, fn, i) is
// the sum of channel co_of(g)+i at local pixel pxl(fn).
template <int MODE, bool U2OUT, int NG, int FN, class ValFn, class CoFn, class PixFn>
__device__ __forceinline__ void epilogue_mode(const ConvLaunch& a,
                                              const uint8_t* lds, ValFn val,
                                              CoFn co_of, int co_blk, int p0,
                                              PixFn pxl, uint8_t* otile,
                                              int orow) {
  int32_t* y32 = reinterpret_cast<int32_t*>(a.y);
  const uint8_t* sc8 = reinterpret_cast<const uint8_t*>(a.shortcut);
  const int32_t* sc32 = reinterpret_cast<const int32_t*>(a.shortcut);
  const bool in8 = a.in_bits == 8;
  const bool full4 = (a.cout & 3) == 0;
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int co = co_of(g);
    if (co >= a.cout) continue;
    const int lc = co - co_blk;
    int corr[4] = {0, 0, 0, 0};
    if (in8) {
#pragma unroll
      for (int i = 0; i < 4; ++i) corr[i] = 128 * a.rowsum[co + i];
    }
    int4 tr[4];
    double cf[4][3];
    if constexpr (MODE == kEpiThr4) {
#pragma unroll
      for (int i = 0; i < 4; ++i) tr[i] = *reinterpret_cast<const int4*>(lds + (lc + i) * 16);
    }
    if constexpr (MODE >= kEpiJoinConv) {
      const double* c = reinterpret_cast<const double*>(lds) + 3 * lc;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        cf[i][0] = c[3 * i];
        cf[i][1] = c[3 * i + 1];
        cf[i][2] = c[3 * i + 2];
      }
    }
    // Pixel blocks are handled in chunks of CH: a chunk's join shortcut values
    // are loaded before any of its stores, so their latencies overlap.
    constexpr int CH = MODE >= kEpiJoinConv ? 4 : FN;
#pragma unroll
    for (int f0 = 0; f0 < FN; f0 += CH) {
      int scv[CH][4];
      if constexpr (MODE >= kEpiJoinConv) {
#pragma unroll
        for (int j = 0; j < CH; ++j) {
          const int fn = f0 + j;
          scv[j][0] = scv[j][1] = scv[j][2] = scv[j][3] = 0;
          if (fn >= FN) continue;
          const int pl = pxl(fn);
          if (pl < 0) continue;
          const int p = p0 + pl;
          const int64_t e = (int64_t)p * a.cout + co;
          if constexpr (MODE == kEpiJoinConv) {
            if (full4) {
              const int4 s4 = *reinterpret_cast<const int4*>(sc32 + e);
              scv[j][0] = s4.x;
              scv[j][1] = s4.y;
              scv[j][2] = s4.z;
              scv[j][3] = s4.w;
            } else {
#pragma unroll
              for (int i = 0; i < 4; ++i) scv[j][i] = co + i < a.cout ? sc32[e + i] : 0;
            }
          } else if constexpr (MODE == kEpiJoinU2) {
            const uint32_t byte = sc8[e >> 2];
#pragma unroll
            for (int i = 0; i < 4; ++i) scv[j][i] = (byte >> (2 * i)) & 3u;
          } else {
            if (full4) {
              const uint32_t w4 = *reinterpret_cast<const uint32_t*>(sc8 + e);
#pragma unroll
              for (int i = 0; i < 4; ++i) scv[j][i] = (w4 >> (8 * i)) & 0xFFu;
            } else {
#pragma unroll
              for (int i = 0; i < 4; ++i) scv[j][i] = co + i < a.cout ? sc8[e + i] : 0;
            }
          }
        }
      }
#pragma unroll
      for (int j = 0; j < CH; ++j) {
        const int fn = f0 + j;
        if (fn >= FN) continue;
        const int pl = pxl(fn);
        if (pl < 0) continue;
        const int p = p0 + pl;
        int v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = val(g, fn, i) + corr[i];
        const int64_t e = (int64_t)p * a.cout + co;
        if constexpr (MODE == kEpiI32) {
          if (full4) {
            *reinterpret_cast<int4*>(y32 + e) = int4{v[0], v[1], v[2], v[3]};
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i)
              if (co + i < a.cout) y32[e + i] = v[i];
          }
        } else {
          int code[4] = {0, 0, 0, 0};
          if constexpr (MODE == kEpiThr4) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int sv = tr[i].x * v[i];
              code[i] = (sv > tr[i].y ? 1 : 0) + (sv > tr[i].z ? 1 : 0) +
                        (sv > tr[i].w ? 1 : 0);
            }
          } else if constexpr (MODE == kEpiThr) {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int32_t* t = reinterpret_cast<const int32_t*>(lds) + (lc + i) * a.rec;
              const int sv = t[0] * v[i];
              int c = 0;
              for (int q = 1; q <= a.nq; ++q) c += sv > t[q] ? 1 : 0;
              code[i] = c;
            }
          } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const double z = fma(cf[i][0], (double)v[i],
                                   fma(cf[i][1], (double)scv[j][i], cf[i][2]));
              int c = 0;
#pragma unroll
              for (int q = 0; q < IFQ_MAX_THRESHOLDS; ++q)
                if (q < a.nq) c += z > a.qthr[q] ? 1 : 0;
              code[i] = c;
            }
          }
          // codes go to the LDS output tile (row pl, this lane's 4 channels)
          if constexpr (U2OUT) {
            otile[pl * orow + (lc >> 2)] =
                (uint8_t)(code[0] | (code[1] << 2) | (code[2] << 4) | (code[3] << 6));
          } else {
            *reinterpret_cast<uint32_t*>(otile + pl * orow + lc) =
                (uint32_t)code[0] | ((uint32_t)code[1] << 8) |
                ((uint32_t)code[2] << 16) | ((uint32_t)code[3] << 24);
          }
        }
      }
    }
  }
}

// Epilogue of one lane. For row block fm the lane holds output channels
// co_lane + 16*fm + {0..3}; for column block fn it holds local pixel pxl(fn)
// of the tile starting at pixel p0 (negative: outside). Writes the optional
// int32 dump and the int32 sums directly; codes (Eq. 7/8 or the join) go to
// the LDS output tile otile (orow bytes per pixel), which copy_out_tile then
// writes to HBM with wide coalesced stores. Per-channel parameters come from
// LDS (stage_epilogue).
template <int NG, int FN, class ValFn, class CoFn, class PixFn>
__device__ __forceinline__ void epilogue_lane(const ConvLaunch& a,
                                              const uint8_t* lds, ValFn val,
                                              CoFn co_of, int co_blk, int p0,
                                              PixFn pxl, uint8_t* otile,
                                              int orow) {
  if (a.acc_dump) {
    int32_t* dump = a.acc_dump;
    const bool in8 = a.in_bits == 8;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const int co = co_of(g);
      if (co >= a.cout) continue;
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        const int pl = pxl(fn);
        if (pl < 0) continue;
        const int64_t e = (int64_t)(p0 + pl) * a.cout + co;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (co + i < a.cout)
            dump[e + i] = val(g, fn, i) + (in8 ? 128 * a.rowsum[co + i] : 0);
      }
    }
  }
  const bool u2 = a.out_mode == 2;
#define IFQ_EPI(M, U) \
  epilogue_mode<M, U, NG, FN>(a, lds, val, co_of, co_blk, p0, pxl, otile, orow)
  if (a.out_mode == 0) {
    IFQ_EPI(kEpiI32, false);
  } else if (a.join_kind == IFQ_JOIN_CONV) {
    if (u2) IFQ_EPI(kEpiJoinConv, true); else IFQ_EPI(kEpiJoinConv, false);
  } else if (a.join_kind == IFQ_JOIN_IDENTITY) {
    if (a.sc_layout == IFQ_LAYOUT_U2_NHWC_PACKED) {
      if (u2) IFQ_EPI(kEpiJoinU2, true); else IFQ_EPI(kEpiJoinU2, false);
    } else {
      if (u2) IFQ_EPI(kEpiJoinI8, true); else IFQ_EPI(kEpiJoinI8, false);
    }
  } else if (a.rec == 4) {
    if (u2) IFQ_EPI(kEpiThr4, true); else IFQ_EPI(kEpiThr4, false);
  } else {
    if (u2) IFQ_EPI(kEpiThr, true); else IFQ_EPI(kEpiThr, false);
  }
#undef IFQ_EPI
}

// Writes the LDS output tile (codes of output channels co0 .. co0+bm-1 for
// the npx pixels starting at p0, orow bytes per pixel) to HBM: each pixel's
// row is contiguous in the NHWC output, so the workgroup copies it with
// 16-byte (else 4- or 1-byte) stores.
__device__ __forceinline__ void copy_out_tile(const ConvLaunch& a, const uint8_t* otile,
                                              int orow, int co0, int bm, int p0,
                                              int npx) {
  if (a.out_mode == 0 || npx <= 0) return;
  const bool u2 = a.out_mode == 2;
  const int ch = a.cout - co0 < bm ? a.cout - co0 : bm;
  const int rbytes = u2 ? ch >> 2 : ch;              // bytes per pixel row
  const int pstride = u2 ? a.cout >> 2 : a.cout;      // output bytes per pixel
  const int cofs = u2 ? co0 >> 2 : co0;
  uint8_t* y8 = reinterpret_cast<uint8_t*>(a.y);
  const int tid = threadIdx.x;
  if ((rbytes & 15) == 0 && (pstride & 15) == 0 && (cofs & 15) == 0) {
    const int per = rbytes >> 4;
    for (int u = tid; u < npx * per; u += blockDim.x) {
      const int pl = u / per, q = u - pl * per;
      *reinterpret_cast<uint4*>(y8 + (int64_t)(p0 + pl) * pstride + cofs + q * 16) =
          *reinterpret_cast<const uint4*>(otile + pl * orow + q * 16);
    }
  } else if ((rbytes & 3) == 0 && (pstride & 3) == 0 && (cofs & 3) == 0) {
    const int per = rbytes >> 2;
    for (int u = tid; u < npx * per; u += blockDim.x) {
      const int pl = u / per, q = u - pl * per;
      *reinterpret_cast<uint32_t*>(y8 + (int64_t)(p0 + pl) * pstride + cofs + q * 4) =
          *reinterpret_cast<const uint32_t*>(otile + pl * orow + q * 4);
    }
  } else {
    for (int u = tid; u < npx * rbytes; u += blockDim.x) {
      const int pl = u / rbytes, q = u - pl * rbytes;
      y8[(int64_t)(p0 + pl) * pstride + cofs + q] = otile[pl * orow + q];
    }
  }
}

template <int BM, int BN, int WAVES_M, int GATHER>
__global__ __launch_bounds__(256) void conv_igemm(ConvLaunch a) {
  constexpr int WAVES_N = 4 / WAVES_M;
  constexpr int WM = BM / WAVES_M;
  constexpr int WN = BN / WAVES_N;
  constexpr int FM = WM / 16;
  constexpr int FN = WN / 16;
  static_assert(FM >= 1 && FN >= 1 && WM % 16 == 0 && WN % 16 == 0, "wave tile");
  constexpr int A_BYTES = BM * 64;
  constexpr int B_ROW = GATHER == kGatherU2 ? 16 : 64;
  constexpr int B_BYTES = BN * B_ROW;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int A_CHUNKS = BM * 4;
  constexpr int A_PER_T = (A_CHUNKS + 255) / 256;
  static_assert((BN * 4) % 256 == 0, "BN must be a multiple of 64");
  constexpr int B_PER_T = BN * 4 / 256;
  constexpr int EPI_BYTES = BM * 16 * 4;        // largest threshold records
  constexpr int OUT_BYTES = BN * BM;            // output tile, byte per code
  constexpr int LDS_BYTES =
      2 * STAGE > EPI_BYTES + OUT_BYTES ? 2 * STAGE : EPI_BYTES + OUT_BYTES;

  __shared__ __attribute__((aligned(16))) uint8_t lds[LDS_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % WAVES_M;
  const int wn = wave / WAVES_M;
  const int p0 = blockIdx.x * BN;
  const int co0 = blockIdx.y * BM;

  // Each thread gathers k16-group j of pixels (tid>>2) + 64*i of the tile.
  const int j = tid & 3;
  const int howo = a.ho * a.wo;
  int pix_row[B_PER_T], pix_iy0[B_PER_T], pix_ix0[B_PER_T];
#pragma unroll
  for (int i = 0; i < B_PER_T; ++i) {
    const int p = p0 + (tid >> 2) + 64 * i;
    if (p < a.m) {
      const int nimg = p / howo;
      const int rem = p - nimg * howo;
      const int oy = rem / a.wo;
      const int ox = rem - oy * a.wo;
      pix_row[i] = nimg * a.h;
      pix_iy0[i] = oy * a.stride - a.pad;
      pix_ix0[i] = ox * a.stride - a.pad;
    } else {
      pix_row[i] = -1;
      pix_iy0[i] = 0;
      pix_ix0[i] = 0;
    }
  }
  const bool in8 = a.in_bits == 8;
  const uint32_t pad_word = in8 ? 0x80808080u : 0u;
  const int cg16 = a.cin >> 4;
  const int ntaps = a.kh * a.kw;

  uint4 areg[A_PER_T];
  uint4 breg[B_PER_T];

  auto load_a = [&](int kt) {
#pragma unroll
    for (int i = 0; i < A_PER_T; ++i) {
      const int q = tid + 256 * i;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (q < A_CHUNKS) {
        const int co = co0 + (q >> 2);
        if (co < a.cout_pad)
          v = *reinterpret_cast<const uint4*>(
              a.wgt + (int64_t)co * a.kpad + kt * kKStep + (q & 3) * 16);
      }
      areg[i] = v;
    }
  };

  auto load_b = [&](int kt) {
    if constexpr (GATHER == kGatherBytes) {
#pragma unroll
      for (int i = 0; i < B_PER_T; ++i) {
        uint32_t wd[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int b = 0; b < 16; ++b) {
          const int k = kt * kKStep + j * 16 + b;
          const int tap = k / a.cin;
          const int c = k - tap * a.cin;
          const int r = tap / a.kw;
          const int s = tap - r * a.kw;
          const int iy = pix_iy0[i] + r;
          const int ix = pix_ix0[i] + s;
          const bool ok = tap < ntaps && pix_row[i] >= 0 &&
                          (unsigned)iy < (unsigned)a.h &&
                          (unsigned)ix < (unsigned)a.w;
          uint32_t val = in8 ? 0x80u : 0u;
          if (ok) {
            val = a.x[((int64_t)(pix_row[i] + iy) * a.w + ix) * a.cin + c];
            if (in8) val ^= 0x80u;
          }
          wd[b >> 2] |= val << (8 * (b & 3));
        }
        breg[i] = make_uint4(wd[0], wd[1], wd[2], wd[3]);
      }
    } else {
      const int k16 = kt * 4 + j;
      const int tap = k16 / cg16;
      const int cg = k16 - tap * cg16;
      const int r = tap / a.kw;
      const int s = tap - r * a.kw;
      const bool tap_ok = tap < ntaps;
#pragma unroll
      for (int i = 0; i < B_PER_T; ++i) {
        const int iy = pix_iy0[i] + r;
        const int ix = pix_ix0[i] + s;
        const bool ok = tap_ok && pix_row[i] >= 0 &&
                        (unsigned)iy < (unsigned)a.h &&
                        (unsigned)ix < (unsigned)a.w;
        const int64_t ch = ((int64_t)(pix_row[i] + iy) * a.w + ix) * a.cin + cg * 16;
        if constexpr (GATHER == kGatherI8) {
          uint4 v = make_uint4(pad_word, pad_word, pad_word, pad_word);
          if (ok) {
            v = *reinterpret_cast<const uint4*>(a.x + ch);
            if (in8) {
              v.x ^= 0x80808080u;
              v.y ^= 0x80808080u;
              v.z ^= 0x80808080u;
              v.w ^= 0x80808080u;
            }
          }
          breg[i] = v;
        } else {
          uint32_t v = 0u;
          if (ok) v = *reinterpret_cast<const uint32_t*>(a.x + (ch >> 2));
          breg[i] = make_uint4(v, 0u, 0u, 0u);
        }
      }
    }
  };

  auto store = [&](int buf) {
    uint8_t* as = lds + buf * STAGE;
    uint8_t* bs = as + A_BYTES;
#pragma unroll
    for (int i = 0; i < A_PER_T; ++i) {
      const int q = tid + 256 * i;
      if (q < A_CHUNKS) {
        const int row = q >> 2;
        *reinterpret_cast<uint4*>(as + row * 64 + (((q & 3) ^ swz(row)) << 4)) = areg[i];
      }
    }
#pragma unroll
    for (int i = 0; i < B_PER_T; ++i) {
      const int pl = (tid >> 2) + 64 * i;
      if constexpr (GATHER == kGatherU2) {
        *reinterpret_cast<uint32_t*>(bs + pl * 16 + j * 4) = breg[i].x;
      } else {
        *reinterpret_cast<uint4*>(bs + pl * 64 + ((j ^ swz(pl)) << 4)) = breg[i];
      }
    }
  };

  v4i acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = v4i{0, 0, 0, 0};

  const int kg = lane >> 4;
  const int l16 = lane & 15;

  auto compute = [&](int buf) {
    const uint8_t* as = lds + buf * STAGE;
    const uint8_t* bs = as + A_BYTES;
    v4i af[FM], bf[FN];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int row = wm * WM + fm * 16 + l16;
      af[fm] = *reinterpret_cast<const v4i*>(as + row * 64 + ((kg ^ swz(row)) << 4));
    }
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int pix = wn * WN + fn * 16 + l16;
      if constexpr (GATHER == kGatherU2) {
        const uint32_t u = *reinterpret_cast<const uint32_t*>(bs + pix * 16 + kg * 4);
        bf[fn] = v4i{(int)(u & kLow2), (int)((u >> 2) & kLow2),
                     (int)((u >> 4) & kLow2), (int)((u >> 6) & kLow2)};
      } else {
        bf[fn] = *reinterpret_cast<const v4i*>(bs + pix * 64 + ((kg ^ swz(pix)) << 4));
      }
    }
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        acc[fm][fn] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[fm], bf[fn], acc[fm][fn], 0, 0, 0);
  };

  load_a(0);
  load_b(0);
  store(0);
  __syncthreads();
  for (int kt = 0; kt < a.nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < a.nk;
    if (more) {
      load_a(kt + 1);
      load_b(kt + 1);
    }
    compute(cur);
    if (more) store(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue: lane holds channels co..co+3 of pixel p per block ----
  stage_epilogue(a, lds, co0, BM);
  __syncthreads();
  const int orow = a.out_mode == 2 ? BM / 4 : BM;
  uint8_t* otile = lds + EPI_BYTES;
  // 16x16 accumulator block (fm, fn): lane holds channels 4*kg..4*kg+3 of
  // the block's rows and pixel l16 of its columns
  epilogue_lane<FM, FN>(
      a, lds, [&](int g, int fn, int i) { return acc[g][fn][i]; },
      [&](int g) { return co0 + wm * WM + g * 16 + 4 * kg; }, co0, p0,
      [&](int fn) {
        const int pl = wn * WN + fn * 16 + l16;
        return p0 + pl < a.m ? pl : -1;
      },
      otile, orow);
  __syncthreads();
  copy_out_tile(a, otile, orow, co0, BM, p0, a.m - p0 < BN ? a.m - p0 : BN);
}


// ---------------------------------------------------------------------------
// Fast path: 2-bit packed input with c_in % 64 == 0. One K step is 64 channels
// of one filter tap (16 packed bytes per pixel). The four waves form a 2 x 2
// grid over (output channels, pixels); each wave owns 16*FM channels x 16*FN
// pixels, a workgroup 32*FM channels x a pixel tile of bn <= 32*FN pixels (bn
// is chosen per layer so that the grid fills the 256 CUs in whole waves).
//
// Operands reach LDS through the LDS-DMA form of the global load: one wave
// instruction moves 64 x 16 bytes, lane i's bytes landing at base + 16*i, with
// no staging registers. The weights are stored in MFMA fragment order, so a
// 1 KB chunk per (16-row block, K step) is one such load and the A fragment is
// a conflict-free 16-byte LDS read. The activations stay 2-bit packed in LDS
// (16 bytes per pixel row and K step) and are unpacked with shifts and masks
// right before the MFMA. S K steps form a stage; a ring of D stages keeps the
// loads of the next D-1 stages in flight while one stage computes, so the
// L2/HBM latency is hidden behind D-1 stages of MFMA work. Each wave issues
// the same number of loads per stage, and waits for a stage with an explicit
// vmcnt that leaves the younger stages in flight. Out-of-range operands are
// read from blocks of zeros, so the loop has no branch around a load.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)p;
}

// One wave-wide LDS-DMA load: 16 bytes per lane from src to LDS dst + 16*lane.
// M0 carries the LDS base; nothing else in these kernels uses M0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const void* src, uint32_t dst) {
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
               :: "s"(dst), "v"(src) : "memory", "m0");
}
#pragma clang diagnostic pop

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}

template <int FM, int FN, int S, int D>
__global__ __launch_bounds__(256) void conv_u2(ConvLaunch a) {
  constexpr int BM = 32 * FM;
  constexpr int BNMAX = 32 * FN;
  static_assert(BNMAX <= 256, "pixel rows");
  constexpr int RB = BM / 16;                   // 16-row blocks per workgroup
  constexpr int NBW = (BNMAX + 63) / 64;        // 64-pixel row groups
  static_assert(NBW == 1 || NBW == 2 || NBW == 4, "row groups");
  constexpr int A_CH = RB * S;                  // 1 KB chunks per stage
  constexpr int B_CH = NBW * S;
  static_assert(A_CH % 4 == 0 && B_CH % 4 == 0, "equal loads per wave");
  constexpr int CA = A_CH / 4, CB = B_CH / 4, C = CA + CB;
  static_assert((D - 2) * C <= 63, "vmcnt range");
  constexpr int A_STAGE = A_CH * 1024;
  constexpr int B_T = NBW * 1024;               // one K step of B
  constexpr int STAGE = A_STAGE + B_CH * 1024;
  constexpr int EPI_BYTES = BM * 16 * 4;        // largest threshold records
  constexpr int OUT_BYTES = BNMAX * BM;         // output tile, byte per code
  constexpr int LDS_BYTES =
      D * STAGE > EPI_BYTES + OUT_BYTES ? D * STAGE : EPI_BYTES + OUT_BYTES;

  __shared__ __attribute__((aligned(1024))) uint8_t lds[LDS_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1;
  const int wn = wave >> 1;
  const int kg = lane >> 4;
  const int l16 = lane & 15;
  const int bn = a.bn;
  const int p0 = blockIdx.x * bn;
  const int co0 = blockIdx.y * BM;
  const int cg64 = a.cin >> 6;
  const int cb = a.cin >> 2;                    // packed bytes per pixel
  const int nk = a.nk;
  const int nst = (nk + S - 1) / S;
  const int rbw = co0 >> 4;                     // first row block of the workgroup
  const int nrb = a.cout_pad >> 4;
  const uint8_t* wbase = reinterpret_cast<const uint8_t*>(a.wgt) + (int64_t)lane * 16;
  const uint8_t* zero_src = reinterpret_cast<const uint8_t*>(&g_zero_chunk);
  const uint32_t lds0 = lds_addr(lds);

  // the pixel row this thread loads: row group wave % NBW, row lane
  const int prow = (wave % NBW) * 64 + lane;
  bool px_ok = false;
  int px_base = 0, px_iy0 = 0, px_ix0 = 0;
  if (prow < BNMAX && prow < bn) {
    const int p = p0 + prow;
    if (p < a.m) {
      const int howo = a.ho * a.wo;
      const int nimg = p / howo;
      const int rem = p - nimg * howo;
      const int oy = rem / a.wo;
      const int ox = rem - oy * a.wo;
      px_ok = true;
      px_iy0 = oy * a.stride - a.pad;
      px_ix0 = ox * a.stride - a.pad;
      // byte offset of input pixel (nimg, iy0, ix0); may be out of the image
      px_base = ((nimg * a.h + px_iy0) * a.w + px_ix0) * cb;
    }
  }

  // K-step state (uniform) of each of this wave's B loads: K step
  // t_j = (wave + 4j) / NBW of the stage being issued, as (tap r, s, group)
  int kr[CB], ks[CB], kc[CB];
#pragma unroll
  for (int j = 0; j < CB; ++j) {
    const int t = (wave + 4 * j) / NBW;
    const int tap = t / cg64;
    kc[j] = t - tap * cg64;
    kr[j] = tap / a.kw;
    ks[j] = tap - kr[j] * a.kw;
  }

  // Issue the loads of stage st into ring slot st % D.
  auto issue = [&](int st) {
    const uint32_t slot = lds0 + (uint32_t)((st % D) * STAGE);
#pragma unroll
    for (int j = 0; j < CA; ++j) {
      const int i = wave + 4 * j;               // chunk: row block i / S, step i % S
      const int rb = i / S;
      const int kt = st * S + (i % S);
      const bool ok = kt < nk && rbw + rb < nrb;
      const int64_t off = ok ? ((int64_t)(rbw + rb) * nk + kt) * 1024 : a.wzero;
      dma16(wbase + off, slot + i * 1024);
    }
#pragma unroll
    for (int j = 0; j < CB; ++j) {
      const int t = (wave + 4 * j) / NBW;
      const bool kok = st * S + t < nk;
      const int iy = px_iy0 + kr[j];
      const int ix = px_ix0 + ks[j];
      const bool ok = kok && px_ok && (unsigned)iy < (unsigned)a.h &&
                      (unsigned)ix < (unsigned)a.w;
      const uint8_t* src =
          ok ? a.x + (px_base + (kr[j] * a.w + ks[j]) * cb + kc[j] * 16) : zero_src;
      dma16(src, slot + A_STAGE + t * B_T + (wave % NBW) * 1024);
      // advance this load's K step by S (uniform selects, no branch)
#pragma unroll
      for (int u = 0; u < S; ++u) {
        kc[j] += 1;
        const bool wc = kc[j] == cg64;
        kc[j] = wc ? 0 : kc[j];
        ks[j] += wc ? 1 : 0;
        const bool wsw = ks[j] == a.kw;
        ks[j] = wsw ? 0 : ks[j];
        kr[j] += wsw ? 1 : 0;
      }
    }
  };

  v4i acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = v4i{0, 0, 0, 0};

  // K steps beyond nk multiply zero A fragments: no branch in the compute.
  auto compute = [&](int st) {
    const uint8_t* as = lds + (st % D) * STAGE;
    const uint8_t* bs = as + A_STAGE;
#pragma unroll
    for (int t = 0; t < S; ++t) {
      v4i af[FM];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
        af[fm] = *reinterpret_cast<const v4i*>(as + ((wm * FM + fm) * S + t) * 1024 +
                                               lane * 16);
      uint32_t braw[FN];
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        braw[fn] = *reinterpret_cast<const uint32_t*>(
            bs + t * B_T + (wn * 16 * FN + fn * 16 + l16) * 16 + kg * 4);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        const uint32_t u = braw[fn];
        const v4i bf = v4i{(int)(u & kLow2), (int)((u >> 2) & kLow2),
                           (int)((u >> 4) & kLow2), (int)((u >> 6) & kLow2)};
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
          acc[fm][fn] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[fm], bf, acc[fm][fn], 0, 0, 0);
      }
    }
  };

#pragma unroll
  for (int st = 0; st < D - 1; ++st) issue(st);
  for (int st = 0; st < nst; ++st) {
    wait_vmcnt<(D - 2) * C>();                  // this wave's part of stage st landed
    __syncthreads();                            // ... and every wave's; slot st-1 is free
    issue(st + D - 1);                          // into the slot freed by stage st-1
    compute(st);
  }
  wait_vmcnt<0>();
  __syncthreads();

  stage_epilogue(a, lds, co0, BM);
  __syncthreads();
  const int orow = a.out_mode == 2 ? BM / 4 : BM;
  uint8_t* otile = lds + EPI_BYTES;
  epilogue_lane<FM, FN>(
      a, lds, [&](int g, int fn, int i) { return acc[g][fn][i]; },
      [&](int g) { return co0 + (wm * FM + g) * 16 + 4 * kg; }, co0, p0,
      [&](int fn) {
        const int pl = wn * 16 * FN + fn * 16 + l16;
        return (pl < bn && p0 + pl < a.m) ? pl : -1;
      },
      otile, orow);
  __syncthreads();
  const int npx = a.m - p0 < bn ? a.m - p0 : bn;
  copy_out_tile(a, otile, orow, co0, BM, p0, npx);
}

template <int BM, int BN, int WAVES_M, int GATHER>
hipError_t launch_tile(const ConvLaunch& a, hipStream_t stream) {
  dim3 grid((a.m + BN - 1) / BN, (a.cout + BM - 1) / BM);
  hipLaunchKernelGGL((conv_igemm<BM, BN, WAVES_M, GATHER>), grid, dim3(256), 0,
                     stream, a);
  return hipGetLastError();
}

// Tile variant by output-channel count: 0: 16x256, 1: 32x128, 2: 64x128,
// 3: 128x128 (output channels x pixels per workgroup).
int tile_variant(const ConvLaunch& a) {
  if (a.cout <= 16) return 0;
  if (a.cout <= 32) return 1;
  if (a.cout <= 64) return 2;
  return 3;
}

int gather_kind(const ConvLaunch& a) {
  if (a.in_layout == IFQ_LAYOUT_U2_NHWC_PACKED) return kGatherU2;
  if (a.cin % 16 == 0) return kGatherI8;
  return kGatherBytes;
}

template <int GATHER>
hipError_t launch_gather(const ConvLaunch& a, hipStream_t stream) {
  switch (tile_variant(a)) {
    case 0: return launch_tile<16, 256, 1, GATHER>(a, stream);
    case 1: return launch_tile<32, 128, 1, GATHER>(a, stream);
    case 2: return launch_tile<64, 128, 2, GATHER>(a, stream);
    default: return launch_tile<128, 128, 2, GATHER>(a, stream);
  }
}

// Fast-path variants (FM, FN): 32*FM output channels x up to 32*FN pixels.
struct FastVariant {
  int fm, fn;
  const char* name;
};
const FastVariant kFast[] = {
    {4, 7, "conv_u2<4, 7, 2, 5>"},
    {2, 7, "conv_u2<2, 7, 2, 8>"},
    {4, 4, "conv_u2<4, 4, 2, 6>"},
    {2, 4, "conv_u2<2, 4, 2, 8>"},
};
constexpr int kNumCUs = 256;

struct FastPlan {
  int variant;   // index into kFast, or -1 for the generic kernel
  int bn;        // pixels per workgroup
  int blocks_m;  // workgroups along pixels
};

// Pick the fast-path tile whose grid covers the 256 CUs in whole waves with
// the least idle MFMA work: for each variant, take the fewest waves that fit
// the layer, spread the pixels evenly over the workgroups of those waves, and
// score useful / issued MFMA work.
FastPlan plan_fast(const ConvLaunch& a) {
  FastPlan best{-1, 0, 0};
  if (a.in_layout != IFQ_LAYOUT_U2_NHWC_PACKED || a.cin % 64 != 0 || a.m == 0)
    return best;
  double best_eff = -1.0;
  for (int v = 0; v < (int)(sizeof(kFast) / sizeof(kFast[0])); ++v) {
    const int bm = 32 * kFast[v].fm;
    const int bnmax = 32 * kFast[v].fn;
    const int64_t nco = (a.cout + bm - 1) / bm;
    const int64_t nb_min = (a.m + bnmax - 1) / bnmax;
    const int64_t waves = (nco * nb_min + kNumCUs - 1) / kNumCUs;
    int64_t nb = waves * kNumCUs / nco;
    if (nb < nb_min) nb = nb_min;
    if (nb > a.m) nb = a.m;
    const int64_t bn = (a.m + nb - 1) / nb;
    const int64_t blocks = nco * ((a.m + bn - 1) / bn);
    const double issued = (double)((blocks + kNumCUs - 1) / kNumCUs) * kNumCUs * bm * bnmax;
    const double eff = (double)a.m * a.cout / issued;
    if (eff > best_eff + 1e-9) {
      best_eff = eff;
      best = FastPlan{v, (int)bn, (int)((a.m + bn - 1) / bn)};
    }
  }
  return best;
}

template <int FM, int FN, int S, int D>
hipError_t launch_fast(ConvLaunch a, const FastPlan& pl, hipStream_t stream) {
  a.bn = pl.bn;
  dim3 grid(pl.blocks_m, (a.cout + 32 * FM - 1) / (32 * FM));
  hipLaunchKernelGGL((conv_u2<FM, FN, S, D>), grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

const char* conv_kernel_name(const ConvLaunch& a) {
  const FastPlan pl = plan_fast(a);
  if (pl.variant >= 0) return kFast[pl.variant].name;
  static const char* names[3][4] = {
      {"conv_igemm<16, 256, 1, 0>", "conv_igemm<32, 128, 1, 0>",
       "conv_igemm<64, 128, 2, 0>", "conv_igemm<128, 128, 2, 0>"},
      {"conv_igemm<16, 256, 1, 1>", "conv_igemm<32, 128, 1, 1>",
       "conv_igemm<64, 128, 2, 1>", "conv_igemm<128, 128, 2, 1>"},
      {"conv_igemm<16, 256, 1, 2>", "conv_igemm<32, 128, 1, 2>",
       "conv_igemm<64, 128, 2, 2>", "conv_igemm<128, 128, 2, 2>"}};
  return names[gather_kind(a)][tile_variant(a)];
}

hipError_t launch_conv(const ConvLaunch& a, hipStream_t stream) {
  if (a.m == 0) return hipSuccess;
  const FastPlan pl = plan_fast(a);
  switch (pl.variant) {
    case 0: return launch_fast<4, 7, 2, 5>(a, pl, stream);
    case 1: return launch_fast<2, 7, 2, 8>(a, pl, stream);
    case 2: return launch_fast<4, 4, 2, 6>(a, pl, stream);
    case 3: return launch_fast<2, 4, 2, 8>(a, pl, stream);
    default: break;
  }
  switch (gather_kind(a)) {
    case kGatherU2: return launch_gather<kGatherU2>(a, stream);
    case kGatherI8: return launch_gather<kGatherI8>(a, stream);
    default: return launch_gather<kGatherBytes>(a, stream);
  }
}

}  // namespace ifq
