// Fused epilogue of the conv kernels (device code, included by each kernel
// source): from the int32 sums a of a lane's accumulators to the layer
// output. One of
//   - the int32 sums themselves (layers without a quantizer),
//   - code = #{i : s*a > T_i}, the integer thresholds of Eq. (7)/(8),
//   - an identity residual join: code = #{i : s*a > T_i(x)}, with the
//     integer records of ifq_fold_join_table for the shortcut code x,
//   - a join with a 1x1 downsample's int32 sum d:
//     z = fma(p, a, fma(q, d, cc)), code = #{i : z > q_i} in fp64.
// Codes are packed four per byte (2-bit output) or one per byte into an LDS
// output tile and then written to HBM with wide coalesced stores.
#pragma once

#include <hip/hip_runtime.h>

#include "ifq_internal.h"

namespace ifq {
namespace {

// Bytes of LDS the per-channel parameters of bm output channels take at
// most (identity join tables of 4-bit codes: bm * 4 shortcut levels * 16).
__host__ __device__ constexpr int epilogue_param_bytes(int bm) { return bm * 4 * 16 * 4; }

// A conv join's parameters in LDS: the quantizer thresholds (16 doubles),
// then {p, q, cc} per channel. Kernel-argument arrays are never indexed with
// a runtime index (that would move the whole argument block to scratch).
constexpr int kJoinCoefOff = 16 * 8;

// Copies the per-channel epilogue parameters of output channels
// [co0, co0 + bm) into LDS once per workgroup: threshold records
// (bm * rec int32), identity join tables (bm * 4 * rec int32) or, for a
// conv join, the quantizer thresholds and bm * 3 coefficients. The caller
// brackets it with barriers.
__device__ __forceinline__ void stage_epilogue(const ConvLaunch& a, uint8_t* lds,
                                               int co0, int bm) {
  if (a.out_mode == 0) return;
  const int tid = threadIdx.x;
  const int nch = a.cout - co0 < bm ? a.cout - co0 : bm;
  if (a.join_kind == IFQ_JOIN_CONV || a.join_kind == IFQ_JOIN_CONV_FUSED) {
    double* qt = reinterpret_cast<double*>(lds);
#pragma unroll
    for (int q = 0; q < IFQ_MAX_THRESHOLDS; ++q)
      if (tid == q) qt[q] = a.qthr[q];
    double* dst = reinterpret_cast<double*>(lds + kJoinCoefOff);
    const double* src = a.coef + (int64_t)co0 * 3;
    for (int i = tid; i < bm * 3; i += blockDim.x) dst[i] = i < nch * 3 ? src[i] : 0.0;
    return;
  }
  const int per = a.join_kind == IFQ_JOIN_IDENTITY ? 4 * a.rec : a.rec;
  const int32_t* src =
      (a.join_kind == IFQ_JOIN_IDENTITY ? a.table : a.thr) + (int64_t)co0 * per;
  int32_t* dst = reinterpret_cast<int32_t*>(lds);
  for (int i = tid; i < bm * per; i += blockDim.x) dst[i] = i < nch * per ? src[i] : 0;
}

// s * v for a record sign s in {+1, -1}, without a multiply
__device__ __forceinline__ int sgn(int v, int s) {
  const int m = s >> 31;
  return (v ^ m) - m;
}

__device__ __forceinline__ int fdiv(int n, FastDiv d) {
  return (int)((__umulhi((uint32_t)n, d.mul) + (uint32_t)n) >> d.shift);
}

// Byte offset of channel co of output pixel p in a BLOCK64 code tensor of
// c channels over n images of howo pixels (dh divides by howo).
__device__ __forceinline__ int64_t block64_byte(int p, int co, int howo, FastDiv dh, int c) {
  const int nimg = fdiv(p, dh);
  const int64_t cell = ((int64_t)nimg * (c >> 6) + (co >> 6)) * howo + (p - nimg * howo);
  return cell * 16 + ((co & 63) >> 2);
}

// The 2-bit shortcut codes of channels co .. co+3 of pixel p, as the four
// low 2-bit fields of the result (field i = channel co+i).
__device__ __forceinline__ uint32_t shortcut_codes(const ConvLaunch& a, int p, int co) {
  const uint8_t* sc8 = reinterpret_cast<const uint8_t*>(a.shortcut);
  const int64_t e = (int64_t)p * a.cout + co;
  if (a.sc_layout == IFQ_LAYOUT_U2_NHWC_PACKED) return sc8[e >> 2];
  if (a.sc_layout == IFQ_LAYOUT_U2_BLOCK64)
    return sc8[block64_byte(p, co, a.ho * a.wo, a.div_howo, a.cout)];
  uint32_t b = 0;  // byte per code
  if ((a.cout & 3) == 0) {
    const uint32_t w4 = *reinterpret_cast<const uint32_t*>(sc8 + e);
#pragma unroll
    for (int i = 0; i < 4; ++i) b |= ((w4 >> (8 * i)) & 3u) << (2 * i);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (co + i < a.cout) b |= (sc8[e + i] & 3u) << (2 * i);
  }
  return b;
}

// Epilogue modes, decided once per launch (uniform branch) so that each
// inlined copy is straight-line code with only that mode's arithmetic.
enum EpiMode {
  kEpiI32 = 0,      // int32 sums are the output
  kEpiThr4 = 1,     // codes from {s, T1, T2, T3} records (2-bit output)
  kEpiThr = 2,      // codes from records of any length 2^out_bits
  kEpiTab4 = 3,     // identity join, records {s, T1, T2, T3} per shortcut code
  kEpiTab = 4,      // identity join, records of any length
  kEpiJoinConv = 5, // join with an int32 shortcut (1x1 downsample sums), fp64
};

// The accumulators of a lane are seen as NG groups of four consecutive output
// channels (co_of(g) .. co_of(g)+3) times FN pixel blocks: val(g, fn, i) is
// the sum of channel co_of(g)+i at local pixel pxl(fn) (negative: outside).
template <int MODE, int NG, int FN, class ValFn, class CoFn, class PixFn>
__device__ __forceinline__ void epilogue_mode(const ConvLaunch& a,
                                              const uint8_t* lds, ValFn val,
                                              CoFn co_of, int co_blk, int p0,
                                              PixFn pxl, uint8_t* otile,
                                              int orow) {
  int32_t* y32 = reinterpret_cast<int32_t*>(a.y);
  const int32_t* sc32 = reinterpret_cast<const int32_t*>(a.shortcut);
  const int32_t* prm = reinterpret_cast<const int32_t*>(lds);
  const bool in8 = a.in_bits == 8;
  const bool full4 = (a.cout & 3) == 0;
  const bool u2 = a.out_mode == 2;
#pragma unroll
  for (int g = 0; g < NG; ++g) {
    const int co = co_of(g);
    if (co >= a.cout) continue;
    const int lc = co - co_blk;
    int corr[4] = {0, 0, 0, 0};
    if (in8) {
#pragma unroll
      for (int i = 0; i < 4; ++i) corr[i] = co + i < a.cout ? 128 * a.rowsum[co + i] : 0;
    }
    // per-channel parameters, shared by the FN pixel blocks
    int4 tr[4];
    double cf[4][3];
    if constexpr (MODE == kEpiThr4) {
#pragma unroll
      for (int i = 0; i < 4; ++i) tr[i] = *reinterpret_cast<const int4*>(prm + (lc + i) * 4);
    }
    if constexpr (MODE == kEpiJoinConv) {
      const double* c = reinterpret_cast<const double*>(lds + kJoinCoefOff) + 3 * lc;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        cf[i][0] = c[3 * i];
        cf[i][1] = c[3 * i + 1];
        cf[i][2] = c[3 * i + 2];
      }
    }
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
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
        continue;
      }
      int code[4];
      if constexpr (MODE == kEpiThr4) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int sv = sgn(v[i], tr[i].x);
          code[i] = (sv > tr[i].y) + (sv > tr[i].z) + (sv > tr[i].w);
        }
      } else if constexpr (MODE == kEpiThr) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int32_t* t = prm + (lc + i) * a.rec;
          const int sv = sgn(v[i], t[0]);
          int c = 0;
          for (int q = 1; q <= a.nq; ++q) c += sv > t[q];
          code[i] = c;
        }
      } else if constexpr (MODE == kEpiTab4 || MODE == kEpiTab) {
        const uint32_t xs = shortcut_codes(a, p, co);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int x = (xs >> (2 * i)) & 3;
          if constexpr (MODE == kEpiTab4) {
            const int4 t = *reinterpret_cast<const int4*>(prm + ((lc + i) * 4 + x) * 4);
            const int sv = sgn(v[i], t.x);
            code[i] = (sv > t.y) + (sv > t.z) + (sv > t.w);
          } else {
            const int32_t* t = prm + ((lc + i) * 4 + x) * a.rec;
            const int sv = sgn(v[i], t[0]);
            int c = 0;
            for (int q = 1; q <= a.nq; ++q) c += sv > t[q];
            code[i] = c;
          }
        }
      } else {
        int d[4];
        if (full4) {
          const int4 s4 = *reinterpret_cast<const int4*>(sc32 + e);
          d[0] = s4.x; d[1] = s4.y; d[2] = s4.z; d[3] = s4.w;
        } else {
#pragma unroll
          for (int i = 0; i < 4; ++i) d[i] = co + i < a.cout ? sc32[e + i] : 0;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const double z = fma(cf[i][0], (double)v[i], fma(cf[i][1], (double)d[i], cf[i][2]));
          const double* qt = reinterpret_cast<const double*>(lds);
          int c = 0;
          for (int q = 0; q < a.nq; ++q) c += z > qt[q];
          code[i] = c;
        }
      }
      // codes go to the LDS output tile (row pl, this lane's 4 channels)
      if (u2) {
        otile[pl * orow + (lc >> 2)] =
            (uint8_t)(code[0] | (code[1] << 2) | (code[2] << 4) | (code[3] << 6));
      } else {
        *reinterpret_cast<uint32_t*>(otile + pl * orow + lc) =
            (uint32_t)code[0] | ((uint32_t)code[1] << 8) | ((uint32_t)code[2] << 16) |
            ((uint32_t)code[3] << 24);
      }
    }
  }
}

// Epilogue of one lane. Writes the optional int32 dump and the int32 sums
// directly; codes go to the LDS output tile otile (orow bytes per pixel),
// which copy_out_tile then writes to HBM. Per-channel parameters come from
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
#define IFQ_EPI(M) \
  epilogue_mode<M, NG, FN>(a, lds, val, co_of, co_blk, p0, pxl, otile, orow)
  if (a.out_mode == 0) {
    IFQ_EPI(kEpiI32);
  } else if (a.join_kind == IFQ_JOIN_CONV) {
    IFQ_EPI(kEpiJoinConv);
  } else if (a.join_kind == IFQ_JOIN_IDENTITY) {
    if (a.rec == 4) IFQ_EPI(kEpiTab4); else IFQ_EPI(kEpiTab);
  } else if (a.rec == 4) {
    IFQ_EPI(kEpiThr4);
  } else {
    IFQ_EPI(kEpiThr);
  }
#undef IFQ_EPI
}

// Writes the LDS output tile (codes of output channels co0 .. co0+bm-1 for
// the npx pixels starting at p0, orow bytes per pixel) to HBM with 16-byte
// (else 8-, 4- or 1-byte) stores. In NHWC layouts each pixel's channel range
// is one contiguous row; in BLOCK64 each 64-channel block of a pixel is a
// 16-byte cell and consecutive pixels of an image are consecutive cells.
__device__ __forceinline__ void copy_out_tile(const ConvLaunch& a, const uint8_t* otile,
                                              int orow, int co0, int bm, int p0,
                                              int npx) {
  if (a.out_mode == 0 || npx <= 0) return;
  const bool u2 = a.out_mode == 2;
  const int ch = a.cout - co0 < bm ? a.cout - co0 : bm;
  uint8_t* y8 = reinterpret_cast<uint8_t*>(a.y);
  const int tid = threadIdx.x;
  if (a.out_layout == IFQ_LAYOUT_U2_BLOCK64) {
    // cells of 64 channels (a tile of 32 channels fills half a cell)
    const int howo = a.ho * a.wo;
    const int G = a.cout >> 6;
    if (ch >= 64) {
      const int ng = ch >> 6;
      for (int u = tid; u < npx * ng; u += blockDim.x) {
        const int pl = u / ng, gg = u - pl * ng;
        const int p = p0 + pl;
        const int nimg = fdiv(p, a.div_howo);
        const int64_t cell =
            ((int64_t)nimg * G + (co0 >> 6) + gg) * howo + (p - nimg * howo);
        *reinterpret_cast<uint4*>(y8 + cell * 16) =
            *reinterpret_cast<const uint4*>(otile + pl * orow + gg * 16);
      }
    } else {
      for (int u = tid; u < npx; u += blockDim.x) {
        const int p = p0 + u;
        const int nimg = fdiv(p, a.div_howo);
        const int64_t cell = ((int64_t)nimg * G + (co0 >> 6)) * howo + (p - nimg * howo);
        *reinterpret_cast<uint2*>(y8 + cell * 16 + ((co0 & 63) >> 2)) =
            *reinterpret_cast<const uint2*>(otile + u * orow);
      }
    }
    return;
  }
  const int rbytes = u2 ? ch >> 2 : ch;              // bytes per pixel row
  const int pstride = u2 ? a.cout >> 2 : a.cout;      // output bytes per pixel
  const int cofs = u2 ? co0 >> 2 : co0;
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

// Max of two words of codes, field by field (Eq. 4 on codes): 2-bit fields
// (bit 1 of a field decides, then bit 0 among equals), or bytes below 128
// (a per-byte a >= b from the top bit of (a | 0x80) - b, which never
// borrows across bytes).
__device__ __forceinline__ uint32_t max_codes_u2(uint32_t a, uint32_t b) {
  constexpr uint32_t M = 0x55555555u;
  const uint32_t ha = (a >> 1) & M, la = a & M, hb = (b >> 1) & M, lb = b & M;
  const uint32_t lo = (ha & ~hb & la) | (hb & ~ha & lb) | (~(ha ^ hb) & (la | lb));
  return ((ha | hb) << 1) | (lo & M);
}
__device__ __forceinline__ uint32_t max_codes_u8(uint32_t a, uint32_t b) {
  const uint32_t ge = (((a | 0x80808080u) - b) & 0x80808080u) >> 7;   // 1 per byte a >= b
  const uint32_t mask = ge * 0xFFu;
  return (a & mask) | (b & ~mask);
}

// copy_out_tile with the max-pool of Eq. 4 fused: the tile's npx pixels are
// whole rows of whole windows (pool_img 0: k == stride, valid, the tile
// starting at a window row) or whole images (pool_img 1: any window), so
// every window of the tile's pooled pixels lies in the LDS tile. One 32-bit
// word of a pixel's channel row per thread and step, the max taken over the
// window's words (clipped at the bottom and right edges in SAME mode).
__device__ __forceinline__ void pool_out_tile(const ConvLaunch& a, const uint8_t* otile,
                                              int orow, int co0, int bm, int p0, int npx) {
  if (npx <= 0) return;
  const int k = a.pool_k, st = a.pool_s;
  const bool u2 = a.out_mode == 2;
  const int ch = a.cout - co0 < bm ? a.cout - co0 : bm;
  const int words = (u2 ? ch >> 2 : ch) >> 2;
  const int howo = a.ho * a.wo;
  // first pooled row (over all images) and pooled pixels of the tile
  int pr0, npo;
  if (a.pool_img) {
    const int i0 = fdiv(p0, a.div_howo);
    pr0 = i0 * a.pho;
    npo = fdiv(npx, a.div_howo) * a.pho * a.pwo;
  } else {
    pr0 = fdiv(p0, a.div_wo) / k;
    npo = npx / (k * k);
  }
  const int pstride = u2 ? a.cout >> 2 : a.cout;
  const int cofs = u2 ? co0 >> 2 : co0;
  const int phowo = a.pho * a.pwo;
  const bool b64 = a.out_layout == IFQ_LAYOUT_U2_BLOCK64;
  uint8_t* y8 = reinterpret_cast<uint8_t*>(a.y);
  for (int u = threadIdx.x; u < npo * words; u += blockDim.x) {
    const int po = u / words, wi = u - po * words;
    const int dr = fdiv(po, a.div_pwo);
    const int px = po - dr * a.pwo;
    const int pr = pr0 + dr;
    const int img = fdiv(pr, a.div_pho);
    const int py = pr - img * a.pho;
    const int y0 = py * st, x0 = px * st;
    const int y1 = y0 + k < a.ho ? y0 + k : a.ho, x1 = x0 + k < a.wo ? x0 + k : a.wo;
    const uint8_t* src = otile + (img * howo - p0) * orow + 4 * wi;
    uint32_t m = 0;
    for (int y = y0; y < y1; ++y)
      for (int x = x0; x < x1; ++x) {
        const uint32_t v = *reinterpret_cast<const uint32_t*>(src + (y * a.wo + x) * orow);
        m = u2 ? max_codes_u2(m, v) : max_codes_u8(m, v);
      }
    const int P = pr * a.pwo + px;
    int64_t off;
    if (b64) {
      const int gb = cofs + 4 * wi;   // byte of the pixel's 2-bit channel row
      off = (((int64_t)img * (a.cout >> 6) + (gb >> 4)) * phowo + (P - img * phowo)) * 16 +
            (gb & 15);
    } else {
      off = (int64_t)P * pstride + cofs + 4 * wi;
    }
    *reinterpret_cast<uint32_t*>(y8 + off) = m;
  }
}

}  // namespace
}  // namespace ifq
