// Device helpers shared by the two MFMA conv kernels (included by each
// kernel source): LDS-DMA loads with explicit vmcnt waits, the 2-bit code
// unpack, and the fused epilogue for the 32x32 accumulator layout.
#pragma once

#include <hip/hip_runtime.h>

#include "ifq_epilogue.h"
#include "ifq_internal.h"

namespace ifq {
namespace {

typedef int v2i __attribute__((ext_vector_type(2)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));

constexpr uint32_t kLow2 = 0x03030303u;

// Sixteen zero bytes in device memory: code loads that fall outside the
// image read them instead of branching around the load.
__device__ uint4 g_zero_cell;

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) uint8_t*)p;
}

// One wave-wide LDS-DMA load: 16 bytes per lane from src to LDS dst + 16*lane.
// M0 carries the LDS base; nothing else in these kernels uses M0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// dst must be wave-uniform (it is moved to SGPRs explicitly).
__device__ __forceinline__ void dma16(const void* src, uint32_t dst) {
  const uint32_t d = __builtin_amdgcn_readfirstlane(dst);
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
               :: "s"(d), "v"(src) : "memory", "m0");
}

// The same load with a wave-uniform 64-bit base in SGPRs and a per-lane
// 32-bit byte offset: no per-lane address arithmetic.
__device__ __forceinline__ void dma16s(const void* base, uint32_t voff, uint32_t dst) {
  const uint32_t d = __builtin_amdgcn_readfirstlane(dst);
  const uint64_t b = (uint64_t)(uintptr_t)base;
  // readfirstlane yields a signed int: widen each half as unsigned, or a low
  // half with bit 31 set would be sign-extended over the high half
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)b);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  const uint64_t bs = ((uint64_t)hi << 32) | (uint64_t)lo;
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, %2"
               :: "s"(d), "v"(voff), "s"(bs) : "memory", "m0");
}
#pragma clang diagnostic pop

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}

// Waits until at most ahead*CPW of this wave's loads are outstanding
// (0 <= ahead <= MAXA).
template <int MAXA, int CPW>
__device__ __forceinline__ void wait_ahead(int ahead) {
  if constexpr (MAXA <= 0) {
    wait_vmcnt<0>();
  } else {
    if (ahead >= MAXA) wait_vmcnt<MAXA * CPW>();
    else wait_ahead<MAXA - 1, CPW>(ahead);
  }
}

// Epilogue for the 32x32 accumulator layout when c_out % 32 == 0 and the
// records have 4 entries (2-bit codes): every lane computes codes for all of
// its accumulators without per-lane branches. A lane holds, per block
// (fm, fn), output channels cb + 8b + 4h + i (b, i = 0..3) of one pixel; the
// per-channel records of a 4-channel group are read from LDS once and used
// for the FN pixel blocks. Codes go to the LDS output tile (rows past the
// last pixel are never copied out); shortcut reads use a clamped pixel index.
enum Epi32 { kE32I32 = 0, kE32Thr4 = 1, kE32Tab4 = 2, kE32Conv = 3 };

template <int MODE, int FM, int FN>
__device__ __forceinline__ void epilogue32(const ConvLaunch& a, const uint8_t* lds,
                                           const v16i (&acc)[FM][FN], int wm, int wn,
                                           int h, int l32, int co0, int p0, int bn,
                                           uint8_t* otile, int orow, int32_t* y32) {
  const int32_t* prm = reinterpret_cast<const int32_t*>(lds);
  const bool u2 = a.out_mode == 2;
  const int howo = a.ho * a.wo;
  const uint8_t* sc8 = reinterpret_cast<const uint8_t*>(a.shortcut);
  const int32_t* sc32 = reinterpret_cast<const int32_t*>(a.shortcut);
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int cb = (wm * FM + fm) * 32;         // local first channel of the block
    if (co0 + cb >= a.cout) continue;           // uniform: whole 32-channel block
    // shortcut codes of the 32 channels of each pixel block (identity join):
    // byte 2b + h of the 8 holds the lane's channels cb + 8b + 4h .. +3
    uint32_t scw[FN][2];
    if constexpr (MODE == kE32Tab4) {
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        int p = p0 + wn * 32 * FN + fn * 32 + l32;
        p = p < a.m ? p : a.m - 1;
        const int co = co0 + cb;
        if (a.sc_layout == IFQ_LAYOUT_I8_NHWC) {
          const uint8_t* src = sc8 + (int64_t)p * a.cout + co;
          uint32_t w[2] = {0u, 0u};
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const uint32_t v = *reinterpret_cast<const uint32_t*>(src + 8 * b + 4 * h) & kLow2;
            const uint32_t byte = v | (v >> 6) | (v >> 12) | (v >> 18);
            w[b >> 1] |= (byte & 0xFFu) << (8 * (2 * (b & 1) + h));
          }
          scw[fn][0] = w[0];
          scw[fn][1] = w[1];
        } else {
          int64_t off;
          if (a.sc_layout == IFQ_LAYOUT_U2_BLOCK64) {
            const int nimg = fdiv(p, a.div_howo);
            off = (((int64_t)nimg * (a.cout >> 6) + (co >> 6)) * howo + (p - nimg * howo)) * 16 +
                  ((co & 63) >> 2);
          } else {
            off = ((int64_t)p * a.cout + co) >> 2;
          }
          const uint2 v = *reinterpret_cast<const uint2*>(sc8 + off);
          scw[fn][0] = v.x;
          scw[fn][1] = v.y;
        }
      }
    }
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int cl = cb + 8 * b + 4 * h;        // local channel of value 4b + 0
      int4 tr[4];
      double cf[4][3];
      if constexpr (MODE == kE32Thr4) {
#pragma unroll
        for (int i = 0; i < 4; ++i) tr[i] = *reinterpret_cast<const int4*>(prm + (cl + i) * 4);
      }
      if constexpr (MODE == kE32Conv) {
        const double* c = reinterpret_cast<const double*>(lds + kJoinCoefOff) + 3 * cl;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          cf[i][0] = c[3 * i];
          cf[i][1] = c[3 * i + 1];
          cf[i][2] = c[3 * i + 2];
        }
      }
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        const int pl = wn * 32 * FN + fn * 32 + l32;
        int v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = acc[fm][fn][4 * b + i];
        if constexpr (MODE == kE32I32) {
          if (pl < bn && p0 + pl < a.m)
            *reinterpret_cast<int4*>(y32 + (int64_t)(p0 + pl) * a.cout + co0 + cl) =
                int4{v[0], v[1], v[2], v[3]};
          continue;
        }
        int code[4];
        if constexpr (MODE == kE32Thr4) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int sv = sgn(v[i], tr[i].x);
            code[i] = (sv > tr[i].y) + (sv > tr[i].z) + (sv > tr[i].w);
          }
        } else if constexpr (MODE == kE32Tab4) {
          const uint32_t xs = (scw[fn][b >> 1] >> (8 * (2 * (b & 1) + h))) & 0xFFu;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int x = (xs >> (2 * i)) & 3;
            const int4 t = *reinterpret_cast<const int4*>(prm + ((cl + i) * 4 + x) * 4);
            const int sv = sgn(v[i], t.x);
            code[i] = (sv > t.y) + (sv > t.z) + (sv > t.w);
          }
        } else {
          int p = p0 + pl;
          p = p < a.m ? p : a.m - 1;
          const int4 d = *reinterpret_cast<const int4*>(sc32 + (int64_t)p * a.cout + co0 + cl);
          const int dv[4] = {d.x, d.y, d.z, d.w};
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const double z = fma(cf[i][0], (double)v[i], fma(cf[i][1], (double)dv[i], cf[i][2]));
            const double* qt = reinterpret_cast<const double*>(lds);
            int c = 0;
            for (int q = 0; q < a.nq; ++q) c += z > qt[q];
            code[i] = c;
          }
        }
        if (u2) {
          otile[pl * orow + (cl >> 2)] =
              (uint8_t)(code[0] | (code[1] << 2) | (code[2] << 4) | (code[3] << 6));
        } else {
          *reinterpret_cast<uint32_t*>(otile + pl * orow + cl) =
              (uint32_t)code[0] | ((uint32_t)code[1] << 8) | ((uint32_t)code[2] << 16) |
              ((uint32_t)code[3] << 24);
        }
      }
    }
  }
}

typedef short s16x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// Threshold records of 2-bit outputs laid out for packed 16-bit compares,
// 32 bytes per group of four consecutive output channels c .. c+3:
//   words 0..2  {T'_i(c), T'_i(c+1)} as int16 pairs, i = 1..3
//   words 3..5  the same for (c+2, c+3)
//   word  6     xor mask of the flipped channels, in the bit layout the codes
//               are packed in by epilogue_thr_pk
// with T' = T for s = +1 and T' = -T - 1 for s = -1. For an integer sum a,
// -a > T holds exactly when a < -T, i.e. when a > -T - 1 is false, so a
// flipped channel's code #{i : -a > T_i} is 3 - #{i : a > T'_i}, which is
// that count xor 3. Needs |T| and |a| below 2^15 (3*K <= 32766); their
// difference can reach 2^16 and is taken with a saturating subtract.
constexpr int kPkRecBytes = 32;

// recs: the bm channels' {s, T1, T2, T3} records (already in LDS; records of
// channels past c_out may hold anything, their codes are never stored).
__device__ __forceinline__ void stage_thr_pk(const int4* recs, uint8_t* lds, int bm) {
  for (int gq = threadIdx.x; gq < bm / 4; gq += blockDim.x) {
    uint32_t w[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int4 r = recs[4 * gq + i];
      const bool flip = r.x < 0;
      const int t[3] = {r.y, r.z, r.w};
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        const int v = flip ? -t[k] - 1 : t[k];
        w[(i >> 1) * 3 + k] |= ((uint32_t)v & 0xFFFFu) << (16 * (i & 1));
      }
      if (flip) w[6] |= 3u << ((i & 1) * 16 + (i >> 1) * 4);
    }
    uint4* dst = reinterpret_cast<uint4*>(lds + gq * kPkRecBytes);
    dst[0] = uint4{w[0], w[1], w[2], w[3]};
    dst[1] = uint4{w[4], w[5], w[6], w[7]};
  }
}

// #{i : a > T'_i} for both halves of a packed pair: T' - a is negative
// exactly when a > T'. With T' and a in [-2^15, 2^15) the difference spans
// twice the int16 range: the subtract saturates (v_pk_sub_i16 with clamp),
// which keeps its sign, where a wrapping one would flip it.
__device__ __forceinline__ uint32_t count3_pk(s16x2 p, uint32_t w1, uint32_t w2, uint32_t w3) {
  const s16x2 d1 = __builtin_elementwise_sub_sat(__builtin_bit_cast(s16x2, w1), p);
  const s16x2 d2 = __builtin_elementwise_sub_sat(__builtin_bit_cast(s16x2, w2), p);
  const s16x2 d3 = __builtin_elementwise_sub_sat(__builtin_bit_cast(s16x2, w3), p);
  const u16x2 s1 = __builtin_bit_cast(u16x2, d1) >> (unsigned short)15;
  const u16x2 s2 = __builtin_bit_cast(u16x2, d2) >> (unsigned short)15;
  const u16x2 s3 = __builtin_bit_cast(u16x2, d3) >> (unsigned short)15;
  return __builtin_bit_cast(uint32_t, s1) + __builtin_bit_cast(uint32_t, s2) +
         __builtin_bit_cast(uint32_t, s3);
}

// Code of two sums (int16 halves of p) against thresholds sorted ascending,
// w1 <= w2 <= w3 (each an int16 pair): the count of thresholds below a sum
// is the same in any order, and with sorted ones it is 2 [p > T2] plus
// [p > T3] where p > T2, else [p > T1]. Saturating differences keep the sign.
__device__ __forceinline__ uint32_t count3_sorted_pk(s16x2 p, uint32_t w1, uint32_t w2,
                                                     uint32_t w3) {
  const s16x2 d2 = __builtin_elementwise_sub_sat(__builtin_bit_cast(s16x2, w2), p);
  uint32_t m = __builtin_bit_cast(uint32_t, d2 >> (short)15);   // 0xFFFF: p > T2
  // opaque to the optimizer, which would otherwise turn the bit-field select
  // below into compares and selects per half
  asm("" : "+v"(m));
  const uint32_t ts = (m & w3) | (~m & w1);
  const s16x2 ds = __builtin_elementwise_sub_sat(__builtin_bit_cast(s16x2, ts), p);
  const uint32_t lo = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, ds) >> (unsigned short)15);
  return (m & 0x00020002u) | lo;
}

// Threshold epilogue for 2-bit packed output from the records of
// stage_thr_pk: per lane, accumulator blocks fm of rows (wm*NB + fm)*32 and
// the pixel column pl of the output tile. Each group of four channels of a
// pixel becomes one byte: codes packed two per 16-bit half, counted with
// packed 16-bit subtracts, flipped channels xor'ed, then folded into a byte.
template <int NB>
__device__ __forceinline__ void epilogue_thr_pk(const ConvLaunch& a, const uint8_t* lds,
                                                const v16i (&acc)[NB], int wm, int h, int co0,
                                                int pl, uint8_t* otile, int orow) {
#pragma unroll
  for (int fm = 0; fm < NB; ++fm) {
    const int cb = (wm * NB + fm) * 32;
    if (co0 + cb >= a.cout) continue;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int cl = cb + 8 * b + 4 * h;
      const uint4* rec = reinterpret_cast<const uint4*>(lds + (cl >> 2) * kPkRecBytes);
      const uint4 r0 = rec[0], r1 = rec[1];
      const s16x2 p01 = __builtin_amdgcn_cvt_pk_i16(acc[fm][4 * b], acc[fm][4 * b + 1]);
      const s16x2 p23 = __builtin_amdgcn_cvt_pk_i16(acc[fm][4 * b + 2], acc[fm][4 * b + 3]);
      const uint32_t c01 = count3_pk(p01, r0.x, r0.y, r0.z);
      const uint32_t c23 = count3_pk(p23, r0.w, r1.x, r1.y);
      const uint32_t t = (c01 | (c23 << 4)) ^ r1.z;
      otile[pl * orow + (cl >> 2)] = (uint8_t)(t | (t >> 14));
    }
  }
}

// Identity-join records laid out for packed 16-bit compares. The shortcut
// code x of each channel selects that channel's thresholds T_i(c, x) (the
// records of ifq_fold_join_table; their sign s depends on the channel only).
// Per group of four channels c .. c+3, 512 bytes: for the pair (c, c+1) 16
// entries of 16 bytes, entry x0 | x1 << 2 holding {T'_i(c, x0), T'_i(c+1, x1)}
// as int16 pairs (i = 1..3) and the pair's xor mask of flipped channels;
// then the same for (c+2, c+3). T' as for stage_thr_pk.
constexpr int kIdjGroupBytes = 512;

// tbl: the bm channels' [4][4] int32 records (global or LDS); channels at or
// past nch get plain records (their codes are never stored). sh > 0: for
// sums kept as 2^sh a, each T' is clamped to [-bnd-1, bnd] (bnd bounds |a|,
// so no comparison changes) and scaled by 2^sh.
__device__ __forceinline__ void stage_idj_pk(const int32_t* tbl, uint8_t* lds, int bm, int nch,
                                             int sh = 0, int bnd = 0) {
  for (int e = threadIdx.x; e < (bm / 4) * 32; e += blockDim.x) {
    const int gq = e >> 5, pr = (e >> 4) & 1, combo = e & 15;
    const int x[2] = {combo & 3, combo >> 2};
    uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int c = 4 * gq + 2 * pr + j;
      int4 r = int4{1, 0, 0, 0};
      if (c < nch) r = *reinterpret_cast<const int4*>(tbl + (c * 4 + x[j]) * 4);
      const bool flip = r.x < 0;
      const int t[3] = {r.y, r.z, r.w};
      int v[3];
#pragma unroll
      for (int k = 0; k < 3; ++k) {
        v[k] = flip ? -t[k] - 1 : t[k];
        if (sh > 0) v[k] = (v[k] < -bnd - 1 ? -bnd - 1 : (v[k] > bnd ? bnd : v[k])) * (1 << sh);
        v[k] = (int16_t)v[k];     // compared as 16-bit halves
      }
      // sorted ascending for count3_sorted_pk (the count is order-free)
      const int lo = min(v[0], min(v[1], v[2])), hi = max(v[0], max(v[1], v[2]));
      const int md = max(min(v[0], v[1]), min(max(v[0], v[1]), v[2]));
      w[0] |= ((uint32_t)lo & 0xFFFFu) << (16 * j);
      w[1] |= ((uint32_t)md & 0xFFFFu) << (16 * j);
      w[2] |= ((uint32_t)hi & 0xFFFFu) << (16 * j);
      if (flip) w[3] |= 3u << (16 * j);
    }
    *reinterpret_cast<uint4*>(lds + gq * kIdjGroupBytes + pr * 256 + combo * 16) =
        uint4{w[0], w[1], w[2], w[3]};
  }
}

// The 2-bit shortcut codes of output channels co .. co+31 of pixel p
// (8 bytes, channel co + 4k + i in bits 2i of byte k), for shortcut layouts
// U2_NHWC_PACKED and U2_BLOCK64 (co % 32 == 0).
__device__ __forceinline__ uint2 shortcut8(const ConvLaunch& a, int p, int co) {
  const uint8_t* sc8 = reinterpret_cast<const uint8_t*>(a.shortcut);
  int64_t off;
  if (a.sc_layout == IFQ_LAYOUT_U2_BLOCK64) {
    const int howo = a.ho * a.wo;
    const int nimg = fdiv(p, a.div_howo);
    off = (((int64_t)nimg * (a.cout >> 6) + (co >> 6)) * howo + (p - nimg * howo)) * 16 +
          ((co & 63) >> 2);
  } else {
    off = ((int64_t)p * a.cout + co) >> 2;
  }
  return *reinterpret_cast<const uint2*>(sc8 + off);
}

// Identity-join epilogue for 2-bit packed output from the records of
// stage_idj_pk; sc[fm]: shortcut8 of the lane's pixel for block fm.
// CK as for epilogue_thr_pk_t.
template <int NB, bool CK = true>
__device__ __forceinline__ void epilogue_idj_pk(const ConvLaunch& a, const uint8_t* lds,
                                                const v16i (&acc)[NB], const uint2 (&sc)[NB],
                                                int wm, int h, int co0, int pl,
                                                uint8_t* otile, int orow) {
#pragma unroll
  for (int fm = 0; fm < NB; ++fm) {
    const int cb = (wm * NB + fm) * 32;
    if (CK && co0 + cb >= a.cout) continue;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int cl = cb + 8 * b + 4 * h;
      const uint32_t word = (b >> 1) ? sc[fm].y : sc[fm].x;
      const uint32_t xs = word >> (8 * (2 * (b & 1) + h));
      const uint8_t* g = lds + (cl >> 2) * kIdjGroupBytes;
      const uint4 e01 = *reinterpret_cast<const uint4*>(g + (xs & 15u) * 16);
      const uint4 e23 = *reinterpret_cast<const uint4*>(g + 256 + ((xs >> 4) & 15u) * 16);
      const s16x2 p01 = __builtin_amdgcn_cvt_pk_i16(acc[fm][4 * b], acc[fm][4 * b + 1]);
      const s16x2 p23 = __builtin_amdgcn_cvt_pk_i16(acc[fm][4 * b + 2], acc[fm][4 * b + 3]);
      const uint32_t c01 = count3_sorted_pk(p01, e01.x, e01.y, e01.z) ^ e01.w;
      const uint32_t c23 = count3_sorted_pk(p23, e23.x, e23.y, e23.z) ^ e23.w;
      const uint32_t t = c01 | (c23 << 4);
      otile[pl * orow + (cl >> 2)] = (uint8_t)(t | (t >> 14));
    }
  }
}

// Conv-join epilogue with both sums in registers (fused downsample): per
// output z = fma(p, a, fma(q, d, cc)) in fp64 with the per-channel {p, q, cc}
// staged at kJoinCoefOff, code = #{i : z > q_i} for the three quantizer
// thresholds of 2-bit output, four codes packed per byte.
template <int NB>
__device__ __forceinline__ void epilogue_cjoin(const ConvLaunch& a, const uint8_t* lds,
                                               const v16i (&acc)[NB], const v16i (&accd)[NB],
                                               int wm, int h, int co0, int pl, uint8_t* otile,
                                               int orow) {
  const double q1 = a.qthr[0], q2 = a.qthr[1], q3 = a.qthr[2];
  const double* cf = reinterpret_cast<const double*>(lds + kJoinCoefOff);
#pragma unroll
  for (int fm = 0; fm < NB; ++fm) {
    const int cb = (wm * NB + fm) * 32;
    if (co0 + cb >= a.cout) continue;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int cl = cb + 8 * b + 4 * h;
      uint32_t byte = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const double* c = cf + 3 * (cl + i);
        const double z = fma(c[0], (double)acc[fm][4 * b + i],
                             fma(c[1], (double)accd[fm][4 * b + i], c[2]));
        const uint32_t code = (uint32_t)(z > q1) + (uint32_t)(z > q2) + (uint32_t)(z > q3);
        byte |= code << (2 * i);
      }
      otile[pl * orow + (cl >> 2)] = (uint8_t)byte;
    }
  }
}

// ---- Epilogues for the transposed accumulator layout --------------------
// With the codes as the MFMA's A operand and the weights as B, a lane
// (h, l32) holds per 32x32 block ONE output channel (column l32) for the 16
// pixel rows 8b + 4h + i (register v = 4b + i) of its wave's 32-pixel column.
// Its channel's thresholds or join coefficients are read once per block, not
// once per output; the four channels of an output byte are the four lanes of
// an aligned quad, merged with two DPP ORs, and lane t = l32 & 3 of the quad
// stores the byte of pixel row 8b + 4h + t.

// OR of w over the four lanes of the lane's quad (every lane gets it).
__device__ __forceinline__ uint32_t quad_or(uint32_t w) {
  w |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w, 0xB1, 0xF, 0xF, false);  // lane ^ 1
  w |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)w, 0x4E, 0xF, 0xF, false);  // lane ^ 2
  return w;
}

__device__ __forceinline__ uint32_t pk2_i16(int v) { return ((uint32_t)v & 0xFFFFu) * 0x10001u; }

// The packed thresholds of one channel for the transposed epilogue: the
// record's three thresholds (sign rule applied, clamped and scaled by 2^SH
// where SH > 0), sorted ascending as int16 pairs, and its flip.
struct ThrPk {
  uint32_t w1, w2, w3;
  bool flip;
};
template <int SH>
__device__ __forceinline__ ThrPk thr_pk_of(const int4 r, int bnd) {
  const bool flip = r.x < 0;
  auto thr = [&](int v) {
    if constexpr (SH > 0) v = (v < -bnd - 1 ? -bnd - 1 : (v > bnd ? bnd : v)) * (1 << SH);
    return (int)(int16_t)v;    // compared as 16-bit halves
  };
  const int v1 = thr(flip ? -r.y - 1 : r.y);
  const int v2 = thr(flip ? -r.z - 1 : r.z);
  const int v3 = thr(flip ? -r.w - 1 : r.w);
  const int tlo = min(v1, min(v2, v3)), thi = max(v1, max(v2, v3));
  const int tmd = max(min(v1, v2), min(max(v1, v2), v3));
  return ThrPk{pk2_i16(tlo), pk2_i16(tmd), pk2_i16(thi), flip};
}

// One 32x32 block of the transposed threshold epilogue, for the lane's
// channel cl (thresholds th) and pixel rows pl0 + 0..31.
__device__ __forceinline__ void epilogue_thr_pk_block(const v16i& acc, const ThrPk& th, int h,
                                                      int l32, int cl, int pl0, uint8_t* otile,
                                                      int orow) {
  const int t = l32 & 3;
  const uint32_t r1 = (t & 1) ? 2u : 30u, r2 = (t & 2) ? 4u : 28u;
  const uint32_t k1 = (t & 1) ? 0xCCCCCCCCu : 0x33333333u;
  const uint32_t k2 = (t & 2) ? 0xF0F0F0F0u : 0x0F0F0F0Fu;
  uint32_t wd = 0;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const s16x2 p01 = __builtin_amdgcn_cvt_pk_i16(acc[4 * b], acc[4 * b + 1]);
    const s16x2 p23 = __builtin_amdgcn_cvt_pk_i16(acc[4 * b + 2], acc[4 * b + 3]);
    const uint32_t c01 = count3_sorted_pk(p01, th.w1, th.w2, th.w3);
    const uint32_t c23 = count3_sorted_pk(p23, th.w1, th.w2, th.w3);
    wd |= (c01 | (c23 << 8)) << (2 * b);
  }
  if (th.flip) wd = ~wd;
  uint32_t q = (uint32_t)__builtin_amdgcn_mov_dpp((int)wd, 0xB1, 0xF, 0xF, true);
  q = __builtin_rotateright32(q, r1);
  wd = q ^ ((wd ^ q) & k1);
  q = (uint32_t)__builtin_amdgcn_mov_dpp((int)wd, 0x4E, 0xF, 0xF, true);
  q = __builtin_rotateright32(q, r2);
  wd = q ^ ((wd ^ q) & k2);
  uint8_t* o = otile + (pl0 + 8 * t + 4 * h) * orow + (cl >> 2);
  const uint32_t w8 = wd >> 8;
  o[0] = (uint8_t)wd;
  o[orow] = (uint8_t)(wd >> 16);
  o[2 * orow] = (uint8_t)w8;
  o[3 * orow] = (uint8_t)(w8 >> 16);
}

// Threshold epilogue (2-bit codes, c_out % 32 == 0, 27 * c_in <= 32766) from
// the raw {s, T1, T2, T3} records of the tile's channels (recs[c - co0]),
// with the same packed 16-bit compare and sign flip as epilogue_thr_pk.
// SH > 0: the sums are 2^SH a (|2^SH a| < 2^15); the thresholds, clamped to
// [-B-1, B] (B = 27 c_in bounds |a|, so no comparison changes), are scaled
// the same way.
// Each lane holds one channel of a block; its 16 codes are gathered into one
// word (byte k: pixels {0, 2, 1, 3}[k] of the four row groups, group g in
// bits 2g), and a 4x4 transpose of 2-bit fields across the lane quad (two
// exchanges with the lanes at xor 1 and xor 2, each a rotate and a bit-field
// select) leaves lane t with the bytes of row group t: the four channels of
// the quad for each of its pixels.
// CK false: the caller guarantees every block's channels exist (no check,
// so the blocks of one call site form one straight-line region).
template <int NB, int SH = 0, bool CK = true>
__device__ __forceinline__ void epilogue_thr_pk_t(const ConvLaunch& a, const int4* recs,
                                                  const v16i (&acc)[NB], int wm, int h,
                                                  int l32, int co0, int pl0, uint8_t* otile,
                                                  int orow) {
  const int bnd = 27 * a.cin;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int cb = (wm * NB + j) * 32;
    if (CK && co0 + cb >= a.cout) continue;
    const int cl = cb + l32;
    epilogue_thr_pk_block(acc[j], thr_pk_of<SH>(recs[cl], bnd), h, l32, cl, pl0, otile, orow);
  }
}

// Conv-join epilogue (fused downsample), the same fp64 evaluation as
// epilogue_cjoin: z = fma(p, a, fma(q, d, cc)), code = #{i : z > q_i}.
template <int NB>
__device__ __forceinline__ void epilogue_cjoin_t(const ConvLaunch& a, const uint8_t* lds,
                                                 const v16i (&acc)[NB], const v16i (&accd)[NB],
                                                 int wm, int h, int l32, int co0, int pl0,
                                                 uint8_t* otile, int orow) {
  const double q1 = a.qthr[0], q2 = a.qthr[1], q3 = a.qthr[2];
  // the three thresholds sorted (the count #{i : z > q_i} is order-free):
  // then the code is 2 [z > mid] + [z > (z > mid ? high : low)], two fp64
  // compares per output instead of three, the same count for every z
  const double qlo = fmin(q1, fmin(q2, q3)), qhi = fmax(q1, fmax(q2, q3));
  const double qmd = fmax(fmin(q1, q2), fmin(fmax(q1, q2), q3));
  const double* cf = reinterpret_cast<const double*>(lds + kJoinCoefOff);
  const int t = l32 & 3;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int cb = (wm * NB + j) * 32;
    if (co0 + cb >= a.cout) continue;
    const int cl = cb + l32;
    const double p = cf[3 * cl], q = cf[3 * cl + 1], cc = cf[3 * cl + 2];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      uint32_t w = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const double z = fma(p, (double)acc[j][4 * b + i], fma(q, (double)accd[j][4 * b + i], cc));
        const bool up = z > qmd;
        const uint32_t code = 2u * (uint32_t)up + (uint32_t)(z > (up ? qhi : qlo));
        w |= code << (8 * i);
      }
      w = quad_or(w << (2 * t));
      otile[(pl0 + 8 * b + 4 * h + t) * orow + (cl >> 2)] = (uint8_t)(w >> (8 * t));
    }
  }
}

// int32 sums of the tile to dump[p * c_out + c] (diagnostic path).
template <int NB>
__device__ __forceinline__ void dump_acc_t(const ConvLaunch& a, const v16i (&acc)[NB], int wm,
                                           int h, int l32, int co0, int p0, int pl0, int bn,
                                           int32_t* dump) {
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int c = co0 + (wm * NB + j) * 32 + l32;
    if (c >= a.cout) continue;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int pl = pl0 + 8 * (v >> 2) + 4 * h + (v & 3);
      if (pl < bn && p0 + pl < a.m) dump[(int64_t)(p0 + pl) * a.cout + c] = acc[j][v];
    }
  }
}

// 16 two-bit codes (one 32-bit word of a cell) -> 16 int8 operand bytes.
__device__ __forceinline__ v4i unpack2(uint32_t u) {
  return v4i{(int)(u & kLow2), (int)((u >> 2) & kLow2), (int)((u >> 4) & kLow2),
             (int)((u >> 6) & kLow2)};
}

}  // namespace
}  // namespace ifq
