// Persistent 3x3 kernel for layers whose weight slab of one 64-channel
// output slice fits in LDS (3x3, stride 1 or 2, pad 1, 2-bit BLOCK64 codes,
// c_in a multiple of 64), on gfx950 (MI355X). The contraction and epilogues
// are those of the register-blocked kernel in ifq_conv_w2.hip: the integer
// part of Eq. (1) on v_mfma_i32_32x32x32_i8 (or exactly on the fp4 scaled
// MFMA, F4), then the 2-bit threshold epilogue of Eq. (7)/(8) (MODE 0) or the
// identity residual join (MODE 1).
//
// Layers with many output pixels and a short K (the 56x56 64-channel layers
// of a ResNet-18 body: K = 576, about three 64x256 tiles per CU) spend most
// of a one-tile-per-workgroup kernel in each tile's prologue and epilogue.
// Here a workgroup loads the weights of its channel slice into LDS once and
// then runs a contiguous range of pixel tiles:
//  - a tile's main loop reads weights and input window from LDS only: no
//    waits and no barriers inside it;
//  - the window (and the identity join's shortcut cells) of the next tile
//    load into the other half of a double buffer while the current tile's
//    main loop and epilogue run;
//  - the output tile is double-buffered too, so one barrier per tile
//    separates every producer from its consumer;
//  - two workgroups share a CU, so one's epilogue (VALU) can overlap the
//    other's MFMAs.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "ifq_epilogue.h"
#include "ifq_internal.h"
#include "ifq_mfma_common.h"

namespace ifq {
namespace {

constexpr int kWpTaps = 9;

__host__ __device__ constexpr int wp_round64(int v) { return (v + 63) & ~63; }

// The images (segments) the output pixels [p0, p0 + bn) of a tile touch and
// the input row span of each (the window layout of ifq_conv_w2.hip: per
// channel block, each segment's rows of cells rounded up to 64 cells).
struct WpTile {
  int n_first, nseg, oy_first, oy_last;
  __device__ void init(const ConvLaunch& a, int p0, int bn) {
    const int howo = a.ho * a.wo;
    const int pend = (p0 + bn < a.m ? p0 + bn : a.m) - 1;
    n_first = fdiv(p0, a.div_howo);
    const int n_last = fdiv(pend, a.div_howo);
    nseg = n_last - n_first + 1;
    oy_first = fdiv(p0 - n_first * howo, a.div_wo);
    oy_last = fdiv(pend - n_last * howo, a.div_wo);
  }
  __device__ int rows(const ConvLaunch& a, int i, int& iya) const {
    const int oya = i == 0 ? oy_first : 0;
    const int oyb = i == nseg - 1 ? oy_last : a.ho - 1;
    iya = oya * a.stride - 1;
    iya = iya < 0 ? 0 : iya;
    int iyb = oyb * a.stride + 1;
    iyb = iyb > a.h - 1 ? a.h - 1 : iyb;
    return iyb - iya + 1;
  }
};

template <int WN, int FM, int FN, int MODE, bool F4, int OCC, int WGTB, int WINB>
__global__ __launch_bounds__(64 * WN, (WN / 4) * OCC) void conv_wp(ConvLaunch a) {
  constexpr bool SW = MODE == 0;                 // transposed sums
  constexpr int NW = WN;
  constexpr int BM = 32 * FM;
  constexpr int BN = 32 * FN * WN;
  constexpr int KH = F4 ? 1 : 2;                 // 1 KB chunks per row block and K64 step
  constexpr int RB = FM;
  static_assert(NW % 4 == 0 && BM == 64, "waves; one 64-channel slice per workgroup");
  // LDS: the slice's weights, two windows, the per-channel records, two
  // shortcut buffers (identity join), two output tiles. The identity join's
  // raw records are only read while the packed ones are staged, before the
  // second window is first written: they sit in that window.
  constexpr int WGT = 0;
  constexpr int WIN = WGTB;
  constexpr int TBL = SW ? WIN + 2 * WINB : WIN + WINB;
  constexpr int TBL_BYTES = SW ? BM * 16 : 0;
  static_assert(SW || BM * 64 <= WINB, "raw join records inside the second window");
  constexpr int EPI = WIN + 2 * WINB + TBL_BYTES;   // past both windows
  constexpr int EPI_BYTES = SW ? 0 : BM * 128;
  constexpr int SCB = EPI + EPI_BYTES;
  constexpr int SC_BYTES = SW ? 0 : (BM / 64) * BN * 16;
  constexpr int OTL = SCB + 2 * SC_BYTES;
  constexpr int OUT_BYTES = BN * BM / 4;
  constexpr int LDS_BYTES = OTL + 2 * OUT_BYTES;
  static_assert(LDS_BYTES <= 160 * 1024 / OCC, "LDS");

  __shared__ __attribute__((aligned(1024))) uint8_t lds[LDS_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wn = wave;
  const int h = lane >> 5;
  const int l32 = lane & 31;
  const int bn = a.bn;
  const int co0 = blockIdx.y * BM;
  const int G = a.cin >> 6;
  const int H = a.h, W = a.w, Wo = a.wo, st = a.stride;
  const int howo = a.ho * a.wo;
  const int HW = H * W;
  const int wcells = a.wcells;                   // host: the largest tile window
  const int wstr = (wcells + 1) * 16;            // block window + its zero cell
  const int ntm = (a.m + bn - 1) / bn;
  const int t_begin = blockIdx.x * a.tiles_wg;
  const int t_end = t_begin + a.tiles_wg < ntm ? t_begin + a.tiles_wg : ntm;
  const uint32_t lds0 = lds_addr(lds);
  const uint8_t* zero_src = reinterpret_cast<const uint8_t*>(&g_zero_cell);
  constexpr int orow = BM / 4;

  // the window of tile tt into window buffer b: chunk j of segment i is 64
  // cells of that image's input rows, the same chunk for every channel block;
  // wave w takes the chunks w, w + NW, .. of the segments' chunk list
  auto load_window = [&](int tt, int b) {
    WpTile tl;
    tl.init(a, tt * bn, bn);
    const uint32_t dst0 = lds0 + WIN + b * WINB;
    int off = 0, jbase = 0;
    for (int i = 0; i < tl.nseg; ++i) {
      int iya;
      const int cells = tl.rows(a, i, iya) * W;
      const int nch = wp_round64(cells) >> 6;
      int j = wave - jbase;
      j += j < 0 ? ((-j + NW - 1) / NW) * NW : 0;
      for (; j < nch; j += NW) {
        const int c = j * 64 + lane;
        const int64_t src = ((int64_t)(tl.n_first + i) * G * HW + iya * W + c) * 16;
        for (int g = 0; g < G; ++g)
          dma16(c < cells ? a.x + src + (int64_t)g * HW * 16 : zero_src,
                dst0 + (uint32_t)(g * wstr + (off + j * 64) * 16));
      }
      jbase += nch;
      off += wp_round64(cells);
    }
  };
  // the shortcut cells of tile tt's pixels (identity join) into buffer b
  auto load_shortcut = [&](int tt, int b) {
    const int p0 = tt * bn;
    const uint8_t* sc8 = reinterpret_cast<const uint8_t*>(a.shortcut);
    const int ncx = (bn + 63) >> 6;
    for (int q = wave; q < (BM / 64) * ncx; q += NW) {
      const int gbl = q / ncx, j = q - gbl * ncx;
      const int pl = j * 64 + lane, p = p0 + pl, gb = (co0 >> 6) + gbl;
      const uint8_t* src = zero_src;
      if (pl < bn && p < a.m && gb * 64 < a.cout) {
        if (a.sc_layout == IFQ_LAYOUT_U2_BLOCK64) {
          const int nimg = fdiv(p, a.div_howo);
          src = sc8 + (((int64_t)nimg * (a.cout >> 6) + gb) * howo + (p - nimg * howo)) * 16;
        } else {
          src = sc8 + ((int64_t)p * a.cout + gb * 64) / 4;
        }
      }
      dma16(src, lds0 + SCB + (uint32_t)(b * SC_BYTES + (gbl * BN + j * 64) * 16));
    }
  };

  // ---- prologue: records, weights, the first tile's window and shortcut ---
  if constexpr (SW) {
    for (int q = wave; q < BM / 64; q += NW) {
      const int c = co0 + q * 64 + lane;
      dma16(c < a.cout ? reinterpret_cast<const uint8_t*>(a.thr + (int64_t)c * 4) : zero_src,
            lds0 + TBL + q * 1024);
    }
  } else {
    for (int q = wave; q < BM / 16; q += NW) {   // 16 channels x 64 B per chunk
      const int c = co0 + q * 16 + (lane >> 2);
      dma16(c < a.cout ? reinterpret_cast<const uint8_t*>(a.table + (int64_t)c * 16 + (lane & 3) * 4)
                       : zero_src,
            lds0 + TBL + q * 1024);
    }
  }
  {
    // weight chunk c = (kk*RB + rb)*KH + t of K64 step kk = g*9 + tap
    const int nrb = a.cout_pad >> 5;
    const int rbw = co0 >> 5;
    const uint8_t* wbase = reinterpret_cast<const uint8_t*>(a.wgt);
    const uint32_t voff = (uint32_t)lane * 16;
    const int nch = G * kWpTaps * RB * KH;
    for (int c = wave; c < nch; c += NW) {
      const int t = c % KH, rb = (c / KH) % RB, kk = c / (KH * RB);
      const int64_t off =
          rbw + rb < nrb ? ((int64_t)(rbw + rb) * (KH * a.nk) + KH * kk + t) * 1024 : a.wzero;
      dma16s(wbase + off, voff, lds0 + WGT + (uint32_t)(c * 1024));
    }
  }
  if (t_begin < t_end) {
    load_window(t_begin, 0);
    if constexpr (!SW) load_shortcut(t_begin, 0);
  }
  // zero cell after every block window (the second window's, for the
  // identity join, once its raw records are staged)
  for (int g = tid; g < G * (SW ? 2 : 1); g += 64 * NW) {
    const int b = g / G, gg = g - b * G;
    *reinterpret_cast<uint4*>(lds + WIN + b * WINB + gg * wstr + wcells * 16) = uint4{0, 0, 0, 0};
  }
  wait_vmcnt<0>();
  __syncthreads();
  if constexpr (!SW) {
    stage_idj_pk(reinterpret_cast<const int32_t*>(lds + TBL), lds + EPI, BM,
                 a.cout - co0 < BM ? a.cout - co0 : BM);
    __syncthreads();
    // ordered before the second window's first read by the first tile's
    // barrier
    for (int g = tid; g < G; g += 64 * NW)
      *reinterpret_cast<uint4*>(lds + WIN + WINB + g * wstr + wcells * 16) = uint4{0, 0, 0, 0};
  }

  struct Frag {
    v4i af[KH][FM];
    v2i braw[FN];
  };
  // Tile i (buffer b = i & 1): issue the next tile's window and shortcut
  // into buffer b ^ 1 (last read by tile i - 1, before its barrier), run the
  // main loop on window b, the epilogue into output tile b, wait for this
  // wave's loads, barrier, then write output tile b to HBM (output tile b is
  // next written by tile i + 2, after tile i + 1's barrier).
  int b = 0;
  for (int tile = t_begin; tile < t_end; ++tile, b ^= 1) {
    const int p0 = tile * bn;
    if (tile + 1 < t_end) {
      load_window(tile + 1, b ^ 1);
      if constexpr (!SW) load_shortcut(tile + 1, b ^ 1);
    }
    // ---- per-lane LDS offsets of the nine taps of each pixel block -------
    int boff[FN][kWpTaps];
    {
      WpTile tl;
      tl.init(a, p0, bn);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        const int pl = (wn * FN + fn) * 32 + l32;
        const int p = p0 + pl;
        const bool pok = pl < bn && p < a.m;
        int my_off = 0, my_iya = 0, oy = 0, ox = 0;
        if (pok) {
          const int n = fdiv(p, a.div_howo);
          const int rem = p - n * howo;
          oy = fdiv(rem, a.div_wo);
          ox = rem - oy * Wo;
          int off = 0;
          for (int i = 0; i < tl.nseg; ++i) {
            int iya;
            const int rows = tl.rows(a, i, iya);
            if (i == n - tl.n_first) {
              my_off = off;
              my_iya = iya;
            }
            off += wp_round64(rows * W);
          }
        }
#pragma unroll
        for (int r = 0; r < 3; ++r)
#pragma unroll
          for (int s = 0; s < 3; ++s) {
            const int iy = oy * st - 1 + r;
            const int ix = ox * st - 1 + s;
            const bool ok = pok && (unsigned)iy < (unsigned)H && (unsigned)ix < (unsigned)W;
            boff[fn][r * 3 + s] =
                (ok ? (my_off + (iy - my_iya) * W + ix) * 16 : wcells * 16) + 8 * h;
          }
      }
    }

    // ---- main loop: every tap of every channel block, operands in LDS ----
    v16i acc[FM][FN];
    v16f accf[F4 ? FM : 1][F4 ? FN : 1];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = v16i{0};
#pragma unroll
    for (int fm = 0; fm < (F4 ? FM : 1); ++fm)
#pragma unroll
      for (int fn = 0; fn < (F4 ? FN : 1); ++fn) accf[fm][fn] = v16f{0.0f};
    const uint8_t* winb = lds + WIN + b * WINB;
    auto read_frags = [&](int g, int tap, Frag& F) {
      const uint8_t* as = lds + WGT + (g * kWpTaps + tap) * RB * KH * 1024;
      const uint8_t* win = winb + g * wstr;
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int t = 0; t < KH; ++t)
          F.af[t][fm] = *reinterpret_cast<const v4i*>(as + (fm * KH + t) * 1024 + lane * 16);
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        F.braw[fn] = *reinterpret_cast<const v2i*>(win + boff[fn][tap]);
    };
    // B operands: int8 bytes of the 2-bit codes per K32 half and pixel
    // block, or the codes as fp4 nibbles (the order of the fp4 weight blob)
    struct Unp {
      v4i b4[F4 ? 1 : 2][FN];
      v8i b8[F4 ? FN : 1];
    };
    constexpr int kGroups = KH * FN;   // MFMA groups of a tap: one B operand, FM MFMAs
    // piece k of the unpack: group k's B operand
    auto unpack_piece = [&](const Frag& F, Unp& U, int k) {
      const int t = k / FN, fn = k % FN;
      if constexpr (F4) {
        const uint32_t w0 = (uint32_t)F.braw[fn][0], w1 = (uint32_t)F.braw[fn][1];
        U.b8[fn] = v8i{(int)(w0 & 0x33333333u), (int)((w0 >> 2) & 0x33333333u),
                       (int)(w1 & 0x33333333u), (int)((w1 >> 2) & 0x33333333u), 0, 0, 0, 0};
      } else {
        U.b4[t][fn] = unpack2((uint32_t)F.braw[fn][t]);
      }
    };
    auto mfma_group = [&](const Frag& F, const Unp& U, int k) {
      const int t = k / FN, fn = k % FN;
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) {
        if constexpr (F4) {
          const v4i w = F.af[0][fm];
          const v8i af = v8i{w.x, w.y, w.z, w.w, 0, 0, 0, 0};
          if constexpr (SW)
            accf[fm][fn] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                U.b8[fn], af, accf[fm][fn], 4, 4, 0, 127, 0, 127);
          else
            accf[fm][fn] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                af, U.b8[fn], accf[fm][fn], 4, 4, 0, 127, 0, 127);
        } else {
          if constexpr (SW)
            acc[fm][fn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(U.b4[t][fn], F.af[t][fm],
                                                                acc[fm][fn], 0, 0, 0);
          else
            acc[fm][fn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(F.af[t][fm], U.b4[t][fn],
                                                                acc[fm][fn], 0, 0, 0);
        }
      }
    };
    // Software pipeline over the taps: during tap i's MFMA groups the
    // fragments of tap i + 1 arrive from LDS and their B operands are
    // unpacked, one piece after each group from the second on, so the VALU
    // work runs while the MFMAs queued before it execute. Scheduling
    // barriers keep that order (the scheduler would otherwise sink each read
    // and unpack to its first use and expose the LDS latency).
    // MFMA phases run at raised wave priority: where the other workgroup on
    // the CU is in its epilogue, its VALU work fills the issue slots this
    // loop leaves and the two drift into complementary phases.
    __builtin_amdgcn_s_setprio(1);
    for (int g = 0; g < G; ++g) {
      Frag f[2];
      Unp u[2];
      read_frags(g, 0, f[0]);
#pragma unroll
      for (int k = 0; k < kGroups; ++k) unpack_piece(f[0], u[0], k);
#pragma unroll
      for (int tap = 0; tap < kWpTaps; ++tap) {
        const int c = tap & 1;
        const bool nxt = tap + 1 < kWpTaps;
        if (nxt) read_frags(g, tap + 1, f[c ^ 1]);
#pragma unroll
        for (int k = 0; k < kGroups; ++k) {
          __builtin_amdgcn_sched_barrier(0);
          mfma_group(f[c], u[c], k);
          __builtin_amdgcn_sched_barrier(0);
          if (nxt && k >= 1) unpack_piece(f[c ^ 1], u[c ^ 1], k - 1);
        }
        if (nxt) unpack_piece(f[c ^ 1], u[c ^ 1], kGroups - 1);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    __builtin_amdgcn_s_setprio(0);
    if constexpr (F4) {
      // exact integers (every partial sum is an integer below 2^24)
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn)
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[fm][fn][i] = (int)accf[fm][fn][i];
    }

    // ---- epilogue into output tile b --------------------------------------
    uint8_t* otile = lds + OTL + b * OUT_BYTES;
#pragma unroll
    for (int q = 0; q < FM * FN; ++q) {
      const int fm = q / FN, fn = q % FN;
      const int pcb = wn * FN + fn;
      const v16i one[1] = {acc[fm][fn]};
      if constexpr (SW) {
        if (a.acc_dump) dump_acc_t<1>(a, one, fm, h, l32, co0, p0, pcb * 32, bn, a.acc_dump);
        epilogue_thr_pk_t<1>(a, reinterpret_cast<const int4*>(lds + TBL), one, fm, h, l32, co0,
                             pcb * 32, otile, orow);
      } else {
        if (a.acc_dump) {
          const v16i one2[1][1] = {{acc[fm][fn]}};
          epilogue32<kE32I32, 1, 1>(a, lds + EPI, one2, fm, pcb, h, l32, co0, p0, bn, otile,
                                    orow, a.acc_dump);
        }
        const int pl = pcb * 32 + l32;
        const int cl = fm * 32;
        const uint2 sc[1] = {*reinterpret_cast<const uint2*>(
            lds + SCB + b * SC_BYTES + (((cl >> 6) * BN + pl) * 16) + ((cl & 63) >> 2))};
        epilogue_idj_pk<1>(a, lds + EPI, one, sc, fm, h, co0, pl, otile, orow);
      }
    }
    wait_vmcnt<0>();
    __syncthreads();
    copy_out_tile(a, otile, orow, co0, BM, p0, a.m - p0 < bn ? a.m - p0 : bn);
  }
}

// ---------------------------------------------------------------------------
// Wave-independent persistent 3x3 kernel
// ---------------------------------------------------------------------------
// The same contraction and epilogues, but the prologue brings everything
// the workgroup will read into LDS at once (the slice's weights and records,
// the input window of the workgroup's whole pixel range and, for the
// identity join, that range's shortcut cells), and after its barrier every
// wave runs its own pixels with no further barrier or wait: per unit the
// main loop, the epilogue into the wave's own output tile and the stores.
// Nothing ties one wave's phases to another's, so while one wave of a SIMD
// is in its epilogue (VALU) the other's MFMAs keep the matrix core busy,
// where the workgroup-wide barrier of conv_wp holds the two workgroups of a
// CU in step. One workgroup of eight waves per CU.
//
// Work is split in half units of 32 output pixels: a workgroup takes a
// contiguous range of them and each wave a contiguous eighth of that, run
// as units of 64 pixels x the 64-channel slice and, where its count is odd,
// one last unit of 32 pixels (half the MFMAs). So the two waves of a SIMD
// carry nearly the same work and neither runs long alone.
// FMT row blocks of 32 channels per workgroup: 2 (conv_wv, a 64-channel
// slice) or 1 (conv_wvh, half of one 64-channel cell of the output, for
// layers whose 64-channel slice of weights does not fit the slab).
template <int MODE, bool F4, int WGTB, int WINB, int FMT>
__device__ __forceinline__ void conv_wv_body(const ConvLaunch& a) {
  constexpr bool SW = MODE == 0;                 // transposed sums
  constexpr int NW = 8, FM = FMT, FN = 2;
  constexpr int BM = 32 * FM, UN = 64, HU = 32;  // unit: BM channels x 64 pixels
  constexpr int KH = F4 ? 1 : 2;
  constexpr int RB = FM;
  static_assert(WGTB % 1024 == 0, "weight chunks");
  // int8 instances for one channel block (K = 576, WGTB = 36 KB): the code
  // operand keeps each 2-bit field in place within its byte (1, 4, 16 or,
  // shifted down once, 16 times the code) and the weight bytes that meet
  // fields 0 and 1 are scaled by 16 and 4 in LDS, so every product is
  // 16 * w * x: the sums are 16 a, |16 a| <= 16 * 3 * 576 < 2^15, compared
  // against 16 T.
  constexpr bool SC16 = !F4 && WGTB == 36864;
  // LDS: the slice's weights, the records (raw for the threshold epilogue,
  // packed for the identity join), one output tile per wave (the identity
  // join's raw records sit there until they are packed), the workgroup's
  // window (per channel block its cells and a zero cell) and shortcut cells.
  constexpr int WGT = 0;
  constexpr int TBL = WGTB;
  // (threshold records: one 64-lane load, 1 KB, whatever BM)
  constexpr int TBL_BYTES = SW ? (BM * 16 > 1024 ? BM * 16 : 1024) : (BM / 4) * kIdjGroupBytes;
  constexpr int OUT = TBL + TBL_BYTES;
  constexpr int OUT_BYTES = UN * BM / 4;
  static_assert(SW || NW * OUT_BYTES >= BM * 64, "raw join records in the output tiles");
  constexpr int WIN = OUT + NW * OUT_BYTES;
  constexpr int SCO = WIN + WINB;
  constexpr int LDS_BYTES = 160 * 1024;
  constexpr int SCB = LDS_BYTES - SCO;
  static_assert(SCO <= LDS_BYTES && (SW || SCB >= 1024), "LDS");
  static_assert(WINB % 1024 == 0, "window bytes");

  __shared__ __attribute__((aligned(1024))) uint8_t lds[LDS_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int h = lane >> 5;
  const int l32 = lane & 31;
  const int co0 = blockIdx.y * BM;
  const int G = a.cin >> 6;
  const int H = a.h, W = a.w, Wo = a.wo, st = a.stride;
  const int howo = a.ho * a.wo;
  const int HW = H * W;
  const int wcells = a.wcells;
  const int wstr = (wcells + 1) * 16;            // block window + its zero cell
  // this workgroup's half units, then this wave's contiguous share
  const int nhu = (a.m + HU - 1) / HU;
  const int g_lo = (int)((int64_t)blockIdx.x * nhu / gridDim.x);
  const int g_hi = (int)((int64_t)(blockIdx.x + 1) * nhu / gridDim.x);
  const int w_lo = g_lo + (g_hi - g_lo) * wave / NW;
  const int w_hi = g_lo + (g_hi - g_lo) * (wave + 1) / NW;
  const int P0 = g_lo * HU;
  const int P1 = g_hi * HU < a.m ? g_hi * HU : a.m;
  const uint32_t lds0 = lds_addr(lds);
  uint8_t* const otile = lds + OUT + wave * OUT_BYTES;
  const uint8_t* zero_src = reinterpret_cast<const uint8_t*>(&g_zero_cell);
  constexpr int orow = BM / 4;
  // half units of the unit starting at half unit c: two, or the last one
  auto unit_len = [&](int c) { return c + 2 <= w_hi ? 2 : 1; };

  // the workgroup's input window: segment i's rows of cells (each image the
  // range touches), rounded up to 64 cells, per channel block; chunk j of
  // the segments' chunk list by wave j % 8
  WpTile wt;
  wt.init(a, P0, P1 - P0);
  auto load_window = [&]() {
    int off = 0, jbase = 0;
    for (int i = 0; i < wt.nseg; ++i) {
      int iya;
      const int cells = wt.rows(a, i, iya) * W;
      const int nch = wp_round64(cells) >> 6;
      int j = wave - jbase;
      j += j < 0 ? ((-j + NW - 1) / NW) * NW : 0;
      for (; j < nch; j += NW) {
        const int c = j * 64 + lane;
        const int64_t src = ((int64_t)(wt.n_first + i) * G * HW + iya * W + c) * 16;
        for (int g = 0; g < G; ++g)
          dma16(c < cells ? a.x + src + (int64_t)g * HW * 16 : zero_src,
                lds0 + WIN + (uint32_t)(g * wstr + (off + j * 64) * 16));
      }
      jbase += nch;
      off += wp_round64(cells);
    }
  };
  // the shortcut cells of the workgroup's pixels (identity join), 64 a chunk
  auto load_shortcut = [&]() {
    const uint8_t* sc8 = reinterpret_cast<const uint8_t*>(a.shortcut);
    for (int q = wave; q * 64 < P1 - P0; q += NW) {
      const int p = P0 + q * 64 + lane;
      const uint8_t* src = zero_src;
      if (p < P1) {
        if (a.sc_layout == IFQ_LAYOUT_U2_BLOCK64) {
          const int nimg = fdiv(p, a.div_howo);
          src = sc8 + (((int64_t)nimg * (a.cout >> 6) + (co0 >> 6)) * howo + (p - nimg * howo)) * 16;
        } else {
          src = sc8 + ((int64_t)p * a.cout + (co0 & ~63)) / 4;
        }
      }
      dma16(src, lds0 + SCO + (uint32_t)(q * 1024));
    }
  };
  // this wave's output tile (npx pixels from p0) to HBM: lane = pixel, BM / 4
  // bytes (of a 64-channel cell: from byte (co0 % 64) / 4)
  auto store_unit = [&](int p0, int npx) {
    const int p = p0 + lane;
    using Row = std::conditional_t<BM == 64, uint4, uint2>;
    const Row v = *reinterpret_cast<const Row*>(otile + lane * orow);
    if (lane < npx && p < a.m) {
      uint8_t* y8 = reinterpret_cast<uint8_t*>(a.y);
      int64_t off;
      if (a.out_layout == IFQ_LAYOUT_U2_BLOCK64) {
        const int nimg = fdiv(p, a.div_howo);
        off = (((int64_t)nimg * (a.cout >> 6) + (co0 >> 6)) * howo + (p - nimg * howo)) * 16 +
              ((co0 & 63) >> 2);
      } else {
        off = ((int64_t)p * a.cout + co0) / 4;
      }
      *reinterpret_cast<Row*>(y8 + off) = v;
    }
  };

  // ---- prologue: records, weights, the window and shortcut cells ---------
  if constexpr (SW) {
    if (wave == 0) {
      const int c = co0 + lane;
      dma16(c < a.cout ? reinterpret_cast<const uint8_t*>(a.thr + (int64_t)c * 4) : zero_src,
            lds0 + TBL);
    }
  } else {
    for (int q = wave; q < BM / 16; q += NW) {   // 16 channels x 64 B per chunk
      const int c = co0 + q * 16 + (lane >> 2);
      dma16(c < a.cout ? reinterpret_cast<const uint8_t*>(a.table + (int64_t)c * 16 + (lane & 3) * 4)
                       : zero_src,
            lds0 + OUT + q * 1024);
    }
  }
  const int nwch = G * kWpTaps * RB * KH;        // 1 KB weight chunks
  {
    const int nrb = a.cout_pad >> 5;
    const int rbw = co0 >> 5;
    const uint8_t* wbase = reinterpret_cast<const uint8_t*>(a.wgt);
    const uint32_t voff = (uint32_t)lane * 16;
    for (int c = wave; c < nwch; c += NW) {
      const int t = c % KH, rb = (c / KH) % RB, kk = c / (KH * RB);
      const int64_t off =
          rbw + rb < nrb ? ((int64_t)(rbw + rb) * (KH * a.nk) + KH * kk + t) * 1024 : a.wzero;
      dma16s(wbase + off, voff, lds0 + WGT + (uint32_t)(c * 1024));
    }
  }
  if (P0 < P1) {
    load_window();
    if constexpr (!SW) load_shortcut();
  }
  // the zero cell after every block window
  if (tid < G) *reinterpret_cast<uint4*>(lds + WIN + tid * wstr + wcells * 16) = uint4{0, 0, 0, 0};
  wait_vmcnt<0>();
  __syncthreads();
  if constexpr (!SW) {
    stage_idj_pk(reinterpret_cast<const int32_t*>(lds + OUT), lds + TBL, BM,
                 a.cout - co0 < BM ? a.cout - co0 : BM, SC16 ? 4 : 0, 27 * a.cin);
    __syncthreads();
  }
  if constexpr (SC16) {
    // dwords 0 and 1 of every lane's 16 weight bytes of a K32 step meet
    // fields 0 and 1: x16 and x4 (bytes are 0 or +-1); all reads issued
    // before the writes
    const int nq = nwch * 64;
    for (int q0 = 0; q0 < nq; q0 += 4 * 64 * NW) {
      uint2 v[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = q0 + i * 64 * NW + tid;
        if (q < nq) v[i] = *reinterpret_cast<const uint2*>(lds + WGT + q * 16);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int q = q0 + i * 64 * NW + tid;
        if (q < nq)
          *reinterpret_cast<uint2*>(lds + WGT + q * 16) =
              uint2{(v[i].x << 4) & 0xF0F0F0F0u, (v[i].y << 2) & 0xFCFCFCFCu};
      }
    }
    __syncthreads();
  }

  // the threshold epilogue's packed thresholds of the lane's channel in each
  // row block: the same for every unit, so taken once
  ThrPk thp[SW ? FM : 1];
  if constexpr (SW) {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
      thp[fm] = thr_pk_of<SC16 ? 4 : 0>(reinterpret_cast<const int4*>(lds + TBL)[fm * 32 + l32],
                                        27 * a.cin);
  }

  struct Unp {
    v4i b4[F4 ? 1 : 2][FN];
    v8i b8[F4 ? FN : 1];
  };

  // ---- one unit: NB pixel blocks of 32 from p0 ----------------------------
  auto run_unit = [&](auto nb_tag, int p0) {
    constexpr int NB = decltype(nb_tag)::value;
    constexpr int kGroups = KH * NB;             // MFMA groups of a tap
    // per-lane LDS offsets of the nine taps of each pixel block: the
    // top-left tap's offset plus row and column steps; taps outside the
    // image, and pixels past the last, read the zero cell
    int boff[NB][kWpTaps];
    {
      const int zc = wcells * 16 + 8 * h;
#pragma unroll
      for (int fn = 0; fn < NB; ++fn) {
        const int p = p0 + fn * 32 + l32;
        const bool pok = p < a.m;
        const int pc = pok ? p : p0;
        const int n = fdiv(pc, a.div_howo);
        const int rem = pc - n * howo;
        const int oy = fdiv(rem, a.div_wo);
        const int ox = rem - oy * Wo;
        int my_off = 0, my_iya = 0, off = 0;
        for (int i = 0; i < wt.nseg; ++i) {
          int iya;
          const int rows = wt.rows(a, i, iya);
          if (i == n - wt.n_first) {
            my_off = off;
            my_iya = iya;
          }
          off += wp_round64(rows * W);
        }
        const int iy0 = oy * st - 1, ix0 = ox * st - 1;
        const int base = (my_off + (iy0 - my_iya) * W + ix0) * 16 + 8 * h;
        const bool rok[3] = {pok && iy0 >= 0, pok, pok && iy0 + 2 < H};
        const bool cok[3] = {ix0 >= 0, true, ix0 + 2 < W};
#pragma unroll
        for (int r = 0; r < 3; ++r)
#pragma unroll
          for (int s2 = 0; s2 < 3; ++s2)
            boff[fn][r * 3 + s2] = rok[r] && cok[s2] ? base + (r * W + s2) * 16 : zc;
      }
    }

    // main loop: written first by the zero-addend MFMAs of the first tap
    v16i acc[FM][NB];
    v16f accf[F4 ? FM : 1][F4 ? NB : 1];
    const uint8_t* winb = lds + WIN;
    // weight fragments of a tap (K32 halves x channel blocks) and the raw
    // codes of its pixel blocks
    auto read_a = [&](int g, int tap, v4i (&af)[KH][FM]) {
      const uint8_t* as = lds + WGT + (g * kWpTaps + tap) * RB * KH * 1024;
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int t = 0; t < KH; ++t)
          af[t][fm] = *reinterpret_cast<const v4i*>(as + (fm * KH + t) * 1024 + lane * 16);
    };
    auto read_b = [&](int g, int tap, v2i (&br)[NB]) {
      const uint8_t* win = winb + g * wstr;
#pragma unroll
      for (int fn = 0; fn < NB; ++fn)
        br[fn] = *reinterpret_cast<const v2i*>(win + boff[fn][tap]);
    };
    auto unpack_piece = [&](const v2i (&br)[NB], Unp& U, int k) {
      const int t = k / NB, fn = k % NB;
      if constexpr (F4) {
        const uint32_t w0 = (uint32_t)br[fn][0], w1 = (uint32_t)br[fn][1];
        U.b8[fn] = v8i{(int)(w0 & 0x33333333u), (int)((w0 >> 2) & 0x33333333u),
                       (int)(w1 & 0x33333333u), (int)((w1 >> 2) & 0x33333333u), 0, 0, 0, 0};
      } else if constexpr (SC16) {
        const uint32_t w = (uint32_t)br[fn][t];
        U.b4[t][fn] = v4i{(int)(w & 0x03030303u), (int)(w & 0x0C0C0C0Cu), (int)(w & 0x30303030u),
                          (int)((w >> 2) & 0x30303030u)};
      } else {
        U.b4[t][fn] = unpack2((uint32_t)br[fn][t]);
      }
    };
    // zc: the first MFMA into each accumulator (zero addend, no clearing)
    auto mfma_group = [&](auto zc, const v4i (&afr)[KH][FM], const Unp& U, int k) {
      constexpr bool ZC = decltype(zc)::value;
      const int t = k / NB, fn = k % NB;
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) {
        if constexpr (F4) {
          const v4i w = afr[0][fm];
          const v8i af = v8i{w.x, w.y, w.z, w.w, 0, 0, 0, 0};
          const v16f cf = ZC ? v16f{0.0f} : accf[fm][fn];
          if constexpr (SW)
            accf[fm][fn] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                U.b8[fn], af, cf, 4, 4, 0, 127, 0, 127);
          else
            accf[fm][fn] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                af, U.b8[fn], cf, 4, 4, 0, 127, 0, 127);
        } else {
          const v16i ci = ZC && t == 0 ? v16i{0} : acc[fm][fn];
          if constexpr (SW)
            acc[fm][fn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(U.b4[t][fn], afr[t][fm], ci, 0,
                                                                0, 0);
          else
            acc[fm][fn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(afr[t][fm], U.b4[t][fn], ci, 0,
                                                                0, 0);
        }
      }
    };
    // Software pipeline over the taps, two deep for the codes: during tap
    // i's MFMA groups the weight fragments of tap i + 1 and the raw codes of
    // tap i + 2 are read, and tap i + 1's B operands are unpacked from codes
    // read a whole tap earlier, one piece after each MFMA group from the
    // second on (the compiler's own schedule of this order measured a few
    // percent faster than one pinned with scheduling barriers).
    // Operand registers rotate through rings of three (weights, raw codes,
    // unpacked codes): an LDS read or an unpack never writes a register that
    // one of the last few MFMAs still reads, which would hold the write (and
    // the wave) until that MFMA has taken its operands. The empty asm at the
    // end of a tap keeps the tap's operands live to there, so the compiler
    // cannot hand their registers to the next tap's reads and unpacks; those
    // of the previous tap too, whose last MFMAs may still be reading them.
    auto run_block = [&](auto zc, int g) {
      v4i af[3][KH][FM];
      v2i br[3][NB];
      Unp uu[3];
      read_b(g, 0, br[0]);
      read_a(g, 0, af[0]);
      read_b(g, 1, br[1]);
#pragma unroll
      for (int k = 0; k < kGroups; ++k) unpack_piece(br[0], uu[0], k);
#pragma unroll
      for (int tap = 0; tap < kWpTaps; ++tap) {
        const int c = tap % 3, n1 = (tap + 1) % 3;
        const bool nxt = tap + 1 < kWpTaps;
        if (nxt) read_a(g, tap + 1, af[n1]);
        if (tap + 2 < kWpTaps) read_b(g, tap + 2, br[(tap + 2) % 3]);
#pragma unroll
        for (int k = 0; k < kGroups; ++k) {
          if (tap == 0)
            mfma_group(zc, af[c], uu[c], k);
          else
            mfma_group(std::false_type{}, af[c], uu[c], k);
          if (nxt && k >= 1) unpack_piece(br[n1], uu[n1], k - 1);
        }
        if (nxt) unpack_piece(br[n1], uu[n1], kGroups - 1);
        // this tap's operands and the previous tap's stay live to here
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          if (e == 1 && tap == 0) break;
          const int q = (tap + 3 - e) % 3;
#pragma unroll
          for (int t = 0; t < KH; ++t)
#pragma unroll
            for (int fm = 0; fm < FM; ++fm) asm volatile("" ::"v"(af[q][t][fm]));
#pragma unroll
          for (int fn = 0; fn < NB; ++fn) {
            if constexpr (F4) {
#pragma unroll
              for (int i = 0; i < 4; ++i) asm volatile("" ::"v"(uu[q].b8[fn][i]));
            } else {
#pragma unroll
              for (int t = 0; t < KH; ++t) asm volatile("" ::"v"(uu[q].b4[t][fn]));
            }
          }
        }
      }
    };
    __builtin_amdgcn_s_setprio(1);
    run_block(std::true_type{}, 0);
    for (int g = 1; g < G; ++g) run_block(std::false_type{}, g);
    __builtin_amdgcn_s_setprio(0);
    if constexpr (F4) {
      // exact integers (every partial sum is an integer below 2^24)
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int fn = 0; fn < NB; ++fn)
#pragma unroll
          for (int i = 0; i < 16; ++i) acc[fm][fn][i] = (int)accf[fm][fn][i];
    }

    // epilogue into this wave's output tile: the int32 sums first where asked
    // for, then the codes of all blocks with no branch between them (c_out is
    // a multiple of 64), so their independent dependency chains interleave
    if (a.acc_dump) {
#pragma unroll
      for (int q = 0; q < FM * NB; ++q) {
        const int fm = q / NB, fn = q % NB;
        if constexpr (SW) {
          const v16i sums[1] = {SC16 ? acc[fm][fn] >> 4 : acc[fm][fn]};
          dump_acc_t<1>(a, sums, fm, h, l32, co0, p0, fn * 32, NB * 32, a.acc_dump);
        } else {
          const v16i one2[1][1] = {{SC16 ? acc[fm][fn] >> 4 : acc[fm][fn]}};
          epilogue32<kE32I32, 1, 1>(a, lds + TBL, one2, fm, fn, h, l32, co0, p0, NB * 32, otile,
                                    orow, a.acc_dump);
        }
      }
    }
#pragma unroll
    for (int q = 0; q < FM * NB; ++q) {
      const int fm = q / NB, fn = q % NB;
      const v16i one[1] = {acc[fm][fn]};
      if constexpr (SW) {
        epilogue_thr_pk_block(one[0], thp[fm], h, l32, fm * 32 + l32, fn * 32, otile, orow);
      } else {
        const int pl = fn * 32 + l32;
        const int cl = fm * 32;
        const uint2 sc[1] = {*reinterpret_cast<const uint2*>(
            lds + SCO + (p0 - P0 + pl) * 16 + ((co0 & 63) >> 2) + (cl >> 2))};
        epilogue_idj_pk<1, false>(a, lds + TBL, one, sc, fm, h, co0, pl, otile, orow);
      }
    }
    // the output tile's bytes (written by other lanes of this wave) are read
    // back by store_unit: LDS operations of one wave complete in order; the
    // empty asm keeps the compiler from moving the reads above the writes
    asm volatile("" ::: "memory");
  };

  for (int c = w_lo; c < w_hi;) {
    const int len = unit_len(c);
    if (len == 2)
      run_unit(std::integral_constant<int, 2>{}, c * HU);
    else
      run_unit(std::integral_constant<int, 1>{}, c * HU);
    store_unit(c * HU, len * HU);
    c += len;
  }
}

template <int MODE, bool F4, int WGTB, int WINB>
__global__ __launch_bounds__(512, 1) void conv_wv(ConvLaunch a) {
  conv_wv_body<MODE, F4, WGTB, WINB, 2>(a);
}

template <int MODE, bool F4, int WGTB, int WINB>
__global__ __launch_bounds__(512, 1) void conv_wvh(ConvLaunch a) {
  conv_wv_body<MODE, F4, WGTB, WINB, 1>(a);
}

// ---------------------------------------------------------------------------
// Variants and planning
// ---------------------------------------------------------------------------
struct WpVariant {
  int wn, fm, fn, occ, wgtb, winb_thr, winb_idj;
  bool f4;
  double c_tile_us;    // fixed cost of a tile (window and tap offsets, epilogue, copy-out)
  double c_blk_us;     // a tile's main loop per 64-channel input block
  const char* thr_name;
  const char* idj_name;
};
// Fitted to kernel times measured on MI355X (the ResNet-18-shaped stack's
// 64-channel layers and VGG-16's conv1_2, int8 and fp4, and the ResNet
// 128-channel layers on fp4), with two workgroups on every busy CU: a fixed
// cost per workgroup (prologue, launch ramp), then per tile the variant's
// fixed and per-channel-block costs, more for the identity join's table
// epilogue.
constexpr double kWpWgUs = 1.27;
constexpr double kWpIdjUs = 1.1;

#define IFQ_WP_NAME(wn, fm, fn, mode, f4, occ, wgtb, winb) \
  "conv_wp<" #wn ", " #fm ", " #fn ", " #mode ", " #f4 ", " #occ ", " #wgtb ", " #winb ">"

// Index order must match the switch in launch_conv_wp.
const WpVariant kWpVariants[] = {
    {4, 2, 2, 2, 36864, 16384, 10240, false, 2.91, 2.34,
     IFQ_WP_NAME(4, 2, 2, 0, false, 2, 36864, 16384),
     IFQ_WP_NAME(4, 2, 2, 1, false, 2, 36864, 10240)},
    {4, 2, 2, 2, 36864, 16384, 10240, true, 3.34, 1.17,
     IFQ_WP_NAME(4, 2, 2, 0, true, 2, 36864, 16384),
     IFQ_WP_NAME(4, 2, 2, 1, true, 2, 36864, 10240)},
};
constexpr int kNumWpBlock = sizeof(kWpVariants) / sizeof(kWpVariants[0]);

// The wave-independent kernel: one workgroup of eight waves per CU, a unit
// of 64 pixels x 64 channels per wave at a time. Fitted the same way (the
// ResNet-18-shaped stack's 64- to 256-channel layers, VGG-16's and
// Tiny-YOLOv2's, small batches, int8 and fp4): a prologue (weights,
// records, the workgroup's window) and, per unit, a fixed and a
// per-channel-block cost, with two waves sharing each SIMD.
struct WvVariant {
  bool f4;
  int fm;                   // row blocks of 32 channels per workgroup (2: conv_wv, 1: conv_wvh)
  int wgtb;                 // weight slab bytes
  int winb_thr, winb_idj;   // window bytes of a workgroup
  double pro_us, c_unit_us, c_blk_us, idj_us;
  const char* thr_name;
  const char* idj_name;
};
#define IFQ_WV_NAME(kern, mode, f4, wgtb, winb) \
  #kern "<" #mode ", " #f4 ", " #wgtb ", " #winb ">"
// The identity join's shortcut cells take the LDS past its window: 160 KB
// less the weights, packed records (BM / 4 groups of 512 B), output tiles
// (eight of 64 pixels x BM / 4 bytes) and window.
constexpr int kWvLds = 160 * 1024;
constexpr int wv_fixed_idj(int bm) { return (bm / 4) * 512 + 8 * 64 * (bm / 4); }
// Index order must match the switch in launch_conv_wp. Weight slabs of
// 36 KB (int8: one channel block; fp4: two) or 72 KB (int8: two; fp4: four)
// for a 64-channel slice; the 32-channel instance's 72 KB slab holds four
// int8 channel blocks (c_in 256). Its window sizes fill the LDS left by its
// smaller records and output tiles; it takes stride 1 only (at stride 2 each
// of twice as many channel slices re-reads a window of the same pixels: the
// ResNet-18 l4.0.conv1 shape measured 14.3 us against 12.1 on conv_w2).
// Coefficients fitted to six measured stride-1 shapes (within about 7%).
const WvVariant kWvVariants[] = {
    {false, 2, 36864, 114688, 77824, 2.86, 0.8, 1.0, 0.4,
     IFQ_WV_NAME(conv_wv, 0, false, 36864, 114688), IFQ_WV_NAME(conv_wv, 1, false, 36864, 77824)},
    {true, 2, 36864, 114688, 77824, 2.0, 0.8, 0.62, 0.53,
     IFQ_WV_NAME(conv_wv, 0, true, 36864, 114688), IFQ_WV_NAME(conv_wv, 1, true, 36864, 77824)},
    {false, 2, 73728, 80896, 49152, 2.58, 0.45, 1.28, 0.37,
     IFQ_WV_NAME(conv_wv, 0, false, 73728, 80896), IFQ_WV_NAME(conv_wv, 1, false, 73728, 49152)},
    {true, 2, 73728, 80896, 49152, 1.73, 0.83, 0.69, 0.6,
     IFQ_WV_NAME(conv_wv, 0, true, 73728, 80896), IFQ_WV_NAME(conv_wv, 1, true, 73728, 49152)},
    {false, 1, 73728, 84992, 57344, 1.25, 0.36, 0.86, 0.37,
     IFQ_WV_NAME(conv_wvh, 0, false, 73728, 84992), IFQ_WV_NAME(conv_wvh, 1, false, 73728, 57344)},
};
constexpr int kNumWv = sizeof(kWvVariants) / sizeof(kWvVariants[0]);
constexpr int kNumWp = kNumWpBlock + kNumWv;
constexpr int kWvWaves = 8;
constexpr int kWvUnit = 64;

bool wp_fit(const ConvLaunch& a, int v, WpPlan* out) {
  const WpVariant& V = kWpVariants[v];
  if (V.f4 != (a.f4 != 0)) return false;
  const int G = a.cin / 64;
  const int bm = 32 * V.fm, bn = 32 * V.fn * V.wn;
  const int kh = V.f4 ? 1 : 2;
  if ((int64_t)G * kWpTaps * (bm / 32) * kh * 1024 > V.wgtb) return false;
  const int winb = a.join_kind == IFQ_JOIN_IDENTITY ? V.winb_idj : V.winb_thr;
  const int64_t cells = window_cells_max(a, bn, (int64_t)winb / 16 / G);
  if (cells < 0 || (int64_t)G * (cells + 1) * 16 > winb) return false;
  const int64_t nco = (a.cout + bm - 1) / bm;
  const int64_t ntm = (a.m + bn - 1) / bn;
  const int64_t slots = (int64_t)kPlanCUs * V.occ;
  const int64_t per = (nco * ntm + slots - 1) / slots;     // tiles per workgroup
  const int64_t gx = (ntm + per - 1) / per;
  const double c_tile = V.c_tile_us + G * V.c_blk_us +
                        (a.join_kind == IFQ_JOIN_IDENTITY ? kWpIdjUs : 0.0);
  const double t = kLaunchUs + kWpWgUs + (double)per * c_tile;
  *out = WpPlan{v, bn, (int)gx, (int)per, (int)cells, t};
  return true;
}

// Cells per channel block of the input window of output pixels [p0, p1)
// (each image's rows rounded up to 64 cells), as the wave kernel lays it.
int64_t wv_window_cells(const ConvLaunch& a, int64_t p0, int64_t p1) {
  const int64_t howo = (int64_t)a.ho * a.wo;
  const int64_t pend = p1 - 1;
  const int64_t nf = p0 / howo, nl = pend / howo;
  const int64_t oyf = (p0 - nf * howo) / a.wo, oyl = (pend - nl * howo) / a.wo;
  int64_t tot = 0;
  for (int64_t i = 0; i <= nl - nf; ++i) {
    const int64_t oya = i == 0 ? oyf : 0, oyb = i == nl - nf ? oyl : a.ho - 1;
    int64_t iya = oya * a.stride - 1, iyb = oyb * a.stride + 1;
    if (iya < 0) iya = 0;
    if (iyb > a.h - 1) iyb = a.h - 1;
    tot += ((iyb - iya + 1) * a.w + 63) / 64 * 64;
  }
  return tot;
}

bool wv_fit(const ConvLaunch& a, int v, WpPlan* out) {
  const WvVariant& V = kWvVariants[v];
  if (V.f4 != (a.f4 != 0) || a.cout % 64 != 0) return false;
  const int G = a.cin / 64;
  const int kh = V.f4 ? 1 : 2;
  const int bm = 32 * V.fm;
  if ((int64_t)G * kWpTaps * V.fm * kh * 1024 > V.wgtb) return false;
  // the 32-channel instance only where no 64-channel slab holds the weights
  // (it measured slower than conv_wv on the 64- and 128-channel layers)
  if (V.fm == 1 && (a.stride != 1 || (int64_t)G * kWpTaps * 2 * kh * 1024 <= 73728))
    return false;
  const bool idj = a.join_kind == IFQ_JOIN_IDENTITY;
  const int64_t winb = idj ? V.winb_idj : V.winb_thr;
  const int64_t scb = idj ? kWvLds - wv_fixed_idj(bm) - V.wgtb - winb : 0;
  const int64_t nco = a.cout / bm;
  const int64_t hu = kWvUnit / 2;
  const int64_t nhu = (a.m + hu - 1) / hu;                      // half units
  int64_t gx = kPlanCUs / nco;
  if (gx < 1) gx = 1;
  if (gx > (nhu + kWvWaves - 1) / kWvWaves) gx = (nhu + kWvWaves - 1) / kWvWaves;
  // more workgroups (in rounds) until each one's window and shortcut cells
  // fit; the window cells of the largest
  int64_t cells = -1;
  for (; gx <= nhu; gx *= 2) {
    int64_t mx = 0, px = 0;
    for (int64_t k = 0; k < gx; ++k) {
      const int64_t p0 = k * nhu / gx * hu;
      int64_t p1 = (k + 1) * nhu / gx * hu;
      if (p1 > a.m) p1 = a.m;
      const int64_t c = wv_window_cells(a, p0, p1);
      if (c > mx) mx = c;
      if (p1 - p0 > px) px = p1 - p0;
    }
    if (G * (mx + 1) * 16 <= winb && (!idj || (px + 63) / 64 * 1024 <= scb)) {
      cells = mx;
      break;
    }
  }
  if (cells < 0 || gx > nhu) return false;
  const int64_t hw = (nhu + gx - 1) / gx;                        // half units per workgroup
  const int64_t per_wave = (hw + kWvWaves - 1) / kWvWaves;
  const int64_t rounds = (gx * nco + kPlanCUs - 1) / kPlanCUs;   // one workgroup per CU
  // the two waves of a SIMD: 2 * per_wave half units between them
  const double c_hu = (V.c_unit_us + G * V.c_blk_us + (idj ? V.idj_us : 0.0)) / 2.0;
  const double t = kLaunchUs + rounds * (V.pro_us + 2 * per_wave * c_hu);
  *out = WpPlan{kNumWpBlock + v, kWvUnit, (int)gx, (int)per_wave, (int)cells, t};
  return true;
}

bool wp_mode_ok(const ConvLaunch& a) {
  if (!(a.out_mode == 2 && a.rec == 4 && (a.cout & 31) == 0 && 27 * a.cin <= 32766 &&
        a.pool_k == 0))
    return false;
  if (a.join_kind == IFQ_JOIN_NONE) return true;
  return a.join_kind == IFQ_JOIN_IDENTITY && a.cout % 64 == 0 &&
         (a.sc_layout == IFQ_LAYOUT_U2_BLOCK64 || a.sc_layout == IFQ_LAYOUT_U2_NHWC_PACKED);
}

}  // namespace

int wp_variant_count() { return kNumWp; }
bool wp_variant_fp4(int v) {
  if (v < 0 || v >= kNumWp) return false;
  return v < kNumWpBlock ? kWpVariants[v].f4 : kWvVariants[v - kNumWpBlock].f4;
}

namespace {
bool wp_any_fit(const ConvLaunch& a, int v, WpPlan* out) {
  return v < kNumWpBlock ? wp_fit(a, v, out) : wv_fit(a, v - kNumWpBlock, out);
}
}  // namespace

bool plan_wp(const ConvLaunch& a, int forced, WpPlan* out) {
  if (!(a.in_layout == IFQ_LAYOUT_U2_BLOCK64 && a.in_bits == 2 && a.cin % 64 == 0 &&
        a.kh == 3 && a.kw == 3 && a.pad == 1 && (a.stride == 1 || a.stride == 2) && a.m > 0))
    return false;
  if (!wp_mode_ok(a)) return false;
  // 32-bit cell indices and offsets
  if ((int64_t)a.n * a.h * a.w * (a.cin / 64) >= (int64_t)1 << 26) return false;
  if (forced >= 0) return forced < kNumWp && wp_any_fit(a, forced, out);
  bool found = false;
  for (int v = 0; v < kNumWp; ++v) {
    WpPlan p;
    if (wp_any_fit(a, v, &p) && (!found || p.t_us < out->t_us)) {
      *out = p;
      found = true;
    }
  }
  return found;
}

const char* conv_wp_name(const WpPlan& p, const ConvLaunch& a) {
  const bool idj = a.join_kind == IFQ_JOIN_IDENTITY;
  if (p.variant >= kNumWpBlock) {
    const WvVariant& V = kWvVariants[p.variant - kNumWpBlock];
    return idj ? V.idj_name : V.thr_name;
  }
  const WpVariant& V = kWpVariants[p.variant];
  return idj ? V.idj_name : V.thr_name;
}

hipError_t launch_conv_wp(ConvLaunch a, const WpPlan& p, hipStream_t stream) {
  a.bn = p.bn;
  a.wcells = p.wcells;
  a.tiles_wg = p.per;
  if (p.variant >= kNumWpBlock) {
    const dim3 grid(p.gx, a.cout / (32 * kWvVariants[p.variant - kNumWpBlock].fm));
    const dim3 block(64 * kWvWaves);
    const int mode = a.join_kind == IFQ_JOIN_IDENTITY ? 1 : 0;
    switch ((p.variant - kNumWpBlock) * 2 + mode) {
#define IFQ_WV_CASE(k, kern, f4, wgtb, winbt, winbi)                                       \
  case 2 * k:                                                                              \
    hipLaunchKernelGGL((kern<0, f4, wgtb, winbt>), grid, block, 0, stream, a);             \
    break;                                                                                 \
  case 2 * k + 1:                                                                          \
    hipLaunchKernelGGL((kern<1, f4, wgtb, winbi>), grid, block, 0, stream, a);             \
    break;
      IFQ_WV_CASE(0, conv_wv, false, 36864, 114688, 77824)
      IFQ_WV_CASE(1, conv_wv, true, 36864, 114688, 77824)
      IFQ_WV_CASE(2, conv_wv, false, 73728, 80896, 49152)
      IFQ_WV_CASE(3, conv_wv, true, 73728, 80896, 49152)
      IFQ_WV_CASE(4, conv_wvh, false, 73728, 84992, 57344)
#undef IFQ_WV_CASE
      default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
  }
  const WpVariant& V = kWpVariants[p.variant];
  const int bm = 32 * V.fm;
  const dim3 grid(p.gx, (a.cout + bm - 1) / bm);
  const dim3 block(64 * V.wn);
  const int mode = a.join_kind == IFQ_JOIN_IDENTITY ? 1 : 0;
  switch (p.variant * 2 + mode) {
#define IFQ_WP_CASE(k, wn, fm, fn, f4, occ, wgtb, winbt, winbi)                             \
  case 2 * k:                                                                               \
    hipLaunchKernelGGL((conv_wp<wn, fm, fn, 0, f4, occ, wgtb, winbt>), grid, block, 0,      \
                       stream, a);                                                          \
    break;                                                                                  \
  case 2 * k + 1:                                                                           \
    hipLaunchKernelGGL((conv_wp<wn, fm, fn, 1, f4, occ, wgtb, winbi>), grid, block, 0,      \
                       stream, a);                                                          \
    break;
    IFQ_WP_CASE(0, 4, 2, 2, false, 2, 36864, 16384, 10240)
    IFQ_WP_CASE(1, 4, 2, 2, true, 2, 36864, 16384, 10240)
#undef IFQ_WP_CASE
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ---- the register-blocked family ------------------------------------------
int reg3_variant_count() { return w2_variant_count() + wp_variant_count(); }

bool reg3_variant_fp4(int v) {
  return v < w2_variant_count() ? w2_variant_fp4(v) : wp_variant_fp4(v - w2_variant_count());
}

bool plan_reg3(const ConvLaunch& a, int forced, Reg3Plan* out) {
  const int n2 = w2_variant_count();
  if (forced >= 0) {
    out->persistent = forced >= n2;
    if (forced < n2) {
      if (!plan_w2(a, forced, &out->w2)) return false;
      out->t_us = out->w2.t_us;
    } else {
      if (!plan_wp(a, forced - n2, &out->wp)) return false;
      out->t_us = out->wp.t_us;
    }
    return true;
  }
  const bool w2 = plan_w2(a, -1, &out->w2);
  const bool wp = plan_wp(a, -1, &out->wp);
  if (!w2 && !wp) return false;
  out->persistent = wp && (!w2 || out->wp.t_us < out->w2.t_us);
  out->t_us = out->persistent ? out->wp.t_us : out->w2.t_us;
  return true;
}

hipError_t launch_reg3(const ConvLaunch& a, const Reg3Plan& p, hipStream_t stream) {
  return p.persistent ? launch_conv_wp(a, p.wp, stream) : launch_conv_w2(a, p.w2, stream);
}

const char* reg3_name(const Reg3Plan& p, const ConvLaunch& a) {
  return p.persistent ? conv_wp_name(p.wp, a) : conv_w2_name(p.w2, a);
}

}  // namespace ifq
