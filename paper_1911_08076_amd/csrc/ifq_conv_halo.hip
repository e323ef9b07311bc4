// Fast path of the integrated fixed-point quantized convolution for 3x3
// filters (stride 1 or 2, zero padding 1) on 2-bit codes in the BLOCK64
// layout, c_in a multiple of 64, on gfx950 (MI355X).
//
// The integer part of Eq. (1), a = W_b (x) X_q, is the implicit GEMM
// D[co][pixel] = sum_k W[co][k] * X[pixel][k] on v_mfma_i32_32x32x32_i8, as in
// ifq_conv_mfma.hip; what differs is how the operands reach the MFMA:
//
//  - Codes: a workgroup's output pixels are a run of consecutive (n, oy, ox)
//    positions. Per image the input rows they touch (plus the filter halo)
//    are one contiguous span of 16-byte cells per channel block g in the
//    BLOCK64 layout, so the whole input window of the tile for block g is
//    brought into LDS with a few 1 KB LDS-DMA chunks, once per g. The nine
//    filter taps of that block then read it at fixed per-lane LDS addresses
//    computed once per workgroup (out-of-image taps point at a zero cell), so
//    the main loop spends no VALU on code addressing or bounds.
//  - Weights stream through a ring of LDS stages, one K64 step per stage and
//    wave group, with a wave-uniform SGPR base (no per-lane address math).
//
// K order: K64 step kk = g*9 + tap (channel block outermost, the weight blob's
// order). The WK wave groups take the channel blocks g = gi*WK + kg, all at
// the same tap, so stage st = 9*gi + tap covers WK K64 steps. The window of
// block gi+1 is loaded into the second of two buffers per group while gi is
// computed: its chunks ride along with the stage loads issued in the first
// 11 - D iterations of gi, after the barrier that ends the use of that
// buffer's previous contents, and before the loads of the first stage of
// gi+1 (loads complete in issue order, so that stage's wait covers them).
// Every wave issues exactly WK + 1 loads per stage (padding with dummy loads
// into a scratch LDS area), which keeps the explicit vmcnt waits exact.
//
// Each of the 8 waves owns a 128-channel x 32-pixel tile (four 32x32
// accumulators): every unpacked code fragment feeds four MFMAs. The WK
// groups' sums are added through LDS; the fused epilogue of ifq_epilogue.h /
// ifq_mfma_common.h produces codes, joins or int32 sums.
#include <hip/hip_runtime.h>

#include "ifq_epilogue.h"
#include "ifq_internal.h"
#include "ifq_mfma_common.h"

namespace ifq {
namespace {

constexpr int kHaloNW = 8;     // waves per workgroup
constexpr int kTaps = 9;

// Cells of one halo buffer (2 buffers per wave group) for WK wave groups and
// FM 32-row blocks per wave (FM = 2: two workgroups share a CU).
__host__ __device__ constexpr int halo_cap_cells(int wk, int fm) {
  return fm == 2 ? 1024 : wk == 1 ? 2560 : wk == 2 ? 1024 : 192;
}

__host__ __device__ constexpr int round64(int v) { return (v + 63) & ~63; }

// SW: the MFMAs take the codes as A and the weights as B, so the sums come
// out transposed (one channel per lane; see the transposed epilogues of
// ifq_mfma_common.h). Those kernels serve the 2-bit threshold epilogue and
// the fused downsample join only.
// F4: the contraction on the fp4 (e2m1) scaled MFMA, 32x32x64 with unit
// scales. A code c is the nibble c, the e2m1 value c/2; a weight is +-2.0, so
// every product is +-c and every partial sum an integer far below 2^24: the
// fp32 accumulators hold the int8 kernel's sums exactly. The weight blob
// holds 32 nibbles per lane and K64 step (half the int8 bytes), and one
// MFMA covers what two int8 ones do.
template <int WN, int WK, int D, bool FUSED, int FM, bool SW, bool F4 = false>
__global__ __launch_bounds__(512, FM == 2 ? 4 : 2) void conv_halo(ConvLaunch a) {
  static_assert(WN * WK == kHaloNW, "8 waves");
  static_assert(FM == 4 || (FM == 2 && !FUSED), "fused downsample needs FM = 4");
  static_assert(!FUSED || SW, "the fused join runs on the transposed layout");
  static_assert(!F4 || FM == 4, "fp4 kernels: 128-channel tiles");
  constexpr int BM = 32 * FM, BN = 32 * WN;
  constexpr int KH = F4 ? 1 : 2;                  // 1 KB chunks per row block and K64 step
  constexpr int A_STEP = BM * 32 * KH;            // one K64 step of weights
  constexpr int STAGE = WK * A_STEP;
  // weight chunks (1 KB) per stage: KH*FM per group; wave w takes chunks
  // w + 8k, k < CPWA (dummy loads where that runs past the stage)
  constexpr int NCH = KH * FM * WK;
  constexpr int CPWA = NCH > kHaloNW ? NCH / kHaloNW : 1;
  static_assert(NCH % kHaloNW == 0 || NCH < kHaloNW, "weight chunks per wave");
  constexpr int CPW = CPWA + 1;                   // loads per wave per stage
  static_assert((D - 3) * CPW <= 63, "vmcnt range");
  static_assert(D >= 3 && D <= 10, "halo window");
  constexpr int HCAP = halo_cap_cells(WK, FM);
  constexpr int HSTRIDE = HCAP * 16 + 16;         // buffer + its zero cell
  constexpr int RING = D * STAGE;
  constexpr int HALO0 = RING;
  constexpr int DUMMY = HALO0 + 2 * WK * HSTRIDE;  // 1 KB sink of dummy loads
  constexpr int EPI_BYTES = epilogue_param_bytes(BM);
  constexpr int OUT_BYTES = BN * BM;
  constexpr int RED_BYTES = WK > 1 ? kHaloNW * FM * 4096 : 0;  // 32x32 partial blocks
  // Prefetched epilogue records, above everything the reduction and the
  // epilogue reuse: BM threshold records of 16 B, or (where LDS allows) the
  // identity-join records of BM channels (64 B each).
  constexpr int TBL_BYTES = WK <= 2 ? BM * 64 : BM * 16;
  constexpr int THR0 = DUMMY + 1024 > RED_BYTES ? DUMMY + 1024 : RED_BYTES;
  constexpr int THR = THR0 > EPI_BYTES + OUT_BYTES ? THR0 : EPI_BYTES + OUT_BYTES;
  constexpr int LDS_BYTES = THR + TBL_BYTES;
  static_assert(LDS_BYTES <= 160 * 1024, "LDS");

  __shared__ __attribute__((aligned(1024))) uint8_t lds[LDS_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = wave / WN;
  const int wn = wave - kg * WN;
  const int h = lane >> 5;
  const int l32 = lane & 31;
  const int bn = a.bn;
  const int p0 = blockIdx.x * bn;
  const int co0 = blockIdx.y * BM;
  const int G = a.cin >> 6;
  const int nG = G / WK;
  const int nst = kTaps * nG;
  const int H = a.h, W = a.w, Wo = a.wo, st = a.stride;
  const int howo = a.ho * a.wo;
  const int HW = H * W;
  const uint32_t lds0 = lds_addr(lds);

  // zero cells after every halo buffer
  if (tid < 2 * WK)
    *reinterpret_cast<uint4*>(lds + HALO0 + tid * HSTRIDE + HCAP * 16) = uint4{0, 0, 0, 0};

  // ---- the tile's images (segments) and their input row spans ----------
  const int pend = (p0 + bn < a.m ? p0 + bn : a.m) - 1;
  const int n_first = fdiv(p0, a.div_howo);
  const int n_last = fdiv(pend, a.div_howo);
  const int nseg = n_last - n_first + 1;
  const int oy_first = fdiv(p0 - n_first * howo, a.div_wo);
  const int oy_last = fdiv(pend - n_last * howo, a.div_wo);
  auto seg_rows = [&](int i, int& iya) {
    const int oya = i == 0 ? oy_first : 0;
    const int oyb = i == nseg - 1 ? oy_last : a.ho - 1;
    iya = oya * st - 1;
    iya = iya < 0 ? 0 : iya;
    int iyb = oyb * st + 1;
    iyb = iyb > H - 1 ? H - 1 : iyb;
    return iyb - iya + 1;
  };

  // ---- per-lane LDS offsets of the nine taps (relative to buffer 0 of the
  // lane's group); a tap outside the image reads the buffer's zero cell ----
  int boff[kTaps];
  {
    const int pl = wn * 32 + l32;
    const int p = p0 + pl;
    const bool pok = pl < bn && p < a.m;
    int my_off = 0, my_iya = 0, oy = 0, ox = 0;
    if (pok) {
      const int n = fdiv(p, a.div_howo);
      const int rem = p - n * howo;
      oy = fdiv(rem, a.div_wo);
      ox = rem - oy * Wo;
      int off = 0;
      for (int i = 0; i < nseg; ++i) {
        int iya;
        const int rows = seg_rows(i, iya);
        if (i == n - n_first) {
          my_off = off;
          my_iya = iya;
        }
        off += round64(rows * W);
      }
    }
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        const int iy = oy * st - 1 + r;
        const int ix = ox * st - 1 + s;
        const bool ok = pok && (unsigned)iy < (unsigned)H && (unsigned)ix < (unsigned)W;
        boff[r * 3 + s] = (ok ? (my_off + (iy - my_iya) * W + ix) * 16 : HCAP * 16) + 8 * h;
      }
  }

  // 2-bit thresholds of a 3x3 layer fit packed 16-bit compares when
  // 3 * 9 * c_in <= 32766 (sums and thresholds below 2^15 in magnitude)
  const bool pk16 = a.out_mode == 2 && a.rec == 4 && (a.cout & 31) == 0 && 27 * a.cin <= 32766;
  const bool pk = pk16 && a.join_kind == IFQ_JOIN_NONE;
  const bool pk_idj = pk16 && a.join_kind == IFQ_JOIN_IDENTITY &&
                      (a.sc_layout == IFQ_LAYOUT_U2_BLOCK64 ||
                       a.sc_layout == IFQ_LAYOUT_U2_NHWC_PACKED);
  const bool tbl_pre = pk_idj && WK <= 2;


  // ---- halo chunks: chunk j of a block's window is 64 cells of one image's
  // span; q = kg'*C_h + j enumerates the WK groups' chunks ----------------
  int C_h = 0;
  for (int i = 0; i < nseg; ++i) {
    int iya;
    C_h += round64(seg_rows(i, iya) * W) >> 6;
  }
  const int nq = WK * C_h;
  // source cell (without the channel-block term; -1: zero) and LDS
  // destination (relative to buffer 0 of group 0) of chunk q for this lane
  auto chunk = [&](int q, int& src_cell, int& dst) {
    const int kq = q / C_h;
    int j = q - kq * C_h;
    int off = 0;
    src_cell = -1;
    dst = kq * 2 * HSTRIDE;
    for (int i = 0; i < nseg; ++i) {
      int iya;
      const int cells = seg_rows(i, iya) * W;
      const int nch = round64(cells) >> 6;
      if (j >= 0 && j < nch) {
        const int c = j * 64 + lane;
        if (c < cells) src_cell = ((n_first + i) * G + kq) * HW + iya * W + c;
        dst += (off + j * 64) * 16;
      }
      j -= nch;
      off += round64(cells);
    }
  };
  const uint8_t* zero_src = reinterpret_cast<const uint8_t*>(&g_zero_cell);
  auto issue_halo = [&](int gi, int src_cell, int dst) {
    // block g = gi*WK + kq: the chunk's group term kq is already in src_cell
    const uint8_t* src =
        src_cell >= 0 ? a.x + ((int64_t)src_cell + (int64_t)gi * WK * HW) * 16 : zero_src;
    dma16(src, lds0 + HALO0 + (uint32_t)((gi & 1) * HSTRIDE + dst));
  };
  auto issue_dummy = [&]() { dma16(zero_src, lds0 + DUMMY); };

  // chunks this wave adds to the stage loads of the first NR iterations of a
  // block (see the loop below for why NR = 11 - D)
  constexpr int NR = 11 - D < kTaps ? 11 - D : kTaps;
  int hs_src[NR], hs_dst[NR];
  bool hs_real[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const int q = r * kHaloNW + wave;
    hs_real[r] = q < nq;
    hs_src[r] = -1;
    hs_dst[r] = 0;
    if (hs_real[r]) chunk(q, hs_src[r], hs_dst[r]);
  }

  // ---- weights: chunk c of a stage is group c / (2*FM)'s row block
  // (c % (2*FM)) / 2, K32 half c % 2 of its K64 step: 1 KB at
  // ((rbw + rb) * KH*nk + KH*kk + t) * 1024 (KH = 1, t = 0 for fp4) ------------
  const int nrb = a.cout_pad >> 5;
  const int rbw = co0 >> 5;
  const uint8_t* wbase = reinterpret_cast<const uint8_t*>(a.wgt);
  const uint32_t voff = (uint32_t)lane * 16;
  auto issue_a = [&](int stg, int tap) {
    const int gi = stg / kTaps;
    const uint32_t slot = lds0 + (uint32_t)((stg % D) * STAGE);
#pragma unroll
    for (int k = 0; k < CPWA; ++k) {
      const int c = wave + kHaloNW * k;
      if (NCH >= kHaloNW || c < NCH) {
        const int i = c / (KH * FM), cc = c - i * KH * FM;
        const int rb = F4 ? cc : cc >> 1, t = F4 ? 0 : cc & 1;
        const int kk = (gi * WK + i) * kTaps + tap;
        const int64_t off =
            rbw + rb < nrb ? ((int64_t)(rbw + rb) * (KH * a.nk) + KH * kk + t) * 1024 : a.wzero;
        dma16s(wbase + off, voff, slot + (uint32_t)(i * A_STEP + cc * 1024));
      } else {
        dma16(zero_src, lds0 + DUMMY);
      }
    }
  };


  // ---- fused downsample (IFQ_JOIN_CONV_FUSED): one extra stage after the
  // 3x3 stages. Its weight chunks are those of the row blocks each group
  // finishes (all Gd = d_cin/64 = WK K64 steps: 8 chunks per group, so the
  // stage has the usual WK chunks per wave); its input cells (stride d_stride
  // gather, one 16-byte cell per pixel and channel block, cell e = g*BN + pixel
  // in 1 KB chunks, one per wave) go into the halo buffers of parity nG % 2,
  // which the last block does not use. ----------------------------------------
  constexpr bool fused = FUSED;   // a.join_kind == IFQ_JOIN_CONV_FUSED
  const int Gd = fused ? a.d_cin >> 6 : 0;
  const int nst_all = nst + (fused ? 1 : 0);
  constexpr int CPB = HCAP / 64;                  // 1 KB chunks per halo buffer
  const int dpar = nG & 1;
  auto dchunk = [&](int q) {                      // LDS offset of down chunk q
    return HALO0 + ((q / CPB) * 2 + dpar) * HSTRIDE + (q % CPB) * 1024;
  };
  const uint8_t* dsrc = zero_src;                 // this wave's down chunk
  if constexpr (FUSED) {
    const int e = wave * 64 + lane;
    const int g = e / BN, pe = e - g * BN;
    const int p = p0 + pe;
    if (g < Gd && pe < bn && p < a.m) {
      const int n = fdiv(p, a.div_howo);
      const int rem = p - n * howo;
      const int oy = fdiv(rem, a.div_wo);
      const int ox = rem - oy * Wo;
      dsrc = a.dx + ((((int64_t)n * Gd + g) * a.d_h + oy * a.d_stride) * a.d_w +
                     ox * a.d_stride) * 16;
    }
  }
  const bool dreal = fused && wave * 64 < Gd * BN;
  auto issue_down = [&]() {
    const uint32_t slot = lds0 + (uint32_t)((nst % D) * STAGE);
    if constexpr (F4) {
      // fp4: FM chunks (FM/WK row blocks x Gd = WK K64 steps) per group,
      // chunk c = wave + 8k as in issue_a (the same loads per wave)
#pragma unroll
      for (int k = 0; k < CPWA; ++k) {
        const int c = wave + kHaloNW * k;
        if (NCH >= kHaloNW || c < NCH) {
          const int i = c / FM, cc = c - i * FM;
          const int j = cc / WK, g = cc - j * WK;
          const int rb = rbw + i * (FM / WK) + j;
          const int64_t off = rb < nrb ? ((int64_t)rb * WK + g) * 1024 : a.d_wzero;
          dma16s(reinterpret_cast<const uint8_t*>(a.dwgt) + off, voff,
                 slot + (uint32_t)(i * A_STEP + cc * 1024));
        } else {
          issue_dummy();
        }
      }
    } else {
      const int gd2 = fused ? 2 * Gd : 1;   // (Gd is 0 in the unfused kernels)
      const int j = wave / gd2, k32 = wave - j * gd2;
#pragma unroll
      for (int i = 0; i < WK; ++i) {
        const int rb = rbw + i * (FM / WK) + j;
        const int64_t off = rb < nrb ? ((int64_t)rb * a.d_nk32 + k32) * 1024 : a.d_wzero;
        dma16s(reinterpret_cast<const uint8_t*>(a.dwgt) + off, voff,
               slot + (uint32_t)(i * A_STEP + wave * 1024));
      }
    }
    if (dreal)
      dma16(dsrc, lds0 + (uint32_t)dchunk(wave));
    else
      issue_dummy();
  };

  // ---- prologue: the tile's threshold records (read by the epilogue, so
  // their latency hides behind the main loop), block 0's windows, then
  // stages 0 .. D-3 ---------------------------------------------------------
  if (pk && wave < BM / 64) {
    const int c = co0 + wave * 64 + lane;
    dma16(c < a.cout ? reinterpret_cast<const uint8_t*>(a.thr + (int64_t)c * 4) : zero_src,
          lds0 + THR + wave * 1024);
  }
  if (tbl_pre && wave < BM / 16) {   // 16 channels x 64 B per wave
    const int c = co0 + wave * 16 + (lane >> 2);
    dma16(c < a.cout ? reinterpret_cast<const uint8_t*>(a.table + (int64_t)c * 16 + (lane & 3) * 4)
                     : zero_src,
          lds0 + THR + wave * 1024);
  }
  for (int q = wave; q < nq; q += kHaloNW) {
    int sc, dst;
    chunk(q, sc, dst);
    issue_halo(0, sc, dst);
  }
  const int pre = nst < D - 2 ? nst : D - 2;
  for (int s_ = 0; s_ < pre; ++s_) {
    issue_a(s_, s_ % kTaps);
    issue_dummy();
  }

  v16i acc[FM];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) acc[fm] = v16i{0};
  v16f accf[F4 ? FM : 1];
#pragma unroll
  for (int fm = 0; fm < (F4 ? FM : 1); ++fm) accf[fm] = v16f{0.0f};

  // Fragments of one stage in registers: A for both K32 halves and the raw
  // 2-bit B words, unpacked only right before the MFMAs that use them (one
  // iteration later), so no instruction waits on these reads in the
  // iteration that issues them.
  struct Frag {
    v4i af[KH][FM];
    v2i braw;
  };
  auto read_frags = [&](int s_, int tap, Frag& F) {
    const uint8_t* as = lds + (s_ % D) * STAGE + kg * A_STEP;
    const int gi = s_ / kTaps;
    F.braw = *reinterpret_cast<const v2i*>(
        lds + HALO0 + kg * 2 * HSTRIDE + (gi & 1) * HSTRIDE + boff[tap]);
#pragma unroll
    for (int t = 0; t < KH; ++t)
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
        F.af[t][fm] = *reinterpret_cast<const v4i*>(as + (fm * KH + t) * 1024 + lane * 16);
  };
  auto mfmas = [&](const Frag& F) {
    if constexpr (F4) {
      // the 32 codes of the lane's half of the cell as nibbles: word 0 holds
      // codes 0, 2, .., 14 of braw.x, word 1 codes 1, 3, .., 15, words 2 and
      // 3 the same of braw.y (the weight blob follows that order)
      const uint32_t w0 = (uint32_t)F.braw[0], w1 = (uint32_t)F.braw[1];
      const v8i bf = v8i{(int)(w0 & 0x33333333u), (int)((w0 >> 2) & 0x33333333u),
                         (int)(w1 & 0x33333333u), (int)((w1 >> 2) & 0x33333333u), 0, 0, 0, 0};
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) {
        const v4i w = F.af[0][fm];
        const v8i af = v8i{w.x, w.y, w.z, w.w, 0, 0, 0, 0};
        if constexpr (SW)
          accf[fm] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(bf, af, accf[fm], 4, 4, 0,
                                                                     127, 0, 127);
        else
          accf[fm] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(af, bf, accf[fm], 4, 4, 0,
                                                                     127, 0, 127);
      }
      return;
    }
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const v4i bf = unpack2((uint32_t)F.braw[t]);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) {
        if constexpr (SW)
          acc[fm] = __builtin_amdgcn_mfma_i32_32x32x32_i8(bf, F.af[t][fm], acc[fm], 0, 0, 0);
        else
          acc[fm] = __builtin_amdgcn_mfma_i32_32x32x32_i8(F.af[t][fm], bf, acc[fm], 0, 0, 0);
      }
    }
  };

  // Iteration s_: wait until stage s_ has landed, barrier, issue stage
  // s_ + D - 2 into the slot of stage s_ - 2 (read in iteration s_ - 2 and
  // consumed by the MFMAs of iteration s_ - 1, both before this barrier),
  // read stage s_'s fragments into registers, then run the MFMAs of stage
  // s_ - 1 while those reads are in flight. The window of block gi + 1 rides
  // along with the loads issued in iterations 9*gi .. 9*gi + NR - 1: after
  // the barrier of iteration 9*gi, which ends the reads of its buffer's
  // previous block gi - 1, and before the loads of stage 9*(gi + 1), issued in
  // iteration 9*gi + 11 - D, whose wait therefore covers them.
  Frag fa, fb;   // even taps read into fa, odd taps into fb
  for (int gi = 0; gi < nG; ++gi) {
#pragma unroll
    for (int tap = 0; tap < kTaps; ++tap) {
      const int s_ = gi * kTaps + tap;
      const int after = nst_all - 1 - s_;
      wait_ahead<D - 3, CPW>(after < D - 3 ? after : D - 3);
      // A bare barrier: no LDS fence is needed here (the slot reused below
      // was read by fragments the previous iteration's MFMAs consumed, and
      // the stage's LDS-DMA data is complete by the vmcnt wait above), and
      // a fence would stall until this iteration's own fragment reads land.
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      if (s_ + D - 2 < nst) {
        issue_a(s_ + D - 2, (tap + D - 2) % kTaps);
        if (tap < NR && gi + 1 < nG && hs_real[tap < NR ? tap : 0])
          issue_halo(gi + 1, hs_src[tap < NR ? tap : 0], hs_dst[tap < NR ? tap : 0]);
        else
          issue_dummy();
      } else if constexpr (FUSED) {
        if (s_ + D - 2 == nst) issue_down();
      }
      if ((tap & 1) == 0) {
        // tap 0 follows tap 8 of the previous block, which was read into fa
        // and moved to fb at the end of that block
        read_frags(s_, tap, fa);
        if (s_ > 0) mfmas(fb);
      } else {
        read_frags(s_, tap, fb);
        mfmas(fa);
      }
    }
    // tap 8 (odd count of taps): its fragments move to fb
#pragma unroll
    for (int t = 0; t < KH; ++t)
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) fb.af[t][fm] = fa.af[t][fm];
    fb.braw = fa.braw;
  }
  mfmas(fb);
  if constexpr (F4) {
    // exact integers (see above)
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 16; ++i) acc[fm][i] = (int)accf[fm][i];
  }
  wait_vmcnt<0>();
  __syncthreads();

  // fused downsample: its sums for the row blocks this wave finishes
  constexpr int OWN = FM / WK;
  v16i accd[OWN];
#pragma unroll
  for (int j = 0; j < OWN; ++j) accd[j] = v16i{0};
  if constexpr (FUSED && F4) {
    const uint8_t* as = lds + (nst % D) * STAGE + kg * A_STEP;
    v16f accdf[OWN];
#pragma unroll
    for (int j = 0; j < OWN; ++j) accdf[j] = v16f{0.0f};
    for (int g = 0; g < Gd; ++g) {
      const int e = g * BN + wn * 32 + l32;
      const v2i braw =
          *reinterpret_cast<const v2i*>(lds + dchunk(e >> 6) + (e & 63) * 16 + 8 * h);
      const uint32_t w0 = (uint32_t)braw[0], w1 = (uint32_t)braw[1];
      const v8i bf = v8i{(int)(w0 & 0x33333333u), (int)((w0 >> 2) & 0x33333333u),
                         (int)(w1 & 0x33333333u), (int)((w1 >> 2) & 0x33333333u), 0, 0, 0, 0};
#pragma unroll
      for (int j = 0; j < OWN; ++j) {
        const v4i w = *reinterpret_cast<const v4i*>(as + (j * Gd + g) * 1024 + lane * 16);
        const v8i af = v8i{w.x, w.y, w.z, w.w, 0, 0, 0, 0};
        accdf[j] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(bf, af, accdf[j], 4, 4, 0,
                                                                   127, 0, 127);
      }
    }
#pragma unroll
    for (int j = 0; j < OWN; ++j)
#pragma unroll
      for (int i = 0; i < 16; ++i) accd[j][i] = (int)accdf[j][i];
    __syncthreads();   // before the K-group exchange reuses this LDS
  } else if constexpr (FUSED) {
    const uint8_t* as = lds + (nst % D) * STAGE + kg * A_STEP;
    for (int g = 0; g < Gd; ++g) {
      const int e = g * BN + wn * 32 + l32;
      const v2i braw =
          *reinterpret_cast<const v2i*>(lds + dchunk(e >> 6) + (e & 63) * 16 + 8 * h);
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const v4i bf = unpack2((uint32_t)braw[t]);
#pragma unroll
        for (int j = 0; j < OWN; ++j) {
          const v4i af = *reinterpret_cast<const v4i*>(
              as + (j * 2 * Gd + 2 * g + t) * 1024 + lane * 16);
          accd[j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(bf, af, accd[j], 0, 0, 0);
        }
      }
    }
    __syncthreads();   // before the K-group exchange reuses this LDS
  }

  // ---- K groups: wave (kg, wn) keeps row blocks kg*OWN .. kg*OWN + OWN - 1
  // of its pixel column; the other groups' sums of those blocks come through
  // LDS (4 KB per 32x32 block) ------------------------------------------------
  v16i own[OWN];
  // (indices of acc stay compile-time: a runtime index would move it to
  // scratch)
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
    if (fm / OWN == kg) own[fm % OWN] = acc[fm];
  if constexpr (WK > 1) {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      if (fm / OWN == kg) continue;
      uint8_t* dst = lds + ((kg * WN + wn) * FM + fm) * 4096;
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *reinterpret_cast<v4i*>(dst + j * 1024 + lane * 16) =
            v4i{acc[fm][4 * j], acc[fm][4 * j + 1], acc[fm][4 * j + 2], acc[fm][4 * j + 3]};
    }
    __syncthreads();
#pragma unroll
    for (int k2 = 0; k2 < WK; ++k2) {
      if (k2 == kg) continue;
#pragma unroll
      for (int j = 0; j < OWN; ++j) {
        const uint8_t* src = lds + ((k2 * WN + wn) * FM + kg * OWN + j) * 4096;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const v4i v = *reinterpret_cast<const v4i*>(src + q * 1024 + lane * 16);
          own[j][4 * q] += v.x;
          own[j][4 * q + 1] += v.y;
          own[j][4 * q + 2] += v.z;
          own[j][4 * q + 3] += v.w;
        }
      }
    }
    __syncthreads();
  }

  if constexpr (SW) {
    // thresholds stay as raw records at THR; the join stages its coefficients
    if (FUSED) stage_epilogue(a, lds, co0, BM);
  } else if (pk)
    stage_thr_pk(reinterpret_cast<const int4*>(lds + THR), lds, BM);
  else if (pk_idj)
    stage_idj_pk(tbl_pre ? reinterpret_cast<const int32_t*>(lds + THR) : a.table + co0 * 16,
                 lds, BM, a.cout - co0 < BM ? a.cout - co0 : BM);
  else
    stage_epilogue(a, lds, co0, BM);
  __syncthreads();
  const int orow = a.out_mode == 2 ? BM / 4 : BM;
  uint8_t* otile = lds + EPI_BYTES;
  const int pl = wn * 32 + l32;
  if constexpr (SW) {
    if (a.acc_dump) dump_acc_t<OWN>(a, own, kg, h, l32, co0, p0, wn * 32, bn, a.acc_dump);
    if constexpr (FUSED)
      epilogue_cjoin_t<OWN>(a, lds, own, accd, kg, h, l32, co0, wn * 32, otile, orow);
    else
      epilogue_thr_pk_t<OWN>(a, reinterpret_cast<const int4*>(lds + THR), own, kg, h, l32, co0,
                             wn * 32, otile, orow);
  } else {
    v16i own2[OWN][1];
#pragma unroll
    for (int j = 0; j < OWN; ++j) own2[j][0] = own[j];
    const bool fast = (a.cout & 31) == 0 && (a.out_mode == 0 || a.rec == 4);
    int32_t* y32 = reinterpret_cast<int32_t*>(a.y);
    if (a.acc_dump)
      epilogue32<kE32I32, OWN, 1>(a, lds, own2, kg, wn, h, l32, co0, p0, bn, otile, orow,
                                  a.acc_dump);
    if (pk) {
      epilogue_thr_pk<OWN>(a, lds, own, kg, h, co0, pl, otile, orow);
    } else if (pk_idj) {
      // shortcut codes of the row blocks this wave finishes (loading them
      // before the main loop, as compiler-visible loads among the explicitly
      // counted DMA, measured slower)
      uint2 scw[OWN];
      const int pc = p0 + pl < a.m ? p0 + pl : a.m - 1;
#pragma unroll
      for (int j = 0; j < OWN; ++j) {
        const int co = co0 + (kg * OWN + j) * 32;
        scw[j] = co < a.cout ? shortcut8(a, pc, co) : uint2{0, 0};
      }
      epilogue_idj_pk<OWN>(a, lds, own, scw, kg, h, co0, pl, otile, orow);
    } else if (fast) {
      if (a.out_mode == 0)
        epilogue32<kE32I32, OWN, 1>(a, lds, own2, kg, wn, h, l32, co0, p0, bn, otile, orow, y32);
      else if (a.join_kind == IFQ_JOIN_IDENTITY)
        epilogue32<kE32Tab4, OWN, 1>(a, lds, own2, kg, wn, h, l32, co0, p0, bn, otile, orow, y32);
      else if (a.join_kind == IFQ_JOIN_CONV)
        epilogue32<kE32Conv, OWN, 1>(a, lds, own2, kg, wn, h, l32, co0, p0, bn, otile, orow, y32);
      else
        epilogue32<kE32Thr4, OWN, 1>(a, lds, own2, kg, wn, h, l32, co0, p0, bn, otile, orow, y32);
    } else {
      epilogue_lane<OWN * 4, 1>(
          a, lds, [&](int g, int fn, int i) { return own2[g >> 2][fn][4 * (g & 3) + i]; },
          [&](int g) { return co0 + (kg * OWN + (g >> 2)) * 32 + 8 * (g & 3) + 4 * h; }, co0,
          p0, [&](int fn) { return (pl < bn && p0 + pl < a.m) ? pl : -1; }, otile, orow);
    }
  }
  __syncthreads();
  const int npx = a.m - p0 < bn ? a.m - p0 : bn;
  if (a.pool_k)
    pool_out_tile(a, otile, orow, co0, BM, p0, npx);
  else
    copy_out_tile(a, otile, orow, co0, BM, p0, npx);
}

// ---------------------------------------------------------------------------
// Variants and per-layer planning
// ---------------------------------------------------------------------------
struct HaloVariant {
  int wn, wk, d, fm;   // waves along pixels, K groups, ring stages, row blocks per wave
  double c0_us;        // fixed cost per round of workgroups on a CU (plan_time)
  double eff;          // MFMA efficiency of a tile's main loop (plan_time)
  const char* name;    // the kernels as a profiler lists them: unfused,
  const char* sw_name;       // unfused on the transposed layout,
  const char* fused_name;    // fused downsample (transposed layout),
  const char* f4_name;       // fp4 contraction (transposed layout),
  const char* f4_idj_name;   // fp4 contraction, identity join (untransposed),
  const char* f4_fused_name; // fp4 contraction, fused downsample (transposed)
};

// Index order must match the switch in launch_conv_halo. Variants with
// fm = 2 (64 output channels) run two workgroups per CU.
// (c0_us, eff) fitted to measured MI355X kernel times (ResNet-18, AlexNet,
// VGG-16, Tiny-YOLOv2 layer shapes).
const HaloVariant kHaloVariants[] = {
    {8, 1, 6, 4, 4.0, 0.55, "conv_halo<8, 1, 6, false, 4, false, false>", "conv_halo<8, 1, 6, false, 4, true, false>",
     "conv_halo<8, 1, 6, true, 4, true, false>", "conv_halo<8, 1, 6, false, 4, true, true>",
     "conv_halo<8, 1, 6, false, 4, false, true>", "conv_halo<8, 1, 6, true, 4, true, true>"},
    {4, 2, 4, 4, 3.5, 0.55, "conv_halo<4, 2, 4, false, 4, false, false>", "conv_halo<4, 2, 4, false, 4, true, false>",
     "conv_halo<4, 2, 4, true, 4, true, false>", "conv_halo<4, 2, 4, false, 4, true, true>",
     "conv_halo<4, 2, 4, false, 4, false, true>", "conv_halo<4, 2, 4, true, 4, true, true>"},
    {2, 4, 4, 4, 5.7, 0.55, "conv_halo<2, 4, 4, false, 4, false, false>", "conv_halo<2, 4, 4, false, 4, true, false>",
     "conv_halo<2, 4, 4, true, 4, true, false>", "conv_halo<2, 4, 4, false, 4, true, true>",
     "conv_halo<2, 4, 4, false, 4, false, true>", "conv_halo<2, 4, 4, true, 4, true, true>"},
    {8, 1, 6, 2, 2.0, 0.33, "conv_halo<8, 1, 6, false, 2, false, false>", "conv_halo<8, 1, 6, false, 2, true, false>",
     nullptr, nullptr, nullptr, nullptr},   // 64 x 256
};
constexpr int kNumHalo = sizeof(kHaloVariants) / sizeof(kHaloVariants[0]);
constexpr int kNumCUs = 256;

// Upper bound of the halo cells (rounded per image to 64) one tile of bn
// output pixels needs per channel block, over every tile of the layer.
int64_t halo_cells_bound(const ConvLaunch& a, int64_t bn) {
  const int64_t howo = (int64_t)a.ho * a.wo;
  const int64_t nseg = (bn - 1) / howo + 2;              // images a tile touches
  const int64_t rows_out = (bn - 1) / a.wo + 2;          // output rows it touches
  int64_t rows_in = rows_out * a.stride + 3;
  if (rows_in > a.h) rows_in = a.h;
  return nseg * round64((int)(rows_in * a.w));
}

}  // namespace

bool plan_halo(const ConvLaunch& a, HaloPlan* out) {
  if (!(a.in_layout == IFQ_LAYOUT_U2_BLOCK64 && a.in_bits == 2 && a.cin % 64 == 0 &&
        a.kh == 3 && a.kw == 3 && a.pad == 1 && (a.stride == 1 || a.stride == 2) && a.m > 0))
    return false;
  // 32-bit cell indices and offsets
  if ((int64_t)a.n * a.h * a.w * (a.cin / 64) >= (int64_t)1 << 26) return false;
  const bool fused = a.join_kind == IFQ_JOIN_CONV_FUSED;
  if (fused && !(a.out_mode == 2 && a.rec == 4 && a.out_layout == IFQ_LAYOUT_U2_BLOCK64 &&
                 a.sc_layout == IFQ_LAYOUT_U2_BLOCK64 && a.d_cin % 64 == 0 &&
                 a.cout % 32 == 0 &&
                 (int64_t)a.n * a.d_h * a.d_w * (a.d_cin / 64) < (int64_t)1 << 26))
    return false;
  if (a.pool_k && !pool_epilogue_ok(a)) return false;
  const int G = a.cin / 64;
  double best_t = 1e30;
  bool found = false;
  for (int v = 0; v < kNumHalo; ++v) {
    const HaloVariant& V = kHaloVariants[v];
    if (G % V.wk) continue;
    // the fp4 instance of the two-workgroups-per-CU variant needs more than
    // its 128 VGPRs (spills): fp4 layers take the 128-channel tiles instead
    if (a.f4 && !V.f4_name) continue;
    const int bm = 32 * V.fm, bnmax = 32 * V.wn;
    const int occ = V.fm == 2 ? 2 : 1;               // workgroups per CU
    const int cap = halo_cap_cells(V.wk, V.fm);
    if (fused) {
      // the downsample's K64 steps split one per group; its input chunks
      // (one per wave) fit the spare halo buffers
      const int gd = a.d_cin / 64, nqd = gd * bnmax / 64;
      if (!V.fused_name || gd != V.wk || nqd > kHaloNW || nqd > V.wk * (cap / 64)) continue;
    }
    const int64_t slots = (int64_t)kNumCUs * occ;
    const int64_t nco = (a.cout + bm - 1) / bm;
    const int64_t nb_min = (a.m + bnmax - 1) / bnmax;
    const int64_t rounds = (nco * nb_min + slots - 1) / slots;
    int64_t nb = rounds * slots / nco;
    if (nb < nb_min) nb = nb_min;
    int64_t bn = (a.m + nb - 1) / nb;
    bn = (bn + 31) / 32 * 32;
    if (bn > bnmax) bn = bnmax;
    if (a.pool_k) {
      // a fused pool needs whole rows of pooling windows (or whole images)
      // per tile
      const int64_t unit = a.pool_img ? (int64_t)a.ho * a.wo : (int64_t)a.pool_k * a.wo;
      bn = (bn + unit - 1) / unit * unit;
      if (bn > bnmax) bn = bnmax / unit * unit;
      if (bn == 0) continue;
    }
    const int64_t cells = halo_cells_bound(a, bn);
    if (cells > cap) continue;
    const int nr = 11 - V.d < kTaps ? 11 - V.d : kTaps;
    if (V.wk * (cells / 64) > kHaloNW * nr) continue;
    const int64_t blocks = nco * ((a.m + bn - 1) / bn);
    // occ workgroups share a CU: each runs at 1/occ of its MFMA rate
    const double t = plan_time(blocks, 2.0 * bm * bnmax * (double)a.kpad, occ, V.c0_us, V.eff);
    if (t < best_t) {
      best_t = t;
      *out = HaloPlan{v, (int)bn, (int)((a.m + bn - 1) / bn), t};
      found = true;
    }
  }
  return found;
}

// Which instance of a variant runs: 0 = unfused, 1 = unfused on the
// transposed layout (the 2-bit threshold epilogue with packed 16-bit
// compares, the same condition as the kernel's pk), 2 = fused downsample,
// 3 = the fp4 contraction (a.f4; the same epilogue as 1, checked by the host),
// 4 = the fp4 contraction with the identity join (untransposed, as 0),
// 5 = the fp4 contraction with the fused downsample (as 2).
int halo_instance(const ConvLaunch& a) {
  if (a.f4)
    return a.join_kind == IFQ_JOIN_IDENTITY ? 4 : a.join_kind == IFQ_JOIN_CONV_FUSED ? 5 : 3;
  if (a.join_kind == IFQ_JOIN_CONV_FUSED) return 2;
  const bool pk = a.out_mode == 2 && a.rec == 4 && (a.cout & 31) == 0 &&
                  27 * a.cin <= 32766 && a.join_kind == IFQ_JOIN_NONE;
  return pk ? 1 : 0;
}

// The kernel's name as a profiler lists it (the template arguments).
const char* conv_halo_name(const HaloPlan& p, const ConvLaunch& a) {
  const HaloVariant& V = kHaloVariants[p.variant];
  const int inst = halo_instance(a);
  return inst == 5   ? V.f4_fused_name
         : inst == 4 ? V.f4_idj_name
         : inst == 3 ? V.f4_name
         : inst == 2 ? V.fused_name
         : inst == 1 ? V.sw_name
                     : V.name;
}

hipError_t launch_conv_halo(ConvLaunch a, const HaloPlan& p, hipStream_t stream) {
  a.bn = p.bn;
  const int bm = 32 * kHaloVariants[p.variant].fm;
  const dim3 grid(p.blocks_m, (a.cout + bm - 1) / bm);
  const int inst = halo_instance(a);
  switch (inst == 5   ? 20 + p.variant
          : inst == 4 ? 16 + p.variant
          : inst == 3 ? 12 + p.variant
                      : p.variant * 3 + inst) {
#define IFQ_HALO_CASE(k, wn, wk, d, fu, fm, sw) \
    case k: hipLaunchKernelGGL((conv_halo<wn, wk, d, fu, fm, sw>), grid, dim3(512), 0, stream, a); break;
#define IFQ_HALO_F4(k, wn, wk, d, fu, fm, sw) \
    case k: hipLaunchKernelGGL((conv_halo<wn, wk, d, fu, fm, sw, true>), grid, dim3(512), 0, stream, a); break;
    IFQ_HALO_CASE(0, 8, 1, 6, false, 4, false)
    IFQ_HALO_CASE(1, 8, 1, 6, false, 4, true)
    IFQ_HALO_CASE(2, 8, 1, 6, true, 4, true)
    IFQ_HALO_CASE(3, 4, 2, 4, false, 4, false)
    IFQ_HALO_CASE(4, 4, 2, 4, false, 4, true)
    IFQ_HALO_CASE(5, 4, 2, 4, true, 4, true)
    IFQ_HALO_CASE(6, 2, 4, 4, false, 4, false)
    IFQ_HALO_CASE(7, 2, 4, 4, false, 4, true)
    IFQ_HALO_CASE(8, 2, 4, 4, true, 4, true)
    IFQ_HALO_CASE(9, 8, 1, 6, false, 2, false)
    IFQ_HALO_CASE(10, 8, 1, 6, false, 2, true)
    IFQ_HALO_F4(12, 8, 1, 6, false, 4, true)
    IFQ_HALO_F4(13, 4, 2, 4, false, 4, true)
    IFQ_HALO_F4(14, 2, 4, 4, false, 4, true)
    IFQ_HALO_F4(16, 8, 1, 6, false, 4, false)
    IFQ_HALO_F4(17, 4, 2, 4, false, 4, false)
    IFQ_HALO_F4(18, 2, 4, 4, false, 4, false)
    IFQ_HALO_F4(20, 8, 1, 6, true, 4, true)
    IFQ_HALO_F4(21, 4, 2, 4, true, 4, true)
    IFQ_HALO_F4(22, 2, 4, 4, true, 4, true)
#undef IFQ_HALO_CASE
#undef IFQ_HALO_F4
    default: return hipErrorInvalidValue;   // no fused kernel for this variant
  }
  return hipGetLastError();
}

}  // namespace ifq
