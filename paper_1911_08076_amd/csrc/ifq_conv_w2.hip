// Windowed 3x3 kernel with register-blocked waves, for 3x3 filters (stride 1
// or 2, zero padding 1) on 2-bit codes in the BLOCK64 layout, c_in a
// multiple of 64, on gfx950 (MI355X).
//
// The integer part of Eq. (1), a = W_b (x) X_q, as the implicit GEMM
// D[co][pixel] = sum_k W[co][k] * X[pixel][k] on v_mfma_i32_32x32x32_i8
// (or, with F4, exactly on the fp4 scaled MFMA, as in ifq_conv_halo.hip).
// What differs from ifq_conv_halo.hip is how the work is spread:
//
//  - Codes: the input window of the tile for EVERY channel block is brought
//    into LDS once, in the prologue (one contiguous span of 16-byte BLOCK64
//    cells per image the tile touches and per block; 2-bit codes make it
//    small: a few KB per block). The main loop never waits on codes.
//  - Weights stream through a ring of D LDS stages; a stage holds T filter
//    taps (T in {1, 3, 9}) of one channel block for each of the WK K groups,
//    so the loop waits and synchronises once per T taps, not once per tap.
//  - Waves: WM x WN x WK. Wave (wm, wn, kg) owns FM 32-channel row blocks x
//    FN 32-pixel column blocks of the tile (FM*FN accumulators) and the
//    channel blocks g with g % WK == kg. Every A fragment (weights) read from
//    LDS feeds FN MFMAs and every unpacked B fragment (codes) FM MFMAs, so
//    fewer LDS bytes and VALU unpacks are spent per MFMA than with one
//    32-pixel column per wave. The K groups add their sums through LDS.
//
// Epilogues (MODE): 0, the 2-bit threshold epilogue of Eq. (7)/(8) on the
// transposed layout (codes as the MFMA's A operand, one output channel per
// lane); 1, the identity residual join on the untransposed layout, both with
// the packed 16-bit compares of ifq_mfma_common.h; 2, the join with a 1x1
// downsample computed in the kernel (its weights arrive as one extra stage of
// the ring, its strided input cells in the prologue) and the fp64 join of
// ifq_epilogue.h on the transposed layout. Optional int32 dump of the sums.
//
// K split across workgroups (MODE 3: the threshold epilogue, a.ksplit > 1): the
// grid's z index picks a range of c_in/64/ksplit channel blocks. Each
// workgroup of a tile writes its int32 partial tile to the workspace,
// fences, and counts its arrival on the tile's counter; the one that
// arrives last adds the other partials to its own (integer addition is
// associative, so the sums are exact) and runs the epilogue. No workgroup
// waits for another, and the counter returns to zero with the last arrival.
#include <hip/hip_runtime.h>

#include "ifq_epilogue.h"
#include "ifq_internal.h"
#include "ifq_mfma_common.h"

namespace ifq {
namespace {

constexpr int kW2Taps = 9;

__host__ __device__ constexpr int w2_round64(int v) { return (v + 63) & ~63; }
__host__ __device__ constexpr int w2_max(int a, int b) { return a > b ? a : b; }

template <int WM, int WN, int WK, int FM, int FN, int T, int D, int MODE, bool F4, int OCC,
          int WINB>
__global__ __launch_bounds__(64 * WM * WN * WK, (WM * WN * WK / 4) * OCC) void conv_w2(
    ConvLaunch a) {
  // MODE 3: the threshold epilogue (0) with the K split across workgroups
  constexpr bool SPLIT = MODE == 3;
  constexpr int EM = SPLIT ? 0 : MODE;           // the epilogue
  constexpr bool SW = EM != 1;                 // transposed sums
  constexpr bool FUSED = EM == 2;
  constexpr int GDM = 4;                         // downsample channel blocks at most
  constexpr int NW = WM * WN * WK;
  constexpr int NT = 64 * NW;
  constexpr int BM = 32 * FM * WM;
  constexpr int BN = 32 * FN * WN;
  constexpr int KH = F4 ? 1 : 2;                 // 1 KB chunks per row block and K64 step
  constexpr int RB = BM / 32;                    // row blocks of the tile
  constexpr int NCH = WK * T * RB * KH;          // 1 KB weight chunks per stage
  constexpr int CPW = (NCH + NW - 1) / NW;       // loads per wave per stage
  constexpr int STAGE = NCH * 1024;
  constexpr int TSTEPS = kW2Taps / T;            // stages per channel block
  constexpr int NB = FM * FN / WK;               // blocks a wave keeps after the K sum
  static_assert(NW % 4 == 0 && NW <= 16, "waves");
  static_assert(kW2Taps % T == 0, "taps per stage");
  static_assert((FM * FN) % WK == 0, "K-group split of the wave's blocks");
  static_assert(BM % 64 == 0, "64-channel record chunks");
  static_assert(D >= 2 && (D - 2) * CPW <= 63, "vmcnt range");
  constexpr int RING = D * STAGE;
  constexpr int WIN0 = RING;
  constexpr int DUMMY = WIN0 + WINB;             // 1 KB sink of padding loads
  constexpr int NOK = FM * FN - NB;              // blocks a wave hands to the others
  constexpr int RED_BYTES = WK > 1 ? NW * NOK * 4096 : 0;
  // staged epilogue parameters: the identity join's records, or the
  // downsample join's {p, q, cc} per channel (at kJoinCoefOff)
  constexpr int EPI_BYTES = EM == 1 ? BM * 128 : EM == 2 ? (kJoinCoefOff + BM * 24 + 15) / 16 * 16 : 0;
  constexpr int OUT_BYTES = BN * BM / 4;         // 2-bit output tile
  // prefetched per-channel records: thresholds, join records or coefficients
  constexpr int TBL_BYTES = EM == 0 ? BM * 16 : EM == 1 ? BM * 64 : (BM * 24 + 1023) / 1024 * 1024;
  constexpr int THR = w2_max(w2_max(DUMMY + 1024, RED_BYTES), EPI_BYTES + OUT_BYTES);
  // the tile's shortcut cells [BM/64 blocks][BN pixels] (identity join) or
  // the downsample's strided input cells [GDM blocks][BN pixels], 16 B each
  constexpr int SCB = THR + TBL_BYTES;
  constexpr int SC_BYTES = EM == 1 ? (BM / 64) * BN * 16 : EM == 2 ? GDM * BN * 16 : 0;
  constexpr int LDS_BYTES = SCB + SC_BYTES;
  static_assert(LDS_BYTES <= 160 * 1024, "LDS");

  __shared__ __attribute__((aligned(1024))) uint8_t lds[LDS_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = wave / (WM * WN);
  const int wmn = wave - kg * WM * WN;
  const int wm = wmn / WN;
  const int wn = wmn - wm * WN;
  const int h = lane >> 5;
  const int l32 = lane & 31;
  const int bn = a.bn;
  const int p0 = blockIdx.x * bn;
  const int co0 = blockIdx.y * BM;
  const int G = a.cin >> 6;                      // channel blocks of the layer
  const int Gs = SPLIT ? G / a.ksplit : G;       // of this workgroup's K range
  const int gbase = SPLIT ? (int)blockIdx.z * Gs : 0;
  const int nst = (Gs / WK) * TSTEPS;
  const int H = a.h, W = a.w, Wo = a.wo, st = a.stride;
  const int howo = a.ho * a.wo;
  const int HW = H * W;
  const int wcells = a.wcells;                   // cells per block window (host bound)
  const int wstr = (wcells + 1) * 16;            // block window + its zero cell
  const uint32_t lds0 = lds_addr(lds);
  const uint8_t* zero_src = reinterpret_cast<const uint8_t*>(&g_zero_cell);

  // zero cell after every block window
  for (int g = tid; g < Gs; g += NT)
    *reinterpret_cast<uint4*>(lds + WIN0 + g * wstr + wcells * 16) = uint4{0, 0, 0, 0};

  // ---- the tile's images (segments) and their input row spans ------------
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

  // ---- prologue: the epilogue's per-channel records, the windows of all
  // channel blocks, then stages 0 .. D-2 of the weight ring --------------------
  if constexpr (EM == 0) {
    for (int q = wave; q < BM / 64; q += NW) {
      const int c = co0 + q * 64 + lane;
      dma16(c < a.cout ? reinterpret_cast<const uint8_t*>(a.thr + (int64_t)c * 4) : zero_src,
            lds0 + THR + q * 1024);
    }
  } else if constexpr (EM == 2) {
    // the join coefficients of the tile's channels (24 bytes each, as 16-byte
    // pieces; c_out % 32 == 0 keeps every piece inside the array or past it)
    const uint8_t* cf8 = reinterpret_cast<const uint8_t*>(a.coef);
    const int nch = a.cout - co0 < BM ? a.cout - co0 : BM;
    for (int q = wave; q < TBL_BYTES / 1024; q += NW) {
      const int e = q * 64 + lane;               // 16-byte piece of the slice
      dma16(e * 16 < nch * 24 ? cf8 + (int64_t)co0 * 24 + e * 16 : zero_src,
            lds0 + THR + q * 1024);
    }
    // the downsample's input cells of the tile's pixels: pixel (n, oy, ox)
    // reads cell (n, gd, oy*d_stride, ox*d_stride) of its BLOCK64 input
    const int Gd = a.d_cin >> 6;
    const int ncx = (bn + 63) >> 6;
    for (int q = wave; q < Gd * ncx; q += NW) {
      const int gd = q / ncx, j = q - gd * ncx;
      const int pl = j * 64 + lane, p = p0 + pl;
      const uint8_t* src = zero_src;
      if (pl < bn && p < a.m) {
        const int n = fdiv(p, a.div_howo);
        const int rem = p - n * howo;
        const int oy = fdiv(rem, a.div_wo);
        const int ox = rem - oy * Wo;
        src = a.dx + ((((int64_t)n * Gd + gd) * a.d_h + oy * a.d_stride) * a.d_w +
                      ox * a.d_stride) * 16;
      }
      dma16(src, lds0 + SCB + (uint32_t)((gd * BN + j * 64) * 16));
    }
  } else {
    for (int q = wave; q < BM / 16; q += NW) {   // 16 channels x 64 B per chunk
      const int c = co0 + q * 16 + (lane >> 2);
      dma16(c < a.cout ? reinterpret_cast<const uint8_t*>(a.table + (int64_t)c * 16 + (lane & 3) * 4)
                       : zero_src,
            lds0 + THR + q * 1024);
    }
    // the shortcut's 16-byte cells (64 channels of one pixel) of the tile's
    // pixels and channel blocks, read by the epilogue: chunk q = 64 pixels
    // of one block (c_out % 64 == 0, checked by the host)
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
      dma16(src, lds0 + SCB + (uint32_t)((gbl * BN + j * 64) * 16));
    }
  }
  {
    // the windows: chunk j of image segment i is 64 cells of that image's
    // input rows, the same chunk for every channel block g; wave w takes the
    // chunks j' = w, w + NW, .. of the segments' chunk list
    int off = 0, jbase = 0;
    for (int i = 0; i < nseg; ++i) {
      int iya;
      const int cells = seg_rows(i, iya) * W;
      const int nch = w2_round64(cells) >> 6;
      int j = wave - jbase;
      j += j < 0 ? ((-j + NW - 1) / NW) * NW : 0;
      for (; j < nch; j += NW) {
        const int c = j * 64 + lane;
        const int64_t src = ((int64_t)(n_first + i) * G * HW + iya * W + c) * 16;
        for (int g = 0; g < Gs; ++g)
          dma16(c < cells ? a.x + src + (int64_t)(gbase + g) * HW * 16 : zero_src,
                lds0 + WIN0 + (uint32_t)(g * wstr + (off + j * 64) * 16));
      }
      jbase += nch;
      off += w2_round64(cells);
    }
  }

  const int nrb = a.cout_pad >> 5;
  const int rbw = co0 >> 5;
  const uint8_t* wbase = reinterpret_cast<const uint8_t*>(a.wgt);
  const uint32_t voff = (uint32_t)lane * 16;
  // stage s: taps (s % TSTEPS)*T .. +T-1 of channel block (s / TSTEPS)*WK + kq
  // for each K group kq; chunk c = ((kq*T + tau)*RB + rb)*KH + t
  auto issue_stage = [&](int s) {
    const int gi = s / TSTEPS;
    const int tap0 = (s - gi * TSTEPS) * T;
    const uint32_t slot = lds0 + (uint32_t)((s % D) * STAGE);
#pragma unroll
    for (int k = 0; k < CPW; ++k) {
      const int c = wave + NW * k;
      if (NCH % NW == 0 || c < NCH) {
        const int t = c % KH;
        const int rb = (c / KH) % RB;
        const int kt = c / (KH * RB);
        const int tau = kt % T, kq = kt / T;
        const int kk = (gbase + gi * WK + kq) * kW2Taps + tap0 + tau;
        const int64_t off =
            rbw + rb < nrb ? ((int64_t)(rbw + rb) * (KH * a.nk) + KH * kk + t) * 1024 : a.wzero;
        dma16s(wbase + off, voff, slot + (uint32_t)(c * 1024));
      } else {
        dma16(zero_src, lds0 + DUMMY);
      }
    }
  };
  // the downsample's weights: one extra stage after the 3x3 stages, chunk
  // c = (gd*RB + rb)*KH + t (Gd * RB * KH <= NCH, checked by the host)
  const int nst_all = nst + (FUSED ? 1 : 0);
  auto issue_down = [&]() {
    const uint32_t slot = lds0 + (uint32_t)((nst % D) * STAGE);
    const int Gd = a.d_cin >> 6;
#pragma unroll
    for (int k = 0; k < CPW; ++k) {
      const int c = wave + NW * k;
      if (c < Gd * RB * KH) {
        const int t = c % KH;
        const int rb = (c / KH) % RB;
        const int gd = c / (KH * RB);
        const int64_t off =
            rbw + rb < nrb
                ? ((int64_t)(rbw + rb) * (KH == 2 ? a.d_nk32 : Gd) + (KH == 2 ? 2 * gd + t : gd)) *
                      1024
                : a.d_wzero;
        dma16s(reinterpret_cast<const uint8_t*>(a.dwgt) + off, voff, slot + (uint32_t)(c * 1024));
      } else {
        dma16(zero_src, lds0 + DUMMY);
      }
    }
  };
  auto issue_any = [&](int s) {
    if (s < nst)
      issue_stage(s);
    else
      issue_down();
  };
  const int pre = nst_all < D - 1 ? nst_all : D - 1;
  for (int s = 0; s < pre; ++s) issue_any(s);

  // ---- per-lane LDS offsets of the nine taps of each pixel column block,
  // relative to a block window (computed while the prologue's loads are in
  // flight); a tap outside the image reads the zero cell (8*h: the lane's
  // half of the cell, the MFMA's K half) ---------------------------------------
  int boff[FN][kW2Taps];
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
      for (int i = 0; i < nseg; ++i) {
        int iya;
        const int rows = seg_rows(i, iya);
        if (i == n - n_first) {
          my_off = off;
          my_iya = iya;
        }
        off += w2_round64(rows * W);
      }
    }
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
      for (int s = 0; s < 3; ++s) {
        const int iy = oy * st - 1 + r;
        const int ix = ox * st - 1 + s;
        const bool ok = pok && (unsigned)iy < (unsigned)H && (unsigned)ix < (unsigned)W;
        boff[fn][r * 3 + s] = (ok ? (my_off + (iy - my_iya) * W + ix) * 16 : wcells * 16) + 8 * h;
      }
  }


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

  struct Frag {
    v4i af[KH][FM];
    v2i braw[FN];
  };
  // fragments of tap `tap` (stage-local tap tau) of the stage in LDS slot
  // `slot`, for this wave; win is the wave's block window
  auto read_frags = [&](int slot, int tau, int tap, const uint8_t* win, Frag& F) {
    const uint8_t* as = lds + slot * STAGE + ((kg * T + tau) * RB + wm * FM) * KH * 1024;
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int t = 0; t < KH; ++t)
        F.af[t][fm] = *reinterpret_cast<const v4i*>(as + (fm * KH + t) * 1024 + lane * 16);
#pragma unroll
    for (int fn = 0; fn < FN; ++fn)
      F.braw[fn] = *reinterpret_cast<const v2i*>(win + boff[fn][tap]);
  };
  auto mfmas = [&](const Frag& F) {
    if constexpr (F4) {
#pragma unroll
      for (int fn = 0; fn < FN; ++fn) {
        // 32 codes of the lane's half cell as nibbles (the fp4 weight blob
        // follows this order): codes 0, 2, .., 14 of braw.x, then 1, 3, ..,
        // 15, then the same of braw.y
        const uint32_t w0 = (uint32_t)F.braw[fn][0], w1 = (uint32_t)F.braw[fn][1];
        const v8i bf = v8i{(int)(w0 & 0x33333333u), (int)((w0 >> 2) & 0x33333333u),
                           (int)(w1 & 0x33333333u), (int)((w1 >> 2) & 0x33333333u), 0, 0, 0, 0};
#pragma unroll
        for (int fm = 0; fm < FM; ++fm) {
          const v4i w = F.af[0][fm];
          const v8i af = v8i{w.x, w.y, w.z, w.w, 0, 0, 0, 0};
          if constexpr (SW)
            accf[fm][fn] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                bf, af, accf[fm][fn], 4, 4, 0, 127, 0, 127);
          else
            accf[fm][fn] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                af, bf, accf[fm][fn], 4, 4, 0, 127, 0, 127);
        }
      }
    } else {
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          const v4i bf = unpack2((uint32_t)F.braw[fn][t]);
#pragma unroll
          for (int fm = 0; fm < FM; ++fm) {
            if constexpr (SW)
              acc[fm][fn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(bf, F.af[t][fm], acc[fm][fn], 0, 0, 0);
            else
              acc[fm][fn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(F.af[t][fm], bf, acc[fm][fn], 0, 0, 0);
          }
        }
    }
  };

  // Iteration s (channel-block step gi, stage ts of its TSTEPS): wait until
  // stage s has landed (loads complete in issue order: at most the stages
  // issued after it may be outstanding), barrier, issue stage s + D - 1 into
  // the slot of stage s - 1 (read in iteration s - 1, before this barrier),
  // then the T taps of stage s, the fragments of tap tau + 1 read before the
  // MFMAs of tap tau. The first wait also covers the windows and records,
  // issued before stage 0. Taps are compile-time indices (the stage loop is
  // unrolled per block), so boff stays in registers.
  const int nG = Gs / WK;
  int slot = 0;
  for (int gi = 0; gi < nG; ++gi) {
    const uint8_t* win = lds + WIN0 + (gi * WK + kg) * wstr;
#pragma unroll
    for (int ts = 0; ts < TSTEPS; ++ts) {
      const int s = gi * TSTEPS + ts;
      const int after = nst_all - 1 - s;
      wait_ahead<D - 2, CPW>(after < D - 2 ? after : D - 2);
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      if (s + D - 1 < nst_all) issue_any(s + D - 1);
      Frag f0, f1;
      read_frags(slot, 0, ts * T, win, f0);
#pragma unroll
      for (int tau = 0; tau < T; ++tau) {
        if (tau + 1 < T) read_frags(slot, tau + 1, ts * T + tau + 1, win, (tau & 1) ? f0 : f1);
        mfmas((tau & 1) ? f1 : f0);
      }
      slot = slot + 1 == D ? 0 : slot + 1;
    }
  }
  if constexpr (F4) {
    // exact integers (every partial sum is an integer below 2^24)
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[fm][fn][i] = (int)accf[fm][fn][i];
  }
  wait_vmcnt<0>();
  __syncthreads();

  // ---- the downsample's sums of the blocks this wave keeps after the K
  // sum (its weights in the extra stage's slot, its cells at SCB) ------------
  v16i accd[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) accd[j] = v16i{0};
  if constexpr (FUSED) {
    const uint8_t* ds = lds + (nst % D) * STAGE;
    const int Gd = a.d_cin >> 6;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int b = kg * NB + j;
      const int fm = b / FN, fn = b - fm * FN;
      const int pl = (wn * FN + fn) * 32 + l32;
      const int rbl = wm * FM + fm;
      v16f df = v16f{0.0f};
      for (int gd = 0; gd < Gd; ++gd) {
        const v2i braw = *reinterpret_cast<const v2i*>(lds + SCB + (gd * BN + pl) * 16 + 8 * h);
        if constexpr (F4) {
          const uint32_t w0 = (uint32_t)braw[0], w1 = (uint32_t)braw[1];
          const v8i bf = v8i{(int)(w0 & 0x33333333u), (int)((w0 >> 2) & 0x33333333u),
                             (int)(w1 & 0x33333333u), (int)((w1 >> 2) & 0x33333333u), 0, 0, 0, 0};
          const v4i w = *reinterpret_cast<const v4i*>(ds + (gd * RB + rbl) * 1024 + lane * 16);
          const v8i af = v8i{w.x, w.y, w.z, w.w, 0, 0, 0, 0};
          df = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(bf, af, df, 4, 4, 0, 127, 0, 127);
        } else {
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            const v4i af =
                *reinterpret_cast<const v4i*>(ds + ((gd * RB + rbl) * 2 + t) * 1024 + lane * 16);
            accd[j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(unpack2((uint32_t)braw[t]), af,
                                                            accd[j], 0, 0, 0);
          }
        }
      }
      if constexpr (F4) {
#pragma unroll
        for (int i = 0; i < 16; ++i) accd[j][i] = (int)df[i];
      }
    }
    __syncthreads();   // before the K-group exchange reuses the ring
  }

  // ---- K groups: wave (wm, wn, kg) keeps blocks b = fm*FN + fn in
  // [kg*NB, kg*NB + NB); the other groups' sums of those blocks come through
  // LDS (4 KB per 32x32 block; wave k2 stores its blocks outside its own
  // range at index b, less NB past that range) -------------------------------------
  v16i own[NB];
#pragma unroll
  for (int b = 0; b < FM * FN; ++b)
    if (b / NB == kg) own[b % NB] = acc[b / FN][b % FN];
  if constexpr (WK > 1) {
#pragma unroll
    for (int b = 0; b < FM * FN; ++b) {
      if (b / NB == kg) continue;
      const int bi = b < kg * NB ? b : b - NB;
      uint8_t* dst = lds + (((kg * WM + wm) * WN + wn) * NOK + bi) * 4096;
      const v16i v = acc[b / FN][b % FN];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        *reinterpret_cast<v4i*>(dst + j * 1024 + lane * 16) =
            v4i{v[4 * j], v[4 * j + 1], v[4 * j + 2], v[4 * j + 3]};
    }
    __syncthreads();
#pragma unroll
    for (int k2 = 0; k2 < WK; ++k2) {
      if (k2 == kg) continue;
#pragma unroll
      for (int j = 0; j < NB; ++j) {
        const int b = kg * NB + j;
        const int bi = b < k2 * NB ? b : b - NB;
        const uint8_t* src = lds + (((k2 * WM + wm) * WN + wn) * NOK + bi) * 4096;
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

  // ---- K split across workgroups: partial tiles through the workspace ------
  if constexpr (SPLIT) {
    const int S = a.ksplit;
    const int tile = blockIdx.y * gridDim.x + blockIdx.x;
    constexpr int PER = NB * 16;                 // int32 per thread
    int32_t* part = a.ws_part + (int64_t)tile * S * (NT * PER);
    int32_t* mine = part + (int64_t)blockIdx.z * (NT * PER) + tid * PER;
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<v4i*>(mine + j * 16 + 4 * q) =
            v4i{own[j][4 * q], own[j][4 * q + 1], own[j][4 * q + 2], own[j][4 * q + 3]};
    // every wave's stores have reached the L2 before the barrier; then one
    // device-scope fence (an L2 write-back for the whole workgroup) and the
    // arrival, whose count wraps to zero at the last of the S arrivals; the
    // last arrival's fence invalidates the caches the partials are read
    // through (one per workgroup: the waves share them)
    wait_vmcnt<0>();
    __syncthreads();
    volatile int* flag = reinterpret_cast<volatile int*>(lds);
    if (tid == 0) {
      __threadfence();
      const bool last = atomicInc(a.ws_cnt + tile, (unsigned)(S - 1)) == (unsigned)(S - 1);
      if (last) __threadfence();
      *flag = last;
    }
    __syncthreads();
    if (!*flag) return;
    for (int z = 0; z < S; ++z) {
      if (z == (int)blockIdx.z) continue;
      const int32_t* src = part + (int64_t)z * (NT * PER) + tid * PER;
#pragma unroll
      for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const v4i v = *reinterpret_cast<const v4i*>(src + j * 16 + 4 * q);
          own[j][4 * q] += v.x;
          own[j][4 * q + 1] += v.y;
          own[j][4 * q + 2] += v.z;
          own[j][4 * q + 3] += v.w;
        }
    }
    __syncthreads();   // the flag word before the epilogue's tile writes
  }

  // ---- epilogue -------------------------------------------------------------
  if constexpr (EM == 1)
    stage_idj_pk(reinterpret_cast<const int32_t*>(lds + THR), lds, BM,
                 a.cout - co0 < BM ? a.cout - co0 : BM);
  if constexpr (EM == 2) {
    const double* src = reinterpret_cast<const double*>(lds + THR);
    double* dst = reinterpret_cast<double*>(lds + kJoinCoefOff);
    for (int i = tid; i < BM * 3; i += NT) dst[i] = src[i];
  }
  __syncthreads();
  constexpr int orow = BM / 4;
  uint8_t* otile = lds + EPI_BYTES;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int b = kg * NB + j;
    const int rbl = wm * FM + b / FN;            // row block in the tile
    const int pcb = wn * FN + b % FN;            // pixel column block in the tile
    const v16i one[1] = {own[j]};
    if constexpr (EM == 0) {
      if (a.acc_dump) dump_acc_t<1>(a, one, rbl, h, l32, co0, p0, pcb * 32, bn, a.acc_dump);
      epilogue_thr_pk_t<1>(a, reinterpret_cast<const int4*>(lds + THR), one, rbl, h, l32, co0,
                           pcb * 32, otile, orow);
    } else if constexpr (EM == 2) {
      if (a.acc_dump) dump_acc_t<1>(a, one, rbl, h, l32, co0, p0, pcb * 32, bn, a.acc_dump);
      const v16i oned[1] = {accd[j]};
      epilogue_cjoin_t<1>(a, lds, one, oned, rbl, h, l32, co0, pcb * 32, otile, orow);
    } else {
      const v16i one2[1][1] = {{own[j]}};
      if (a.acc_dump)
        epilogue32<kE32I32, 1, 1>(a, lds, one2, rbl, pcb, h, l32, co0, p0, bn, otile, orow,
                                  a.acc_dump);
      const int pl = pcb * 32 + l32;
      const int cl = rbl * 32;                   // local first channel of the block
      const uint2 sc[1] = {*reinterpret_cast<const uint2*>(
          lds + SCB + (((cl >> 6) * BN + pl) * 16) + ((cl & 63) >> 2))};
      epilogue_idj_pk<1>(a, lds, one, sc, rbl, h, co0, pl, otile, orow);
    }
  }
  __syncthreads();
  const int npx = a.m - p0 < bn ? a.m - p0 : bn;
  copy_out_tile(a, otile, orow, co0, BM, p0, npx);
}

// ---------------------------------------------------------------------------
// Variants and planning
// ---------------------------------------------------------------------------
struct W2Variant {
  int wm, wn, wk, fm, fn, t, d, occ, winb;
  bool f4;
  double c0_us;        // fixed cost per round of occ workgroups on a CU
  double cj_us;        // more per round with a join epilogue
  double cs_us;        // cost of one weight stage (T taps of the tile's MFMAs)
  const char* thr_name;   // the kernels as a profiler lists them: threshold
  const char* idj_name;   // epilogue, identity join, fused downsample join
  const char* fused_name;
};

#define IFQ_W2_NAME(wm, wn, wk, fm, fn, t, d, mode, f4, occ, winb)                          \
  "conv_w2<" #wm ", " #wn ", " #wk ", " #fm ", " #fn ", " #t ", " #d ", " #mode ", " #f4 ", " \
  #occ ", " #winb ">"
#define IFQ_W2_NAMES(wm, wn, wk, fm, fn, t, d, f4, occ, winb)      \
  IFQ_W2_NAME(wm, wn, wk, fm, fn, t, d, 0, f4, occ, winb),         \
      IFQ_W2_NAME(wm, wn, wk, fm, fn, t, d, 1, f4, occ, winb),     \
      IFQ_W2_NAME(wm, wn, wk, fm, fn, t, d, 2, f4, occ, winb)

// Index order must match the switch in launch_conv_w2.
// (c0_us, cj_us, cs_us) are least-squares fits to kernel times measured on
// MI355X for every variant on every 3x3 layer of the ResNet-18, AlexNet,
// VGG-16 and Tiny-YOLOv2 stacks it takes (rms error 2-4%, 7% for the
// one-tap-stage tiles): a stage's cost holds its MFMAs at the efficiency the
// tile reaches and the barrier and DMA issue that bracket it.
const W2Variant kW2Variants[] = {
    {2, 4, 1, 2, 2, 3, 3, 1, 49152, false, 4.14, 0.75, 0.927, IFQ_W2_NAMES(2, 4, 1, 2, 2, 3, 3, false, 1, 49152)},
    {1, 4, 2, 2, 2, 3, 2, 1, 53248, false, 3.64, 0.68, 0.919, IFQ_W2_NAMES(1, 4, 2, 2, 2, 3, 2, false, 1, 53248)},
    {1, 2, 4, 2, 2, 3, 2, 1, 36864, false, 4.05, 0.75, 0.917, IFQ_W2_NAMES(1, 2, 4, 2, 2, 3, 2, false, 1, 36864)},
    {1, 4, 1, 2, 2, 3, 3, 2, 20480, false, 3.46, 1.71, 0.457, IFQ_W2_NAMES(1, 4, 1, 2, 2, 3, 3, false, 2, 20480)},
    {1, 8, 1, 2, 1, 3, 3, 2, 20480, false, 3.52, 0.90, 0.477, IFQ_W2_NAMES(1, 8, 1, 2, 1, 3, 3, false, 2, 20480)},
    {2, 4, 1, 2, 2, 1, 3, 2, 24576, false, 3.33, 2.11, 0.298, IFQ_W2_NAMES(2, 4, 1, 2, 2, 1, 3, false, 2, 24576)},
    // the same tiles on the fp4 scaled MFMA (half the weight bytes per K64
    // step: a stage holds three times the taps)
    {2, 4, 1, 2, 2, 9, 2, 1, 49152, true, 3.68, 1.14, 1.656, IFQ_W2_NAMES(2, 4, 1, 2, 2, 9, 2, true, 1, 49152)},
    {1, 4, 2, 2, 2, 9, 2, 1, 53248, true, 3.84, 0.62, 1.645, IFQ_W2_NAMES(1, 4, 2, 2, 2, 9, 2, true, 1, 53248)},
    {1, 2, 4, 2, 2, 3, 2, 1, 36864, true, 3.91, 0.70, 0.569, IFQ_W2_NAMES(1, 2, 4, 2, 2, 3, 2, true, 1, 36864)},
    {1, 4, 1, 2, 2, 9, 2, 2, 20480, true, 3.60, 1.59, 0.782, IFQ_W2_NAMES(1, 4, 1, 2, 2, 9, 2, true, 2, 20480)},
};
constexpr int kNumW2 = sizeof(kW2Variants) / sizeof(kW2Variants[0]);
constexpr int kW2CUs = 256;
// K split across workgroups: at most 4 ways; per round of a split tile, the
// partial's write, fence and arrival, and each other partial the last
// arrival adds. Measured on MI355X (Tiny-YOLOv2 c7, 13x13x512 -> 512 at
// batch 8, split 2 on 2 x 88 workgroups): 26-30 us against 11.5 us
// unsplit. The device-scope fence that publishes a partial is an L2
// write-back of the whole XCD's L2, one per workgroup, and those serialise;
// so the fixed cost below keeps the planner from splitting any layer of
// the benchmark stacks, and ifq_conv_forward_split runs it on request.
constexpr int kW2MaxSplit = 4;
constexpr double kW2SplitUs = 19.0;
constexpr double kW2SplitAddUs = 0.3;

// The epilogues this kernel has: 2-bit codes with the packed 16-bit compares
// (sums and thresholds below 2^15), no pool, and either thresholds or an
// identity join with a 2-bit shortcut.
bool w2_mode_ok(const ConvLaunch& a) {
  if (!(a.out_mode == 2 && a.rec == 4 && (a.cout & 31) == 0 && 27 * a.cin <= 32766 &&
        a.pool_k == 0))
    return false;
  if (a.join_kind == IFQ_JOIN_NONE) return true;
  // identity join: the shortcut is prefetched as whole 16-byte cells
  if (a.join_kind == IFQ_JOIN_IDENTITY)
    return a.cout % 64 == 0 &&
           (a.sc_layout == IFQ_LAYOUT_U2_BLOCK64 || a.sc_layout == IFQ_LAYOUT_U2_NHWC_PACKED);
  // downsample join: 1x1 conv on BLOCK64 codes with at most 4 channel blocks
  return a.join_kind == IFQ_JOIN_CONV_FUSED && a.sc_layout == IFQ_LAYOUT_U2_BLOCK64 &&
         a.d_cin % 64 == 0 && a.d_cin / 64 <= 4 &&
         (int64_t)a.n * a.d_h * a.d_w * (a.d_cin / 64) < (int64_t)1 << 26;
}

// Pixels per workgroup and the predicted time of variant v on layer a, or
// false if v cannot take it.
bool w2_fit(const ConvLaunch& a, int v, W2Plan* out, int want_split) {
  const W2Variant& V = kW2Variants[v];
  if (V.f4 != (a.f4 != 0)) return false;
  const int G = a.cin / 64;
  if (G % V.wk) return false;
  // the downsample's weights fit one stage; the two-per-CU eight-wave tiles'
  // join instance needs more than their 128 VGPRs
  if (a.join_kind == IFQ_JOIN_CONV_FUSED &&
      (a.d_cin / 64 > V.wk * V.t || (V.occ == 2 && V.wm * V.wn * V.wk == 8 && V.fn == 2)))
    return false;
  const int bm = 32 * V.fm * V.wm, bnmax = 32 * V.fn * V.wn;
  const int64_t nco = (a.cout + bm - 1) / bm;
  const int64_t nb_min = (a.m + bnmax - 1) / bnmax;
  // per K split S (S workgroups per tile, each over 1/S of the channel
  // blocks): pixel tiles sized so that the S * tiles workgroups fill whole
  // rounds of occ per CU; the busiest CU's rounds and weight stages (the
  // fused downsample's weights are one more stage), and for S > 1 the
  // partial tile's round trip through the workspace per round
  const double c_round = V.c0_us + (a.join_kind != IFQ_JOIN_NONE ? V.cj_us : 0.0);
  W2Plan best{};
  bool have = false;
  for (int S = 1; S <= kW2MaxSplit; S *= 2) {
    if (S > 1 && !(a.split_ok && a.join_kind == IFQ_JOIN_NONE && !V.f4 && G % (S * V.wk) == 0))
      break;
    if (want_split > 0 && S != want_split) continue;
    const int64_t slots = (int64_t)kW2CUs * V.occ / S;
    const int64_t rounds = (nco * nb_min + slots - 1) / slots;
    int64_t nb = rounds * slots / nco;
    if (nb < nb_min) nb = nb_min;
    int64_t bn = (a.m + nb - 1) / nb;
    bn = (bn + 31) / 32 * 32;
    if (bn > bnmax) bn = bnmax;
    // a workgroup holds the windows of its own G / S channel blocks
    const int64_t gs = G / S;
    const int64_t cells = window_cells_max(a, bn, (int64_t)V.winb / 16 / gs);
    if (cells < 0 || gs * (cells + 1) * 16 > V.winb) continue;
    const int64_t blocks = nco * ((a.m + bn - 1) / bn);
    if (S > 1 && blocks > kSplitMaxTiles) continue;
    const int64_t wgs = blocks * S;
    const int64_t per_cu = (wgs + kW2CUs - 1) / kW2CUs;
    const int64_t cu_rounds = (per_cu + V.occ - 1) / V.occ;
    const int64_t stages =
        (G / S / V.wk) * (kW2Taps / V.t) + (a.join_kind == IFQ_JOIN_CONV_FUSED);
    const double split_us = S > 1 ? kW2SplitUs + kW2SplitAddUs * (S - 1) : 0.0;
    const double t = kLaunchUs + (double)cu_rounds * (c_round + split_us) +
                     (double)(per_cu * stages) * V.cs_us;
    if (!have || t < best.t_us) {
      best = W2Plan{v, (int)bn, (int)((a.m + bn - 1) / bn), (int)cells, t, S};
      have = true;
    }
  }
  if (!have) return false;
  *out = best;
  return true;
}

}  // namespace

int w2_variant_count() { return kNumW2; }

int64_t w2_split_bytes(const ConvLaunch& a, const W2Plan& p) {
  if (p.ksplit <= 1) return 0;
  const W2Variant& V = kW2Variants[p.variant];
  const int64_t bm = 32 * V.fm * V.wm, bn = 32 * V.fn * V.wn;
  const int64_t tiles = (int64_t)p.blocks_m * ((a.cout + bm - 1) / bm);
  return kSplitCounterBytes + tiles * p.ksplit * bm * bn * 4;
}
bool w2_variant_fp4(int v) { return v >= 0 && v < kNumW2 && kW2Variants[v].f4; }

bool plan_w2(const ConvLaunch& a, int forced, W2Plan* out, int want_split) {
  if (!(a.in_layout == IFQ_LAYOUT_U2_BLOCK64 && a.in_bits == 2 && a.cin % 64 == 0 &&
        a.kh == 3 && a.kw == 3 && a.pad == 1 && (a.stride == 1 || a.stride == 2) && a.m > 0))
    return false;
  if (!w2_mode_ok(a)) return false;
  // 32-bit cell indices and offsets
  if ((int64_t)a.n * a.h * a.w * (a.cin / 64) >= (int64_t)1 << 26) return false;
  if (forced >= 0) return forced < kNumW2 && w2_fit(a, forced, out, want_split);
  bool found = false;
  for (int v = 0; v < kNumW2; ++v) {
    W2Plan p;
    if (w2_fit(a, v, &p, want_split) && (!found || p.t_us < out->t_us)) {
      *out = p;
      found = true;
    }
  }
  return found;
}

const char* conv_w2_name(const W2Plan& p, const ConvLaunch& a) {
  const W2Variant& V = kW2Variants[p.variant];
  return a.join_kind == IFQ_JOIN_IDENTITY    ? V.idj_name
         : a.join_kind == IFQ_JOIN_CONV_FUSED ? V.fused_name
                                              : V.thr_name;
}

hipError_t launch_conv_w2(ConvLaunch a, const W2Plan& p, hipStream_t stream) {
  a.bn = p.bn;
  a.wcells = p.wcells;
  const W2Variant& V = kW2Variants[p.variant];
  const int bm = 32 * V.fm * V.wm;
  a.ksplit = p.ksplit > 1 ? p.ksplit : 1;
  if (a.ksplit > 1) {
    if (!a.ws_cnt) return hipErrorInvalidValue;   // the caller's workspace
    a.ws_part = reinterpret_cast<int32_t*>(reinterpret_cast<uint8_t*>(a.ws_cnt) +
                                           kSplitCounterBytes);
  }
  const dim3 grid(p.blocks_m, (a.cout + bm - 1) / bm, a.ksplit);
  const dim3 block(64 * V.wm * V.wn * V.wk);
  const int mode = a.ksplit > 1                            ? 3
                   : a.join_kind == IFQ_JOIN_IDENTITY    ? 1
                   : a.join_kind == IFQ_JOIN_CONV_FUSED ? 2
                                                         : 0;
  switch (p.variant * 4 + mode) {
// the K-split instances (int8 variants only)
#define IFQ_W2_SPLIT(k, wm, wn, wk, fm, fn, t, d, f4, occ, winb)                                \
  case 4 * k + 3:                                                                               \
    hipLaunchKernelGGL((conv_w2<wm, wn, wk, fm, fn, t, d, 3, f4, occ, winb>), grid, block, 0,   \
                       stream, a);                                                              \
    break;
#define IFQ_W2_CASE(k, wm, wn, wk, fm, fn, t, d, f4, occ, winb)                                 \
  case 4 * k:                                                                                   \
    hipLaunchKernelGGL((conv_w2<wm, wn, wk, fm, fn, t, d, 0, f4, occ, winb>), grid, block, 0,   \
                       stream, a);                                                              \
    break;                                                                                      \
  case 4 * k + 1:                                                                               \
    hipLaunchKernelGGL((conv_w2<wm, wn, wk, fm, fn, t, d, 1, f4, occ, winb>), grid, block, 0,   \
                       stream, a);                                                              \
    break;                                                                                      \
  case 4 * k + 2:                                                                               \
    hipLaunchKernelGGL((conv_w2<wm, wn, wk, fm, fn, t, d, 2, f4, occ, winb>), grid, block, 0,   \
                       stream, a);                                                              \
    break;
    IFQ_W2_SPLIT(0, 2, 4, 1, 2, 2, 3, 3, false, 1, 49152)
    IFQ_W2_SPLIT(1, 1, 4, 2, 2, 2, 3, 2, false, 1, 53248)
    IFQ_W2_SPLIT(2, 1, 2, 4, 2, 2, 3, 2, false, 1, 36864)
    IFQ_W2_SPLIT(3, 1, 4, 1, 2, 2, 3, 3, false, 2, 20480)
    IFQ_W2_SPLIT(4, 1, 8, 1, 2, 1, 3, 3, false, 2, 20480)
    IFQ_W2_SPLIT(5, 2, 4, 1, 2, 2, 1, 3, false, 2, 24576)
    IFQ_W2_CASE(0, 2, 4, 1, 2, 2, 3, 3, false, 1, 49152)
    IFQ_W2_CASE(1, 1, 4, 2, 2, 2, 3, 2, false, 1, 53248)
    IFQ_W2_CASE(2, 1, 2, 4, 2, 2, 3, 2, false, 1, 36864)
    IFQ_W2_CASE(3, 1, 4, 1, 2, 2, 3, 3, false, 2, 20480)
    IFQ_W2_CASE(4, 1, 8, 1, 2, 1, 3, 3, false, 2, 20480)
    IFQ_W2_CASE(5, 2, 4, 1, 2, 2, 1, 3, false, 2, 24576)
    IFQ_W2_CASE(6, 2, 4, 1, 2, 2, 9, 2, true, 1, 49152)
    IFQ_W2_CASE(7, 1, 4, 2, 2, 2, 9, 2, true, 1, 53248)
    IFQ_W2_CASE(8, 1, 2, 4, 2, 2, 3, 2, true, 1, 36864)
    IFQ_W2_CASE(9, 1, 4, 1, 2, 2, 9, 2, true, 2, 20480)
#undef IFQ_W2_CASE
#undef IFQ_W2_SPLIT
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace ifq
