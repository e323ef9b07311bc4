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
  int ncg;         // register-pooled epilogues: groups of pooled columns per
  FastDiv div_ncg; // row pair (4 in small8, 8 in small2), the division by it
  FastDiv div_phowo;  // small2: division by pho * pwo (pooled copy-out)
};

__host__ __device__ inline int small_orow(const ConvLaunch& a, int bm) {
  return a.out_mode == 2 ? bm / 4 : bm;
}

// EPI: the epilogue, fixed per launch by small8_epi: 0 the generic one
// through the LDS output tile, 1 the register epilogue of 2-bit codes
// stored straight to HBM, 2 the register epilogue into the LDS tile for the
// fused pool, 3 a 2x2/2 max-pool taken on the sums in registers before the
// threshold compare.
//
// EPI 3. The code #{i : s*a > T_i} does not decrease as s*a grows, so the
// largest code of a window is the code of the window's largest s*a (the
// order of Eq. 4 and Eq. 7 swapped: pool the sums, max where s = +1 and min
// where s = -1). Rows of the weights with s = -1 are negated in registers,
// which makes every sum s*a and the pool a plain max. A 16-pixel block is
// four 2x2 windows, the four pixels of a window in one lane quad; four
// blocks are in flight, and two DPP exchanges inside each quad leave lane e
// of a quad with block e's pooled window (a reduce-scatter), so the compare
// and packing run once per pooled pixel instead of once per pixel.
template <int FM, int EPI>
__global__ __launch_bounds__(kSmallThreads) void conv_small8(ConvLaunch a, SmallGeom sg) {
  constexpr int BM = 16 * FM;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int kg = lane >> 4;     // K bytes 16*kg .. 16*kg+15: taps 4*kg .. 4*kg+3
  const int l16 = lane & 15;

  const int nimg = blockIdx.x / sg.tiles;
  const int oy0 = (blockIdx.x - nimg * sg.tiles) * sg.rows;
  const int rows = a.ho - oy0 < sg.rows ? a.ho - oy0 : sg.rows;
  const int npx = rows * a.wo;
  const int p0 = (nimg * a.ho + oy0) * a.wo;
  const int st = a.stride;
  const int ntaps = a.kh * a.kw;
  constexpr bool fast = EPI != 0;

  // ---- operands kept in registers, loaded before the input rows so that
  // their latency overlaps the staging loads: from clamped addresses, the
  // lanes out of range masked afterwards. A lane group's 4*c_in weight bytes
  // (taps 4*kg .. 4*kg+3) are one 4-aligned span of its row, inside the row's
  // kpad >= 64 bytes.
  uint32_t wraw[FM][4];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const int co = fm * 16 + l16;
    const int coc = co < a.cout_pad ? co : a.cout_pad - 1;
    const uint32_t* wr =
        reinterpret_cast<const uint32_t*>(a.wgt + (int64_t)coc * a.kpad + 4 * kg * a.cin);
#pragma unroll
    for (int d = 0; d < 4; ++d) wraw[fm][d] = wr[d];
  }
  int asgn[FM];   // EPI 3: s of the lane's weight row fm*16 + l16
  if constexpr (EPI == 3) {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int co = fm * 16 + l16;
      asgn[fm] = a.thr[(int64_t)(co < a.cout ? co : a.cout - 1) * 4];
    }
  }
  int4 rrec[FM][4];
  int rsum[FM][4];
  if constexpr (fast) {
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int co = fm * 16 + 4 * kg + i;
        const int coc = co < a.cout ? co : a.cout - 1;
        rrec[fm][i] = *reinterpret_cast<const int4*>(a.thr + (int64_t)coc * 4);
        rsum[fm][i] = a.rowsum[coc];
      }
  }

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
      // unconditional loads and stores at clamped indices (the lanes past the
      // end store the last cell's value again), so that every load of a
      // batch is in flight before the first store waits
      auto batch = [&](int i0) {
        uint4 v[VB];
#pragma unroll
        for (int k = 0; k < VB; ++k) {
          const int i = i0 + k * kSmallThreads + tid;
          v[k] = src[i < nfull ? i : nfull - 1];
        }
#pragma unroll
        for (int k = 0; k < VB; ++k) {
          const int i = i0 + k * kSmallThreads + tid;
          reinterpret_cast<uint4*>(raw)[i < nfull ? i : nfull - 1] = v[k];
        }
      };
      if (nfull > 0) batch(0);   // outside the loop: no loop-header wait
      for (int i0 = VB * kSmallThreads; i0 < nfull; i0 += VB * kSmallThreads) batch(i0);
      for (int i = nfull * 16 + tid; i < nb; i += kSmallThreads) raw[i] = a.x[gs16 + i];
    }
    __syncthreads();
    // a pixel's c_in bytes from the two aligned words that hold them (the
    // raw buffer has 16 bytes of slack past its end), the channels past c_in
    // masked to the zero code
    const uint32_t keep = a.cin >= 4 ? 0xFFFFFFFFu : (1u << (8 * a.cin)) - 1u;
    // EB pixels per thread and pass, their LDS reads all issued before the
    // first is used (positions outside the image read byte 0 and are masked)
    constexpr int EB = 4;
    for (int e0 = tid; e0 < nin; e0 += EB * kSmallThreads) {
      uint32_t lo[EB], hi[EB];
      int sh[EB];
      bool in[EB];
#pragma unroll
      for (int k = 0; k < EB; ++k) {
        const int e = e0 + k * kSmallThreads;
        const int r = fdiv(e, sg.div_win);
        const int iy = iy0 + r, ix = e - r * sg.win - a.pad;
        in[k] = e < nin && (unsigned)iy < (unsigned)a.h && (unsigned)ix < (unsigned)a.w;
        const int b = in[k] ? lead + ((iy - iy_lo) * a.w + ix) * a.cin : 0;
        const uint32_t* w32 = reinterpret_cast<const uint32_t*>(raw + (b & ~3));
        lo[k] = w32[0];
        hi[k] = w32[1];
        sh[k] = b & 3;
      }
#pragma unroll
      for (int k = 0; k < EB; ++k) {
        const int e = e0 + k * kSmallThreads;
        const uint32_t v = __builtin_amdgcn_alignbyte(hi[k], lo[k], (uint32_t)sh[k]) & keep;
        if (e < nin) *reinterpret_cast<uint32_t*>(tile + e * 4) = 0x80808080u ^ (in[k] ? v : 0u);
      }
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
  if (!fast) stage_epilogue(a, lds, 0, BM);

  // ---- weight fragments (A: rows = output channels), K byte 4*j + c of
  // lane group kg = channel c of tap 4*kg + j: tap j's c_in bytes start at
  // byte j*c_in of the lane group's span -------------------------------------
  v4i af[FM];
  const uint32_t keep = a.cin >= 4 ? 0xFFFFFFFFu : (1u << (8 * a.cin)) - 1u;
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) {
    const bool row_ok = fm * 16 + l16 < a.cout_pad;
    uint32_t w4[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int o = j * a.cin, q = o >> 2;
      const uint32_t lo = q == 0 ? wraw[fm][0] : q == 1 ? wraw[fm][1] : q == 2 ? wraw[fm][2] : wraw[fm][3];
      const uint32_t hi = q == 0 ? wraw[fm][1] : q == 1 ? wraw[fm][2] : q == 2 ? wraw[fm][3] : 0u;
      const uint32_t v = __builtin_amdgcn_alignbyte(hi, lo, (uint32_t)(o & 3)) & keep;
      w4[j] = (row_ok && 4 * kg + j < ntaps) ? v : 0u;
      if (EPI == 3 && asgn[fm] < 0) {   // bytes in {-1, 0, 1}: negate each
        uint32_t nv = 0;
#pragma unroll
        for (int b = 0; b < 4; ++b)
          nv |= (uint32_t)(uint8_t)(-(int8_t)(w4[j] >> (8 * b))) << (8 * b);
        w4[j] = nv;
      }
    }
    af[fm] = v4i{(int)w4[0], (int)w4[1], (int)w4[2], (int)w4[3]};
  }
  // LDS byte offsets of this lane's four taps from a pixel's window corner
  // (taps past kh*kw read the corner: their weights are zero)
  int toff[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int tap = 4 * kg + j;
    const bool valid = tap < ntaps;
    const int ty = valid ? tap / a.kw : 0, tx = valid ? tap - ty * a.kw : 0;
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
        r = rrec[fm][i];
        corr[fm][i] = 128 * rsum[fm][i];
      }
      const bool flip = r.x < 0;
      const int tt[3] = {r.y, r.z, r.w};
      if constexpr (EPI == 3) {
        // the sums are s*a - s*128*rowsum (negated rows): compare them with
        // T - s*128*rowsum; |sum| <= 128*64, so the clamp keeps every answer
        if (flip) corr[fm][i] = -corr[fm][i];
#pragma unroll
        for (int k = 0; k < 3; ++k) {
          int64_t v = (int64_t)tt[k] - corr[fm][i];
          v = v > 32767 ? 32767 : v < -32768 ? -32768 : v;
          t16[i][k] = (uint32_t)v & 0xFFFFu;
        }
      } else {
#pragma unroll
        for (int k = 0; k < 3; ++k) {
          int v = flip ? -tt[k] - 1 : tt[k];
          v = v > 32767 ? 32767 : v < -32768 ? -32768 : v;   // |sum| < 2^15 anyway
          t16[i][k] = (uint32_t)v & 0xFFFFu;
        }
        if (flip) txm[fm] |= 3u << ((i & 1) * 16 + (i >> 1) * 4);
      }
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
  const bool pooled = EPI == 2 || (EPI == 0 && a.pool_k > 0);
  uint8_t* y8 = reinterpret_cast<uint8_t*>(a.y);
  const int nblk = (npx + 15) / 16;
  // UB independent blocks of 16 pixels per iteration, so the LDS reads, the
  // MFMAs and the epilogues of different blocks overlap (one block at a time
  // past 32 output channels, where four would not fit the registers)
  constexpr int UB = FM <= 2 ? 4 : 1;
  constexpr int NW = kSmallThreads / 64;
  if constexpr (EPI == 3) {
    static_assert(FM <= 2, "four blocks in flight");
    // block b: row pair b / ncg, pooled columns 4*(b % ncg) .. +3; lane
    // l16 = 4*w + e: window w, pixel (e >> 1, e & 1) of it
    const int w = l16 >> 2, e = l16 & 3;
    const int pwo = a.wo >> 1;
    const int nb3 = (rows >> 1) * sg.ncg;
    const int prow = pwo * orow;   // pooled tile bytes per row pair
    // the lane's fixed offset inside a block: pixel (e >> 1, e & 1) of
    // window w (columns 2w, 2w + 1 of the block's 8)
    const int lane_off = ((e >> 1) * st * sg.win + (2 * w + (e & 1)) * st) * 4;
    const int last_off = ((e >> 1) * st * sg.win + (2 * (pwo - 1) + (e & 1)) * st) * 4;
    for (int blk0 = wave; blk0 < nb3; blk0 += NW * 4) {
      v4i accu[4][FM];
      int rps[4], cgs[4];   // wave-uniform block coordinates (scalar)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int b = blk0 + NW * u;
        const int bc = b < nb3 ? b : nb3 - 1;
        rps[u] = fdiv(bc, sg.div_ncg);
        cgs[u] = bc - rps[u] * sg.ncg;
        // window w of the block's group, or the row's last window past pwo
        const int pc = 4 * cgs[u] + w;
        const int base = (2 * rps[u] * st * sg.win + 8 * cgs[u] * st) * 4;
        const uint8_t* win =
            tile + (pc < pwo ? base + lane_off : (2 * rps[u] * st * sg.win) * 4 + last_off);
        uint32_t b4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) b4[j] = *reinterpret_cast<const uint32_t*>(win + toff[j]);
        const v4i bf = v4i{(int)b4[0], (int)b4[1], (int)b4[2], (int)b4[3]};
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
          accu[u][fm] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[fm], bf, v4i{0, 0, 0, 0}, 0, 0, 0);
      }   // (a pooled launch carries no sum dump)
      // int16 pairs (|sum| <= 128*64), then the reduce-scatter over the quad
      s16x2 pk[4][FM][2];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int fm = 0; fm < FM; ++fm) {
          pk[u][fm][0] = __builtin_amdgcn_cvt_pk_i16(accu[u][fm][0], accu[u][fm][1]);
          pk[u][fm][1] = __builtin_amdgcn_cvt_pk_i16(accu[u][fm][2], accu[u][fm][3]);
        }
      const bool odd = (e & 1) != 0, high = (e & 2) != 0;
      auto xchg = [](s16x2 v, int ctrl) {
        const int iv = __builtin_bit_cast(int, v);
        const int r = ctrl == 0xB1 ? __builtin_amdgcn_mov_dpp(iv, 0xB1, 0xF, 0xF, false)
                                   : __builtin_amdgcn_mov_dpp(iv, 0x4E, 0xF, 0xF, false);
        return __builtin_bit_cast(s16x2, r);
      };
      s16x2 red[FM][2];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          // lanes e ^ 1: the even lane keeps blocks 0, 2, the odd lane 1, 3
          s16x2 k1[2];
#pragma unroll
          for (int j = 0; j < 2; ++j) {
            const s16x2 send = odd ? pk[2 * j][fm][hf] : pk[2 * j + 1][fm][hf];
            const s16x2 keep = odd ? pk[2 * j + 1][fm][hf] : pk[2 * j][fm][hf];
            k1[j] = __builtin_elementwise_max(keep, xchg(send, 0xB1));
          }
          // lanes e ^ 2: lane e keeps block e
          const s16x2 send = high ? k1[0] : k1[1];
          const s16x2 keep = high ? k1[1] : k1[0];
          red[fm][hf] = __builtin_elementwise_max(keep, xchg(send, 0x4E));
        }
      // lane e: block blk0 + NW*e, pooled pixel (row pair, 4*group + w)
      const int be = blk0 + NW * e;
      const int rpe = e == 0 ? rps[0] : e == 1 ? rps[1] : e == 2 ? rps[2] : rps[3];
      const int pce = 4 * (e == 0 ? cgs[0] : e == 1 ? cgs[1] : e == 2 ? cgs[2] : cgs[3]) + w;
      const bool store = be < nb3 && pce < pwo;
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) {
        const uint32_t c01 = count3_pk(red[fm][0], tw[fm][0][0], tw[fm][0][1], tw[fm][0][2]);
        const uint32_t c23 = count3_pk(red[fm][1], tw[fm][1][0], tw[fm][1][1], tw[fm][1][2]);
        const uint32_t t = c01 | (c23 << 4);
        if (store) otile[rpe * prow + pce * orow + fm * 4 + kg] = (uint8_t)(t | (t >> 14));
      }
    }
  } else
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
        b4[j] = *reinterpret_cast<const uint32_t*>(win + toff[j]);
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
  if constexpr (EPI == 3) {
    // the pooled rows are one contiguous span of the packed NHWC output
    // (c_out == BM, 4-byte rows of 16 channels)
    __syncthreads();
    const int nw = (rows >> 1) * (a.wo >> 1) * orow / 4;
    const int64_t pp0 = ((int64_t)nimg * a.pho + (oy0 >> 1)) * a.pwo;
    uint32_t* dst = reinterpret_cast<uint32_t*>(y8 + pp0 * orow);
    const uint32_t* srcw = reinterpret_cast<const uint32_t*>(otile);
    for (int i = tid; i < nw; i += kSmallThreads) dst[i] = srcw[i];
  } else if (!fast || pooled) {
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
    // 16 bytes of alignment lead plus 8 of slack for the two-word pixel reads
    const int64_t rawb = ((int64_t)rin * a.w * a.cin + 24 + 15) & ~(int64_t)15;
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
      g->ncg = ((a.wo >> 1) + 3) / 4;
      g->div_ncg = make_fastdiv((uint32_t)(g->ncg > 0 ? g->ncg : 1));
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
// RP: the 2x2/2 max-pool taken on the sums in registers, as in conv_small8's
// EPI 3: weight rows with s = -1 negated, a 32-pixel block is eight 2x2
// windows (lane l32 = 4*w + e), UB blocks in flight, a reduce-scatter over
// each lane quad (UB = 4: lane e ends with block e; UB = 2: a scatter over
// e ^ 1 and a butterfly over e ^ 2), and the compare once per pooled pixel.
template <int FM, int CIN, bool RP>
__global__ __launch_bounds__(kSmallThreads) void conv_small2(ConvLaunch a, SmallGeom sg) {
  constexpr int BM = 32 * FM;
  constexpr int KS = (9 * CIN + 31) / 32;        // K32 steps
  constexpr int BPP = CIN / 4;                   // bytes per packed pixel (4 or 8)
  constexpr int WPP = CIN / 16;                  // 32-bit words per pixel (1 or 2)
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int h = lane >> 5;
  const int l32 = lane & 31;

  const int nimg = blockIdx.x / sg.tiles;
  const int oy0 = (blockIdx.x - nimg * sg.tiles) * sg.rows;
  const int rows = a.ho - oy0 < sg.rows ? a.ho - oy0 : sg.rows;
  const int npx = rows * a.wo;
  const int p0 = (nimg * a.ho + oy0) * a.wo;

  // ---- weight fragments and threshold records into registers first, so
  // that their latency overlaps the staging loads (clamped addresses; rows
  // past cout_pad are zeroed once loaded, records past c_out never used) ----
  v4i af[KS][FM];
#pragma unroll
  for (int s = 0; s < KS; ++s)
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int row = fm * 32 + l32;
      const int rowc = row < a.cout_pad ? row : a.cout_pad - 1;
      af[s][fm] = *reinterpret_cast<const v4i*>(a.wgt + (int64_t)rowc * a.kpad + 32 * s + 16 * h);
    }
  int4 rrec[4];
  if (tid < BM / 4) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int c = 4 * tid + i;
      const int cc = c < a.cout ? c : a.cout - 1;
      rrec[i] = *reinterpret_cast<const int4*>(a.thr + (int64_t)cc * 4);
    }
  }

  // ---- stage the input rows (1 or 2 words per pixel) ------------------------
  uint32_t* tile = reinterpret_cast<uint32_t*>(lds + sg.in_off);
  const int iy0 = oy0 - 1;
  const int nwords = sg.rin * sg.win * WPP;
  const uint32_t* x32 = reinterpret_cast<const uint32_t*>(a.x);
  constexpr int SB = 8;
  auto stage = [&](int e0) {
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
  };
  // the first batch outside the loop: a loop header would wait for every
  // load in flight, the register operands' included
  stage(0);
  for (int e0 = SB * kSmallThreads; e0 < nwords; e0 += SB * kSmallThreads) stage(e0);
  // ---- threshold records (stage_thr_pk's layout; channels past c_out get
  // records whose codes are never stored) and weight fragments --------------
  if (tid < BM / 4) {
    uint32_t w[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      // opaque here, so that no use of the record moves above the staging
      asm volatile("" : "+v"(rrec[i].x), "+v"(rrec[i].y), "+v"(rrec[i].z), "+v"(rrec[i].w));
      const int4 r = rrec[i];
      const bool flip = !RP && r.x < 0;   // RP: the sums are s*a already
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
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
    if (fm * 32 + l32 >= a.cout_pad)
#pragma unroll
      for (int s = 0; s < KS; ++s) af[s][fm] = v4i{0, 0, 0, 0};
  if constexpr (RP) {
    // s of the lane's weight row: rows with s = -1 negated (bytes in {-1, 0, 1})
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int row = fm * 32 + l32;
      if (row < a.cout && a.thr[(int64_t)row * 4] < 0)
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const uint32_t w4 = (uint32_t)af[s][fm][k];
            uint32_t nv = 0;
#pragma unroll
            for (int b = 0; b < 4; ++b)
              nv |= (uint32_t)(uint8_t)(-(int8_t)(w4 >> (8 * b))) << (8 * b);
            af[s][fm][k] = (int)nv;
          }
    }
  }
  // LDS byte offset of this lane's word of K step s from a pixel's window
  // corner (K past 9*c_in reads the corner: its weights are zero)
  int toff[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int k0 = 32 * s + 16 * h;
    const int tap = k0 / CIN, c0 = k0 - tap * CIN;
    const int ty = tap / 3, tx = tap - ty * 3;
    toff[s] = tap < 9 ? ((ty * sg.win + tx) * BPP + (c0 >> 2)) : 0;
  }
  __syncthreads();

  const int orow = small_orow(a, BM);
  uint8_t* otile = lds + sg.out_off;
  const int nblk = (npx + 31) / 32;
  constexpr int NW = kSmallThreads / 64;
  if constexpr (RP) {
    constexpr int UB = FM == 1 ? 4 : 2;
    const int w = l32 >> 2, e = l32 & 3;
    const int pwo = a.wo >> 1;
    const int nb = (rows >> 1) * sg.ncg;
    const int prow = pwo * orow;
    auto xchg = [](s16x2 v, int ctrl) {
      const int iv = __builtin_bit_cast(int, v);
      const int r = ctrl == 0xB1 ? __builtin_amdgcn_mov_dpp(iv, 0xB1, 0xF, 0xF, false)
                                 : __builtin_amdgcn_mov_dpp(iv, 0x4E, 0xF, 0xF, false);
      return __builtin_bit_cast(s16x2, r);
    };
    for (int blk0 = wave; blk0 < nb; blk0 += NW * UB) {
      s16x2 pk[UB][FM][8];
#pragma unroll
      for (int u = 0; u < UB; ++u) {
        const int b = blk0 + NW * u;
        const int bc = b < nb ? b : nb - 1;
        const int rp = fdiv(bc, sg.div_ncg);
        const int pc = 8 * (bc - rp * sg.ncg) + w;
        const int pcc = pc < pwo ? pc : pwo - 1;
        const int r = 2 * rp + (e >> 1), ox = 2 * pcc + (e & 1);
        const uint8_t* win = lds + sg.in_off + (r * sg.win + ox) * BPP;
        v16i acc[FM];
#pragma unroll
        for (int fm = 0; fm < FM; ++fm) acc[fm] = v16i{0};
        uint32_t uw[KS];
#pragma unroll
        for (int s = 0; s < KS; ++s) uw[s] = *reinterpret_cast<const uint32_t*>(win + toff[s]);
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          const v4i bf = unpack2(uw[s]);
#pragma unroll
          for (int fm = 0; fm < FM; ++fm)
            acc[fm] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[s][fm], bf, acc[fm], 0, 0, 0);
        }
        // int16 pairs: |sum| <= 3 * 288
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
          for (int v2 = 0; v2 < 8; ++v2)
            pk[u][fm][v2] = __builtin_amdgcn_cvt_pk_i16(acc[fm][2 * v2], acc[fm][2 * v2 + 1]);
      }   // (a pooled launch carries no sum dump)
      const bool odd = (e & 1) != 0, high = (e & 2) != 0;
      s16x2 red[FM][8];
#pragma unroll
      for (int fm = 0; fm < FM; ++fm)
#pragma unroll
        for (int v2 = 0; v2 < 8; ++v2) {
          if constexpr (UB == 4) {
            s16x2 k1[2];
#pragma unroll
            for (int j = 0; j < 2; ++j) {
              const s16x2 send = odd ? pk[2 * j][fm][v2] : pk[2 * j + 1][fm][v2];
              const s16x2 keep = odd ? pk[2 * j + 1][fm][v2] : pk[2 * j][fm][v2];
              k1[j] = __builtin_elementwise_max(keep, xchg(send, 0xB1));
            }
            const s16x2 send = high ? k1[0] : k1[1];
            const s16x2 keep = high ? k1[1] : k1[0];
            red[fm][v2] = __builtin_elementwise_max(keep, xchg(send, 0x4E));
          } else {
            const s16x2 send = odd ? pk[0][fm][v2] : pk[1][fm][v2];
            const s16x2 keep = odd ? pk[1][fm][v2] : pk[0][fm][v2];
            const s16x2 k1 = __builtin_elementwise_max(keep, xchg(send, 0xB1));
            red[fm][v2] = __builtin_elementwise_max(k1, xchg(k1, 0x4E));
          }
        }
      // lane e: block blk0 + NW*ub (ub = e, or e & 1 for two blocks)
      const int ub = UB == 4 ? e : (e & 1);
      const int be = blk0 + NW * ub;
      const int bec = be < nb ? be : nb - 1;
      const int rpe = fdiv(bec, sg.div_ncg);
      const int pce = 8 * (bec - rpe * sg.ncg) + w;
      const bool store = be < nb && pce < pwo && (UB == 4 || e < 2);
#pragma unroll
      for (int fm = 0; fm < FM; ++fm) {
        if (fm * 32 >= a.cout) continue;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int cl = fm * 32 + 8 * b + 4 * h;
          const uint4* rec = reinterpret_cast<const uint4*>(lds + (cl >> 2) * kPkRecBytes);
          const uint4 r0 = rec[0], r1 = rec[1];
          const uint32_t c01 = count3_pk(red[fm][2 * b], r0.x, r0.y, r0.z);
          const uint32_t c23 = count3_pk(red[fm][2 * b + 1], r0.w, r1.x, r1.y);
          const uint32_t t = c01 | (c23 << 4);
          if (store) otile[rpe * prow + pce * orow + (cl >> 2)] = (uint8_t)(t | (t >> 14));
        }
      }
    }
    __syncthreads();
    // the pooled rows of the tile, as an output of pho x pwo pixels
    ConvLaunch ap = a;
    ap.ho = a.pho;
    ap.wo = a.pwo;
    ap.div_howo = sg.div_phowo;
    copy_out_tile(ap, otile, orow, 0, BM, (nimg * a.pho + (oy0 >> 1)) * a.pwo,
                  (rows >> 1) * a.pwo);
    return;
  }
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
      u[s] = *reinterpret_cast<const uint32_t*>(win + toff[s]);
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
      g->ncg = ((a.wo >> 1) + 7) / 8;
      g->div_ncg = make_fastdiv((uint32_t)(g->ncg > 0 ? g->ncg : 1));
      g->div_phowo = make_fastdiv((uint32_t)(a.pool_k ? (a.pho * a.pwo > 0 ? a.pho * a.pwo : 1) : 1));
      return true;
    }
  }
}

// ---------------------------------------------------------------------------
// 1x1 convolutions with int32 sums out and at most 64 output channels (a
// detector's head: c_in 512 -> 30 channels), on 2-bit codes in BLOCK64 or
// packed NHWC with c_in a multiple of 64. M is small (the head of Tiny-YOLOv2
// at batch 8 has 1352 pixels), so the kernel is built for latency: one wave
// per 32 pixels, no LDS and no barrier. Each lane loads its pixel's 16-byte
// cells (one per 64-channel block) and its A fragments (the weight blob's
// fragment order) straight into registers, all loads of a chunk of eight
// channel blocks in flight at once; K32 step 2g + t takes the 32-bit word
// 2h + t of cell g (the 16 channels 32h + 16t .. +15 the blob's K order puts
// in that half of the step) through unpack2, then v_mfma_i32_32x32x32_i8.
template <int FM>
__global__ __launch_bounds__(64, 1) void conv_head(ConvLaunch a) {
  constexpr int GC = 8;                            // channel blocks per chunk
  const int lane = threadIdx.x;
  const int h = lane >> 5;
  const int l32 = lane & 31;
  const int G = a.cin >> 6;
  const int nk32 = 2 * G;                          // kpad = c_in for 1x1
  const int p0 = blockIdx.x * 32;
  const int p = p0 + l32;
  const int pc = p < a.m ? p : a.m - 1;
  // byte offset of the pixel's cell g: g * gstride + cbase
  int64_t cbase, gstride;
  if (a.in_layout == IFQ_LAYOUT_U2_BLOCK64) {
    const int howo = a.h * a.w;
    const int n = fdiv(pc, a.div_howo);
    cbase = ((int64_t)n * G * howo + (pc - n * howo)) * 16;
    gstride = (int64_t)howo * 16;
  } else {
    cbase = (int64_t)pc * G * 16;
    gstride = 16;
  }
  const uint8_t* x8 = reinterpret_cast<const uint8_t*>(a.x);
  const uint8_t* w8 = reinterpret_cast<const uint8_t*>(a.wgt);
  v16i acc[FM];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm) acc[fm] = v16i{0};
  for (int g0 = 0; g0 < G; g0 += GC) {
    uint2 cw[GC];                                  // words 2h, 2h+1 of each cell
    v4i af[GC][2][FM];
#pragma unroll
    for (int j = 0; j < GC; ++j) {
      const int g = g0 + j < G ? g0 + j : G - 1;
      cw[j] = *reinterpret_cast<const uint2*>(x8 + cbase + g * gstride + 8 * h);
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
          af[j][t][fm] = *reinterpret_cast<const v4i*>(
              w8 + (((int64_t)fm * nk32 + 2 * g + t) * 64 + lane) * 16);
    }
    // blocks past G (the last chunk) multiply zero codes: no branch, and no
    // instruction scheduled across this point, so that every load of the
    // chunk is issued before the first MFMA
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < GC; ++j) {
      const bool in = g0 + j < G;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const v4i bf = unpack2(in ? (t == 0 ? cw[j].x : cw[j].y) : 0u);
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
          acc[fm] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[j][t][fm], bf, acc[fm], 0, 0, 0);
      }
    }
  }
  if (p >= a.m) return;
  // lane: pixel p, channels fm*32 + 8b + 4h + i (b = v >> 2, i = v & 3)
  int32_t* y32 = reinterpret_cast<int32_t*>(a.y);
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int c = fm * 32 + 8 * (v >> 2) + 4 * h + (v & 3);
      if (c < a.cout) {
        y32[(int64_t)p * a.cout + c] = acc[fm][v];
        if (a.acc_dump) a.acc_dump[(int64_t)p * a.cout + c] = acc[fm][v];
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

// The epilogue kind of a small8 launch (the EPI template argument).
static int small8_epi(const ConvLaunch& a) {
  const bool fast = a.out_mode != 0 && a.rec == 4 && a.join_kind == IFQ_JOIN_NONE &&
                    (a.out_layout == IFQ_LAYOUT_I8_NHWC ||
                     (a.out_layout == IFQ_LAYOUT_U2_NHWC_PACKED && (a.cout & 3) == 0));
  if (!fast) return 0;
  if (a.pool_k == 0) return 1;
  // the register pool: 2x2/2 windows in whole row pairs, packed NHWC codes,
  // c_out 16 or 32 (one or two row blocks, the whole tile row)
  const bool reg_pool = a.pool_k == 2 && a.pool_s == 2 && !a.pool_same && !a.pool_img &&
                        a.out_layout == IFQ_LAYOUT_U2_NHWC_PACKED &&
                        (a.cout == 16 || a.cout == 32) && ((uintptr_t)a.y & 3) == 0;
  return reg_pool ? 3 : 2;
}

const char* conv_small8_name(const ConvLaunch& a) {
  static const char* names[4][4] = {
      {"conv_small8<1, 0>", "conv_small8<1, 1>", "conv_small8<1, 2>", "conv_small8<1, 3>"},
      {"conv_small8<2, 0>", "conv_small8<2, 1>", "conv_small8<2, 2>", "conv_small8<2, 3>"},
      {"conv_small8<3, 0>", "conv_small8<3, 1>", "conv_small8<3, 2>", ""},
      {"conv_small8<4, 0>", "conv_small8<4, 1>", "conv_small8<4, 2>", ""}};
  return names[(a.cout + 15) / 16 - 1][small8_epi(a)];
}

template <int FM>
static hipError_t launch_small8_fm(const ConvLaunch& a, const SmallGeom& g, hipStream_t stream) {
  const dim3 grid(a.n * g.tiles);
  switch (small8_epi(a)) {
    case 0: hipLaunchKernelGGL((conv_small8<FM, 0>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g); break;
    case 1: hipLaunchKernelGGL((conv_small8<FM, 1>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g); break;
    case 2: hipLaunchKernelGGL((conv_small8<FM, 2>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g); break;
    default:
      if constexpr (FM <= 2) {
        hipLaunchKernelGGL((conv_small8<FM, 3>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g);
      } else {
        return hipErrorInvalidValue;
      }
      break;
  }
  return hipGetLastError();
}

hipError_t launch_conv_small8(const ConvLaunch& a, hipStream_t stream) {
  SmallGeom g;
  if (!small_geom(a, &g)) return hipErrorInvalidValue;
  switch ((a.cout + 15) / 16) {
    case 1: return launch_small8_fm<1>(a, g, stream);
    case 2: return launch_small8_fm<2>(a, g, stream);
    case 3: return launch_small8_fm<3>(a, g, stream);
    case 4: return launch_small8_fm<4>(a, g, stream);
    default: return hipErrorInvalidValue;
  }
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

// The register pool: 2x2/2 windows in whole row pairs (even ho and wo),
// one row block of 32 output channels (four blocks in flight; with two row
// blocks and two blocks in flight it measured slower than the LDS pool on
// the detector's third layer: 10.4 against 9.8 us).
static bool small2_reg_pool(const ConvLaunch& a) {
  return a.pool_k == 2 && a.pool_s == 2 && !a.pool_same && !a.pool_img && a.cout <= 32;
}

const char* conv_small2_name(const ConvLaunch& a) {
  static const char* names[2][2][2] = {
      {{"conv_small2<1, 16, false>", "conv_small2<1, 16, true>"},
       {"conv_small2<1, 32, false>", "conv_small2<1, 32, true>"}},
      {{"conv_small2<2, 16, false>", "conv_small2<2, 16, true>"},
       {"conv_small2<2, 32, false>", "conv_small2<2, 32, true>"}}};
  return names[a.cout > 32][a.cin == 32][small2_reg_pool(a)];
}

template <int FM, int CIN>
static void launch_small2_rp(const ConvLaunch& a, const SmallGeom& g, hipStream_t stream) {
  const dim3 grid(a.n * g.tiles);
  if (small2_reg_pool(a))
    hipLaunchKernelGGL((conv_small2<FM, CIN, true>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g);
  else
    hipLaunchKernelGGL((conv_small2<FM, CIN, false>), grid, dim3(kSmallThreads), g.lds_bytes, stream, a, g);
}

hipError_t launch_conv_small2(const ConvLaunch& a, hipStream_t stream) {
  SmallGeom g;
  if (!small2_geom(a, &g)) return hipErrorInvalidValue;
  const int key = (a.cout > 32 ? 2 : 0) + (a.cin == 32 ? 1 : 0);
  switch (key) {
    case 0: launch_small2_rp<1, 16>(a, g, stream); break;
    case 1: launch_small2_rp<1, 32>(a, g, stream); break;
    case 2: launch_small2_rp<2, 16>(a, g, stream); break;
    case 3: launch_small2_rp<2, 32>(a, g, stream); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

bool head_eligible(const ConvLaunch& a) {
  return a.in_bits == 2 && a.cin % 64 == 0 &&
         (a.in_layout == IFQ_LAYOUT_U2_BLOCK64 || a.in_layout == IFQ_LAYOUT_U2_NHWC_PACKED) &&
         a.kh == 1 && a.kw == 1 && a.stride == 1 && a.pad == 0 && a.cout <= 64 &&
         a.out_mode == 0 && a.join_kind == IFQ_JOIN_NONE && a.m > 0 &&
         ((uintptr_t)a.x & 7) == 0 && (int64_t)a.n * a.h * a.w * (a.cin / 4) < ((int64_t)1 << 40);
}

const char* conv_head_name(const ConvLaunch& a) {
  return a.cout > 32 ? "conv_head<2>" : "conv_head<1>";
}

hipError_t launch_conv_head(const ConvLaunch& a, hipStream_t stream) {
  const dim3 grid((a.m + 31) / 32);
  if (a.cout > 32)
    hipLaunchKernelGGL((conv_head<2>), grid, dim3(64), 0, stream, a);
  else
    hipLaunchKernelGGL((conv_head<1>), grid, dim3(64), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ifq
