// Internal declarations shared by the host entry points and the HIP kernels.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "ifq.h"

namespace ifq {

// Device weight blob of one layer (written by ifq_pack_weights):
//   int8  W[cout_pad][kpad]      W_b, zero beyond K = kh*kw*c_in and beyond
//                                c_out
//   int32 rowsum[cout_pad]       sum over k of W[co][k]
//   int8  zeros[1024]            a zero block: fragment loads that fall
//                                outside W read it instead of branching
//
// Generic kernel (row-major W, byte co*kpad + k): K index k = (r*kw + s)*c_in
// + c', with c' = c for byte-per-code input; for 2-bit NHWC input the 16
// channels of each group are stored transposed as 4x4 (position 4*i + m holds
// channel 4*m + i) to match the order in which four codes are unpacked from a
// byte.
//
// Fast path (mfma_layout(d): 2-bit input, c_in % 64 == 0): W is in the A
// fragment order of v_mfma_i32_32x32x32_i8. K runs over K64 steps
// kk = g*kh*kw + (r*kw + s), G = c_in/64 channel blocks g with the filter
// taps fastest, each split into two K32 steps
// k32 = 2*kk + t. For each block of 32 rows rb and K32 step k32 one 1 KB
// chunk at byte (rb*nk32 + k32)*1024 holds the 64 lanes' 16-byte fragments:
// lane l = 32*h + r carries row 32*rb + r, and its byte 4*q + i is the weight
// of input channel 64*g + 32*h + 16*t + 4*i + q. That is the order in which a
// lane unpacks its 16 codes of a pixel from four packed bytes.
constexpr int kKStep = 64;   // K per LDS stage step (one K64 step)
constexpr int kRowAlign = 16;
constexpr int kMfmaRows = 32;

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

// Division of a non-negative int32 n < 2^31 by a fixed divisor d >= 1 as
// (umulhi(n, mul) + n) >> shift, with shift = ceil(log2 d) and
// mul = floor(2^32 * (2^shift - d) / d) + 1 (division by invariant integers,
// Granlund and Montgomery); exact for every such n.
struct FastDiv {
  uint32_t mul;
  uint32_t shift;
};

inline FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while ((1ull << l) < d) ++l;
  const uint64_t m = ((1ull << 32) * ((1ull << l) - d)) / d + 1;
  return FastDiv{(uint32_t)m, l};
}

struct WeightGeom {
  int64_t k;         // kh*kw*c_in
  int64_t kpad;      // k rounded up to kKStep
  int64_t cout_pad;  // c_out rounded up to the row block
  int64_t rows_bytes;
  int64_t zero_off;     // byte offset of the zero block
  int64_t total_bytes;
};

// Layers that run on the MFMA fast path keep W in fragment order.
inline bool mfma_layout(const ifq_conv_desc& d) {
  return d.in_bits == 2 && d.c_in % 64 == 0 &&
         (d.in_layout == IFQ_LAYOUT_U2_NHWC_PACKED ||
          d.in_layout == IFQ_LAYOUT_U2_BLOCK64);
}

inline WeightGeom weight_geom(const ifq_conv_desc& d) {
  WeightGeom g;
  g.k = (int64_t)d.kh * d.kw * d.c_in;
  g.kpad = round_up(g.k, kKStep);
  g.cout_pad = round_up(d.c_out, mfma_layout(d) ? kMfmaRows : kRowAlign);
  g.rows_bytes = g.cout_pad * g.kpad;
  g.zero_off = round_up(g.rows_bytes + 4 * g.cout_pad, 16);
  g.total_bytes = g.zero_off + 1024;
  return g;
}

// Arguments of one conv launch (resolved and validated on the host).
struct ConvLaunch {
  const uint8_t* x;
  const int8_t* wgt;
  const int32_t* rowsum;
  const int32_t* thr;
  void* y;
  int32_t* acc_dump;
  const void* shortcut;
  const double* coef;      // conv join: {p, q, cc} per channel
  const int32_t* table;    // identity join: [c_out][4][rec] integer records
  double qthr[IFQ_MAX_THRESHOLDS];
  int32_t nq;          // thresholds per channel (codes) or 0
  int32_t rec;         // threshold record length 2^out_bits
  int32_t join_kind;
  int32_t sc_layout;
  int32_t n, h, w, cin, cout, cout_pad;
  int32_t kh, kw, stride, pad, ho, wo;
  int32_t m;           // n*ho*wo
  int32_t kpad, nk;    // nk: K64 steps
  int32_t in_layout, in_bits;
  int32_t out_layout;
  int32_t out_mode;    // 0 int32 sums, 1 codes byte per code, 2 codes 2-bit packed
  int32_t bn;          // pixels per workgroup (set by the launcher)
  int64_t wzero;       // byte offset of the weight blob's zero block
  FastDiv div_howo;    // division by ho*wo (output pixel -> image)
  FastDiv div_wo;      // division by wo (pixel in image -> row)
  // IFQ_JOIN_CONV_FUSED: the 1x1 downsample conv computed in this kernel
  const uint8_t* dx;   // its input codes (BLOCK64)
  const int8_t* dwgt;  // its packed weights (fragment order)
  int64_t d_wzero;     // byte offset of its weight blob's zero block
  int32_t d_cin, d_h, d_w, d_stride;
  int32_t d_nk32;      // its K32 steps (2 * c_in / 64)
  // Max-pool fused into the epilogue (Eq. 4): pool_k x pool_k windows at
  // stride pool_s over the codes (pool_same: SAME mode, windows clipped at
  // the bottom and right edges), y then the pooled tensor
  // [n][pho][pwo][cout]. pool_k 0: no pool. Tiles hold whole rows of
  // windows (pool_img 0: k == stride, valid, ho and wo multiples of k) or
  // whole images (pool_img 1: any window).
  int32_t pool_k, pool_s, pool_same, pool_img;
  // The contraction on the fp4 scaled MFMA (windowed 3x3 kernel, 2-bit
  // threshold epilogue): wgt is then the fp4 weight blob, wzero its zero
  // block.
  int32_t f4;
  int32_t pho, pwo;
  FastDiv div_pwo;     // division by pwo (pooled pixel -> pooled row)
  FastDiv div_pho;     // division by pho (pooled row -> image)
  int32_t wcells;      // register-blocked 3x3 kernels: window cells per channel block
  int32_t tiles_wg;    // persistent 3x3 kernel: consecutive pixel tiles per workgroup
  // K split across workgroups (register-blocked 3x3 kernel, threshold
  // epilogue): split_ok lets the planner split (a workspace is at hand);
  // ksplit workgroups per tile, each over c_in/64/ksplit channel blocks,
  // their int32 partial tiles in ws_part and one arrival counter per tile in
  // ws_cnt (zero before the launch, zero again after it)
  int32_t split_ok;
  int32_t ksplit;
  uint32_t* ws_cnt;
  int32_t* ws_part;
};

// Whether the pooled epilogue takes this launch: codes out (no join), and
// every output tile row of the tile's channels a whole number of 32-bit
// words. The kernel's planner then fits whole rows of windows (or whole
// images, pool_img) into each tile.
inline bool pool_epilogue_ok(const ConvLaunch& a) {
  if (a.pool_k < 1 || a.out_mode == 0 || a.join_kind != IFQ_JOIN_NONE) return false;
  return a.out_mode == 2 ? a.cout % 16 == 0 : a.cout % 4 == 0;
}

hipError_t launch_conv(const ConvLaunch& a, hipStream_t stream);

// Workspace bytes launch_conv needs for these arguments (a K split planned
// with a.split_ok set), 0 if none.
int64_t conv_workspace_bytes(const ConvLaunch& a);
int64_t conv_mfma_workspace_bytes(const ConvLaunch& a);

// Name of the kernel launch_conv would pick for these arguments.
const char* conv_kernel_name(const ConvLaunch& a);

// Fast path (MFMA 32x32x32 kernel): whether it takes the layer, its launch,
// and the name of the variant it picks.
bool mfma_eligible(const ConvLaunch& a);

// 3x3 kernel with per-tile input windows in LDS (BLOCK64 input): the
// variant, pixels per workgroup, workgroups along pixels and the predicted
// time of the best variant that fits the layer, if any.
// Predicted time (us) of a conv launch of `tiles` workgroup tiles of
// tile_ops dense int8 ops each, occ of them sharing a CU: the launch, the
// MFMA work of the busiest CU at a fitted efficiency eff, and a fitted fixed
// cost c0_us per round of occ tiles on a CU (prologue latency, epilogue,
// drain). One form for every kernel, so that the planners' predictions
// compare.
constexpr double kLaunchUs = 2.0;
constexpr int kPlanCUs = 256;
constexpr double kCuOpsPerUsInt8 = 2.4e3 * 8192;   // dense int8 ops per us of one CU
inline double plan_time(int64_t tiles, double tile_ops, int occ, double c0_us, double eff) {
  const int64_t per_cu = (tiles + kPlanCUs - 1) / kPlanCUs;
  const int64_t rounds = (per_cu + occ - 1) / occ;
  return kLaunchUs + (double)per_cu * tile_ops / (kCuOpsPerUsInt8 * eff) +
         (double)rounds * c0_us;
}

struct HaloPlan {
  int variant;
  int bn;
  int blocks_m;
  double t_us;
};
bool plan_halo(const ConvLaunch& a, HaloPlan* out);
hipError_t launch_conv_halo(ConvLaunch a, const HaloPlan& p, hipStream_t stream);
const char* conv_halo_name(const HaloPlan& p, const ConvLaunch& a);
hipError_t launch_conv_mfma(const ConvLaunch& a, hipStream_t stream);

// The largest input window (cells per channel block, each image's rows of
// cells rounded up to 64) that a tile of bn consecutive output pixels of a
// 3x3 pad-1 conv needs, over the layer's tiles, or -1 once it exceeds limit.
// Tiles start at the multiples of step (0: bn), the last ones clipped at m.
// Tile starts repeat modulo ho*wo with period ho*wo / gcd(step, ho*wo), so
// one period and the layer's last starts cover every distinct tile.
inline int64_t window_cells_max(const ConvLaunch& a, int64_t bn, int64_t limit,
                                int64_t step = 0) {
  if (step <= 0) step = bn;
  const int64_t howo = (int64_t)a.ho * a.wo;
  int64_t g = step, r = howo;
  while (r) {
    const int64_t t = g % r;
    g = r;
    r = t;
  }
  const int64_t nst = (a.m + step - 1) / step;           // tile starts
  const int64_t period = howo / g;
  const int64_t tail = (bn + step - 1) / step;           // starts whose tile reaches m
  int64_t mx = 0;
  for (int64_t t = 0; t < nst; ++t) {
    if (t == period && nst - tail > period) t = nst - tail;   // then only the last starts
    const int64_t p0 = t * step;
    const int64_t pend = (p0 + bn < a.m ? p0 + bn : a.m) - 1;
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
    if (tot > mx) mx = tot;
    if (mx > limit) return -1;
  }
  return mx;
}

// 3x3 kernel with register-blocked waves and every channel block's window
// resident in LDS (BLOCK64 input, 2-bit threshold or identity-join
// epilogue): the variant, pixels per workgroup, workgroups along pixels,
// window cells per channel block and the predicted time. forced >= 0 plans
// that variant only (false if it cannot take the layer).
struct W2Plan {
  int variant;
  int bn;
  int blocks_m;
  int wcells;
  double t_us;
  int ksplit;     // workgroups per tile along K (1: no split)
};
// Workspace of a K-split conv: a fixed region of arrival counters (one per
// tile, at most kSplitMaxTiles) at offset 0, which must be zero before the
// first use and is zero again after every launch, then the partial tiles.
// The region sits at the same place for every layer and every stack, so no
// layer's partials or slots ever land on another layer's counters.
constexpr int64_t kSplitCounterBytes = 64 << 10;
constexpr int64_t kSplitMaxTiles = kSplitCounterBytes / 4;
// Workspace bytes of a K-split launch of plan p (0 without a split).
int64_t w2_split_bytes(const ConvLaunch& a, const W2Plan& p);
int w2_variant_count();
bool w2_variant_fp4(int v);   // variant v runs the fp4 contraction (fp4 weight blob)
// want_split > 0: only plans with that K split (a.split_ok must be set for
// any split above 1).
bool plan_w2(const ConvLaunch& a, int forced, W2Plan* out, int want_split = 0);
hipError_t launch_conv_w2(ConvLaunch a, const W2Plan& p, hipStream_t stream);
const char* conv_w2_name(const W2Plan& p, const ConvLaunch& a);

// Persistent 3x3 kernel (BLOCK64 input, every weight of a 64-channel slice
// resident in LDS, 2-bit threshold or identity-join epilogue): the variant,
// pixels per tile, workgroups along pixels, tiles per workgroup, window cells
// per channel block and the predicted time.
struct WpPlan {
  int variant;
  int bn;
  int gx;
  int per;
  int wcells;
  double t_us;
};
int wp_variant_count();
bool wp_variant_fp4(int v);
bool plan_wp(const ConvLaunch& a, int forced, WpPlan* out);
hipError_t launch_conv_wp(ConvLaunch a, const WpPlan& p, hipStream_t stream);
const char* conv_wp_name(const WpPlan& p, const ConvLaunch& a);

// The register-blocked 3x3 kernels as one family: variants 0 ..
// w2_variant_count()-1 are conv_w2's, the rest conv_wp's. plan_reg3 with
// forced < 0 takes the faster prediction of the two planners.
struct Reg3Plan {
  bool persistent;
  W2Plan w2;
  WpPlan wp;
  double t_us;
};
int reg3_variant_count();
bool reg3_variant_fp4(int v);
bool plan_reg3(const ConvLaunch& a, int forced, Reg3Plan* out);
hipError_t launch_reg3(const ConvLaunch& a, const Reg3Plan& p, hipStream_t stream);
const char* reg3_name(const Reg3Plan& p, const ConvLaunch& a);

// Whether a launch with a fused downsample (IFQ_JOIN_CONV_FUSED) is covered
// by one of the 3x3 kernels.
inline bool fused_supported(const ConvLaunch& a) {
  HaloPlan p;
  W2Plan w;
  return plan_halo(a, &p) || plan_w2(a, -1, &w);
}

// 8-bit input codes with c_in <= 4 (a detector's first layer): whether the
// small-channel kernel takes the layer, its launch and its name.
bool small8_eligible(const ConvLaunch& a);
hipError_t launch_conv_small8(const ConvLaunch& a, hipStream_t stream);
const char* conv_small8_name(const ConvLaunch& a);
// 2-bit packed NHWC input codes with c_in 16 or 32, 3x3 s1 p1, 2-bit output
// codes with thresholds (a detector's second and third layers).
bool small2_eligible(const ConvLaunch& a);
hipError_t launch_conv_small2(const ConvLaunch& a, hipStream_t stream);
const char* conv_small2_name(const ConvLaunch& a);
// 1x1, stride 1, c_in a multiple of 64 on 2-bit codes, c_out <= 64, int32
// sums out (a detector's head): a latency-bound kernel without LDS.
bool head_eligible(const ConvLaunch& a);
hipError_t launch_conv_head(const ConvLaunch& a, hipStream_t stream);
const char* conv_head_name(const ConvLaunch& a);
const char* conv_mfma_name(const ConvLaunch& a);

struct PoolLaunch {
  const uint8_t* x;
  uint8_t* y;
  int32_t n, h, w, c, k, stride, ho, wo;
  int32_t layout;
  int32_t bits;
};

hipError_t launch_pool(const PoolLaunch& a, hipStream_t stream);

// Compact thresholds (Eq. 8) -> {s, T_1..T_nq} records of c_out channels.
hipError_t launch_expand_thresholds(const ifq_thr_compact* recs, int c_out, int out_bits,
                                    double bound, int32_t* thr, hipStream_t stream);

// Sets the thread's last-error text (ifq_last_error) and returns st.
ifq_status set_error(ifq_status st, const char* msg);

hipError_t launch_convert(int64_t n, int64_t hw, int32_t c, int32_t src_layout,
                          int32_t dst_layout, const void* src, void* dst,
                          hipStream_t stream);

}  // namespace ifq
