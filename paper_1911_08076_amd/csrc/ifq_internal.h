// Internal declarations shared by the host entry points and the HIP kernels.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "ifq.h"

namespace ifq {

// Device weight blob of one layer (written by ifq_pack_weights):
//   int8  W[cout_pad][kpad]      W_b, K index k = (r*kw + s)*c_in + c', zero
//                                beyond K = kh*kw*c_in and beyond c_out
//   int32 rowsum[cout_pad]       sum over k of W[co][k]
//   int8  zeros[1024]            a zero block: fast-path fragment loads that
//                                fall outside W read it instead of branching
// c' is c itself for byte-per-code input; for 2-bit packed input the 16
// channels of each group are stored transposed as 4x4 (position 4*i + m holds
// channel 4*m + i) to match the order in which the kernels unpack four codes
// from each byte.
// W is stored either row-major (byte co*kpad + k) or, for layers that take the
// fast path (frag_layout), in MFMA fragment order: for each block of 16 rows
// rb and K step kt, 1 KB holding the 64 lanes' 16-byte A fragments of
// v_mfma_i32_16x16x64_i8, lane l = 16*g + i carrying row 16*rb + i and
// K bytes 64*kt + 16*g .. +15; byte ((rb*nk + kt)*64 + l)*16 + b.
constexpr int kKStep = 64;   // K per MFMA step (v_mfma_i32_16x16x64_i8)
constexpr int kRowAlign = 16;

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

struct WeightGeom {
  int64_t k;         // kh*kw*c_in
  int64_t kpad;      // k rounded up to kKStep
  int64_t cout_pad;  // c_out rounded up to kRowAlign
  int64_t rows_bytes;
  int64_t zero_off;     // byte offset of the zero block
  int64_t total_bytes;
};

// Layers that run on the 2-bit fast path keep W in MFMA fragment order.
inline bool frag_layout(const ifq_conv_desc& d) {
  return d.in_layout == IFQ_LAYOUT_U2_NHWC_PACKED && d.c_in % 64 == 0;
}

inline WeightGeom weight_geom(const ifq_conv_desc& d) {
  WeightGeom g;
  g.k = (int64_t)d.kh * d.kw * d.c_in;
  g.kpad = round_up(g.k, kKStep);
  g.cout_pad = round_up(d.c_out, kRowAlign);
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
  const double* coef;
  double qthr[IFQ_MAX_THRESHOLDS];
  int32_t nq;          // thresholds per channel (codes) or 0
  int32_t rec;         // threshold record length 2^out_bits
  int32_t join_kind;
  int32_t sc_layout;
  int32_t n, h, w, cin, cout, cout_pad;
  int32_t kh, kw, stride, pad, ho, wo;
  int32_t m;           // n*ho*wo
  int32_t kpad, nk;
  int32_t in_layout, in_bits;
  int32_t out_mode;    // 0 int32 sums, 1 codes byte per code, 2 codes 2-bit packed
  int32_t bn;          // pixels per workgroup (set by the launcher)
  int64_t wzero;       // byte offset of the weight blob's zero block
};

hipError_t launch_conv(const ConvLaunch& a, hipStream_t stream);

// Name of the kernel launch_conv would pick for these arguments.
const char* conv_kernel_name(const ConvLaunch& a);

struct PoolLaunch {
  const uint8_t* x;
  uint8_t* y;
  int32_t n, h, w, c, k, stride, ho, wo;
  int32_t layout;
  int32_t bits;
};

hipError_t launch_pool(const PoolLaunch& a, hipStream_t stream);

hipError_t launch_convert(int64_t ncodes, int32_t src_layout,
                          const void* src, void* dst, hipStream_t stream);

}  // namespace ifq
