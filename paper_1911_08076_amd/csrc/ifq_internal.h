// Internal declarations shared by the host entry points and the HIP kernels.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#include "ifq.h"

namespace ifq {

// Device weight blob of one layer (written by ifq_pack_weights):
//   int8  rows[cout_pad][kpad]   W_b, K index k = (r*kw + s)*c_in + c', zero
//                                beyond K = kh*kw*c_in and beyond c_out
//   int32 rowsum[cout_pad]       sum over k of rows[co][k]
// c' is c itself for byte-per-code input; for 2-bit packed input the 16
// channels of each group are stored transposed as 4x4 (position 4*i + m holds
// channel 4*m + i) to match the order in which the kernel unpacks four codes
// from each byte.
constexpr int kKStep = 64;   // K per MFMA step (v_mfma_i32_16x16x64_i8)
constexpr int kRowAlign = 16;

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

struct WeightGeom {
  int64_t k;         // kh*kw*c_in
  int64_t kpad;      // k rounded up to kKStep
  int64_t cout_pad;  // c_out rounded up to kRowAlign
  int64_t rows_bytes;
  int64_t total_bytes;
};

inline WeightGeom weight_geom(const ifq_conv_desc& d) {
  WeightGeom g;
  g.k = (int64_t)d.kh * d.kw * d.c_in;
  g.kpad = round_up(g.k, kKStep);
  g.cout_pad = round_up(d.c_out, kRowAlign);
  g.rows_bytes = g.cout_pad * g.kpad;
  g.total_bytes = g.rows_bytes + 4 * g.cout_pad;
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
};

hipError_t launch_conv(const ConvLaunch& a, hipStream_t stream);

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
