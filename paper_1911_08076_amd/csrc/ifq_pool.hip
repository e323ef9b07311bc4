// Integer max-pool on codes (Eq. 4 applied to the quantizer output) and
// conversion between the code layouts.
//
// Both are HBM-bound streaming kernels: each thread owns a vector of V bytes
// of one output pixel (V = 16, 4 or 1, the widest that divides the bytes per
// pixel), reads the k x k window of input vectors (in-bounds positions only)
// and keeps a per-code running maximum with SWAR byte arithmetic.
#include <hip/hip_runtime.h>

#include "ifq_internal.h"

namespace ifq {
namespace {

// Per-byte unsigned max of four bytes, valid for byte values below 128:
// (b | 0x80) - a never borrows across bytes and its top bit says b >= a.
__device__ __forceinline__ uint32_t max7(uint32_t a, uint32_t b) {
  const uint32_t d = (b | 0x80808080u) - a;
  const uint32_t m = ((d >> 7) & 0x01010101u) * 0xFFu;
  return (b & m) | (a & ~m);
}

// Per-byte unsigned max for any byte values.
__device__ __forceinline__ uint32_t max8(uint32_t a, uint32_t b) {
  uint32_t r = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t x = (a >> (8 * i)) & 0xFFu;
    const uint32_t y = (b >> (8 * i)) & 0xFFu;
    r |= (x > y ? x : y) << (8 * i);
  }
  return r;
}

// Per-field max of sixteen 2-bit codes packed four per byte.
__device__ __forceinline__ uint32_t max2(uint32_t a, uint32_t b) {
  uint32_t r = 0;
#pragma unroll
  for (int f = 0; f < 4; ++f) {
    const uint32_t x = (a >> (2 * f)) & 0x03030303u;
    const uint32_t y = (b >> (2 * f)) & 0x03030303u;
    r |= max7(x, y) << (2 * f);
  }
  return r;
}

// MODE 0: byte codes below 128; 1: any byte codes; 2: 2-bit packed codes.
template <int MODE>
__device__ __forceinline__ uint32_t vmax(uint32_t a, uint32_t b) {
  if constexpr (MODE == 0) return max7(a, b);
  else if constexpr (MODE == 1) return max8(a, b);
  else return max2(a, b);
}

template <int V, int MODE>
__global__ __launch_bounds__(256) void maxpool_codes(PoolLaunch a, int64_t total,
                                                     int cb) {
  const int nv = cb / V;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
       t += (int64_t)gridDim.x * blockDim.x) {
    const int chunk = (int)(t % nv);
    int64_t pix = t / nv;
    const int px = (int)(pix % a.wo);
    pix /= a.wo;
    const int py = (int)(pix % a.ho);
    const int b = (int)(pix / a.ho);
    uint32_t m[(V + 3) / 4];
#pragma unroll
    for (int q = 0; q < (V + 3) / 4; ++q) m[q] = 0u;
    for (int i = 0; i < a.k; ++i) {
      const int iy = py * a.stride + i;
      if (iy >= a.h) break;
      for (int jx = 0; jx < a.k; ++jx) {
        const int ix = px * a.stride + jx;
        if (ix >= a.w) break;
        const uint8_t* src = a.x + ((int64_t)(b * a.h + iy) * a.w + ix) * cb + chunk * V;
        if constexpr (V == 16) {
          const uint4 v = *reinterpret_cast<const uint4*>(src);
          m[0] = vmax<MODE>(m[0], v.x);
          m[1] = vmax<MODE>(m[1], v.y);
          m[2] = vmax<MODE>(m[2], v.z);
          m[3] = vmax<MODE>(m[3], v.w);
        } else if constexpr (V == 4) {
          m[0] = vmax<MODE>(m[0], *reinterpret_cast<const uint32_t*>(src));
        } else {
          m[0] = vmax<MODE>(m[0], (uint32_t)*src);
        }
      }
    }
    uint8_t* dst = a.y + t * V;
    if constexpr (V == 16) {
      *reinterpret_cast<uint4*>(dst) = make_uint4(m[0], m[1], m[2], m[3]);
    } else if constexpr (V == 4) {
      *reinterpret_cast<uint32_t*>(dst) = m[0];
    } else {
      *dst = (uint8_t)m[0];
    }
  }
}

template <int MODE>
hipError_t launch_pool_mode(const PoolLaunch& a, int cb, hipStream_t stream) {
  const int64_t pixels = (int64_t)a.n * a.ho * a.wo;
  auto go = [&](auto kern, int v) {
    const int64_t total = pixels * (cb / v);
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(kern, dim3((unsigned)blocks), dim3(256), 0, stream, a,
                       total, cb);
    return hipGetLastError();
  };
  if (cb % 16 == 0) return go(maxpool_codes<16, MODE>, 16);
  if (cb % 4 == 0) return go(maxpool_codes<4, MODE>, 4);
  return go(maxpool_codes<1, MODE>, 1);
}

// Byte offset of the four codes of channel group cg (channels 4cg..4cg+3)
// of pixel p in a 2-bit code tensor: NHWC packed, or BLOCK64 cells.
__device__ __forceinline__ int64_t u2_offset(int32_t layout, int64_t p, int64_t cg,
                                             int64_t hw, int32_t c) {
  if (layout == IFQ_LAYOUT_U2_NHWC_PACKED) return p * (c >> 2) + cg;
  const int64_t nimg = p / hw;
  return ((nimg * (c >> 6) + (cg >> 4)) * hw + (p - nimg * hw)) * 16 + (cg & 15);
}

// One thread per group of four codes: reads them in the source layout and
// writes them in the destination layout (byte per code or 2-bit).
__global__ __launch_bounds__(256) void convert_codes(const uint8_t* src, uint8_t* dst,
                                                     int64_t groups, int64_t hw,
                                                     int32_t c, int32_t sl, int32_t dl) {
  const int64_t cgs = c >> 2;
  for (int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; g < groups;
       g += (int64_t)gridDim.x * blockDim.x) {
    const int64_t p = g / cgs, cg = g - p * cgs;
    uint32_t codes;  // byte i = code of channel 4cg + i
    if (sl == IFQ_LAYOUT_I8_NHWC) {
      codes = *reinterpret_cast<const uint32_t*>(src + 4 * g) & 0x03030303u;
    } else {
      const uint32_t b = src[u2_offset(sl, p, cg, hw, c)];
      codes = (b & 3u) | ((b & 0x0Cu) << 6) | ((b & 0x30u) << 12) | ((b & 0xC0u) << 18);
    }
    if (dl == IFQ_LAYOUT_I8_NHWC) {
      *reinterpret_cast<uint32_t*>(dst + 4 * g) = codes;
    } else {
      dst[u2_offset(dl, p, cg, hw, c)] =
          (uint8_t)((codes & 3u) | ((codes >> 6) & 0x0Cu) | ((codes >> 12) & 0x30u) |
                    ((codes >> 18) & 0xC0u));
    }
  }
}

}  // namespace

hipError_t launch_pool(const PoolLaunch& a, hipStream_t stream) {
  if ((int64_t)a.n * a.ho * a.wo == 0) return hipSuccess;
  if (a.layout == IFQ_LAYOUT_U2_NHWC_PACKED)
    return launch_pool_mode<2>(a, a.c / 4, stream);
  if (a.bits < 8) return launch_pool_mode<0>(a, a.c, stream);
  return launch_pool_mode<1>(a, a.c, stream);
}

hipError_t launch_convert(int64_t n, int64_t hw, int32_t c, int32_t src_layout,
                          int32_t dst_layout, const void* src, void* dst,
                          hipStream_t stream) {
  const int64_t groups = n * hw * (c / 4);
  if (groups == 0) return hipSuccess;
  int64_t blocks = (groups + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(convert_codes, dim3((unsigned)blocks), dim3(256), 0, stream,
                     reinterpret_cast<const uint8_t*>(src), reinterpret_cast<uint8_t*>(dst),
                     groups, hw, c, src_layout, dst_layout);
  return hipGetLastError();
}

}  // namespace ifq
