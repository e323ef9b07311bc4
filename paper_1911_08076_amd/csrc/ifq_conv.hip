// Generic integrated fixed-point quantized convolution on gfx950 (MI355X):
// every layer shape and code layout the fast path (ifq_conv_mfma.hip) does
// not take: byte-per-code input, 8-bit input codes, c_in not a multiple of
// 64, 2-bit NHWC input with 16 | c_in.
//
// One kernel computes a quantized substructure of IFQ-Net:
//   a    = W_b (x) X_q            integer part of Eq. (1), as an implicit GEMM
//                                 D[co][pixel] = sum_k W[co][k] * X[pixel][k]
//                                 on v_mfma_i32_16x16x64_i8 (int8 x int8 -> int32)
//   code = #{i : s*a > T_i}       Eq. (7)/(8): integer thresholds folded on the
//                                 host (Sec. 3.2); or the residual join, or the
//                                 int32 sum itself for layers without quantizer
//
// K runs over (tap, channel): k = (r*kw + s)*c_in + c. The A operand (rows =
// output channels) is the packed +-1 weight matrix, the B operand (columns =
// output pixels) is gathered on the fly from the NHWC codes, 16 channels of
// one tap at a time, with zero codes for padded positions. Both tiles go
// through LDS, double-buffered, one barrier per 64-wide K step.
//
// Output channels sit on the MFMA row dimension, so each lane of a 16x16
// accumulator block holds four consecutive output channels of one pixel:
// four codes pack into one 32-bit word (byte per code) or one byte (2-bit)
// without any cross-lane traffic.
//
// 8-bit input codes (0..255) do not fit signed int8. They enter the MFMA as
// x - 128 (XOR 0x80), padded positions as -128 (i.e. x = 0), and the epilogue
// adds back 128 * rowsum(W[co]): sum W*x = sum W*(x-128) + 128 * sum W, exact.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "ifq_epilogue.h"
#include "ifq_internal.h"

namespace ifq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

enum Gather {
  kGatherI8 = 0,     // byte-per-code input, c_in % 16 == 0: 16-byte loads
  kGatherU2 = 1,     // 2-bit packed input, c_in % 16 == 0: 4-byte loads
  kGatherBytes = 2,  // byte-per-code input, any c_in: byte loads
};

constexpr uint32_t kLow2 = 0x03030303u;

// XOR swizzle of the four 16-byte chunks of a 64-byte LDS row, so that the
// 16-byte reads of eight consecutive rows hit distinct banks.
__device__ __forceinline__ int swz(int row) { return (row >> 1) & 3; }

template <int BM, int BN, int WAVES_M, int GATHER>
__global__ __launch_bounds__(256) void conv_igemm(ConvLaunch a) {
  constexpr int WAVES_N = 4 / WAVES_M;
  constexpr int WM = BM / WAVES_M;
  constexpr int WN = BN / WAVES_N;
  constexpr int FM = WM / 16;
  constexpr int FN = WN / 16;
  static_assert(FM >= 1 && FN >= 1 && WM % 16 == 0 && WN % 16 == 0, "wave tile");
  constexpr int A_BYTES = BM * 64;
  constexpr int B_ROW = GATHER == kGatherU2 ? 16 : 64;
  constexpr int B_BYTES = BN * B_ROW;
  constexpr int STAGE = A_BYTES + B_BYTES;
  constexpr int A_CHUNKS = BM * 4;
  constexpr int A_PER_T = (A_CHUNKS + 255) / 256;
  static_assert((BN * 4) % 256 == 0, "BN must be a multiple of 64");
  constexpr int B_PER_T = BN * 4 / 256;
  constexpr int EPI_BYTES = epilogue_param_bytes(BM);  // per-channel parameters
  constexpr int OUT_BYTES = BN * BM;            // output tile, byte per code
  constexpr int LDS_BYTES =
      2 * STAGE > EPI_BYTES + OUT_BYTES ? 2 * STAGE : EPI_BYTES + OUT_BYTES;

  __shared__ __attribute__((aligned(16))) uint8_t lds[LDS_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % WAVES_M;
  const int wn = wave / WAVES_M;
  const int p0 = blockIdx.x * BN;
  const int co0 = blockIdx.y * BM;

  // Each thread gathers k16-group j of pixels (tid>>2) + 64*i of the tile.
  const int j = tid & 3;
  const int howo = a.ho * a.wo;
  int pix_row[B_PER_T], pix_iy0[B_PER_T], pix_ix0[B_PER_T];
#pragma unroll
  for (int i = 0; i < B_PER_T; ++i) {
    const int p = p0 + (tid >> 2) + 64 * i;
    if (p < a.m) {
      const int nimg = p / howo;
      const int rem = p - nimg * howo;
      const int oy = rem / a.wo;
      const int ox = rem - oy * a.wo;
      pix_row[i] = nimg * a.h;
      pix_iy0[i] = oy * a.stride - a.pad;
      pix_ix0[i] = ox * a.stride - a.pad;
    } else {
      pix_row[i] = -1;
      pix_iy0[i] = 0;
      pix_ix0[i] = 0;
    }
  }
  const bool in8 = a.in_bits == 8;
  const uint32_t pad_word = in8 ? 0x80808080u : 0u;
  const int cg16 = a.cin >> 4;
  const int ntaps = a.kh * a.kw;

  uint4 areg[A_PER_T];
  uint4 breg[B_PER_T];

  auto load_a = [&](int kt) {
#pragma unroll
    for (int i = 0; i < A_PER_T; ++i) {
      const int q = tid + 256 * i;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (q < A_CHUNKS) {
        const int co = co0 + (q >> 2);
        if (co < a.cout_pad)
          v = *reinterpret_cast<const uint4*>(
              a.wgt + (int64_t)co * a.kpad + kt * kKStep + (q & 3) * 16);
      }
      areg[i] = v;
    }
  };

  auto load_b = [&](int kt) {
    if constexpr (GATHER == kGatherBytes) {
#pragma unroll
      for (int i = 0; i < B_PER_T; ++i) {
        uint32_t wd[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int b = 0; b < 16; ++b) {
          const int k = kt * kKStep + j * 16 + b;
          const int tap = k / a.cin;
          const int c = k - tap * a.cin;
          const int r = tap / a.kw;
          const int s = tap - r * a.kw;
          const int iy = pix_iy0[i] + r;
          const int ix = pix_ix0[i] + s;
          const bool ok = tap < ntaps && pix_row[i] >= 0 &&
                          (unsigned)iy < (unsigned)a.h &&
                          (unsigned)ix < (unsigned)a.w;
          uint32_t val = in8 ? 0x80u : 0u;
          if (ok) {
            val = a.x[((int64_t)(pix_row[i] + iy) * a.w + ix) * a.cin + c];
            if (in8) val ^= 0x80u;
          }
          wd[b >> 2] |= val << (8 * (b & 3));
        }
        breg[i] = make_uint4(wd[0], wd[1], wd[2], wd[3]);
      }
    } else {
      const int k16 = kt * 4 + j;
      const int tap = k16 / cg16;
      const int cg = k16 - tap * cg16;
      const int r = tap / a.kw;
      const int s = tap - r * a.kw;
      const bool tap_ok = tap < ntaps;
#pragma unroll
      for (int i = 0; i < B_PER_T; ++i) {
        const int iy = pix_iy0[i] + r;
        const int ix = pix_ix0[i] + s;
        const bool ok = tap_ok && pix_row[i] >= 0 &&
                        (unsigned)iy < (unsigned)a.h &&
                        (unsigned)ix < (unsigned)a.w;
        const int64_t ch = ((int64_t)(pix_row[i] + iy) * a.w + ix) * a.cin + cg * 16;
        if constexpr (GATHER == kGatherI8) {
          uint4 v = make_uint4(pad_word, pad_word, pad_word, pad_word);
          if (ok) {
            v = *reinterpret_cast<const uint4*>(a.x + ch);
            if (in8) {
              v.x ^= 0x80808080u;
              v.y ^= 0x80808080u;
              v.z ^= 0x80808080u;
              v.w ^= 0x80808080u;
            }
          }
          breg[i] = v;
        } else {
          uint32_t v = 0u;
          if (ok) v = *reinterpret_cast<const uint32_t*>(a.x + (ch >> 2));
          breg[i] = make_uint4(v, 0u, 0u, 0u);
        }
      }
    }
  };

  auto store = [&](int buf) {
    uint8_t* as = lds + buf * STAGE;
    uint8_t* bs = as + A_BYTES;
#pragma unroll
    for (int i = 0; i < A_PER_T; ++i) {
      const int q = tid + 256 * i;
      if (q < A_CHUNKS) {
        const int row = q >> 2;
        *reinterpret_cast<uint4*>(as + row * 64 + (((q & 3) ^ swz(row)) << 4)) = areg[i];
      }
    }
#pragma unroll
    for (int i = 0; i < B_PER_T; ++i) {
      const int pl = (tid >> 2) + 64 * i;
      if constexpr (GATHER == kGatherU2) {
        *reinterpret_cast<uint32_t*>(bs + pl * 16 + j * 4) = breg[i].x;
      } else {
        *reinterpret_cast<uint4*>(bs + pl * 64 + ((j ^ swz(pl)) << 4)) = breg[i];
      }
    }
  };

  v4i acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = v4i{0, 0, 0, 0};

  const int kg = lane >> 4;
  const int l16 = lane & 15;

  auto compute = [&](int buf) {
    const uint8_t* as = lds + buf * STAGE;
    const uint8_t* bs = as + A_BYTES;
    v4i af[FM], bf[FN];
#pragma unroll
    for (int fm = 0; fm < FM; ++fm) {
      const int row = wm * WM + fm * 16 + l16;
      af[fm] = *reinterpret_cast<const v4i*>(as + row * 64 + ((kg ^ swz(row)) << 4));
    }
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) {
      const int pix = wn * WN + fn * 16 + l16;
      if constexpr (GATHER == kGatherU2) {
        const uint32_t u = *reinterpret_cast<const uint32_t*>(bs + pix * 16 + kg * 4);
        bf[fn] = v4i{(int)(u & kLow2), (int)((u >> 2) & kLow2),
                     (int)((u >> 4) & kLow2), (int)((u >> 6) & kLow2)};
      } else {
        bf[fn] = *reinterpret_cast<const v4i*>(bs + pix * 64 + ((kg ^ swz(pix)) << 4));
      }
    }
#pragma unroll
    for (int fm = 0; fm < FM; ++fm)
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        acc[fm][fn] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[fm], bf[fn], acc[fm][fn], 0, 0, 0);
  };

  load_a(0);
  load_b(0);
  store(0);
  __syncthreads();
  for (int kt = 0; kt < a.nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < a.nk;
    if (more) {
      load_a(kt + 1);
      load_b(kt + 1);
    }
    compute(cur);
    if (more) store(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue: lane holds channels co..co+3 of pixel p per block ----
  stage_epilogue(a, lds, co0, BM);
  __syncthreads();
  const int orow = a.out_mode == 2 ? BM / 4 : BM;
  uint8_t* otile = lds + EPI_BYTES;
  // 16x16 accumulator block (fm, fn): lane holds channels 4*kg..4*kg+3 of
  // the block's rows and pixel l16 of its columns
  epilogue_lane<FM, FN>(
      a, lds, [&](int g, int fn, int i) { return acc[g][fn][i]; },
      [&](int g) { return co0 + wm * WM + g * 16 + 4 * kg; }, co0, p0,
      [&](int fn) {
        const int pl = wn * WN + fn * 16 + l16;
        return p0 + pl < a.m ? pl : -1;
      },
      otile, orow);
  __syncthreads();
  copy_out_tile(a, otile, orow, co0, BM, p0, a.m - p0 < BN ? a.m - p0 : BN);
}


template <int BM, int BN, int WAVES_M, int GATHER>
hipError_t launch_tile(const ConvLaunch& a, hipStream_t stream) {
  dim3 grid((a.m + BN - 1) / BN, (a.cout + BM - 1) / BM);
  hipLaunchKernelGGL((conv_igemm<BM, BN, WAVES_M, GATHER>), grid, dim3(256), 0,
                     stream, a);
  return hipGetLastError();
}

// Tile variant by output-channel count: 0: 16x256, 1: 32x128, 2: 64x128,
// 3: 128x128 (output channels x pixels per workgroup).
int tile_variant(const ConvLaunch& a) {
  if (a.cout <= 16) return 0;
  if (a.cout <= 32) return 1;
  if (a.cout <= 64) return 2;
  return 3;
}

int gather_kind(const ConvLaunch& a) {
  if (a.in_layout == IFQ_LAYOUT_U2_NHWC_PACKED) return kGatherU2;
  if (a.cin % 16 == 0) return kGatherI8;
  return kGatherBytes;
}

template <int GATHER>
hipError_t launch_gather(const ConvLaunch& a, hipStream_t stream) {
  switch (tile_variant(a)) {
    case 0: return launch_tile<16, 256, 1, GATHER>(a, stream);
    case 1: return launch_tile<32, 128, 1, GATHER>(a, stream);
    case 2: return launch_tile<64, 128, 2, GATHER>(a, stream);
    default: return launch_tile<128, 128, 2, GATHER>(a, stream);
  }
}

}  // namespace

// A fused pool (a.pool_k) runs in the windowed 3x3 kernel or one of the
// small-channel kernels, where their planners fit whole rows of pooling
// windows into a tile; no other kernel takes it.
const char* conv_kernel_name(const ConvLaunch& a) {
  if (a.m == 0) return "";   // nothing is launched
  if (a.pool_k) {
    HaloPlan hp;
    if (mfma_eligible(a) && plan_halo(a, &hp)) return conv_halo_name(hp, a);
    if (small8_eligible(a)) return conv_small8_name(a);
    if (small2_eligible(a)) return conv_small2_name(a);
    return "";
  }
  if (head_eligible(a)) return conv_head_name(a);
  if (mfma_eligible(a)) return conv_mfma_name(a);
  if (small8_eligible(a)) return conv_small8_name(a);
  if (small2_eligible(a)) return conv_small2_name(a);
  static const char* names[3][4] = {
      {"conv_igemm<16, 256, 1, 0>", "conv_igemm<32, 128, 1, 0>",
       "conv_igemm<64, 128, 2, 0>", "conv_igemm<128, 128, 2, 0>"},
      {"conv_igemm<16, 256, 1, 1>", "conv_igemm<32, 128, 1, 1>",
       "conv_igemm<64, 128, 2, 1>", "conv_igemm<128, 128, 2, 1>"},
      {"conv_igemm<16, 256, 1, 2>", "conv_igemm<32, 128, 1, 2>",
       "conv_igemm<64, 128, 2, 2>", "conv_igemm<128, 128, 2, 2>"}};
  return names[gather_kind(a)][tile_variant(a)];
}

int64_t conv_workspace_bytes(const ConvLaunch& a) {
  if (a.m == 0 || a.pool_k || head_eligible(a)) return 0;
  return mfma_eligible(a) ? conv_mfma_workspace_bytes(a) : 0;
}

hipError_t launch_conv(const ConvLaunch& a, hipStream_t stream) {
  if (a.m == 0) return hipSuccess;
  if (a.pool_k) {
    HaloPlan hp;
    if (mfma_eligible(a) && plan_halo(a, &hp)) return launch_conv_halo(a, hp, stream);
    if (small8_eligible(a)) return launch_conv_small8(a, stream);
    if (small2_eligible(a)) return launch_conv_small2(a, stream);
    return hipErrorNotSupported;
  }
  if (head_eligible(a)) return launch_conv_head(a, stream);
  if (mfma_eligible(a)) return launch_conv_mfma(a, stream);
  if (small8_eligible(a)) return launch_conv_small8(a, stream);
  if (small2_eligible(a)) return launch_conv_small2(a, stream);
  switch (gather_kind(a)) {
    case kGatherU2: return launch_gather<kGatherU2>(a, stream);
    case kGatherI8: return launch_gather<kGatherI8>(a, stream);
    default: return launch_gather<kGatherBytes>(a, stream);
  }
}

}  // namespace ifq
