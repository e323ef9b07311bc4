// Fast path of the integrated fixed-point quantized convolution on gfx950
// (MI355X): 2-bit input codes with c_in a multiple of 64, in the BLOCK64 or
// the NHWC packed layout.
//
// The integer part of Eq. (1), a = W_b (x) X_q, is an implicit GEMM
// D[co][pixel] = sum_k W[co][k] * X[pixel][k] on v_mfma_i32_32x32x32_i8:
// A (rows = output channels) is the +-1 weight matrix in fragment order, B
// (columns = output pixels) the input codes of one filter tap and 64 channels
// per K64 step, unpacked from 2 bits to int8 in registers right before the
// MFMA. K runs over K64 steps kk = g*kh*kw + (r*kw + s) (G = c_in/64
// channel blocks g, filter taps (r, s) fastest).
//
// A workgroup of WM x WN x WK waves computes a tile of 32*FM*WM output
// channels x up to 32*FN*WN pixels (bn, chosen per layer on the host); the
// WK wave groups split the K64 steps and their sums are added in LDS at the
// end. Operands reach LDS through the LDS-DMA form of the global load (one
// wave instruction moves 64 x 16 bytes, lane i's bytes landing at base +
// 16*i, no staging registers): a weight chunk is 1 KB of fragments, a code
// chunk the 16-byte cells of 64 consecutive output pixels for one tap and
// 64 channels, which in the BLOCK64 layout is one contiguous 1 KB span for a
// stride-1 conv. A ring of D stages of S K64 steps per wave group keeps the
// loads of the next D-1 stages in flight while one computes; every wave
// issues the same number of loads per stage and waits for its part of a
// stage with an explicit vmcnt that leaves younger stages in flight.
// Out-of-range operands are read from blocks of zeros, so the main loop has
// no branch around a load.
//
// Accumulator layout (32x32 MFMA): lane l = 32*h + j holds, for register v,
// row 8*(v/4) + 4*h + v%4 and column j; each lane therefore holds groups of
// four consecutive output channels of one pixel, and the fused epilogue of
// ifq_epilogue.h turns them into codes with integer compares (Eq. 7/8) or the
// residual join without cross-lane traffic.
#include <hip/hip_runtime.h>

#include <cstring>
#include <mutex>

#include "ifq_epilogue.h"
#include "ifq_internal.h"
#include "ifq_mfma_common.h"

namespace ifq {
namespace {

template <int WM, int WN, int WK, int FM, int FN, int S, int D>
__global__ __launch_bounds__(64 * WM * WN * WK) void conv_mfma(ConvLaunch a) {
  constexpr int NWG = WM * WN;                  // waves per K group
  constexpr int NW = NWG * WK;
  constexpr int BM = 32 * FM * WM;
  constexpr int BN = 32 * FN * WN;
  constexpr int BNL = (BN + 63) / 64 * 64;      // pixels loaded per K64 step
  constexpr int A_STEP = BM * 64;               // BM/32 row blocks x 2 K32 x 1 KB
  constexpr int B_STEP = BNL * 16;
  constexpr int STEP = A_STEP + B_STEP;
  constexpr int SK = S * WK;                    // K64 steps per stage
  constexpr int STAGE = SK * STEP;
  constexpr int CA1 = BM / 16, CB1 = BNL / 64;  // 1 KB chunks per K64 step
  constexpr int C = SK * (CA1 + CB1);
  static_assert(C % NW == 0, "equal loads per wave");
  constexpr int CPW = C / NW;
  static_assert((D - 2) * CPW <= 63, "vmcnt range");
  constexpr int EPI_BYTES = epilogue_param_bytes(BM);  // per-channel parameters
  constexpr int OUT_BYTES = BN * BM;            // byte-per-code output tile
  constexpr int RED_BYTES = (WK / 2) * NWG * FM * FN * 4096;
  constexpr int LDS0 = D * STAGE > RED_BYTES ? D * STAGE : RED_BYTES;
  constexpr int LDS_BYTES = LDS0 > EPI_BYTES + OUT_BYTES ? LDS0 : EPI_BYTES + OUT_BYTES;
  static_assert(LDS_BYTES <= 160 * 1024, "LDS");

  __shared__ __attribute__((aligned(1024))) uint8_t lds[LDS_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kg = wave / NWG;                    // K group
  const int wig = wave - kg * NWG;              // wave in group
  const int wm = wig % WM;
  const int wn = wig / WM;
  const int h = lane >> 5;
  const int l32 = lane & 31;
  const int bn = a.bn;
  const int p0 = blockIdx.x * bn;
  const int co0 = blockIdx.y * BM;
  const int G = a.cin >> 6;
  const int nk = a.nk;
  const int nk32 = 2 * nk;
  const int nst = (nk + SK - 1) / SK;
  const int rbw = co0 >> 5;                     // first row block
  const int nrb = a.cout_pad >> 5;
  const int howo = a.ho * a.wo;
  const uint8_t* wbase = reinterpret_cast<const uint8_t*>(a.wgt) + lane * 16;
  const uint8_t* zero_src = reinterpret_cast<const uint8_t*>(&g_zero_cell);
  const uint32_t lds0 = lds_addr(lds);

  // input strides in 16-byte cells: n, channel block, row, column
  int sN, sG, sH, sW;
  if (a.in_layout == IFQ_LAYOUT_U2_BLOCK64) {
    sW = 1; sH = a.w; sG = a.h * a.w; sN = G * sG;
  } else {
    sG = 1; sW = G; sH = a.w * G; sN = a.h * sH;
  }

  // The loads of wave w are chunks c = w + NW*i of a stage; for code chunks
  // the lane's pixel is fixed across stages, so its position is computed once.
  int px_base[CPW], px_iy0[CPW], px_ix0[CPW];
  bool px_ok[CPW];
#pragma unroll
  for (int i = 0; i < CPW; ++i) {
    const int c = wave + NW * i;
    const int cb = (c % (CA1 + CB1)) - CA1;     // code chunk index in the step
    px_ok[i] = false;
    px_base[i] = px_iy0[i] = px_ix0[i] = 0;
    if (cb >= 0) {
      const int pl = cb * 64 + lane;
      const int p = p0 + pl;
      if (pl < bn && p < a.m) {
        const int nimg = fdiv(p, a.div_howo);
        const int rem = p - nimg * howo;
        const int oy = fdiv(rem, a.div_wo);
        const int ox = rem - oy * a.wo;
        px_ok[i] = true;
        px_iy0[i] = oy * a.stride - a.pad;
        px_ix0[i] = ox * a.stride - a.pad;
        px_base[i] = nimg * sN + px_iy0[i] * sH + px_ix0[i] * sW;
      }
    }
  }

  // Filter tap (r, s) and channel block g of K64 step kk, kept incrementally
  // (taps fastest): kpos is the position of the first step of the next stage
  // to issue.
  struct KPos {
    int g, s, r;
  };
  auto adv1 = [&](KPos& q) {
    q.s += 1;
    const bool ws = q.s == a.kw;
    q.s = ws ? 0 : q.s;
    q.r += ws ? 1 : 0;
    const bool wr = q.r == a.kh;
    q.r = wr ? 0 : q.r;
    q.g += wr ? 1 : 0;
  };
  KPos kpos{0, 0, 0};

  // Issue the loads of stage st into ring slot st % D (stages are issued in
  // order). Chunk c covers K64 step kk = st*SK + c / (CA1 + CB1) of the
  // stage; within the step the first CA1 chunks are weights (row block, K32
  // half), the rest codes.
  auto issue = [&](int st) {
    const uint32_t slot = lds0 + (uint32_t)((st % D) * STAGE);
#pragma unroll
    for (int i = 0; i < CPW; ++i) {
      const int c = wave + NW * i;
      const int s_ = c / (CA1 + CB1);
      const int local = c - s_ * (CA1 + CB1);
      const int kk = st * SK + s_;
      const uint32_t dst = slot + (uint32_t)(s_ * STEP + local * 1024);
      if (local < CA1) {
        const int rb = local >> 1, t = local & 1;
        const bool ok = kk < nk && rbw + rb < nrb;
        const int64_t off = ok ? ((int64_t)(rbw + rb) * nk32 + 2 * kk + t) * 1024 : a.wzero;
        dma16(wbase + off, dst);
      } else {
        KPos q = kpos;
        for (int u = 0; u < s_; ++u) adv1(q);
        const int g = q.g, r = q.r, s = q.s;
        const int iy = px_iy0[i] + r;
        const int ix = px_ix0[i] + s;
        const bool ok = kk < nk && px_ok[i] && (unsigned)iy < (unsigned)a.h &&
                        (unsigned)ix < (unsigned)a.w;
        const uint8_t* src =
            ok ? a.x + (int64_t)(px_base[i] + g * sG + r * sH + s * sW) * 16 : zero_src;
        dma16(src, dst);
      }
    }
#pragma unroll
    for (int u = 0; u < SK; ++u) adv1(kpos);
  };

  v16i acc[FM][FN];
#pragma unroll
  for (int fm = 0; fm < FM; ++fm)
#pragma unroll
    for (int fn = 0; fn < FN; ++fn) acc[fm][fn] = v16i{0};

  // K64 steps beyond nk multiply zero weight fragments: no branch here.
  auto compute = [&](int st) {
    const uint8_t* sb = lds + (st % D) * STAGE + kg * S * STEP;
#pragma unroll
    for (int s_ = 0; s_ < S; ++s_) {
      const uint8_t* as = sb + s_ * STEP;
      const uint8_t* bs = as + A_STEP;
      v2i braw[FN];
#pragma unroll
      for (int fn = 0; fn < FN; ++fn)
        braw[fn] = *reinterpret_cast<const v2i*>(
            bs + (wn * 32 * FN + fn * 32 + l32) * 16 + 8 * h);
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        v4i af[FM];
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
          af[fm] = *reinterpret_cast<const v4i*>(as + ((wm * FM + fm) * 2 + t) * 1024 +
                                                 lane * 16);
#pragma unroll
        for (int fn = 0; fn < FN; ++fn) {
          const v4i bf = unpack2((uint32_t)braw[fn][t]);
#pragma unroll
          for (int fm = 0; fm < FM; ++fm)
            acc[fm][fn] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[fm], bf, acc[fm][fn],
                                                                0, 0, 0);
        }
      }
    }
  };

  const int pre = nst < D - 1 ? nst : D - 1;
  for (int st = 0; st < pre; ++st) issue(st);
  for (int st = 0; st < nst; ++st) {
    const int issued_after = nst - 1 - st;      // stages issued after st, capped
    wait_ahead<D - 2, CPW>(issued_after < D - 2 ? issued_after : D - 2);
    __syncthreads();                            // every wave's part landed; slot st-1 free
    if (st + D - 1 < nst) issue(st + D - 1);
    compute(st);
  }
  wait_vmcnt<0>();
  __syncthreads();

  // K groups: sums of groups half..2*half-1 are added into groups 0..half-1
  if constexpr (WK > 1) {
#pragma unroll
    for (int half = WK / 2; half >= 1; half /= 2) {
      if (kg >= half && kg < 2 * half) {
        uint8_t* dst = lds + (((kg - half) * NWG + wig) * FM * FN) * 4096;
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
          for (int fn = 0; fn < FN; ++fn)
#pragma unroll
            for (int j = 0; j < 4; ++j)
              *reinterpret_cast<v4i*>(dst + (fm * FN + fn) * 4096 + j * 1024 + lane * 16) =
                  v4i{acc[fm][fn][4 * j], acc[fm][fn][4 * j + 1], acc[fm][fn][4 * j + 2],
                      acc[fm][fn][4 * j + 3]};
      }
      __syncthreads();
      if (kg < half) {
        const uint8_t* src = lds + ((kg * NWG + wig) * FM * FN) * 4096;
#pragma unroll
        for (int fm = 0; fm < FM; ++fm)
#pragma unroll
          for (int fn = 0; fn < FN; ++fn)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const v4i v = *reinterpret_cast<const v4i*>(src + (fm * FN + fn) * 4096 +
                                                          j * 1024 + lane * 16);
              acc[fm][fn][4 * j] += v.x;
              acc[fm][fn][4 * j + 1] += v.y;
              acc[fm][fn][4 * j + 2] += v.z;
              acc[fm][fn][4 * j + 3] += v.w;
            }
      }
      __syncthreads();
    }
  }

  stage_epilogue(a, lds, co0, BM);
  __syncthreads();
  const int orow = a.out_mode == 2 ? BM / 4 : BM;
  uint8_t* otile = lds + EPI_BYTES;
  if (kg == 0) {
    const bool fast = (a.cout & 31) == 0 && (a.out_mode == 0 || a.rec == 4);
    if (fast) {
      int32_t* y32 = reinterpret_cast<int32_t*>(a.y);
      if (a.acc_dump)
        epilogue32<kE32I32, FM, FN>(a, lds, acc, wm, wn, h, l32, co0, p0, bn, otile, orow,
                                    a.acc_dump);
      if (a.out_mode == 0)
        epilogue32<kE32I32, FM, FN>(a, lds, acc, wm, wn, h, l32, co0, p0, bn, otile, orow, y32);
      else if (a.join_kind == IFQ_JOIN_IDENTITY)
        epilogue32<kE32Tab4, FM, FN>(a, lds, acc, wm, wn, h, l32, co0, p0, bn, otile, orow, y32);
      else if (a.join_kind == IFQ_JOIN_CONV)
        epilogue32<kE32Conv, FM, FN>(a, lds, acc, wm, wn, h, l32, co0, p0, bn, otile, orow, y32);
      else
        epilogue32<kE32Thr4, FM, FN>(a, lds, acc, wm, wn, h, l32, co0, p0, bn, otile, orow, y32);
    } else {
      epilogue_lane<FM * 4, FN>(
          a, lds, [&](int g, int fn, int i) { return acc[g >> 2][fn][4 * (g & 3) + i]; },
          [&](int g) { return co0 + (wm * FM + (g >> 2)) * 32 + 8 * (g & 3) + 4 * h; }, co0,
          p0,
          [&](int fn) {
            const int pl = wn * 32 * FN + fn * 32 + l32;
            return (pl < bn && p0 + pl < a.m) ? pl : -1;
          },
          otile, orow);
    }
  }
  __syncthreads();
  const int npx = a.m - p0 < bn ? a.m - p0 : bn;
  copy_out_tile(a, otile, orow, co0, BM, p0, npx);
}

// ---------------------------------------------------------------------------
// Variants and per-layer planning
// ---------------------------------------------------------------------------
struct Variant {
  int wm, wn, wk, fm, fn;
  double c0_us;      // fixed cost of one round of workgroups (measured)
  double eff;        // MFMA efficiency of the main loop (measured)
  const char* name;
};

// Index order must match the switch in launch_conv_mfma. The two constants
// of each variant are fitted to kernel times on the ResNet-18 layer shapes
// (batch 64); the ones of the 64 x 256 tile are a conservative guess.
const Variant kVariants[] = {
    {2, 4, 1, 2, 4, 9.0, 0.45, "conv_mfma<2, 4, 1, 2, 4, 1, 6>"},    // 128 x 512
    {2, 4, 1, 2, 2, 8.3, 0.443, "conv_mfma<2, 4, 1, 2, 2, 2, 4>"},   // 128 x 256
    {1, 8, 1, 2, 2, 7.7, 0.415, "conv_mfma<1, 8, 1, 2, 2, 2, 4>"},   //  64 x 512
    {2, 4, 1, 1, 2, 9.0, 0.30, "conv_mfma<2, 4, 1, 1, 2, 2, 6>"},    //  64 x 256
    {2, 2, 2, 2, 2, 9.5, 0.309, "conv_mfma<2, 2, 2, 2, 2, 2, 3>"},   // 128 x 128, K split 2
    {2, 1, 4, 1, 4, 6.7, 0.19, "conv_mfma<2, 1, 4, 1, 4, 1, 6>"},    //  64 x 128, K split 4
};
constexpr int kNumVariants = sizeof(kVariants) / sizeof(kVariants[0]);
constexpr int kNumCUs = 256;

struct Plan {
  int variant;
  int bn;        // pixels per workgroup
  int blocks_m;  // workgroups along pixels
  double t_us;   // predicted time
};

// For each variant take the fewest rounds of one workgroup per CU that fit
// the layer and spread the pixels evenly over the workgroups of those rounds
// (in multiples of 32). The predicted time is rounds x (fixed cost + the
// tile's MFMA work at the variant's loop efficiency); the fastest wins.
Plan plan_mfma(const ConvLaunch& a) {
  Plan best{0, 0, 0, 0.0};
  double best_t = 1e30;
  for (int v = 0; v < kNumVariants; ++v) {
    const Variant& V = kVariants[v];
    const int bm = 32 * V.fm * V.wm;
    const int bnmax = 32 * V.fn * V.wn;
    const int64_t nco = (a.cout + bm - 1) / bm;
    const int64_t nb_min = (a.m + bnmax - 1) / bnmax;
    const int64_t rounds = (nco * nb_min + kNumCUs - 1) / kNumCUs;
    int64_t nb = rounds * kNumCUs / nco;
    if (nb < nb_min) nb = nb_min;
    int64_t bn = (a.m + nb - 1) / nb;
    bn = (bn + 31) / 32 * 32;
    if (bn > bnmax) bn = bnmax;
    const int64_t blocks = nco * ((a.m + bn - 1) / bn);
    const double t = plan_time(blocks, 2.0 * bm * bnmax * (double)a.kpad, 1, V.c0_us, V.eff);
    if (t < best_t - 1e-9) {
      best_t = t;
      best = Plan{v, (int)bn, (int)((a.m + bn - 1) / bn), t};
    }
  }
  return best;
}

template <int WM, int WN, int WK, int FM, int FN, int S, int D>
hipError_t launch_variant(ConvLaunch a, const Plan& pl, hipStream_t stream) {
  a.bn = pl.bn;
  dim3 grid(pl.blocks_m, (a.cout + 32 * FM * WM - 1) / (32 * FM * WM));
  hipLaunchKernelGGL((conv_mfma<WM, WN, WK, FM, FN, S, D>), grid,
                     dim3(64 * WM * WN * WK), 0, stream, a);
  return hipGetLastError();
}

}  // namespace

bool mfma_eligible(const ConvLaunch& a) {
  return a.in_bits == 2 && a.cin % 64 == 0 &&
         (a.in_layout == IFQ_LAYOUT_U2_NHWC_PACKED || a.in_layout == IFQ_LAYOUT_U2_BLOCK64);
}

// The dispatcher's choice among the three MFMA kernels for one layer, and
// their plans. Every planner reads only the launch's geometry, layouts,
// epilogue and K-split fields (no pointer, no quantizer threshold value), so
// launches with equal values there get the same choice: it is kept in a
// small table keyed by those fields, which saves the planners' host time
// (several microseconds per layer, against kernels of ten) on every launch
// after the first.
namespace {

struct MfmaChoice {
  int kind;   // 0 register-blocked (reg3), 1 windowed, 2 tiled, -1 none
  HaloPlan hp;
  Reg3Plan rp;
  Plan pl;
};

MfmaChoice plan_choice(const ConvLaunch& a) {
  MfmaChoice c{};
  const bool halo = plan_halo(a, &c.hp);
  const bool r3 = plan_reg3(a, -1, &c.rp);
  if (a.join_kind == IFQ_JOIN_CONV_FUSED) {
    c.kind = r3 ? 0 : (halo ? 1 : -1);
    return c;
  }
  c.pl = plan_mfma(a);
  if (r3 && c.rp.t_us <= c.pl.t_us && (!halo || c.rp.t_us <= c.hp.t_us))
    c.kind = 0;
  else if (halo && c.hp.t_us < c.pl.t_us)
    c.kind = 1;
  else
    c.kind = 2;
  return c;
}

// The launch with its pointers and threshold values cleared (whether a sum
// dump is asked for stays a flag); compared byte for byte, so equal keys
// have equal fields.
ConvLaunch choice_key(const ConvLaunch& a) {
  ConvLaunch k;
  std::memcpy(&k, &a, sizeof(k));
  k.x = nullptr;
  k.wgt = nullptr;
  k.rowsum = nullptr;
  k.thr = nullptr;
  k.y = nullptr;
  k.acc_dump = a.acc_dump ? reinterpret_cast<int32_t*>(alignof(int32_t)) : nullptr;
  k.shortcut = nullptr;
  k.coef = nullptr;
  k.table = nullptr;
  k.dx = nullptr;
  k.dwgt = nullptr;
  k.ws_cnt = nullptr;
  k.ws_part = nullptr;
  for (double& q : k.qthr) q = 0.0;
  return k;
}

struct ChoiceSlot {
  bool used;
  ConvLaunch key;
  MfmaChoice c;
};
constexpr int kChoiceSlots = 256;
ChoiceSlot g_choice[kChoiceSlots];
std::mutex g_choice_mu;

MfmaChoice choose_mfma(const ConvLaunch& a) {
  const ConvLaunch k = choice_key(a);
  uint64_t hsh = 1469598103934665603ull;   // FNV-1a over the key's bytes
  const unsigned char* b = reinterpret_cast<const unsigned char*>(&k);
  for (size_t i = 0; i < sizeof(k); ++i) hsh = (hsh ^ b[i]) * 1099511628211ull;
  ChoiceSlot& slot = g_choice[hsh % kChoiceSlots];
  {
    std::lock_guard<std::mutex> lock(g_choice_mu);
    if (slot.used && std::memcmp(&slot.key, &k, sizeof(k)) == 0) return slot.c;
  }
  const MfmaChoice c = plan_choice(a);
  std::lock_guard<std::mutex> lock(g_choice_mu);
  std::memcpy(&slot.key, &k, sizeof(k));
  slot.c = c;
  slot.used = true;
  return c;
}

}  // namespace

// The fast path picks the kernel with the lowest predicted time among the
// register-blocked 3x3 kernels (one tile per workgroup or persistent), the
// windowed 3x3 kernel and the tiled kernel. A fused downsample join runs on
// the register-blocked kernel wherever it takes the layer (faster on every
// downsampling block of the ResNet-18-shaped stack as measured), else on the
// windowed kernel (the host checks fused_supported before launching one).
const char* conv_mfma_name(const ConvLaunch& a) {
  const MfmaChoice c = choose_mfma(a);
  if (c.kind == 0) return reg3_name(c.rp, a);
  if (c.kind == 1) return conv_halo_name(c.hp, a);
  if (c.kind < 0) return "";
  return kVariants[c.pl.variant].name;
}

// The workspace of the kernel launch_conv_mfma picks (the same choice).
int64_t conv_mfma_workspace_bytes(const ConvLaunch& a) {
  const MfmaChoice c = choose_mfma(a);
  if (c.kind != 0 || c.rp.persistent) return 0;
  return w2_split_bytes(a, c.rp.w2);
}

hipError_t launch_conv_mfma(const ConvLaunch& a, hipStream_t stream) {
  const MfmaChoice c = choose_mfma(a);
  if (c.kind == 0) return launch_reg3(a, c.rp, stream);
  if (c.kind == 1) return launch_conv_halo(a, c.hp, stream);
  if (c.kind < 0) return hipErrorNotSupported;
  const Plan& pl = c.pl;
  switch (pl.variant) {
    case 0: return launch_variant<2, 4, 1, 2, 4, 1, 6>(a, pl, stream);
    case 1: return launch_variant<2, 4, 1, 2, 2, 2, 4>(a, pl, stream);
    case 2: return launch_variant<1, 8, 1, 2, 2, 2, 4>(a, pl, stream);
    case 3: return launch_variant<2, 4, 1, 1, 2, 2, 6>(a, pl, stream);
    case 4: return launch_variant<2, 2, 2, 2, 2, 2, 3>(a, pl, stream);
    default: return launch_variant<2, 1, 4, 1, 4, 1, 6>(a, pl, stream);
  }
}

}  // namespace ifq
