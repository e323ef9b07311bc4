// Host side of the C ABI declared in include/ifq.h: argument validation,
// the weight packer, the threshold and join folds (Sec. 3.2, Eq. 6 -> 7 -> 8),
// launch resolution and the layer-chain driver. Compiled with
// -ffp-contract=off: the folds evaluate their fp64 expressions one operation
// per statement in a fixed order.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "ifq.h"
#include "ifq_internal.h"

namespace {

thread_local std::string g_last_error;

ifq_status fail(ifq_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

ifq_status ok() {
  g_last_error.clear();
  return IFQ_OK;
}

}  // namespace

namespace ifq {
ifq_status set_error(ifq_status st, const char* msg) {
  g_last_error = msg;
  return st;
}
}  // namespace ifq

namespace {

constexpr int64_t kMaxIndex = (int64_t)1 << 31;  // byte offsets kept below 2^31

bool is_finite(double v) { return std::isfinite(v); }

int64_t out_extent(int64_t in, int64_t k, int64_t stride, int64_t pad) {
  return (in + 2 * pad - k) / stride + 1;
}

int64_t tensor_bytes(int64_t n, int64_t h, int64_t w, int64_t c, int layout) {
  if (n < 0 || h < 0 || w < 0 || c < 0) return -1;
  const int64_t e = n * h * w * c;
  switch (layout) {
    case IFQ_LAYOUT_I8_NHWC: return e;
    case IFQ_LAYOUT_U2_NHWC_PACKED: return (c % 4) ? -1 : e / 4;
    case IFQ_LAYOUT_U2_BLOCK64: return (c % 64) ? -1 : e / 4;
    case IFQ_LAYOUT_I32_NHWC: return 4 * e;
    default: return -1;
  }
}

// Structural validation of a conv descriptor. UNSUPPORTED marks shapes the
// kernels do not handle although the descriptor itself is meaningful.
ifq_status check_conv(const ifq_conv_desc* d, int64_t* ho_out = nullptr,
                      int64_t* wo_out = nullptr) {
  if (!d) return fail(IFQ_ERR_INVALID_ARGUMENT, "conv desc is NULL");
  if (d->n < 0 || d->h < 1 || d->w < 1 || d->c_in < 1 || d->c_out < 1)
    return fail(IFQ_ERR_INVALID_ARGUMENT,
                "conv: need n >= 0 and h, w, c_in, c_out >= 1 (got n=%d h=%d "
                "w=%d c_in=%d c_out=%d)", d->n, d->h, d->w, d->c_in, d->c_out);
  if (d->kh < 1 || d->kw < 1 || d->stride < 1 || d->pad < 0)
    return fail(IFQ_ERR_INVALID_ARGUMENT,
                "conv: need kh, kw, stride >= 1 and pad >= 0");
  if (d->h + 2 * d->pad < d->kh || d->w + 2 * d->pad < d->kw)
    return fail(IFQ_ERR_INVALID_ARGUMENT,
                "conv: filter larger than the padded input");
  if (d->in_bits < 1 || d->in_bits > 8)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "conv: in_bits must be 1..8");
  if (d->out_bits < 0 || d->out_bits > 4)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "conv: out_bits must be 0..4");
  if (d->in_layout == IFQ_LAYOUT_U2_NHWC_PACKED) {
    if (d->in_bits != 2)
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "conv: 2-bit packed input needs in_bits == 2");
    if (d->c_in % 4)
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "conv: 2-bit packed input needs c_in %% 4 == 0");
    if (d->c_in % 16)
      return fail(IFQ_ERR_UNSUPPORTED,
                  "conv: 2-bit packed input needs c_in %% 16 == 0");
  } else if (d->in_layout == IFQ_LAYOUT_U2_BLOCK64) {
    if (d->in_bits != 2 || d->c_in % 64)
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "conv: BLOCK64 input needs in_bits == 2 and c_in %% 64 == 0");
  } else if (d->in_layout != IFQ_LAYOUT_I8_NHWC) {
    return fail(IFQ_ERR_INVALID_ARGUMENT, "conv: bad in_layout %d", d->in_layout);
  }
  if (d->out_bits == 0) {
    if (d->out_layout != IFQ_LAYOUT_I32_NHWC)
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "conv: out_bits == 0 needs out_layout I32_NHWC");
  } else if (d->out_layout == IFQ_LAYOUT_U2_NHWC_PACKED) {
    if (d->out_bits != 2)
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "conv: 2-bit packed output needs out_bits == 2");
    if (d->c_out % 4)
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "conv: 2-bit packed output needs c_out %% 4 == 0");
  } else if (d->out_layout == IFQ_LAYOUT_U2_BLOCK64) {
    if (d->out_bits != 2 || d->c_out % 64)
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "conv: BLOCK64 output needs out_bits == 2 and c_out %% 64 == 0");
  } else if (d->out_layout != IFQ_LAYOUT_I8_NHWC) {
    return fail(IFQ_ERR_INVALID_ARGUMENT, "conv: bad out_layout %d", d->out_layout);
  }
  const int64_t ho = out_extent(d->h, d->kh, d->stride, d->pad);
  const int64_t wo = out_extent(d->w, d->kw, d->stride, d->pad);
  const int64_t xb = tensor_bytes(d->n, d->h, d->w, d->c_in, d->in_layout);
  const int64_t yb = tensor_bytes(d->n, ho, wo, d->c_out, IFQ_LAYOUT_I32_NHWC);
  if (xb >= kMaxIndex || yb >= kMaxIndex)
    return fail(IFQ_ERR_UNSUPPORTED, "conv: tensors of 2^31 bytes or more");
  const int64_t k = (int64_t)d->kh * d->kw * d->c_in;
  if (k * ((1 << d->in_bits) - 1) >= kMaxIndex / 2)
    return fail(IFQ_ERR_UNSUPPORTED, "conv: sums could overflow int32");
  if (ho_out) *ho_out = ho;
  if (wo_out) *wo_out = wo;
  return IFQ_OK;
}

ifq_status check_pool(const ifq_pool_desc* d, int64_t* ho, int64_t* wo) {
  if (!d) return fail(IFQ_ERR_INVALID_ARGUMENT, "pool desc is NULL");
  if (d->n < 0 || d->h < 1 || d->w < 1 || d->c < 1)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "pool: need n >= 0, h, w, c >= 1");
  if (d->k < 1 || d->stride < 1)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "pool: need k, stride >= 1");
  if (d->bits < 1 || d->bits > 8)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "pool: bits must be 1..8");
  if (d->layout == IFQ_LAYOUT_U2_NHWC_PACKED) {
    if (d->bits != 2 || d->c % 4)
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "pool: 2-bit packed codes need bits == 2 and c %% 4 == 0");
  } else if (d->layout == IFQ_LAYOUT_U2_BLOCK64) {
    if (d->bits != 2 || d->c % 64)
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "pool: BLOCK64 codes need bits == 2 and c %% 64 == 0");
  } else if (d->layout != IFQ_LAYOUT_I8_NHWC) {
    return fail(IFQ_ERR_INVALID_ARGUMENT, "pool: bad layout %d", d->layout);
  }
  if (d->mode == IFQ_POOL_VALID) {
    if (d->k > d->h || d->k > d->w)
      return fail(IFQ_ERR_INVALID_ARGUMENT, "pool: window larger than input");
    *ho = (d->h - d->k) / d->stride + 1;
    *wo = (d->w - d->k) / d->stride + 1;
  } else if (d->mode == IFQ_POOL_SAME) {
    *ho = (d->h + d->stride - 1) / d->stride;
    *wo = (d->w + d->stride - 1) / d->stride;
  } else {
    return fail(IFQ_ERR_INVALID_ARGUMENT, "pool: bad mode %d", d->mode);
  }
  if (tensor_bytes(d->n, d->h, d->w, d->c, IFQ_LAYOUT_I8_NHWC) >= kMaxIndex)
    return fail(IFQ_ERR_UNSUPPORTED, "pool: tensors of 2^31 bytes or more");
  return IFQ_OK;
}

ifq_status check_join(const ifq_join* j, const ifq_conv_desc* d) {
  if (j->kind != IFQ_JOIN_IDENTITY && j->kind != IFQ_JOIN_CONV &&
      j->kind != IFQ_JOIN_CONV_FUSED)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "join: bad kind %d", j->kind);
  if (d->out_bits == 0)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "join: needs a quantized output");
  if (j->n_q != (1 << d->out_bits) - 1)
    return fail(IFQ_ERR_INVALID_ARGUMENT,
                "join: n_q must be 2^out_bits - 1 = %d", (1 << d->out_bits) - 1);
  for (int i = 0; i < j->n_q; ++i) {
    if (!is_finite(j->q_thr[i]) || (i > 0 && !(j->q_thr[i] > j->q_thr[i - 1])))
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "join: q_thr must be finite and strictly increasing");
  }
  if ((j->kind == IFQ_JOIN_CONV || j->kind == IFQ_JOIN_CONV_FUSED) && !j->coef)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "join: conv join needs coef");
  if (j->kind == IFQ_JOIN_CONV_FUSED) {
    const ifq_conv_desc& dd = j->down;
    int64_t dho, dwo;
    if (check_conv(&dd, &dho, &dwo) != IFQ_OK)
      return fail(IFQ_ERR_INVALID_ARGUMENT, "join: fused downsample: %s",
                  g_last_error.c_str());
    int64_t ho, wo;
    check_conv(d, &ho, &wo);
    if (!j->down_w)
      return fail(IFQ_ERR_INVALID_ARGUMENT, "join: fused downsample needs down_w");
    if (dd.kh != 1 || dd.kw != 1 || dd.pad != 0 || dd.in_bits != 2 || dd.out_bits != 0 ||
        dd.out_layout != IFQ_LAYOUT_I32_NHWC)
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "join: fused downsample must be 1x1, pad 0, 2-bit input, int32 output");
    if (dd.n != d->n || dd.c_out != d->c_out || dho != ho || dwo != wo)
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "join: fused downsample output must match the conv's (n, size, c_out)");
    if (j->layout != dd.in_layout)
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "join: fused shortcut layout must be the downsample's input layout");
  }
  if (j->kind == IFQ_JOIN_IDENTITY && !j->table)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "join: identity join needs table");
  if (j->kind == IFQ_JOIN_IDENTITY && j->sc_bits != 0 && j->sc_bits != 2)
    return fail(IFQ_ERR_UNSUPPORTED,
                "join: identity shortcut codes must be 2-bit (sc_bits %d)", j->sc_bits);
  if (j->kind == IFQ_JOIN_CONV && j->layout != IFQ_LAYOUT_I32_NHWC)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "join: conv shortcut must be I32_NHWC");
  if (j->kind == IFQ_JOIN_IDENTITY) {
    if (j->layout == IFQ_LAYOUT_U2_NHWC_PACKED) {
      if (d->c_out % 4)
        return fail(IFQ_ERR_INVALID_ARGUMENT,
                    "join: packed shortcut needs c_out %% 4 == 0");
    } else if (j->layout == IFQ_LAYOUT_U2_BLOCK64) {
      if (d->c_out % 64)
        return fail(IFQ_ERR_INVALID_ARGUMENT,
                    "join: BLOCK64 shortcut needs c_out %% 64 == 0");
    } else if (j->layout != IFQ_LAYOUT_I8_NHWC) {
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "join: identity shortcut must be codes (I8, U2 or BLOCK64)");
    }
  }
  return IFQ_OK;
}

// Resolve a validated conv into kernel arguments.
ifq::ConvLaunch make_launch(const ifq_conv_desc* d, int64_t ho, int64_t wo,
                            const void* x, const void* w, const int32_t* thr,
                            const ifq_join* join, const void* shortcut, void* y,
                            int32_t* acc_dump) {
  const ifq::WeightGeom g = ifq::weight_geom(*d);
  ifq::ConvLaunch a;
  std::memset(&a, 0, sizeof(a));
  a.x = static_cast<const uint8_t*>(x);
  a.wgt = static_cast<const int8_t*>(w);
  a.rowsum = w ? reinterpret_cast<const int32_t*>(static_cast<const uint8_t*>(w) +
                                                  g.rows_bytes)
                : nullptr;
  a.wzero = g.zero_off;
  a.thr = thr;
  a.y = y;
  a.acc_dump = acc_dump;
  a.join_kind = IFQ_JOIN_NONE;
  if (join && join->kind != IFQ_JOIN_NONE) {
    a.join_kind = join->kind;
    a.sc_layout = join->layout;
    a.shortcut = shortcut;
    a.coef = join->coef;
    a.table = join->table;
    for (int i = 0; i < join->n_q; ++i) a.qthr[i] = join->q_thr[i];
    if (join->kind == IFQ_JOIN_CONV_FUSED) {
      const ifq::WeightGeom gd = ifq::weight_geom(join->down);
      a.dx = static_cast<const uint8_t*>(shortcut);
      a.dwgt = static_cast<const int8_t*>(join->down_w);
      a.d_wzero = gd.zero_off;
      a.d_cin = join->down.c_in;
      a.d_h = join->down.h;
      a.d_w = join->down.w;
      a.d_stride = join->down.stride;
      a.d_nk32 = (int32_t)(gd.kpad / 32);
    }
  }
  a.nq = d->out_bits ? (1 << d->out_bits) - 1 : 0;
  a.rec = d->out_bits ? (1 << d->out_bits) : 0;
  a.n = d->n;
  a.h = d->h;
  a.w = d->w;
  a.cin = d->c_in;
  a.cout = d->c_out;
  a.cout_pad = (int32_t)g.cout_pad;
  a.kh = d->kh;
  a.kw = d->kw;
  a.stride = d->stride;
  a.pad = d->pad;
  a.ho = (int32_t)ho;
  a.wo = (int32_t)wo;
  a.m = (int32_t)((int64_t)d->n * ho * wo);
  a.kpad = (int32_t)g.kpad;
  a.nk = (int32_t)(g.kpad / ifq::kKStep);
  a.in_layout = d->in_layout;
  a.in_bits = d->in_bits;
  a.out_layout = d->out_layout;
  a.out_mode = d->out_bits == 0 ? 0 : d->out_layout == IFQ_LAYOUT_I8_NHWC ? 1 : 2;
  a.div_howo = ifq::make_fastdiv((uint32_t)(ho * wo > 0 ? ho * wo : 1));
  a.div_wo = ifq::make_fastdiv((uint32_t)(wo > 0 ? wo : 1));
  a.ksplit = 1;
  return a;
}

// A conv with a fused pool: both descs valid, the pool over the conv's own
// output (shape, code width, layout), non-overlapping valid windows that
// tile it exactly, codes out and no join.
ifq_status check_conv_pool(const ifq_conv_desc* d, const ifq_pool_desc* p, int64_t* ho,
                           int64_t* wo) {
  ifq_status st = check_conv(d, ho, wo);
  if (st != IFQ_OK) return st;
  int64_t pho, pwo;
  st = check_pool(p, &pho, &pwo);
  if (st != IFQ_OK) return st;
  if (p->n != d->n || p->h != *ho || p->w != *wo || p->c != d->c_out)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "conv+pool: pool input is not the conv output");
  if (d->out_bits == 0 || p->bits != d->out_bits || p->layout != d->out_layout)
    return fail(IFQ_ERR_INVALID_ARGUMENT,
                "conv+pool: codes out, with the pool's bits and layout the conv's");
  return IFQ_OK;
}

// Pool fields of a conv launch (p checked by check_conv_pool): tiles of
// whole window rows where the windows tile the output exactly, else of whole
// images.
void add_pool(ifq::ConvLaunch& a, const ifq_pool_desc& p) {
  int64_t pho, pwo;
  check_pool(&p, &pho, &pwo);
  a.pool_k = p.k;
  a.pool_s = p.stride;
  a.pool_same = p.mode == IFQ_POOL_SAME ? 1 : 0;
  a.pool_img = (p.mode == IFQ_POOL_VALID && p.k == p.stride && a.ho % p.k == 0 &&
                a.wo % p.k == 0) ? 0 : 1;
  a.pho = (int32_t)pho;
  a.pwo = (int32_t)pwo;
  a.div_pwo = ifq::make_fastdiv((uint32_t)(a.pwo > 0 ? a.pwo : 1));
  a.div_pho = ifq::make_fastdiv((uint32_t)(a.pho > 0 ? a.pho : 1));
}

// A BLOCK64 tensor of n images and c channels is pooled as the NHWC packed
// tensor of n*c/64 images of 64 channels it is laid out as.
ifq::PoolLaunch make_pool(const ifq_pool_desc& d, int64_t ho, int64_t wo,
                          const void* x, void* y) {
  ifq::PoolLaunch a;
  a.x = static_cast<const uint8_t*>(x);
  a.y = static_cast<uint8_t*>(y);
  const bool b64 = d.layout == IFQ_LAYOUT_U2_BLOCK64;
  a.n = b64 ? d.n * (d.c / 64) : d.n;
  a.h = d.h;
  a.w = d.w;
  a.c = b64 ? 64 : d.c;
  a.k = d.k;
  a.stride = d.stride;
  a.ho = (int32_t)ho;
  a.wo = (int32_t)wo;
  a.layout = b64 ? IFQ_LAYOUT_U2_NHWC_PACKED : d.layout;
  a.bits = d.bits;
  return a;
}

ifq_status hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess)
    return fail(IFQ_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
  return IFQ_OK;
}

ifq_status conv_args_check(const ifq_conv_desc* d, const void* x,
                           const void* w, const int32_t* thr,
                           const ifq_join* join, const void* shortcut,
                           const void* y) {
  const bool joined = join && join->kind != IFQ_JOIN_NONE;
  if (joined) {
    ifq_status st = check_join(join, d);
    if (st != IFQ_OK) return st;
    if (!shortcut) return fail(IFQ_ERR_INVALID_ARGUMENT, "join: shortcut is NULL");
    if (join->kind == IFQ_JOIN_CONV_FUSED) {
      int64_t ho, wo;
      check_conv(d, &ho, &wo);
      const ifq::ConvLaunch a =
          make_launch(d, ho, wo, x, w, thr, join, shortcut, const_cast<void*>(y), nullptr);
      if (!ifq::mfma_eligible(a) || !ifq::fused_supported(a))
        return fail(IFQ_ERR_UNSUPPORTED,
                    "join: no fused kernel for this conv and downsample shape");
    }
  }
  if (d->n > 0 && (!x || !w || !y))
    return fail(IFQ_ERR_INVALID_ARGUMENT, "conv: x, w_packed and y are required");
  // the kernels read the blob and the records with 16-byte loads
  if ((reinterpret_cast<uintptr_t>(w) & 15) || (reinterpret_cast<uintptr_t>(thr) & 15))
    return fail(IFQ_ERR_INVALID_ARGUMENT, "conv: w_packed and thr must be 16-byte aligned");
  const bool want_thr = d->out_bits != 0 && !joined;
  if (want_thr && !thr)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "conv: thresholds required");
  if (!want_thr && thr)
    return fail(IFQ_ERR_INVALID_ARGUMENT,
                "conv: thr must be NULL for int32 output or a join");
  return IFQ_OK;
}

// Checks of a fold's parameters shared by the table and the compact folds
// (the quantizer thresholds only where need_q), before anything is written.
ifq_status check_fold_params(const ifq_fold_params* p, bool need_q) {
  if (p->c_out < 1) return fail(IFQ_ERR_INVALID_ARGUMENT, "fold: c_out < 1");
  if (p->in_bits < 1 || p->in_bits > 8)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "fold: in_bits must be 1..8");
  if (p->out_bits < 1 || p->out_bits > 4)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "fold: out_bits must be 1..4");
  if (p->k < 1 || p->k * ((1 << p->in_bits) - 1) >= kMaxIndex / 2)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "fold: bad contraction length");
  if (!p->alpha || (need_q && !p->q_thr))
    return fail(IFQ_ERR_INVALID_ARGUMENT, "fold: alpha and q_thr are required");
  if (!(p->beta_in > 0.0) || !is_finite(p->beta_in))
    return fail(IFQ_ERR_INVALID_ARGUMENT, "fold: beta_in must be > 0");
  if (!is_finite(p->eps)) return fail(IFQ_ERR_INVALID_ARGUMENT, "fold: eps not finite");
  const int nq = (1 << p->out_bits) - 1;
  for (int i = 0; need_q && i < nq; ++i)
    if (!is_finite(p->q_thr[i]) || (i > 0 && !(p->q_thr[i] > p->q_thr[i - 1])))
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "fold: q_thr must be finite and strictly increasing");
  for (int c = 0; c < p->c_out; ++c) {
    const double al = p->alpha[c];
    const double bi = p->bias ? p->bias[c] : 0.0;
    const double mu = p->mean ? p->mean[c] : 0.0;
    const double va = p->var ? p->var[c] : 1.0;
    const double ga = p->gamma ? p->gamma[c] : 1.0;
    const double be = p->bn_beta ? p->bn_beta[c] : 0.0;
    if (!(al > 0.0) || !is_finite(al))
      return fail(IFQ_ERR_INVALID_ARGUMENT, "fold: alpha[%d] must be > 0", c);
    if (!is_finite(bi) || !is_finite(mu) || !is_finite(va) || !is_finite(ga) || !is_finite(be))
      return fail(IFQ_ERR_INVALID_ARGUMENT, "fold: channel %d not finite", c);
    if (!(va + p->eps > 0.0))
      return fail(IFQ_ERR_INVALID_ARGUMENT, "fold: var[%d] + eps must be > 0", c);
  }
  return IFQ_OK;
}

// fp4 weight blob: 1 KB per 32-row block and K64 step, then a zero block.
int64_t fp4_zero_off(const ifq::WeightGeom& g) { return (g.cout_pad / 32) * (g.kpad / 64) * 1024; }

// The fp4 kernels: the windowed kernel's 2-bit threshold epilogue on the
// transposed layout (the conditions of its packed 16-bit compares), no join,
// no pool, and a plan of the windowed kernel.
bool fp4_plan(const ifq::ConvLaunch& a, ifq::HaloPlan* hp) {
  const bool join_ok =
      a.join_kind == IFQ_JOIN_NONE || a.join_kind == IFQ_JOIN_CONV_FUSED ||
      (a.join_kind == IFQ_JOIN_IDENTITY && (a.sc_layout == IFQ_LAYOUT_U2_BLOCK64 ||
                                            a.sc_layout == IFQ_LAYOUT_U2_NHWC_PACKED));
  if (!(a.out_mode == 2 && a.rec == 4 && a.cout % 32 == 0 && 27 * a.cin <= 32766 && join_ok &&
        (a.pool_k == 0 || a.join_kind == IFQ_JOIN_NONE) && a.m > 0))
    return false;
  // only where the int8 plan's variant has an fp4 instance: the
  // 64-channel layers, whose two-workgroups-per-CU variant has none, measured
  // 16 -> 24 us on the 128-channel fp4 tiles (half their rows padding)
  ifq::HaloPlan h8;
  if (!ifq::plan_halo(a, &h8)) return false;
  ifq::ConvLaunch f = a;
  f.f4 = 1;   // the variants with an fp4 instance
  if (!ifq::plan_halo(f, hp)) return false;
  return hp->variant == h8.variant;
}

}  // namespace

extern "C" {

IFQ_API const char* ifq_version(void) { return "ifq 1.0.0 gfx950"; }

IFQ_API const char* ifq_last_error(void) { return g_last_error.c_str(); }

IFQ_API size_t ifq_tensor_bytes(int64_t n, int64_t h, int64_t w, int64_t c,
                                int32_t layout) {
  const int64_t b = tensor_bytes(n, h, w, c, layout);
  return b < 0 ? 0 : (size_t)b;
}

IFQ_API ifq_status ifq_conv_output_dims(const ifq_conv_desc* d, int32_t* ho,
                                        int32_t* wo) {
  int64_t h, w;
  ifq_status st = check_conv(d, &h, &w);
  if (st != IFQ_OK) return st;
  if (!ho || !wo) return fail(IFQ_ERR_INVALID_ARGUMENT, "NULL output pointer");
  *ho = (int32_t)h;
  *wo = (int32_t)w;
  return ok();
}

IFQ_API size_t ifq_packed_weight_bytes(const ifq_conv_desc* d) {
  if (check_conv(d) != IFQ_OK) return 0;
  return (size_t)ifq::weight_geom(*d).total_bytes;
}

IFQ_API ifq_status ifq_pack_weights(const ifq_conv_desc* d,
                                    const int8_t* w_oihw, void* dst,
                                    size_t dst_bytes) {
  ifq_status st = check_conv(d);
  if (st != IFQ_OK) return st;
  if (!w_oihw || !dst) return fail(IFQ_ERR_INVALID_ARGUMENT, "NULL pointer");
  const ifq::WeightGeom g = ifq::weight_geom(*d);
  if (dst_bytes < (size_t)g.total_bytes)
    return fail(IFQ_ERR_INSUFFICIENT_BUFFER, "pack: need %lld bytes, got %zu",
                (long long)g.total_bytes, dst_bytes);
  const int64_t total = (int64_t)d->c_out * d->c_in * d->kh * d->kw;
  for (int64_t i = 0; i < total; ++i)
    if (w_oihw[i] != 1 && w_oihw[i] != -1)
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "pack: weight %lld is %d, must be +1 or -1", (long long)i,
                  (int)w_oihw[i]);
  const bool mfma = ifq::mfma_layout(*d);
  const bool u2 = d->in_layout == IFQ_LAYOUT_U2_NHWC_PACKED;
  const int64_t nk32 = g.kpad / 32;
  const int64_t groups = d->c_in / 64;
  int8_t* rows = static_cast<int8_t*>(dst);
  int32_t* rowsum = reinterpret_cast<int32_t*>(static_cast<uint8_t*>(dst) + g.rows_bytes);
  std::memset(dst, 0, (size_t)g.total_bytes);
  for (int64_t co = 0; co < d->c_out; ++co) {
    int32_t sum = 0;
    for (int64_t r = 0; r < d->kh; ++r)
      for (int64_t s = 0; s < d->kw; ++s)
        for (int64_t c = 0; c < d->c_in; ++c) {
          const int8_t v = w_oihw[((co * d->c_in + c) * d->kh + r) * d->kw + s];
          const int64_t tap = r * d->kw + s;
          int64_t pos;
          if (mfma) {
            // K64 step kk = (c/64)*T + tap (T = kh*kw taps); channel
            // c' = c%64 = 32h + 16t + 4i + q sits in K32 step 2*kk + t,
            // lane 32h + co%32, byte 4q + i
            const int64_t kk = (c / 64) * (d->kh * d->kw) + tap, cp = c % 64;
            const int64_t h = cp / 32, t = (cp % 32) / 16, i = (cp % 16) / 4, q = cp % 4;
            const int64_t k32 = 2 * kk + t;
            const int64_t lane = 32 * h + co % 32;
            pos = (((co / 32) * nk32 + k32) * 64 + lane) * 16 + 4 * q + i;
          } else {
            int64_t cp = c;
            if (u2) {  // 4x4 transpose inside each group of 16 channels
              const int64_t base = c & ~(int64_t)15, in = c & 15;
              cp = base + (in & 3) * 4 + (in >> 2);
            }
            pos = co * g.kpad + tap * d->c_in + cp;
          }
          rows[pos] = v;
          sum += v;
        }
    rowsum[co] = sum;
  }
  return ok();
}

IFQ_API ifq_status ifq_fold_thresholds(const ifq_fold_params* p,
                                       int32_t* thr_out) {
  if (!p || !thr_out) return fail(IFQ_ERR_INVALID_ARGUMENT, "NULL pointer");
  ifq_status st = check_fold_params(p, true);
  if (st != IFQ_OK) return st;
  const int nq = (1 << p->out_bits) - 1;
  const int rec = nq + 1;
  const double bound = (double)p->k * (double)((1 << p->in_bits) - 1);
  for (int c = 0; c < p->c_out; ++c) {
    const double alpha = p->alpha[c];
    const double bias = p->bias ? p->bias[c] : 0.0;
    const double mean = p->mean ? p->mean[c] : 0.0;
    const double var = p->var ? p->var[c] : 1.0;
    const double gamma = p->gamma ? p->gamma[c] : 1.0;
    const double bn_beta = p->bn_beta ? p->bn_beta[c] : 0.0;
    int32_t* rec_c = thr_out + (int64_t)c * rec;
    const double sd = std::sqrt(var + p->eps);
    const double ab = alpha * p->beta_in;
    if (gamma == 0.0) {
      // BN output is the constant bn_beta: the code is #{i : bn_beta > q_i}
      rec_c[0] = 1;
      int level = 0;
      for (int i = 0; i < nq; ++i) level += bn_beta > p->q_thr[i] ? 1 : 0;
      for (int i = 0; i < nq; ++i)
        rec_c[1 + i] = i < level ? (int32_t)(-bound - 1.0) : (int32_t)bound;
      continue;
    }
    // a negative BN scale flips the direction of every comparison
    const double sign = gamma > 0.0 ? 1.0 : -1.0;
    rec_c[0] = gamma > 0.0 ? 1 : -1;
    for (int i = 0; i < nq; ++i) {
      double t = p->q_thr[i] - bn_beta;
      t = t * sd;
      t = t / gamma;
      t = t + mean;
      t = t - bias;
      t = t / ab;
      // integer sums: s*a > s*t  <=>  s*a > floor(s*t)
      double f = std::floor(sign * t);
      if (f < -bound - 1.0) f = -bound - 1.0;
      if (f > bound) f = bound;
      rec_c[1 + i] = (int32_t)f;
    }
  }
  return ok();
}

IFQ_API ifq_status ifq_fold_thresholds_compact(const ifq_fold_params* p, double base,
                                               double offset, ifq_thr_compact* out) {
  if (!p || !out) return fail(IFQ_ERR_INVALID_ARGUMENT, "NULL pointer");
  ifq_status st = check_fold_params(p, false);
  if (st != IFQ_OK) return st;
  if (!(base > 0.0) || !is_finite(base) || !is_finite(offset))
    return fail(IFQ_ERR_INVALID_ARGUMENT, "fold: base must be > 0 and offset finite");
  const int nq = (1 << p->out_bits) - 1;
  for (int c = 0; c < p->c_out; ++c) {
    const double alpha = p->alpha[c];
    const double bias = p->bias ? p->bias[c] : 0.0;
    const double mean = p->mean ? p->mean[c] : 0.0;
    const double var = p->var ? p->var[c] : 1.0;
    const double gamma = p->gamma ? p->gamma[c] : 1.0;
    const double bn_beta = p->bn_beta ? p->bn_beta[c] : 0.0;
    ifq_thr_compact& r = out[c];
    r.base = 0.0;
    r.offset = 0.0;
    r.cstar = 0;
    if (gamma == 0.0) {
      r.s = 0;
      for (int i = 1; i <= nq; ++i) {
        double q = (double)i * base;
        q = q + offset;
        r.cstar += bn_beta > q ? 1 : 0;
      }
      continue;
    }
    r.s = gamma > 0.0 ? 1 : -1;
    const double sd = std::sqrt(var + p->eps);
    const double ab = alpha * p->beta_in;
    double b = base * sd;
    b = b / gamma;
    r.base = b / ab;
    double o = offset - bn_beta;
    o = o * sd;
    o = o / gamma;
    o = o + mean;
    o = o - bias;
    r.offset = o / ab;
  }
  return ok();
}

IFQ_API ifq_status ifq_expand_thresholds(const ifq_thr_compact* recs, int32_t c_out,
                                         int32_t in_bits, int64_t k, int32_t out_bits,
                                         int32_t* thr, hipStream_t stream) {
  if (!recs || !thr) return fail(IFQ_ERR_INVALID_ARGUMENT, "expand: NULL pointer");
  if (c_out < 1 || in_bits < 1 || in_bits > 8 || out_bits < 1 || out_bits > 4 || k < 1 ||
      k * ((1 << in_bits) - 1) >= kMaxIndex / 2)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "expand: bad c_out, bits or k");
  const double bound = (double)k * (double)((1 << in_bits) - 1);
  ifq_status st = hip_status(ifq::launch_expand_thresholds(recs, c_out, out_bits, bound, thr,
                                                           stream),
                             "expand launch");
  if (st != IFQ_OK) return st;
  return ok();
}

IFQ_API ifq_status ifq_fold_join(const ifq_join_params* p, double* coef_out) {
  if (!p || !coef_out) return fail(IFQ_ERR_INVALID_ARGUMENT, "NULL pointer");
  if (p->c_out < 1) return fail(IFQ_ERR_INVALID_ARGUMENT, "join: c_out < 1");
  if (p->kind != IFQ_JOIN_IDENTITY && p->kind != IFQ_JOIN_CONV)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "join: bad kind %d", p->kind);
  const bool conv = p->kind == IFQ_JOIN_CONV;
  if (!p->alpha || !p->mean || !p->var || !p->gamma || !p->bn_beta)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "join: main-branch arrays required");
  if (conv && (!p->alpha_d || !p->mean_d || !p->var_d || !p->gamma_d || !p->bn_beta_d))
    return fail(IFQ_ERR_INVALID_ARGUMENT, "join: shortcut arrays required");
  if (!(p->beta_in > 0.0) || !is_finite(p->beta_in) || !(p->beta_x > 0.0) ||
      !is_finite(p->beta_x) || !is_finite(p->eps) || (conv && !is_finite(p->eps_d)))
    return fail(IFQ_ERR_INVALID_ARGUMENT, "join: steps must be > 0");
  for (int c = 0; c < p->c_out; ++c) {
    const double b = p->bias ? p->bias[c] : 0.0;
    if (!(p->alpha[c] > 0.0) || !is_finite(p->alpha[c]) || !is_finite(b) ||
        !is_finite(p->mean[c]) || !is_finite(p->gamma[c]) || !is_finite(p->bn_beta[c]) ||
        !is_finite(p->var[c]) || !(p->var[c] + p->eps > 0.0))
      return fail(IFQ_ERR_INVALID_ARGUMENT, "join: bad main channel %d", c);
    if (conv) {
      const double bd = p->bias_d ? p->bias_d[c] : 0.0;
      if (!(p->alpha_d[c] > 0.0) || !is_finite(p->alpha_d[c]) || !is_finite(bd) ||
          !is_finite(p->mean_d[c]) || !is_finite(p->gamma_d[c]) ||
          !is_finite(p->bn_beta_d[c]) || !is_finite(p->var_d[c]) ||
          !(p->var_d[c] + p->eps_d > 0.0))
        return fail(IFQ_ERR_INVALID_ARGUMENT, "join: bad shortcut channel %d", c);
    }
  }
  for (int c = 0; c < p->c_out; ++c) {
    const double sd = std::sqrt(p->var[c] + p->eps);
    double pm = p->alpha[c] * p->beta_in;
    pm = p->gamma[c] * pm;
    pm = pm / sd;
    double c2 = (p->bias ? p->bias[c] : 0.0) - p->mean[c];
    c2 = p->gamma[c] * c2;
    c2 = c2 / sd;
    c2 = c2 + p->bn_beta[c];
    double q = p->beta_x;
    double cd = 0.0;
    if (conv) {
      const double sdd = std::sqrt(p->var_d[c] + p->eps_d);
      q = p->alpha_d[c] * p->beta_x;
      q = p->gamma_d[c] * q;
      q = q / sdd;
      cd = (p->bias_d ? p->bias_d[c] : 0.0) - p->mean_d[c];
      cd = p->gamma_d[c] * cd;
      cd = cd / sdd;
      cd = cd + p->bn_beta_d[c];
    }
    coef_out[3 * c + 0] = pm;
    coef_out[3 * c + 1] = q;
    coef_out[3 * c + 2] = c2 + cd;
  }
  return ok();
}

IFQ_API ifq_status ifq_fold_join_table(const ifq_join_params* p, int32_t in_bits,
                                       int64_t k, int32_t x_bits, int32_t out_bits,
                                       const double* q_thr, int32_t* table_out) {
  if (!p || !q_thr || !table_out) return fail(IFQ_ERR_INVALID_ARGUMENT, "NULL pointer");
  if (p->kind != IFQ_JOIN_IDENTITY)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "join table: kind must be IFQ_JOIN_IDENTITY");
  if (in_bits < 1 || in_bits > 8 || x_bits < 1 || x_bits > 8 || out_bits < 1 ||
      out_bits > 4)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "join table: bad bit widths");
  if (k < 1 || k * ((1 << in_bits) - 1) >= kMaxIndex / 2)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "join table: bad contraction length");
  const int nq = (1 << out_bits) - 1;
  for (int i = 0; i < nq; ++i)
    if (!is_finite(q_thr[i]) || (i > 0 && !(q_thr[i] > q_thr[i - 1])))
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "join table: q_thr must be finite and strictly increasing");
  std::vector<double> coef((size_t)p->c_out * 3);
  ifq_status st = ifq_fold_join(p, coef.data());
  if (st != IFQ_OK) return st;
  const int64_t bound = k * ((1 << in_bits) - 1);
  const int nx = 1 << x_bits, rec = nq + 1;
  for (int c = 0; c < p->c_out; ++c) {
    const double pc = coef[3 * c], qc = coef[3 * c + 1], cc = coef[3 * c + 2];
    const int32_t s = pc < 0.0 ? -1 : 1;
    for (int x = 0; x < nx; ++x) {
      const double inner = std::fma(qc, (double)x, cc);
      int32_t* r = table_out + ((int64_t)c * nx + x) * rec;
      r[0] = s;
      for (int i = 0; i < nq; ++i) {
        // with u = s*a the join value is non-decreasing in u (fma is
        // correctly rounded), so "z > q_i" is false up to some u and true
        // after it: T_i is the last u where it is false
        auto pred = [&](int64_t u) {
          return std::fma(pc, (double)(s * u), inner) > q_thr[i];
        };
        int64_t t;
        if (pred(-bound)) {
          t = -bound - 1;
        } else if (!pred(bound)) {
          t = bound;
        } else {
          int64_t lo = -bound, hi = bound;  // pred(lo) false, pred(hi) true
          while (hi - lo > 1) {
            const int64_t mid = lo + (hi - lo) / 2;
            if (pred(mid)) hi = mid; else lo = mid;
          }
          t = lo;
        }
        r[1 + i] = (int32_t)t;
      }
    }
  }
  return ok();
}

IFQ_API const char* ifq_conv_kernel_name(const ifq_conv_desc* d, const ifq_join* join) {
  int64_t ho, wo;
  if (check_conv(d, &ho, &wo) != IFQ_OK) return "";
  const ifq::ConvLaunch a = make_launch(d, ho, wo, nullptr, nullptr, nullptr, join,
                                        nullptr, nullptr, nullptr);
  return ifq::conv_kernel_name(a);
}

IFQ_API int32_t ifq_conv_variant_count(void) { return ifq::reg3_variant_count(); }

IFQ_API int32_t ifq_conv_variant_fp4(int32_t variant) {
  if (variant < 0 || variant >= ifq::reg3_variant_count()) return -1;
  return ifq::reg3_variant_fp4(variant) ? 1 : 0;
}

IFQ_API const char* ifq_conv_variant_name(const ifq_conv_desc* d, const ifq_join* join,
                                          int32_t variant) {
  int64_t ho, wo;
  if (check_conv(d, &ho, &wo) != IFQ_OK) return "";
  ifq::ConvLaunch a = make_launch(d, ho, wo, nullptr, nullptr, nullptr, join, nullptr,
                                  nullptr, nullptr);
  a.f4 = ifq::reg3_variant_fp4(variant) ? 1 : 0;
  ifq::Reg3Plan p;
  if (variant < 0 || !ifq::plan_reg3(a, variant, &p)) return "";
  return ifq::reg3_name(p, a);
}

IFQ_API ifq_status ifq_conv_forward_variant(const ifq_conv_desc* d, const void* x,
                                            const void* w_packed, const int32_t* thr,
                                            const ifq_join* join, void* y, int32_t* acc_dump,
                                            int32_t variant, hipStream_t stream) {
  int64_t ho, wo;
  ifq_status st = check_conv(d, &ho, &wo);
  if (st != IFQ_OK) return st;
  const void* sc = (join && join->kind != IFQ_JOIN_NONE) ? join->shortcut : nullptr;
  st = conv_args_check(d, x, w_packed, thr, join, sc, y);
  if (st != IFQ_OK) return st;
  if (d->n == 0) return ok();
  ifq::ConvLaunch a = make_launch(d, ho, wo, x, w_packed, thr, join, sc, y, acc_dump);
  if (ifq::reg3_variant_fp4(variant)) {   // w_packed (and a fused join's down_w): fp4 blobs
    a.f4 = 1;
    a.rowsum = nullptr;
    a.wzero = fp4_zero_off(ifq::weight_geom(*d));
    if (a.join_kind == IFQ_JOIN_CONV_FUSED) a.d_wzero = fp4_zero_off(ifq::weight_geom(join->down));
  }
  ifq::Reg3Plan p;
  if (variant < 0 || !ifq::plan_reg3(a, variant, &p))
    return fail(IFQ_ERR_UNSUPPORTED, "conv variant %d: cannot take this layer", variant);
  st = hip_status(ifq::launch_reg3(a, p, stream), "conv variant launch");
  if (st != IFQ_OK) return st;
  return ok();
}

namespace {
// The plan of a forced K split (int8 register-blocked variant, thresholds).
bool split_plan(const ifq_conv_desc* d, int32_t variant, int32_t ksplit, ifq::ConvLaunch* a,
                ifq::W2Plan* p) {
  if (variant < 0 || variant >= ifq::w2_variant_count() || ifq::w2_variant_fp4(variant) ||
      ksplit < 2 || ksplit > 4 || d->out_bits == 0)
    return false;
  a->split_ok = 1;
  return ifq::plan_w2(*a, variant, p, ksplit) && p->ksplit == ksplit;
}
}  // namespace

IFQ_API size_t ifq_conv_split_workspace_bytes(const ifq_conv_desc* d, int32_t variant,
                                              int32_t ksplit) {
  int64_t ho, wo;
  if (!d || check_conv(d, &ho, &wo) != IFQ_OK || d->n == 0) return 0;
  ifq::ConvLaunch a = make_launch(d, ho, wo, nullptr, nullptr, nullptr, nullptr, nullptr,
                                  nullptr, nullptr);
  ifq::W2Plan p;
  if (!split_plan(d, variant, ksplit, &a, &p)) return 0;
  return (size_t)ifq::w2_split_bytes(a, p);
}

IFQ_API ifq_status ifq_conv_forward_split(const ifq_conv_desc* d, const void* x,
                                          const void* w_packed, const int32_t* thr, void* y,
                                          int32_t* acc_dump, int32_t variant, int32_t ksplit,
                                          void* ws, size_t ws_bytes, hipStream_t stream) {
  int64_t ho, wo;
  ifq_status st = check_conv(d, &ho, &wo);
  if (st != IFQ_OK) return st;
  st = conv_args_check(d, x, w_packed, thr, nullptr, nullptr, y);
  if (st != IFQ_OK) return st;
  if (d->n == 0) return ok();
  ifq::ConvLaunch a = make_launch(d, ho, wo, x, w_packed, thr, nullptr, nullptr, y, acc_dump);
  ifq::W2Plan p;
  if (!split_plan(d, variant, ksplit, &a, &p))
    return fail(IFQ_ERR_UNSUPPORTED, "conv split: variant %d cannot take this layer in %d",
                variant, ksplit);
  const int64_t need = ifq::w2_split_bytes(a, p);
  if ((int64_t)ws_bytes < need || !ws)
    return fail(IFQ_ERR_INSUFFICIENT_BUFFER, "conv split: workspace needs %lld bytes",
                (long long)need);
  a.ws_cnt = static_cast<uint32_t*>(ws);
  st = hip_status(ifq::launch_conv_w2(a, p, stream), "conv split launch");
  if (st != IFQ_OK) return st;
  return ok();
}

IFQ_API size_t ifq_conv_workspace_bytes(const ifq_conv_desc* d) {
  int64_t ho, wo;
  if (!d || check_conv(d, &ho, &wo) != IFQ_OK) return 0;
  ifq::ConvLaunch a = make_launch(d, ho, wo, nullptr, nullptr, nullptr, nullptr, nullptr,
                                  nullptr, nullptr);
  a.split_ok = 1;
  return (size_t)ifq::conv_workspace_bytes(a);
}

IFQ_API ifq_status ifq_conv_forward(const ifq_conv_desc* d, const void* x,
                                    const void* w_packed, const int32_t* thr,
                                    const ifq_join* join, void* y,
                                    int32_t* acc_dump, void* ws,
                                    size_t ws_bytes, hipStream_t stream) {
  int64_t ho, wo;
  ifq_status st = check_conv(d, &ho, &wo);
  if (st != IFQ_OK) return st;
  const void* sc = (join && join->kind != IFQ_JOIN_NONE) ? join->shortcut : nullptr;
  st = conv_args_check(d, x, w_packed, thr, join, sc, y);
  if (st != IFQ_OK) return st;
  const size_t need = ifq_conv_workspace_bytes(d);
  if (ws_bytes < need || (need && !ws))
    return fail(IFQ_ERR_INSUFFICIENT_BUFFER, "conv: workspace needs %zu bytes", need);
  ifq::ConvLaunch a = make_launch(d, ho, wo, x, w_packed, thr, join, sc, y, acc_dump);
  if (need) {   // the K split the workspace was sized for
    a.split_ok = 1;
    a.ws_cnt = static_cast<uint32_t*>(ws);
  }
  st = hip_status(ifq::launch_conv(a, stream), "conv launch");
  if (st != IFQ_OK) return st;
  return ok();
}

IFQ_API size_t ifq_packed_weight_bytes_fp4(const ifq_conv_desc* d) {
  if (check_conv(d) != IFQ_OK || !ifq::mfma_layout(*d)) return 0;
  const ifq::WeightGeom g = ifq::weight_geom(*d);
  return (size_t)(fp4_zero_off(g) + 1024);
}

IFQ_API ifq_status ifq_pack_weights_fp4(const ifq_conv_desc* d, const int8_t* w_oihw,
                                        void* dst, size_t dst_bytes) {
  ifq_status st = check_conv(d);
  if (st != IFQ_OK) return st;
  if (!w_oihw || !dst) return fail(IFQ_ERR_INVALID_ARGUMENT, "NULL pointer");
  if (!ifq::mfma_layout(*d))
    return fail(IFQ_ERR_INVALID_ARGUMENT,
                "pack fp4: needs in_bits 2, c_in %% 64 == 0 and a 2-bit packed input");
  const ifq::WeightGeom g = ifq::weight_geom(*d);
  const int64_t bytes = fp4_zero_off(g) + 1024;
  if (dst_bytes < (size_t)bytes)
    return fail(IFQ_ERR_INSUFFICIENT_BUFFER, "pack fp4: need %lld bytes, got %zu",
                (long long)bytes, dst_bytes);
  const int64_t total = (int64_t)d->c_out * d->c_in * d->kh * d->kw;
  for (int64_t i = 0; i < total; ++i)
    if (w_oihw[i] != 1 && w_oihw[i] != -1)
      return fail(IFQ_ERR_INVALID_ARGUMENT, "pack fp4: weight %lld is %d, must be +1 or -1",
                  (long long)i, (int)w_oihw[i]);
  uint8_t* out = static_cast<uint8_t*>(dst);
  std::memset(dst, 0, (size_t)bytes);
  const int64_t nk = g.kpad / 64;
  for (int64_t co = 0; co < d->c_out; ++co)
    for (int64_t r = 0; r < d->kh; ++r)
      for (int64_t s = 0; s < d->kw; ++s)
        for (int64_t c = 0; c < d->c_in; ++c) {
          const int8_t v = w_oihw[((co * d->c_in + c) * d->kh + r) * d->kw + s];
          // K64 step kk = (c/64)*T + tap; channel c' = c%64 = 32h + m sits in
          // lane 32h + co%32 at nibble 8*qw + j, where the kernel expands
          // code m = 16*(qw/2) + 2*j + qw%2 of the lane's half cell
          const int64_t kk = (c / 64) * (d->kh * d->kw) + r * d->kw + s, cp = c % 64;
          const int64_t h = cp / 32, m = cp % 32;
          const int64_t qw = 2 * (m / 16) + (m % 2), j = (m % 16) / 2;
          const int64_t lane = 32 * h + co % 32, nib = 8 * qw + j;
          const int64_t pos = (((co / 32) * nk + kk) * 64 + lane) * 16 + nib / 2;
          out[pos] |= (uint8_t)((v > 0 ? 0x4 : 0xC) << (4 * (nib % 2)));
        }
  return ok();
}

IFQ_API const char* ifq_conv_fp4_kernel_name(const ifq_conv_desc* d, const ifq_join* join) {
  int64_t ho, wo;
  if (check_conv(d, &ho, &wo) != IFQ_OK) return "";
  ifq::ConvLaunch a = make_launch(d, ho, wo, nullptr, nullptr, nullptr, join, nullptr,
                                  nullptr, nullptr);
  a.f4 = 1;
  ifq::Reg3Plan wp;
  if (ifq::plan_reg3(a, -1, &wp)) return ifq::reg3_name(wp, a);
  a.f4 = 0;
  ifq::HaloPlan hp;
  if (!fp4_plan(a, &hp)) return "";
  a.f4 = 1;
  return ifq::conv_halo_name(hp, a);
}

IFQ_API ifq_status ifq_conv_forward_fp4(const ifq_conv_desc* d, const void* x,
                                        const void* w_fp4, const int32_t* thr,
                                        const ifq_join* join, void* y, hipStream_t stream) {
  int64_t ho, wo;
  ifq_status st = check_conv(d, &ho, &wo);
  if (st != IFQ_OK) return st;
  const void* sc = (join && join->kind != IFQ_JOIN_NONE) ? join->shortcut : nullptr;
  st = conv_args_check(d, x, w_fp4, thr, join, sc, y);
  if (st != IFQ_OK) return st;
  ifq::ConvLaunch a = make_launch(d, ho, wo, x, w_fp4, thr, join, sc, y, nullptr);
  if (d->n == 0) return ok();
  // the register-blocked kernels' fp4 instances where they take the layer
  // (thresholds or an identity join), else the windowed kernel's
  ifq::Reg3Plan wp;
  {
    ifq::ConvLaunch f = a;
    f.f4 = 1;
    if (ifq::plan_reg3(f, -1, &wp)) {
      f.rowsum = nullptr;
      f.wzero = fp4_zero_off(ifq::weight_geom(*d));
      if (f.join_kind == IFQ_JOIN_CONV_FUSED)   // join->down_w is the down conv's fp4 blob
        f.d_wzero = fp4_zero_off(ifq::weight_geom(join->down));
      st = hip_status(ifq::launch_reg3(f, wp, stream), "conv fp4 launch");
      if (st != IFQ_OK) return st;
      return ok();
    }
  }
  ifq::HaloPlan hp;
  if (!fp4_plan(a, &hp))
    return fail(IFQ_ERR_UNSUPPORTED, "conv fp4: no fp4 kernel covers this layer");
  a.f4 = 1;
  a.rowsum = nullptr;
  a.wzero = fp4_zero_off(ifq::weight_geom(*d));
  if (a.join_kind == IFQ_JOIN_CONV_FUSED)   // join->down_w is the down conv's fp4 blob
    a.d_wzero = fp4_zero_off(ifq::weight_geom(join->down));
  st = hip_status(ifq::launch_conv_halo(a, hp, stream), "conv fp4 launch");
  if (st != IFQ_OK) return st;
  return ok();
}

IFQ_API const char* ifq_conv_pool_kernel_name(const ifq_conv_desc* d,
                                              const ifq_pool_desc* p) {
  int64_t ho, wo;
  if (check_conv_pool(d, p, &ho, &wo) != IFQ_OK) return "";
  ifq::ConvLaunch a = make_launch(d, ho, wo, nullptr, nullptr, nullptr, nullptr, nullptr,
                                  nullptr, nullptr);
  add_pool(a, *p);
  return ifq::conv_kernel_name(a);
}

IFQ_API ifq_status ifq_conv_pool_forward(const ifq_conv_desc* d, const ifq_pool_desc* p,
                                         const void* x, const void* w_packed,
                                         const int32_t* thr, void* y, hipStream_t stream) {
  int64_t ho, wo;
  ifq_status st = check_conv_pool(d, p, &ho, &wo);
  if (st != IFQ_OK) return st;
  st = conv_args_check(d, x, w_packed, thr, nullptr, nullptr, y);
  if (st != IFQ_OK) return st;
  if (d->n == 0) return ok();
  ifq::ConvLaunch a = make_launch(d, ho, wo, x, w_packed, thr, nullptr, nullptr, y, nullptr);
  add_pool(a, *p);
  if (!*ifq::conv_kernel_name(a))
    return fail(IFQ_ERR_UNSUPPORTED, "conv+pool: no fused kernel covers this shape");
  st = hip_status(ifq::launch_conv(a, stream), "conv+pool launch");
  if (st != IFQ_OK) return st;
  return ok();
}

IFQ_API const char* ifq_conv_pool_fp4_kernel_name(const ifq_conv_desc* d,
                                                  const ifq_pool_desc* p) {
  int64_t ho, wo;
  if (check_conv_pool(d, p, &ho, &wo) != IFQ_OK) return "";
  ifq::ConvLaunch a = make_launch(d, ho, wo, nullptr, nullptr, nullptr, nullptr, nullptr,
                                  nullptr, nullptr);
  add_pool(a, *p);
  ifq::HaloPlan hp;
  if (!ifq::mfma_eligible(a) || !fp4_plan(a, &hp)) return "";
  a.f4 = 1;
  return ifq::conv_halo_name(hp, a);
}

IFQ_API ifq_status ifq_conv_pool_forward_fp4(const ifq_conv_desc* d, const ifq_pool_desc* p,
                                             const void* x, const void* w_fp4,
                                             const int32_t* thr, void* y, hipStream_t stream) {
  int64_t ho, wo;
  ifq_status st = check_conv_pool(d, p, &ho, &wo);
  if (st != IFQ_OK) return st;
  st = conv_args_check(d, x, w_fp4, thr, nullptr, nullptr, y);
  if (st != IFQ_OK) return st;
  if (d->n == 0) return ok();
  ifq::ConvLaunch a = make_launch(d, ho, wo, x, w_fp4, thr, nullptr, nullptr, y, nullptr);
  add_pool(a, *p);
  ifq::HaloPlan hp;
  if (!ifq::mfma_eligible(a) || !fp4_plan(a, &hp))
    return fail(IFQ_ERR_UNSUPPORTED, "conv+pool fp4: no fp4 kernel covers this pair");
  a.f4 = 1;
  a.rowsum = nullptr;
  a.wzero = fp4_zero_off(ifq::weight_geom(*d));
  st = hip_status(ifq::launch_conv_halo(a, hp, stream), "conv+pool fp4 launch");
  if (st != IFQ_OK) return st;
  return ok();
}

IFQ_API ifq_status ifq_maxpool_codes(const ifq_pool_desc* d, const void* x,
                                     void* y, hipStream_t stream) {
  int64_t ho, wo;
  ifq_status st = check_pool(d, &ho, &wo);
  if (st != IFQ_OK) return st;
  if (d->n > 0 && (!x || !y)) return fail(IFQ_ERR_INVALID_ARGUMENT, "pool: NULL tensor");
  const ifq::PoolLaunch a = make_pool(*d, ho, wo, x, y);
  st = hip_status(ifq::launch_pool(a, stream), "pool launch");
  if (st != IFQ_OK) return st;
  return ok();
}

IFQ_API ifq_status ifq_convert_codes(int64_t n, int64_t h, int64_t w, int32_t c,
                                     int32_t src_layout, int32_t dst_layout,
                                     const void* src, void* dst,
                                     hipStream_t stream) {
  auto code_layout = [](int32_t l) {
    return l == IFQ_LAYOUT_I8_NHWC || l == IFQ_LAYOUT_U2_NHWC_PACKED ||
           l == IFQ_LAYOUT_U2_BLOCK64;
  };
  if (n < 0 || h < 0 || w < 0 || c < 1 || c % 4)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "convert: need n, h, w >= 0, c %% 4 == 0");
  if (!code_layout(src_layout) || !code_layout(dst_layout) || src_layout == dst_layout)
    return fail(IFQ_ERR_INVALID_ARGUMENT,
                "convert: layouts must be two different code layouts");
  if ((src_layout == IFQ_LAYOUT_U2_BLOCK64 || dst_layout == IFQ_LAYOUT_U2_BLOCK64) && c % 64)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "convert: BLOCK64 needs c %% 64 == 0");
  if (n * h * w * c >= kMaxIndex) return fail(IFQ_ERR_UNSUPPORTED, "convert: too large");
  if (n * h * w > 0 && (!src || !dst))
    return fail(IFQ_ERR_INVALID_ARGUMENT, "convert: NULL");
  ifq_status st = hip_status(
      ifq::launch_convert(n, h * w, c, src_layout, dst_layout, src, dst, stream),
      "convert launch");
  if (st != IFQ_OK) return st;
  return ok();
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Layer-chain driver
// ---------------------------------------------------------------------------
namespace {

struct SlotPlan {
  std::vector<int64_t> offset;  // byte offset of each work slot in ws
  std::vector<int64_t> bytes;   // capacity of each slot
  int64_t slots_bytes = 0;      // end of the slot area
  int64_t conv_ws = 0;          // per-conv workspace (shared by all layers)
  int64_t total = 0;
};

int64_t layer_out_bytes(const ifq_layer& L) {
  if (L.kind == IFQ_LAYER_CONV_POOL || L.kind == IFQ_LAYER_CONV_POOL_FP4) {
    // the pooled tensor (pool checked by plan_stack before this is used)
    int64_t pho = 0, pwo = 0;
    if (check_pool(&L.pool, &pho, &pwo) != IFQ_OK) return 0;
    return tensor_bytes(L.conv.n, pho, pwo, L.conv.c_out, L.conv.out_layout);
  }
  if (L.kind == IFQ_LAYER_CONV || L.kind == IFQ_LAYER_CONV_FP4) {
    const int64_t ho = out_extent(L.conv.h, L.conv.kh, L.conv.stride, L.conv.pad);
    const int64_t wo = out_extent(L.conv.w, L.conv.kw, L.conv.stride, L.conv.pad);
    return tensor_bytes(L.conv.n, ho, wo, L.conv.c_out, L.conv.out_layout);
  }
  int64_t ho, wo;
  if (L.pool.mode == IFQ_POOL_VALID) {
    ho = (L.pool.h - L.pool.k) / L.pool.stride + 1;
    wo = (L.pool.w - L.pool.k) / L.pool.stride + 1;
  } else {
    ho = (L.pool.h + L.pool.stride - 1) / L.pool.stride;
    wo = (L.pool.w + L.pool.stride - 1) / L.pool.stride;
  }
  return tensor_bytes(L.pool.n, ho, wo, L.pool.c, L.pool.layout);
}

int64_t layer_in_bytes(const ifq_layer& L) {
  if (L.kind == IFQ_LAYER_CONV || L.kind == IFQ_LAYER_CONV_POOL || L.kind == IFQ_LAYER_CONV_FP4 ||
      L.kind == IFQ_LAYER_CONV_POOL_FP4)
    return tensor_bytes(L.conv.n, L.conv.h, L.conv.w, L.conv.c_in, L.conv.in_layout);
  return tensor_bytes(L.pool.n, L.pool.h, L.pool.w, L.pool.c, L.pool.layout);
}

// Bytes the join of a conv layer reads from its join_src slot: the block
// input codes [n][ho][wo][c_out] (identity), the downsample's int32 sums
// (conv) or the downsample's input codes (fused downsample); 0 without a join.
int64_t join_in_bytes(const ifq_layer& L) {
  if (L.kind != IFQ_LAYER_CONV && L.kind != IFQ_LAYER_CONV_FP4) return 0;
  const ifq_join& j = L.join;
  const int64_t ho = out_extent(L.conv.h, L.conv.kh, L.conv.stride, L.conv.pad);
  const int64_t wo = out_extent(L.conv.w, L.conv.kw, L.conv.stride, L.conv.pad);
  switch (j.kind) {
    case IFQ_JOIN_IDENTITY: return tensor_bytes(L.conv.n, ho, wo, L.conv.c_out, j.layout);
    case IFQ_JOIN_CONV:
      return tensor_bytes(L.conv.n, ho, wo, L.conv.c_out, IFQ_LAYOUT_I32_NHWC);
    case IFQ_JOIN_CONV_FUSED:
      return tensor_bytes(j.down.n, j.down.h, j.down.w, j.down.c_in, j.down.in_layout);
    default: return 0;
  }
}

// Code width a layer writes into its dst slot (0: int32 sums).
int layer_out_bits(const ifq_layer& L) {
  return L.kind == IFQ_LAYER_POOL ? L.pool.bits : L.conv.out_bits;
}

ifq_status plan_stack(const ifq_stack* s, SlotPlan* plan) {
  if (!s) return fail(IFQ_ERR_INVALID_ARGUMENT, "stack is NULL");
  if (s->n_layers < 0 || (s->n_layers > 0 && !s->layers))
    return fail(IFQ_ERR_INVALID_ARGUMENT, "stack: bad layer array");
  if (s->n_slots < 2) return fail(IFQ_ERR_INVALID_ARGUMENT, "stack: n_slots < 2");
  plan->offset.assign(s->n_slots, 0);
  plan->bytes.assign(s->n_slots, 0);
  std::vector<char> written(s->n_slots, 0);
  written[0] = 1;
  // bytes and code width of the last write of each slot (the caller's x
  // and y have no size known here; their bits are unknown, -1)
  std::vector<int64_t> last_bytes(s->n_slots, 0);
  std::vector<int> last_bits(s->n_slots, -1);
  for (int i = 0; i < s->n_layers; ++i) {
    const ifq_layer& L = s->layers[i];
    ifq_status st;
    if (L.kind == IFQ_LAYER_CONV) {
      st = check_conv(&L.conv);
      if (st != IFQ_OK) return fail(st, "layer %d: %s", i, g_last_error.c_str());
      const bool joined = L.join.kind != IFQ_JOIN_NONE;
      st = conv_args_check(&L.conv, (const void*)1, L.w_packed, L.thr, &L.join,
                           joined ? (const void*)1 : nullptr, (const void*)1);
      if (st != IFQ_OK) return fail(st, "layer %d: %s", i, g_last_error.c_str());
      if (joined) {
        if (L.join_src < 0 || L.join_src >= s->n_slots || !written[L.join_src] ||
            L.join_src == L.dst)
          return fail(IFQ_ERR_INVALID_ARGUMENT,
                      "layer %d: join slot %d not written before", i, L.join_src);
      }
      plan->conv_ws = std::max<int64_t>(plan->conv_ws,
                                        (int64_t)ifq_conv_workspace_bytes(&L.conv));
    } else if (L.kind == IFQ_LAYER_POOL) {
      int64_t ho, wo;
      st = check_pool(&L.pool, &ho, &wo);
      if (st != IFQ_OK) return fail(st, "layer %d: %s", i, g_last_error.c_str());
    } else if (L.kind == IFQ_LAYER_CONV_FP4) {
      st = check_conv(&L.conv);
      if (st != IFQ_OK) return fail(st, "layer %d: %s", i, g_last_error.c_str());
      const bool joined = L.join.kind != IFQ_JOIN_NONE;
      st = conv_args_check(&L.conv, (const void*)1, L.w_packed, L.thr, &L.join,
                           joined ? (const void*)1 : nullptr, (const void*)1);
      if (st != IFQ_OK) return fail(st, "layer %d: %s", i, g_last_error.c_str());
      if (joined && (L.join_src < 0 || L.join_src >= s->n_slots || !written[L.join_src] ||
                     L.join_src == L.dst))
        return fail(IFQ_ERR_INVALID_ARGUMENT, "layer %d: join slot %d not written before", i,
                    L.join_src);
      if (L.conv.n > 0 && !*ifq_conv_fp4_kernel_name(&L.conv, &L.join))
        return fail(IFQ_ERR_UNSUPPORTED, "layer %d: no fp4 kernel covers it", i);
    } else if (L.kind == IFQ_LAYER_CONV_POOL_FP4) {
      int64_t ho, wo;
      st = check_conv_pool(&L.conv, &L.pool, &ho, &wo);
      if (st != IFQ_OK) return fail(st, "layer %d: %s", i, g_last_error.c_str());
      st = conv_args_check(&L.conv, (const void*)1, L.w_packed, L.thr, nullptr, nullptr,
                           (const void*)1);
      if (st != IFQ_OK) return fail(st, "layer %d: %s", i, g_last_error.c_str());
      if (L.conv.n > 0 && !*ifq_conv_pool_fp4_kernel_name(&L.conv, &L.pool))
        return fail(IFQ_ERR_UNSUPPORTED, "layer %d: no fp4 conv+pool kernel covers it", i);
    } else if (L.kind == IFQ_LAYER_CONV_POOL) {
      int64_t ho, wo;
      st = check_conv_pool(&L.conv, &L.pool, &ho, &wo);
      if (st != IFQ_OK) return fail(st, "layer %d: %s", i, g_last_error.c_str());
      st = conv_args_check(&L.conv, (const void*)1, L.w_packed, L.thr, nullptr, nullptr,
                           (const void*)1);
      if (st != IFQ_OK) return fail(st, "layer %d: %s", i, g_last_error.c_str());
      if (L.conv.n > 0 && !*ifq_conv_pool_kernel_name(&L.conv, &L.pool))
        return fail(IFQ_ERR_UNSUPPORTED, "layer %d: no fused conv+pool kernel covers it", i);
    } else {
      return fail(IFQ_ERR_INVALID_ARGUMENT, "layer %d: bad kind %d", i, L.kind);
    }
    if (L.src < 0 || L.src >= s->n_slots || !written[L.src])
      return fail(IFQ_ERR_INVALID_ARGUMENT, "layer %d: src slot %d not written before",
                  i, L.src);
    if (L.dst < 1 || L.dst >= s->n_slots || L.dst == L.src)
      return fail(IFQ_ERR_INVALID_ARGUMENT, "layer %d: bad dst slot %d", i, L.dst);
    if (L.src >= 2 && layer_in_bytes(L) > last_bytes[L.src])
      return fail(IFQ_ERR_INVALID_ARGUMENT,
                  "layer %d: reads %lld bytes from slot %d holding %lld", i,
                  (long long)layer_in_bytes(L), L.src, (long long)last_bytes[L.src]);
    const bool joins = (L.kind == IFQ_LAYER_CONV || L.kind == IFQ_LAYER_CONV_FP4) &&
                       L.join.kind != IFQ_JOIN_NONE;
    if (joins) {
      const int64_t jb = join_in_bytes(L);
      if (jb < 0 || (L.join_src >= 2 && jb > last_bytes[L.join_src]))
        return fail(IFQ_ERR_INVALID_ARGUMENT,
                    "layer %d: the join reads %lld bytes from slot %d holding %lld", i,
                    (long long)jb, L.join_src, (long long)last_bytes[L.join_src]);
      if (L.join.kind == IFQ_JOIN_IDENTITY && last_bits[L.join_src] >= 0 &&
          last_bits[L.join_src] != 2)
        return fail(IFQ_ERR_UNSUPPORTED,
                    "layer %d: identity shortcut slot %d holds %d-bit codes (2-bit only)", i,
                    L.join_src, last_bits[L.join_src]);
    }
    const int64_t ob = layer_out_bytes(L);
    if (ob > plan->bytes[L.dst]) plan->bytes[L.dst] = ob;
    last_bytes[L.dst] = ob;
    last_bits[L.dst] = layer_out_bits(L);
    written[L.dst] = 1;
  }
  // the conv workspace first, its K-split counters at offset 0 for every
  // stack (at least the counter region, so that no stack's slots overwrite
  // another's counters in a shared workspace), then the slots
  plan->conv_ws = ifq::round_up(std::max<int64_t>(plan->conv_ws, ifq::kSplitCounterBytes), 256);
  int64_t off = plan->conv_ws;
  for (int k = 2; k < s->n_slots; ++k) {
    plan->offset[k] = off;
    off += ifq::round_up(plan->bytes[k], 256);
  }
  plan->slots_bytes = off;
  plan->total = off;
  return IFQ_OK;
}

}  // namespace

extern "C" {

IFQ_API size_t ifq_stack_workspace_bytes(const ifq_stack* s) {
  SlotPlan plan;
  if (plan_stack(s, &plan) != IFQ_OK) return 0;
  return (size_t)plan.total;
}

IFQ_API ifq_status ifq_stack_slot_info(const ifq_stack* s, int32_t slot,
                                       size_t* offset, size_t* bytes) {
  SlotPlan plan;
  ifq_status st = plan_stack(s, &plan);
  if (st != IFQ_OK) return st;
  if (slot < 2 || slot >= s->n_slots || !offset || !bytes)
    return fail(IFQ_ERR_INVALID_ARGUMENT, "slot_info: bad slot %d", slot);
  *offset = (size_t)plan.offset[slot];
  *bytes = (size_t)plan.bytes[slot];
  return ok();
}

IFQ_API ifq_status ifq_run_stack(const ifq_stack* s, const void* x, void* y,
                                 void* ws, size_t ws_bytes, hipStream_t stream) {
  SlotPlan plan;
  ifq_status st = plan_stack(s, &plan);
  if (st != IFQ_OK) return st;
  if ((int64_t)ws_bytes < plan.total || (plan.total > 0 && !ws))
    return fail(IFQ_ERR_INSUFFICIENT_BUFFER, "stack: workspace needs %lld bytes",
                (long long)plan.total);
  if (!x || !y) return fail(IFQ_ERR_INVALID_ARGUMENT, "stack: x and y are required");
  uint8_t* base = static_cast<uint8_t*>(ws);
  auto slot = [&](int k) -> void* {
    if (k == 0) return const_cast<void*>(x);
    if (k == 1) return y;
    return base + plan.offset[k];
  };
  void* conv_ws = base;   // offset 0: the K-split counters, then partials
  for (int i = 0; i < s->n_layers; ++i) {
    const ifq_layer& L = s->layers[i];
    if (s->events) {
      st = hip_status(hipEventRecord(s->events[i], stream), "event record");
      if (st != IFQ_OK) return st;
    }
    if (L.kind == IFQ_LAYER_CONV) {
      ifq_join j = L.join;
      const void* sc = nullptr;
      if (j.kind != IFQ_JOIN_NONE) sc = slot(L.join_src);
      int64_t ho = out_extent(L.conv.h, L.conv.kh, L.conv.stride, L.conv.pad);
      int64_t wo = out_extent(L.conv.w, L.conv.kw, L.conv.stride, L.conv.pad);
      ifq::ConvLaunch a = make_launch(&L.conv, ho, wo, slot(L.src), L.w_packed,
                                      L.thr, &j, sc, slot(L.dst), nullptr);
      if (ifq_conv_workspace_bytes(&L.conv) > 0) {   // sized into plan.conv_ws
        a.split_ok = 1;
        a.ws_cnt = static_cast<uint32_t*>(conv_ws);
      }
      st = hip_status(ifq::launch_conv(a, stream), "conv launch");
    } else if (L.kind == IFQ_LAYER_CONV_POOL_FP4) {
      st = ifq_conv_pool_forward_fp4(&L.conv, &L.pool, slot(L.src), L.w_packed, L.thr,
                                     slot(L.dst), stream);
    } else if (L.kind == IFQ_LAYER_CONV_FP4) {
      ifq_join j = L.join;
      if (j.kind != IFQ_JOIN_NONE) j.shortcut = slot(L.join_src);
      st = ifq_conv_forward_fp4(&L.conv, slot(L.src), L.w_packed, L.thr, &j, slot(L.dst),
                                stream);
    } else if (L.kind == IFQ_LAYER_CONV_POOL) {
      int64_t ho = out_extent(L.conv.h, L.conv.kh, L.conv.stride, L.conv.pad);
      int64_t wo = out_extent(L.conv.w, L.conv.kw, L.conv.stride, L.conv.pad);
      ifq::ConvLaunch a = make_launch(&L.conv, ho, wo, slot(L.src), L.w_packed, L.thr,
                                      nullptr, nullptr, slot(L.dst), nullptr);
      add_pool(a, L.pool);
      st = hip_status(ifq::launch_conv(a, stream), "conv+pool launch");
    } else {
      int64_t ho, wo;
      check_pool(&L.pool, &ho, &wo);
      const ifq::PoolLaunch a = make_pool(L.pool, ho, wo, slot(L.src), slot(L.dst));
      st = hip_status(ifq::launch_pool(a, stream), "pool launch");
    }
    if (st != IFQ_OK) return fail(st, "layer %d: %s", i, g_last_error.c_str());
  }
  if (s->events) {
    st = hip_status(hipEventRecord(s->events[s->n_layers], stream), "event record");
    if (st != IFQ_OK) return st;
  }
  return ok();
}

}  // extern "C"
