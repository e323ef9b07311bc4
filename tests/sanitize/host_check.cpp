// Host-side calls of libifq under AddressSanitizer and UndefinedBehavior-
// Sanitizer: descriptor checks, weight packing, threshold and join folding,
// kernel planning for many layer shapes, and stack validation. Nothing here
// touches a GPU; device pointers are placeholders that are never
// dereferenced. Exit status 0 when every call returned the expected status.
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <vector>

#include "ifq.h"

static int g_fail = 0;

#define EXPECT(cond)                                                          \
  do {                                                                        \
    if (!(cond)) {                                                            \
      std::fprintf(stderr, "%s:%d: %s (%s)\n", __FILE__, __LINE__, #cond,     \
                   ifq_last_error());                                         \
      ++g_fail;                                                               \
    }                                                                         \
  } while (0)

static ifq_conv_desc desc(int n, int h, int w, int cin, int cout, int k, int st, int pad,
                          int ib, int ob, int il, int ol) {
  ifq_conv_desc d;
  d.n = n; d.h = h; d.w = w; d.c_in = cin; d.c_out = cout;
  d.kh = k; d.kw = k; d.stride = st; d.pad = pad;
  d.in_bits = ib; d.out_bits = ob; d.in_layout = il; d.out_layout = ol;
  return d;
}

static void conv_shapes(std::mt19937& rng) {
  const int B64 = IFQ_LAYOUT_U2_BLOCK64, U2 = IFQ_LAYOUT_U2_NHWC_PACKED,
            I8 = IFQ_LAYOUT_I8_NHWC, I32 = IFQ_LAYOUT_I32_NHWC;
  std::vector<ifq_conv_desc> ds = {
      desc(64, 56, 56, 64, 64, 3, 1, 1, 2, 2, B64, B64),
      desc(64, 56, 56, 64, 128, 3, 2, 1, 2, 2, B64, B64),
      desc(64, 28, 28, 128, 128, 3, 1, 1, 2, 2, B64, B64),
      desc(64, 14, 14, 256, 256, 3, 1, 1, 2, 2, B64, B64),
      desc(64, 7, 7, 512, 512, 3, 1, 1, 2, 2, B64, B64),
      desc(64, 56, 56, 64, 128, 1, 2, 0, 2, 0, B64, I32),
      desc(3, 13, 11, 64, 96, 3, 1, 1, 2, 2, B64, U2),
      desc(2, 6, 6, 1024, 64, 3, 1, 1, 2, 2, B64, B64),
      desc(8, 416, 416, 3, 16, 3, 1, 1, 8, 2, I8, U2),
      desc(8, 208, 208, 16, 32, 3, 1, 1, 2, 2, U2, U2),
      desc(8, 104, 104, 32, 64, 3, 1, 1, 2, 2, U2, B64),
      desc(3, 1, 1, 32, 36, 3, 1, 1, 2, 2, U2, U2),
      desc(32, 27, 27, 96, 256, 5, 1, 2, 2, 2, I8, I8),
      desc(8, 13, 13, 512, 30, 1, 1, 0, 2, 0, B64, I32),
      desc(2, 9, 9, 32, 200, 3, 1, 1, 2, 4, I8, I8),
      desc(1, 1, 1, 64, 64, 3, 1, 1, 2, 2, B64, B64),
      desc(0, 5, 5, 64, 64, 3, 1, 1, 2, 2, B64, B64),      // no pixels
      desc(1, 5, 5, 60, 64, 3, 1, 1, 2, 2, B64, B64),      // c_in not a multiple of 64
      desc(1, 5, 5, 64, 64, 7, 1, 0, 2, 2, B64, B64),      // no output pixel
      desc(1, 5, 5, 64, 64, 3, 0, 1, 2, 2, B64, B64),      // stride 0
  };
  const int nvar = ifq_conv_variant_count();
  EXPECT(nvar > 0);
  EXPECT(ifq_conv_variant_fp4(-1) == -1 && ifq_conv_variant_fp4(nvar) == -1);
  for (const ifq_conv_desc& d : ds) {
    int32_t ho = -1, wo = -1;
    const ifq_status st = ifq_conv_output_dims(&d, &ho, &wo);
    (void)ifq_conv_kernel_name(&d, nullptr);
    (void)ifq_conv_fp4_kernel_name(&d, nullptr);
    (void)ifq_conv_workspace_bytes(&d);
    for (int v = 0; v < nvar; ++v) (void)ifq_conv_variant_name(&d, nullptr, v);
    ifq_join j;
    std::memset(&j, 0, sizeof(j));
    j.kind = IFQ_JOIN_IDENTITY;
    j.layout = d.out_layout;
    j.table = reinterpret_cast<const int32_t*>(0x1000);
    j.n_q = 3;
    (void)ifq_conv_kernel_name(&d, &j);
    for (int v = 0; v < nvar; ++v) (void)ifq_conv_variant_name(&d, &j, v);
    ifq_pool_desc p;
    p.n = d.n; p.h = ho > 0 ? ho : 1; p.w = wo > 0 ? wo : 1; p.c = d.c_out;
    p.k = 2; p.stride = 2; p.mode = IFQ_POOL_VALID; p.bits = d.out_bits;
    p.layout = d.out_layout;
    (void)ifq_conv_pool_kernel_name(&d, &p);
    (void)ifq_conv_pool_fp4_kernel_name(&d, &p);
    if (st != IFQ_OK) continue;
    const size_t wb = ifq_packed_weight_bytes(&d);
    const size_t nw = (size_t)d.c_out * d.c_in * d.kh * d.kw;
    if (wb == 0 || nw > (size_t)1 << 26) continue;
    std::vector<int8_t> w(nw);
    for (auto& e : w) e = (rng() & 1) ? 1 : -1;
    std::vector<uint8_t> blob(wb);
    EXPECT(ifq_pack_weights(&d, w.data(), blob.data(), blob.size()) == IFQ_OK);
    EXPECT(ifq_pack_weights(&d, w.data(), blob.data(), blob.size() - 1) ==
           IFQ_ERR_INSUFFICIENT_BUFFER);
    w[nw / 2] = 0;
    EXPECT(ifq_pack_weights(&d, w.data(), blob.data(), blob.size()) ==
           IFQ_ERR_INVALID_ARGUMENT);
    w[nw / 2] = 1;
    const size_t fb = ifq_packed_weight_bytes_fp4(&d);
    if (fb) {
      std::vector<uint8_t> f(fb);
      EXPECT(ifq_pack_weights_fp4(&d, w.data(), f.data(), f.size()) == IFQ_OK);
    }
  }
  for (int layout = -1; layout <= 4; ++layout)
    for (int c : {3, 16, 64, 100})
      (void)ifq_tensor_bytes(2, 7, 9, c, layout);
}

static void folds(std::mt19937& rng) {
  std::uniform_real_distribution<double> u(0.0, 1.0);
  std::normal_distribution<double> nd(0.0, 1.0);
  const int c_out = 37;
  std::vector<double> alpha(c_out), bias(c_out), mean(c_out), var(c_out), gamma(c_out),
      beta(c_out);
  for (int c = 0; c < c_out; ++c) {
    alpha[c] = 0.01 + 0.09 * u(rng);
    bias[c] = 0.1 * nd(rng);
    mean[c] = 2.0 * nd(rng);
    var[c] = 0.5 + 1.5 * u(rng);
    gamma[c] = (0.5 + u(rng)) * (c % 10 == 3 ? -1.0 : 1.0);
    beta[c] = nd(rng);
  }
  gamma[5] = 0.0;
  for (int ob = 1; ob <= 4; ++ob) {
    const int nq = (1 << ob) - 1;
    std::vector<double> q(nq);
    for (int i = 0; i < nq; ++i) q[i] = 0.25 + 0.5 * i;
    ifq_fold_params p;
    std::memset(&p, 0, sizeof(p));
    p.c_out = c_out; p.in_bits = 2; p.out_bits = ob; p.k = 576;
    p.alpha = alpha.data(); p.beta_in = 0.5; p.bias = bias.data(); p.mean = mean.data();
    p.var = var.data(); p.gamma = gamma.data(); p.bn_beta = beta.data(); p.eps = 1e-5;
    p.q_thr = q.data();
    std::vector<int32_t> thr((size_t)c_out * (1 << ob));
    EXPECT(ifq_fold_thresholds(&p, thr.data()) == IFQ_OK);
    std::vector<ifq_thr_compact> rec(c_out);
    (void)ifq_fold_thresholds_compact(&p, 0.5, -0.25, rec.data());
    p.eps = -1.0;
    EXPECT(ifq_fold_thresholds(&p, thr.data()) != IFQ_OK);
    p.eps = 1e-5;
    EXPECT(ifq_fold_thresholds(nullptr, thr.data()) != IFQ_OK);
  }
  for (int kind : {IFQ_JOIN_IDENTITY, IFQ_JOIN_CONV}) {
    ifq_join_params jp;
    std::memset(&jp, 0, sizeof(jp));
    jp.c_out = c_out; jp.kind = kind; jp.alpha = alpha.data(); jp.beta_in = 0.5;
    jp.bias = bias.data(); jp.mean = mean.data(); jp.var = var.data(); jp.gamma = gamma.data();
    jp.bn_beta = beta.data(); jp.eps = 1e-5; jp.beta_x = 0.5;
    jp.alpha_d = alpha.data(); jp.bias_d = bias.data(); jp.mean_d = mean.data();
    jp.var_d = var.data(); jp.gamma_d = gamma.data(); jp.bn_beta_d = beta.data();
    jp.eps_d = 1e-5;
    std::vector<double> coef((size_t)c_out * 3);
    EXPECT(ifq_fold_join(&jp, coef.data()) == IFQ_OK);
    if (kind == IFQ_JOIN_IDENTITY) {
      const double q[3] = {0.25, 0.75, 1.25};
      std::vector<int32_t> table((size_t)c_out * 16);
      EXPECT(ifq_fold_join_table(&jp, 2, 576, 2, 2, q, table.data()) == IFQ_OK);
    }
  }
}

static void stacks() {
  const int B64 = IFQ_LAYOUT_U2_BLOCK64;
  const void* fake = reinterpret_cast<const void*>(0x1000);
  std::vector<ifq_layer> L(3);
  std::memset(L.data(), 0, sizeof(ifq_layer) * L.size());
  for (int i = 0; i < 3; ++i) {
    L[i].kind = IFQ_LAYER_CONV;
    L[i].conv = desc(4, 14, 14, 64, 64, 3, 1, 1, 2, 2, B64, B64);
    L[i].w_packed = fake;
    L[i].thr = reinterpret_cast<const int32_t*>(fake);
    L[i].join_src = -1;
  }
  L[0].src = 0; L[0].dst = 2;
  L[1].src = 2; L[1].dst = 3;
  L[2].src = 3; L[2].dst = 1;
  L[2].join.kind = IFQ_JOIN_IDENTITY;
  L[2].join.layout = B64;
  L[2].join.table = reinterpret_cast<const int32_t*>(fake);
  L[2].join.n_q = 3;
  L[2].join.q_thr[0] = 0.25;
  L[2].join.q_thr[1] = 0.75;
  L[2].join.q_thr[2] = 1.25;
  L[2].join_src = 2;
  L[2].thr = nullptr;
  ifq_stack s;
  s.n_layers = 3; s.n_slots = 4; s.layers = L.data(); s.events = nullptr;
  const size_t ws = ifq_stack_workspace_bytes(&s);
  EXPECT(ws > 0);
  size_t off = 0, bytes = 0;
  EXPECT(ifq_stack_slot_info(&s, 2, &off, &bytes) == IFQ_OK);
  EXPECT(ifq_stack_slot_info(&s, 9, &off, &bytes) != IFQ_OK);
  L[1].conv.c_in = 128;   // disagrees with the tensor slot 2 holds
  EXPECT(ifq_stack_workspace_bytes(&s) == 0);
  L[1].conv.c_in = 64;
  L[2].join_src = 7;      // no such slot
  EXPECT(ifq_stack_workspace_bytes(&s) == 0);
}

int main() {
  std::printf("%s\n", ifq_version());
  std::mt19937 rng(2026);
  conv_shapes(rng);
  folds(rng);
  stacks();
  if (g_fail) {
    std::fprintf(stderr, "%d check(s) failed\n", g_fail);
    return 1;
  }
  std::printf("host checks passed\n");
  return 0;
}
