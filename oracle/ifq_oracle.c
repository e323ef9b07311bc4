/*
 * Plain CPU oracle for the integrated fixed-point quantized convolution of
 * IFQ-Net (Integrated Fixed-point Quantization Networks for Embedded Vision).
 *
 * TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
 * baseline may load this library. It shares no code with the GPU library.
 *
 * Each function follows the paper's statement of the layer:
 *   oracle_conv_acc   integer part of Eq. (1): W_b (x) X_q, accumulated in int64
 *   oracle_fold       Eq. (6) -> Eq. (7): thresholds moved onto the integer
 *                     side, then floored (Sec. 3.2), with the comparison
 *                     direction flipped for channels whose BN scale is negative
 *   oracle_codes      Eq. (7)/(8): the output code is the number of new
 *                     thresholds the integer sum exceeds
 *   oracle_maxpool    Eq. (4) applied to the codes (max over the window,
 *                     in-bounds elements only)
 *   oracle_join_*     residual join of two dequantized branches before the
 *                     quantizer (not in the paper; ResNet-shaped stack only)
 *
 * Build: gcc -O2 -ffp-contract=off -fopenmp -fPIC -shared (no fast-math).
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_MUTATE_NO_FLIP 1 /* mutation-test knob: ignore the sign of gamma */

static int64_t out_size(int64_t in, int64_t k, int64_t stride, int64_t pad) {
  return (in + 2 * pad - k) / stride + 1;
}

/*
 * Integer part of Eq. (1). x: NHWC codes (uint8, values < 2^in_bits).
 * w: PyTorch OIHW int8 in {-1,+1}. acc: NHWC int32 [n][ho][wo][cout].
 * Input positions outside the image hold code 0 (zero padding).
 * Returns 0, or -1 if a sum leaves the bound K*(2^in_bits - 1) or int32.
 */
int oracle_conv_acc(const uint8_t* x, int n, int h, int w, int cin,
                    const int8_t* wt, int cout, int kh, int kw, int stride,
                    int pad, int in_bits, int32_t* acc) {
  const int64_t ho = out_size(h, kh, stride, pad);
  const int64_t wo = out_size(w, kw, stride, pad);
  const int64_t bound = (int64_t)kh * kw * cin * ((1 << in_bits) - 1);
  int bad = 0;
#pragma omp parallel for collapse(2) schedule(static) reduction(| : bad)
  for (int64_t b = 0; b < n; ++b) {
    for (int64_t oy = 0; oy < ho; ++oy) {
      for (int64_t ox = 0; ox < wo; ++ox) {
        for (int64_t o = 0; o < cout; ++o) {
          int64_t sum = 0;
          for (int64_t i = 0; i < kh; ++i) {
            const int64_t iy = oy * stride - pad + i;
            if (iy < 0 || iy >= h) continue;
            for (int64_t j = 0; j < kw; ++j) {
              const int64_t ix = ox * stride - pad + j;
              if (ix < 0 || ix >= w) continue;
              const uint8_t* xp = x + ((b * h + iy) * w + ix) * cin;
              for (int64_t c = 0; c < cin; ++c) {
                const int64_t wv = wt[((o * cin + c) * kh + i) * kw + j];
                sum += wv * (int64_t)xp[c];
              }
            }
          }
          if (sum > bound || sum < -bound) bad = 1;
          acc[((b * ho + oy) * wo + ox) * cout + o] = (int32_t)sum;
        }
      }
    }
  }
  return bad ? -1 : 0;
}

/*
 * Threshold fold, Eq. (6) -> Eq. (7) -> floor (Sec. 3.2), per output channel.
 *
 * The float chain of one substructure is
 *   Y_conv = alpha*beta * a + b                       (Eq. 1, a = W_b (x) X_q)
 *   Y_bn   = gamma * (Y_conv - mean) / sd + bn_beta   (Eq. 2, sd = sqrt(var+eps))
 *   code   = #{ i : Y_bn > q_i }                      (Eq. 3, ties go low)
 * Y_bn > q_i is rearranged into a comparison of the integer a with
 *   t_i = ((q_i - bn_beta) * sd / gamma + mean - b) / (alpha*beta).
 * For gamma > 0: a > t_i, and for an integer a that is a > floor(t_i).
 * For gamma < 0 the division flips the inequality: a < t_i, i.e.
 * -a > floor(-t_i). So with s = sign(gamma): s*a > floor(s*t_i).
 * gamma == 0 makes the code the constant #{i : bn_beta > q_i}.
 * Thresholds are clamped to [-B-1, B], B = K*(2^in_bits - 1) bounding |a|,
 * which changes no comparison and keeps them in int32.
 *
 * Operation order (fp64, no contraction) is fixed:
 *   sd = sqrt(var + eps); ab = alpha * beta_in;
 *   u = q_i - bn_beta; u = u * sd; u = u / gamma; u = u + mean; u = u - bias;
 *   t_i = u / ab;  T_i = clamp(floor(s * t_i), -B-1, B).
 *
 * Outputs: s_out[c] in {+1,-1}; t_out[c*nq + i] = T_{i+1}, nq = 2^out_bits - 1.
 * Nullable inputs default to bias 0, mean 0, var 1, gamma 1, bn_beta 0.
 * Returns 0, or -1 on invalid input (alpha<=0, beta<=0, var+eps<=0, NaN,
 * non-increasing q).
 */
int oracle_fold(int c_out, int in_bits, int64_t k, int out_bits,
                const double* alpha, double beta_in, const double* bias,
                const double* mean, const double* var, const double* gamma,
                const double* bn_beta, double eps, const double* q,
                int flags, int32_t* s_out, int32_t* t_out) {
  const int nq = (1 << out_bits) - 1;
  const double bound = (double)k * (double)((1 << in_bits) - 1);
  if (!(beta_in > 0.0)) return -1;
  for (int i = 1; i < nq; ++i)
    if (!(q[i] > q[i - 1])) return -1;
  for (int c = 0; c < c_out; ++c) {
    const double al = alpha[c];
    const double bi = bias ? bias[c] : 0.0;
    const double mu = mean ? mean[c] : 0.0;
    const double va = var ? var[c] : 1.0;
    const double ga = gamma ? gamma[c] : 1.0;
    const double be = bn_beta ? bn_beta[c] : 0.0;
    if (!(al > 0.0) || !(va + eps > 0.0) || isnan(bi) || isnan(mu) ||
        isnan(ga) || isnan(be))
      return -1;
    const double sd = sqrt(va + eps);
    const double ab = al * beta_in;
    if (ga == 0.0) {
      int cstar = 0;
      for (int i = 0; i < nq; ++i)
        if (be > q[i]) ++cstar;
      s_out[c] = 1;
      for (int i = 0; i < nq; ++i)
        t_out[(int64_t)c * nq + i] =
            (i < cstar) ? (int32_t)(-bound - 1.0) : (int32_t)bound;
      continue;
    }
    int s = ga > 0.0 ? 1 : -1;
    if (flags & ORACLE_MUTATE_NO_FLIP) s = 1;
    s_out[c] = s;
    for (int i = 0; i < nq; ++i) {
      double u = q[i] - be;
      u = u * sd;
      u = u / ga;
      u = u + mu;
      u = u - bi;
      const double t = u / ab;
      double f = floor((double)s * t);
      if (f < -bound - 1.0) f = -bound - 1.0;
      if (f > bound) f = bound;
      t_out[(int64_t)c * nq + i] = (int32_t)f;
    }
  }
  return 0;
}

/* Eq. (7)/(8): code = #{ i : s*a > T_i } for every element of an NHWC tensor. */
void oracle_codes(const int32_t* acc, int64_t npix, int c_out,
                  const int32_t* s, const int32_t* t, int nq, uint8_t* codes) {
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < npix; ++p) {
    for (int c = 0; c < c_out; ++c) {
      const int64_t sa = (int64_t)s[c] * acc[p * c_out + c];
      int code = 0;
      for (int i = 0; i < nq; ++i)
        if (sa > t[(int64_t)c * nq + i]) ++code;
      codes[p * c_out + c] = (uint8_t)code;
    }
  }
}

/*
 * Eq. (4) on codes: y = max over the k x k window with the given stride.
 * mode 0 (valid): ho = (h - k) / stride + 1, every window fully inside.
 * mode 1 (same):  ho = ceil(h / stride), window rows p*stride .. p*stride+k-1
 *                 clipped at the bottom/right edge (max over in-bounds only).
 */
int oracle_maxpool(const uint8_t* x, int n, int h, int w, int c, int k,
                   int stride, int mode, uint8_t* y) {
  int64_t ho, wo;
  if (mode == 0) {
    ho = (h - k) / stride + 1;
    wo = (w - k) / stride + 1;
  } else if (mode == 1) {
    ho = (h + stride - 1) / stride;
    wo = (w + stride - 1) / stride;
  } else {
    return -1;
  }
#pragma omp parallel for collapse(2) schedule(static)
  for (int64_t b = 0; b < n; ++b)
    for (int64_t py = 0; py < ho; ++py)
      for (int64_t px = 0; px < wo; ++px)
        for (int64_t ch = 0; ch < c; ++ch) {
          int m = 0;
          for (int64_t i = 0; i < k; ++i) {
            const int64_t iy = py * stride + i;
            if (iy >= h) continue;
            for (int64_t j = 0; j < k; ++j) {
              const int64_t ix = px * stride + j;
              if (ix >= w) continue;
              const int v = x[((b * h + iy) * w + ix) * c + ch];
              if (v > m) m = v;
            }
          }
          y[((b * ho + py) * wo + px) * c + ch] = (uint8_t)m;
        }
  return 0;
}

/*
 * Residual join coefficients. The join adds the main branch after its BN to
 * the dequantized shortcut and quantizes the sum:
 *   z = gamma2*(alpha2*beta2*a + b2 - mean2)/sd2 + bn_beta2 + sc,
 *   sc = beta_x * x_q                                  (identity shortcut)
 *   sc = gamma_d*(alpha_d*beta_x*d + b_d - mean_d)/sd_d + bn_beta_d  (1x1 conv)
 * which is z = p*a + q*s + cc with, in this fixed fp64 order,
 *   p  = gamma2 * (alpha2*beta2) / sd2
 *   c2 = (gamma2 * (b2 - mean2)) / sd2 + bn_beta2
 *   identity: q = beta_x,                          cd = 0
 *   conv:     q = gamma_d * (alpha_d*beta_x) / sd_d,
 *             cd = (gamma_d * (b_d - mean_d)) / sd_d + bn_beta_d
 *   cc = c2 + cd.
 * out[c*3 + {0,1,2}] = {p, q, cc}. kind: 1 identity, 2 conv.
 */
int oracle_join_coeffs(int c_out, int kind, const double* alpha2,
                       double beta2, const double* bias2, const double* mean2,
                       const double* var2, const double* gamma2,
                       const double* bnb2, double eps2, double beta_x,
                       const double* alphad, const double* biasd,
                       const double* meand, const double* vard,
                       const double* gammad, const double* bnbd, double epsd,
                       double* out) {
  for (int c = 0; c < c_out; ++c) {
    const double sd2 = sqrt(var2[c] + eps2);
    double p = alpha2[c] * beta2;
    p = gamma2[c] * p;
    p = p / sd2;
    double c2 = (bias2 ? bias2[c] : 0.0) - mean2[c];
    c2 = gamma2[c] * c2;
    c2 = c2 / sd2;
    c2 = c2 + bnb2[c];
    double q, cd;
    if (kind == 1) {
      q = beta_x;
      cd = 0.0;
    } else if (kind == 2) {
      const double sdd = sqrt(vard[c] + epsd);
      q = alphad[c] * beta_x;
      q = gammad[c] * q;
      q = q / sdd;
      cd = (biasd ? biasd[c] : 0.0) - meand[c];
      cd = gammad[c] * cd;
      cd = cd / sdd;
      cd = cd + bnbd[c];
    } else {
      return -1;
    }
    out[3 * c + 0] = p;
    out[3 * c + 1] = q;
    out[3 * c + 2] = c2 + cd;
  }
  return 0;
}

/* Join codes: z = fma(p, a, fma(q, s, cc)); code = #{ i : z > q_i }. */
void oracle_join_codes(const int32_t* a, const int32_t* sc, int64_t npix,
                       int c_out, const double* coef, const double* qthr,
                       int nq, uint8_t* codes) {
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < npix; ++p) {
    for (int c = 0; c < c_out; ++c) {
      const int64_t e = p * c_out + c;
      const double z = fma(coef[3 * c], (double)a[e],
                           fma(coef[3 * c + 1], (double)sc[e], coef[3 * c + 2]));
      int code = 0;
      for (int i = 0; i < nq; ++i)
        if (z > qthr[i]) ++code;
      codes[e] = (uint8_t)code;
    }
  }
}

int oracle_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
