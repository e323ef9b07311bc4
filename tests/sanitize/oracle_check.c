/* The C oracle under AddressSanitizer and UndefinedBehaviorSanitizer: every
 * entry point on small seeded inputs, including padding, strides, SAME pools
 * clipped at the edges and the conv join. Exit status 0 when all calls
 * return their expected status. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int oracle_conv_acc(const uint8_t* x, int n, int h, int w, int cin, const int8_t* wt,
                    int cout, int kh, int kw, int stride, int pad, int in_bits, int32_t* acc);
int oracle_fold(int c_out, int in_bits, int64_t k, int out_bits, const double* alpha,
                double beta_in, const double* bias, const double* mean, const double* var,
                const double* gamma, const double* bn_beta, double eps, const double* q,
                int flags, int32_t* s_out, int32_t* t_out);
void oracle_codes(const int32_t* acc, int64_t npix, int c_out, const int32_t* s,
                  const int32_t* t, int nq, uint8_t* codes);
int oracle_maxpool(const uint8_t* x, int n, int h, int w, int c, int k, int stride, int mode,
                   uint8_t* y);
int oracle_join_coeffs(int c_out, int kind, const double* alpha2, double beta2,
                       const double* bias2, const double* mean2, const double* var2,
                       const double* gamma2, const double* bnb2, double eps2, double beta_x,
                       const double* alphad, const double* biasd, const double* meand,
                       const double* vard, const double* gammad, const double* bnbd,
                       double epsd, double* out);
void oracle_join_codes(const int32_t* a, const int32_t* sc, int64_t npix, int c_out,
                       const double* coef, const double* qthr, int nq, uint8_t* codes);

static unsigned rng_state = 12345u;
static unsigned rnd(void) {
  rng_state = rng_state * 1664525u + 1013904223u;
  return rng_state >> 8;
}
static double urand(void) { return (double)(rnd() & 0xFFFF) / 65536.0; }

static int fails = 0;
#define EXPECT(c)                                                     \
  do {                                                                \
    if (!(c)) {                                                       \
      fprintf(stderr, "%s:%d: %s\n", __FILE__, __LINE__, #c);         \
      ++fails;                                                        \
    }                                                                 \
  } while (0)

static int out_size(int h, int k, int s, int p) { return (h + 2 * p - k) / s + 1; }

int main(void) {
  /* conv shapes: (n, h, w, cin, cout, k, stride, pad, in_bits) */
  const int shapes[][9] = {{2, 7, 5, 5, 6, 3, 1, 1, 2}, {1, 9, 9, 3, 4, 3, 2, 1, 8},
                           {3, 6, 6, 8, 3, 1, 2, 0, 2}, {1, 5, 7, 4, 5, 5, 1, 2, 4}};
  for (size_t si = 0; si < sizeof(shapes) / sizeof(shapes[0]); ++si) {
    const int* S = shapes[si];
    const int n = S[0], h = S[1], w = S[2], cin = S[3], cout = S[4], k = S[5], st = S[6],
              pad = S[7], ib = S[8];
    const int ho = out_size(h, k, st, pad), wo = out_size(w, k, st, pad);
    uint8_t* x = malloc((size_t)n * h * w * cin);
    int8_t* wt = malloc((size_t)cout * cin * k * k);
    int32_t* acc = malloc(sizeof(int32_t) * (size_t)n * ho * wo * cout);
    for (int i = 0; i < n * h * w * cin; ++i) x[i] = (uint8_t)(rnd() % (1u << ib));
    for (int i = 0; i < cout * cin * k * k; ++i) wt[i] = (rnd() & 1) ? 1 : -1;
    EXPECT(oracle_conv_acc(x, n, h, w, cin, wt, cout, k, k, st, pad, ib, acc) == 0);
    /* thresholds for 1..3-bit outputs, then codes */
    for (int ob = 1; ob <= 3; ++ob) {
      const int nq = (1 << ob) - 1;
      double *alpha = malloc(sizeof(double) * cout), *bias = malloc(sizeof(double) * cout),
             *mean = malloc(sizeof(double) * cout), *var = malloc(sizeof(double) * cout),
             *gamma = malloc(sizeof(double) * cout), *beta = malloc(sizeof(double) * cout),
             *q = malloc(sizeof(double) * nq);
      for (int c = 0; c < cout; ++c) {
        alpha[c] = 0.01 + 0.09 * urand();
        bias[c] = urand() - 0.5;
        mean[c] = 4.0 * (urand() - 0.5);
        var[c] = 0.5 + 1.5 * urand();
        gamma[c] = (0.5 + urand()) * (c % 3 == 1 ? -1.0 : 1.0);
        beta[c] = urand() - 0.5;
      }
      gamma[0] = 0.0;
      for (int i = 0; i < nq; ++i) q[i] = 0.25 + 0.5 * i;
      int32_t* s = malloc(sizeof(int32_t) * cout);
      int32_t* t = malloc(sizeof(int32_t) * cout * nq);
      uint8_t* codes = malloc((size_t)n * ho * wo * cout);
      EXPECT(oracle_fold(cout, ib, (int64_t)k * k * cin, ob, alpha, 0.5, bias, mean, var, gamma,
                         beta, 1e-5, q, 0, s, t) == 0);
      oracle_codes(acc, (int64_t)n * ho * wo, cout, s, t, nq, codes);
      for (int i = 0; i < n * ho * wo * cout; ++i) EXPECT(codes[i] <= nq);
      /* pools on the codes: valid and same */
      for (int mode = 0; mode <= 1; ++mode) {
        const int pk = 2, ps = 2;
        const int ph = mode ? (ho + ps - 1) / ps : (ho - pk) / ps + 1;
        const int pw = mode ? (wo + ps - 1) / ps : (wo - pk) / ps + 1;
        if (ph <= 0 || pw <= 0) continue;
        uint8_t* y = malloc((size_t)n * ph * pw * cout);
        EXPECT(oracle_maxpool(codes, n, ho, wo, cout, pk, ps, mode, y) == 0);
        free(y);
      }
      /* join on these sums with a second tensor as the shortcut */
      double* coef = malloc(sizeof(double) * 3 * cout);
      EXPECT(oracle_join_coeffs(cout, 2, alpha, 0.5, bias, mean, var, gamma, beta, 1e-5, 0.5,
                                alpha, bias, mean, var, gamma, beta, 1e-5, coef) == 0);
      EXPECT(oracle_join_coeffs(cout, 7, alpha, 0.5, bias, mean, var, gamma, beta, 1e-5, 0.5,
                                alpha, bias, mean, var, gamma, beta, 1e-5, coef) != 0);
      oracle_join_codes(acc, acc, (int64_t)n * ho * wo, cout, coef, q, nq, codes);
      free(coef);
      free(codes);
      free(s);
      free(t);
      free(alpha); free(bias); free(mean); free(var); free(gamma); free(beta); free(q);
    }
    free(x);
    free(wt);
    free(acc);
  }
  if (fails) {
    fprintf(stderr, "%d check(s) failed\n", fails);
    return 1;
  }
  printf("oracle checks passed\n");
  return 0;
}
