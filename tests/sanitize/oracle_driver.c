/* Calls every function of the oracle's C library on small geometries
 * (padding, strides, ragged windows, one-token rows) with heap buffers of
 * exactly the size each function reads or writes, under AddressSanitizer and
 * UBSan.  Prints "OK <calls>" on success. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

void oracle_conv2d(const double *x, int N, int C, int H, int W, const double *w, int O, int kh, int kw,
                   int stride, int pad, const double *bias, double *y);
void oracle_batchnorm(double *x, int N, int C, int64_t HW, const double *gamma, const double *beta,
                      const double *mean, const double *var, double eps);
void oracle_relu(double *x, int64_t n);
void oracle_add(double *y, const double *x, int64_t n);
void oracle_maxpool2d(const double *x, int N, int C, int H, int W, int k, int stride, int pad, double *y);
void oracle_avgpool2d(const double *x, int N, int C, int H, int W, int k, int stride, double *y);
void oracle_avgpool_global(const double *x, int N, int C, int64_t HW, double *y);
void oracle_linear(const double *x, int64_t M, int K, const double *w, int O, const double *b, double *y);
void oracle_layernorm(const double *x, int64_t M, int D, const double *gamma, const double *beta, double eps,
                      double *y);
void oracle_gelu(double *x, int64_t n);
void oracle_attention(const double *qkv, int N, int T, int D, int heads, double *out);

static double *buf(int64_t n) {
  double *p = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
  for (int64_t i = 0; i < n; ++i) p[i] = sin(0.37 * (double)i) * 2.0;
  return p;
}

int main(void) {
  long calls = 0;
  const int geo[][6] = {{1, 3, 9, 7, 3, 1}, {2, 4, 8, 8, 7, 2}, {1, 2, 5, 6, 1, 1}, {2, 3, 11, 9, 5, 3},
                        {1, 1, 4, 4, 4, 4}};
  for (unsigned g = 0; g < sizeof geo / sizeof geo[0]; ++g) {
    const int N = geo[g][0], C = geo[g][1], H = geo[g][2], W = geo[g][3], k = geo[g][4], s = geo[g][5];
    for (int pad = 0; pad < k && pad <= 3; ++pad) {
      const int Ho = (H + 2 * pad - k) / s + 1, Wo = (W + 2 * pad - k) / s + 1;
      if (Ho < 1 || Wo < 1) continue;
      const int O = 3;
      double *x = buf((int64_t)N * C * H * W), *w = buf((int64_t)O * C * k * k), *b = buf(O);
      double *y = buf((int64_t)N * O * Ho * Wo);
      oracle_conv2d(x, N, C, H, W, w, O, k, k, s, pad, b, y);
      oracle_conv2d(x, N, C, H, W, w, O, k, k, s, pad, NULL, y);
      if (2 * pad <= k) {
        double *p = buf((int64_t)N * C * Ho * Wo);
        oracle_maxpool2d(x, N, C, H, W, k, s, pad, p);
        free(p);
        calls++;
      }
      if (pad == 0) {
        double *p = buf((int64_t)N * C * Ho * Wo);
        oracle_avgpool2d(x, N, C, H, W, k, s, p);
        free(p);
        calls++;
      }
      free(x); free(w); free(b); free(y);
      calls += 2;
    }
    double *x = buf((int64_t)N * C * H * W), *ga = buf(C), *be = buf(C), *mu = buf(C), *va = buf(C);
    for (int c = 0; c < C; ++c) va[c] = 1.0 + va[c] * va[c];
    oracle_batchnorm(x, N, C, (int64_t)H * W, ga, be, mu, va, 1e-5);
    oracle_relu(x, (int64_t)N * C * H * W);
    double *x2 = buf((int64_t)N * C * H * W);
    oracle_add(x, x2, (int64_t)N * C * H * W);
    double *gp = buf((int64_t)N * C);
    oracle_avgpool_global(x, N, C, (int64_t)H * W, gp);
    free(x); free(x2); free(ga); free(be); free(mu); free(va); free(gp);
    calls += 4;
  }
  const int lin[][3] = {{1, 8, 3}, {5, 16, 24}, {7, 3, 1}};
  for (unsigned i = 0; i < 3; ++i) {
    const int M = lin[i][0], K = lin[i][1], O = lin[i][2];
    double *x = buf((int64_t)M * K), *w = buf((int64_t)O * K), *b = buf(O), *y = buf((int64_t)M * O);
    oracle_linear(x, M, K, w, O, b, y);
    oracle_linear(x, M, K, w, O, NULL, y);
    double *g = buf(K), *be = buf(K), *z = buf((int64_t)M * K);
    oracle_layernorm(x, M, K, g, be, 1e-6, z);
    oracle_gelu(z, (int64_t)M * K);
    free(x); free(w); free(b); free(y); free(g); free(be); free(z);
    calls += 4;
  }
  const int att[][4] = {{1, 1, 8, 2}, {2, 5, 16, 4}, {1, 33, 128, 2}};
  for (unsigned i = 0; i < 3; ++i) {
    const int N = att[i][0], T = att[i][1], D = att[i][2], h = att[i][3];
    double *qkv = buf((int64_t)N * T * 3 * D), *o = buf((int64_t)N * T * D);
    oracle_attention(qkv, N, T, D, h, o);
    free(qkv); free(o);
    calls++;
  }
  printf("OK %ld calls\n", calls);
  return 0;
}
