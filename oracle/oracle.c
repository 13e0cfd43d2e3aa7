/*
 * Oracle layer definitions in plain C, float64 throughout.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the reference against which the HIP
 * feature-extraction path is checked; only the test-suite, the smoke check and
 * the benchmark's CPU-baseline leg may load it.  It shares no code, header or
 * table with the HIP path.
 *
 * Each routine is the textbook definition of one layer of the frozen
 * feature-extraction networks the paper splits (Measurement study; Evaluation,
 * Table 2: AlexNet, ResNet18/50, Vgg, the TorchVision Vision Transformer),
 * written as loops.  OpenMP only distributes independent output elements over
 * threads; every sum runs in a fixed sequential order.
 *
 * Layout: activations are NCHW ([N, C, H, W]) or row-major token matrices
 * ([T, D]); conv weights are OIHW; linear weights are [out, in].
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

/* y[n,o,i,j] = b[o] + sum_c sum_u sum_v w[o,c,u,v] * x[n,c,i*s-p+u, j*s-p+v],
 * with zero padding; Ho = floor((H + 2p - kh)/s) + 1, Wo likewise. */
void oracle_conv2d(const double *x, int N, int C, int H, int W,
                   const double *w, int O, int kh, int kw, int stride, int pad,
                   const double *bias, double *y) {
  const int Ho = (H + 2 * pad - kh) / stride + 1;
  const int Wo = (W + 2 * pad - kw) / stride + 1;
#pragma omp parallel for collapse(2) schedule(dynamic)
  for (int n = 0; n < N; ++n) {
    for (int o = 0; o < O; ++o) {
      double *yo = y + ((int64_t)n * O + o) * Ho * Wo;
      for (int i = 0; i < Ho * Wo; ++i) yo[i] = bias ? bias[o] : 0.0;
      for (int c = 0; c < C; ++c) {
        const double *xc = x + ((int64_t)n * C + c) * H * W;
        for (int u = 0; u < kh; ++u) {
          for (int v = 0; v < kw; ++v) {
            const double wv = w[(((int64_t)o * C + c) * kh + u) * kw + v];
            for (int i = 0; i < Ho; ++i) {
              const int hi = i * stride - pad + u;
              if (hi < 0 || hi >= H) continue;
              for (int j = 0; j < Wo; ++j) {
                const int wi = j * stride - pad + v;
                if (wi < 0 || wi >= W) continue;
                yo[i * Wo + j] += wv * xc[hi * W + wi];
              }
            }
          }
        }
      }
    }
  }
}

/* Inference batch normalisation, in place over [N, C, HW]:
 * x <- gamma * (x - mean) / sqrt(var + eps) + beta. */
void oracle_batchnorm(double *x, int N, int C, int64_t HW, const double *gamma,
                      const double *beta, const double *mean, const double *var,
                      double eps) {
#pragma omp parallel for collapse(2)
  for (int n = 0; n < N; ++n) {
    for (int c = 0; c < C; ++c) {
      double *xc = x + ((int64_t)n * C + c) * HW;
      const double inv = 1.0 / sqrt(var[c] + eps);
      for (int64_t i = 0; i < HW; ++i) xc[i] = gamma[c] * (xc[i] - mean[c]) * inv + beta[c];
    }
  }
}

void oracle_relu(double *x, int64_t n) {
#pragma omp parallel for
  for (int64_t i = 0; i < n; ++i) x[i] = x[i] > 0.0 ? x[i] : 0.0;
}

/* y += x, elementwise. */
void oracle_add(double *y, const double *x, int64_t n) {
#pragma omp parallel for
  for (int64_t i = 0; i < n; ++i) y[i] += x[i];
}

/* Max over k x k windows (stride s, padding p counted as -infinity, floor mode). */
void oracle_maxpool2d(const double *x, int N, int C, int H, int W, int k,
                      int stride, int pad, double *y) {
  const int Ho = (H + 2 * pad - k) / stride + 1;
  const int Wo = (W + 2 * pad - k) / stride + 1;
#pragma omp parallel for collapse(2)
  for (int n = 0; n < N; ++n) {
    for (int c = 0; c < C; ++c) {
      const double *xc = x + ((int64_t)n * C + c) * H * W;
      double *yc = y + ((int64_t)n * C + c) * Ho * Wo;
      for (int i = 0; i < Ho; ++i) {
        for (int j = 0; j < Wo; ++j) {
          double m = -INFINITY;
          for (int u = 0; u < k; ++u) {
            const int hi = i * stride - pad + u;
            if (hi < 0 || hi >= H) continue;
            for (int v = 0; v < k; ++v) {
              const int wi = j * stride - pad + v;
              if (wi < 0 || wi >= W) continue;
              if (xc[hi * W + wi] > m) m = xc[hi * W + wi];
            }
          }
          yc[i * Wo + j] = m;
        }
      }
    }
  }
}

/* Mean over k x k windows (stride s, no padding), as used by dense-net transitions. */
void oracle_avgpool2d(const double *x, int N, int C, int H, int W, int k,
                      int stride, double *y) {
  const int Ho = (H - k) / stride + 1;
  const int Wo = (W - k) / stride + 1;
#pragma omp parallel for collapse(2)
  for (int n = 0; n < N; ++n) {
    for (int c = 0; c < C; ++c) {
      const double *xc = x + ((int64_t)n * C + c) * H * W;
      double *yc = y + ((int64_t)n * C + c) * Ho * Wo;
      for (int i = 0; i < Ho; ++i)
        for (int j = 0; j < Wo; ++j) {
          double s = 0.0;
          for (int u = 0; u < k; ++u)
            for (int v = 0; v < k; ++v) s += xc[(i * stride + u) * W + j * stride + v];
          yc[i * Wo + j] = s / (double)(k * k);
        }
    }
  }
}

/* Global average: y[n,c] = mean over the HW positions of x[n,c,:]. */
void oracle_avgpool_global(const double *x, int N, int C, int64_t HW, double *y) {
#pragma omp parallel for collapse(2)
  for (int n = 0; n < N; ++n) {
    for (int c = 0; c < C; ++c) {
      const double *xc = x + ((int64_t)n * C + c) * HW;
      double s = 0.0;
      for (int64_t i = 0; i < HW; ++i) s += xc[i];
      y[(int64_t)n * C + c] = s / (double)HW;
    }
  }
}

/* y[m, o] = b[o] + sum_k x[m, k] * w[o, k]   (x: [M, K], w: [O, K], y: [M, O]). */
void oracle_linear(const double *x, int64_t M, int K, const double *w, int O,
                   const double *bias, double *y) {
#pragma omp parallel for collapse(2)
  for (int64_t m = 0; m < M; ++m) {
    for (int o = 0; o < O; ++o) {
      double s = bias ? bias[o] : 0.0;
      const double *xr = x + m * K;
      const double *wr = w + (int64_t)o * K;
      for (int k = 0; k < K; ++k) s += xr[k] * wr[k];
      y[m * O + o] = s;
    }
  }
}

/* Per-row layer normalisation over D features with affine (gamma, beta):
 * y = gamma * (x - mean) / sqrt(var + eps) + beta, var the biased (1/D) variance. */
void oracle_layernorm(const double *x, int64_t M, int D, const double *gamma,
                      const double *beta, double eps, double *y) {
#pragma omp parallel for
  for (int64_t m = 0; m < M; ++m) {
    const double *xr = x + m * D;
    double mean = 0.0;
    for (int d = 0; d < D; ++d) mean += xr[d];
    mean /= (double)D;
    double var = 0.0;
    for (int d = 0; d < D; ++d) var += (xr[d] - mean) * (xr[d] - mean);
    var /= (double)D;
    const double inv = 1.0 / sqrt(var + eps);
    for (int d = 0; d < D; ++d) y[m * D + d] = gamma[d] * (xr[d] - mean) * inv + beta[d];
  }
}

/* GELU with the exact error function: x * (1 + erf(x / sqrt 2)) / 2, in place. */
void oracle_gelu(double *x, int64_t n) {
#pragma omp parallel for
  for (int64_t i = 0; i < n; ++i) x[i] = 0.5 * x[i] * (1.0 + erf(x[i] / sqrt(2.0)));
}

/* Multi-head self-attention core for N independent sequences.
 * qkv: [N, T, 3D] with query columns [0, D), key columns [D, 2D), value
 * columns [2D, 3D); head h uses the dh = D/heads wide slice h of each.
 * out[n, t, h*dh + e] = sum_s P[t, s] * V[s, e], where
 * P = softmax_s(Q K^T / sqrt(dh)) row by row (max-subtracted). */
void oracle_attention(const double *qkv, int N, int T, int D, int heads, double *out) {
  const int dh = D / heads;
  const double scale = 1.0 / sqrt((double)dh);
#pragma omp parallel for collapse(3)
  for (int n = 0; n < N; ++n) {
    for (int h = 0; h < heads; ++h) {
      for (int t = 0; t < T; ++t) {
        double p[4096];
        const double *base = qkv + (int64_t)n * T * 3 * D;
        const double *q = base + (int64_t)t * 3 * D + h * dh;
        double mx = -INFINITY;
        for (int s = 0; s < T; ++s) {
          const double *k = base + (int64_t)s * 3 * D + D + h * dh;
          double dot = 0.0;
          for (int e = 0; e < dh; ++e) dot += q[e] * k[e];
          p[s] = dot * scale;
          if (p[s] > mx) mx = p[s];
        }
        double sum = 0.0;
        for (int s = 0; s < T; ++s) {
          p[s] = exp(p[s] - mx);
          sum += p[s];
        }
        double *o = out + ((int64_t)n * T + t) * D + h * dh;
        for (int e = 0; e < dh; ++e) {
          double acc = 0.0;
          for (int s = 0; s < T; ++s) acc += p[s] * base[(int64_t)s * 3 * D + 2 * D + h * dh + e];
          o[e] = acc / sum;
        }
      }
    }
  }
}

int oracle_max_tokens(void) { return 4096; }
