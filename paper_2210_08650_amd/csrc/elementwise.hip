// Memory-bound kernels for gfx950: pooling, layout changes, token assembly,
// layernorm, copies and weight packing.  They move data in 16-byte vectors
// along the contiguous channel (NHWC) or feature dimension so that each wave
// reads and writes whole cache lines; their roofline is HBM bandwidth.
#include <algorithm>

#include "internal.h"

namespace hapi {
namespace {

__device__ __forceinline__ float bf2f(uint16_t u) { return __uint_as_float((uint32_t)u << 16); }


inline int blocks_for(int64_t n, int per_block) { return (int)((n + per_block - 1) / per_block); }

// Activation element access for both types.
template <typename T> struct Elt;
template <> struct Elt<float> {
  __device__ static float ld(const float *p, int64_t i) { return p[i]; }
  __device__ static void st(float *p, int64_t i, float v) { p[i] = v; }
};
template <> struct Elt<uint16_t> {
  __device__ static float ld(const uint16_t *p, int64_t i) { return bf2f(p[i]); }
  __device__ static void st(uint16_t *p, int64_t i, float v) { p[i] = f2bf(v); }
};

// --------------------------------------------------------------- max pool
// NHWC, 8 channels per thread (16 B for bf16, 2 x 16 B for fp32).  The max of
// bf16 values is exact, so no rounding happens.
template <typename T>
__global__ void maxpool_kernel(const T *__restrict__ x, T *__restrict__ y, int n, int H, int W,
                               int C, int k, int stride, int pad, int Ho, int Wo) {
  const int cg = C / 8;
  const int64_t total = (int64_t)n * Ho * Wo * cg;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int g = (int)(i % cg);
  int64_t p = i / cg;
  const int wo = (int)(p % Wo); p /= Wo;
  const int ho = (int)(p % Ho);
  const int img = (int)(p / Ho);
  float m[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) m[j] = -INFINITY;
  for (int u = 0; u < k; ++u) {
    const int hi = ho * stride - pad + u;
    if (hi < 0 || hi >= H) continue;
    for (int v = 0; v < k; ++v) {
      const int wi = wo * stride - pad + v;
      if (wi < 0 || wi >= W) continue;
      const int64_t base = (((int64_t)img * H + hi) * W + wi) * C + g * 8;
      if constexpr (sizeof(T) == 2) {
        const uint4 q = *reinterpret_cast<const uint4 *>(x + base);
        const uint32_t w4[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          m[2 * j] = fmaxf(m[2 * j], bf2f((uint16_t)(w4[j] & 0xffff)));
          m[2 * j + 1] = fmaxf(m[2 * j + 1], bf2f((uint16_t)(w4[j] >> 16)));
        }
      } else {
        const float4 a = *reinterpret_cast<const float4 *>(x + base);
        const float4 b = *reinterpret_cast<const float4 *>(x + base + 4);
        m[0] = fmaxf(m[0], a.x); m[1] = fmaxf(m[1], a.y); m[2] = fmaxf(m[2], a.z); m[3] = fmaxf(m[3], a.w);
        m[4] = fmaxf(m[4], b.x); m[5] = fmaxf(m[5], b.y); m[6] = fmaxf(m[6], b.z); m[7] = fmaxf(m[7], b.w);
      }
    }
  }
  const int64_t ob = (((int64_t)img * Ho + ho) * Wo + wo) * C + g * 8;
  if constexpr (sizeof(T) == 2) {
    uint4 q;
    q.x = f2bf2(m[0], m[1]);
    q.y = f2bf2(m[2], m[3]);
    q.z = f2bf2(m[4], m[5]);
    q.w = f2bf2(m[6], m[7]);
    *reinterpret_cast<uint4 *>(y + ob) = q;
  } else {
    *reinterpret_cast<float4 *>(y + ob) = make_float4(m[0], m[1], m[2], m[3]);
    *reinterpret_cast<float4 *>(y + ob + 4) = make_float4(m[4], m[5], m[6], m[7]);
  }
}

// --------------------------------------------------------------- avg pool
// k == 0: global mean over H x W; else k x k windows, no padding.  One
// thread per (output pixel, channel); consecutive threads take consecutive
// channels so loads coalesce along C.
template <typename T>
__global__ void avgpool_kernel(const T *__restrict__ x, T *__restrict__ y, int n, int H, int W,
                               int C, int k, int stride, int Ho, int Wo) {
  const int64_t total = (int64_t)n * Ho * Wo * C;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int c = (int)(i % C);
  int64_t p = i / C;
  const int wo = (int)(p % Wo); p /= Wo;
  const int ho = (int)(p % Ho);
  const int img = (int)(p / Ho);
  const int kh = k ? k : H, kw = k ? k : W;
  const int h0 = k ? ho * stride : 0, w0 = k ? wo * stride : 0;
  float s = 0.0f;
  for (int u = 0; u < kh; ++u)
    for (int v = 0; v < kw; ++v)
      s += Elt<T>::ld(x, (((int64_t)img * H + h0 + u) * W + w0 + v) * C + c);
  Elt<T>::st(y, i, s / (float)(kh * kw));
}

// bf16 NHWC with C % 8 == 0: 8 channels per thread, 16-byte loads and
// stores; the same summation order and rounding as avgpool_kernel.
__global__ void avgpool8_kernel(const uint16_t *__restrict__ x, uint16_t *__restrict__ y, int n, int H,
                                int W, int C, int k, int stride, int Ho, int Wo) {
  const int cg = C / 8;
  const int64_t total = (int64_t)n * Ho * Wo * cg;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int g = (int)(i % cg);
  int64_t p = i / cg;
  const int wo = (int)(p % Wo); p /= Wo;
  const int ho = (int)(p % Ho);
  const int img = (int)(p / Ho);
  const int kh = k ? k : H, kw = k ? k : W;
  const int h0 = k ? ho * stride : 0, w0 = k ? wo * stride : 0;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int u = 0; u < kh; ++u)
    for (int v = 0; v < kw; ++v) {
      const uint4 q = *reinterpret_cast<const uint4 *>(x + (((int64_t)img * H + h0 + u) * W + w0 + v) * C + g * 8);
      const uint32_t w4[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[2 * e] += bf2f((uint16_t)(w4[e] & 0xffff));
        acc[2 * e + 1] += bf2f((uint16_t)(w4[e] >> 16));
      }
    }
  const float d = (float)(kh * kw);
  uint32_t o[4];
#pragma unroll
  for (int e = 0; e < 4; ++e) o[e] = f2bf2(acc[2 * e] / d, acc[2 * e + 1] / d);
  *reinterpret_cast<uint4 *>(y + i * 8) = make_uint4(o[0], o[1], o[2], o[3]);
}

// ------------------------------------------------------------- transposes
// [n, R, S] -> [n, S, R] through a 64 x 64 LDS tile (rows padded by one
// element against bank conflicts); both global sides are coalesced.
template <typename T>
__global__ void transpose_kernel(const T *__restrict__ x, T *__restrict__ y, int R, int S) {
  __shared__ T tile[64][65];
  const int img = blockIdx.z;
  const int r0 = blockIdx.y * 64, s0 = blockIdx.x * 64;
  const T *xi = x + (int64_t)img * R * S;
  T *yi = y + (int64_t)img * R * S;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;  // 256 threads: 4 rows per pass
  for (int r = ty; r < 64; r += 4) {
    const int gr = r0 + r, gs = s0 + tx;
    if (gr < R && gs < S) tile[r][tx] = xi[(int64_t)gr * S + gs];
  }
  __syncthreads();
  for (int s = ty; s < 64; s += 4) {
    const int gs = s0 + s, gr = r0 + tx;
    if (gr < R && gs < S) yi[(int64_t)gs * R + gr] = tile[tx][s];
  }
}

// ------------------------------------------------------------------ copies
__global__ void copy16_kernel(const uint4 *__restrict__ x, uint4 *__restrict__ y, int64_t n16) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) y[i] = x[i];
}

__global__ void copy1_kernel(const uint8_t *__restrict__ x, uint8_t *__restrict__ y, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] = x[i];
}

__global__ void copy_f32_kernel(const float *__restrict__ x, float *__restrict__ y, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) y[i] = x[i];
}

// Deterministic pseudo-random fill in [-scale, scale) (profiling inputs only).
template <typename T>
__global__ void fill_kernel(T *__restrict__ y, int64_t n, uint32_t seed, float scale) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  uint32_t h = (uint32_t)i * 2654435761u ^ seed;
  h ^= h >> 16; h *= 0x7feb352du; h ^= h >> 15; h *= 0x846ca68bu; h ^= h >> 16;
  const float u = (float)(h >> 8) * (1.0f / 16777216.0f);
  Elt<T>::st(y, i, (2.0f * u - 1.0f) * scale);
}

// ------------------------------------------------------------------ tokens
// patch: [n, T-1, D] (NHWC patch-embedding output), y: [n, T, D].
// y[i, 0] = cls + pos[0];  y[i, 1 + t] = patch[i, t] + pos[1 + t].
__global__ void tokens_kernel(const uint16_t *__restrict__ patch, const float *__restrict__ cls,
                              const float *__restrict__ pos, uint16_t *__restrict__ y, int n,
                              int T, int D) {
  const int dg = D / 8;
  const int64_t total = (int64_t)n * T * dg;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int g = (int)(i % dg);
  const int64_t row = i / dg;
  const int tok = (int)(row % T);
  const int img = (int)(row / T);
  float v[8];
  if (tok == 0) {
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = cls[g * 8 + j];
  } else {
    const uint4 q = *reinterpret_cast<const uint4 *>(patch + ((int64_t)img * (T - 1) + tok - 1) * D + g * 8);
    const uint32_t w4[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[2 * j] = bf2f((uint16_t)(w4[j] & 0xffff));
      v[2 * j + 1] = bf2f((uint16_t)(w4[j] >> 16));
    }
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) v[j] += pos[(int64_t)tok * D + g * 8 + j];
  uint4 o;
  o.x = f2bf2(v[0], v[1]);
  o.y = f2bf2(v[2], v[3]);
  o.z = f2bf2(v[4], v[5]);
  o.w = f2bf2(v[6], v[7]);
  *reinterpret_cast<uint4 *>(y + row * D + g * 8) = o;
}

// --------------------------------------------------------------- layernorm
// One wave per row; each lane holds up to 4 chunks of 8 features (D <= 2048,
// D % 8 == 0).  Mean and variance in fp32 from registers (two passes).
__global__ __launch_bounds__(256) void layernorm_kernel(const uint16_t *__restrict__ x,
                                                        const float *__restrict__ gamma,
                                                        const float *__restrict__ beta,
                                                        uint16_t *__restrict__ y, int64_t rows,
                                                        int D, float eps) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= rows) return;
  const int nch = D / 8;
  const uint16_t *xr = x + row * D;
  float v[4][8];
  float s = 0.0f;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int ch = lane + 64 * c;
    if (ch < nch) {
      const uint4 q = *reinterpret_cast<const uint4 *>(xr + ch * 8);
      const uint32_t w4[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        v[c][2 * j] = bf2f((uint16_t)(w4[j] & 0xffff));
        v[c][2 * j + 1] = bf2f((uint16_t)(w4[j] >> 16));
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) s += v[c][j];
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
  const float mean = s / (float)D;
  float q2 = 0.0f;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    if (lane + 64 * c < nch) {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float d = v[c][j] - mean;
        q2 += d * d;
      }
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) q2 += __shfl_xor(q2, o, 64);
  const float inv = rsqrtf(q2 / (float)D + eps);
  uint16_t *yr = y + row * D;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int ch = lane + 64 * c;
    if (ch < nch) {
      uint16_t o[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int d = ch * 8 + j;
        o[j] = f2bf((v[c][j] - mean) * inv * gamma[d] + beta[d]);
      }
      uint4 q;
      q.x = o[0] | ((uint32_t)o[1] << 16);
      q.y = o[2] | ((uint32_t)o[3] << 16);
      q.z = o[4] | ((uint32_t)o[5] << 16);
      q.w = o[6] | ((uint32_t)o[7] << 16);
      *reinterpret_cast<uint4 *>(yr + ch * 8) = q;
    }
  }
}

// ------------------------------------------------------------- weight pack
// wp[n][k'] = W[n, c, u, v] * s[n] for k' < K, 0 for K <= k' < Kp, where
// s[n] = gamma[n] / sqrt(var[n] + 1e-5) (1 without batch-norm), computed in fp32;
// bias_out[n] = (b[n] - mean[n]) * s[n] + beta[n]  (b = conv bias or 0).
template <typename T>
__global__ void pack_conv_kernel(const float *__restrict__ w, const float *__restrict__ cb,
                                 const float *__restrict__ gamma, const float *__restrict__ beta,
                                 const float *__restrict__ mean, const float *__restrict__ var,
                                 int N, int C, int kh, int kw, int kcols, int ldw, int koff,
                                 int acc_bias, int order, T *__restrict__ wp,
                                 float *__restrict__ bias_out) {
  const int64_t total = (int64_t)N * kcols;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int n = (int)(i / kcols), k = (int)(i % kcols);
  const int K = C * kh * kw;
  const float sc = gamma ? gamma[n] / sqrtf(var[n] + 1e-5f) : 1.0f;
  float val = 0.0f;
  if (order == PACK_S2D) {
    // k = (du, dv, a, b, c4) over kh2 x kw2 cells: tap (u, v) = (2 du + a, 2 dv + b)
    const int kw2 = (kw + 1) / 2;
    const int c = k & 3, b = (k >> 2) & 1, a = (k >> 3) & 1;
    const int cell = k >> 4, du = cell / kw2, dv = cell % kw2;
    const int u = 2 * du + a, v = 2 * dv + b;
    if (c < C && u < kh && v < kw) val = w[(((int64_t)n * C + c) * kh + u) * kw + v] * sc;
  } else if (order == PACK_KHKWC8) {
    const int tap = k >> 3, c = k & 7;
    if (c < C && tap < kh * kw) val = w[(((int64_t)n * C + c) * kh + tap / kw) * kw + tap % kw] * sc;
  } else if (k < K) {
    int c, u, v;
    if (order == PACK_CKHKW) {
      c = k / (kh * kw);
      const int r = k % (kh * kw);
      u = r / kw; v = r % kw;
    } else {
      const int tap = k / C;
      c = k % C;
      u = tap / kw; v = tap % kw;
    }
    val = w[(((int64_t)n * C + c) * kh + u) * kw + v] * sc;
  }
  Elt<T>::st(wp, (int64_t)n * ldw + koff + k, val);
  if (k == 0) {
    const float b = cb ? cb[n] : 0.0f;
    const float folded = gamma ? (b - mean[n]) * sc + beta[n] : b;
    bias_out[n] = acc_bias ? bias_out[n] + folded : folded;
  }
}

// Space-to-depth: one thread per output cell, writing its 16 channels (32 B).
__global__ void s2d_kernel(const uint16_t *__restrict__ x, uint16_t *__restrict__ y, int n, int C,
                           int H, int W, int pad, int HP, int WP) {
  const int64_t total = (int64_t)n * HP * WP;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= total) return;
  const int Q = (int)(i % WP);
  const int64_t r = i / WP;
  const int P = (int)(r % HP);
  const int img = (int)(r / HP);
  uint16_t v[16];
#pragma unroll
  for (int q = 0; q < 16; ++q) {
    const int c = q & 3, b = (q >> 2) & 1, a = (q >> 3) & 1;
    const int h = 2 * P + a - pad, w = 2 * Q + b - pad;
    v[q] = (c < C && (unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W)
               ? x[(((int64_t)img * C + c) * H + h) * W + w]
               : (uint16_t)0;
  }
  uint4 *dst = reinterpret_cast<uint4 *>(y + i * 16);
  dst[0] = make_uint4(v[0] | ((uint32_t)v[1] << 16), v[2] | ((uint32_t)v[3] << 16),
                      v[4] | ((uint32_t)v[5] << 16), v[6] | ((uint32_t)v[7] << 16));
  dst[1] = make_uint4(v[8] | ((uint32_t)v[9] << 16), v[10] | ((uint32_t)v[11] << 16),
                      v[12] | ((uint32_t)v[13] << 16), v[14] | ((uint32_t)v[15] << 16));
}

// NCHW (C <= 8) -> NHWC with 8 channel slots: one thread per pixel (16 bytes).
__global__ void nhwc8_kernel(const uint16_t *__restrict__ x, uint16_t *__restrict__ y, int n, int C,
                             int64_t HW) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)n * HW) return;
  const int64_t img = i / HW, p = i - img * HW;
  uint32_t v[8];
#pragma unroll
  for (int c = 0; c < 8; ++c) v[c] = c < C ? x[(img * C + c) * HW + p] : 0u;
  *reinterpret_cast<uint4 *>(y + i * 8) =
      make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16), v[6] | (v[7] << 16));
}

// Concatenation along channels: one thread per 8 channels (16 bytes).
__global__ void channel_copy_kernel(const uint16_t *__restrict__ x, uint16_t *__restrict__ y,
                                    int64_t pixels, int C, int cx, int cy, int off) {
  const int cg = C / 8;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= pixels * cg) return;
  const int64_t p = i / cg;
  const int g = (int)(i % cg);
  *reinterpret_cast<uint4 *>(y + p * cy + off + g * 8) =
      *reinterpret_cast<const uint4 *>(x + p * cx + g * 8);
}

// Inference batch-norm (per-channel scale and shift) and optional ReLU on a
// channel prefix of C of the cx channels of x, 8 channels per thread.
template <bool RELU>
__global__ void affine_kernel(const uint16_t *__restrict__ x, const float *__restrict__ scale,
                              const float *__restrict__ shift, uint16_t *__restrict__ y,
                              int64_t pixels, int C, int cx) {
  const int cg = C / 8;
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= pixels * cg) return;
  const int64_t p = i / cg;
  const int g = (int)(i % cg);
  const uint4 q = *reinterpret_cast<const uint4 *>(x + p * cx + g * 8);
  const uint32_t w4[4] = {q.x, q.y, q.z, q.w};
  uint32_t o[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int c = g * 8 + 2 * j;
    float lo = __builtin_fmaf(bf2f((uint16_t)(w4[j] & 0xffff)), scale[c], shift[c]);
    float hi = __builtin_fmaf(bf2f((uint16_t)(w4[j] >> 16)), scale[c + 1], shift[c + 1]);
    if (RELU) {
      lo = fmaxf(lo, 0.0f);
      hi = fmaxf(hi, 0.0f);
    }
    o[j] = f2bf2(lo, hi);
  }
  *reinterpret_cast<uint4 *>(y + p * C + g * 8) = make_uint4(o[0], o[1], o[2], o[3]);
}

__global__ void pack_affine_kernel(const float *__restrict__ bn, int C, float *__restrict__ scale,
                                   float *__restrict__ shift) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= C) return;
  const float sc = bn[c] / sqrtf(bn[3 * C + c] + 1e-5f);
  scale[c] = sc;
  shift[c] = bn[C + c] - bn[2 * C + c] * sc;
}

}  // namespace

hipError_t launch_channel_copy(const void *x, void *y, int64_t pixels, int C, int cx, int cy,
                               int off, hipStream_t s) {
  const int64_t total = pixels * (C / 8);
  hapi_launch(channel_copy_kernel, dim3(blocks_for(total, 256)), dim3(256), 0, s,
                     (const uint16_t *)x, (uint16_t *)y, pixels, C, cx, cy, off);
  return hipGetLastError();
}

hipError_t launch_affine(const void *x, const float *scale, const float *shift, void *y,
                         int64_t pixels, int C, int cx, bool relu, hipStream_t s) {
  const int64_t total = pixels * (C / 8);
  hapi_launch(relu ? affine_kernel<true> : affine_kernel<false>, dim3(blocks_for(total, 256)),
              dim3(256), 0, s, (const uint16_t *)x, scale, shift, (uint16_t *)y, pixels, C, cx);
  return hipGetLastError();
}

hipError_t launch_pack_affine(const float *bn, int C, float *scale, float *shift, hipStream_t s) {
  hapi_launch(pack_affine_kernel, dim3(blocks_for(C, 256)), dim3(256), 0, s, bn, C, scale,
                     shift);
  return hipGetLastError();
}

hipError_t launch_nchw_to_nhwc8(const void *x, void *y, int n, int C, int H, int W, hipStream_t s) {
  if (C < 1 || C > 8) return hipErrorInvalidValue;
  const int64_t total = (int64_t)n * H * W;
  hapi_launch(nhwc8_kernel, dim3(blocks_for(total, 256)), dim3(256), 0, s, (const uint16_t *)x, (uint16_t *)y, n,
              C, (int64_t)H * W);
  return hipGetLastError();
}

hipError_t launch_space_to_depth(const void *x, void *y, int n, int C, int H, int W, int pad,
                                 int HP, int WP, hipStream_t s) {
  const int64_t total = (int64_t)n * HP * WP;
  hapi_launch(s2d_kernel, dim3(blocks_for(total, 256)), dim3(256), 0, s,
                     (const uint16_t *)x, (uint16_t *)y, n, C, H, W, pad, HP, WP);
  return hipGetLastError();
}

hipError_t launch_maxpool(bool bf16, const void *x, void *y, int n, int H, int W, int C, int k,
                          int stride, int pad, int Ho, int Wo, hipStream_t s) {
  const int64_t total = (int64_t)n * Ho * Wo * (C / 8);
  if (bf16)
    hapi_launch(maxpool_kernel<uint16_t>, dim3(blocks_for(total, 256)), dim3(256), 0, s,
                       (const uint16_t *)x, (uint16_t *)y, n, H, W, C, k, stride, pad, Ho, Wo);
  else
    hapi_launch(maxpool_kernel<float>, dim3(blocks_for(total, 256)), dim3(256), 0, s,
                       (const float *)x, (float *)y, n, H, W, C, k, stride, pad, Ho, Wo);
  return hipGetLastError();
}

hipError_t launch_avgpool(bool bf16, const void *x, void *y, int n, int H, int W, int C, int k,
                          int stride, int Ho, int Wo, hipStream_t s) {
  const int64_t total = (int64_t)n * Ho * Wo * C;
  if (bf16 && C % 8 == 0 && (uintptr_t)x % 16 == 0 && (uintptr_t)y % 16 == 0)
    hapi_launch(avgpool8_kernel, dim3(blocks_for(total / 8, 256)), dim3(256), 0, s, (const uint16_t *)x,
                (uint16_t *)y, n, H, W, C, k, stride, Ho, Wo);
  else if (bf16)
    hapi_launch(avgpool_kernel<uint16_t>, dim3(blocks_for(total, 256)), dim3(256), 0, s,
                       (const uint16_t *)x, (uint16_t *)y, n, H, W, C, k, stride, Ho, Wo);
  else
    hapi_launch(avgpool_kernel<float>, dim3(blocks_for(total, 256)), dim3(256), 0, s,
                       (const float *)x, (float *)y, n, H, W, C, k, stride, Ho, Wo);
  return hipGetLastError();
}

static hipError_t launch_transpose(bool bf16, const void *x, void *y, int n, int R, int S,
                                   hipStream_t s) {
  const dim3 grid((S + 63) / 64, (R + 63) / 64, n);
  if (bf16)
    hapi_launch(transpose_kernel<uint16_t>, grid, dim3(256), 0, s, (const uint16_t *)x,
                       (uint16_t *)y, R, S);
  else
    hapi_launch(transpose_kernel<float>, grid, dim3(256), 0, s, (const float *)x,
                       (float *)y, R, S);
  return hipGetLastError();
}

hipError_t launch_nhwc_to_nchw(bool bf16, const void *x, void *y, int n, int HW, int C,
                               hipStream_t s) {
  return launch_transpose(bf16, x, y, n, HW, C, s);
}

hipError_t launch_nchw_to_nhwc(bool bf16, const void *x, void *y, int n, int HW, int C,
                               hipStream_t s) {
  return launch_transpose(bf16, x, y, n, C, HW, s);
}

hipError_t launch_copy(const void *x, void *y, size_t bytes, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  if (((uintptr_t)x % 16) == 0 && ((uintptr_t)y % 16) == 0 && bytes % 16 == 0) {
    const int64_t n16 = (int64_t)(bytes / 16);
    const int blocks = (int)std::min<int64_t>(blocks_for(n16, 256), 8192);
    hapi_launch(copy16_kernel, dim3(blocks), dim3(256), 0, s, (const uint4 *)x, (uint4 *)y, n16);
  } else {
    hapi_launch(copy1_kernel, dim3(blocks_for((int64_t)bytes, 256)), dim3(256), 0, s,
                       (const uint8_t *)x, (uint8_t *)y, (int64_t)bytes);
  }
  return hipGetLastError();
}

hipError_t launch_copy_f32(const float *x, float *y, int64_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hapi_launch(copy_f32_kernel, dim3(blocks_for(n, 256)), dim3(256), 0, s, x, y, n);
  return hipGetLastError();
}

hipError_t launch_fill_pattern(bool bf16, void *y, int64_t n, uint32_t seed, float scale,
                               hipStream_t s) {
  if (n == 0) return hipSuccess;
  if (bf16)
    hapi_launch(fill_kernel<uint16_t>, dim3(blocks_for(n, 256)), dim3(256), 0, s,
                       (uint16_t *)y, n, seed, scale);
  else
    hapi_launch(fill_kernel<float>, dim3(blocks_for(n, 256)), dim3(256), 0, s, (float *)y,
                       n, seed, scale);
  return hipGetLastError();
}

hipError_t launch_tokens(const void *patch, const float *cls, const float *pos, void *y, int n,
                         int T, int D, hipStream_t s) {
  const int64_t total = (int64_t)n * T * (D / 8);
  hapi_launch(tokens_kernel, dim3(blocks_for(total, 256)), dim3(256), 0, s,
                     (const uint16_t *)patch, cls, pos, (uint16_t *)y, n, T, D);
  return hipGetLastError();
}

hipError_t launch_layernorm(const void *x, const float *gamma, const float *beta, void *y,
                            int64_t rows, int D, float eps, hipStream_t s) {
  hapi_launch(layernorm_kernel, dim3(blocks_for(rows, 4)), dim3(256), 0, s,
                     (const uint16_t *)x, gamma, beta, (uint16_t *)y, rows, D, eps);
  return hipGetLastError();
}

hipError_t launch_pack_conv(bool bf16, const float *w, const float *conv_bias, const float *gamma,
                            const float *beta, const float *mean, const float *var, int N, int C,
                            int kh, int kw, int kcols, int ldw, int koff, bool acc_bias,
                            PackOrder order, void *wp, float *bias_out, hipStream_t s) {
  const int64_t total = (int64_t)N * kcols;
  if (bf16)
    hapi_launch(pack_conv_kernel<uint16_t>, dim3(blocks_for(total, 256)), dim3(256), 0, s,
                       w, conv_bias, gamma, beta, mean, var, N, C, kh, kw, kcols, ldw, koff,
                       (int)acc_bias, (int)order, (uint16_t *)wp, bias_out);
  else
    hapi_launch(pack_conv_kernel<float>, dim3(blocks_for(total, 256)), dim3(256), 0, s,
                       w, conv_bias, gamma, beta, mean, var, N, C, kh, kw, kcols, ldw, koff,
                       (int)acc_bias, (int)order, (float *)wp, bias_out);
  return hipGetLastError();
}

}  // namespace hapi
