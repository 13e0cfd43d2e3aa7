// Internal declarations shared by the host runtime and the HIP kernels of libhapi.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdlib>

#include "hapi.h"

namespace hapi {

// bfloat16 from float32 on the device, rounded to nearest even
// (v_cvt_pk_bf16_f32: identical to integer RNE on every finite value,
// denormals included; a NaN stays a NaN).  f2bf2 packs (lo, hi) into one word.
typedef __bf16 bf16x2_dev_t __attribute__((ext_vector_type(2)));
typedef float f32x2_dev_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ __forceinline__ uint32_t f2bf2(float lo, float hi) {
  const f32x2_dev_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_dev_t));
}
// Per-half maximum of two packed pairs of non-negative bf16 values: for those
// the order of the bit patterns as unsigned integers is the order of the values.
__device__ __forceinline__ uint32_t bf16x2_max(uint32_t x, uint32_t y) {
  return max(x & 0xffffu, y & 0xffffu) | (max(x >> 16, y >> 16) << 16);
}

// ---------------------------------------------------------------- launches

// Timing events for the next kernel launch of this thread (kernel
// statistics).  When set, the launch records them at the start and the end of
// the dispatch itself, so the measured time is the kernel's own duration.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
LaunchEvents &launch_events();

// Records a printf-style message for hapi_last_error() and returns `code`.
int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));

// Every kernel of the library is launched through here.
template <typename F, typename... Args>
inline void hapi_launch(F kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s, Args... args) {
  LaunchEvents &e = launch_events();
  hipEvent_t a = e.start, b = e.stop;
  e.start = e.stop = nullptr;
  hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, a, b, 0u, args...);
}

// ---------------------------------------------------------------- kernels

// Where a convolution reads its input from.
enum Loader : int {
  LD_NHWC = 0,       // NHWC activation, cin % 64 == 0 (bf16) / cin % 16 == 0 (f32)
  LD_GEMM = 1,       // row-major [M, K] matrix: a 1x1 / stride 1 / pad 0 convolution
  LD_NCHW = 2,       // NCHW images, any geometry, element gather (first layer)
  LD_NCHW_PATCH = 3, // NCHW images, non-overlapping patches with k % 8 == 0 (bf16)
  LD_S2D = 4,        // space-to-depth cells (see launch_space_to_depth): every k-tile
                     // is one contiguous 64-element run, zero border, no bounds checks
  LD_CAT = 5,        // two sources along K: k < K1 as LD_NHWC over x, k >= K1 a 1x1
                     // convolution with stride s2 over x2 (a residual block's shortcut)
  LD_NHWC8 = 6       // NHWC with 8 channel slots per pixel (C <= 8, zero padded; see
                     // launch_nchw_to_nhwc8): k = (tap, c8), a 64-wide k-tile holds 8
                     // taps, 9 .. 16 taps in two k-tiles (first layers over images)
};

// Weight order of a packed convolution.
enum PackOrder : int {
  PACK_KHKWC = 0,  // k = (kh, kw, c)       NHWC inputs
  PACK_CKHKW = 1,  // k = (c, kh, kw)       NCHW inputs
  PACK_S2D = 2,    // k = (du, dv, a, b, c4) stride-2 convolution on 2x2 cells
  PACK_KHKWC8 = 3  // k = (kh, kw, c8): 8 channel slots per tap (LD_NHWC8)
};

// One convolution / linear layer as an implicit GEMM:
//   y[m, n] = act( sum_k A[m, k] * Wp[n, k] + bias[n] (+ res[m, n]) )
// m = (image, ho, wo) in NHWC order, n = output channel,
// k = (kh, kw, c) for NHWC inputs and (c, kh, kw) for NCHW inputs.
struct ConvArgs {
  const void *x;       // input activation
  const void *w;       // packed weights [N][Kp], zero padded beyond K
  const float *bias;   // [N] float32, may be null
  const void *res;     // residual [M][ldr] in the activation type, may be null
  void *y;             // output [M][ldc]
  int n_img, H, W, C;  // input geometry
  int Ho, Wo;
  int kh, kw, stride, pad;
  int M, N, K, Kp;
  int ldc, ldr;
  int relu, gelu;
  // LD_CAT only: second source [n, H2, W2, C2] NHWC, read at stride s2; K1 = % 64
  const void *x2;
  int H2, W2, C2, s2, K1;
  // LD_GEMM only: row stride of x in elements (0: K), and a pre-activation
  // applied to every element of x as it is read, x' = ReLU(x * pre_scale[k] +
  // pre_shift[k]) rounded to bf16 (pre_scale null: none; K <= kPreMax).
  int lda;
  const float *pre_scale, *pre_shift;
  // Workgroups of the persistent kernels (0: one per CU).
  int cus;
  // Tiles in reverse order (results do not depend on the order).
  int rev;
  // Partitions in flight on the device (kernels of the others may fill the
  // CUs this launch leaves idle); tile choice only, never the results.
  int lanes;
  // > 0: y is the caller's NCHW tensor [n][N][out_hw] (a split output stored
  // from the epilogue, out_hw = Ho * Wo); 0: NHWC rows y[M][ldc].  bf16 only;
  // launch_conv_bf16 returns hipErrorNotSupported when the layer's kernel
  // cannot store it, before launching anything.
  int out_hw;
  // 1: the convolution is followed by 2 x 2 / 2 max pooling, which the
  // epilogue applies before storing: GEMM row m is pixel
  // (2 hp + (m & 2) / 2, 2 wp + (m & 1)) of pooling window m / 4 =
  // (image, hp, wp), and y is the pooled output [M / 4][ldc].  bf16, NHWC
  // loader, ReLU, even Ho and Wo, N % 16 == 0, no residual; launch_conv_bf16
  // returns hipErrorNotSupported, having launched nothing, otherwise.
  int pool;
  // fp32 only: the k-tiles split into `splits` consecutive slices computed by
  // separate workgroups into part [splits][M][N] (float32), then summed in
  // slice order (fixed, so results do not depend on M); splits <= 1: none.
  float *part;
  int splits;
};
// Slices of an fp32 convolution's reduction: a function of the padded K only.
inline int f32_splits(int Kp) {
  // One slice per 256 k (16 k-tiles), at most 16: AlexNet b4 23.2k -> 25.5k
  // img/s against one per 512 (at most 8); one per 128 is slower again (the
  // partial sums' traffic).
  const int s = Kp / 256;
  return s < 1 ? 1 : s > 16 ? 16 : s;
}
constexpr int kPreMax = 1024;

hipError_t launch_conv_bf16(const ConvArgs &a, Loader ld, hipStream_t s);
hipError_t launch_conv_f32(const ConvArgs &a, Loader ld, hipStream_t s);
// The ordered sum of an fp32 convolution's slices (a.splits > 1), then its
// bias, residual and activation, into a.y.
hipError_t launch_f32_split_reduce(const ConvArgs &a, hipStream_t s);

// Elementwise / memory-bound kernels; `bf16` selects the activation type.
hipError_t launch_maxpool(bool bf16, const void *x, void *y, int n, int H, int W, int C, int k,
                          int stride, int pad, int Ho, int Wo, hipStream_t s);
hipError_t launch_avgpool(bool bf16, const void *x, void *y, int n, int H, int W, int C, int k,
                          int stride, int Ho, int Wo, hipStream_t s);
// [n, HW, C] <-> [n, C, HW]
hipError_t launch_nhwc_to_nchw(bool bf16, const void *x, void *y, int n, int HW, int C,
                               hipStream_t s);
hipError_t launch_nchw_to_nhwc(bool bf16, const void *x, void *y, int n, int HW, int C,
                               hipStream_t s);
hipError_t launch_copy(const void *x, void *y, size_t bytes, hipStream_t s);
hipError_t launch_fill_pattern(bool bf16, void *y, int64_t n, uint32_t seed, float scale,
                               hipStream_t s);
hipError_t launch_tokens(const void *patch, const float *cls, const float *pos, void *y, int n,
                         int T, int D, hipStream_t s);
hipError_t launch_layernorm(const void *x, const float *gamma, const float *beta, void *y,
                            int64_t rows, int D, float eps, hipStream_t s);
hipError_t launch_attention(const void *qkv, void *out, int n, int T, int D, int heads,
                            hipStream_t s);
// Weight packing in the given k order (see PackOrder): writes columns
// [koff, koff + kcols) of rows n < N with row pitch ldw (columns past the
// weight's own K are zero), and the folded bias (added to bias_out when
// acc_bias, else stored).
hipError_t launch_pack_conv(bool bf16, const float *w, const float *conv_bias, const float *gamma,
                            const float *beta, const float *mean, const float *var, int N, int C,
                            int kh, int kw, int kcols, int ldw, int koff, bool acc_bias,
                            PackOrder order, void *wp, float *bias_out, hipStream_t s);
// Space-to-depth for a stride-2 convolution with C <= 4 input channels:
// y[n][P][Q][(a*2 + b)*4 + c] = x[n][c][2P + a - pad][2Q + b - pad] (0 outside
// the image or for c >= C), P < HP, Q < WP.  bf16 only.
// NCHW bf16 images with C <= 8 channels -> NHWC with 8 channel slots per
// pixel, the slots past C zero: y[n][h][w][0..7].
hipError_t launch_nchw_to_nhwc8(const void *x, void *y, int n, int C, int H, int W, hipStream_t s);
hipError_t launch_space_to_depth(const void *x, void *y, int n, int C, int H, int W, int pad,
                                 int HP, int WP, hipStream_t s);
constexpr int kS2DChannels = 16;
// Fused ResNet stem: 7 x 7 stride-2 pad-3 convolution on space-to-depth cells
// (packed weights [64][ldw] in PACK_S2D order, float32 bias, ReLU, one bf16
// rounding) and 3 x 3 stride-2 pad-1 max pooling, from NCHW bf16 images to the
// pooled NHWC output [n, Hp, Wp, 64].  bf16 only; see stem_pool_supported.
// Row-streaming 3 x 3 stride-1 pad-1 convolution with 64 input and output
// channels (NHWC bf16, width <= 64): weights resident in LDS, input rows
// streamed once.  k = (kh, kw, c), packed [64][ldw]; optional residual;
// cus = CUs to fill.
bool conv3x3_c64_supported(int C, int N, int kh, int kw, int stride, int pad, int W, int Kp, int ldc, int ldr);
// With w3 (packed [256][ldw3], K = 64) the ReLU'd, bf16-rounded result is
// expanded in the same kernel by a 1 x 1 convolution to 256 channels with
// bias3, the residual res [.][ldr] (required: hipErrorInvalidValue without)
// and ReLU, into y [.][ldc] (a bottleneck's last two convolutions); see
// conv3x3_c64_expand_supported.
// pool: the ReLU'd result goes through 2 x 2 / 2 max pooling first, y being
// the pooled output [n, H/2, W/2][ldc] (relu, no residual, no expansion;
// see conv3x3_c64_pool_supported).
hipError_t launch_conv3x3_c64(const void *x, const void *w, int ldw, const float *bias, const void *res, int ldr,
                              void *y, int ldc, int n, int H, int W, bool relu, int cus, hipStream_t s,
                              const void *w3 = nullptr, int ldw3 = 0, const float *bias3 = nullptr,
                              bool pool = false);
bool conv3x3_c64_pool_supported(int H, int W, int ldc);
bool conv3x3_c64_expand_supported(int N3, int K3, int Kp3, int ldc, int ldr);
// First layer over an 8-slot NHWC input (LD_NHWC8) with 64 outputs, no
// residual: weights in registers, operands loaded straight from memory.
bool conv_first_supported(const ConvArgs &a);
hipError_t launch_conv_first(const ConvArgs &a, hipStream_t s);
// Compute units of the current device.
int cu_count();
// Two consecutive bottlenecks joined at their boundary: block i's expanding
// 1 x 1 convolution (b3 [M][ci] -> y [M][e], bias3, residual res [M][e],
// ReLU; y may equal res) and block i + 1's reducing 1 x 1 convolution
// (y -> a1 [M][co], bias1, ReLU) in one kernel, bit for bit the two
// convolutions.  w3 [e][ci] and w1 [co][e] packed bf16 (Kp == K).  Shapes
// outside bottleneck_link_supported: hipErrorInvalidValue, nothing launched.
bool bottleneck_link_supported(int ci, int e, int co, int kp3, int kp1);
hipError_t launch_bottleneck_link(const void *b3, const void *w3, const float *bias3, const void *res, void *y,
                                  const void *w1, const float *bias1, void *a1, int M, int ci, int e, int co,
                                  hipStream_t s);
bool stem_pool_supported(int C, int H, int W, int cout, int Ho, int Wo, int Hp, int Wp);
hipError_t launch_stem_pool_bf16(const void *x, const void *w, int ldw, const float *bias, void *y, int n, int C,
                                 int H, int W, int Ho, int Wo, int Hp, int Wp, int cus, hipStream_t s);
hipError_t launch_copy_f32(const float *x, float *y, int64_t n, hipStream_t s);
// Channel-slice copy (concatenation): y[p * cy + off + c] = x[p * cx + c], c < C,
// for `pixels` NHWC pixels.  C, cx, cy, off multiples of 8.  bf16.
hipError_t launch_channel_copy(const void *x, void *y, int64_t pixels, int C, int cx, int cy,
                               int off, hipStream_t s);
// Per-channel affine (+ ReLU) over the first C channels of NHWC pixels with
// row stride cx: y[p * C + c] = [max(0,] x[p * cx + c] * scale[c] + shift[c]).
// C and cx multiples of 8.  bf16.
hipError_t launch_affine(const void *x, const float *scale, const float *shift, void *y,
                         int64_t pixels, int C, int cx, bool relu, hipStream_t s);
// Inference batch-norm as a per-channel affine: scale = g / sqrt(v + 1e-5),
// shift = b - m * scale, from raw [g | b | m | v] (C each).
hipError_t launch_pack_affine(const float *bn, int C, float *scale, float *shift, hipStream_t s);

constexpr int kAttnMaxTokens = 256;
constexpr int kHeadDim = 64;

}  // namespace hapi
