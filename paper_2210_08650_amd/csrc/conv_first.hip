// First convolution over few input channels for gfx950 (VGG-16's 3 x 3 over
// RGB): the images in NHWC with 8 channel slots (16 bytes per pixel, zeros
// past the real channels), 64 output channels, bf16.
//
// Such a layer writes 64 channels for every 8-slot input pixel, so it is
// bound by its output stores; the implicit-GEMM pipeline spends most of its
// time in LDS staging and per-tile epilogues instead.  Here a wave keeps the
// whole packed weight matrix [64][k] in registers as MFMA A fragments and
// walks an output row 32 pixels at a time: each lane loads the 16-byte slot
// chunk of its pixel under two kernel taps per k-step straight from global
// memory (one B fragment); LDS only stages the output for whole-pixel stores.
//
// Reduction order: k = (tap, slot) in sequence, 16 columns (two taps) per
// MFMA step, as the implicit-GEMM kernels run it; their further k-steps only
// add exact zeros (taps past kh x kw), so the results are the same bits.
// Operands are swapped (weights as A) so a lane's accumulators hold 4
// consecutive channels of one pixel; half-wave exchanges give each lane 8
// consecutive channels, stored as 16-byte chunks after bias, ReLU and one
// rounding, staged through LDS so that stores cover whole pixels.
#include <cstdint>

#include "internal.h"

namespace hapi {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kFirstN = 64;     // output channels
constexpr int kFirstWaves = 4;  // waves per workgroup, one output row each

// KS k-steps of two taps each (kh x kw <= 2 KS).
template <int KS>
__global__ __launch_bounds__(64 * kFirstWaves) void conv_first_kernel(ConvArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lrow = lane & 31, lh = lane >> 5;
  // Each wave's 32 x 64 output block is staged here so that every store
  // instruction writes 8 whole pixels (1 KB contiguous): chunk c (8
  // channels) of pixel p sits at p * 8 + (c ^ (p & 7)).
  __shared__ uint4 stage[kFirstWaves][32 * 8];
  const int64_t row = (int64_t)blockIdx.x * kFirstWaves + wave;  // (image, output row)
  if (row >= (int64_t)a.n_img * a.Ho) return;
  const int img = (int)(row / a.Ho), ho = (int)(row - (int64_t)img * a.Ho);
  const uint16_t *x = static_cast<const uint16_t *>(a.x);
  const uint16_t *w = static_cast<const uint16_t *>(a.w);
  uint16_t *y = static_cast<uint16_t *>(a.y);

  // A fragments: output channel 32 j + lane % 32, k = 16 s + 8 (lane / 32) .. + 8.
  bf16x8_t wf[2][KS];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int s = 0; s < KS; ++s)
      wf[j][s] = *reinterpret_cast<const bf16x8_t *>(w + (int64_t)(32 * j + lrow) * a.Kp + 16 * s + 8 * lh);
  // Bias of the 8 channels 32 j + 16 q + 8 (lane / 32) .. + 8 this lane stores.
  float bs[2][2][8];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int e = 0; e < 8; ++e) bs[j][q][e] = a.bias ? a.bias[32 * j + 16 * q + 8 * lh + e] : 0.0f;

  // This lane's tap of k-step s is 2 s + lane / 32: input offset (du, dv).
  int du[KS], dv[KS];
  bool tap_ok[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    const int t = 2 * s + lh;
    tap_ok[s] = t < a.kh * a.kw;
    du[s] = tap_ok[s] ? t / a.kw : 0;
    dv[s] = tap_ok[s] ? t - (t / a.kw) * a.kw : 0;
  }
  const int64_t img_px = (int64_t)img * a.H * a.W;
  const int hi0 = ho * a.stride - a.pad;

  // B fragments of the 32 output pixels from column wo0: the 8 slots of the
  // input pixel under this lane's tap, zero outside the image.  Branch-free:
  // a chunk outside reads the image's first pixel; bit s of the mask says
  // whether k-step s is inside, and the zeroing (a select) happens where the
  // fragment is used: zeroing a load's destination right after issuing it
  // would make the wave wait for that load first.
  auto load = [&](int wo0, bf16x8_t xf[KS], uint32_t &okm) {
    const int wo = wo0 + lrow;
    const int wi0 = wo * a.stride - a.pad;
    okm = 0;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int hi = hi0 + du[s], wi = wi0 + dv[s];
      const bool ok = tap_ok[s] && wo < a.Wo && (unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W;
      const int64_t pix = ok ? img_px + (int64_t)hi * a.W + wi : img_px;
      xf[s] = __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const uint4 *>(x + pix * 8));
      okm |= ok ? 1u << s : 0u;
    }
  };
  auto masked = [](bf16x8_t f, uint32_t okm, int s) {
    const uint32_t keep = (okm >> s) & 1u ? ~0u : 0u;
    const uint4 v = __builtin_bit_cast(uint4, f);
    return __builtin_bit_cast(bf16x8_t, make_uint4(v.x & keep, v.y & keep, v.z & keep, v.w & keep));
  };

  bf16x8_t cur[KS], nxt[KS];
  uint32_t okc, okn = 0;
  load(0, cur, okc);
  for (int wo0 = 0; wo0 < a.Wo; wo0 += 32) {
    if (wo0 + 32 < a.Wo) load(wo0 + 32, nxt, okn);  // next block's loads fly over this block's MFMAs and stores
    f32x16_t acc[2];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[j][e] = 0.0f;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const bf16x8_t b = masked(cur[s], okc, s);
      acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[0][s], b, acc[0], 0, 0, 0);
      acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[1][s], b, acc[1], 0, 0, 0);
    }
    // acc[j][4 g + e] = channel 32 j + 8 g + 4 (lane / 32) + e of pixel wo0 + lane % 32;
    // after the exchange of part q a lane owns channels 32 j + 16 q + 8 (lane / 32) .. + 8.
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        float v[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[j][8 * q + e]),
                                                           __float_as_uint(acc[j][8 * q + 4 + e]), false, false);
          v[e] = __uint_as_float(sw[0]) + bs[j][q][e];
          v[4 + e] = __uint_as_float(sw[1]) + bs[j][q][4 + e];
        }
        uint32_t o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e)
          o[e] = a.relu ? f2bf2(fmaxf(v[2 * e], 0.0f), fmaxf(v[2 * e + 1], 0.0f)) : f2bf2(v[2 * e], v[2 * e + 1]);
        const int c = 4 * j + 2 * q + lh;
        stage[wave][lrow * 8 + (c ^ (lrow & 7))] = make_uint4(o[0], o[1], o[2], o[3]);
      }
    // The wave's LDS accesses complete in order; the fences keep the compiler
    // from moving the reads above the other lanes' writes (and the next
    // block's writes above these reads).
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int p = (lane >> 3) + 8 * i, c = lane & 7;
      const uint4 v = stage[wave][p * 8 + (c ^ (p & 7))];
      if (wo0 + p < a.Wo) *reinterpret_cast<uint4 *>(y + (row * a.Wo + wo0 + p) * a.ldc + 8 * c) = v;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int s = 0; s < KS; ++s) cur[s] = nxt[s];
    okc = okn;
  }
}

}  // namespace

bool conv_first_supported(const ConvArgs &a) {
  // the kernel reads 16 KS weight columns per row (KS = 5 or 8)
  const int ks = a.kh * a.kw <= 10 ? 5 : 8;
  return a.N == kFirstN && !a.res && !a.gelu && a.C == 8 && a.kh * a.kw <= 16 && a.Kp >= 16 * ks &&
         a.ldc >= kFirstN && a.ldc % 8 == 0 && (int64_t)a.n_img * a.Ho <= 0x7fffffffLL * kFirstWaves;
}

hipError_t launch_conv_first(const ConvArgs &a, hipStream_t s) {
  if (!conv_first_supported(a)) return hipErrorInvalidValue;
  const int64_t rows = (int64_t)a.n_img * a.Ho;
  const dim3 grid((unsigned)((rows + kFirstWaves - 1) / kFirstWaves));
  if (a.kh * a.kw <= 10)
    hapi_launch(conv_first_kernel<5>, grid, dim3(64 * kFirstWaves), 0, s, a);
  else
    hapi_launch(conv_first_kernel<8>, grid, dim3(64 * kFirstWaves), 0, s, a);
  return hipGetLastError();
}

}  // namespace hapi
