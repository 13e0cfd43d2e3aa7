// Fused ResNet stem for gfx950: 7 x 7 stride-2 convolution (inference
// batch-norm folded into the packed weights and bias, ReLU) followed by 3 x 3
// stride-2 max pooling with padding 1, in one pass over the images.
//
// The convolution runs on 2 x 2 space-to-depth cells of the input, exactly
// as the implicit-GEMM kernels do for the unfused stem (k = (du, dv, a, b, c)
// over a 4 x 4 window of cells, 16 channels per cell, the same MFMA, operand
// order and k-step order, one rounding after bias and ReLU), so the pooled
// result is bit-identical to running the stem and the pooling separately.
// What changes is the data movement:
// - the cells of one input row pair are built straight from the NCHW images
//   into a ring of LDS rows (no space-to-depth buffer in HBM);
// - all 64 x 256 weight fragments stay in registers, so the MFMAs read only
//   one contiguous 1 KB slice of a cell row per k-step and wave;
// - the 112 x 112 stem output never reaches HBM: each conv row's 3-wide
//   horizontal maxima are formed in registers (half-wave exchanges and one
//   edge pixel through LDS), and a running vertical maximum emits every
//   pooled row as soon as its three conv rows are done.
// One workgroup of 4 waves handles a band of pooled rows of one image (two
// bands per image, more when the batch is too small to fill the CUs); wave w
// computes conv pixels [32 w, 32 w + 32) of every conv row of the band.
#include <cstdint>

#include "internal.h"

namespace hapi {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kStemWaves = 4;
constexpr int kStemCols = 32 * kStemWaves;  // conv pixels per row the workgroup covers
constexpr int kCellPitch = kStemCols + 4;   // cells per LDS row: pixels + 3-cell window, padded
constexpr int kRing = 6;                    // conv row r reads cell rows r .. r + 3; r + 4 is stored, r + 5 loading
constexpr int kStemN = 64;                  // output channels

__device__ __forceinline__ uint16_t bf_bits(float f) { return (uint16_t)(__float_as_uint(f) >> 16); }

struct StemArgs {
  const uint16_t *x;  // [n, C, H, W] bf16 images
  const uint16_t *w;  // packed [64][ldw] bf16, k = (du, dv, a, b, c)
  const float *bias;  // [64]
  uint16_t *y;        // [n, Hp, Wp, 64] pooled output (NHWC)
  int n, C, H, W, ldw;
  int Ho, Wo, Hp, Wp;
  int bands;  // bands of pooled rows per image
};

// Cell (P, Q) of image img: element (a * 2 + b) * 4 + c is input pixel
// (2 P + a - 3, 2 Q + b - 3) of channel c (zero outside the image or c >= C).
// Cell rows are built from dword-aligned input pairs: item (a, u) reads
// columns 2u and 2u + 1 of input row 2 P + a - 3 for every channel; column 2u
// is element b = 1 of cell u + 1 and column 2u + 1 element b = 0 of cell
// u + 2.  Cells and elements no item writes (the image border, channels
// >= C) stay zero from the ring's initialisation.
struct CellLoad {
  uint32_t v[4];  // channels 0 .. 3: columns (2u, 2u + 1), unmasked
  uint32_t keep;  // per channel bit: the item lies in the image and c < C
};

__device__ __forceinline__ CellLoad load_cells(const StemArgs &a, int img, int P, int item) {
  CellLoad L;
  const int aa = item / (a.W / 2), u = item - aa * (a.W / 2);
  const int h = 2 * P + aa - 3;
  const bool in = item < a.W && (unsigned)h < (unsigned)a.H;
  // Branch-free: an item outside the image reads pixel (0, 0) and keeps zero.
  const int64_t pix = in ? (int64_t)h * a.W + 2 * u : 0;
  const uint16_t *base = a.x + (int64_t)img * a.C * a.H * a.W + pix;
  // The mask is applied when the row is stored (a row later), so the loads
  // stay in flight across the MFMAs.
  L.keep = in ? (1u << (a.C < 4 ? a.C : 4)) - 1u : 0u;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int cc = c < a.C ? c : 0;
    L.v[c] = __builtin_nontemporal_load(reinterpret_cast<const uint32_t *>(base + (int64_t)cc * a.H * a.W));
  }
  return L;
}

__device__ __forceinline__ void store_cells(const StemArgs &a, uint16_t *row, int item, const CellLoad &L) {
  if (item >= a.W) return;
  const int aa = item / (a.W / 2), u = item - aa * (a.W / 2);
  uint32_t v[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) v[c] = (L.keep >> c) & 1u ? L.v[c] : 0u;
  const uint2 lo = make_uint2((v[0] & 0xffffu) | (v[1] << 16), (v[2] & 0xffffu) | (v[3] << 16));
  const uint2 hi = make_uint2((v[0] >> 16) | (v[1] & 0xffff0000u), (v[2] >> 16) | (v[3] & 0xffff0000u));
  *reinterpret_cast<uint2 *>(row + (u + 1) * 16 + (aa * 2 + 1) * 4) = lo;
  *reinterpret_cast<uint2 *>(row + (u + 2) * 16 + (aa * 2 + 0) * 4) = hi;
}

__global__ __launch_bounds__(64 * kStemWaves, 2) void stem_pool_kernel(StemArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t cells[kRing][kCellPitch * 16];
  __shared__ float edge[2][kStemWaves][kStemN];

  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int lrow = lane & 31, lh = lane >> 5;
  const int img = blockIdx.x / a.bands, band = blockIdx.x - img * a.bands;
  // Pooled rows [p0, p1) of this image; pooled row i takes conv rows 2i-1 .. 2i+1.
  const int p0 = band * a.Hp / a.bands, p1 = (band + 1) * a.Hp / a.bands;
  const int r0 = p0 > 0 ? 2 * p0 - 1 : 0, r1 = 2 * p1;  // conv rows [r0, r1)
  const int plast = r1 - 1 + 3;                          // last cell row needed

  // Weight fragments: column n = 32 j + lane % 32, k-step s = 4 du + dv holds
  // k = 16 s + 8 (lane / 32) .. + 8.
  bf16x8_t bw[2][16];
#pragma unroll
  for (int j = 0; j < 2; ++j)
#pragma unroll
    for (int s = 0; s < 16; ++s)
      bw[j][s] = *reinterpret_cast<const bf16x8_t *>(a.w + (int64_t)(32 * j + lrow) * a.ldw + 16 * s + 8 * lh);
  const float bias0 = a.bias ? a.bias[lrow] : 0.0f, bias1 = a.bias ? a.bias[32 + lrow] : 0.0f;
  // Every weight fragment has landed before the row loop, so no wait inside
  // the loop is attributed to them (the loop's only loads are the cell-row
  // prefetches, which must stay in flight across the MFMAs).
  __builtin_amdgcn_s_waitcnt(0x0f70);  // vmcnt(0)

  // Zero the ring once (borders and absent channels stay zero), then the
  // first four cell rows; cell row r0 + 4 is loaded into registers.
  for (int i = t; i < kRing * kCellPitch * 2; i += 64 * kStemWaves)
    reinterpret_cast<uint4 *>(&cells[0][0])[i] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  for (int P = r0; P < r0 + 4; ++P) store_cells(a, cells[P % kRing], t, load_cells(a, img, P, t));
  CellLoad pre = load_cells(a, img, r0 + 4, t);
  __syncthreads();

  const int wo = 32 * wave + lrow;  // this lane's conv pixel (may lie past Wo: computed, never pooled)
  float run[2][8];                  // running vertical maximum of the current pooled row
  // A finished pooled row is stored one conv row later, before that row's
  // cell prefetch is issued: the wait for the prefetch then finds no store
  // younger than it, and the stores had a whole row of MFMAs to complete.
  uint16_t pend[2][8];
  int pend_row = -1;
  auto store_pending = [&] {
#pragma unroll
    for (int k2 = 0; k2 < 4; ++k2) {
      // pooled columns 16 wave + 4 k2 .. + 3: all inside or all outside (Wp % 4 == 0)
      if (16 * wave + 4 * k2 < a.Wp) {
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int k1 = 0; k1 < 2; ++k1) {
            const int pc = 16 * wave + 4 * k2 + 2 * lh + k1;
            a.y[(((int64_t)img * a.Hp + pend_row) * a.Wp + pc) * kStemN + 32 * j + lrow] = pend[j][2 * k2 + k1];
          }
      }
    }
  };
  for (int r = r0; r < r1; ++r) {
    // Cell row r + 4 (loaded during the previous row) goes to the ring and
    // row r + 5 is fetched while row r computes.
    if (r + 4 <= plast) store_cells(a, cells[(r + 4) % kRing], t, pre);
    if (pend_row >= 0) {
      store_pending();
      pend_row = -1;
    }
    if (r + 5 <= plast) pre = load_cells(a, img, r + 5, t);
    f32x16_t acc0, acc1;
#pragma unroll
    for (int e = 0; e < 16; ++e) { acc0[e] = 0.0f; acc1[e] = 0.0f; }
    // A fragments of cell row r + du are read one row ahead of their MFMAs.
    bf16x8_t afr[2][4];
#pragma unroll
    for (int dv = 0; dv < 4; ++dv)
      afr[0][dv] = *reinterpret_cast<const bf16x8_t *>(cells[r % kRing] + (wo + dv) * 16 + 8 * lh);
#pragma unroll
    for (int du = 0; du < 4; ++du) {
      if (du < 3) {
        const uint16_t *row = cells[(r + du + 1) % kRing];
#pragma unroll
        for (int dv = 0; dv < 4; ++dv)
          afr[(du + 1) & 1][dv] = *reinterpret_cast<const bf16x8_t *>(row + (wo + dv) * 16 + 8 * lh);
      }
      __builtin_amdgcn_sched_barrier(0);  // keep the next row's reads ahead of these MFMAs
#pragma unroll
      for (int dv = 0; dv < 4; ++dv) {
        acc0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(afr[du & 1][dv], bw[0][4 * du + dv], acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(afr[du & 1][dv], bw[1][4 * du + dv], acc1, 0, 0, 0);
      }
    }
    // Conv outputs, rounded once: v[j][e] is channel 32 j + lane % 32 of
    // pixel 32 wave + 8 (e / 4) + 4 (lane / 32) + e % 4.
    float v[2][16];
#pragma unroll
    for (int e = 0; e < 16; e += 2) {
      const uint32_t p0 = f2bf2(fmaxf(acc0[e] + bias0, 0.0f), fmaxf(acc0[e + 1] + bias0, 0.0f));
      const uint32_t p1 = f2bf2(fmaxf(acc1[e] + bias1, 0.0f), fmaxf(acc1[e + 1] + bias1, 0.0f));
      v[0][e] = __uint_as_float(p0 << 16);
      v[0][e + 1] = __uint_as_float(p0 & 0xffff0000u);
      v[1][e] = __uint_as_float(p1 << 16);
      v[1][e + 1] = __uint_as_float(p1 & 0xffff0000u);
    }
    // Pixel 31 of this wave is the left neighbour of the next wave's pixel 0.
    if (lh) {
      edge[r & 1][wave][lrow] = v[0][15];
      edge[r & 1][wave][32 + lrow] = v[1][15];
    }
    __syncthreads();
    // Horizontal maxima: pooled column c' = 4 q + 2 (lane / 32) + {0, 1} of
    // this wave's 16 takes pixels 2c' - 1 .. 2c' + 1.
    float hm[2][8];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      float o[4];  // the other half-wave's pixel of group q, e = 3
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t u = __float_as_uint(v[j][4 * q + 3]);
        const auto sw = __builtin_amdgcn_permlane32_swap(u, u, false, false);
        o[q] = __uint_as_float(lh ? sw[0] : sw[1]);
      }
      const float left = wave > 0 ? edge[r & 1][wave - 1][32 * j + lrow] : -__builtin_inff();
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float prev = lh ? o[q] : (q == 0 ? left : o[q - 1]);
        hm[j][2 * q] = fmaxf(prev, fmaxf(v[j][4 * q], v[j][4 * q + 1]));
        hm[j][2 * q + 1] = fmaxf(v[j][4 * q + 1], fmaxf(v[j][4 * q + 2], v[j][4 * q + 3]));
      }
    }
    // Vertical: an odd conv row r = 2i + 1 completes pooled row i and starts
    // pooled row i + 1; an even row extends the current one.
    if (r & 1) {
      const int pi = (r - 1) >> 1;
      if (pi >= p0) {
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int k = 0; k < 8; ++k) pend[j][k] = bf_bits(fmaxf(run[j][k], hm[j][k]));
        pend_row = pi;
      }
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int k = 0; k < 8; ++k) run[j][k] = hm[j][k];
    } else {
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int k = 0; k < 8; ++k) run[j][k] = r == r0 ? hm[j][k] : fmaxf(run[j][k], hm[j][k]);
    }
  }
  if (pend_row >= 0) store_pending();
}

}  // namespace

bool stem_pool_supported(int C, int H, int W, int cout, int Ho, int Wo, int Hp, int Wp) {
  // one cell-load item per thread: 2 input rows x W / 2 column pairs
  return C >= 1 && C <= 4 && cout == kStemN && Wo <= kStemCols && Ho == 2 * Hp && Wo == 2 * Wp && Hp >= 2 &&
         W % 2 == 0 && W <= 64 * kStemWaves && Wp % 4 == 0 &&
         Ho == (H + 6 - 7) / 2 + 1 && Wo == (W + 6 - 7) / 2 + 1;
}

hipError_t launch_stem_pool_bf16(const void *x, const void *w, int ldw, const float *bias, void *y, int n, int C,
                                 int H, int W, int Ho, int Wo, int Hp, int Wp, int cus, hipStream_t s) {
  // Two bands per image, or enough for one workgroup per CU, with at least
  // four pooled rows per band (each band recomputes one conv row of halo).
  int bands = n > 0 ? (cus + n - 1) / n : 2;
  bands = bands < 2 ? 2 : bands;
  const int max_bands = Hp / 4 < 2 ? 2 : Hp / 4;
  bands = bands > max_bands ? max_bands : bands;
  bands = bands > Hp ? Hp : bands;
  StemArgs a{static_cast<const uint16_t *>(x), static_cast<const uint16_t *>(w), bias, static_cast<uint16_t *>(y),
             n, C, H, W, ldw, Ho, Wo, Hp, Wp, bands};
  hapi_launch(stem_pool_kernel, dim3(bands * n), dim3(64 * kStemWaves), 0, s, a);
  return hipGetLastError();
}

}  // namespace hapi
