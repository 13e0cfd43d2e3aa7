// Row-streaming 3 x 3 convolution for gfx950: stride 1, padding 1, 64 input
// and 64 output channels, NHWC bf16 (the ResNet stage-1 bottleneck and
// basic-block convolutions, VGG's second convolution).  Rows wider than 64
// pixels are cut into strips of 64 output columns, each streamed by its own
// workgroups with a one-column halo on either side.
//
// The implicit-GEMM kernels gather every k-tile of such a layer from L2 (each
// input pixel is fetched nine times, once per tap) and are bound by the
// latency of that traffic.  Here a workgroup (one per CU) keeps the whole
// weight matrix [64][576] in LDS and streams the input rows of one image band
// through a ring of LDS rows, so every input element moves from HBM to LDS
// once.  Each step computes four output rows, each split over two waves (32
// pixels x 64 channels, 36 k-steps of 2 MFMAs; two waves per SIMD) while the
// next four input rows load.
//
// Reduction order: k = (kh, kw, c) in sequence, 16 channels per MFMA step, as
// in the implicit-GEMM kernels.  The MFMA operands are swapped (weights as A)
// so a lane's accumulators hold 4 consecutive channels of one pixel; half-wave
// exchanges give each lane 8 consecutive channels, stored as 16-byte chunks
// after bias, optional residual, ReLU and one rounding.
#include <cstdint>
#include <type_traits>
#include <utility>

#include "internal.h"

namespace hapi {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kC = 64;                 // input and output channels
constexpr int kK = 9 * kC;             // 576
constexpr int kWPitch = kK + 8;        // bf16 pitch of a weight row in LDS (conflict-free fragment reads)
constexpr int kPix = 66;               // pixels per ring row: columns -1 .. 64
constexpr int kRows = 10;              // ring rows: a step reads 6, the next 4 are loading
constexpr int kStepRows = 4;           // output rows per step
constexpr int kWaves = 2 * kStepRows;  // two waves per row: 32-pixel halves
constexpr int kThreads = 64 * kWaves;
constexpr int kRowChunks = kPix * 8;   // 16-byte chunks per ring row

template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
// Calls f(integral_constant<int, i>) for i = 0 .. N-1 (compile-time indices).
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Chunk c (8 channels) of pixel slot p sits at chunk c ^ ((p >> 1) & 7): the
// 16 pixels a quarter-wave reads land in 16 distinct bank groups.
__device__ __forceinline__ int ring_off(int slot, int p, int c) { return (slot * kPix + p) * kC + ((c ^ ((p >> 1) & 7)) << 3); }

struct Conv3Args {
  const uint16_t *x;    // [n, H, W, 64]
  const uint16_t *w;    // packed [64][ldw], k = (kh, kw, c)
  const float *bias;    // [64] or null
  const uint16_t *res;  // [n * H * W][ldr] or null
  uint16_t *y;          // [n * H * W][ldc]
  int H, W, ldw, ldc, ldr, relu;
  int bands, band_rows;  // output rows [b * band_rows, ...) of each image per workgroup
  int strips;            // 64-column strips per row: workgroup (img, band, strip)
  // Expansion (EXPAND kernels): the 3 x 3 result, with bias and ReLU and
  // rounded to bf16, is the 64-channel input of a 1 x 1 convolution to
  // kExpand channels (packed [kExpand][ldw3]) with bias3, the residual res
  // and ReLU; y and res then have kExpand channels per pixel.
  const uint16_t *w3;
  const float *bias3;
  int ldw3;
};

constexpr int kExpand = 256;             // output channels of the expansion
constexpr int kW3Pitch = kC + 8;         // bf16 pitch of an expansion weight row in LDS

// EXPAND = false: the 3 x 3 convolution alone, input rows double-buffered in
// a ring of 10 (a step reads 6 while the next 4 are stored).
// EXPAND = true: the expansion weights take the LDS of four ring rows; the
// ring holds the 6 rows a step reads, and the next step's rows replace the 4
// oldest after a barrier, while the expansion runs.
// POOL = true (with EXPAND = false): the ReLU'd, rounded 3 x 3 result goes
// through 2 x 2 / 2 max pooling before it is stored, y being the pooled
// output [n, H/2, W/2][ldc] (H % 4 == 0, W even).  Each wave then computes two
// output rows x 16 columns (lane % 32 = 16 dr + dc), so that a pooling
// window's four pixels are lanes l, l ^ 1, l ^ 16 and l ^ 17 of one wave.
template <bool EXPAND, bool POOL = false>
__global__ __launch_bounds__(kThreads, 1) void conv3x3_c64_kernel(Conv3Args a) {
  static_assert(!(EXPAND && POOL), "pooling follows the plain 3 x 3 only");
  constexpr int kRing = EXPAND ? 6 : kRows;
  __shared__ __attribute__((aligned(16))) uint16_t wts[kC * kWPitch];
  __shared__ __attribute__((aligned(16))) uint16_t ring[kRing * kPix * kC];
  __shared__ __attribute__((aligned(16))) uint16_t w3s[EXPAND ? kExpand * kW3Pitch : 8];
  __shared__ __attribute__((aligned(16))) float bias_s[kC];
  __shared__ __attribute__((aligned(16))) float bias3_s[EXPAND ? kExpand : 4];

  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int lrow = lane & 31, lh = lane >> 5;
  const int per_img = a.bands * a.strips;
  const int img = blockIdx.x / per_img, rest = blockIdx.x - img * per_img;
  const int band = rest / a.strips, strip = rest - band * a.strips;
  const int c0 = strip * (kPix - 2);  // first output column of the strip
  const int r0 = band * a.band_rows;
  const int r1 = min(a.H, r0 + a.band_rows);
  const int64_t img_px = (int64_t)img * a.H * a.W;

  // Input row h (-1 .. H) lives in ring slot (h + 1) % kRing; outside the
  // image and in the padding columns it is zero.  Item it moves 16 bytes.
  // Branch-free: a chunk outside the image reads the image's first pixel and
  // is zeroed (a select) only when stored, so the loads of a whole row set
  // stay in flight; zeroing a load's destination right after issuing it
  // would make the wave wait for that load first.
  auto row_ok = [&](int h, int it) {
    const int col = c0 + (it >> 3) - 1;  // ring pixel p holds column c0 + p - 1
    return it < kRowChunks && (unsigned)h < (unsigned)a.H && (unsigned)col < (unsigned)a.W;
  };
  auto load_row = [&](int h, int it) -> uint4 {
    const int p = it >> 3, c = it & 7;
    const int64_t pix = row_ok(h, it) ? (int64_t)h * a.W + c0 + p - 1 : 0;
    return *reinterpret_cast<const uint4 *>(a.x + ((img_px + pix) << 6) + c * 8);
  };
  constexpr int kPer = (kRowChunks + kThreads - 1) / kThreads;  // chunks per thread per row
  auto store_row = [&](int h, int it, const uint4 &v) {
    const int p = it >> 3, c = it & 7;
    const uint32_t keep = row_ok(h, it) ? ~0u : 0u;
    *reinterpret_cast<uint4 *>(ring + ring_off((h + 1) % kRing, p, c)) =
        make_uint4(v.x & keep, v.y & keep, v.z & keep, v.w & keep);
  };

  // Prologue: every load (weights and the first six input rows) is issued
  // before any store, so their latencies overlap.
  {
    constexpr int kWPer = kC * (kK / 8) / kThreads;  // chunks of 16 bytes
    constexpr int kW3Per = EXPAND ? kExpand * (kC / 8) / kThreads : 1;
    uint4 wv[kWPer], w3v[kW3Per];
    uint4 iv[6][kPer];
#pragma unroll
    for (int e = 0; e < kWPer; ++e) {
      const int i = t + e * kThreads, n = i / (kK / 8), k8 = i - n * (kK / 8);
      wv[e] = *reinterpret_cast<const uint4 *>(a.w + (int64_t)n * a.ldw + k8 * 8);
    }
    if constexpr (EXPAND) {
#pragma unroll
      for (int e = 0; e < kW3Per; ++e) {
        const int i = t + e * kThreads, n = i / (kC / 8), k8 = i - n * (kC / 8);
        w3v[e] = *reinterpret_cast<const uint4 *>(a.w3 + (int64_t)n * a.ldw3 + k8 * 8);
      }
    }
#pragma unroll
    for (int q = 0; q < 6; ++q)
#pragma unroll
      for (int e = 0; e < kPer; ++e) iv[q][e] = load_row(r0 - 1 + q, t + e * kThreads);
#pragma unroll
    for (int e = 0; e < kWPer; ++e) {
      const int i = t + e * kThreads, n = i / (kK / 8), k8 = i - n * (kK / 8);
      *reinterpret_cast<uint4 *>(wts + n * kWPitch + k8 * 8) = wv[e];
    }
    if constexpr (EXPAND) {
#pragma unroll
      for (int e = 0; e < kW3Per; ++e) {
        const int i = t + e * kThreads, n = i / (kC / 8), k8 = i - n * (kC / 8);
        *reinterpret_cast<uint4 *>(w3s + n * kW3Pitch + k8 * 8) = w3v[e];
      }
    }
#pragma unroll
    for (int q = 0; q < 6; ++q)
#pragma unroll
      for (int e = 0; e < kPer; ++e)
        if (t + e * kThreads < kRowChunks) store_row(r0 - 1 + q, t + e * kThreads, iv[q][e]);
  }
  if (t < kC) bias_s[t] = a.bias ? a.bias[t] : 0.0f;
  if constexpr (EXPAND) {
    if (t < kExpand) bias3_s[t] = a.bias3 ? a.bias3[t] : 0.0f;
  }
  __syncthreads();

  // Fragment offsets: A (weights) row n = 32 j + lane % 32 at k = 16 s + 8 lh;
  // B (activations) pixel 32 i + lane % 32 (+ kw) at channel chunk 2 cs + lh.
  const int aoff0 = lrow * kWPitch + 8 * lh, aoff1 = (32 + lrow) * kWPitch + 8 * lh;
  uint16_t *y = a.y;

  for (int ho = r0; ho < r1; ho += kStepRows) {
    // The input rows of the next step load while this one computes.
    uint4 pre[4][kPer];
    const bool more = ho + kStepRows < r1;
    if (more) {
#pragma unroll
      for (int q = 0; q < 4; ++q)
#pragma unroll
        for (int e = 0; e < kPer; ++e) {
          pre[q][e] = load_row(ho + 5 + q, t + e * kThreads);
        }
    }
    // This lane's output pixel: row `row`, ring pixel px + 1, output column
    // c0 + px.  Plain: the wave's row (ho + wave % 4) and 32-pixel half;
    // POOL: rows ho + 2 (wave % 2) + lrow / 16, columns 16 (wave / 2) + lrow % 16.
    const int row = POOL ? ho + 2 * (wave & 1) + (lrow >> 4) : ho + (wave & (kStepRows - 1));
    const int px = POOL ? 16 * (wave >> 1) + (lrow & 15) : 32 * (wave / kStepRows) + lrow;
    const int64_t m = img_px + (int64_t)row * a.W + c0 + px;
    const bool live = row < r1 && c0 + px < a.W;
    // EXPAND: the residual of this lane's outputs, loaded now so that its
    // latency hides behind the 3 x 3 MFMAs.  Part (h, jn, q) holds channels
    // 128 h + 32 jn + 16 q + 8 lh .. + 8 of pixel px.  The loads are
    // unconditional (a lane outside the band reads its image's first pixel;
    // its outputs are never stored): a register zeroed for some lanes before
    // its load is issued makes the wave wait for every load in flight,
    // the next rows' included.
    uint4 rr[EXPAND ? 2 : 1][EXPAND ? 4 : 1][2];
    if constexpr (EXPAND) {
      const int64_t mr = live ? m : img_px;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int jn = 0; jn < 4; ++jn)
#pragma unroll
          for (int q = 0; q < 2; ++q)
            rr[h][jn][q] = *reinterpret_cast<const uint4 *>(a.res + mr * a.ldr + 128 * h + 32 * jn + 16 * q + 8 * lh);
    }
    f32x16_t acc[2];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[j][e] = 0.0f;
    if (POOL ? ho < r1 : row < r1) {  // POOL: the step's four rows are all inside the band
      // Fragments are read kAhead k-steps before their MFMAs (a ring of
      // kAhead + 1 register sets), so the LDS latency hides behind 2 kAhead
      // MFMAs of this wave plus those of the other wave on the SIMD.
      constexpr int kSteps = 36, kAhead = 3, kSlots = kAhead + 1;
      int slot_base[3];
#pragma unroll
      for (int kh = 0; kh < 3; ++kh) slot_base[kh] = ((row + kh) % kRing) * kPix * kC;
      bf16x8_t fw0[kSlots], fw1[kSlots], fx[kSlots];
      auto read_step = [&](int st, int sl) {
        const int kh = st / 12, kw = (st / 4) % 3, cs = st % 4;
        fw0[sl] = *reinterpret_cast<const bf16x8_t *>(wts + aoff0 + 16 * st);
        fw1[sl] = *reinterpret_cast<const bf16x8_t *>(wts + aoff1 + 16 * st);
        const int p = px + kw;
        fx[sl] = *reinterpret_cast<const bf16x8_t *>(ring + slot_base[kh] + p * kC + (((2 * cs + lh) ^ ((p >> 1) & 7)) << 3));
      };
      static_for<kAhead>([&](auto sc) { read_step(decltype(sc)::value, decltype(sc)::value); });
      static_for<kSteps>([&](auto sc) {
        constexpr int st = decltype(sc)::value, sl = st % kSlots;
        if constexpr (st + kAhead < kSteps) read_step(st + kAhead, (st + kAhead) % kSlots);
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw0[sl], fx[sl], acc[0], 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw1[sl], fx[sl], acc[1], 0, 0, 0);
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    // acc[j][4 g + e] = channel 32 j + 8 g + 4 lh + e of pixel px.  After the
    // half-wave exchange of part q, a lane owns channels 32 j + 16 q + 8 lh
    // .. + 8 of that pixel, with bias added.
    auto finish8 = [&](const f32x16_t &c, int q, const float *bsrc, float v[8]) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(c[8 * q + e]),
                                                         __float_as_uint(c[8 * q + 4 + e]), false, false);
        v[e] = __uint_as_float(sw[0]);
        v[4 + e] = __uint_as_float(sw[1]);
      }
      const float4 b0 = *reinterpret_cast<const float4 *>(bsrc);
      const float4 b1 = *reinterpret_cast<const float4 *>(bsrc + 4);
      v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
      v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
    };
    auto add_res = [&](const uint4 &rv, float v[8]) {
      const uint32_t w4[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] += __uint_as_float(w4[e] << 16);
        v[2 * e + 1] += __uint_as_float(w4[e] & 0xffff0000u);
      }
    };
    if constexpr (POOL) {
      // Max over the window (lanes l, l ^ 1, l ^ 16, l ^ 17) of the rounded,
      // non-negative bf16 values, compared as unsigned integers, as the
      // separate pooling layer computes it; the window's top-left lane stores.
      if (ho < r1) {
        const bool store = (lrow & 0x11) == 0 && c0 + px < a.W;
        const int64_t pm = ((int64_t)img * (a.H / 2) + (row >> 1)) * (a.W / 2) + ((c0 + px) >> 1);
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            const int n = 32 * j + 16 * q + 8 * lh;
            float v[8];
            finish8(acc[j], q, bias_s + n, v);
            uint32_t o[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              o[e] = f2bf2(fmaxf(v[2 * e], 0.0f), fmaxf(v[2 * e + 1], 0.0f));
              o[e] = bf16x2_max(o[e], (uint32_t)__shfl_xor((int)o[e], 1, 64));
              o[e] = bf16x2_max(o[e], (uint32_t)__shfl_xor((int)o[e], 16, 64));
            }
            if (store) *reinterpret_cast<uint4 *>(y + pm * a.ldc + n) = make_uint4(o[0], o[1], o[2], o[3]);
          }
      }
      if (more) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int e = 0; e < kPer; ++e) {
            const int it = t + e * kThreads;
            if (it < kRowChunks) store_row(ho + 5 + q, it, pre[q][e]);
          }
      }
    } else if constexpr (!EXPAND) {
      if (row < r1) {
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            const int n = 32 * j + 16 * q + 8 * lh;
            float v[8];
            finish8(acc[j], q, bias_s + n, v);
            if (c0 + px < a.W) {
              if (a.res) add_res(*reinterpret_cast<const uint4 *>(a.res + m * a.ldr + n), v);
              uint32_t o[4];
#pragma unroll
              for (int e = 0; e < 4; ++e)
                o[e] = a.relu ? f2bf2(fmaxf(v[2 * e], 0.0f), fmaxf(v[2 * e + 1], 0.0f)) : f2bf2(v[2 * e], v[2 * e + 1]);
              *reinterpret_cast<uint4 *>(y + m * a.ldc + n) = make_uint4(o[0], o[1], o[2], o[3]);
            }
          }
      }
      if (more) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int e = 0; e < kPer; ++e) {
            const int it = t + e * kThreads;
            if (it < kRowChunks) store_row(ho + 5 + q, it, pre[q][e]);
          }
      }
    } else {
      // Every wave has read the ring rows the next step's rows replace.
      __syncthreads();
      if (more) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
#pragma unroll
          for (int e = 0; e < kPer; ++e) {
            const int it = t + e * kThreads;
            if (it < kRowChunks) store_row(ho + 5 + q, it, pre[q][e]);
          }
      }
      if (row < r1) {
        // The 3 x 3 result, rounded once, is the expansion's B operand: k-step
        // s = 2 j + q covers channels 16 s .. 16 s + 15, of which this lane
        // holds 16 s + 8 lh .. + 8 of pixel px.
        bf16x8_t xb[4];
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            float v[8];
            finish8(acc[j], q, bias_s + 32 * j + 16 * q + 8 * lh, v);
            uint32_t o[4];
#pragma unroll
            for (int e = 0; e < 4; ++e)
              o[e] = a.relu ? f2bf2(fmaxf(v[2 * e], 0.0f), fmaxf(v[2 * e + 1], 0.0f)) : f2bf2(v[2 * e], v[2 * e + 1]);
            xb[2 * j + q] = __builtin_bit_cast(bf16x8_t, make_uint4(o[0], o[1], o[2], o[3]));
          }
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          f32x16_t e3[4];
#pragma unroll
          for (int jn = 0; jn < 4; ++jn)
#pragma unroll
            for (int e = 0; e < 16; ++e) e3[jn][e] = 0.0f;
#pragma unroll
          for (int s3 = 0; s3 < 4; ++s3)
#pragma unroll
            for (int jn = 0; jn < 4; ++jn) {
              const bf16x8_t wf =
                  *reinterpret_cast<const bf16x8_t *>(w3s + (128 * h + 32 * jn + lrow) * kW3Pitch + 16 * s3 + 8 * lh);
              e3[jn] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf, xb[s3], e3[jn], 0, 0, 0);
            }
#pragma unroll
          for (int jn = 0; jn < 4; ++jn)
#pragma unroll
            for (int q = 0; q < 2; ++q) {
              const int n = 128 * h + 32 * jn + 16 * q + 8 * lh;
              float v[8];
              finish8(e3[jn], q, bias3_s + n, v);
              if (c0 + px < a.W) {
                add_res(rr[h][jn][q], v);
                uint32_t o[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) o[e] = f2bf2(fmaxf(v[2 * e], 0.0f), fmaxf(v[2 * e + 1], 0.0f));
                *reinterpret_cast<uint4 *>(y + m * a.ldc + n) = make_uint4(o[0], o[1], o[2], o[3]);
              }
            }
        }
      }
    }
    __syncthreads();
  }
}

}  // namespace

bool conv3x3_c64_supported(int C, int N, int kh, int kw, int stride, int pad, int W, int Kp, int ldc, int ldr) {
  return C == kC && N == kC && kh == 3 && kw == 3 && stride == 1 && pad == 1 && W >= 1 && Kp == kK &&
         ldc % 8 == 0 && ldr % 8 == 0;
}

bool conv3x3_c64_pool_supported(int H, int W, int ldc) { return H % 4 == 0 && W % 2 == 0 && ldc % 8 == 0; }

bool conv3x3_c64_expand_supported(int N3, int K3, int Kp3, int ldc, int ldr) {
  return N3 == kExpand && K3 == kC && Kp3 == kC && ldc % 8 == 0 && ldr % 8 == 0;
}

hipError_t launch_conv3x3_c64(const void *x, const void *w, int ldw, const float *bias, const void *res, int ldr,
                              void *y, int ldc, int n, int H, int W, bool relu, int cus, hipStream_t s,
                              const void *w3, int ldw3, const float *bias3, bool pool) {
  if (pool && (w3 || res || !relu || !conv3x3_c64_pool_supported(H, W, ldc))) return hipErrorInvalidValue;
  if (w3 && !res) return hipErrorInvalidValue;
  // Enough workgroups to fill the CUs: split images into strips of columns,
  // then into bands of rows.
  const int strips = (W + kPix - 3) / (kPix - 2);
  int bands = (cus + n * strips - 1) / (n * strips);
  bands = bands < 1 ? 1 : bands;
  const int max_bands = (H + kStepRows - 1) / kStepRows;
  bands = bands > max_bands ? max_bands : bands;
  int band_rows = (H + bands - 1) / bands;
  band_rows = (band_rows + kStepRows - 1) / kStepRows * kStepRows;
  bands = (H + band_rows - 1) / band_rows;
  Conv3Args a{static_cast<const uint16_t *>(x), static_cast<const uint16_t *>(w), bias,
              static_cast<const uint16_t *>(res), static_cast<uint16_t *>(y), H, W, ldw, ldc, ldr, relu ? 1 : 0,
              bands, band_rows, strips, static_cast<const uint16_t *>(w3), bias3, ldw3};
  const int64_t grid = (int64_t)n * bands * strips;
  if (grid > 0x7fffffff) return hipErrorInvalidValue;
  if (w3)
    hapi_launch(conv3x3_c64_kernel<true>, dim3((unsigned)grid), dim3(kThreads), 0, s, a);
  else if (pool)
    hapi_launch((conv3x3_c64_kernel<false, true>), dim3((unsigned)grid), dim3(kThreads), 0, s, a);
  else
    hapi_launch(conv3x3_c64_kernel<false>, dim3((unsigned)grid), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace hapi
