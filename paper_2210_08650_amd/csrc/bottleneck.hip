// Two consecutive ResNet bottleneck blocks joined at their boundary on gfx950:
// block i's expanding 1x1 convolution (bias, identity residual, ReLU) and
// block i + 1's reducing 1x1 convolution (bias, ReLU) in one kernel, so the
// block output, which the reduction reads, never makes the round trip
// through HBM a second time.
//
// A workgroup owns 64 rows (output pixels).  The expansion's E output
// channels are produced in 64-wide chunks; each finished chunk is both
// stored (it is block i's output and block i + 1's residual) and kept in LDS
// as one 64-wide k-tile of the reduction, which accumulates it one step later.
// The arithmetic is that of the two separate convolutions exactly: the same
// v_mfma_f32_32x32x16_bf16, k-steps in the same order, the epilogues adding
// bias, then the residual, then applying ReLU with one bf16 rounding, so the
// outputs equal the unfused layers bit for bit.
//
// Waves 0-3 compute the expansion (one 32 x 32 block of each chunk per
// wave) and store it; waves 4-7 accumulate the reduction (the 64 rows x CO
// outputs split by columns); waves 8-9 only move operands into LDS by DMA:
// the 3x3 output tile once, then per step an expansion weight chunk, a
// residual chunk and a reduction weight k-tile, each P steps ahead.  Step s:
// the expansion computes chunk s while the reduction consumes chunk s - 1;
// one barrier ends the step.  The DMA waves never store and, past the bias,
// the others never load from global memory, so each wave's waits on the
// vector-memory counter (which loads and stores share) cover exactly the
// transfers it needs.
#include "internal.h"

namespace hapi {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

#define LINK_LDS(p) ((__attribute__((address_space(3))) void *)(p))

constexpr unsigned kLinkOob = 0x80000000u;  // a byte offset outside every buffer range
constexpr int kLinkBM = 64;                  // rows per workgroup
constexpr int kLinkTile = kLinkBM * 64;      // elements of a 64-row x 64-wide k-tile

// 16 bytes per lane from base + voff (offsets at or beyond kLinkOob read
// zeros) into LDS at lds + 16 * lane.
__device__ __forceinline__ void link_dma(const void *base, uint16_t *lds, unsigned voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, 0x7fffffff, 0x00020000), LINK_LDS(lds), 16,
      voff, 0, 0, 0);
}

// One DMA instruction of a 64-wide k-tile: rows 8 g .. 8 g + 7 of the tile,
// lane l moving row 8 g + l / 8, physical 16-byte chunk l % 8, which holds
// logical chunk (l % 8) ^ ((row >> 1) & 7) (the XOR swizzle that keeps
// fragment reads free of bank conflicts).  Source: row r0 + row of a
// row-major [rows][ld] bf16 matrix, columns k0 ...
__device__ __forceinline__ void link_dma_rows(const uint16_t *src, int rows, int ld, int r0, int k0, uint16_t *tile,
                                              int g, int lane) {
  const int row = 8 * g + (lane >> 3);
  const int lc = (lane & 7) ^ ((row >> 1) & 7);
  const unsigned voff = r0 + row < rows ? (unsigned)((((int64_t)(r0 + row) * ld) + k0 + lc * 8) * 2) : kLinkOob;
  link_dma(src, tile + g * 512, voff);
}

// Fragment of k-step ks (16 k values) for row r (32-aligned block + lane % 32)
// of a swizzled 64-wide k-tile.
__device__ __forceinline__ bf16x8_t link_frag(const uint16_t *tile, int r, int ks, int lh) {
  return *reinterpret_cast<const bf16x8_t *>(tile + r * 64 + (((2 * ks + lh) ^ ((r >> 1) & 7)) << 3));
}

// Workgroup barrier after this wave's LDS writes completed (no wait on its
// global memory operations, unlike __syncthreads).
__device__ __forceinline__ void link_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_s_barrier();
}

template <int N>
__device__ __forceinline__ void link_vmwait() {
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

struct LinkArgs {
  const uint16_t *b3;  // [M][CI] block i's 3x3 output, the expansion's input
  const uint16_t *w3;  // [E][CI] packed expansion weights
  const float *bias3;  // [E]
  const uint16_t *res; // [M][E] the residual (block i's input or its projection shortcut)
  uint16_t *y;         // [M][E] block i's output; may be res itself (each element is read
                       // by the lane that later writes it)
  const uint16_t *w1;  // [CO][E] packed reduction weights of block i + 1
  const float *bias1;  // [CO]
  uint16_t *a1;        // [M][CO] block i + 1's reduction output
  int M;
};

template <int... I, class F>
__device__ __forceinline__ void link_steps_impl(F &&f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void link_steps(F &&f) {
  link_steps_impl(f, std::make_integer_sequence<int, N>{});
}

constexpr int kLinkDmaWaves = 2;  // waves that only move operands into LDS
constexpr int kLinkThreads = 64 * (8 + kLinkDmaWaves);

// DMA instructions per DMA wave that carry the operands of step q (see the
// kernel), and those of steps lo .. hi together.
template <int KTI, int NS, int CO>
constexpr int link_issued(int q) {
  return ((q < NS ? KTI * 8 + 8 : 0) + (q >= 1 && q <= NS ? CO / 8 : 0)) / kLinkDmaWaves;
}
template <int KTI, int NS, int CO>
constexpr int link_in_flight(int lo, int hi) {
  int n = 0;
  for (int q = lo; q <= hi && q <= NS; ++q) n += link_issued<KTI, NS, CO>(q);
  return n;
}

// P: prefetch distance in steps of every streamed operand (expansion weight
// chunks, residual chunks, reduction weight k-tiles); rings of P + 1 buffers.
// Each role runs its own loop over the steps, so that the waits the compiler
// places for one role's memory operations never land in another's.
template <int CI, int E, int CO, int P>
__global__ __launch_bounds__(kLinkThreads, 1) void bottleneck_link_kernel(LinkArgs a) {
  static_assert(CI % 64 == 0 && E % 64 == 0 && CO % 128 == 0 && CO <= 256 && P >= 1, "shape");
  constexpr int KTI = CI / 64;   // expansion k-tiles
  constexpr int NS = E / 64;     // chunks = reduction k-tiles
  constexpr int TNR = CO / 128;  // reduction 32-column blocks per wave
  constexpr int D = P + 1;       // ring depth
  static_assert((KTI * 8) % kLinkDmaWaves == 0 && 8 % kLinkDmaWaves == 0 && (CO / 8) % kLinkDmaWaves == 0, "DMA split");
  __shared__ __attribute__((aligned(16))) uint16_t b3s[KTI][kLinkTile];
  __shared__ __attribute__((aligned(16))) uint16_t w3s[D][KTI][kLinkTile];
  __shared__ __attribute__((aligned(16))) uint16_t w1s[D][CO * 64];
  __shared__ __attribute__((aligned(16))) uint16_t rs[D][kLinkTile];
  __shared__ __attribute__((aligned(16))) uint16_t xs[2][kLinkTile];
  __shared__ __attribute__((aligned(16))) float b3f[E];
  __shared__ __attribute__((aligned(16))) float b1f[CO];

  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int lrow = lane & 31, lh = lane >> 5;
  const int m0 = blockIdx.x * kLinkBM;

  for (int i = t; i < E; i += kLinkThreads) b3f[i] = a.bias3 ? a.bias3[i] : 0.0f;
  for (int i = t; i < CO; i += kLinkThreads) b1f[i] = a.bias1 ? a.bias1[i] : 0.0f;

  if (wave >= 8) {
    // ---- DMA waves.  Operands of step q: expansion weight chunk q and
    // residual chunk q (q < NS), reduction weight k-tile q - 1 (q >= 1);
    // instruction i of a transfer goes to DMA wave i % kLinkDmaWaves.
    const int dw = wave - 8;
    constexpr int kW3 = KTI * 8 / kLinkDmaWaves, kRs = 8 / kLinkDmaWaves, kW1 = CO / 8 / kLinkDmaWaves;
    auto issue = [&](auto qc) {
      constexpr int q = decltype(qc)::value;
      if constexpr (q < NS) {
#pragma unroll
        for (int i = 0; i < kW3; ++i) {
          const int qq = dw + kLinkDmaWaves * i, kt = qq >> 3, g = qq & 7;
          link_dma_rows(a.w3, E, CI, 64 * q, 64 * kt, w3s[q % D][kt], g, lane);
        }
#pragma unroll
        for (int i = 0; i < kRs; ++i)
          link_dma_rows(a.res, a.M, E, m0, 64 * q, rs[q % D], dw + kLinkDmaWaves * i, lane);
      }
      if constexpr (q >= 1 && q <= NS) {
#pragma unroll
        for (int i = 0; i < kW1; ++i)
          link_dma_rows(a.w1, CO, E, 0, 64 * (q - 1), w1s[(q - 1) % D], dw + kLinkDmaWaves * i, lane);
      }
    };
#pragma unroll
    for (int i = 0; i < KTI * 8 / kLinkDmaWaves; ++i) {
      const int qq = dw + kLinkDmaWaves * i, kt = qq >> 3, g = qq & 7;
      link_dma_rows(a.b3, a.M, CI, m0, 64 * kt, b3s[kt], g, lane);
    }
    link_steps<P>([&](auto qc) { issue(qc); });
    // the 3x3 tile and the operands of step 0 landed; steps 1 .. P - 1 may fly
    link_vmwait<link_in_flight<KTI, NS, CO>(1, P - 1)>();
    link_barrier();
    link_steps<NS + 1>([&](auto sc) {
      constexpr int s = decltype(sc)::value;
      if constexpr (s + P <= NS) issue(std::integral_constant<int, s + P>{});
      // operands of step s + 1 landed; those of steps s + 2 .. s + P may fly
      if constexpr (s + 1 <= NS) link_vmwait<link_in_flight<KTI, NS, CO>(s + 2, s + P)>();
      __builtin_amdgcn_s_barrier();
    });
    return;
  }
  link_barrier();

  if (wave < 4) {
    // ---- Expansion waves: block rows eb .. eb + 31, columns ec .. ec + 31
    // of every chunk.
    const int eb = 32 * (wave >> 1 & 1), ec = 32 * (wave & 1);
    const int r = eb + lrow, em = m0 + r;  // this lane's row
    link_steps<NS + 1>([&](auto sc) {
      constexpr int s = decltype(sc)::value;
      if constexpr (s < NS) {
        // acc[4 g + e] = chunk s, row r, column ec + 8 g + 4 lh + e
        f32x16_t acc;
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
#pragma unroll
        for (int kt = 0; kt < KTI; ++kt)
#pragma unroll
          for (int ks = 0; ks < 4; ++ks) {
            const bf16x8_t af = link_frag(b3s[kt], r, ks, lh);
            const bf16x8_t bf = link_frag(w3s[s % D][kt], ec + lrow, ks, lh);
            acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bf, af, acc, 0, 0, 0);
          }
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          // lower half-wave keeps group 2 p and receives the upper half's; the
          // upper half receives the lower half's group 2 p + 1
          float v[8];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[8 * p + e]),
                                                             __float_as_uint(acc[8 * p + 4 + e]), false, false);
            v[e] = __uint_as_float(sw[0]);
            v[4 + e] = __uint_as_float(sw[1]);
          }
          const int c = ec + 16 * p + 8 * lh;               // column within the chunk
          const int pc = ((c >> 3) ^ ((r >> 1) & 7)) << 3;  // its swizzled place in a tile row
          const float4 b0 = *reinterpret_cast<const float4 *>(b3f + 64 * s + c);
          const float4 b1 = *reinterpret_cast<const float4 *>(b3f + 64 * s + c + 4);
          v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
          v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
          const uint4 rv = *reinterpret_cast<const uint4 *>(rs[s % D] + r * 64 + pc);
          const uint32_t w4[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            v[2 * e] += __uint_as_float(w4[e] << 16);
            v[2 * e + 1] += __uint_as_float(w4[e] & 0xffff0000u);
          }
          uint32_t o[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) o[e] = f2bf2(fmaxf(v[2 * e], 0.0f), fmaxf(v[2 * e + 1], 0.0f));
          const uint4 ov = make_uint4(o[0], o[1], o[2], o[3]);
          if (em < a.M) *reinterpret_cast<uint4 *>(a.y + (int64_t)em * E + 64 * s + c) = ov;
          *reinterpret_cast<uint4 *>(xs[s & 1] + r * 64 + pc) = ov;  // the reduction's k-tile
        }
      }
      link_barrier();  // publishes this step's LDS writes
    });
    return;
  }

  // ---- Reduction waves: output columns rc .. rc + CO / 4 - 1 of the 64 rows.
  const int rc = (CO / 4) * (wave - 4);
  f32x16_t racc[2][TNR];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < TNR; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) racc[i][j][e] = 0.0f;
  link_steps<NS + 1>([&](auto sc) {
    constexpr int s = decltype(sc)::value;
    if constexpr (s >= 1) {
      // k-tile s - 1 of the reduction: chunk s - 1 of the expansion output
      const uint16_t *xa = xs[(s - 1) & 1], *wb = w1s[(s - 1) % D];
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        bf16x8_t af[2], bfr[TNR];
#pragma unroll
        for (int i = 0; i < 2; ++i) af[i] = link_frag(xa, 32 * i + lrow, ks, lh);
#pragma unroll
        for (int j = 0; j < TNR; ++j) bfr[j] = link_frag(wb, rc + 32 * j + lrow, ks, lh);
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < TNR; ++j)
            racc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], racc[i][j], 0, 0, 0);
      }
    }
    link_barrier();  // this step's LDS reads are done: their buffers are free
  });
  // Epilogue: bias, ReLU, one rounding, 16-byte stores.
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int m = m0 + 32 * i + lrow;
#pragma unroll
    for (int j = 0; j < TNR; ++j)
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        float v[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(racc[i][j][8 * p + e]),
                                                           __float_as_uint(racc[i][j][8 * p + 4 + e]), false, false);
          v[e] = __uint_as_float(sw[0]);
          v[4 + e] = __uint_as_float(sw[1]);
        }
        const int n = rc + 32 * j + 16 * p + 8 * lh;
        const float4 b0 = *reinterpret_cast<const float4 *>(b1f + n);
        const float4 b1 = *reinterpret_cast<const float4 *>(b1f + n + 4);
        v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
        v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
        uint32_t o[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = f2bf2(fmaxf(v[2 * e], 0.0f), fmaxf(v[2 * e + 1], 0.0f));
        if (m < a.M) *reinterpret_cast<uint4 *>(a.a1 + (int64_t)m * CO + n) = make_uint4(o[0], o[1], o[2], o[3]);
      }
  }
}

}  // namespace

bool bottleneck_link_supported(int ci, int e, int co, int kp3, int kp1) {
  return ci == 128 && e == 512 && (co == 128 || co == 256) && kp3 == ci && kp1 == e;
}

hipError_t launch_bottleneck_link(const void *b3, const void *w3, const float *bias3, const void *res, void *y,
                                  const void *w1, const float *bias1, void *a1, int M, int ci, int e, int co,
                                  hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (!bottleneck_link_supported(ci, e, co, ci, e) || (int64_t)M * e * 2 >= ((int64_t)1 << 31))
    return hipErrorInvalidValue;
  LinkArgs a{};
  a.b3 = static_cast<const uint16_t *>(b3);
  a.w3 = static_cast<const uint16_t *>(w3);
  a.bias3 = bias3;
  a.res = static_cast<const uint16_t *>(res);
  a.y = static_cast<uint16_t *>(y);
  a.w1 = static_cast<const uint16_t *>(w1);
  a.bias1 = bias1;
  a.a1 = static_cast<uint16_t *>(a1);
  a.M = M;
  const dim3 grid((M + kLinkBM - 1) / kLinkBM);
  if (co == 128)
    hapi_launch(bottleneck_link_kernel<128, 512, 128, 2>, grid, dim3(kLinkThreads), 0, s, a);
  else
    hapi_launch(bottleneck_link_kernel<128, 512, 256, 1>, grid, dim3(kLinkThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace hapi
