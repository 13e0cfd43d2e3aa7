// Two consecutive ResNet bottleneck blocks joined at their boundary on gfx950:
// block i's expanding 1x1 convolution (bias, identity residual, ReLU) and
// block i + 1's reducing 1x1 convolution (bias, ReLU) in one kernel, so the
// block output, which the reduction reads, never makes the round trip
// through HBM a second time.
//
// A workgroup owns 128 rows (output pixels); each of its four compute waves
// owns 32 of them and keeps their 3x3 output (the expansion's A operand) in
// registers.  The expansion's E output channels are produced one 64-wide
// chunk per step.  After the epilogue's half-wave exchange a lane holds 8
// consecutive channels of its row, rounded to bf16: exactly the A fragment
// of the reduction for those 8 k values.  So the wave stores the chunk (it
// is block i's output and block i + 1's residual) and accumulates it into
// the reduction straight from registers.  The arithmetic is that of the two
// separate convolutions exactly: the same v_mfma_f32_32x32x16_bf16, k-steps
// in the same order, epilogues adding bias, then the residual, then applying
// ReLU with one bf16 rounding, so the outputs equal the unfused layers bit
// for bit.
//
// Three more waves only move operands into LDS with buffer_load ... lds, one
// stream each: residual chunks, expansion weight chunks and reduction weight
// k-tiles, each some steps ahead in a ring of buffers.  A DMA wave never
// stores and the compute waves never load from global memory inside the step
// loop, so every wait on a wave's vector-memory counter (which loads and
// stores share, completing in issue order) covers exactly the transfers it
// needs.  One barrier ends each step.
#include "internal.h"

namespace hapi {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

#define LINK_LDS(p) ((__attribute__((address_space(3))) void *)(p))

constexpr unsigned kLinkOob = 0x80000000u;  // a byte offset outside every buffer range
constexpr int kLinkBM = 128;                 // rows per workgroup
constexpr int kLinkComputeWaves = kLinkBM / 32;
constexpr int kLinkThreads = 64 * (kLinkComputeWaves + 3);

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

// Workgroup barrier after this wave's LDS operations completed (no wait on
// its global memory operations, unlike __syncthreads).
__device__ __forceinline__ void link_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);
  __builtin_amdgcn_s_barrier();
}

template <int N>
__device__ __forceinline__ void link_vmwait() {
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <int... I, class F>
__device__ __forceinline__ void link_steps_impl(F &&f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void link_steps(F &&f) {
  link_steps_impl(f, std::make_integer_sequence<int, N>{});
}

// DMA instructions in flight when items lo .. hi (of n, `per` instructions
// each) have been issued and not yet waited for.
template <int N, int PER>
constexpr int link_fly(int lo, int hi) {
  if (hi > N - 1) hi = N - 1;
  return hi >= lo ? (hi - lo + 1) * PER : 0;
}

// One DMA stream over the N steps: item q (PER instructions, issued by
// issue(q)) is needed in step q; it is issued during step q - P (P steps
// ahead, the first P before step 0) and waited for at the end of step q - 1.
template <int N, int P, int PER, class F>
__device__ __forceinline__ void link_stream(F &&issue) {
  link_steps<P>([&](auto qc) {
    if constexpr (decltype(qc)::value < N) issue(decltype(qc)::value);
  });
  link_vmwait<link_fly<N, PER>(1, P - 1)>();
  link_barrier();
  link_steps<N>([&](auto sc) {
    constexpr int s = decltype(sc)::value;
    if constexpr (s + P < N) issue(s + P);
    if constexpr (s + 1 < N) link_vmwait<link_fly<N, PER>(s + 2, s + P)>();
    __builtin_amdgcn_s_barrier();
  });
}

struct LinkArgs {
  const uint16_t *b3;  // [M][CI] block i's 3x3 output, the expansion's input
  const uint16_t *w3;  // [E][CI] packed expansion weights
  const float *bias3;  // [E]
  const uint16_t *res; // [M][E] the residual (block i's input)
  uint16_t *y;         // [M][E] block i's output; may be res itself (each element is read
                       // by the lane that later writes it)
  const uint16_t *w1;  // [CO][E] packed reduction weights of block i + 1
  const float *bias1;  // [CO]
  uint16_t *a1;        // [M][CO] block i + 1's reduction output
  int M;
};

// Prefetch distances in steps: PW for expansion weight chunks, PR for
// residual chunks, PK for reduction weight k-tiles (rings of P + 1 buffers).
// Each role runs its own loop over the steps, so that the waits the compiler
// places for one role's memory operations never land in another's.
template <int CI, int E, int CO, int PW, int PR, int PK>
__global__ __launch_bounds__(kLinkThreads, 1) void bottleneck_link_kernel(LinkArgs a) {
  static_assert(CI % 64 == 0 && E % 64 == 0 && CO % 32 == 0 && PW >= 1 && PR >= 1 && PK >= 1, "shape");
  constexpr int KTI = CI / 64;  // expansion k-tiles
  constexpr int NS = E / 64;    // steps: expansion chunks = reduction k-tiles
  constexpr int TN = CO / 32;   // reduction 32-column blocks
  __shared__ __attribute__((aligned(16))) uint16_t w3s[PW + 1][KTI][64 * 64];
  __shared__ __attribute__((aligned(16))) uint16_t w1s[PK + 1][CO * 64];
  __shared__ __attribute__((aligned(16))) uint16_t rs[PR + 1][kLinkBM * 64];
  __shared__ __attribute__((aligned(16))) float b3f[E];
  __shared__ __attribute__((aligned(16))) float b1f[CO];

  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int lrow = lane & 31, lh = lane >> 5;
  const int m0 = blockIdx.x * kLinkBM;

  for (int i = t; i < E; i += kLinkThreads) b3f[i] = a.bias3 ? a.bias3[i] : 0.0f;
  for (int i = t; i < CO; i += kLinkThreads) b1f[i] = a.bias1 ? a.bias1[i] : 0.0f;

  if (wave >= kLinkComputeWaves) {
    // ---- DMA waves.  Step q needs residual chunk q, expansion weight chunk q
    // (output channels 64 q ..) and reduction weight k-tile q.
    const int dw = wave - kLinkComputeWaves;
    if (dw == 0) {
      link_stream<NS, PR, kLinkBM / 8>([&](int c) {
#pragma unroll
        for (int g = 0; g < kLinkBM / 8; ++g) link_dma_rows(a.res, a.M, E, m0, 64 * c, rs[c % (PR + 1)], g, lane);
      });
    } else if (dw == 1) {
      link_stream<NS, PW, KTI * 8>([&](int c) {
#pragma unroll
        for (int q = 0; q < KTI * 8; ++q)
          link_dma_rows(a.w3, E, CI, 64 * c, 64 * (q >> 3), w3s[c % (PW + 1)][q >> 3], q & 7, lane);
      });
    } else {
      link_stream<NS, PK, CO / 8>([&](int k) {
#pragma unroll
        for (int g = 0; g < CO / 8; ++g) link_dma_rows(a.w1, CO, E, 0, 64 * k, w1s[k % (PK + 1)], g, lane);
      });
    }
    return;
  }

  // ---- Compute wave: rows r = 32 wave + lane % 32 of the workgroup's tile.
  const int r = 32 * wave + lrow, m = m0 + r;
  // The expansion's A fragments (k = 16 i + 8 lh ..), for the whole tile.
  bf16x8_t a3[KTI * 4];
#pragma unroll
  for (int i = 0; i < KTI * 4; ++i)
    a3[i] = m < a.M ? *reinterpret_cast<const bf16x8_t *>(a.b3 + (int64_t)m * CI + 16 * i + 8 * lh)
                    : bf16x8_t{};
  f32x16_t racc[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int e = 0; e < 16; ++e) racc[j][e] = 0.0f;
  link_barrier();

  link_steps<NS>([&](auto sc) {
    constexpr int s = decltype(sc)::value;
    // eacc[j][4 g + e] = chunk s, row r, channel 32 j + 8 g + 4 lh + e
    f32x16_t eacc[2];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) eacc[j][e] = 0.0f;
#pragma unroll
    for (int kt = 0; kt < KTI; ++kt)
#pragma unroll
      for (int ks = 0; ks < 4; ++ks)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          eacc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(link_frag(w3s[s % (PW + 1)][kt], 32 * j + lrow, ks, lh),
                                                            a3[4 * kt + ks], eacc[j], 0, 0, 0);
    // Epilogue: part (j, p) gives this lane channels c = 32 j + 16 p + 8 lh ..
    // c + 7 of row r, which is the reduction's A fragment of k-step 2 j + p.
    bf16x8_t xa[4];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        // lower half-wave keeps group 2 p and receives the upper half's; the
        // upper half receives the lower half's group 2 p + 1
        float v[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(eacc[j][8 * p + e]),
                                                           __float_as_uint(eacc[j][8 * p + 4 + e]), false, false);
          v[e] = __uint_as_float(sw[0]);
          v[4 + e] = __uint_as_float(sw[1]);
        }
        const int c = 32 * j + 16 * p + 8 * lh;
        const float4 b0 = *reinterpret_cast<const float4 *>(b3f + 64 * s + c);
        const float4 b1 = *reinterpret_cast<const float4 *>(b3f + 64 * s + c + 4);
        v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
        v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
        const uint4 rv =
            *reinterpret_cast<const uint4 *>(rs[s % (PR + 1)] + r * 64 + (((c >> 3) ^ ((r >> 1) & 7)) << 3));
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
        if (m < a.M) *reinterpret_cast<uint4 *>(a.y + (int64_t)m * E + 64 * s + c) = ov;
        xa[2 * j + p] = __builtin_bit_cast(bf16x8_t, ov);
      }
    // k-tile s of the reduction, k-steps in order
#pragma unroll
    for (int ks = 0; ks < 4; ++ks)
#pragma unroll
      for (int j = 0; j < TN; ++j)
        racc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(link_frag(w1s[s % (PK + 1)], 32 * j + lrow, ks, lh),
                                                          xa[ks], racc[j], 0, 0, 0);
    link_barrier();  // this step's LDS reads are done: their buffers are free
  });

  // Reduction epilogue: bias, ReLU, one rounding, 16-byte stores.
#pragma unroll
  for (int j = 0; j < TN; ++j)
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(racc[j][8 * p + e]),
                                                         __float_as_uint(racc[j][8 * p + 4 + e]), false, false);
        v[e] = __uint_as_float(sw[0]);
        v[4 + e] = __uint_as_float(sw[1]);
      }
      const int n = 32 * j + 16 * p + 8 * lh;
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
  // Prefetch distances within 150 KB of LDS; the residual, from HBM, travels
  // furthest ahead (128 -> 512 -> 128 with two partitions in flight: 124 us per
  // pair of launches, against 132-134 us with other distances).
  if (co == 128)
    hapi_launch(bottleneck_link_kernel<128, 512, 128, 1, 3, 2>, grid, dim3(kLinkThreads), 0, s, a);
  else
    hapi_launch(bottleneck_link_kernel<128, 512, 256, 1, 2, 1>, grid, dim3(kLinkThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace hapi
