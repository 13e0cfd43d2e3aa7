// Implicit-GEMM convolution / linear kernels for gfx950 (CDNA4).
//
// A convolution y = act(W * x + b [+ r]) is the GEMM C[M, N] = A[M, K] * B[K, N]
// with M = images x output pixels (NHWC order), N = output channels and
// K = kernel taps x input channels.  A is never materialised: each k-tile of
// the im2col matrix is gathered from the activation straight into LDS.  The
// packed weights are B^T ([N][Kp], K contiguous, zero padded to the k-tile).
//
// bf16 path: v_mfma_f32_32x32x16_bf16 with fp32 accumulation, k-tile 64,
// 256 threads = 4 waves in a 2 x 2 grid, double-buffered LDS with one barrier
// per k-tile, global loads of the next tile in flight during the MFMAs.
// fp32 path: v_mfma_f32_32x32x2f32, k-tile 16, same structure.
//
// Every output element's reduction visits the k-tiles in order and, inside a
// tile, the MFMA k-steps in order, independent of the tile shape (BM, BN) and
// of M.  Results are therefore bit-identical for any batch split.
#include <cstdio>
#include <cstdlib>
#include <type_traits>
#include <utility>

#include "internal.h"

namespace hapi {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;

__device__ __forceinline__ int xcd_remap(int bid, int nb) {
  // Workgroups are dispatched round-robin over the 8 XCDs (block b -> XCD b % 8).
  // Renumber so that consecutive logical tiles run on one XCD and share its L2.
  const int xcd = bid & 7, idx = bid >> 3;
  const int q = nb >> 3, r = nb & 7;
  return (xcd < r) ? xcd * (q + 1) + idx : r * (q + 1) + (xcd - r) * q + idx;
}

__device__ __forceinline__ float bf2f(uint16_t u) { return __uint_as_float((uint32_t)u << 16); }


// erf by Abramowitz & Stegun, Handbook of Mathematical Functions, 7.1.26:
// erf(x) = 1 - t (a1 + t (a2 + t (a3 + t (a4 + t a5)))) exp(-x^2), t = 1 / (1 + p x)
// for x >= 0 (odd extension), absolute error <= 1.5e-7: branch-free, one
// reciprocal and one exponential, against a piecewise library erf.
__device__ __forceinline__ float erf_as(float x) {
  const float ax = fabsf(x);
  const float t = __builtin_amdgcn_rcpf(fmaf(0.3275911f, ax, 1.0f));
  float q = fmaf(t, 1.061405429f, -1.453152027f);
  q = fmaf(t, q, 1.421413741f);
  q = fmaf(t, q, -0.284496736f);
  q = fmaf(t, q, 0.254829592f);
  const float y = fmaf(-t * q, __builtin_amdgcn_exp2f(-ax * ax * 1.4426950408889634f), 1.0f);
  return copysignf(y, x);
}

// GELU is the exact (erf) form: v * Phi(v) = 0.5 v (1 + erf(v / sqrt 2)).
__device__ __forceinline__ float epilogue_act(float v, int relu, int gelu) {
  if (relu) v = fmaxf(v, 0.0f);
  if (gelu) v = 0.5f * v * (1.0f + erf_as(v * 0.70710678118654752f));
  return v;
}

// ------------------------------------------------------------------ bf16

constexpr int BK = 64;         // k-tile (bf16 elements)
constexpr int LDSW = BK + 8;   // LDS row pitch in elements: 144 B spreads rows over banks

// Per-row state of the rows a thread gathers for the A tile.
struct RowState {
  int base;  // element offset of the row's image (NHWC / NCHW) or of the row (GEMM)
  int hi0;   // ho * stride - pad  (large negative: row beyond M)
  int wi0;   // wo * stride - pad
};

template <int LD>
__device__ __forceinline__ RowState make_row(const ConvArgs &a, int m) {
  RowState r;
  if (m >= a.M) {
    r.base = 0; r.hi0 = -(1 << 28); r.wi0 = 0;
    return r;
  }
  if (LD == LD_GEMM) {
    r.base = m * (a.lda ? a.lda : a.K); r.hi0 = 0; r.wi0 = 0;
    return r;
  }
  const int hw = a.Ho * a.Wo;
  const int n = m / hw, rem = m - n * hw;
  const int ho = rem / a.Wo, wo = rem - ho * a.Wo;
  r.base = n * a.H * a.W * a.C;
  r.hi0 = ho * a.stride - a.pad;
  r.wi0 = wo * a.stride - a.pad;
  return r;
}

// Gather the 8 consecutive k values [k0, k0 + 8) of one im2col row.
template <int LD>
__device__ __forceinline__ uint4 load_a_chunk(const ConvArgs &a, const RowState &r, int k0,
                                              int kh_, int kw_, int c0) {
  const uint16_t *x = static_cast<const uint16_t *>(a.x);
  uint4 v = make_uint4(0, 0, 0, 0);
  if (LD == LD_GEMM) {  // K % 8 == 0; chunks past K read nothing
    if (r.hi0 >= 0 && k0 < a.K) v = *reinterpret_cast<const uint4 *>(x + r.base + k0);
  } else if (LD == LD_NHWC) {
    const int hi = r.hi0 + kh_, wi = r.wi0 + kw_;
    if ((unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W)
      v = *reinterpret_cast<const uint4 *>(x + r.base + (hi * a.W + wi) * a.C + c0);
  } else if (LD == LD_NCHW_PATCH) {
    // k = (c, u, v) with 8 | kw: the 8 taps are contiguous pixels of one image row.
    if (r.hi0 > -(1 << 27) && k0 < a.K) {
      const int khw = a.kh * a.kw;
      const int c = k0 / khw, rem = k0 - c * khw;
      const int u = rem / a.kw, vv = rem - u * a.kw;
      const int hi = r.hi0 + u, wi = r.wi0 + vv;
      v = *reinterpret_cast<const uint4 *>(x + r.base + (c * a.H + hi) * a.W + wi);
    }
  } else {  // LD_NCHW: element gather, k = (c, u, v)
    if (r.hi0 > -(1 << 27)) {
      uint16_t e[8];
      const int khw = a.kh * a.kw;
      int c = k0 / khw, rem = k0 - c * khw;
      int u = rem / a.kw, vv = rem - u * a.kw;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int hi = r.hi0 + u, wi = r.wi0 + vv;
        e[j] = (k0 + j < a.K && (unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W)
                   ? x[r.base + (c * a.H + hi) * a.W + wi]
                   : (uint16_t)0;
        if (++vv == a.kw) { vv = 0; if (++u == a.kh) { u = 0; ++c; } }
      }
      v.x = e[0] | ((uint32_t)e[1] << 16);
      v.y = e[2] | ((uint32_t)e[3] << 16);
      v.z = e[4] | ((uint32_t)e[5] << 16);
      v.w = e[6] | ((uint32_t)e[7] << 16);
    }
  }
  return v;
}

template <int BM, int BN, int LD>
__global__ __launch_bounds__(kThreads) void conv_bf16_kernel(ConvArgs a) {
  constexpr int WM = 2, WN = 2;
  constexpr int TM = BM / (WM * 32), TN = BN / (WN * 32);
  constexpr int A_PER = BM * (BK / 8) / kThreads;  // 16-byte chunks per thread
  constexpr int B_PER = BN * (BK / 8) / kThreads;
  static_assert(TM >= 1 && TN >= 1 && A_PER >= 1 && B_PER >= 1, "tile");

  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (BM + BN) * LDSW];

  const int tiles_n = (a.N + BN - 1) / BN;
  const int tile = a.rev ? (int)gridDim.x - 1 - xcd_remap(blockIdx.x, gridDim.x) : xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * BN;

  const int t = threadIdx.x;
  const int kc = t & 7;    // which 16-byte chunk of the 64-wide k-tile this thread moves
  const int r0 = t >> 3;   // first row it moves; then every 32nd

  RowState rs[A_PER];
#pragma unroll
  for (int i = 0; i < A_PER; ++i) rs[i] = make_row<LD>(a, m0 + r0 + 32 * i);

  const uint16_t *wp = static_cast<const uint16_t *>(a.w);
  uint4 ra[A_PER], rb[B_PER];

  auto load_tile = [&](int kt) {
    const int kbase = kt * BK;
    int kh_ = 0, kw_ = 0, c0 = 0;
    if (LD == LD_NHWC) {  // C % 64 == 0: the whole k-tile lies in one (kh, kw) tap
      const int tap = kbase / a.C;
      c0 = kbase - tap * a.C + kc * 8;
      kh_ = tap / a.kw;
      kw_ = tap - kh_ * a.kw;
    }
#pragma unroll
    for (int i = 0; i < A_PER; ++i) ra[i] = load_a_chunk<LD>(a, rs[i], kbase + kc * 8, kh_, kw_, c0);
#pragma unroll
    for (int j = 0; j < B_PER; ++j) {
      const int n = n0 + r0 + 32 * j;
      rb[j] = (n < a.N) ? *reinterpret_cast<const uint4 *>(wp + (size_t)n * a.Kp + kbase + kc * 8)
                        : make_uint4(0, 0, 0, 0);
    }
  };
  auto store_tile = [&](int buf) {
    uint16_t *As = smem + buf * (BM + BN) * LDSW;
    uint16_t *Bs = As + BM * LDSW;
#pragma unroll
    for (int i = 0; i < A_PER; ++i)
      *reinterpret_cast<uint4 *>(As + (r0 + 32 * i) * LDSW + kc * 8) = ra[i];
#pragma unroll
    for (int j = 0; j < B_PER; ++j)
      *reinterpret_cast<uint4 *>(Bs + (r0 + 32 * j) * LDSW + kc * 8) = rb[j];
  };

  const int lane = t & 63, wave = t >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int lrow = lane & 31, lk = (lane >> 5) * 8;

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = a.Kp / BK;
  load_tile(0);
  store_tile(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load_tile(kt + 1);
    const uint16_t *As = smem + cur * (BM + BN) * LDSW + (wm * TM * 32 + lrow) * LDSW + lk;
    const uint16_t *Bs = smem + cur * (BM + BN) * LDSW + BM * LDSW + (wn * TN * 32 + lrow) * LDSW + lk;
#pragma unroll
    for (int ks = 0; ks < BK / 16; ++ks) {
      bf16x8_t af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *reinterpret_cast<const bf16x8_t *>(As + i * 32 * LDSW + ks * 16);
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8_t *>(Bs + j * 32 * LDSW + ks * 16);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) store_tile(cur ^ 1);
    __syncthreads();
  }

  // Epilogue: lane holds column n = lane % 32 and rows 8*(r/4) + 4*(lane/32) + r%4.
  uint16_t *y = static_cast<uint16_t *>(a.y);
  const uint16_t *res = static_cast<const uint16_t *>(a.res);
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int n = n0 + wn * TN * 32 + j * 32 + lrow;
    if (n >= a.N) continue;
    const float bv = a.bias ? a.bias[n] : 0.0f;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * TM * 32 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (m >= a.M) continue;
        float v = acc[i][j][r] + bv;
        if (res) v += bf2f(res[(int64_t)m * a.ldr + n]);
        y[(int64_t)m * a.ldc + n] = f2bf(epilogue_act(v, a.relu, a.gelu));
      }
    }
  }
}

// ----------------------------------------------- bf16, LDS-DMA pipeline
//
// For inputs whose 8-element k-chunks are contiguous 16-byte runs (NHWC with
// C % 64 == 0, row-major matrices, NCHW patches) the tiles are moved by
// buffer_load ... lds (16 bytes per lane): each lane's 16 bytes land directly
// in LDS, so no registers or ds_write instructions are spent on staging and
// STAGES - 1 k-tiles are in flight while the MFMAs consume the oldest one.
// Padding taps and rows beyond M / N use a byte offset outside the buffer's
// range, which reads zeros.
//
// LDS rows hold 64 bf16 (128 B) without padding; the 16-byte chunk kc of row
// r is stored at position kc ^ ((r >> 1) & 7).  The LDS serves 256 bytes (64
// banks) per clock, i.e. two 128-byte rows: with this swizzle the 16 rows a
// quarter-wave fragment read touches land in 16 distinct 16-byte slots of
// that 256-byte window, so fragment reads are free of bank conflicts.

#define LDS_PTR(p) ((__attribute__((address_space(3))) void *)(p))

// Wait until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

constexpr unsigned kOob = 0x80000000u;  // a byte offset outside every buffer range

// Moves 16 bytes per lane from base + soff + voff (a raw buffer of 2^31 - 1
// bytes: offsets at or beyond kOob read zeros) into LDS at lds + 16 * lane.
// Only scalar instructions besides the load itself.
__device__ __forceinline__ void dma16(const void *base, uint16_t *lds, unsigned voff, unsigned soff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), 0, 0x7fffffff, 0x00020000), LDS_PTR(lds), 16,
      voff, soff, 0, 0);
}

// Addressing of the LDS DMA that moves one k-tile (64 k values) of the
// implicit-GEMM operands: A rows (output pixels, gathered through the loader
// LD) and B rows (packed weights [N][Kp]).  One DMA instruction moves 8 rows of
// 8 16-byte chunks; this thread's instructions are A row-groups ga0 .. ga0+NA-1
// and B row-groups gb0 .. gb0+NB-1.  Rows beyond M / N and padding taps get
// an out-of-range offset (zeros), so the address arithmetic stays
// branch-free.
//
// Lane l of row-group g fills row 8 g + l / 8, physical chunk l % 8, i.e.
// logical chunk (l % 8) ^ ((row >> 1) & 7) = (l % 8) ^ ((4 g + l / 16) & 7).
template <int NA, int NB, int LD>
struct DmaPlan {
  int roff[NA], rhi[NA], rwi[NA], rkc[NA], roff2[LD == LD_CAT ? NA : 1];
  int boffs[NB];
  bool bok[NB];
  int ga0, gb0;

  __device__ __forceinline__ void init(const ConvArgs &a, int m0, int n0, int ga, int gb, int lane) {
    ga0 = ga;
    gb0 = gb;
    const int kcA = ((lane & 7) ^ ((lane >> 4) & 7)) * 8;        // even g
    const int kcB = ((lane & 7) ^ ((4 + (lane >> 4)) & 7)) * 8;  // odd g
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      // Per-row gather state: element offset of the row's first tap (may
      // point into padding) and the tap origin for bounds checks.
      const int m = m0 + (ga + i) * 8 + (lane >> 3);
      const RowState r = make_row<LD == LD_CAT ? LD_NHWC : LD>(a, m);
      const int kc8 = ((ga + i) & 1) ? kcB : kcA;
      rkc[i] = kc8;
      rhi[i] = r.hi0;
      rwi[i] = r.wi0;
      if (LD == LD_NHWC || LD == LD_S2D || LD == LD_CAT)
        roff[i] = r.base + (r.hi0 * a.W + r.wi0) * a.C + kc8;
      else if (LD == LD_GEMM) roff[i] = r.base + kc8;
      else roff[i] = r.base;
      if (LD == LD_CAT) {
        // shortcut pixel (n, ho * s2, wo * s2) of x2, relative to roff
        const int hw = a.Ho * a.Wo;
        const int mm = m < a.M ? m : 0;
        const int n = mm / hw, rem = mm - n * hw;
        const int ho = rem / a.Wo, wo = rem - ho * a.Wo;
        roff2[i] = ((n * a.H2 + ho * a.s2) * a.W2 + wo * a.s2) * a.C2 + kc8 - a.K1 - roff[i];
      }
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int n = n0 + (gb + j) * 8 + (lane >> 3);
      bok[j] = n < a.N;
      boffs[j] = (bok[j] ? n : 0) * a.Kp + (((gb + j) & 1) ? kcB : kcA);
    }
  }

  // Moves instructions q0 <= q < q1 (A first, then B) of k-tile kt into the
  // stage whose A and B parts start at As and Bs.
  __device__ __forceinline__ void issue(const ConvArgs &a, int kt, uint16_t *As, uint16_t *Bs, int q0,
                                        int q1) const {
    const uint16_t *x = static_cast<const uint16_t *>(a.x);
    const uint16_t *wp = static_cast<const uint16_t *>(a.w);
    const int kbase = kt * BK;
    int kh_ = 0, kw_ = 0, tapoff = 0;
    if (LD == LD_NHWC || LD == LD_CAT) {  // C % 64 == 0: the k-tile lies in one tap
      const int tap = kbase / a.C;
      kh_ = tap / a.kw;
      kw_ = tap - kh_ * a.kw;
      tapoff = (kh_ * a.W + kw_) * a.C + (kbase - tap * a.C);
    }
    // LD_CAT: k-tiles past K1 read the shortcut pixel of x2.  The first part
    // is a stride-1 convolution at output resolution, so taps (pad, pad) are
    // in bounds exactly for the real rows.  Both parts share one formula with
    // uniform selectors, so the per-row arrays stay in registers.
    const bool second = LD == LD_CAT && kbase >= a.K1;
    const uint16_t *xs = second ? static_cast<const uint16_t *>(a.x2) : x;
    const int cat_sel = second ? 1 : 0;
    if (second) {
      kh_ = kw_ = a.pad;
      tapoff = kbase;
    }
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      if (i < q0 || i >= q1) continue;
      bool ok;
      int off;
      if (LD == LD_GEMM) {  // K % 8 == 0; chunks past K (ragged last k-tile) read zeros
        ok = rhi[i] >= 0 && kbase + rkc[i] < a.K;
        off = roff[i] + kbase;
      } else if (LD == LD_NHWC || LD == LD_CAT) {
        ok = (unsigned)(rhi[i] + kh_) < (unsigned)a.H && (unsigned)(rwi[i] + kw_) < (unsigned)a.W;
        off = roff[i] + tapoff + (LD == LD_CAT ? cat_sel * roff2[i] : 0);
      } else if (LD == LD_S2D) {
        // k-tile kt is the contiguous run of cell row du = kt (kw x 16 = 64 elements)
        ok = rhi[i] >= 0;
        off = roff[i] + kt * a.W * a.C;
      } else {  // LD_NCHW_PATCH: k = (c, u, v), 8 | kw
        const int k0 = kbase + rkc[i];
        const int khw = a.kh * a.kw;
        const int c = k0 / khw, rem = k0 - c * khw;
        const int u = rem / a.kw, vv = rem - u * a.kw;
        ok = rhi[i] > -(1 << 27) && k0 < a.K;
        off = roff[i] + (c * a.H + rhi[i] + u) * a.W + rwi[i] + vv;
      }
      // 32-bit byte offsets (the launcher checks every operand fits in
      // 2^31 bytes); a chunk outside the image or past K reads zeros
      dma16(xs, As + (ga0 + i) * 512, ok ? (unsigned)off * 2u : kOob, 0);
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      if (NA + j < q0 || NA + j >= q1) continue;
      dma16(wp, Bs + (gb0 + j) * 512, bok[j] ? (unsigned)(boffs[j] + kbase) * 2u : kOob, 0);
    }
  }
};

template <typename F, int... I>
__device__ __forceinline__ void static_for_impl(F &&f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
// Calls f(integral_constant<int, i>) for i = 0 .. N-1 (compile-time indices).
template <int N, typename F>
__device__ __forceinline__ void static_for(F &&f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// Scheduling recipe of one MFMA k-step: NMF MFMAs with NRD fragment reads
// and NDMA DMA issues (each with its address arithmetic) spread evenly
// between them.
template <int Q, int NMF, int NRD, int NDMA>
__device__ __forceinline__ void sched_step() {
  if constexpr (Q < NMF) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
    constexpr int r0 = Q * NRD / NMF, r1 = (Q + 1) * NRD / NMF;
    if constexpr (r1 > r0) __builtin_amdgcn_sched_group_barrier(0x100, r1 - r0, 0);  // DS read
    constexpr int d0 = Q * NDMA / NMF, d1 = (Q + 1) * NDMA / NMF;
    if constexpr (d1 > d0) {
      __builtin_amdgcn_sched_group_barrier(0x002, 6 * (d1 - d0), 0);  // VALU
      __builtin_amdgcn_sched_group_barrier(0x020, d1 - d0, 0);        // VMEM (DMA)
    }
    sched_step<Q + 1, NMF, NRD, NDMA>();
  }
}

template <int BM, int BN, int STAGES, int EPI>
struct PipeSmem {
  static constexpr int kStage = (BM + BN) * BK;  // elements per stage
  static constexpr int kCPitch = BN + 8;         // fp32 pitch of the staged C tile
  static constexpr int kStages = STAGES * kStage * 2;
  static constexpr int kBytes =
      (EPI || kStages > BM * kCPitch * 4) ? kStages : BM * kCPitch * 4;
};

// EPI = 0: C tile staged through LDS, 16-byte stores.  EPI = 1: MFMA operands
// swapped (weights as A, activations as B) so each lane's accumulators hold 4
// consecutive output channels of one output pixel; the epilogue stores them
// directly as 8-byte writes and the kernel needs no LDS beyond the stages.
// EPI = 2 (warp-specialised kernel): operands swapped as for 1, a half-wave
// exchange gives each lane 8 consecutive channels of its pixel, stored as one
// 16-byte write; bias and residual are fetched before the k-loop.
// ReLU(x * scale + shift) on 8 consecutive channels, rounded to bf16 once.
__device__ __forceinline__ bf16x8_t preact8(bf16x8_t v, float4 s0, float4 s1, float4 h0, float4 h1) {
  typedef float f32x8_t __attribute__((ext_vector_type(8)));
  f32x8_t f = __builtin_convertvector(v, f32x8_t);
  const float sc[8] = {s0.x, s0.y, s0.z, s0.w, s1.x, s1.y, s1.z, s1.w};
  const float sh[8] = {h0.x, h0.y, h0.z, h0.w, h1.x, h1.y, h1.z, h1.w};
#pragma unroll
  for (int e = 0; e < 8; ++e) f[e] = fmaxf(__builtin_fmaf(f[e], sc[e], sh[e]), 0.0f);
  return __builtin_convertvector(f, bf16x8_t);
}

// PRE: the A operand is pre-activated (ConvArgs::pre_scale) between LDS and
// the MFMAs; the per-channel scale and shift are staged in LDS once.
template <int BM, int BN, int WM, int WN, int STAGES, int LD, int SCHED, int EPI, bool PRE = false>
__global__ __launch_bounds__(WM * WN * 64) void conv_bf16_pipe_kernel(ConvArgs a) {
  constexpr int NT = WM * WN * 64;                    // threads: WM x WN waves
  constexpr int TM = BM / (WM * 32), TN = BN / (WN * 32);
  constexpr int NA = BM * 8 / NT, NB = BN * 8 / NT;   // DMA instructions per thread per stage
  constexpr int KS = BK / 16;                         // MFMA k-steps per k-tile
  using SM = PipeSmem<BM, BN, STAGES, EPI>;
  static_assert(TM >= 1 && TN >= 1 && NA >= 1 && NB >= 1, "tile");
  static_assert(STAGES >= 2 && STAGES <= 4, "stages");
  static_assert((STAGES - 2) * (NA + NB) < 64, "vmcnt range");
  __shared__ __attribute__((aligned(16))) uint8_t smem_raw[SM::kBytes];
  uint16_t *smem = reinterpret_cast<uint16_t *>(smem_raw);
  __shared__ __attribute__((aligned(16))) float pre_s[PRE ? 2 * kPreMax : 4];

  const int tiles_n = (a.N + BN - 1) / BN;
  const int tile = a.rev ? (int)gridDim.x - 1 - xcd_remap(blockIdx.x, gridDim.x) : xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * BN;

  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  if constexpr (PRE) {
    // Zero beyond K: the padded k columns read zeros and stay zero.
    for (int c = t; c < a.Kp; c += NT) {
      pre_s[c] = c < a.K ? a.pre_scale[c] : 0.0f;
      pre_s[kPreMax + c] = c < a.K ? a.pre_shift[c] : 0.0f;
    }
    __syncthreads();
  }
  DmaPlan<NA, NB, LD> dp;
  dp.init(a, m0, n0, wave * NA, wave * NB, lane);
  const int nk = a.Kp / BK;
  // Only instructions q0 <= q < q1 of the tile's NA + NB (A first, then B)
  // are issued, so the DMA of one k-tile can be spread over several k-steps.
  auto issue = [&](int kt, int st, int q0, int q1) {
    uint16_t *As = smem + st * SM::kStage;
    dp.issue(a, kt, As, As + BM * BK, q0, q1);
  };

  const int wm = wave / WN, wn = wave % WN;
  const int lrow = lane & 31, lh = lane >> 5;
  // Fragment offsets inside a stage; k-step ks reads logical chunk 2 ks + lh,
  // stored at physical chunk (2 ks + lh) ^ ((row >> 1) & 7), and fragment rows
  // are 32-aligned, so (row >> 1) & 7 == (lrow >> 1) & 7.
  int aoff[TM], boff[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) aoff[i] = (wm * TM * 32 + i * 32 + lrow) * BK;
#pragma unroll
  for (int j = 0; j < TN; ++j) boff[j] = BM * BK + (wn * TN * 32 + j * 32 + lrow) * BK;
  const int sw = (lrow >> 1) & 7;

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // The residual block this thread adds in the staged epilogue, loaded
  // before the first DMA (so it is older than every DMA the k-loop waits
  // for): its latency overlaps the whole k-loop instead of the epilogue.
  constexpr int CPR = BN / 8;   // 8-column chunks per row
  constexpr int RPP = NT / CPR; // rows per pass
  constexpr int RPT = BM / RPP; // rows per thread
  uint4 rpre[EPI ? 1 : RPT];
  if (!EPI && a.res) {
    const uint16_t *res = static_cast<const uint16_t *>(a.res);
    const int n = n0 + (t % CPR) * 8;
#pragma unroll
    for (int k = 0; k < RPT; ++k) {
      const int m = m0 + t / CPR + k * RPP;
      rpre[k] = (m < a.M && n < a.N) ? *reinterpret_cast<const uint4 *>(res + (int64_t)m * a.ldr + n)
                                      : make_uint4(0, 0, 0, 0);
    }
  }
  // The staged epilogue's bias (8 channels per thread), loaded here for the
  // same reason: read after the k-loop, its latency would fall in the epilogue.
  float bpre[EPI ? 1 : 8];
  if constexpr (!EPI) {
    const int n = n0 + (t % CPR) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) bpre[e] = (a.bias && n < a.N) ? a.bias[n + e] : 0.0f;
  }

#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < nk) issue(st, st, 0, NA + NB);

  bf16x8_t af[2][TM], bfr[2][TN];
  auto read_frags = [&](const uint16_t *S, int ks, int buf, int kt) {
    const int ch = ((2 * ks + lh) ^ sw) * 8;
#pragma unroll
    for (int i = 0; i < TM; ++i) af[buf][i] = *reinterpret_cast<const bf16x8_t *>(S + aoff[i] + ch);
#pragma unroll
    for (int j = 0; j < TN; ++j) bfr[buf][j] = *reinterpret_cast<const bf16x8_t *>(S + boff[j] + ch);
    if constexpr (PRE) {
      // this lane's 8 channels: logical chunk 2 ks + lh of k-tile kt
      const float *ps = pre_s + kt * BK + (2 * ks + lh) * 8;
      const float4 s0 = *reinterpret_cast<const float4 *>(ps), s1 = *reinterpret_cast<const float4 *>(ps + 4);
      const float4 h0 = *reinterpret_cast<const float4 *>(ps + kPreMax);
      const float4 h1 = *reinterpret_cast<const float4 *>(ps + kPreMax + 4);
#pragma unroll
      for (int i = 0; i < TM; ++i) af[buf][i] = preact8(af[buf][i], s0, s1, h0, h1);
    }
  };
  // One k-tile from LDS stage S: KS MFMA k-steps; step ks reads the
  // fragments of step ks + 1 while its MFMAs run.  With a DMA (WITH_DMA), the
  // instructions of a later k-tile are spread evenly over the first KS - 1
  // steps: the memory pipeline accepts about one 1 KB DMA per 16 clocks per CU,
  // and a burst would stall the issuing wave (and its MFMAs) on a full queue;
  // the last step is left as slack for the DMAs to land.
  // With SCHED each step is its own scheduling region in which the reads and
  // DMA issues are placed between the MFMAs, so one wait per step covers the
  // next step's operands.
  auto run_tile = [&](const uint16_t *S, int kc, int kn, int sn, auto with_dma) {
    constexpr bool WITH_DMA = decltype(with_dma)::value;
    read_frags(S, 0, 0, kc);
    if (SCHED) __builtin_amdgcn_sched_barrier(0);
    static_for<KS>([&](auto ksc) {
      constexpr int ks = decltype(ksc)::value;
      constexpr int cur = ks & 1;
      if constexpr (ks + 1 < KS) read_frags(S, ks + 1, cur ^ 1, kc);
      constexpr int NDS = KS > 1 ? KS - 1 : 1, NQ = NA + NB;
      constexpr int q0 = !WITH_DMA || ks >= NDS ? 0 : ks * NQ / NDS;
      constexpr int q1 = !WITH_DMA || ks >= NDS ? 0 : (ks + 1) * NQ / NDS;
      if constexpr (q1 > q0) issue(kn, sn, q0, q1);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = EPI ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[cur][j], af[cur][i], acc[i][j], 0, 0, 0)
                          : __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0);
      if constexpr (SCHED != 0) {
        constexpr int ndma = q1 - q0;
        sched_step<0, TM * TN, (ks + 1 < KS) ? TM + TN : 0, ndma>();
        __builtin_amdgcn_sched_barrier(0);
      }
    });
  };

  int kt = 0;
  // Steady state: STAGES - 2 younger tiles in flight at the wait, and the
  // tile STAGES - 1 ahead is issued every iteration.
  for (; kt + STAGES - 1 < nk; ++kt) {
    wait_vmcnt<(STAGES - 2) * (NA + NB)>();
    __builtin_amdgcn_s_barrier();
    const int kn = kt + STAGES - 1;
    run_tile(smem + (kt % STAGES) * SM::kStage, kt, kn, kn % STAGES, std::true_type{});
  }
  // Drain: no more tiles to issue.
  for (; kt < nk; ++kt) {
    if (STAGES >= 3 && nk - 1 - kt >= 1) wait_vmcnt<(STAGES >= 3 ? 1 : 0) * (NA + NB)>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    run_tile(smem + (kt % STAGES) * SM::kStage, kt, 0, 0, std::false_type{});
  }
  if (EPI) {
    // acc[i][j][4g + e] = C[m][n + e], m = block row + lane % 32,
    // n = block column + 8 g + 4 (lane / 32).
    uint16_t *y = static_cast<uint16_t *>(a.y);
    const uint16_t *res = static_cast<const uint16_t *>(a.res);
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n0 + wn * TN * 32 + j * 32 + 8 * g + 4 * lh;
        if (n >= a.N) continue;
        const float4 bv = a.bias ? *reinterpret_cast<const float4 *>(a.bias + n)
                                 : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int m = m0 + wm * TM * 32 + i * 32 + lrow;
          if (m >= a.M) continue;
          float v[4] = {acc[i][j][4 * g] + bv.x, acc[i][j][4 * g + 1] + bv.y,
                        acc[i][j][4 * g + 2] + bv.z, acc[i][j][4 * g + 3] + bv.w};
          if (res) {
            const uint2 rv = *reinterpret_cast<const uint2 *>(res + (int64_t)m * a.ldr + n);
            v[0] += bf2f((uint16_t)(rv.x & 0xffff));
            v[1] += bf2f((uint16_t)(rv.x >> 16));
            v[2] += bf2f((uint16_t)(rv.y & 0xffff));
            v[3] += bf2f((uint16_t)(rv.y >> 16));
          }
          uint2 o;
          o.x = f2bf2(epilogue_act(v[0], a.relu, a.gelu), epilogue_act(v[1], a.relu, a.gelu));
          o.y = f2bf2(epilogue_act(v[2], a.relu, a.gelu), epilogue_act(v[3], a.relu, a.gelu));
          *reinterpret_cast<uint2 *>(y + (int64_t)m * a.ldc + n) = o;
        }
      }
    }
    return;
  }

  // Epilogue: stage the fp32 tile in LDS, then each thread finishes 8
  // consecutive output channels of a row and stores them as one 16-byte write.
  __syncthreads();
  float *Cs = reinterpret_cast<float *>(smem_raw);
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wm * TM * 32 + i * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
        const int col = wn * TN * 32 + j * 32 + lrow;
        Cs[row * SM::kCPitch + col] = acc[i][j][r];
      }
  __syncthreads();
  const int cc = t % CPR;
  const int n = n0 + cc * 8;
  if (n >= a.N && !a.out_hw) return;
  const float *bias = bpre;
  uint16_t *y = static_cast<uint16_t *>(a.y);
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int rr = t / CPR + k * RPP;
    const int m = m0 + rr;
    if (m >= a.M || n >= a.N) break;
    const float4 p = *reinterpret_cast<const float4 *>(Cs + rr * SM::kCPitch + cc * 8);
    const float4 q = *reinterpret_cast<const float4 *>(Cs + rr * SM::kCPitch + cc * 8 + 4);
    // bias, then the residual: the order of every epilogue in the library
    float v[8] = {p.x + bias[0], p.y + bias[1], p.z + bias[2], p.w + bias[3],
                  q.x + bias[4], q.y + bias[5], q.z + bias[6], q.w + bias[7]};
    if (a.res) {
      const uint4 rv = rpre[EPI ? 0 : k];
      const uint32_t w4[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] += bf2f((uint16_t)(w4[e] & 0xffff));
        v[2 * e + 1] += bf2f((uint16_t)(w4[e] >> 16));
      }
    }
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = epilogue_act(v[2 * e], a.relu, a.gelu);
      const float hi = epilogue_act(v[2 * e + 1], a.relu, a.gelu);
      o[e] = f2bf2(lo, hi);
    }
    if (a.out_hw) {
      // the finished chunk back into the first half of its own staging
      // slot (no other thread reads that slot)
      *reinterpret_cast<uint4 *>(Cs + rr * SM::kCPitch + cc * 8) = make_uint4(o[0], o[1], o[2], o[3]);
    } else {
      *reinterpret_cast<uint4 *>(y + (int64_t)m * a.ldc + n) = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
  if (a.out_hw) {
    // NCHW store: consecutive threads take consecutive rows (pixels) of one
    // channel, which are consecutive addresses within an image.
    __syncthreads();
    const uint16_t *Cb = reinterpret_cast<const uint16_t *>(Cs);
    for (int idx = t; idx < BM * BN; idx += NT) {
      const int c = idx / BM, rr = idx - c * BM;
      const int m = m0 + rr, nn = n0 + c;
      if (m >= a.M || nn >= a.N) continue;
      const int img = m / a.out_hw, px = m - img * a.out_hw;
      y[((int64_t)img * a.N + nn) * a.out_hw + px] = Cb[rr * (2 * SM::kCPitch) + (c / 8) * 16 + (c % 8)];
    }
  }
}

// ------------------------------------------ bf16, warp-specialised pipeline
//
// WM x WN consumer waves only read fragments and run MFMAs; as many producer
// waves move the k-tiles STAGES - 1 ahead into LDS with buffer loads that
// write LDS directly.  A SIMD whose MFMA pipe is kept busy by one wave issues
// VALU instructions of its other waves only rarely, so the producers' steady
// state holds no VALU instruction at all: every per-lane byte offset is
// computed once (one per kernel tap), padding taps and rows beyond M / N get
// an offset outside the buffer's range, for which the hardware writes zeros,
// and a k-tile only moves scalar values (the LDS address in M0 and the
// buffer's scalar offset).  One s_barrier per k-tile, reached by all waves,
// hands a landed stage to the consumers and a consumed stage back to the
// producers.
// Per-lane offsets of one producer lane.  Row-group g = ga + i (A) or gb + j
// (B) covers rows 8 g .. 8 g + 7; lane l moves row 8 g + l / 8 and logical
// chunk (l % 8) ^ ((row >> 1) & 7) of the 64-wide k-tile, as in DmaPlan.
template <int NA, int NB, int LD, int KW>
struct WsPlan {
  // LD_NHWC8: one offset per k-tile (two k-tiles of 8 taps each)
  static constexpr int TAPS = (LD == LD_NHWC || LD == LD_CAT) ? KW * KW : LD == LD_NHWC8 ? 2 : 1;
  unsigned va[TAPS][NA];                // A, first part: per kernel tap
  unsigned va2[LD == LD_CAT ? NA : 1];  // LD_CAT: shortcut pixel (n, ho s2, wo s2) of x2
  unsigned vb[NB];

  __device__ __forceinline__ void init(const ConvArgs &a, int m0, int n0, int ga, int gb, int lane) {
    const int kcA = ((lane & 7) ^ ((lane >> 4) & 7)) * 8;        // even g
    const int kcB = ((lane & 7) ^ ((4 + (lane >> 4)) & 7)) * 8;  // odd g
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      const int m = m0 + (ga + i) * 8 + (lane >> 3);
      const int kc8 = ((ga + i) & 1) ? kcB : kcA;
      const bool valid = m < a.M;
      const int mm = valid ? m : 0;
      int n, ho, wo;
      if (LD == LD_NHWC && a.pool) {  // row 4 window + 2 dy + dx
        const int wp_n = a.Wo >> 1, hwp = (a.Ho >> 1) * wp_n;
        const int win = mm >> 2;
        n = win / hwp;
        const int rem = win - n * hwp, hp = rem / wp_n;
        ho = 2 * hp + ((mm >> 1) & 1);
        wo = 2 * (rem - hp * wp_n) + (mm & 1);
      } else {
        const int hw = a.Ho * a.Wo;
        n = mm / hw;
        const int rem = mm - n * hw;
        ho = rem / a.Wo;
        wo = rem - ho * a.Wo;
      }
      if (LD == LD_NHWC8) {
        // chunk kc8 / 8 of k-tile t is tap 8 t + kc8 / 8: the 8 channel slots
        // of one input pixel, or zeros (padding, taps past kh x kw)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int tap = 8 * t + kc8 / 8;
          const int hi = ho * a.stride - a.pad + tap / a.kw, wi = wo * a.stride - a.pad + tap % a.kw;
          const bool in = valid && tap < a.kh * a.kw && (unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W;
          va[t][i] = in ? (unsigned)(((((int64_t)n * a.H + hi) * a.W + wi) * 8) * 2) : kOob;
        }
      } else if (LD == LD_GEMM) {
        va[0][i] = valid ? (unsigned)(((int64_t)m * (a.lda ? a.lda : a.K) + kc8) * 2) : kOob;
      } else if (LD == LD_S2D) {  // k-tile du adds du * W * C (scalar)
        va[0][i] = valid ? (unsigned)(((((int64_t)n * a.H + ho) * a.W + wo) * a.C + kc8) * 2) : kOob;
      } else if (LD == LD_NCHW_PATCH) {  // kw == 16: k-tile = 4 kernel rows of one channel
        const int du = kc8 >> 4, dv = kc8 & 15;
        va[0][i] = valid ? (unsigned)((((int64_t)n * a.C * a.H + ho * a.kh + du) * a.W + wo * a.kw + dv) * 2)
                         : kOob;
      } else {  // LD_NHWC, LD_CAT first part
#pragma unroll
        for (int tap = 0; tap < TAPS; ++tap) {
          const int hi = ho * a.stride - a.pad + tap / KW, wi = wo * a.stride - a.pad + tap % KW;
          const bool in = valid && (unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W;
          va[tap][i] = in ? (unsigned)(((((int64_t)n * a.H + hi) * a.W + wi) * a.C + kc8) * 2) : kOob;
        }
        if (LD == LD_CAT)
          va2[LD == LD_CAT ? i : 0] =
              valid ? (unsigned)(((((int64_t)n * a.H2 + ho * a.s2) * a.W2 + wo * a.s2) * a.C2 + kc8) * 2) : kOob;
      }
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int n = n0 + (gb + j) * 8 + (lane >> 3);
      vb[j] = n < a.N ? (unsigned)(((int64_t)n * a.Kp + (((gb + j) & 1) ? kcB : kcA)) * 2) : kOob;
    }
  }
};

template <int BM, int BN, int WM, int WN, int STAGES, int LD, int KW, int EPI, bool PRE = false>
__device__ __forceinline__ void conv_bf16_ws_body(const ConvArgs &a) {
  constexpr int CW = WM * WN;                      // consumer waves (= producer waves)
  constexpr int NT = 2 * CW * 64;
  constexpr int TM = BM / (WM * 32), TN = BN / (WN * 32);
  constexpr int NA = BM / (8 * CW), NB = BN / (8 * CW);  // DMA instructions per producer lane
  constexpr int NQ = NA + NB;
  constexpr int KS = BK / 16;
  using SM = PipeSmem<BM, BN, STAGES, EPI>;
  using Plan = WsPlan<NA, NB, LD, KW>;
  static_assert(NA * 8 * CW == BM && NB * 8 * CW == BN && TM >= 1 && TN >= 1, "tile");
  static_assert(STAGES >= 2 && STAGES <= 4 && (STAGES - 2) * NQ < 64, "stages");
  __shared__ __attribute__((aligned(16))) uint8_t smem_raw[SM::kBytes];
  uint16_t *smem = reinterpret_cast<uint16_t *>(smem_raw);
  __shared__ __attribute__((aligned(16))) float pre_s[PRE ? 2 * kPreMax : 4];
  __shared__ __attribute__((aligned(16))) float bias_s[EPI == 2 ? BN : 4];

  const int tiles_n = (a.N + BN - 1) / BN;
  const int tile = a.rev ? (int)gridDim.x - 1 - xcd_remap(blockIdx.x, gridDim.x) : xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * BN;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);  // uniform: keeps LDS addresses scalar
  const bool producer = wave >= CW;
  const int nk = a.Kp / BK;
  if constexpr (PRE) {
    // Zero beyond K: the columns of the last k-tile past K (which the loader
    // reads from the next channels of the row) become exact zeros, whatever
    // they hold (ReLU maps NaN to 0).
    for (int c = t; c < a.Kp; c += NT) {
      pre_s[c] = c < a.K ? a.pre_scale[c] : 0.0f;
      pre_s[kPreMax + c] = c < a.K ? a.pre_shift[c] : 0.0f;
    }
    __syncthreads();
  }

  const int wm = (wave % CW) / WN, wn = (wave % CW) % WN;
  const int lrow = lane & 31, lh = lane >> 5;
  f32x16_t acc[TM][TN];

  // Residual rows of the staged epilogue, loaded before any DMA (so they are
  // older than every DMA a producer waits for): the latency overlaps the
  // k-loop instead of the epilogue.
  constexpr int CPR = BN / 8;    // 8-column chunks per row
  constexpr int RPP = NT / CPR;  // rows per pass
  constexpr int RPT = BM / RPP;  // rows per thread
  uint4 rpre[EPI ? 1 : RPT];
  if (!EPI && a.res) {
    const uint16_t *res = static_cast<const uint16_t *>(a.res);
    const int n = n0 + (t % CPR) * 8;
#pragma unroll
    for (int k = 0; k < RPT; ++k) {
      const int m = m0 + t / CPR + k * RPP;
      rpre[k] = (m < a.M && n < a.N) ? *reinterpret_cast<const uint4 *>(res + (int64_t)m * a.ldr + n)
                                      : make_uint4(0, 0, 0, 0);
    }
  }
  // EPI = 2: the tile's bias into LDS (written before this wave's first
  // barrier, read after the last), and each consumer lane's residual chunks
  // into registers: 8 channels at column 32 j + 16 p + 8 lh of row
  // 32 i + lane % 32 of its block.
  uint4 rdir[EPI == 2 ? TM : 1][EPI == 2 ? TN : 1][2];
  if constexpr (EPI == 2) {
    if (t < BN) bias_s[t] = (a.bias && n0 + t < a.N) ? a.bias[n0 + t] : 0.0f;
    if (!producer && a.res) {
      const uint16_t *res = static_cast<const uint16_t *>(a.res);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int p = 0; p < 2; ++p) {
            const int m = m0 + wm * TM * 32 + 32 * i + lrow;
            const int n = n0 + wn * TN * 32 + 32 * j + 16 * p + 8 * lh;
            rdir[i][j][p] = (m < a.M && n < a.N) ? *reinterpret_cast<const uint4 *>(res + (int64_t)m * a.ldr + n)
                                                 : make_uint4(0, 0, 0, 0);
          }
    }
    // LDS writes done before the barrier that publishes them (lgkmcnt(0)
    // only: the residual loads stay in flight)
    __builtin_amdgcn_s_waitcnt(0xC07F);
  }

  if (producer) {
    const int pw = wave - CW;
    Plan pl;
    pl.init(a, m0, n0, pw * NA, pw * NB, lane);
    // k-tiles per tap of the first part; the scalar A offset of k-tile (tap, cb)
    const int cpt = (LD == LD_NHWC || LD == LD_CAT) ? a.C / BK : LD == LD_NHWC8 ? 1 : nk;
    auto soff_a = [&](int cb) -> unsigned {
      if (LD == LD_NHWC8) return 0u;
      if (LD == LD_GEMM || LD == LD_NHWC || LD == LD_CAT) return (unsigned)(cb * BK * 2);
      if (LD == LD_S2D) return (unsigned)(cb * a.W * a.C * 2);
      // LD_NCHW_PATCH: channel c = cb / (kh / 4), kernel rows u0 = 4 (cb % (kh / 4))
      const int rpc = a.kh / 4, c = cb / rpc, u0 = (cb - c * rpc) * 4;
      return (unsigned)((((int64_t)c * a.H + u0) * a.W) * 2);
    };
    int q = 0;  // next k-tile to issue
    // Before issuing k-tile q into stage q % STAGES: once STAGES - 1 tiles are
    // in flight, wait until k-tile q - STAGES + 1 has landed, then meet the
    // consumers at its barrier (which also frees the stage it reuses).
    auto gate = [&] {
      if (q >= STAGES - 1) {
        wait_vmcnt<(STAGES - 2) * NQ>();
        __builtin_amdgcn_s_barrier();
      }
    };
    auto issue_b = [&](uint16_t *Bs) {
#pragma unroll
      for (int j = 0; j < NB; ++j)
        dma16(a.w, Bs + (pw * NB + j) * 512, pl.vb[j], (unsigned)(q * BK * 2));
    };
    static_for<Plan::TAPS>([&](auto tc) {
      constexpr int tap = decltype(tc)::value;
      for (int cb = 0; cb < cpt; ++cb) {
        gate();
        uint16_t *As = smem + (q % STAGES) * SM::kStage;
        const unsigned so = soff_a(cb);
#pragma unroll
        for (int i = 0; i < NA; ++i)
          dma16(a.x, As + (pw * NA + i) * 512, pl.va[tap][i], so);
        issue_b(As + BM * BK);
        ++q;
      }
    });
    if (LD == LD_CAT) {  // shortcut part: 1 x 1 on x2
      const int cpt2 = a.C2 / BK;
      for (int cb = 0; cb < cpt2; ++cb) {
        gate();
        uint16_t *As = smem + (q % STAGES) * SM::kStage;
#pragma unroll
        for (int i = 0; i < NA; ++i)
          dma16(a.x2, As + (pw * NA + i) * 512, pl.va2[LD == LD_CAT ? i : 0], (unsigned)(cb * BK * 2));
        issue_b(As + BM * BK);
        ++q;
      }
    }
    // Drain: the last min(nk, STAGES - 1) barriers; k-tile b has nk - 1 - b
    // younger tiles in flight.
    for (int b = max(0, nk - STAGES + 1); b < nk; ++b) {
      const int younger = nk - 1 - b;
      if (STAGES >= 4 && younger >= 2) wait_vmcnt<(STAGES >= 4 ? 2 : 0) * NQ>();
      else if (STAGES >= 3 && younger >= 1) wait_vmcnt<(STAGES >= 3 ? 1 : 0) * NQ>();
      else wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();
    }
  } else {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
    // Fragment offsets inside a stage; k-step ks reads logical chunk 2 ks + lh,
    // stored at physical chunk (2 ks + lh) ^ ((row >> 1) & 7).
    int aoff[TM], boff[TN];
#pragma unroll
    for (int i = 0; i < TM; ++i) aoff[i] = (wm * TM * 32 + i * 32 + lrow) * BK;
#pragma unroll
    for (int j = 0; j < TN; ++j) boff[j] = BM * BK + (wn * TN * 32 + j * 32 + lrow) * BK;
    const int sw = (lrow >> 1) & 7;
    bf16x8_t af[2][TM], bfr[2][TN];
    auto read_frags = [&](const uint16_t *S, int ks, int buf, int kt) {
      const int ch = ((2 * ks + lh) ^ sw) * 8;
#pragma unroll
      for (int i = 0; i < TM; ++i) af[buf][i] = *reinterpret_cast<const bf16x8_t *>(S + aoff[i] + ch);
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[buf][j] = *reinterpret_cast<const bf16x8_t *>(S + boff[j] + ch);
      if constexpr (PRE) {
        const float *ps = pre_s + kt * BK + (2 * ks + lh) * 8;
        const float4 s0 = *reinterpret_cast<const float4 *>(ps), s1 = *reinterpret_cast<const float4 *>(ps + 4);
        const float4 h0 = *reinterpret_cast<const float4 *>(ps + kPreMax);
        const float4 h1 = *reinterpret_cast<const float4 *>(ps + kPreMax + 4);
#pragma unroll
        for (int i = 0; i < TM; ++i) af[buf][i] = preact8(af[buf][i], s0, s1, h0, h1);
      }
    };
    for (int kt = 0; kt < nk; ++kt) {
      __builtin_amdgcn_s_barrier();
      const uint16_t *S = smem + (kt % STAGES) * SM::kStage;
      read_frags(S, 0, 0, kt);
      __builtin_amdgcn_sched_barrier(0);
      static_for<KS>([&](auto ksc) {
        constexpr int ks = decltype(ksc)::value;
        constexpr int cur = ks & 1;
        if constexpr (ks + 1 < KS) read_frags(S, ks + 1, cur ^ 1, kt);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = EPI ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[cur][j], af[cur][i], acc[i][j], 0, 0, 0)
                            : __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0);
        sched_step<0, TM * TN, (ks + 1 < KS) ? TM + TN : 0, 0>();
        __builtin_amdgcn_sched_barrier(0);
      });
    }
  }

  uint16_t *y = static_cast<uint16_t *>(a.y);
  const uint16_t *res = static_cast<const uint16_t *>(a.res);
  if constexpr (EPI == 2) {
    if (producer) return;
    // The residual loads, issued before the k-loop, have landed long ago:
    // one explicit wait here tells the compiler so, and spares every later
    // part the wait it would otherwise place behind the earlier parts'
    // stores (loads and stores share the vector-memory counter).
    wait_vmcnt<0>();
    // acc[i][j][4 g + e] = C[row 32 i + lane % 32][column 32 j + 8 g + 4 lh + e]
    // of this wave's block; the lower half-wave keeps group 2 p and receives
    // the upper half's, the upper half receives the lower half's group 2 p + 1.
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const int m = m0 + wm * TM * 32 + 32 * i + lrow;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          float v[8];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const auto sw2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[i][j][8 * p + e]),
                                                              __float_as_uint(acc[i][j][8 * p + 4 + e]), false, false);
            v[e] = __uint_as_float(sw2[0]);
            v[4 + e] = __uint_as_float(sw2[1]);
          }
          const int c = wn * TN * 32 + 32 * j + 16 * p + 8 * lh, n = n0 + c;
          if (n >= a.N) continue;
          const float4 b0 = *reinterpret_cast<const float4 *>(bias_s + c);
          const float4 b1 = *reinterpret_cast<const float4 *>(bias_s + c + 4);
          v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
          v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
          if (res) {
            const uint4 rv = rdir[i][j][p];
            const uint32_t w4[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              v[2 * e] += bf2f((uint16_t)(w4[e] & 0xffff));
              v[2 * e + 1] += bf2f((uint16_t)(w4[e] >> 16));
            }
          }
          uint32_t o[4];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            o[e] = f2bf2(epilogue_act(v[2 * e], a.relu, a.gelu), epilogue_act(v[2 * e + 1], a.relu, a.gelu));
          if (a.pool) {
            // 2 x 2 max pooling: rows 4 w .. 4 w + 3 (window w) are lanes
            // l, l ^ 1, l ^ 2, l ^ 3; the window's first lane stores.
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              o[e] = bf16x2_max(o[e], (uint32_t)__shfl_xor((int)o[e], 1, 64));
              o[e] = bf16x2_max(o[e], (uint32_t)__shfl_xor((int)o[e], 2, 64));
            }
            if ((lrow & 3) == 0 && m < a.M)
              *reinterpret_cast<uint4 *>(y + (int64_t)(m >> 2) * a.ldc + n) = make_uint4(o[0], o[1], o[2], o[3]);
          } else if (m < a.M) {
            *reinterpret_cast<uint4 *>(y + (int64_t)m * a.ldc + n) = make_uint4(o[0], o[1], o[2], o[3]);
          }
        }
    }
    return;
  }
  if (EPI == 1) {
    if (producer) return;
    // acc[i][j][4g + e] = C[m][n + e], m = block row + lane % 32,
    // n = block column + 8 g + 4 (lane / 32).
#pragma unroll
    for (int j = 0; j < TN; ++j) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n0 + wn * TN * 32 + j * 32 + 8 * g + 4 * lh;
        if (n >= a.N) continue;
        const float4 bv = a.bias ? *reinterpret_cast<const float4 *>(a.bias + n)
                                 : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          const int m = m0 + wm * TM * 32 + i * 32 + lrow;
          if (m >= a.M) continue;
          float v[4] = {acc[i][j][4 * g] + bv.x, acc[i][j][4 * g + 1] + bv.y,
                        acc[i][j][4 * g + 2] + bv.z, acc[i][j][4 * g + 3] + bv.w};
          if (res) {
            const uint2 rv = *reinterpret_cast<const uint2 *>(res + (int64_t)m * a.ldr + n);
            v[0] += bf2f((uint16_t)(rv.x & 0xffff));
            v[1] += bf2f((uint16_t)(rv.x >> 16));
            v[2] += bf2f((uint16_t)(rv.y & 0xffff));
            v[3] += bf2f((uint16_t)(rv.y >> 16));
          }
          uint2 o;
          o.x = f2bf2(epilogue_act(v[0], a.relu, a.gelu), epilogue_act(v[1], a.relu, a.gelu));
          o.y = f2bf2(epilogue_act(v[2], a.relu, a.gelu), epilogue_act(v[3], a.relu, a.gelu));
          *reinterpret_cast<uint2 *>(y + (int64_t)m * a.ldc + n) = o;
        }
      }
    }
    return;
  }

  // Epilogue: the consumers stage the fp32 tile in LDS (the stages are free:
  // every DMA has landed and every fragment was read before this barrier),
  // then all waves finish 8 consecutive output channels of a row per thread
  // and store them as one 16-byte write.
  __syncthreads();
  float *Cs = reinterpret_cast<float *>(smem_raw);
  if (!producer) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wm * TM * 32 + i * 32 + 8 * (r >> 2) + 4 * lh + (r & 3);
          const int col = wn * TN * 32 + j * 32 + lrow;
          Cs[row * SM::kCPitch + col] = acc[i][j][r];
        }
  }
  __syncthreads();
  const int cc = t % CPR;
  const int n = n0 + cc * 8;
  if (n >= a.N && !a.out_hw) return;
  float bias[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) bias[e] = (a.bias && n < a.N) ? a.bias[n + e] : 0.0f;
#pragma unroll
  for (int k = 0; k < RPT; ++k) {
    const int rr = t / CPR + k * RPP;
    const int m = m0 + rr;
    if (m >= a.M || n >= a.N) break;
    const float4 p = *reinterpret_cast<const float4 *>(Cs + rr * SM::kCPitch + cc * 8);
    const float4 q = *reinterpret_cast<const float4 *>(Cs + rr * SM::kCPitch + cc * 8 + 4);
    // bias, then the residual: the order of every epilogue in the library
    float v[8] = {p.x + bias[0], p.y + bias[1], p.z + bias[2], p.w + bias[3],
                  q.x + bias[4], q.y + bias[5], q.z + bias[6], q.w + bias[7]};
    if (res) {
      const uint4 rv = rpre[EPI ? 0 : k];
      const uint32_t w4[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        v[2 * e] += bf2f((uint16_t)(w4[e] & 0xffff));
        v[2 * e + 1] += bf2f((uint16_t)(w4[e] >> 16));
      }
    }
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = epilogue_act(v[2 * e], a.relu, a.gelu);
      const float hi = epilogue_act(v[2 * e + 1], a.relu, a.gelu);
      o[e] = f2bf2(lo, hi);
    }
    if (a.out_hw) {
      // the finished chunk back into the first half of its own staging
      // slot (no other thread reads that slot)
      *reinterpret_cast<uint4 *>(Cs + rr * SM::kCPitch + cc * 8) = make_uint4(o[0], o[1], o[2], o[3]);
    } else {
      *reinterpret_cast<uint4 *>(y + (int64_t)m * a.ldc + n) = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
  if (a.out_hw) {
    // NCHW store: consecutive threads take consecutive rows (pixels) of one
    // channel, which are consecutive addresses within an image.
    __syncthreads();
    const uint16_t *Cb = reinterpret_cast<const uint16_t *>(Cs);
    for (int idx = t; idx < BM * BN; idx += NT) {
      const int c = idx / BM, rr = idx - c * BM;
      const int m = m0 + rr, nn = n0 + c;
      if (m >= a.M || nn >= a.N) continue;
      const int img = m / a.out_hw, px = m - img * a.out_hw;
      y[((int64_t)img * a.N + nn) * a.out_hw + px] = Cb[rr * (2 * SM::kCPitch) + (c / 8) * 16 + (c % 8)];
    }
  }
}

// One workgroup per CU (large tiles), or two (the register budget halves).
template <int BM, int BN, int WM, int WN, int STAGES, int LD, int KW, int EPI>
__global__ __launch_bounds__(2 * WM * WN * 64) void conv_bf16_ws_kernel(ConvArgs a) {
  conv_bf16_ws_body<BM, BN, WM, WN, STAGES, LD, KW, EPI>(a);
}
template <int BM, int BN, int WM, int WN, int STAGES, int LD, int KW, int EPI, bool PRE = false>
__global__ __launch_bounds__(2 * WM * WN * 64, 2) void conv_bf16_ws2_kernel(ConvArgs a) {
  conv_bf16_ws_body<BM, BN, WM, WN, STAGES, LD, KW, EPI, PRE>(a);
}

template <int BM, int BN, int WM, int WN, int STAGES, int LD, int KW, int EPI>
__global__ __launch_bounds__(2 * WM * WN * 64, 3) void conv_bf16_ws3_kernel(ConvArgs a) {
  conv_bf16_ws_body<BM, BN, WM, WN, STAGES, LD, KW, EPI>(a);
}

template <int BM, int BN, int WM, int WN, int STAGES, int LD, int KW, int EPI = 0, int MINB = 1, bool PRE = false>
hipError_t launch_ws_cfg(const ConvArgs &a, hipStream_t s) {
  // the NCHW split store needs the staged epilogue
  if constexpr (EPI == 2)
    if (a.out_hw) return launch_ws_cfg<BM, BN, WM, WN, STAGES, LD, KW, 0, MINB, PRE>(a, s);
  if (a.pool && (EPI != 2 || LD != LD_NHWC)) return hipErrorNotSupported;  // pooling: register epilogue
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  if constexpr (MINB >= 3 && !PRE)
    hapi_launch((conv_bf16_ws3_kernel<BM, BN, WM, WN, STAGES, LD, KW, EPI>), dim3(tiles),
                       dim3(2 * WM * WN * 64), 0, s, a);
  else if constexpr (MINB >= 2)
    hapi_launch((conv_bf16_ws2_kernel<BM, BN, WM, WN, STAGES, LD, KW, EPI, PRE>), dim3(tiles),
                       dim3(2 * WM * WN * 64), 0, s, a);
  else
    hapi_launch((conv_bf16_ws_kernel<BM, BN, WM, WN, STAGES, LD, KW, EPI>), dim3(tiles),
                       dim3(2 * WM * WN * 64), 0, s, a);
  return hipGetLastError();
}

template <int BM, int BN, int LD>
hipError_t launch_bf16_cfg(const ConvArgs &a, hipStream_t s) {
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  hapi_launch((conv_bf16_kernel<BM, BN, LD>), dim3(tiles), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

// Whether every element offset the pipelined kernel's DMA forms stays below
// 2^30 (byte offsets below 2^31).
template <int LD>
bool pipe_offsets_fit(const ConvArgs &a) {
  const int64_t lim = (int64_t)1 << 30;
  if ((int64_t)a.N * a.Kp >= lim) return false;
  if (LD == LD_GEMM) return (int64_t)a.M * (a.lda ? a.lda : a.K) < lim;
  if (LD == LD_CAT && (int64_t)a.n_img * a.H2 * a.W2 * a.C2 >= lim) return false;
  return (int64_t)a.n_img * a.C * a.H * a.W < lim;
}

template <int BM, int BN, int WM, int WN, int STAGES, int LD, int SCHED = 1, int EPI = 0, bool PRE = false>
hipError_t launch_pipe_cfg(const ConvArgs &a, hipStream_t s) {
  // The DMA addresses every operand with 32-bit byte offsets: past 2^31 bytes
  // the register-staged kernel (64-bit addresses) takes the element-gather
  // loaders, and the others report the size as unsupported.
  if (!pipe_offsets_fit<LD>(a)) {
    if constexpr (!PRE && (LD == LD_GEMM || LD == LD_NHWC || LD == LD_NCHW_PATCH))
      return launch_bf16_cfg<BM, BN, LD>(a, s);
    return hipErrorInvalidValue;
  }
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  hapi_launch((conv_bf16_pipe_kernel<BM, BN, WM, WN, STAGES, LD, SCHED, EPI, PRE>), dim3(tiles),
                     dim3(WM * WN * 64), 0, s, a);
  return hipGetLastError();
}

// ------------------------------- bf16, persistent warp-specialised pipeline
//
// As the warp-specialised kernel, but one workgroup per CU processes a
// contiguous range of output tiles, and its PW producer waves stream the
// k-tiles of consecutive tiles through one STAGES-deep ring.  The ring never
// drains between tiles: the first k-tiles of the next tile load while the
// WM x WN consumer waves finish the current one, so layers with a few k-tiles
// per tile no longer pay the pipeline fill once per tile.  Consumers prefetch
// the residual of a tile into registers before its first k-tile, so its
// latency overlaps the whole k-loop.  The MFMA operands are swapped (weights
// as A) so that a lane's accumulators hold 4 consecutive output channels of
// one pixel.  Epilogue EP = 0 stores those 8 bytes per lane directly; EP = 1
// finishes 32-row slabs in a private LDS area per wave and stores 16-byte
// row chunks; EP = 2 exchanges accumulator halves between the two half-waves
// (v_permlane32_swap) so that every lane owns 8 consecutive channels of one
// pixel, then loads the residual and stores the result as 16-byte chunks,
// without LDS.
template <int BM, int BN, int WM, int WN, int PW, int STAGES, int LD, int KW, int EP, bool PRE = false>
__global__ __launch_bounds__((WM * WN + PW) * 64, 1) void conv_bf16_pws_kernel(ConvArgs a) {
  constexpr int CW = WM * WN;                             // consumer waves
  constexpr int TM = BM / (WM * 32), TN = BN / (WN * 32);
  constexpr int NA = BM / (8 * PW), NB = BN / (8 * PW);   // DMA instructions per producer lane
  constexpr int NQ = NA + NB;
  constexpr int KS = BK / 16;
  constexpr int kStage = (BM + BN) * BK;                  // elements per stage
  constexpr int kWC = TN * 32;                            // columns of a consumer wave's block
  constexpr int kEP = kWC + 8;                            // bf16 pitch of a staged slab row
  constexpr int kSlab = EP == 1 ? 32 * kEP : 0;           // elements of a wave's slab
  using Plan = WsPlan<NA, NB, LD, KW>;
  static_assert(NA * 8 * PW == BM && NB * 8 * PW == BN && TM >= 1 && TN >= 1, "tile");
  static_assert(STAGES >= 2 && STAGES <= 6 && (STAGES - 2) * NQ < 64, "stages");
  static_assert((STAGES * kStage + CW * kSlab) * 2 <= 163840, "LDS");
  static_assert((CW + PW) * 64 <= 1024, "workgroup size");
  // The bias is read from LDS in the epilogue: a global load there would sit
  // behind the wave's earlier stores in the one vector-memory counter, and
  // every wait for it would also wait for those stores to be acknowledged.
  constexpr int kPreLds = PRE ? 2 * kPreMax * 4 : 16;
  constexpr int kLdsUsed = (STAGES * kStage + CW * kSlab) * 2 + kPreLds;
  constexpr int kBiasMax = (163840 - kLdsUsed) / 4 < 4096 ? (163840 - kLdsUsed) / 4 : 4096;
  static_assert(kBiasMax >= 256, "LDS for the bias");
  __shared__ __attribute__((aligned(16))) uint16_t smem[STAGES * kStage + CW * kSlab];
  __shared__ __attribute__((aligned(16))) float bias_s[kBiasMax];
  // PRE: the A operand's per-channel scale [0, kPreMax) and shift
  // [kPreMax, 2 kPreMax), zero past K (the ragged last k-tile's extra
  // columns, read from the row's next channels, become exact zeros).
  __shared__ __attribute__((aligned(16))) float pre_s[kPreLds / 4];

  const int tiles_n = (a.N + BN - 1) / BN;
  const int tiles = ((a.M + BM - 1) / BM) * tiles_n;
  const int G = gridDim.x;
  // Logical workgroup index: consecutive indices share an XCD (and its L2),
  // so an XCD works through one contiguous range of tiles.
  const int wg = xcd_remap(blockIdx.x, G);
  const int t_lo = (int)((int64_t)tiles * wg / G), t_hi = (int)((int64_t)tiles * (wg + 1) / G);
  const int nk = a.Kp / BK;
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);  // uniform: keeps LDS addresses scalar
  // Bias in LDS when it fits (one barrier, met by every wave before the
  // producer / consumer split); zero when absent.
  const bool bias_lds = a.N <= kBiasMax;
  if (bias_lds) {
    for (int c = t; c < a.N; c += (CW + PW) * 64) bias_s[c] = a.bias ? a.bias[c] : 0.0f;
  }
  if constexpr (PRE) {
    for (int c = t; c < a.Kp; c += (CW + PW) * 64) {
      pre_s[c] = c < a.K ? a.pre_scale[c] : 0.0f;
      pre_s[kPreMax + c] = c < a.K ? a.pre_shift[c] : 0.0f;
    }
  }
  if (bias_lds || PRE) __syncthreads();

  if (wave >= CW) {
    // ---- producers: k-tile q of the workgroup's stream goes to stage q % STAGES.
    const int pw = wave - CW;
    const int cpt = (LD == LD_NHWC || LD == LD_CAT) ? a.C / BK : nk;  // k-tiles per tap
    auto soff_a = [&](int cb) -> unsigned {
      if (LD == LD_GEMM || LD == LD_NHWC || LD == LD_CAT) return (unsigned)(cb * BK * 2);
      if (LD == LD_S2D) return (unsigned)(cb * a.W * a.C * 2);
      const int rpc = a.kh / 4, c = cb / rpc, u0 = (cb - c * rpc) * 4;  // LD_NCHW_PATCH
      return (unsigned)((((int64_t)c * a.H + u0) * a.W) * 2);
    };
    int q = 0;
    // Before issuing k-tile q: once STAGES - 1 are in flight, wait until k-tile
    // q - STAGES + 1 has landed and meet the consumers at its barrier, which
    // also frees the stage that k-tile q reuses.
    auto gate = [&] {
      if (q >= STAGES - 1) {
        wait_vmcnt<(STAGES - 2) * NQ>();
        __builtin_amdgcn_s_barrier();
      }
    };
    for (int ti = t_lo; ti < t_hi; ++ti) {
      const int tile = a.rev ? t_lo + t_hi - 1 - ti : ti;
      const int m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * BN;
      Plan pl;
      pl.init(a, m0, n0, pw * NA, pw * NB, lane);
      int kq = 0;  // k-tile within the tile
      auto issue_b = [&](uint16_t *Bs) {
#pragma unroll
        for (int j = 0; j < NB; ++j)
          dma16(a.w, Bs + (pw * NB + j) * 512, pl.vb[j], (unsigned)(kq * BK * 2));
      };
      static_for<Plan::TAPS>([&](auto tc) {
        constexpr int tap = decltype(tc)::value;
        for (int cb = 0; cb < cpt; ++cb) {
          gate();
          uint16_t *As = smem + (q % STAGES) * kStage;
          const unsigned so = soff_a(cb);
#pragma unroll
          for (int i = 0; i < NA; ++i) dma16(a.x, As + (pw * NA + i) * 512, pl.va[tap][i], so);
          issue_b(As + BM * BK);
          ++q;
          ++kq;
        }
      });
      if (LD == LD_CAT) {  // shortcut part: 1 x 1 on x2
        const int cpt2 = a.C2 / BK;
        for (int cb = 0; cb < cpt2; ++cb) {
          gate();
          uint16_t *As = smem + (q % STAGES) * kStage;
#pragma unroll
          for (int i = 0; i < NA; ++i)
            dma16(a.x2, As + (pw * NA + i) * 512, pl.va2[LD == LD_CAT ? i : 0], (unsigned)(cb * BK * 2));
          issue_b(As + BM * BK);
          ++q;
          ++kq;
        }
      }
    }
    // Drain: the last min(q, STAGES - 1) barriers; k-tile b has q - 1 - b
    // younger k-tiles in flight.
    for (int b = max(0, q - STAGES + 1); b < q; ++b) {
      const int younger = q - 1 - b;
      static_for<STAGES - 1>([&](auto yc) {
        constexpr int yv = decltype(yc)::value;
        if (younger == yv) wait_vmcnt<yv * NQ>();
      });
      __builtin_amdgcn_s_barrier();
    }
    return;  // every barrier of the stream has been met
  }

  // ---- consumers
  const int wm = wave / WN, wn = wave % WN;
  const int lrow = lane & 31, lh = lane >> 5;
  const int sw = (lrow >> 1) & 7;
  // Fragment offsets inside a stage; k-step ks reads logical chunk 2 ks + lh,
  // stored at physical chunk (2 ks + lh) ^ ((row >> 1) & 7).
  int aoff[TM], boff[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) aoff[i] = (wm * TM * 32 + i * 32 + lrow) * BK;
#pragma unroll
  for (int j = 0; j < TN; ++j) boff[j] = BM * BK + (wn * kWC + j * 32 + lrow) * BK;
  uint16_t *y = static_cast<uint16_t *>(a.y);
  const uint16_t *res = static_cast<const uint16_t *>(a.res);
  uint16_t *slab = smem + STAGES * kStage + wave * kSlab;
  bf16x8_t af[2][TM], bfr[2][TN];
  auto read_frags = [&](const uint16_t *S, int ks, int buf, int kt) {
    const int ch = ((2 * ks + lh) ^ sw) * 8;
#pragma unroll
    for (int i = 0; i < TM; ++i) af[buf][i] = *reinterpret_cast<const bf16x8_t *>(S + aoff[i] + ch);
#pragma unroll
    for (int j = 0; j < TN; ++j) bfr[buf][j] = *reinterpret_cast<const bf16x8_t *>(S + boff[j] + ch);
    if constexpr (PRE) {  // channels kt BK + 16 ks + 8 lh .. + 8 of this lane's rows
      const float *ps = pre_s + kt * BK + (2 * ks + lh) * 8;
      const float4 s0 = *reinterpret_cast<const float4 *>(ps), s1 = *reinterpret_cast<const float4 *>(ps + 4);
      const float4 h0 = *reinterpret_cast<const float4 *>(ps + kPreMax);
      const float4 h1 = *reinterpret_cast<const float4 *>(ps + kPreMax + 4);
#pragma unroll
      for (int i = 0; i < TM; ++i) af[buf][i] = preact8(af[buf][i], s0, s1, h0, h1);
    }
  };
  // Residual chunk of (i, j, part): EP 0 / 1: 4 channels at column
  // 32 j + 8 part + 4 lh (part = g, 0..3); EP 2: 8 channels at column
  // 32 j + 16 part + 8 lh (part 0..1).  Row 32 i + lane % 32 of the block.
  constexpr int NPART = EP == 2 ? 2 : 4;
  using ResT = typename std::conditional<EP == 2, uint4, uint2>::type;
  // The tile loop is instantiated twice, reading the bias from LDS or (N
  // beyond the LDS copy) from global memory, so that no epilogue wait
  // covers the other path's counter.
  auto consume = [&](auto lds_bias) {
  constexpr bool kLdsBias = decltype(lds_bias)::value;
  int q = 0;
  for (int ti = t_lo; ti < t_hi; ++ti) {
    const int tile = a.rev ? t_lo + t_hi - 1 - ti : ti;
    const int m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * BN;
    const int mw = m0 + wm * TM * 32, nw = n0 + wn * kWC;  // origin of this wave's block
    ResT rr[TM][TN][NPART];
    if (res) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int p = 0; p < NPART; ++p) {
            const int m = mw + 32 * i + lrow;
            const int n = nw + 32 * j + (EP == 2 ? 16 * p + 8 * lh : 8 * p + 4 * lh);
            if (m < a.M && n < a.N) rr[i][j][p] = *reinterpret_cast<const ResT *>(res + (int64_t)m * a.ldr + n);
            else if constexpr (EP == 2) rr[i][j][p] = make_uint4(0u, 0u, 0u, 0u);
            else rr[i][j][p] = make_uint2(0u, 0u);
          }
    }
    // acc[i][j][4 g + e] = C[mw + 32 i + lrow][nw + 32 j + 8 g + 4 lh + e]
    f32x16_t acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
    for (int kt = 0; kt < nk; ++kt, ++q) {
      __builtin_amdgcn_s_barrier();
      const uint16_t *S = smem + (q % STAGES) * kStage;
      read_frags(S, 0, 0, kt);
      __builtin_amdgcn_sched_barrier(0);
      static_for<KS>([&](auto ksc) {
        constexpr int ks = decltype(ksc)::value;
        constexpr int cur = ks & 1;
        if constexpr (ks + 1 < KS) read_frags(S, ks + 1, cur ^ 1, kt);
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[cur][j], af[cur][i], acc[i][j], 0, 0, 0);
        sched_step<0, TM * TN, (ks + 1 < KS) ? TM + TN : 0, 0>();
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    // Epilogue: bias, residual, activation and one rounding per element.
    if constexpr (EP == 2) {
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int m = mw + 32 * i + lrow;
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int p = 0; p < 2; ++p) {
            // Lower half-wave keeps group 2p and receives the upper half's
            // group 2p; the upper half receives the lower half's group 2p + 1.
            float v[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const auto sw2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[i][j][8 * p + e]),
                                                                __float_as_uint(acc[i][j][8 * p + 4 + e]), false, false);
              v[e] = __uint_as_float(sw2[0]);
              v[4 + e] = __uint_as_float(sw2[1]);
            }
            const int n = nw + 32 * j + 16 * p + 8 * lh;
            if (n < a.N) {
              // LDS or global memory, never one pointer to either: that
              // would be a flat load, which waits for every store of the
              // wave still in flight.
              float4 b0 = make_float4(0.f, 0.f, 0.f, 0.f), b1 = b0;
              if constexpr (kLdsBias) {
                b0 = *reinterpret_cast<const float4 *>(bias_s + n);
                b1 = *reinterpret_cast<const float4 *>(bias_s + n + 4);
              } else if (a.bias) {
                b0 = *reinterpret_cast<const float4 *>(a.bias + n);
                b1 = *reinterpret_cast<const float4 *>(a.bias + n + 4);
              }
              v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
              v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
              if (res) {
                const uint4 rv = rr[i][j][p];
                const uint32_t w4[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  v[2 * e] += bf2f((uint16_t)(w4[e] & 0xffff));
                  v[2 * e + 1] += bf2f((uint16_t)(w4[e] >> 16));
                }
              }
              uint32_t o[4];
#pragma unroll
              for (int e = 0; e < 4; ++e)
                o[e] = f2bf2(epilogue_act(v[2 * e], a.relu, a.gelu), epilogue_act(v[2 * e + 1], a.relu, a.gelu));
              if (a.pool) {
                // 2 x 2 max pooling: rows 4 w .. 4 w + 3 (window w) are lanes
                // l, l ^ 1, l ^ 2, l ^ 3; the window's first lane stores.
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                  o[e] = bf16x2_max(o[e], (uint32_t)__shfl_xor((int)o[e], 1, 64));
                  o[e] = bf16x2_max(o[e], (uint32_t)__shfl_xor((int)o[e], 2, 64));
                }
                if ((lrow & 3) == 0 && m < a.M)
                  *reinterpret_cast<uint4 *>(y + (int64_t)(m >> 2) * a.ldc + n) = make_uint4(o[0], o[1], o[2], o[3]);
              } else if (m < a.M) {
                *reinterpret_cast<uint4 *>(y + (int64_t)m * a.ldc + n) = make_uint4(o[0], o[1], o[2], o[3]);
              }
            }
          }
      }
    } else {
#pragma unroll
      for (int i = 0; i < TM; ++i) {
        const int m = mw + 32 * i + lrow;
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int col = 32 * j + 8 * g + 4 * lh, n = nw + col;
            float4 bv = make_float4(0.f, 0.f, 0.f, 0.f);  // LDS or global, never a flat load
            if (n < a.N) {
              if constexpr (kLdsBias) bv = *reinterpret_cast<const float4 *>(bias_s + n);
              else if (a.bias) bv = *reinterpret_cast<const float4 *>(a.bias + n);
            }
            float v[4] = {acc[i][j][4 * g] + bv.x, acc[i][j][4 * g + 1] + bv.y, acc[i][j][4 * g + 2] + bv.z,
                          acc[i][j][4 * g + 3] + bv.w};
            if (res) {
              const uint2 rv = *reinterpret_cast<const uint2 *>(&rr[i][j][g]);
              v[0] += bf2f((uint16_t)(rv.x & 0xffff));
              v[1] += bf2f((uint16_t)(rv.x >> 16));
              v[2] += bf2f((uint16_t)(rv.y & 0xffff));
              v[3] += bf2f((uint16_t)(rv.y >> 16));
            }
            uint2 o;
            o.x = f2bf2(epilogue_act(v[0], a.relu, a.gelu), epilogue_act(v[1], a.relu, a.gelu));
            o.y = f2bf2(epilogue_act(v[2], a.relu, a.gelu), epilogue_act(v[3], a.relu, a.gelu));
            if (EP == 1) *reinterpret_cast<uint2 *>(slab + lrow * kEP + col) = o;
            else if (m < a.M && n < a.N) *reinterpret_cast<uint2 *>(y + (int64_t)m * a.ldc + n) = o;
          }
        if (EP == 1) {
          // The slab is private to this wave: order its writes before the
          // reads of other lanes, then store row segments of kWC columns.
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
          constexpr int CPR = kWC / 8;  // 16-byte chunks per slab row
#pragma unroll
          for (int c = lane; c < 32 * CPR; c += 64) {
            const int row = c / CPR, col = (c % CPR) * 8;
            const int mm = mw + 32 * i + row, n = nw + col;
            const uint4 val = *reinterpret_cast<const uint4 *>(slab + row * kEP + col);
            if (mm < a.M && n < a.N) *reinterpret_cast<uint4 *>(y + (int64_t)mm * a.ldc + n) = val;
          }
          __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
          __builtin_amdgcn_wave_barrier();
          __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }
      }
    }
  }
  };
  if (bias_lds) consume(std::true_type{});
  else consume(std::false_type{});
}

// ------------------------------------- bf16, short-K (one or two k-tiles)
//
// For GEMMs with K <= 128 (the memory-bound 1 x 1 layers) a tile's whole
// A and B fit in LDS, and the time per tile is one memory round trip, which
// under load is several microseconds.  Each workgroup issues all of its loads
// at once (the k-tiles by LDS DMA, its residual block into registers, its
// bias slice into LDS), waits once, runs the MFMAs and stores 16-byte chunks
// after a half-wave exchange (as the persistent kernel's epilogue).  Several
// workgroups per CU at different phases keep the loads of the whole device in
// flight.
template <int BM, int BN, int WM, int WN, int KT, int LD, int MINB>
__global__ __launch_bounds__(WM * WN * 64, MINB) void conv_bf16_short_kernel(ConvArgs a) {
  constexpr int NT = WM * WN * 64;
  constexpr int TM = BM / (WM * 32), TN = BN / (WN * 32);
  constexpr int NA = BM * 8 / NT, NB = BN * 8 / NT;  // DMA instructions per thread per k-tile
  constexpr int KS = BK / 16;
  constexpr int kStage = (BM + BN) * BK;
  constexpr int kWC = TN * 32;
  static_assert(TM >= 1 && TN >= 1 && NA >= 1 && NB >= 1 && KT >= 1 && KT <= 8, "tile");
  static_assert(KT * (BM + BN) * BK * 2 + BN * 4 <= 163840, "LDS");
  __shared__ __attribute__((aligned(16))) uint16_t smem[KT * kStage];
  __shared__ __attribute__((aligned(16))) float bias_s[BN];

  const int tiles_n = (a.N + BN - 1) / BN;
  const int tile = a.rev ? (int)gridDim.x - 1 - xcd_remap(blockIdx.x, gridDim.x) : xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * BN;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int lrow = lane & 31, lh = lane >> 5;
  const int mw = m0 + wm * TM * 32, nw = n0 + wn * kWC;  // this wave's block

  // All loads first: the k-tiles (LDS DMA), then the residual block and the
  // bias slice into registers; one wait covers them all.
  DmaPlan<NA, NB, LD> dp;
  dp.init(a, m0, n0, wave * NA, wave * NB, lane);
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) {
    uint16_t *As = smem + kt * kStage;
    dp.issue(a, kt, As, As + BM * BK, 0, NA + NB);
  }
  // Residual chunks of (i, j, part): 8 channels at column 32 j + 16 part + 8 lh
  // of row 32 i + lane % 32 of the block.
  uint4 rr[TM][TN][2];
  const uint16_t *res = static_cast<const uint16_t *>(a.res);
  if (res) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const int m = mw + 32 * i + lrow, n = nw + 32 * j + 16 * p + 8 * lh;
          rr[i][j][p] = (m < a.M && n < a.N) ? *reinterpret_cast<const uint4 *>(res + (int64_t)m * a.ldr + n)
                                             : make_uint4(0u, 0u, 0u, 0u);
        }
  }
  const float bv = (t < BN && a.bias && n0 + t < a.N) ? a.bias[n0 + t] : 0.0f;
  wait_vmcnt<0>();  // every load of this tile (the DMAs, the residual, the bias)
  if (t < BN) bias_s[t] = bv;
  __syncthreads();

  int aoff[TM], boff[TN];
#pragma unroll
  for (int i = 0; i < TM; ++i) aoff[i] = (wm * TM * 32 + i * 32 + lrow) * BK;
#pragma unroll
  for (int j = 0; j < TN; ++j) boff[j] = BM * BK + (wn * kWC + j * 32 + lrow) * BK;
  const int sw = (lrow >> 1) & 7;
  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
#pragma unroll
  for (int kt = 0; kt < KT; ++kt) {
    const uint16_t *S = smem + kt * kStage;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int ch = ((2 * ks + lh) ^ sw) * 8;
      bf16x8_t af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) af[i] = *reinterpret_cast<const bf16x8_t *>(S + aoff[i] + ch);
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[j] = *reinterpret_cast<const bf16x8_t *>(S + boff[j] + ch);
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
    }
  }
  uint16_t *y = static_cast<uint16_t *>(a.y);
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    const int m = mw + 32 * i + lrow;
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        float v[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const auto sw2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[i][j][8 * p + e]),
                                                            __float_as_uint(acc[i][j][8 * p + 4 + e]), false, false);
          v[e] = __uint_as_float(sw2[0]);
          v[4 + e] = __uint_as_float(sw2[1]);
        }
        const int nl = wn * kWC + 32 * j + 16 * p + 8 * lh, n = n0 + nl;
        if (n < a.N && m < a.M) {
          const float4 b0 = *reinterpret_cast<const float4 *>(bias_s + nl);
          const float4 b1 = *reinterpret_cast<const float4 *>(bias_s + nl + 4);
          v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
          v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
          if (res) {
            const uint4 rv = rr[i][j][p];
            const uint32_t w4[4] = {rv.x, rv.y, rv.z, rv.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              v[2 * e] += bf2f((uint16_t)(w4[e] & 0xffff));
              v[2 * e + 1] += bf2f((uint16_t)(w4[e] >> 16));
            }
          }
          uint32_t o[4];
#pragma unroll
          for (int e = 0; e < 4; ++e)
            o[e] = f2bf2(epilogue_act(v[2 * e], a.relu, a.gelu), epilogue_act(v[2 * e + 1], a.relu, a.gelu));
          *reinterpret_cast<uint4 *>(y + (int64_t)m * a.ldc + n) = make_uint4(o[0], o[1], o[2], o[3]);
        }
      }
  }
}

template <int BM, int BN, int WM, int WN, int KT, int LD, int MINB>
hipError_t launch_short_cfg(const ConvArgs &a, hipStream_t s) {
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  hapi_launch((conv_bf16_short_kernel<BM, BN, WM, WN, KT, LD, MINB>), dim3(tiles), dim3(WM * WN * 64), 0, s, a);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, int LD, int MINB>
hipError_t launch_short_ld(const ConvArgs &a, hipStream_t s) {
  if (a.Kp == 2 * BK) return launch_short_cfg<BM, BN, WM, WN, 2, LD, MINB>(a, s);
  return launch_short_cfg<BM, BN, WM, WN, 1, LD, MINB>(a, s);
}

}  // namespace

// CUs of the current device (persistent grids use one workgroup per CU).
int cu_count() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cached[dev] <= 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) v = 256;
    cached[dev] = v;
  }
  return cached[dev];
}

namespace {

template <int BM, int BN, int WM, int WN, int PW, int STAGES, int LD, int KW, int EP, bool PRE = false>
hipError_t launch_pws_cfg(const ConvArgs &a, hipStream_t s) {
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  const int cus = a.cus > 0 ? a.cus : cu_count();
  const int grid = tiles < cus ? tiles : cus;
  if (PRE && a.Kp > kPreMax) return hipErrorInvalidValue;
  if (a.pool && (EP != 2 || LD != LD_NHWC)) return hipErrorNotSupported;  // pooling: 8-channel epilogue
  hapi_launch((conv_bf16_pws_kernel<BM, BN, WM, WN, PW, STAGES, LD, KW, EP, PRE>), dim3(grid),
                     dim3((WM * WN + PW) * 64), 0, s, a);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, int PW, int STAGES, int LD, int EP>
hipError_t launch_pws_ld(const ConvArgs &a, hipStream_t s) {
  if ((LD == LD_NHWC || LD == LD_CAT) && a.kh == 3)
    return launch_pws_cfg<BM, BN, WM, WN, PW, STAGES, LD, 3, EP>(a, s);
  return launch_pws_cfg<BM, BN, WM, WN, PW, STAGES, LD, 1, EP>(a, s);
}

// Whether the warp-specialised kernel handles this launch: whole 64-wide
// k-tiles, kernel taps it was built for, and every operand addressable with
// 31-bit byte offsets.
bool ws_eligible(const ConvArgs &a, Loader ld) {
  const int64_t lim = (int64_t)1 << 31;
  if ((int64_t)a.N * a.Kp * 2 >= lim) return false;
  switch (ld) {
    case LD_GEMM: return a.K % BK == 0 && (int64_t)a.M * a.K * 2 < lim;
    case LD_NHWC:
    case LD_CAT:
      if (a.C % BK != 0 || a.kh != a.kw || (a.kh != 1 && a.kh != 3)) return false;
      if ((int64_t)a.n_img * a.H * a.W * a.C * 2 >= lim) return false;
      return ld == LD_NHWC || (a.C2 % BK == 0 && (int64_t)a.n_img * a.H2 * a.W2 * a.C2 * 2 < lim);
    case LD_S2D: return (int64_t)a.n_img * a.H * a.W * a.C * 2 < lim;
    case LD_NHWC8:
      return a.Kp == 2 * BK && a.kh * a.kw > 8 && a.kh * a.kw <= 16 && (int64_t)a.n_img * a.H * a.W * 16 < lim;
    case LD_NCHW_PATCH:
      return a.kw == 16 && a.kh % 4 == 0 && (int64_t)a.n_img * a.C * a.H * a.W * 2 < lim;
    default: return false;
  }
}

template <int BM, int BN, int WM, int WN, int STAGES, int LD, int EPI, int MINB>
hipError_t launch_ws_ld(const ConvArgs &a, hipStream_t s) {
  if (LD == LD_NHWC || LD == LD_CAT) {
    if (a.kh == 3) return launch_ws_cfg<BM, BN, WM, WN, STAGES, LD, 3, EPI, MINB>(a, s);
    return launch_ws_cfg<BM, BN, WM, WN, STAGES, LD, 1, EPI, MINB>(a, s);
  }
  return launch_ws_cfg<BM, BN, WM, WN, STAGES, LD, 1, EPI, MINB>(a, s);
}

// Tile shape per layer.  Every shape uses the same k-tile and MFMA, so the
// choice never changes a result bit.
// A split output stored as NCHW from the epilogue: the warp-specialised
// kernel with the LDS-staged epilogue, in the tile shape the layer would get
// (tile shapes never change results).
template <int LD>
hipError_t launch_nchw_out(const ConvArgs &a, hipStream_t s) {
  if (!ws_eligible(a, (Loader)LD) || LD == LD_S2D || a.N % 8) return hipErrorNotSupported;
  if (a.lanes <= 1 && a.N >= 64 && 2 * (int64_t)((a.M + 127) / 128) * ((a.N + 127) / 128) < a.cus)
    return launch_ws_ld<64, 64, 2, 2, 4, LD, 0, 2>(a, s);
  if (a.N <= 64) return launch_ws_ld<128, 64, 2, 2, 3, LD, 0, 2>(a, s);
  if (a.res && a.N >= 1024) return launch_ws_ld<128, 64, 2, 2, 2, LD, 0, 3>(a, s);
  return launch_ws_ld<128, 128, 2, 2, 2, LD, 0, 2>(a, s);
}

template <int LD>
hipError_t launch_pipe_ld(const ConvArgs &a, hipStream_t s) {
  if (a.out_hw > 0) return launch_nchw_out<LD>(a, s);
  // Measured on MI355X over the ResNet-50 conv shapes (per-layer kernel
  // traces of every configuration above):
  // - the warp-specialised kernel with two workgroups per CU (128 x 64 tiles)
  //   for the space-to-depth stem and 64-channel outputs with K = 64 or
  //   K >= 512; with 128 x 128 tiles for residual layers with < 1024 output
  //   channels and for 128-channel 3 x 3 layers; with three workgroups per CU
  //   (128 x 64 tiles, two stages: more loads in flight for these
  //   latency-bound layers) for residual layers with >= 1024 output channels
  //   and, with one partition in flight, 128-channel 1 x 1 layers with
  //   K >= 512;
  // - the persistent kernel (one workgroup of 8 consumer and 4 producer waves
  //   per CU) with 128 x 256 tiles for the fused shortcut GEMMs and the other
  //   layers, and with 256 x 128 tiles for 128-channel 1 x 1 layers with short
  //   K and for >= 512 channels with K >= 2048;
  // - the three-stage pipelined kernel for other single k-tiles (and 64-channel
  //   outputs with K = 128 .. 448), where warp specialisation does not pay.
  // Single k-tile 64-channel 1 x 1 layers and 512-channel residual 1 x 1
  // layers with two k-tiles: all loads of a tile at once, several workgroups
  // per CU (short-K kernel).
  if (LD == LD_GEMM && a.Kp == BK && a.N <= 64 && !a.res) return launch_short_ld<128, 64, 2, 2, LD, 3>(a, s);
  if (LD == LD_GEMM && a.Kp == 2 * BK && a.N == 512 && a.res) return launch_short_ld<128, 64, 2, 2, LD, 3>(a, s);
  if (ws_eligible(a, (Loader)LD)) {
    if (LD == LD_S2D) return launch_ws_ld<128, 64, 2, 2, 3, LD, 2, 2>(a, s);
    // With one partition in flight (none other fills the CUs this launch
    // leaves idle):
    // - fewer 128 x 128 tiles than half the CUs: 64 x 64 tiles, four stages
    //   (ResNet-50 b8: 706 -> 528 us of convolutions per pass; b32 stage-4
    //   3 x 3s 30 -> 20 us);
    // - long reductions with fewer 256-row tiles than half the CUs:
    //   persistent 128 x 128 tiles (ResNet-18 b64 stage 3: 111 -> 82 us,
    //   ResNet-50 b32 31.8k -> 37.4k img/s).  With more (ResNet-50 stage 4 at
    //   M = 12544: 196 tiles) 256 x 128 stays faster, 60 against 73 us, and
    //   with two partitions in flight the larger tiles win throughout
    //   (ResNet-50 b256: 70.1k against 67.2k img/s).
    // - 3 x 3 reductions of K >= 2048 with at most half as many 64 x 64 tiles
    //   as CUs: 32 x 64 tiles, four stages, so twice the CUs walk the long
    //   k-chain (ResNet-50 b8 stage-3 3 x 3 11.3 -> 10.3 us, stage 4
    //   18.9 -> 16.7 us; with more tiles, as at b32, 64 x 64 stays faster);
    if (a.lanes <= 1 && a.kh == 3 && a.K >= 2048 && a.N >= 64 &&
        2 * (int64_t)((a.M + 63) / 64) * ((a.N + 63) / 64) <= a.cus)
      return launch_ws_ld<32, 64, 1, 2, 4, LD, 2, 2>(a, s);
    if (a.lanes <= 1 && a.N >= 64 && 2 * (int64_t)((a.M + 127) / 128) * ((a.N + 127) / 128) < a.cus)
      return launch_ws_ld<64, 64, 2, 2, 4, LD, 2, 2>(a, s);
    if (a.lanes <= 1 && a.N >= 128 && a.K >= 1024 &&
        2 * (int64_t)((a.M + 255) / 256) * ((a.N + 127) / 128) < a.cus)
      return launch_pws_ld<128, 128, 2, 2, 4, 4, LD, 2>(a, s);
    // 32 output channels (DenseNet growth): a 32-column tile, so no MFMA
    // works on padding; 32 x 32 per consumer wave, three stages (DenseNet-121
    // b256: 56.8k -> 57.7k img/s against 256 x 32 tiles for large M and
    // 128 x 64 tiles, half of them padding, for small M).
    if (a.N <= 32 && a.K >= 2 * BK) return launch_ws_ld<128, 32, 4, 1, 3, LD, 2, 2>(a, s);
    if (a.N <= 64) {
      if (a.K >= 512 || a.K == BK) return launch_ws_ld<128, 64, 2, 2, 3, LD, 2, 2>(a, s);
    } else if (a.res) {
      if (a.K >= 2 * BK) {
        if (a.N >= 1024) return launch_ws_ld<128, 64, 2, 2, 2, LD, 2, 3>(a, s);
        return launch_ws_ld<128, 128, 2, 2, 2, LD, 2, 2>(a, s);
      }
    } else if (LD == LD_CAT) {
      if (a.N <= 128) return launch_pws_ld<256, 128, 4, 2, 4, 3, LD, 2>(a, s);
      return launch_pws_ld<128, 256, 2, 4, 4, 3, LD, 2>(a, s);
    } else if (a.N <= 128) {
      if (a.kh == 1 && a.K <= 256 && a.K >= 2 * BK) return launch_pws_ld<256, 128, 4, 2, 4, 3, LD, 2>(a, s);
      // 3 x 3 over 64 channels to 128 (VGG conv2_1): persistent 256 x 128
      // tiles (VGG-16 b128 +1.6%)
      if (a.kh == 3 && a.K <= 9 * 64 && a.K >= 2 * BK) return launch_pws_ld<256, 128, 4, 2, 4, 3, LD, 2>(a, s);
      // 1 x 1 with K >= 512 (ResNet-50 stage-2 reductions): with partitions
      // in flight persistent 256 x 128 tiles (b256 +1.0%, b512 +0.8%), alone
      // the latency-bound three-workgroups-per-CU tiles
      if (a.kh == 1 && a.K >= 512) {
        if (a.lanes >= 2) return launch_pws_ld<256, 128, 4, 2, 4, 3, LD, 2>(a, s);
        return launch_ws_ld<128, 64, 2, 2, 2, LD, 2, 3>(a, s);
      }
      if (a.K >= 2 * BK) return launch_ws_ld<128, 128, 2, 2, 2, LD, 2, 2>(a, s);
    } else if (LD == LD_GEMM && a.N >= 2048 && a.K <= 1024) {
      // Wide linear layers with a short reduction (ViT qkv and fc1):
      // warp-specialised 128 x 128 tiles (ViT-B/16 qkv at 64 images 56.8 us
      // against 58-65 us with persistent 128 x 256 tiles).
      return launch_ws_ld<128, 128, 2, 2, 2, LD, 2, 2>(a, s);
    } else if (a.N >= 512 && a.K >= 2048) {
      // The longest reductions with enough rows, partitions in flight:
      // 128 x 256 tiles (VGG-16 b128 conv4/conv5 and ResNet-50 b256 stage-4
      // 3 x 3s: +2% and +0.6%); with fewer rows (ResNet-50 b128) or one
      // partition (ResNet-50 stage 4 at M = 12544: 60 against 73 us),
      // 256 x 128 stays faster.
      if (a.K >= 4096 && a.M >= 6272 && a.lanes >= 2) return launch_pws_ld<128, 256, 2, 4, 4, 3, LD, 2>(a, s);
      return launch_pws_ld<256, 128, 4, 2, 4, 3, LD, 2>(a, s);
    } else if (a.K >= 2 * BK) {
      return launch_pws_ld<128, 256, 2, 4, 4, 3, LD, 2>(a, s);
    }
    // The pipelined kernels below do not pool.
    if (a.pool) {
      if (a.N <= 64) return launch_ws_ld<128, 64, 2, 2, 3, LD, 2, 2>(a, s);
      return launch_ws_ld<128, 128, 2, 2, 2, LD, 2, 2>(a, s);
    }
  }
  if (a.N <= 64) {
    if (a.K > 256) return launch_pipe_cfg<128, 64, 2, 2, 2, LD, 1, 1>(a, s);
    return launch_pipe_cfg<128, 64, 2, 2, 3, LD, 1, 0>(a, s);
  }
  return launch_pipe_cfg<128, 128, 2, 2, 2, LD, 1, 0>(a, s);
}

template <int LD>
hipError_t launch_bf16_ld(const ConvArgs &a, hipStream_t s) {
  if (a.N <= 64) return launch_bf16_cfg<128, 64, LD>(a, s);
  const long big_tiles = (long)((a.M + 255) / 256) * ((a.N + 127) / 128);
  if (big_tiles >= 512) return launch_bf16_cfg<256, 128, LD>(a, s);
  return launch_bf16_cfg<128, 128, LD>(a, s);
}

// ------------------------------------------------------------------ fp32

constexpr int BKF = 16;        // k-tile (fp32 elements)
constexpr int LDSF = BKF + 4;  // LDS row pitch in floats (80 B)

template <int LD>
__device__ __forceinline__ float4 load_a_chunk_f32(const ConvArgs &a, const RowState &r, int k0,
                                                   int kh_, int kw_, int c0) {
  const float *x = static_cast<const float *>(a.x);
  float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
  if (LD == LD_GEMM) {
    if (r.hi0 >= 0) v = *reinterpret_cast<const float4 *>(x + r.base + k0);
  } else if (LD == LD_NHWC) {
    const int hi = r.hi0 + kh_, wi = r.wi0 + kw_;
    if ((unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W)
      v = *reinterpret_cast<const float4 *>(x + r.base + (hi * a.W + wi) * a.C + c0);
  } else {  // LD_NCHW element gather, k = (c, u, v)
    if (r.hi0 > -(1 << 27)) {
      float e[4];
      const int khw = a.kh * a.kw;
      int c = k0 / khw, rem = k0 - c * khw;
      int u = rem / a.kw, vv = rem - u * a.kw;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int hi = r.hi0 + u, wi = r.wi0 + vv;
        e[j] = (k0 + j < a.K && (unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W)
                   ? x[r.base + (c * a.H + hi) * a.W + wi]
                   : 0.0f;
        if (++vv == a.kw) { vv = 0; if (++u == a.kh) { u = 0; ++c; } }
      }
      v = make_float4(e[0], e[1], e[2], e[3]);
    }
  }
  return v;
}

template <int BM, int BN, int LD>
__global__ __launch_bounds__(kThreads) void conv_f32_kernel(ConvArgs a) {
  constexpr int WN = 2;
  constexpr int TM = BM / 64, TN = BN / 64;
  constexpr int A_PER = BM * (BKF / 4) / kThreads;  // float4 chunks per thread
  constexpr int B_PER = BN * (BKF / 4) / kThreads;
  static_assert(TM >= 1 && TN >= 1 && A_PER >= 1 && B_PER >= 1, "tile");

  __shared__ __attribute__((aligned(16))) float smem[2 * (BM + BN) * LDSF];

  const int tiles_n = (a.N + BN - 1) / BN;
  const int tile = a.rev ? (int)gridDim.x - 1 - xcd_remap(blockIdx.x, gridDim.x) : xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * BN;

  const int t = threadIdx.x;
  const int kc = t & 3;   // float4 chunk of the 16-wide k-tile
  const int r0 = t >> 2;  // first row; then every 64th

  RowState rs[A_PER];
#pragma unroll
  for (int i = 0; i < A_PER; ++i) rs[i] = make_row<LD>(a, m0 + r0 + 64 * i);

  const float *wp = static_cast<const float *>(a.w);
  float4 ra[A_PER], rb[B_PER];
  auto load_tile = [&](int kt) {
    const int kbase = kt * BKF;
    int kh_ = 0, kw_ = 0, c0 = 0;
    if (LD == LD_NHWC) {  // C % 16 == 0: the k-tile lies in one tap
      const int tap = kbase / a.C;
      c0 = kbase - tap * a.C + kc * 4;
      kh_ = tap / a.kw;
      kw_ = tap - kh_ * a.kw;
    }
#pragma unroll
    for (int i = 0; i < A_PER; ++i) ra[i] = load_a_chunk_f32<LD>(a, rs[i], kbase + kc * 4, kh_, kw_, c0);
#pragma unroll
    for (int j = 0; j < B_PER; ++j) {
      const int n = n0 + r0 + 64 * j;
      rb[j] = (n < a.N) ? *reinterpret_cast<const float4 *>(wp + (size_t)n * a.Kp + kbase + kc * 4)
                        : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto store_tile = [&](int buf) {
    float *As = smem + buf * (BM + BN) * LDSF;
    float *Bs = As + BM * LDSF;
#pragma unroll
    for (int i = 0; i < A_PER; ++i) *reinterpret_cast<float4 *>(As + (r0 + 64 * i) * LDSF + kc * 4) = ra[i];
#pragma unroll
    for (int j = 0; j < B_PER; ++j) *reinterpret_cast<float4 *>(Bs + (r0 + 64 * j) * LDSF + kc * 4) = rb[j];
  };

  const int lane = t & 63, wave = t >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int lrow = lane & 31, lk = (lane >> 5) * 8;

  f32x16_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  // k-tiles [kt0, kt1): slice blockIdx.y of a split reduction, or all of them.
  const int nk_all = a.Kp / BKF;
  const int S = a.splits > 1 ? a.splits : 1;
  const int kt0 = (int)((int64_t)nk_all * blockIdx.y / S), kt1 = (int)((int64_t)nk_all * (blockIdx.y + 1) / S);
  load_tile(kt0);
  store_tile(0);
  __syncthreads();
  for (int kt = kt0; kt < kt1; ++kt) {
    const int cur = (kt - kt0) & 1;
    if (kt + 1 < kt1) load_tile(kt + 1);
    const float *As = smem + cur * (BM + BN) * LDSF + (wm * TM * 32 + lrow) * LDSF + lk;
    const float *Bs = smem + cur * (BM + BN) * LDSF + BM * LDSF + (wn * TN * 32 + lrow) * LDSF + lk;
    // Lane half h feeds k = 8h + s at step s to both operands, so the 8 steps
    // cover the 16 k of the tile exactly once.
    float av[TM][8], bv[TN][8];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
      const float4 p = *reinterpret_cast<const float4 *>(As + i * 32 * LDSF);
      const float4 q = *reinterpret_cast<const float4 *>(As + i * 32 * LDSF + 4);
      av[i][0] = p.x; av[i][1] = p.y; av[i][2] = p.z; av[i][3] = p.w;
      av[i][4] = q.x; av[i][5] = q.y; av[i][6] = q.z; av[i][7] = q.w;
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const float4 p = *reinterpret_cast<const float4 *>(Bs + j * 32 * LDSF);
      const float4 q = *reinterpret_cast<const float4 *>(Bs + j * 32 * LDSF + 4);
      bv[j][0] = p.x; bv[j][1] = p.y; bv[j][2] = p.z; bv[j][3] = p.w;
      bv[j][4] = q.x; bv[j][5] = q.y; bv[j][6] = q.z; bv[j][7] = q.w;
    }
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av[i][s], bv[j][s], acc[i][j], 0, 0, 0);
    if (kt + 1 < kt1) store_tile(cur ^ 1);
    __syncthreads();
  }

  if (S > 1) {  // partial sums of this slice; bias and activation come after the sum
    float *part = a.part + (int64_t)blockIdx.y * a.M * a.N;
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = n0 + wn * TN * 32 + j * 32 + lrow;
      if (n >= a.N) continue;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int m = m0 + wm * TM * 32 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (m < a.M) part[(int64_t)m * a.N + n] = acc[i][j][r];
        }
    }
    return;
  }
  float *y = static_cast<float *>(a.y);
  const float *res = static_cast<const float *>(a.res);
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int n = n0 + wn * TN * 32 + j * 32 + lrow;
    if (n >= a.N) continue;
    const float bvv = a.bias ? a.bias[n] : 0.0f;
#pragma unroll
    for (int i = 0; i < TM; ++i) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int m = m0 + wm * TM * 32 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        if (m >= a.M) continue;
        float v = acc[i][j][r] + bvv;
        if (res) v += res[(int64_t)m * a.ldr + n];
        y[(int64_t)m * a.ldc + n] = epilogue_act(v, a.relu, a.gelu);
      }
    }
  }
}

// Sum of the slices in slice order, then bias, residual and activation (the
// unsplit epilogue's order), 4 channels per thread.
__global__ void f32_split_reduce_kernel(ConvArgs a) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int ng = a.N / 4;
  if (i >= (int64_t)a.M * ng) return;
  const int64_t m = i / ng;
  const int n = (int)(i - m * ng) * 4;
  const int64_t stride = (int64_t)a.M * a.N;
  float4 v = *reinterpret_cast<const float4 *>(a.part + m * a.N + n);
  for (int sl = 1; sl < a.splits; ++sl) {
    const float4 p = *reinterpret_cast<const float4 *>(a.part + sl * stride + m * a.N + n);
    v.x += p.x; v.y += p.y; v.z += p.z; v.w += p.w;
  }
  float o[4] = {v.x, v.y, v.z, v.w};
  const float *res = static_cast<const float *>(a.res);
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    float x = o[e] + (a.bias ? a.bias[n + e] : 0.0f);
    if (res) x += res[m * a.ldr + n + e];
    o[e] = epilogue_act(x, a.relu, a.gelu);
  }
  float *y = static_cast<float *>(a.y);
#pragma unroll
  for (int e = 0; e < 4; ++e) y[m * a.ldc + n + e] = o[e];
}

template <int BM, int BN, int LD>
hipError_t launch_f32_cfg(const ConvArgs &a, hipStream_t s) {
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  const int S = a.splits > 1 ? a.splits : 1;
  if (S > 1 && (!a.part || a.N % 4 != 0 || a.Kp / BKF < S)) return hipErrorInvalidValue;
  hapi_launch((conv_f32_kernel<BM, BN, LD>), dim3(tiles, S), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_bf16(const ConvArgs &a, Loader ld, hipStream_t s) {
  if (a.pool && (ld != LD_NHWC || !a.relu || a.gelu || a.res || a.out_hw || a.pre_scale || a.lda || (a.Ho & 1) ||
                 (a.Wo & 1) || a.N % 16 || a.ldc % 8 || !ws_eligible(a, ld)))
    return hipErrorNotSupported;
  if (a.out_hw > 0 && ((ld != LD_GEMM && ld != LD_NHWC && ld != LD_CAT) || a.pre_scale || (a.lda && a.lda != a.K) ||
                       a.gelu || a.N % 8 || a.ldr % 8))
    return hipErrorNotSupported;
  if (a.pre_scale || (a.lda && a.lda != a.K)) {
    // Pre-activated or strided A (a channel prefix of a wider tensor): the
    // pipelined kernel, whose loader zero-fills the ragged last k-tile.
    if (ld != LD_GEMM || a.N % 8 || a.ldc % 8 || a.ldr % 8 || a.K % 8 || a.lda % 8 || a.Kp > kPreMax ||
        (a.lda && a.lda < a.K) || (int64_t)a.M * (a.lda ? a.lda : a.K) * 2 >= ((int64_t)1 << 31))
      return hipErrorInvalidValue;
    if (!a.pre_scale) return launch_pipe_cfg<128, 128, 2, 2, 2, LD_GEMM, 1, 0>(a, s);
    if (a.N <= 64) return launch_pipe_cfg<128, 64, 2, 2, 3, LD_GEMM, 1, 0, true>(a, s);
    // Warp-specialised with the pre-activation: the ragged last k-tile reads
    // the row's next channels (inside the row when lda >= Kp), which the
    // zero scale and shift turn into zeros.
    if (a.Kp >= 2 * BK && (a.lda ? a.lda : a.K) >= a.Kp &&
        (int64_t)a.M * (a.lda ? a.lda : a.K) * 2 < ((int64_t)1 << 31)) {
      // Persistent 256 x 128 tiles, two stages (the scale and shift take
      // the LDS of a third): DenseNet-121 b256 56.7k -> 57.9k img/s against
      // the warp-specialised 128 x 128 tiles; 128 x 128 persistent tiles
      // were 5% slower.
      return launch_pws_cfg<256, 128, 4, 2, 4, 2, LD_GEMM, 1, 2, true>(a, s);
    }
    return launch_pipe_cfg<128, 128, 2, 2, 2, LD_GEMM, 1, 0, true>(a, s);
  }
  switch (ld) {
    // The pipelined kernel needs 16-byte output rows; the register-staged one
    // handles element gathers (NCHW stems) and any other width.
    case LD_NHWC:
      if (!a.gelu && !a.out_hw && !a.pool && a.Ho == a.H && a.Wo == a.W && conv3x3_c64_supported(a.C, a.N, a.kh, a.kw, a.stride, a.pad, a.W, a.Kp, a.ldc, a.ldr))
        return launch_conv3x3_c64(a.x, a.w, a.Kp, a.bias, a.res, a.ldr, a.y, a.ldc, a.n_img, a.H, a.W, a.relu != 0,
                                  a.cus > 0 ? a.cus : cu_count(), s);
      return (a.N % 8 == 0 && a.ldc % 8 == 0 && a.ldr % 8 == 0) ? launch_pipe_ld<LD_NHWC>(a, s)
                                                                 : launch_bf16_ld<LD_NHWC>(a, s);
    case LD_GEMM:
      return (a.N % 8 == 0 && a.ldc % 8 == 0 && a.ldr % 8 == 0) ? launch_pipe_ld<LD_GEMM>(a, s)
                                                                 : launch_bf16_ld<LD_GEMM>(a, s);
    case LD_NCHW: return launch_bf16_ld<LD_NCHW>(a, s);
    case LD_NCHW_PATCH:
      return (a.N % 8 == 0 && a.ldc % 8 == 0 && a.ldr % 8 == 0) ? launch_pipe_ld<LD_NCHW_PATCH>(a, s)
                                                                 : launch_bf16_ld<LD_NCHW_PATCH>(a, s);
    case LD_S2D:
      if (a.N % 8 == 0 && a.ldc % 8 == 0 && a.ldr % 8 == 0) return launch_pipe_ld<LD_S2D>(a, s);
      break;
    case LD_CAT:
      if (a.N % 8 == 0 && a.ldc % 8 == 0 && a.ldr % 8 == 0) return launch_pipe_ld<LD_CAT>(a, s);
      break;
    case LD_NHWC8:
      if (conv_first_supported(a)) return launch_conv_first(a, s);
      if (a.N % 8 != 0 || a.ldc % 8 != 0 || a.ldr % 8 != 0 || !ws_eligible(a, LD_NHWC8)) break;
      if (a.N <= 64) return launch_ws_cfg<128, 64, 2, 2, 3, LD_NHWC8, 1, 0, 2>(a, s);
      return launch_ws_cfg<128, 128, 2, 2, 2, LD_NHWC8, 1, 0, 2>(a, s);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_f32_split_reduce(const ConvArgs &a, hipStream_t s) {
  if (a.splits <= 1 || !a.part || a.N % 4 != 0) return hipErrorInvalidValue;
  const int64_t items = (int64_t)a.M * (a.N / 4);
  hapi_launch(f32_split_reduce_kernel, dim3((unsigned)((items + 255) / 256)), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_conv_f32(const ConvArgs &a, Loader ld, hipStream_t s) {
  switch (ld) {
    case LD_NHWC: return launch_f32_cfg<64, 64, LD_NHWC>(a, s);
    case LD_GEMM: return launch_f32_cfg<64, 64, LD_GEMM>(a, s);
    case LD_NCHW: return launch_f32_cfg<64, 64, LD_NCHW>(a, s);
    default: break;
  }
  return hipErrorInvalidValue;
}

}  // namespace hapi
