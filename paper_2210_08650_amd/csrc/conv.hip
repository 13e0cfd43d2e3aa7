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
#include <cstdlib>

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

__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;  // NaN stays NaN
  u += 0x7fffu + ((u >> 16) & 1u);                      // round to nearest even
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float epilogue_act(float v, int relu, int gelu) {
  if (relu) v = fmaxf(v, 0.0f);
  if (gelu) v = 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
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
    r.base = m * a.K; r.hi0 = 0; r.wi0 = 0;
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
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
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
// global_load_lds_dwordx4: each lane's 16 bytes land directly in LDS, so no
// registers or ds_write instructions are spent on staging and STAGES - 1
// k-tiles are in flight while the MFMAs consume the oldest one.  Padding taps
// and rows beyond M / N read a zero chunk in global memory instead.
//
// LDS rows hold 64 bf16 (128 B) without padding; the 16-byte chunk kc of row
// r is stored at position kc ^ ((r >> 1) & 7).  The LDS serves 256 bytes (64
// banks) per clock, i.e. two 128-byte rows: with this swizzle the 16 rows a
// quarter-wave fragment read touches land in 16 distinct 16-byte slots of
// that 256-byte window, so fragment reads are free of bank conflicts.

__device__ __attribute__((aligned(64))) uint4 g_zero_chunk[4];

#define LDS_PTR(p) ((__attribute__((address_space(3))) void *)(p))

// Wait until at most N vector-memory operations of this wave are outstanding.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
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
template <int BM, int BN, int WM, int WN, int STAGES, int LD, int SCHED, int EPI>
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

  const int tiles_n = (a.N + BN - 1) / BN;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int m0 = (tile / tiles_n) * BM, n0 = (tile % tiles_n) * BN;

  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  // Lane l of DMA instruction q (q = wave * NA + i, 8 rows of 8 chunks) fills
  // row 8 q + l / 8, physical chunk l % 8, i.e. logical chunk
  // (l % 8) ^ ((row >> 1) & 7) = (l % 8) ^ ((4 q + l / 16) & 7).
  const int kcA = ((lane & 7) ^ ((lane >> 4) & 7)) * 8;        // even q
  const int kcB = ((lane & 7) ^ ((4 + (lane >> 4)) & 7)) * 8;  // odd q
  const uint16_t *zero = reinterpret_cast<const uint16_t *>(g_zero_chunk);
  const uint16_t *x = static_cast<const uint16_t *>(a.x);
  const uint16_t *wp = static_cast<const uint16_t *>(a.w);

  // Per-row gather state, computed once: element offset of the row's first
  // tap (may point into padding), and the tap origin for bounds checks.
  int roff[NA], rhi[NA], rwi[NA], rkc[NA], roff2[LD == LD_CAT ? NA : 1];
  const uint16_t *x2 = static_cast<const uint16_t *>(a.x2);
#pragma unroll
  for (int i = 0; i < NA; ++i) {
    const int m = m0 + (wave * NA + i) * 8 + (lane >> 3);
    const RowState r = make_row<LD == LD_CAT ? LD_NHWC : LD>(a, m);
    const int kc8 = ((wave * NA + i) & 1) ? kcB : kcA;
    rkc[i] = kc8;
    rhi[i] = r.hi0;
    rwi[i] = r.wi0;
    if (LD == LD_NHWC || LD == LD_S2D || LD == LD_CAT)
      roff[i] = r.base + (r.hi0 * a.W + r.wi0) * a.C + kc8;
    else if (LD == LD_GEMM) roff[i] = r.base + kc8;
    else roff[i] = r.base;
    if (LD == LD_CAT) {
      // shortcut pixel (n, ho * s2, wo * s2) of x2
      const int hw = a.Ho * a.Wo;
      const int mm = m < a.M ? m : 0;
      const int n = mm / hw, rem = mm - n * hw;
      const int ho = rem / a.Wo, wo = rem - ho * a.Wo;
      roff2[i] = ((n * a.H2 + ho * a.s2) * a.W2 + wo * a.s2) * a.C2 + kc8 - a.K1;
    }
  }
  int boffs[NB];
  bool bok[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int n = n0 + (wave * NB + j) * 8 + (lane >> 3);
    bok[j] = n < a.N;
    boffs[j] = (bok[j] ? n : 0) * a.Kp + (((wave * NB + j) & 1) ? kcB : kcA);
  }
  const int nk = a.Kp / BK;

  // Moves k-tile kt (< nk) into stage st.  Only per-lane conditions select
  // the zero chunk, so the address arithmetic stays branch-free.
  auto issue = [&](int kt, int st) {
    uint16_t *As = smem + st * SM::kStage;
    uint16_t *Bs = As + BM * BK;
    const int kbase = kt * BK;
    int kh_ = 0, kw_ = 0, tapoff = 0;
    if (LD == LD_NHWC || LD == LD_CAT) {
      const int tap = kbase / a.C;
      kh_ = tap / a.kw;
      kw_ = tap - kh_ * a.kw;
      tapoff = (kh_ * a.W + kw_) * a.C + (kbase - tap * a.C);
    }
    const uint16_t *xs = (LD == LD_CAT && kbase >= a.K1) ? x2 : x;
#pragma unroll
    for (int i = 0; i < NA; ++i) {
      bool ok;
      int off;
      if (LD == LD_GEMM) {  // K % 8 == 0; chunks past K (ragged last k-tile) read zeros
        ok = rhi[i] >= 0 && kbase + rkc[i] < a.K;
        off = roff[i] + kbase;
      } else if (LD == LD_NHWC) {
        ok = (unsigned)(rhi[i] + kh_) < (unsigned)a.H && (unsigned)(rwi[i] + kw_) < (unsigned)a.W;
        off = roff[i] + tapoff;
      } else if (LD == LD_S2D) {
        // k-tile kt is the contiguous run of cell row du = kt (kw x 16 = 64 elements)
        ok = rhi[i] >= 0;
        off = roff[i] + kt * a.W * a.C;
      } else if (LD == LD_CAT) {
        if (kbase < a.K1) {
          ok = (unsigned)(rhi[i] + kh_) < (unsigned)a.H && (unsigned)(rwi[i] + kw_) < (unsigned)a.W;
          off = roff[i] + tapoff;
        } else {
          ok = rhi[i] > -(1 << 27);
          off = roff2[i] + kbase;
        }
      } else {  // LD_NCHW_PATCH: k = (c, u, v), 8 | kw
        const int k0 = kbase + rkc[i];
        const int khw = a.kh * a.kw;
        const int c = k0 / khw, rem = k0 - c * khw;
        const int u = rem / a.kw, vv = rem - u * a.kw;
        ok = rhi[i] > -(1 << 27) && k0 < a.K;
        off = roff[i] + (c * a.H + rhi[i] + u) * a.W + rwi[i] + vv;
      }
      const uint16_t *src = ok ? xs + off : zero;
      __builtin_amdgcn_global_load_lds(src, LDS_PTR(As + (wave * NA + i) * 512), 16, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const uint16_t *src = bok[j] ? wp + boffs[j] + kbase : zero;
      __builtin_amdgcn_global_load_lds(src, LDS_PTR(Bs + (wave * NB + j) * 512), 16, 0, 0);
    }
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

#pragma unroll
  for (int st = 0; st < STAGES - 1; ++st)
    if (st < nk) issue(st, st);

  bf16x8_t af[2][TM], bfr[2][TN];
  // One k-tile from LDS stage S: 4 MFMA k-steps, the next step's fragments
  // read while the current step's MFMAs run.  `pre` issues the DMA of a later
  // k-tile after the first fragments are read.
  auto run_tile = [&](const uint16_t *S, auto &&pre) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
      af[0][i] = *reinterpret_cast<const bf16x8_t *>(S + aoff[i] + ((lh ^ sw) * 8));
#pragma unroll
    for (int j = 0; j < TN; ++j)
      bfr[0][j] = *reinterpret_cast<const bf16x8_t *>(S + boff[j] + ((lh ^ sw) * 8));
    pre();
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int cur = ks & 1;
      if (ks + 1 < KS) {
        const int ch = ((2 * (ks + 1) + lh) ^ sw) * 8;
#pragma unroll
        for (int i = 0; i < TM; ++i)
          af[cur ^ 1][i] = *reinterpret_cast<const bf16x8_t *>(S + aoff[i] + ch);
#pragma unroll
        for (int j = 0; j < TN; ++j)
          bfr[cur ^ 1][j] = *reinterpret_cast<const bf16x8_t *>(S + boff[j] + ch);
      }
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = EPI ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[cur][j], af[cur][i], acc[i][j], 0, 0, 0)
                          : __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cur][i], bfr[cur][j], acc[i][j], 0, 0, 0);
    }
  };

  int kt = 0;
  // Steady state: STAGES - 2 younger tiles in flight at the wait, and the
  // tile STAGES - 1 ahead is issued every iteration.
  for (; kt + STAGES - 1 < nk; ++kt) {
    wait_vmcnt<(STAGES - 2) * (NA + NB)>();
    __builtin_amdgcn_s_barrier();
    run_tile(smem + (kt % STAGES) * SM::kStage,
             [&] { issue(kt + STAGES - 1, (kt + STAGES - 1) % STAGES); });
    if (SCHED) {
      // Spread the next k-steps' LDS reads and the DMA issue (address
      // arithmetic + global_load_lds) between the MFMAs of this k-tile.
      constexpr int NMF = KS * TM * TN;
      constexpr int NRD = (KS - 1) * (TM + TN);
      constexpr int NDMA = NA + NB;
#pragma unroll
      for (int q = 0; q < NMF; ++q) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                 // MFMA
        if (q < NRD) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);    // DS read
        if (q < NDMA) {
          __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);               // VALU
          __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);               // VMEM (DMA)
        }
      }
    }
  }
  // Drain: no more tiles to issue.
  for (; kt < nk; ++kt) {
    if (STAGES >= 3 && nk - 1 - kt >= 1) wait_vmcnt<(STAGES >= 3 ? 1 : 0) * (NA + NB)>();
    else wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    run_tile(smem + (kt % STAGES) * SM::kStage, [] {});
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
          o.x = f2bf(epilogue_act(v[0], a.relu, a.gelu)) | ((uint32_t)f2bf(epilogue_act(v[1], a.relu, a.gelu)) << 16);
          o.y = f2bf(epilogue_act(v[2], a.relu, a.gelu)) | ((uint32_t)f2bf(epilogue_act(v[3], a.relu, a.gelu)) << 16);
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
  constexpr int CPR = BN / 8;             // 8-column chunks per row
  constexpr int RPP = NT / CPR;           // rows per pass
  const int cc = t % CPR;
  const int n = n0 + cc * 8;
  if (n >= a.N) return;
  float bias[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) bias[e] = a.bias ? a.bias[n + e] : 0.0f;
  uint16_t *y = static_cast<uint16_t *>(a.y);
  const uint16_t *res = static_cast<const uint16_t *>(a.res);
#pragma unroll 4
  for (int rr = t / CPR; rr < BM; rr += RPP) {
    const int m = m0 + rr;
    if (m >= a.M) break;
    const float4 p = *reinterpret_cast<const float4 *>(Cs + rr * SM::kCPitch + cc * 8);
    const float4 q = *reinterpret_cast<const float4 *>(Cs + rr * SM::kCPitch + cc * 8 + 4);
    float v[8] = {p.x, p.y, p.z, p.w, q.x, q.y, q.z, q.w};
    if (res) {
      const uint4 rv = *reinterpret_cast<const uint4 *>(res + (int64_t)m * a.ldr + n);
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
      const float lo = epilogue_act(v[2 * e] + bias[2 * e], a.relu, a.gelu);
      const float hi = epilogue_act(v[2 * e + 1] + bias[2 * e + 1], a.relu, a.gelu);
      o[e] = f2bf(lo) | ((uint32_t)f2bf(hi) << 16);
    }
    *reinterpret_cast<uint4 *>(y + (int64_t)m * a.ldc + n) = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

template <int BM, int BN, int LD>
hipError_t launch_bf16_cfg(const ConvArgs &a, hipStream_t s) {
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  hipLaunchKernelGGL((conv_bf16_kernel<BM, BN, LD>), dim3(tiles), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, int STAGES, int LD, int SCHED = 1, int EPI = 0>
hipError_t launch_pipe_cfg(const ConvArgs &a, hipStream_t s) {
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  hipLaunchKernelGGL((conv_bf16_pipe_kernel<BM, BN, WM, WN, STAGES, LD, SCHED, EPI>), dim3(tiles),
                     dim3(WM * WN * 64), 0, s, a);
  return hipGetLastError();
}

// Tuning override: HAPI_CONV_CFG=<index> forces one tile configuration.
int forced_cfg() {
  static const int v = [] {
    const char *e = getenv("HAPI_CONV_CFG");
    return e ? atoi(e) : -1;
  }();
  return v;
}

// Tile shape per layer.  Every shape uses the same k-tile and MFMA, so the
// choice never changes a result bit.
template <int LD>
hipError_t launch_pipe_ld(const ConvArgs &a, hipStream_t s) {
  switch (forced_cfg()) {
    case 0: return launch_pipe_cfg<128, 128, 2, 2, 2, LD, 1, 0>(a, s);
    case 1: return launch_pipe_cfg<128, 64, 2, 2, 3, LD, 1, 0>(a, s);
    case 2: return launch_pipe_cfg<128, 128, 2, 2, 2, LD, 1, 1>(a, s);
    case 3: return launch_pipe_cfg<128, 64, 2, 2, 3, LD, 1, 1>(a, s);
    case 4: return launch_pipe_cfg<128, 64, 2, 2, 2, LD, 1, 1>(a, s);
    case 5: return launch_pipe_cfg<256, 128, 4, 2, 2, LD, 1, 1>(a, s);
    case 6: return launch_pipe_cfg<256, 256, 4, 2, 2, LD, 1, 1>(a, s);
    case 7: return launch_pipe_cfg<128, 256, 2, 4, 2, LD, 1, 1>(a, s);
    case 8: return launch_pipe_cfg<256, 128, 2, 2, 2, LD, 1, 1>(a, s);
    case 9: return launch_pipe_cfg<128, 128, 2, 2, 3, LD, 1, 1>(a, s);
    case 10: return launch_pipe_cfg<256, 64, 4, 1, 2, LD, 1, 1>(a, s);
    case 11: return launch_pipe_cfg<64, 128, 1, 4, 3, LD, 1, 1>(a, s);
    default: break;
  }
  // Measured on MI355X over the ResNet-50 conv shapes: two or three
  // workgroups per CU beat larger single-workgroup tiles for every shape; the
  // direct-store epilogue (48 KB of LDS, 3 workgroups per CU) wins only for
  // 64-channel outputs with long K.
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
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
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

  const int nk = a.Kp / BKF;
  load_tile(0);
  store_tile(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    if (kt + 1 < nk) load_tile(kt + 1);
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
    if (kt + 1 < nk) store_tile(cur ^ 1);
    __syncthreads();
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

template <int BM, int BN, int LD>
hipError_t launch_f32_cfg(const ConvArgs &a, hipStream_t s) {
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  hipLaunchKernelGGL((conv_f32_kernel<BM, BN, LD>), dim3(tiles), dim3(kThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_conv_bf16(const ConvArgs &a, Loader ld, hipStream_t s) {
  switch (ld) {
    // The pipelined kernel needs 16-byte output rows; the register-staged one
    // handles element gathers (NCHW stems) and any other width.
    case LD_NHWC:
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
  }
  return hipErrorInvalidValue;
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
