// Multi-head self-attention core for the ViT encoder on gfx950.
//
// Persistent workgroups of 8 waves, one per CU, each walking a range of
// (image, head) pairs.  A pair's keys (row-major) and values (transposed)
// sit in LDS, padded to a multiple of 32 tokens with zeros, in one of two
// buffers: while the waves compute pair i from one buffer, the keys and
// values of pair i + 1 are loaded into registers and written to the other
// after the compute, so the loads of one pair overlap the MFMAs of the last.
// Wave w takes the block of 32 queries starting at 32 w (7 blocks for 197
// tokens) and computes the transposed scores S^T = K Q^T with
// v_mfma_f32_32x32x16_bf16, so that every lane owns one query's scores: the
// softmax (fp32, max-subtracted, exp2 with the 1/sqrt(d) scale folded in)
// needs only in-lane work plus one exchange with the other half-wave.  The
// probabilities are rounded to bf16 and fed straight from the score registers
// into O^T = V^T P^T: the MFMA k-slots of lane half h hold the keys whose
// scores that lane already holds, and the V^T operand is read from LDS in the
// same key order, so no transpose of P through LDS is needed.  The query
// fragments of the next pair are loaded as soon as the scores no longer need
// the current ones.
#include "internal.h"

namespace hapi {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kAttnWaves = 8;

template <int TP>
__global__ __launch_bounds__(64 * kAttnWaves, 1) void attention_kernel(const uint16_t *__restrict__ qkv,
                                                                     uint16_t *__restrict__ out, int T, int D,
                                                                     int heads, int pairs, float scale_log2) {
  constexpr int DH = kHeadDim;       // 64
  constexpr int NT = TP / 32;        // key tiles (= query blocks)
  constexpr int KP = DH + 8;         // key row pitch (elements)
  constexpr int VP = TP + 8;         // transposed value row pitch
  static_assert(NT <= kAttnWaves, "one query block per wave");
  __shared__ __attribute__((aligned(16))) uint16_t Ks[2][TP * KP];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[2][DH * VP];

  const int ld = 3 * D;
  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int hl = lane >> 5, col = lane & 31;

  // Staging: thread t < 2 TP owns keys 4 (t / 8) .. + 3 x channels
  // 8 (t % 8) .. + 7 of the pair: 8 loads, then the key rows as they are and
  // the 4 x 8 value block transposed in registers, written as 8 rows of V^T.
  const bool stager = t < 2 * TP;
  const int kb = t >> 3, sc = t & 7;
  uint4 kv[4], vv[4];
  // Keys past T read key T - 1 and are zeroed when stored (a select): a
  // register zeroed before its load is issued makes the wave wait for every
  // load in flight first.
  auto stage_load = [&](int pair) {
    if (!stager) return;
    const int img = pair / heads, h = pair - img * heads;
    const uint16_t *base = qkv + (int64_t)img * T * ld;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int s = min(4 * kb + r, T - 1);
      kv[r] = *reinterpret_cast<const uint4 *>(base + (int64_t)s * ld + D + h * DH + sc * 8);
      vv[r] = *reinterpret_cast<const uint4 *>(base + (int64_t)s * ld + 2 * D + h * DH + sc * 8);
    }
  };
  auto stage_store = [&](int buf) {
    if (!stager) return;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const uint32_t keep = 4 * kb + r < T ? ~0u : 0u;
      kv[r] = make_uint4(kv[r].x & keep, kv[r].y & keep, kv[r].z & keep, kv[r].w & keep);
      vv[r] = make_uint4(vv[r].x & keep, vv[r].y & keep, vv[r].z & keep, vv[r].w & keep);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) *reinterpret_cast<uint4 *>(Ks[buf] + (4 * kb + r) * KP + sc * 8) = kv[r];
    auto half = [&](const uint4 &q, int e) -> uint32_t {
      const uint32_t w = (e >> 1) == 0 ? q.x : (e >> 1) == 1 ? q.y : (e >> 1) == 2 ? q.z : q.w;
      return (e & 1) ? (w >> 16) : (w & 0xffffu);
    };
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint2 o;
      o.x = half(vv[0], e) | (half(vv[1], e) << 16);
      o.y = half(vv[2], e) | (half(vv[3], e) << 16);
      *reinterpret_cast<uint2 *>(Vt[buf] + (sc * 8 + e) * VP + 4 * kb) = o;
    }
  };
  // This wave's query block: queries 32 wave .. + 31 (none past T).
  const int q = wave * 32 + col;
  const bool qblock = wave * 32 < T;
  bf16x8_t qf[DH / 16];
  // Query rows past T read query T - 1: their scores and outputs stay in
  // their own rows, which are never stored.
  auto load_q = [&](int pair) {
    const int img = pair / heads, h = pair - img * heads;
    const uint16_t *base = qkv + (int64_t)img * T * ld;
    const int qr = min(q, T - 1);
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks)
      qf[ks] = *reinterpret_cast<const bf16x8_t *>(base + (int64_t)qr * ld + h * DH + ks * 16 + hl * 8);
  };

  int p = blockIdx.x;
  if (p >= pairs) return;
  stage_load(p);
  if (qblock) load_q(p);
  stage_store(0);
  __syncthreads();
  for (int buf = 0; p < pairs; p += gridDim.x, buf ^= 1) {
    const int pn = p + gridDim.x;
    if (pn < pairs) stage_load(pn);  // in flight during this pair's compute
    if (qblock) {
      const uint16_t *K = Ks[buf], *V = Vt[buf];
      // s[t][r] = S^T[key 32t + 8(r/4) + 4hl + r%4][query col]; k-steps
      // outermost, so each step issues NT independent MFMAs (every tile still
      // accumulates its k-steps in order)
      f32x16_t s[NT];
#pragma unroll
      for (int tt = 0; tt < NT; ++tt)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[tt][r] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < DH / 16; ++ks) {
        bf16x8_t ka[NT];
#pragma unroll
        for (int tt = 0; tt < NT; ++tt)
          ka[tt] = *reinterpret_cast<const bf16x8_t *>(K + (32 * tt + col) * KP + ks * 16 + hl * 8);
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) s[tt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka[tt], qf[ks], s[tt], 0, 0, 0);
      }
      const int img = p / heads, h = p - img * heads;
      if (pn < pairs) load_q(pn);  // the scores no longer need this pair's queries
      // Only the last key tile can hold padding keys (TP is T rounded up to 32).
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int key = 32 * (NT - 1) + 8 * (r >> 2) + 4 * hl + (r & 3);
        if (key >= T) s[NT - 1][r] = -INFINITY;
      }
      float mx = -INFINITY;
#pragma unroll
      for (int tt = 0; tt < NT; ++tt)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[tt][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      float sum = 0.0f;
#pragma unroll
      for (int tt = 0; tt < NT; ++tt)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          // arguments are <= 0: the hardware exp2 (v_exp_f32) is exact enough
          const float pr = __builtin_amdgcn_exp2f((s[tt][r] - mx) * scale_log2);
          s[tt][r] = pr;
          sum += pr;
        }
      sum += __shfl_xor(sum, 32, 64);

      f32x16_t o[DH / 32];
#pragma unroll
      for (int db = 0; db < DH / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          // k-slot e of lane half hl <-> key 32t + 16j + 4hl + e (e < 4), + 8 + (e - 4) (e >= 4)
          bf16x8_t pb;
#pragma unroll
          for (int e = 0; e < 8; ++e) pb[e] = (__bf16)s[tt][8 * j + e];
          const int k0 = 32 * tt + 16 * j + 4 * hl;
#pragma unroll
          for (int db = 0; db < DH / 32; ++db) {
            const uint16_t *vr = V + (32 * db + col) * VP + k0;
            const uint2 lo = *reinterpret_cast<const uint2 *>(vr);
            const uint2 hi = *reinterpret_cast<const uint2 *>(vr + 8);
            uint4 pack = make_uint4(lo.x, lo.y, hi.x, hi.y);
            const bf16x8_t va = *reinterpret_cast<const bf16x8_t *>(&pack);
            o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o[db], 0, 0, 0);
          }
        }
      }
      if (q < T) {
        const float inv = 1.0f / sum;
        uint16_t *orow = out + ((int64_t)img * T + q) * D + h * DH;
#pragma unroll
        for (int db = 0; db < DH / 32; ++db)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int d0 = 32 * db + 8 * g + 4 * hl;
            uint2 w;
            w.x = f2bf2(o[db][4 * g] * inv, o[db][4 * g + 1] * inv);
            w.y = f2bf2(o[db][4 * g + 2] * inv, o[db][4 * g + 3] * inv);
            *reinterpret_cast<uint2 *>(orow + d0) = w;
          }
      }
    }
    // The other buffer: last read before the previous barrier.
    if (pn < pairs) stage_store(buf ^ 1);
    __syncthreads();
  }
}

template <int TP>
hipError_t launch_tp(const void *qkv, void *out, int n, int T, int D, int heads, hipStream_t s) {
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)kHeadDim);
  const int pairs = n * heads, cus = cu_count();
  hapi_launch(attention_kernel<TP>, dim3(pairs < cus ? pairs : cus), dim3(64 * kAttnWaves), 0, s,
              (const uint16_t *)qkv, (uint16_t *)out, T, D, heads, pairs, scale_log2);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const void *qkv, void *out, int n, int T, int D, int heads,
                            hipStream_t s) {
  const int tp = (T + 31) / 32 * 32;
  switch (tp) {
    case 32: return launch_tp<32>(qkv, out, n, T, D, heads, s);
    case 64: return launch_tp<64>(qkv, out, n, T, D, heads, s);
    case 96: return launch_tp<96>(qkv, out, n, T, D, heads, s);
    case 128: return launch_tp<128>(qkv, out, n, T, D, heads, s);
    case 160: return launch_tp<160>(qkv, out, n, T, D, heads, s);
    case 192: return launch_tp<192>(qkv, out, n, T, D, heads, s);
    case 224: return launch_tp<224>(qkv, out, n, T, D, heads, s);
    case 256: return launch_tp<256>(qkv, out, n, T, D, heads, s);
    default: break;
  }
  return hipErrorInvalidValue;
}

}  // namespace hapi
