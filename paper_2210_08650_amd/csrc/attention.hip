// Multi-head self-attention core for the ViT encoder on gfx950.
//
// One workgroup per (image, head); the head's keys (row-major) and values
// (transposed) sit in LDS, padded to a multiple of 32 tokens with zeros.
// Each wave takes blocks of 32 queries and computes the transposed scores
// S^T = K Q^T with v_mfma_f32_32x32x16_bf16, so that every lane owns one
// query's scores: the softmax (fp32, max-subtracted, exp2 with the 1/sqrt(d)
// scale folded in) needs only in-lane work plus one exchange with the other
// half-wave.  The probabilities are rounded to bf16 and fed straight from the
// score registers into O^T = V^T P^T: the MFMA k-slots of lane half h hold the
// keys whose scores that lane already holds, and the V^T operand is read from
// LDS in the same key order, so no transpose of P through LDS is needed.
#include "internal.h"

namespace hapi {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));


template <int TP>
__global__ __launch_bounds__(256, 2) void attention_kernel(const uint16_t *__restrict__ qkv,
                                                        uint16_t *__restrict__ out, int T, int D,
                                                        int heads, float scale_log2) {
  constexpr int DH = kHeadDim;       // 64
  constexpr int NT = TP / 32;        // key tiles
  constexpr int KP = DH + 8;         // key row pitch (elements)
  constexpr int VP = TP + 8;         // transposed value row pitch
  __shared__ __attribute__((aligned(16))) uint16_t Ks[TP * KP];
  __shared__ __attribute__((aligned(16))) uint16_t Vt[DH * VP];

  const int img = blockIdx.x / heads, h = blockIdx.x % heads;
  const int ld = 3 * D;
  const uint16_t *base = qkv + (int64_t)img * T * ld;

  // Staging: thread t < TP owns 8 keys (8 (t / 8) ..) x 8 channels (8 (t % 8) ..):
  // all 16 loads first, then the key rows as they are and the 8 x 8 value
  // block transposed in registers, written as 8 rows of V^T with 16-byte stores.
  static_assert(TP <= 256, "one 8 x 8 block per thread");
  if (threadIdx.x < TP) {
    const int kb = threadIdx.x >> 3, c = threadIdx.x & 7;
    uint4 kv[8], vv[8];
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      const int s = 8 * kb + r;
      kv[r] = vv[r] = make_uint4(0, 0, 0, 0);
      if (s < T) {
        kv[r] = *reinterpret_cast<const uint4 *>(base + (int64_t)s * ld + D + h * DH + c * 8);
        vv[r] = *reinterpret_cast<const uint4 *>(base + (int64_t)s * ld + 2 * D + h * DH + c * 8);
      }
    }
#pragma unroll
    for (int r = 0; r < 8; ++r) *reinterpret_cast<uint4 *>(Ks + (8 * kb + r) * KP + c * 8) = kv[r];
    auto half = [&](const uint4 &q, int e) -> uint32_t {
      const uint32_t w = (e >> 1) == 0 ? q.x : (e >> 1) == 1 ? q.y : (e >> 1) == 2 ? q.z : q.w;
      return (e & 1) ? (w >> 16) : (w & 0xffffu);
    };
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint4 o;
      o.x = half(vv[0], e) | (half(vv[1], e) << 16);
      o.y = half(vv[2], e) | (half(vv[3], e) << 16);
      o.z = half(vv[4], e) | (half(vv[5], e) << 16);
      o.w = half(vv[6], e) | (half(vv[7], e) << 16);
      *reinterpret_cast<uint4 *>(Vt + (c * 8 + e) * VP + 8 * kb) = o;
    }
  }
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int hl = lane >> 5, col = lane & 31;

  for (int qb = wave; qb * 32 < T; qb += 4) {
    const int q = qb * 32 + col;
    bf16x8_t qf[DH / 16];
#pragma unroll
    for (int ks = 0; ks < DH / 16; ++ks) {
      if (q < T) {
        qf[ks] = *reinterpret_cast<const bf16x8_t *>(base + (int64_t)q * ld + h * DH + ks * 16 + hl * 8);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) qf[ks][e] = (__bf16)0.0f;
      }
    }
    // s[t][r] = S^T[key 32t + 8(r/4) + 4hl + r%4][query col]
    f32x16_t s[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
      for (int r = 0; r < 16; ++r) s[t][r] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < DH / 16; ++ks) {
        const bf16x8_t ka = *reinterpret_cast<const bf16x8_t *>(Ks + (32 * t + col) * KP + ks * 16 + hl * 8);
        s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[ks], s[t], 0, 0, 0);
      }
      // one key tile's fragments live at a time (keeps two waves per SIMD)
      __builtin_amdgcn_sched_barrier(0);
    }
    // Only the last key tile can hold padding keys (TP is T rounded up to 32).
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = 32 * (NT - 1) + 8 * (r >> 2) + 4 * hl + (r & 3);
      if (key >= T) s[NT - 1][r] = -INFINITY;
    }
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[t][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float sum = 0.0f;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        // arguments are <= 0: the hardware exp2 (v_exp_f32) is exact enough
        const float p = __builtin_amdgcn_exp2f((s[t][r] - mx) * scale_log2);
        s[t][r] = p;
        sum += p;
      }
    sum += __shfl_xor(sum, 32, 64);

    f32x16_t o[DH / 32];
#pragma unroll
    for (int db = 0; db < DH / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) o[db][r] = 0.0f;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        // k-slot e of lane half hl <-> key 32t + 16j + 4hl + e (e < 4), + 8 + (e - 4) (e >= 4)
        bf16x8_t pb;
#pragma unroll
        for (int e = 0; e < 8; ++e) pb[e] = (__bf16)s[t][8 * j + e];
        const int k0 = 32 * t + 16 * j + 4 * hl;
#pragma unroll
        for (int db = 0; db < DH / 32; ++db) {
          const uint16_t *vr = Vt + (32 * db + col) * VP + k0;
          const uint2 lo = *reinterpret_cast<const uint2 *>(vr);
          const uint2 hi = *reinterpret_cast<const uint2 *>(vr + 8);
          uint4 pack = make_uint4(lo.x, lo.y, hi.x, hi.y);
          const bf16x8_t va = *reinterpret_cast<const bf16x8_t *>(&pack);
          o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, o[db], 0, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
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
}

template <int TP>
hipError_t launch_tp(const void *qkv, void *out, int n, int T, int D, int heads, hipStream_t s) {
  const float scale_log2 = 1.4426950408889634f / sqrtf((float)kHeadDim);
  hapi_launch(attention_kernel<TP>, dim3(n * heads), dim3(256), 0, s,
                     (const uint16_t *)qkv, (uint16_t *)out, T, D, heads, scale_log2);
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
