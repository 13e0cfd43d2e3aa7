// Host runtime of libhapi: descriptor validation and shape calculus, weight
// layout and packing, the chunked (storage-side batch) executor, per-layer
// profiling and per-kernel timing.  Entry points are declared in hapi.h.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"

namespace hapi {

// ------------------------------------------------------------------ errors

thread_local std::string g_err;

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

namespace {

#define HIP_TRY(expr)                                                                  \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail(HAPI_E_DEVICE, "%s failed: %s", #expr, hipGetErrorString(e_));       \
  } while (0)

// ------------------------------------------------------------------ model

constexpr int64_t kAlign = 256;
constexpr int64_t kIndexLimit = (int64_t)1 << 31;  // kernels index a partition with int32
constexpr int kAutoChunk = 256;
constexpr int kMaxInflight = 4;
constexpr int kAutoInflightBatch = 128;

int64_t align_up(int64_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Act {  // per-image activation, stored NHWC (tokens: h = T, w = 1, c = D)
  int c = 0, h = 0, w = 0;
  bool tok = false;
  int64_t elems() const { return (int64_t)c * h * w; }
};

struct ConvSpec {
  int cin, cout, k, stride, pad;
  bool bias, bn;
  bool s2d;  // stride-2 stem on 2x2 space-to-depth cells (first layer, few channels)
  bool nhwc8; // first layer over <= 8 channels, 9..16 taps: NHWC with 8 channel slots,
              // k = (tap, slot), two k-tiles of 8 taps
  int K, Kp;
  int64_t raw_w, raw_b, raw_bn;  // float offsets into the raw buffer (-1: absent)
  int64_t pk_w, pk_b;            // byte offsets into the packed buffer
  // A residual block's last convolution fused with its projection shortcut:
  // one GEMM over K = K1 (this convolution) + cin2 (1x1, stride stride2, on the
  // block input); both batch-norms folded, biases summed.
  bool fused;
  int K1, cin2, stride2;
  int64_t raw_w2, raw_bn2;
  int splits;  // fp32 CONV layers: reduction slices (see f32_splits); else 1
};

struct Extra {  // float32 parameters: copied verbatim (tokens, layernorm), or an
               // inference batch-norm [g|b|m|v] packed as scale[n], shift[n]
  int64_t raw, pk, n;
  bool bn_affine;
};

struct LayerPlan {
  hapi_layer L;
  Act in, out;
  std::vector<ConvSpec> convs;
  std::vector<Extra> extras;
  bool has_sc = false;
  int64_t tmp_elems = 0;  // largest per-image tensor the layer reads or writes
  int64_t part_elems = 0; // per-image fp32 partial sums of a split reduction
  int64_t pk_end = 0;     // packed-weight bytes of layers 1..this one
};

struct Model {
  bool bf16 = true;
  int esz = 2;
  Act input;
  std::vector<LayerPlan> layers;
  int64_t raw_count = 0, packed_bytes = 0;
  bool first_reads_nchw = false;
};

int conv_out(int x, int k, int s, int p) { return (x + 2 * p - k) / s + 1; }

int analyze(const hapi_model_desc *d, Model &m) {
  if (!d) return fail(HAPI_E_INVAL, "desc is NULL");
  if (d->n_layers < 1 || !d->layers) return fail(HAPI_E_INVAL, "desc has no layers");
  if (d->dtype != HAPI_F32 && d->dtype != HAPI_BF16)
    return fail(HAPI_E_INVAL, "unknown dtype %d", d->dtype);
  if (d->in_c < 1 || d->in_h < 1 || d->in_w < 1)
    return fail(HAPI_E_INVAL, "bad input shape %dx%dx%d", d->in_c, d->in_h, d->in_w);
  if (d->chunk < 0) return fail(HAPI_E_INVAL, "chunk must be >= 0");
  if (d->inflight < 0 || d->inflight > kMaxInflight)
    return fail(HAPI_E_INVAL, "inflight must be in [0, %d]", kMaxInflight);
  if (d->direct != 0 && d->direct != 1) return fail(HAPI_E_INVAL, "direct must be 0 or 1");
  m = Model();
  m.bf16 = d->dtype == HAPI_BF16;
  m.esz = m.bf16 ? 2 : 4;
  m.input = Act{d->in_c, d->in_h, d->in_w, false};
  const int kq = m.bf16 ? 64 : 16;  // k-tile of the conv kernels
  Act cur = m.input;
  int64_t raw = 0, pk = 0;

  auto add_conv = [&](LayerPlan &lp, int cin, int cout, int k, int s, int p, bool bias, bool bn,
                      bool s2d = false, bool nhwc8 = false) {
    ConvSpec c{};
    c.cin = cin; c.cout = cout; c.k = k; c.stride = s; c.pad = p; c.bias = bias; c.bn = bn;
    c.s2d = s2d;
    c.nhwc8 = nhwc8;
    c.splits = 1;
    c.K = s2d ? ((k + 1) / 2) * ((k + 1) / 2) * kS2DChannels : nhwc8 ? 16 * 8 : cin * k * k;
    c.Kp = (c.K + kq - 1) / kq * kq;
    c.raw_w = raw; raw += (int64_t)cout * cin * k * k;
    c.raw_b = -1; c.raw_bn = -1;
    if (bias) { c.raw_b = raw; raw += cout; }
    if (bn) { c.raw_bn = raw; raw += 4 * (int64_t)cout; }
    c.pk_w = pk; pk = align_up(pk + (int64_t)cout * c.Kp * m.esz);
    c.pk_b = pk; pk = align_up(pk + (int64_t)cout * 4);
    lp.convs.push_back(c);
  };
  auto add_fused = [&](LayerPlan &lp, int cin1, int cout, int k, int pad, int cin2, int s2) {
    ConvSpec c{};
    c.cin = cin1; c.cout = cout; c.k = k; c.stride = 1; c.pad = pad; c.bn = true;
    c.fused = true;
    c.K1 = cin1 * k * k; c.cin2 = cin2; c.stride2 = s2;
    c.K = c.Kp = c.K1 + cin2;
    c.raw_b = -1;
    c.raw_w = raw; raw += (int64_t)cout * c.K1;
    c.raw_bn = raw; raw += 4 * (int64_t)cout;
    c.raw_w2 = raw; raw += (int64_t)cout * cin2;
    c.raw_bn2 = raw; raw += 4 * (int64_t)cout;
    c.pk_w = pk; pk = align_up(pk + (int64_t)cout * c.Kp * m.esz);
    c.pk_b = pk; pk = align_up(pk + (int64_t)cout * 4);
    lp.convs.push_back(c);
  };
  auto add_extra = [&](LayerPlan &lp, int64_t n) {
    lp.extras.push_back(Extra{raw, pk, n, false});
    raw += n;
    pk = align_up(pk + n * 4);
  };
  auto add_bn_affine = [&](LayerPlan &lp, int64_t c) {
    lp.extras.push_back(Extra{raw, pk, c, true});
    raw += 4 * c;
    pk = align_up(pk + 2 * c * 4);
  };
  // NHWC-input convolutions need whole 16-byte chunks of channels per k-tile.
  auto nhwc_ok = [&](int cin) { return cin % kq == 0; };

  for (int li = 0; li < d->n_layers; ++li) {
    const hapi_layer &L = d->layers[li];
    LayerPlan lp;
    lp.L = L;
    lp.in = cur;
    for (int r = 0; r < 4; ++r)
      if (L.reserved[r]) return fail(HAPI_E_INVAL, "layer %d: reserved fields must be 0", li + 1);
    const bool first = li == 0;
    switch (L.kind) {
      case HAPI_CONV: {
        if (cur.tok) return fail(HAPI_E_INVAL, "layer %d: CONV on token input", li + 1);
        if (L.cin != cur.c) return fail(HAPI_E_INVAL, "layer %d: cin %d != input channels %d", li + 1, L.cin, cur.c);
        if (L.cout < 1 || L.k < 1 || L.stride < 1 || L.pad < 0 || L.pad >= L.k)
          return fail(HAPI_E_INVAL, "layer %d: bad conv geometry", li + 1);
        const int ho = conv_out(cur.h, L.k, L.stride, L.pad), wo = conv_out(cur.w, L.k, L.stride, L.pad);
        if (ho < 1 || wo < 1) return fail(HAPI_E_INVAL, "layer %d: empty conv output", li + 1);
        if (!first && !nhwc_ok(L.cin))
          return fail(HAPI_E_UNSUPPORTED, "layer %d: conv with cin %% %d != 0 after the first layer", li + 1, kq);
        // A stride-2 first layer over <= 4 channels whose receptive field spans
        // 4 x 4 cells of 2 x 2 pixels runs on the space-to-depth layout.
        const bool s2d = first && m.bf16 && L.stride == 2 && L.cin <= 4 && (L.k + 1) / 2 == 4 &&
                         L.cout % 8 == 0;
        // Any other first layer over <= 8 channels with 9..16 taps (VGG's 3 x 3
        // over RGB) reads an NHWC copy of its input with 8 channel slots.
        const bool nhwc8 = first && m.bf16 && !s2d && L.cin <= 8 && L.k * L.k > 8 && L.k * L.k <= 16 &&
                           L.cout % 8 == 0;
        add_conv(lp, L.cin, L.cout, L.k, L.stride, L.pad, L.has_bias != 0, L.has_bn != 0, s2d, nhwc8);
        lp.out = Act{L.cout, ho, wo, false};
        if (s2d) lp.tmp_elems = (int64_t)(ho + 3) * (wo + 3) * kS2DChannels;
        if (nhwc8) lp.tmp_elems = (int64_t)cur.h * cur.w * 8;
        if (!m.bf16 && L.cout % 4 == 0) {
          // fp32: long reductions run as slices (the slice count depends on K
          // only, so results do not depend on the batch or its partitions)
          ConvSpec &cs = lp.convs.back();
          cs.splits = f32_splits(cs.Kp);
          if (cs.splits > 1) lp.part_elems = (int64_t)cs.splits * ho * wo * L.cout;
        }
        if (first) m.first_reads_nchw = true;
        break;
      }
      case HAPI_MAXPOOL:
      case HAPI_AVGPOOL: {
        if (cur.tok) return fail(HAPI_E_INVAL, "layer %d: pooling on token input", li + 1);
        if (L.kind == HAPI_AVGPOOL && L.k == 0) {
          lp.out = Act{cur.c, 1, 1, false};
          break;
        }
        if (L.k < 1 || L.stride < 1 || L.pad < 0 || 2 * L.pad > L.k)
          return fail(HAPI_E_INVAL, "layer %d: bad pooling geometry", li + 1);
        if (L.kind == HAPI_AVGPOOL && L.pad != 0)
          return fail(HAPI_E_UNSUPPORTED, "layer %d: padded average pooling", li + 1);
        if (L.kind == HAPI_MAXPOOL && cur.c % 8 != 0)
          return fail(HAPI_E_UNSUPPORTED, "layer %d: max pooling needs channels %% 8 == 0", li + 1);
        const int ho = conv_out(cur.h, L.k, L.stride, L.pad), wo = conv_out(cur.w, L.k, L.stride, L.pad);
        if (ho < 1 || wo < 1) return fail(HAPI_E_INVAL, "layer %d: empty pooling output", li + 1);
        lp.out = Act{cur.c, ho, wo, false};
        break;
      }
      case HAPI_BASIC_BLOCK:
      case HAPI_BOTTLENECK: {
        if (cur.tok) return fail(HAPI_E_INVAL, "layer %d: residual block on token input", li + 1);
        if (L.cin != cur.c) return fail(HAPI_E_INVAL, "layer %d: cin %d != input channels %d", li + 1, L.cin, cur.c);
        if (L.stride < 1) return fail(HAPI_E_INVAL, "layer %d: stride must be >= 1", li + 1);
        const bool basic = L.kind == HAPI_BASIC_BLOCK;
        const int width = basic ? L.cout : L.width;
        const int cout = basic ? L.cout : 4 * L.width;
        if (width < 1) return fail(HAPI_E_INVAL, "layer %d: bad block width", li + 1);
        if (!basic && L.cout != 0 && L.cout != cout)
          return fail(HAPI_E_INVAL, "layer %d: bottleneck cout must be 4 * width", li + 1);
        if (!nhwc_ok(L.cin) || !nhwc_ok(width) || !nhwc_ok(cout))
          return fail(HAPI_E_UNSUPPORTED, "layer %d: block channels must be multiples of %d", li + 1, kq);
        const int ho = conv_out(cur.h, 3, L.stride, 1), wo = conv_out(cur.w, 3, L.stride, 1);
        if (ho < 1 || wo < 1) return fail(HAPI_E_INVAL, "layer %d: empty block output", li + 1);
        lp.has_sc = L.stride != 1 || L.cin != cout;
        // bf16: the projection shortcut joins the last convolution's GEMM when
        // both K parts are whole 64-wide k-tiles of NHWC channels
        const bool fuse = lp.has_sc && m.bf16 && L.cin % 64 == 0 &&
                          (basic ? cout : width) % 64 == 0 && cout % 8 == 0;
        if (basic) {
          add_conv(lp, L.cin, cout, 3, L.stride, 1, false, true);
          if (fuse) add_fused(lp, cout, cout, 3, 1, L.cin, L.stride);
          else add_conv(lp, cout, cout, 3, 1, 1, false, true);
        } else {
          add_conv(lp, L.cin, width, 1, 1, 0, false, true);
          add_conv(lp, width, width, 3, L.stride, 1, false, true);
          if (fuse) add_fused(lp, width, cout, 1, 0, L.cin, L.stride);
          else add_conv(lp, width, cout, 1, 1, 0, false, true);
        }
        if (lp.has_sc && !fuse) add_conv(lp, L.cin, cout, 1, L.stride, 0, false, true);
        lp.out = Act{cout, ho, wo, false};
        lp.tmp_elems = std::max<int64_t>(lp.tmp_elems, (int64_t)width * cur.h * cur.w);
        lp.tmp_elems = std::max<int64_t>(lp.tmp_elems, (int64_t)width * ho * wo);
        break;
      }
      case HAPI_PATCH_EMBED: {
        if (!m.bf16) return fail(HAPI_E_UNSUPPORTED, "layer %d: PATCH_EMBED needs bf16", li + 1);
        if (cur.tok || L.cin != cur.c) return fail(HAPI_E_INVAL, "layer %d: bad PATCH_EMBED input", li + 1);
        if (L.k < 1 || (L.stride != 0 && L.stride != L.k) || L.pad != 0 || L.cout < 1)
          return fail(HAPI_E_INVAL, "layer %d: bad patch geometry", li + 1);
        if (!first && !nhwc_ok(L.cin))
          return fail(HAPI_E_UNSUPPORTED, "layer %d: PATCH_EMBED after the first layer needs cin %% 64 == 0", li + 1);
        const int ho = cur.h / L.k, wo = cur.w / L.k;
        if (ho < 1 || wo < 1) return fail(HAPI_E_INVAL, "layer %d: image smaller than a patch", li + 1);
        add_conv(lp, L.cin, L.cout, L.k, L.k, 0, true, false);
        lp.out = Act{L.cout, ho, wo, false};
        if (first) m.first_reads_nchw = true;
        break;
      }
      case HAPI_TOKENS: {
        if (!m.bf16) return fail(HAPI_E_UNSUPPORTED, "layer %d: TOKENS needs bf16", li + 1);
        if (cur.tok || L.cout != cur.c) return fail(HAPI_E_INVAL, "layer %d: TOKENS width mismatch", li + 1);
        if (L.cout % 8 != 0) return fail(HAPI_E_UNSUPPORTED, "layer %d: TOKENS width %% 8 != 0", li + 1);
        const int T = 1 + cur.h * cur.w;
        add_extra(lp, L.cout);
        add_extra(lp, (int64_t)T * L.cout);
        lp.out = Act{L.cout, T, 1, true};
        break;
      }
      case HAPI_VIT_BLOCK: {
        if (!m.bf16) return fail(HAPI_E_UNSUPPORTED, "layer %d: VIT_BLOCK needs bf16", li + 1);
        const int D = L.cout;
        if (!cur.tok || D != cur.c) return fail(HAPI_E_INVAL, "layer %d: VIT_BLOCK input mismatch", li + 1);
        if (L.heads < 1 || D % L.heads != 0 || L.mlp_dim < 1)
          return fail(HAPI_E_INVAL, "layer %d: bad heads / mlp_dim", li + 1);
        if (D / L.heads != kHeadDim)
          return fail(HAPI_E_UNSUPPORTED, "layer %d: head dim %d (only %d built)", li + 1, D / L.heads, kHeadDim);
        if (D % 64 != 0 || L.mlp_dim % 64 != 0)
          return fail(HAPI_E_UNSUPPORTED, "layer %d: width and mlp_dim must be multiples of 64", li + 1);
        if (cur.h > kAttnMaxTokens)
          return fail(HAPI_E_UNSUPPORTED, "layer %d: %d tokens (at most %d)", li + 1, cur.h, kAttnMaxTokens);
        add_extra(lp, D);  // ln1 gamma
        add_extra(lp, D);  // ln1 beta
        add_conv(lp, D, 3 * D, 1, 1, 0, true, false);  // in-projection
        add_conv(lp, D, D, 1, 1, 0, true, false);      // out-projection
        add_extra(lp, D);  // ln2 gamma
        add_extra(lp, D);  // ln2 beta
        add_conv(lp, D, L.mlp_dim, 1, 1, 0, true, false);  // fc1
        add_conv(lp, L.mlp_dim, D, 1, 1, 0, true, false);  // fc2
        lp.out = cur;
        lp.tmp_elems = (int64_t)cur.h * std::max(3 * D, L.mlp_dim);
        break;
      }
      case HAPI_LAYERNORM: {
        if (!m.bf16) return fail(HAPI_E_UNSUPPORTED, "layer %d: LAYERNORM needs bf16", li + 1);
        if (!cur.tok || L.cout != cur.c) return fail(HAPI_E_INVAL, "layer %d: LAYERNORM input mismatch", li + 1);
        if (L.cout % 8 != 0 || L.cout > 2048)
          return fail(HAPI_E_UNSUPPORTED, "layer %d: LAYERNORM width must be a multiple of 8, <= 2048", li + 1);
        add_extra(lp, L.cout);
        add_extra(lp, L.cout);
        lp.out = cur;
        break;
      }
      case HAPI_PREACT_CONV: {
        if (!m.bf16) return fail(HAPI_E_UNSUPPORTED, "layer %d: PREACT_CONV needs bf16", li + 1);
        if (cur.tok || L.cin != cur.c)
          return fail(HAPI_E_INVAL, "layer %d: PREACT_CONV input mismatch", li + 1);
        if (L.k < 1 || L.stride < 1 || L.pad < 0 || L.cout < 1)
          return fail(HAPI_E_INVAL, "layer %d: bad conv geometry", li + 1);
        if (first || !nhwc_ok(L.cin))
          return fail(HAPI_E_UNSUPPORTED, "layer %d: PREACT_CONV needs cin %% %d == 0 after the first layer",
                      li + 1, kq);
        const int ho = conv_out(cur.h, L.k, L.stride, L.pad), wo = conv_out(cur.w, L.k, L.stride, L.pad);
        if (ho < 1 || wo < 1) return fail(HAPI_E_INVAL, "layer %d: empty conv output", li + 1);
        add_bn_affine(lp, L.cin);
        add_conv(lp, L.cin, L.cout, L.k, L.stride, L.pad, false, false);
        lp.out = Act{L.cout, ho, wo, false};
        break;
      }
      case HAPI_BATCHNORM: {
        if (!m.bf16) return fail(HAPI_E_UNSUPPORTED, "layer %d: BATCHNORM needs bf16", li + 1);
        if (cur.tok || L.cout != cur.c) return fail(HAPI_E_INVAL, "layer %d: BATCHNORM input mismatch", li + 1);
        if (L.cout % 8 != 0) return fail(HAPI_E_UNSUPPORTED, "layer %d: BATCHNORM needs channels %% 8 == 0", li + 1);
        add_bn_affine(lp, L.cout);
        lp.out = cur;
        break;
      }
      case HAPI_DENSE_BLOCK: {
        if (!m.bf16) return fail(HAPI_E_UNSUPPORTED, "layer %d: DENSE_BLOCK needs bf16", li + 1);
        if (cur.tok || L.cin != cur.c) return fail(HAPI_E_INVAL, "layer %d: DENSE_BLOCK input mismatch", li + 1);
        const int growth = L.width, bott = L.mlp_dim;
        if (growth < 1 || bott < 1 || L.cout <= L.cin || (L.cout - L.cin) % growth != 0)
          return fail(HAPI_E_INVAL, "layer %d: bad dense block (cin %d, cout %d, growth %d)", li + 1,
                      L.cin, L.cout, growth);
        if (L.cin % 8 != 0 || growth % 8 != 0 || bott % 64 != 0)
          return fail(HAPI_E_UNSUPPORTED,
                      "layer %d: dense block needs cin, growth %% 8 == 0 and bottleneck %% 64 == 0", li + 1);
        for (int c = L.cin; c < L.cout; c += growth) {
          add_bn_affine(lp, c);
          add_conv(lp, c, bott, 1, 1, 0, false, true);
          add_conv(lp, bott, growth, 3, 1, 1, false, false);
        }
        lp.out = Act{L.cout, cur.h, cur.w, false};
        lp.tmp_elems = (int64_t)std::max(L.cout, bott) * cur.h * cur.w;
        break;
      }
      default:
        return fail(HAPI_E_INVAL, "layer %d: unknown kind %d", li + 1, L.kind);
    }
    if (first && !m.first_reads_nchw && m.input.c % 8 != 0 && L.kind == HAPI_MAXPOOL)
      return fail(HAPI_E_UNSUPPORTED, "layer 1: max pooling needs channels %% 8 == 0");
    lp.tmp_elems = std::max({lp.tmp_elems, lp.in.elems(), lp.out.elems()});
    lp.pk_end = pk;
    m.layers.push_back(lp);
    cur = lp.out;
  }
  m.raw_count = raw;
  m.packed_bytes = pk;
  return HAPI_OK;
}

int64_t max_tmp(const Model &m, int split) {
  int64_t t = m.first_reads_nchw ? 0 : m.input.elems();
  for (int i = 0; i < split; ++i) t = std::max(t, m.layers[i].tmp_elems);
  return t;
}

// Partitions in flight at once: the caller's choice, else two for a large
// batch split automatically (one partition alone leaves each layer's ramp and
// tail idle, and memory-bound layers of one partition overlap compute-bound
// layers of the other), else one -- an explicit storage-side batch keeps the
// paper's sequential partitions.
int inflight_for(const hapi_model_desc *d, int batch) {
  if (d->inflight > 0) return std::min(d->inflight, kMaxInflight);
  return (d->chunk == 0 && batch >= kAutoInflightBatch) ? 2 : 1;
}

int64_t max_part(const Model &m, int split) {
  int64_t p = 0;
  for (int i = 0; i < split; ++i) p = std::max(p, m.layers[i].part_elems);
  return p;
}

int chunk_for(const hapi_model_desc *d, const Model &m, int batch) {
  const int lanes = inflight_for(d, batch);
  int c = d->chunk > 0 ? std::min(d->chunk, batch)
                       : std::min((batch + lanes - 1) / lanes, kAutoChunk);
  if (d->chunk == 0) {
    const int64_t per = std::max<int64_t>(1, max_tmp(m, (int)m.layers.size()));
    const int64_t lim = (kIndexLimit - 1) / per;
    c = (int)std::max<int64_t>(1, std::min<int64_t>(c, lim));
  }
  return c;
}

int64_t slot_bytes(const Model &m, int split, int chunk) {
  return align_up((int64_t)chunk * max_tmp(m, split) * m.esz);
}

// Streams a batch actually uses: no more than it has partitions.
int lanes_for(const hapi_model_desc *d, int chunk, int batch) {
  return std::max(1, std::min(inflight_for(d, batch), (batch + chunk - 1) / chunk));
}

// Bytes of one lane's fp32 partial-sum region.
int64_t part_bytes(const Model &m, int split, int chunk) {
  return align_up((int64_t)chunk * max_part(m, split) * 4);
}

// Workspace of one partition in flight: three activation slots and the
// partial-sum region, each followed by a guard gap of kGuardBytes that no
// kernel writes (a write past a region's end lands in its gap, where a check
// of the gap's contents sees it instead of it corrupting the next region).
constexpr int64_t kGuardBytes = 4096;
struct LaneLayout {
  int64_t slot[3], part, bytes;
  int64_t guard[4];
};
LaneLayout lane_layout(const Model &m, int split, int chunk) {
  LaneLayout L;
  const int64_t sb = slot_bytes(m, split, chunk);
  int64_t o = 0;
  for (int i = 0; i < 3; ++i) {
    L.slot[i] = o;
    L.guard[i] = o + sb;
    o += sb + kGuardBytes;
  }
  L.part = o;
  L.guard[3] = o + part_bytes(m, split, chunk);
  L.bytes = L.guard[3] + kGuardBytes;
  return L;
}

// One lane layout per partition in flight (profiling runs one), then for
// profiling the synthetic packed weights and images.
int64_t workspace_for(const Model &m, int split, int chunk, bool profile, int batch, int lanes) {
  int64_t b = split > 0 ? (profile ? 1 : lanes) * lane_layout(m, split, chunk).bytes : 0;
  if (profile) b += align_up(m.packed_bytes) + align_up((int64_t)batch * m.input.elems() * m.esz);
  return b;
}

// ------------------------------------------------------------- kernel stats

}  // namespace

LaunchEvents &launch_events() {
  static thread_local LaunchEvents e;
  return e;
}

namespace {

enum Family { F_CONV_BF16, F_CONV_F32, F_ATTN, F_LN, F_MAXPOOL, F_AVGPOOL, F_TOKENS, F_LAYOUT,
              F_COPY, F_AFFINE, F_SPLIT_SUM, F_COUNT };
const char *kFamily[F_COUNT] = {"conv_bf16", "conv_f32", "attention", "layernorm", "maxpool",
                                "avgpool", "tokens", "layout", "copy", "affine_relu", "split_sum"};

struct StatRec {
  int fam;
  hipEvent_t a, b;
  double flops, bytes;
};

std::mutex g_stats_mu;
bool g_stats_on = false;
std::vector<StatRec> g_recs;
std::vector<hipEvent_t> g_pool;

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

template <class F>
hipError_t timed(hipStream_t s, int fam, double flops, double bytes, F &&launch) {
  if (!g_stats_on) return launch();
  (void)s;
  std::lock_guard<std::mutex> g(g_stats_mu);
  hipEvent_t a = take_event(), b = take_event();
  // The launch records a and b as part of its dispatch (hapi_launch).
  if (a && b) launch_events() = LaunchEvents{a, b};
  hipError_t r = launch();
  const bool used = launch_events().start == nullptr;
  launch_events() = LaunchEvents{};
  if (a && b && used && r == hipSuccess) {
    g_recs.push_back(StatRec{fam, a, b, flops, bytes});
  } else {
    if (a) g_pool.push_back(a);
    if (b) g_pool.push_back(b);
  }
  return r;
}

// ------------------------------------------------------------------ executor

struct Ctx {
  const Model &m;
  hipStream_t s;
  const uint8_t *pk;
  uint8_t *slot[3];
  std::function<void(int, bool)> on_layer;  // (layer index, begin) for profiling
  int cus;      // workgroups of persistent kernels
  float *part;  // fp32 partial sums of split reductions
  int lanes;    // partitions in flight
  mutable int seq = 0;  // convolutions issued in this partition
};

// Per-channel scale and shift (an inference batch-norm) that a 1 x 1
// convolution applies with ReLU to its input as it reads it; lda: the input's
// row stride when it is a channel prefix of a wider tensor.
struct PreAct {
  const float *scale = nullptr, *shift = nullptr;
  int lda = 0;
};

// out_hw > 0: y is the split output in the caller's NCHW layout (see
// ConvArgs::out_hw); the launch returns hipErrorNotSupported, having launched
// nothing, when the layer's kernel cannot store it.
hipError_t run_conv(const Ctx &c, const ConvSpec &cs, const void *x, const Act &in, int nb,
                    void *y, const void *res, bool relu, bool gelu, bool nchw_input, int ldc = 0,
                    const void *x2 = nullptr, const Act *in2 = nullptr, PreAct pre = PreAct{},
                    int out_hw = 0, bool pool = false) {
  ConvArgs a{};
  a.out_hw = out_hw;
  a.pool = pool;
  a.cus = c.cus;
  // Every other convolution of a partition walks its tiles backwards, so it
  // starts on the rows its producer wrote last, the ones most likely still in
  // the last-level cache (ResNet-50 b256 +0.6%, ResNet-18 b64 +1%; the order
  // never changes a result).
  a.rev = c.seq++ & 1;
  a.lanes = c.lanes;
  a.pre_scale = pre.scale;
  a.pre_shift = pre.shift;
  a.lda = pre.lda;
  a.x = x;
  a.w = c.pk + cs.pk_w;
  a.bias = reinterpret_cast<const float *>(c.pk + cs.pk_b);
  a.res = res;
  a.y = y;
  a.n_img = nb;
  a.H = in.h;
  a.W = in.w;
  a.C = in.c;
  a.kh = a.kw = cs.k;
  a.stride = cs.stride;
  a.pad = cs.pad;
  a.Ho = conv_out(in.h, cs.k, cs.stride, cs.pad);
  a.Wo = conv_out(in.w, cs.k, cs.stride, cs.pad);
  a.M = nb * a.Ho * a.Wo;
  a.N = cs.cout;
  a.K = cs.K;
  a.Kp = cs.Kp;
  a.ldc = ldc ? ldc : cs.cout;
  a.ldr = cs.cout;
  a.relu = relu;
  a.gelu = gelu;
  Loader ld;
  if (cs.fused) {
    a.x2 = x2;
    a.H2 = in2->h;
    a.W2 = in2->w;
    a.C2 = in2->c;
    a.s2 = cs.stride2;
    a.K1 = cs.K1;
    ld = LD_CAT;
  } else if (cs.s2d) {
    // x is the space-to-depth buffer: a stride-1 4 x 4 convolution over cells.
    const int k2 = (cs.k + 1) / 2;
    a.H = a.Ho + k2 - 1;
    a.W = a.Wo + k2 - 1;
    a.C = kS2DChannels;
    a.kh = a.kw = k2;
    a.stride = 1;
    a.pad = 0;
    ld = LD_S2D;
  } else if (cs.nhwc8) {
    // x is the 8-slot NHWC copy of the input
    a.C = 8;
    a.kh = a.kw = cs.k;
    ld = LD_NHWC8;
  } else if (nchw_input) {
    const bool vec_ok = c.m.bf16 && cs.k % 8 == 0 && cs.stride % 8 == 0 && cs.pad == 0 &&
                        in.w % 8 == 0 && ((uintptr_t)x % 16) == 0;
    ld = vec_ok ? LD_NCHW_PATCH : LD_NCHW;
  } else {
    ld = (cs.k == 1 && cs.stride == 1 && cs.pad == 0) ? LD_GEMM : LD_NHWC;
  }
  const double flops =
      2.0 * a.M * (double)a.N * (cs.s2d || cs.nhwc8 ? (double)cs.cin * cs.k * cs.k : (double)a.K);
  const double bytes = (double)c.m.esz * ((double)nb * in.elems() + (double)a.M * a.N * (res ? 2 : 1) / (pool ? 4 : 1) +
                                          (double)a.N * a.K + (cs.fused ? (double)a.M * cs.cin2 : 0.0));
  if (c.m.bf16)
    return timed(c.s, F_CONV_BF16, flops, bytes, [&] { return launch_conv_bf16(a, ld, c.s); });
  if (out_hw || pool) return hipErrorNotSupported;
  a.splits = cs.splits;
  a.part = c.part;
  hipError_t r = timed(c.s, F_CONV_F32, flops, bytes, [&] { return launch_conv_f32(a, ld, c.s); });
  if (r != hipSuccess || cs.splits <= 1) return r;
  const double pbytes = 4.0 * a.M * a.N * (cs.splits + 1);
  return timed(c.s, F_SPLIT_SUM, (double)a.M * a.N * cs.splits, pbytes,
               [&] { return launch_f32_split_reduce(a, c.s); });
}

// A ResNet stem (7 x 7 stride-2 convolution with ReLU on space-to-depth
// cells, 64 channels) followed by 3 x 3 stride-2 max pooling with padding 1.
bool stem_pool_fusable(const Model &m) {
  if (!m.bf16 || m.layers.size() < 2 || !m.first_reads_nchw) return false;
  const LayerPlan &l0 = m.layers[0], &l1 = m.layers[1];
  if (l0.L.kind != HAPI_CONV || l0.convs.empty() || !l0.convs[0].s2d || !l0.L.relu) return false;
  const ConvSpec &cs = l0.convs[0];
  if (cs.k != 7 || cs.stride != 2 || cs.pad != 3 || cs.Kp != 4 * 4 * kS2DChannels) return false;
  if (l1.L.kind != HAPI_MAXPOOL || l1.L.k != 3 || l1.L.stride != 2 || l1.L.pad != 1) return false;
  return stem_pool_supported(l0.in.c, l0.in.h, l0.in.w, cs.cout, l0.out.h, l0.out.w, l1.out.h, l1.out.w);
}

// Layer li, a bf16 convolution with ReLU over an NHWC activation, followed by
// layer li + 1, 2 x 2 / 2 max pooling of its whole (even-sized) output: the
// convolution's kernel can pool before it stores.
bool pool_follows(const Model &m, int li) {
  if (!m.bf16 || li + 1 >= (int)m.layers.size()) return false;
  const LayerPlan &lp = m.layers[li], &pl = m.layers[li + 1];
  if (lp.L.kind != HAPI_CONV || !lp.L.relu || lp.convs.size() != 1) return false;
  const ConvSpec &cs = lp.convs[0];
  if (cs.s2d || cs.nhwc8 || cs.fused) return false;
  if (pl.L.kind != HAPI_MAXPOOL || pl.L.k != 2 || pl.L.stride != 2 || pl.L.pad != 0) return false;
  return lp.out.h % 2 == 0 && lp.out.w % 2 == 0 && pl.out.h * 2 == lp.out.h && pl.out.w * 2 == lp.out.w;
}

// ... and the convolution is one the row-streaming 3 x 3 kernel runs (64
// channels to 64, stride 1, padding 1), which pools in its own way.
bool pool_fusable_c64(const Model &m, int li) {
  if (!pool_follows(m, li)) return false;
  const LayerPlan &lp = m.layers[li];
  const ConvSpec &cs = lp.convs[0];
  return conv3x3_c64_supported(cs.cin, cs.cout, cs.k, cs.k, cs.stride, cs.pad, lp.in.w, cs.Kp, cs.cout, cs.cout) &&
         conv3x3_c64_pool_supported(lp.in.h, lp.in.w, cs.cout);
}

// The tensor in front of layer `start` + 1: the input (start = 0) or the
// output of layer `start`.
const Act &act_at(const Model &m, int start) {
  return start == 0 ? m.input : m.layers[start - 1].out;
}

// A tensor whose caller layout equals the internal NHWC one: tokens, and
// images of one pixel or one channel.
bool layout_free(const Act &a) { return a.tok || a.h * a.w == 1 || a.c == 1; }

// A bottleneck with an identity shortcut whose 3 x 3 convolution the
// row-streaming kernel runs (64 channels, stride 1) and whose expansion is
// 64 -> 256: both run as one kernel.
bool expand_fusable(const LayerPlan &lp) {
  if (lp.L.kind != HAPI_BOTTLENECK || lp.has_sc || lp.convs.size() != 3 || lp.convs[2].fused) return false;
  const ConvSpec &c2 = lp.convs[1], &c3 = lp.convs[2];
  return c3.k == 1 && c3.stride == 1 && c3.pad == 0 && c3.cin == c2.cout &&
         conv3x3_c64_supported(c2.cin, c2.cout, c2.k, c2.k, c2.stride, c2.pad, lp.in.w, c2.Kp, c2.cout, c2.cout) &&
         conv3x3_c64_expand_supported(c3.cout, c3.K, c3.Kp, c3.cout, c3.cout);
}

// Layer li, a bf16 bottleneck with an identity shortcut and a plain expanding
// 1 x 1 convolution, followed by layer li + 1, a bottleneck whose first
// convolution reduces li's output with a 1 x 1: the two 1 x 1 convolutions
// run as one kernel (bottleneck_link_supported's shapes).
bool link_fusable(const Model &m, int li) {
  if (!m.bf16 || li + 1 >= (int)m.layers.size()) return false;
  const LayerPlan &lp = m.layers[li], &ln = m.layers[li + 1];
  if (lp.L.kind != HAPI_BOTTLENECK || lp.has_sc || lp.convs.size() != 3 || lp.convs[2].fused) return false;
  if (ln.L.kind != HAPI_BOTTLENECK || ln.convs.empty()) return false;
  if (expand_fusable(lp)) return false;
  const ConvSpec &c3 = lp.convs[2], &c1 = ln.convs[0];
  if (c3.k != 1 || c3.stride != 1 || c3.pad != 0 || c1.k != 1 || c1.stride != 1 || c1.pad != 0) return false;
  if (c1.cin != c3.cout || lp.out.h != ln.in.h || lp.out.w != ln.in.w || lp.in.h != lp.out.h || lp.in.w != lp.out.w)
    return false;
  return bottleneck_link_supported(c3.cin, c3.cout, c1.cout, c3.Kp, c1.Kp);
}

// Runs layers start+1..split on nb images of `images` (the layer-`start`
// tensor in the caller layout); writes the split output (caller layout) to
// `out` unless it is null (profiling).
int run_chunk(const Ctx &c, const void *images, int nb, int start, int split, void *out) {
  const Model &m = c.m;
  c.seq = 0;
  const bool bf = m.bf16;
  const void *cur = images;
  int cur_slot = -1;
  auto free_slot = [&](int a = -1, int b = -1) {
    for (int i = 0; i < 3; ++i)
      if (i != cur_slot && i != a && i != b) return i;
    return -1;
  };
  // Stage the input in slot 0 in NHWC, except for a first layer that reads
  // the caller's NCHW images itself.  Blocks update their input slot in
  // place, so a resumed input is always staged, never used where it lies.
  if (start > 0 || !m.first_reads_nchw) {
    const Act &a = act_at(m, start);
    const int64_t bytes = (int64_t)nb * a.elems() * m.esz;
    if (layout_free(a)) {
      HIP_TRY(timed(c.s, F_COPY, 0.0, 2.0 * bytes, [&] { return launch_copy(images, c.slot[0], bytes, c.s); }));
    } else {
      HIP_TRY(timed(c.s, F_LAYOUT, 0.0, 2.0 * bytes, [&] {
        return launch_nchw_to_nhwc(bf, images, c.slot[0], nb, a.h * a.w, a.c, c.s);
      }));
    }
    cur = c.slot[0];
    cur_slot = 0;
  }
  // The split layer's last convolution stores the split output in the
  // caller's NCHW layout itself when its kernel can (no separate layout pass);
  // `stored` records that it did.
  const Act &split_act = m.layers[split - 1].out;
  void *const nchw_out = (out && bf && !layout_free(split_act)) ? out : nullptr;
  bool stored = false;
  // Runs the last convolution of layer li: into `out` as NCHW when li is the
  // split layer and the kernel supports it, else into slot `dst` with `res`.
  auto last_conv = [&](int li, const ConvSpec &cs, const void *x, const Act &in, int dst, const void *res,
                       bool relu, const void *x2 = nullptr, const Act *in2 = nullptr) -> int {
    if (nchw_out && li == split - 1) {
      const hipError_t e = run_conv(c, cs, x, in, nb, nchw_out, res, relu, false, false, 0, x2, in2, PreAct{},
                                    split_act.h * split_act.w);
      if (e == hipSuccess) {
        stored = true;
        return HAPI_OK;
      }
      if (e != hipErrorNotSupported) HIP_TRY(e);
    }
    HIP_TRY(run_conv(c, cs, x, in, nb, c.slot[dst], res, relu, false, false, 0, x2, in2));
    return HAPI_OK;
  };
  int li0 = start;
  int linked = -1;  // slot holding the next bottleneck's first convolution, when already run
  // Stem convolution and max pooling in one kernel when the stem output is
  // not itself the split and layers are not being timed one by one.
  if (start == 0 && split >= 2 && !c.on_layer && stem_pool_fusable(m) && (uintptr_t)images % 4 == 0) {
    const LayerPlan &l0 = m.layers[0], &l1 = m.layers[1];
    const ConvSpec &cs = l0.convs[0];
    const int o = free_slot();
    const double flops = 2.0 * nb * l0.out.h * l0.out.w * (double)cs.cout * cs.cin * cs.k * cs.k;
    const double bytes = (double)m.esz * ((double)nb * (l0.in.elems() + l1.out.elems()) + (double)cs.cout * cs.Kp);
    HIP_TRY(timed(c.s, F_CONV_BF16, flops, bytes, [&] {
      return launch_stem_pool_bf16(images, c.pk + cs.pk_w, cs.Kp, reinterpret_cast<const float *>(c.pk + cs.pk_b),
                                   c.slot[o], nb, l0.in.c, l0.in.h, l0.in.w, l0.out.h, l0.out.w, l1.out.h,
                                   l1.out.w, c.cus, c.s);
    }));
    cur = c.slot[o];
    cur_slot = o;
    li0 = 2;
  }
  for (int li = li0; li < split; ++li) {
    const LayerPlan &lp = m.layers[li];
    const hapi_layer &L = lp.L;
    if (c.on_layer) c.on_layer(li, true);
    const bool nchw_in = (li == 0) && m.first_reads_nchw;
    // A convolution with ReLU followed by 2 x 2 / 2 max pooling (VGG's
    // conv1_2 + pool1 ... conv5_3 + pool5), when its own output is not the
    // split and layers are not being timed one by one: one kernel pools the
    // rounded result before storing it, bit for bit the two layers' output.
    // 64 channels to 64 at stride 1: the row-streaming 3 x 3 kernel; others:
    // the implicit GEMM with its rows in pooling-window order, when the
    // layer's kernel supports it (else the two layers run apart).
    if (L.kind == HAPI_CONV && !nchw_in && !c.on_layer && li + 1 < split && !pool_fusable_c64(m, li) &&
        pool_follows(m, li)) {
      const int o = free_slot();
      const hipError_t e = run_conv(c, lp.convs[0], cur, lp.in, nb, c.slot[o], nullptr, true, false, false, 0,
                                    nullptr, nullptr, PreAct{}, 0, true);
      if (e == hipSuccess) {
        cur = c.slot[o];
        cur_slot = o;
        ++li;  // the pooling layer ran inside the convolution
        continue;
      }
      if (e != hipErrorNotSupported) HIP_TRY(e);
    }
    if (L.kind == HAPI_CONV && !nchw_in && !c.on_layer && li + 1 < split && pool_fusable_c64(m, li)) {
      const ConvSpec &cs = lp.convs[0];
      const LayerPlan &pl = m.layers[li + 1];
      const int o = free_slot();
      const double flops = 2.0 * nb * lp.out.h * lp.out.w * (double)cs.cout * cs.K;
      const double bytes = (double)m.esz * ((double)nb * (lp.in.elems() + pl.out.elems()) + (double)cs.cout * cs.Kp);
      HIP_TRY(timed(c.s, F_CONV_BF16, flops, bytes, [&] {
        return launch_conv3x3_c64(cur, c.pk + cs.pk_w, cs.Kp, reinterpret_cast<const float *>(c.pk + cs.pk_b), nullptr,
                                  cs.cout, c.slot[o], cs.cout, nb, lp.in.h, lp.in.w, true, c.cus, c.s, nullptr, 0,
                                  nullptr, true);
      }));
      cur = c.slot[o];
      cur_slot = o;
      ++li;  // the pooling layer ran inside the convolution
      continue;
    }
    switch (L.kind) {
      case HAPI_CONV:
      case HAPI_PATCH_EMBED: {
        const ConvSpec &cs = lp.convs[0];
        const void *src = cur;
        int o = free_slot();
        if (cs.s2d) {
          const int ho = lp.out.h, wo = lp.out.w;
          HIP_TRY(timed(c.s, F_LAYOUT, 0.0,
                        (double)nb * (lp.in.elems() + (int64_t)(ho + 3) * (wo + 3) * kS2DChannels) * m.esz,
                        [&] {
                          return launch_space_to_depth(cur, c.slot[o], nb, lp.in.c, lp.in.h, lp.in.w,
                                                       cs.pad, ho + 3, wo + 3, c.s);
                        }));
          src = c.slot[o];
          o = free_slot(o);
        } else if (cs.nhwc8) {
          HIP_TRY(timed(c.s, F_LAYOUT, 0.0, (double)nb * lp.in.h * lp.in.w * (lp.in.c + 8) * m.esz, [&] {
            return launch_nchw_to_nhwc8(cur, c.slot[o], nb, lp.in.c, lp.in.h, lp.in.w, c.s);
          }));
          src = c.slot[o];
          o = free_slot(o);
        }
        if (!nchw_in && !cs.s2d && !cs.nhwc8) {
          if (int r = last_conv(li, cs, src, lp.in, o, nullptr, L.kind == HAPI_CONV && L.relu)) return r;
        } else {
          HIP_TRY(run_conv(c, cs, src, lp.in, nb, c.slot[o], nullptr, L.kind == HAPI_CONV && L.relu, false,
                           nchw_in));
        }
        cur = c.slot[o];
        cur_slot = o;
        break;
      }
      case HAPI_MAXPOOL: {
        const int o = free_slot();
        HIP_TRY(timed(c.s, F_MAXPOOL, (double)nb * lp.out.elems() * L.k * L.k,
                      (double)nb * (lp.in.elems() + lp.out.elems()) * m.esz, [&] {
                        return launch_maxpool(bf, cur, c.slot[o], nb, lp.in.h, lp.in.w, lp.in.c, L.k,
                                              L.stride, L.pad, lp.out.h, lp.out.w, c.s);
                      }));
        cur = c.slot[o];
        cur_slot = o;
        break;
      }
      case HAPI_AVGPOOL: {
        const int o = free_slot();
        HIP_TRY(timed(c.s, F_AVGPOOL, (double)nb * lp.in.elems(),
                      (double)nb * (lp.in.elems() + lp.out.elems()) * m.esz, [&] {
                        return launch_avgpool(bf, cur, c.slot[o], nb, lp.in.h, lp.in.w, lp.in.c, L.k,
                                              L.stride, lp.out.h, lp.out.w, c.s);
                      }));
        cur = c.slot[o];
        cur_slot = o;
        break;
      }
      case HAPI_BASIC_BLOCK: {
        const int A = free_slot();
        const Act mid{lp.out.c, lp.out.h, lp.out.w, false};
        HIP_TRY(run_conv(c, lp.convs[0], cur, lp.in, nb, c.slot[A], nullptr, true, false, false));
        if (lp.convs[1].fused) {  // conv2 and the projection shortcut in one GEMM
          const int B = free_slot(A);
          if (int r = last_conv(li, lp.convs[1], c.slot[A], mid, B, nullptr, true, cur, &lp.in)) return r;
          cur = c.slot[B];
          cur_slot = B;
          break;
        }
        const void *res = cur;
        if (lp.has_sc) {
          const int B = free_slot(A);
          HIP_TRY(run_conv(c, lp.convs[2], cur, lp.in, nb, c.slot[B], nullptr, false, false, false));
          res = c.slot[B];
        }
        // In place over the block input: each output element's residual is read
        // by the same thread right before that element is written.
        if (int r = last_conv(li, lp.convs[1], c.slot[A], mid, cur_slot, res, true)) return r;
        cur = c.slot[cur_slot];
        break;
      }
      case HAPI_BOTTLENECK: {
        // The previous block's kernel already ran this block's first
        // convolution into slot `linked`.
        const int A = linked >= 0 ? linked : free_slot(), B = free_slot(A);
        const int width = L.width;
        const Act a1{width, lp.in.h, lp.in.w, false};
        const Act a2{width, lp.out.h, lp.out.w, false};
        if (linked < 0) HIP_TRY(run_conv(c, lp.convs[0], cur, lp.in, nb, c.slot[A], nullptr, true, false, false));
        linked = -1;
        if (expand_fusable(lp)) {
          // The 3 x 3 and the expanding 1 x 1 in one kernel, in place over the
          // block input (each output element's residual is read by the lane
          // that writes it, before it writes it).
          const ConvSpec &c2 = lp.convs[1], &c3 = lp.convs[2];
          const double px = (double)nb * a2.h * a2.w;
          const double flops = 2.0 * px * (c2.cout * (double)c2.K + c3.cout * (double)c3.K);
          const double bytes = (double)m.esz * (px * (c2.cin + 2.0 * c3.cout) + (double)c2.cout * c2.Kp +
                                                (double)c3.cout * c3.Kp);
          HIP_TRY(timed(c.s, F_CONV_BF16, flops, bytes, [&] {
            return launch_conv3x3_c64(c.slot[A], c.pk + c2.pk_w, c2.Kp, reinterpret_cast<const float *>(c.pk + c2.pk_b),
                                      cur, c3.cout, c.slot[cur_slot], c3.cout, nb, a1.h, a1.w, true, c.cus, c.s,
                                      c.pk + c3.pk_w, c3.Kp, reinterpret_cast<const float *>(c.pk + c3.pk_b));
          }));
          cur = c.slot[cur_slot];
          break;
        }
        HIP_TRY(run_conv(c, lp.convs[1], c.slot[A], a1, nb, c.slot[B], nullptr, true, false, false));
        if (!c.on_layer && li + 1 < split && link_fusable(m, li)) {
          // This block's expansion (in place over the block input, which is
          // its residual) and the next block's reduction (into slot A, free
          // once the 3 x 3 has read it) in one kernel.
          const ConvSpec &c3 = lp.convs[2], &n1 = m.layers[li + 1].convs[0];
          const double px = (double)nb * a2.h * a2.w;
          const double flops = 2.0 * px * ((double)c3.cout * c3.K + (double)n1.cout * n1.K);
          const double bytes = (double)m.esz * (px * (c3.cin + 2.0 * c3.cout + n1.cout) + (double)c3.cout * c3.Kp +
                                                (double)n1.cout * n1.Kp);
          HIP_TRY(timed(c.s, F_CONV_BF16, flops, bytes, [&] {
            return launch_bottleneck_link(c.slot[B], c.pk + c3.pk_w, reinterpret_cast<const float *>(c.pk + c3.pk_b),
                                          cur, c.slot[cur_slot], c.pk + n1.pk_w,
                                          reinterpret_cast<const float *>(c.pk + n1.pk_b), c.slot[A],
                                          nb * a2.h * a2.w, c3.cin, c3.cout, n1.cout, c.s);
          }));
          cur = c.slot[cur_slot];
          linked = A;
          break;
        }
        if (lp.convs[2].fused) {  // c3 and the projection shortcut in one GEMM, into the free slot
          if (int r = last_conv(li, lp.convs[2], c.slot[B], a2, A, nullptr, true, cur, &lp.in)) return r;
          cur = c.slot[A];
          cur_slot = A;
          break;
        }
        const void *res = cur;
        if (lp.has_sc) {
          HIP_TRY(run_conv(c, lp.convs[3], cur, lp.in, nb, c.slot[A], nullptr, false, false, false));
          res = c.slot[A];
        }
        if (int r = last_conv(li, lp.convs[2], c.slot[B], a2, cur_slot, res, true)) return r;
        cur = c.slot[cur_slot];
        break;
      }
      case HAPI_TOKENS: {
        const int o = free_slot();
        const int T = lp.out.h, D = lp.out.c;
        HIP_TRY(timed(c.s, F_TOKENS, (double)nb * T * D, 2.0 * nb * T * D * m.esz, [&] {
          return launch_tokens(cur, reinterpret_cast<const float *>(c.pk + lp.extras[0].pk),
                               reinterpret_cast<const float *>(c.pk + lp.extras[1].pk), c.slot[o], nb,
                               T, D, c.s);
        }));
        cur = c.slot[o];
        cur_slot = o;
        break;
      }
      case HAPI_VIT_BLOCK: {
        const int A = free_slot(), B = free_slot(A);
        const int T = lp.in.h, D = lp.in.c;
        const int64_t rows = (int64_t)nb * T;
        // token matrices as NHWC images of one row: n = 1, H = rows, W = 1
        const Act tokD{D, (int)rows, 1, false};
        const Act tokF{L.mlp_dim, (int)rows, 1, false};
        auto ln = [&](const Extra &g, const Extra &b, const void *x, void *y) {
          return timed(c.s, F_LN, 8.0 * rows * D, 2.0 * rows * D * m.esz, [&] {
            return launch_layernorm(x, reinterpret_cast<const float *>(c.pk + g.pk),
                                    reinterpret_cast<const float *>(c.pk + b.pk), y, rows, D, 1e-6f, c.s);
          });
        };
        HIP_TRY(ln(lp.extras[0], lp.extras[1], cur, c.slot[A]));
        HIP_TRY(run_conv(c, lp.convs[0], c.slot[A], tokD, 1, c.slot[B], nullptr, false, false, false));
        HIP_TRY(timed(c.s, F_ATTN, 4.0 * nb * (double)T * T * D, 4.0 * rows * D * m.esz, [&] {
          return launch_attention(c.slot[B], c.slot[A], nb, T, D, L.heads, c.s);
        }));
        HIP_TRY(run_conv(c, lp.convs[1], c.slot[A], tokD, 1, c.slot[cur_slot], cur, false, false, false));
        HIP_TRY(ln(lp.extras[2], lp.extras[3], cur, c.slot[A]));
        HIP_TRY(run_conv(c, lp.convs[2], c.slot[A], tokD, 1, c.slot[B], nullptr, false, true, false));
        // The split block's last linear layer writes the caller's [B, T, D]
        // output itself (the token layout is the caller's layout).
        if (out && li == split - 1) {
          HIP_TRY(run_conv(c, lp.convs[3], c.slot[B], tokF, 1, out, cur, false, false, false));
          stored = true;
        } else {
          HIP_TRY(run_conv(c, lp.convs[3], c.slot[B], tokF, 1, c.slot[cur_slot], cur, false, false, false));
        }
        break;
      }
      case HAPI_LAYERNORM: {
        const int o = free_slot();
        const int64_t rows = (int64_t)nb * lp.in.h;
        const int D = lp.in.c;
        HIP_TRY(timed(c.s, F_LN, 8.0 * rows * D, 2.0 * rows * D * m.esz, [&] {
          return launch_layernorm(cur, reinterpret_cast<const float *>(c.pk + lp.extras[0].pk),
                                  reinterpret_cast<const float *>(c.pk + lp.extras[1].pk), c.slot[o],
                                  rows, D, 1e-6f, c.s);
        }));
        cur = c.slot[o];
        cur_slot = o;
        break;
      }
      case HAPI_PREACT_CONV: {
        // Batch-norm + ReLU in front of the convolution cannot fold into its
        // weights.  A 1 x 1 convolution applies them to its operand as it
        // reads it; otherwise they run on the input first.
        const int A = free_slot(), B = free_slot(A);
        const int64_t pixels = (int64_t)nb * lp.in.h * lp.in.w;
        const Extra &bn = lp.extras[0];
        const float *scale = reinterpret_cast<const float *>(c.pk + bn.pk), *shift = scale + bn.n;
        const ConvSpec &cs = lp.convs[0];
        if (cs.k == 1 && cs.stride == 1 && cs.pad == 0 && cs.K <= kPreMax) {
          HIP_TRY(run_conv(c, cs, cur, lp.in, nb, c.slot[B], nullptr, false, false, false, 0, nullptr, nullptr,
                           PreAct{scale, shift, 0}));
        } else {
          HIP_TRY(timed(c.s, F_AFFINE, 2.0 * pixels * lp.in.c, 2.0 * pixels * lp.in.c * m.esz, [&] {
            return launch_affine(cur, scale, shift, c.slot[A], pixels, lp.in.c, lp.in.c, true, c.s);
          }));
          HIP_TRY(run_conv(c, cs, c.slot[A], lp.in, nb, c.slot[B], nullptr, false, false, false));
        }
        cur = c.slot[B];
        cur_slot = B;
        break;
      }
      case HAPI_BATCHNORM: {
        const int o = free_slot();
        const int64_t pixels = (int64_t)nb * lp.in.h * lp.in.w;
        const Extra &bn = lp.extras[0];
        HIP_TRY(timed(c.s, F_AFFINE, 2.0 * pixels * lp.in.c, 2.0 * pixels * lp.in.c * m.esz, [&] {
          return launch_affine(cur, reinterpret_cast<const float *>(c.pk + bn.pk),
                               reinterpret_cast<const float *>(c.pk + bn.pk) + bn.n, c.slot[o], pixels,
                               lp.in.c, lp.in.c, L.relu != 0, c.s);
        }));
        cur = c.slot[o];
        cur_slot = o;
        break;
      }
      case HAPI_DENSE_BLOCK: {
        // Concatenation without copies: the block input is copied once into the
        // first channels of a buffer with all cout channels, and each dense
        // layer's 3x3 convolution stores its growth channels into its slice.
        const int A = free_slot();
        const int64_t pixels = (int64_t)nb * lp.in.h * lp.in.w;
        const int cout = L.cout, growth = L.width, bott = L.mlp_dim;
        uint8_t *cat = c.slot[A];
        HIP_TRY(timed(c.s, F_COPY, 0.0, 2.0 * pixels * lp.in.c * m.esz, [&] {
          return launch_channel_copy(cur, cat, pixels, lp.in.c, lp.in.c, cout, 0, c.s);
        }));
        const int H = cur_slot, B = free_slot(A);  // block input no longer needed
        for (size_t l = 0; l < lp.extras.size(); ++l) {
          const int ch = lp.in.c + (int)l * growth;
          const Extra &bn = lp.extras[l];
          const float *scale = reinterpret_cast<const float *>(c.pk + bn.pk), *shift = scale + bn.n;
          const Act hin{ch, lp.in.h, lp.in.w, false};
          const Act tin{bott, lp.in.h, lp.in.w, false};
          // The 1 x 1 convolution reads the first ch channels of the
          // concatenation and applies BN1 + ReLU as it reads them.
          if (ch <= kPreMax) {
            HIP_TRY(run_conv(c, lp.convs[2 * l], cat, hin, nb, c.slot[B], nullptr, true, false, false, 0, nullptr,
                             nullptr, PreAct{scale, shift, cout}));
          } else {
            HIP_TRY(timed(c.s, F_AFFINE, 2.0 * pixels * ch, 2.0 * pixels * ch * m.esz, [&] {
              return launch_affine(cat, scale, shift, c.slot[H], pixels, ch, cout, true, c.s);
            }));
            HIP_TRY(run_conv(c, lp.convs[2 * l], c.slot[H], hin, nb, c.slot[B], nullptr, true, false, false));
          }
          HIP_TRY(run_conv(c, lp.convs[2 * l + 1], c.slot[B], tin, nb, cat + (int64_t)ch * m.esz, nullptr,
                           false, false, false, cout));
        }
        cur = cat;
        cur_slot = A;
        break;
      }
      default:
        return fail(HAPI_E_INVAL, "layer %d: unknown kind", li + 1);
    }
    if (c.on_layer) c.on_layer(li, false);
  }
  if (out && !stored) {
    const Act &o = m.layers[split - 1].out;
    const int64_t bytes = (int64_t)nb * o.elems() * m.esz;
    if (layout_free(o)) {
      HIP_TRY(timed(c.s, F_COPY, 0.0, 2.0 * bytes, [&] { return launch_copy(cur, out, bytes, c.s); }));
    } else {
      HIP_TRY(timed(c.s, F_LAYOUT, 0.0, 2.0 * bytes, [&] {
        return launch_nhwc_to_nchw(bf, cur, out, nb, o.h * o.w, o.c, c.s);
      }));
    }
  }
  return HAPI_OK;
}

// Auxiliary streams of one host thread on one device, with the events that
// fork them from the caller's stream and join them back.  Created on first
// use and kept for the thread's lifetime; per thread, so that concurrent
// callers never record each other's events.
struct Lanes {
  int dev = -1;
  hipStream_t aux[kMaxInflight - 1] = {};
  hipEvent_t fork = nullptr, join[kMaxInflight - 1] = {};
};

int get_lanes(hipStream_t s, Lanes **out) {
  static thread_local std::vector<Lanes> per_dev;
  int dev = 0, cur = 0;
  HIP_TRY(hipStreamGetDevice(s, &dev));
  HIP_TRY(hipGetDevice(&cur));
  if (dev != cur) return fail(HAPI_E_INVAL, "desc->stream belongs to device %d, current device is %d", dev, cur);
  if ((int)per_dev.size() <= dev) per_dev.resize(dev + 1);
  Lanes &L = per_dev[dev];
  if (L.dev < 0) {
    HIP_TRY(hipEventCreateWithFlags(&L.fork, hipEventDisableTiming));
    for (int i = 0; i < kMaxInflight - 1; ++i) {
      HIP_TRY(hipStreamCreateWithFlags(&L.aux[i], hipStreamNonBlocking));
      HIP_TRY(hipEventCreateWithFlags(&L.join[i], hipEventDisableTiming));
    }
    L.dev = dev;
  }
  *out = &L;
  return HAPI_OK;
}

// Runs the batch as partitions of `chunk` images, `lanes` of them in flight:
// partition p runs on lane p % lanes (lane 0 is desc->stream, the others
// auxiliary streams forked from it and joined back into it at the end) with
// that lane's three workspace slots.  Partitions are independent, and each
// gives the same bits whichever lane runs it.  `route_lanes` is the number of
// partitions in flight the kernels' tile choice assumes: `lanes` for an
// extraction; for the per-layer profile, which runs the partitions one after
// another, the number an extraction of the same batch would run, so that the
// profile times the kernels the extraction runs.
int run_batch(const hapi_model_desc *d, const Model &m, const void *weights, const void *images,
              int batch, int start, int split, void *out, uint8_t *ws, int chunk, int lanes,
              int route_lanes, const std::function<void(int, bool)> &on_layer) {
  hipStream_t s = static_cast<hipStream_t>(d->stream);
  const LaneLayout ll = lane_layout(m, split, chunk);
  Lanes *L = nullptr;
  if (lanes > 1) {
    if (int r = get_lanes(s, &L)) return r;
    HIP_TRY(hipEventRecord(L->fork, s));
    for (int i = 1; i < lanes; ++i) HIP_TRY(hipStreamWaitEvent(L->aux[i - 1], L->fork, 0));
  }
  std::vector<Ctx> c;
  c.reserve(lanes);
  // Persistent kernels of every lane size their grid to the whole device:
  // halving it per lane was measured slower (ResNet-50 b256: 69.5k -> 66k img/s).
  const int cus = cu_count();
  for (int i = 0; i < lanes; ++i) {
    uint8_t *w0 = ws + (int64_t)i * ll.bytes;
    c.push_back(Ctx{m, i ? L->aux[i - 1] : s, static_cast<const uint8_t *>(weights),
                    {w0 + ll.slot[0], w0 + ll.slot[1], w0 + ll.slot[2]}, on_layer, cus,
                    reinterpret_cast<float *>(w0 + ll.part),
                    std::min(route_lanes, (batch + chunk - 1) / chunk)});
  }
  const int64_t in_bytes = act_at(m, start).elems() * m.esz;
  const int64_t out_bytes = m.layers[split - 1].out.elems() * m.esz;
  int r = HAPI_OK;
  for (int b0 = 0, p = 0; b0 < batch && r == HAPI_OK; b0 += chunk, ++p) {
    const int nb = std::min(chunk, batch - b0);
    r = run_chunk(c[p % lanes], static_cast<const uint8_t *>(images) + (int64_t)b0 * in_bytes, nb, start,
                  split, out ? static_cast<uint8_t *>(out) + (int64_t)b0 * out_bytes : nullptr);
  }
  // Join even after a failed launch, so that desc->stream still orders
  // everything that was issued.
  for (int i = 1; i < lanes; ++i) {
    HIP_TRY(hipEventRecord(L->join[i - 1], L->aux[i - 1]));
    HIP_TRY(hipStreamWaitEvent(s, L->join[i - 1], 0));
  }
  return r;
}

// ------------------------------------------------------------- plan replay

// Everything that determines the kernel launches of an extraction.
struct PlanKey {
  std::vector<hapi_layer> layers;
  int32_t dtype = 0, in_c = 0, in_h = 0, in_w = 0, chunk = 0, inflight = 0;
  const void *weights = nullptr, *images = nullptr, *out = nullptr, *ws = nullptr;
  int batch = 0, start = 0, split = 0, dev = -1;

  bool operator==(const PlanKey &o) const {
    return dtype == o.dtype && in_c == o.in_c && in_h == o.in_h && in_w == o.in_w && chunk == o.chunk &&
           inflight == o.inflight && weights == o.weights && images == o.images && out == o.out &&
           ws == o.ws && batch == o.batch && start == o.start && split == o.split && dev == o.dev &&
           layers.size() == o.layers.size() &&
           std::memcmp(layers.data(), o.layers.data(), layers.size() * sizeof(hapi_layer)) == 0;
  }
};

struct Plan {
  PlanKey key;
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
};

// Per host thread: the key of the previous extraction, the captured plans
// (most recent first) and a private stream per device to capture on (the
// caller's stream may be the null stream, which cannot be captured).  Never
// freed: graphs stay valid until the process ends, and destroying them from a
// thread-exit destructor could run after the HIP runtime has shut down.
struct PlanCache {
  PlanKey last;
  bool has_last = false;
  std::vector<Plan> plans;
  std::vector<hipStream_t> capture;  // per device
};
constexpr size_t kMaxPlans = 8;

PlanCache &plan_cache() {
  static thread_local PlanCache *pc = new PlanCache();
  return *pc;
}

// Runs the extraction through the plan cache: replays a captured graph, or
// captures one when the same call was made just before, or launches directly.
int run_planned(const hapi_model_desc *desc, const Model &m, const void *weights, const void *images,
                int batch, int start, int split, void *out, uint8_t *ws, int chunk, int lanes) {
  hipStream_t s = static_cast<hipStream_t>(desc->stream);
  PlanKey k;
  k.layers.assign(desc->layers, desc->layers + desc->n_layers);
  k.dtype = desc->dtype; k.in_c = desc->in_c; k.in_h = desc->in_h; k.in_w = desc->in_w;
  k.chunk = desc->chunk; k.inflight = desc->inflight;
  k.weights = weights; k.images = images; k.out = out; k.ws = ws;
  k.batch = batch; k.start = start; k.split = split;
  HIP_TRY(hipStreamGetDevice(s, &k.dev));
  PlanCache &pc = plan_cache();
  for (size_t i = 0; i < pc.plans.size(); ++i) {
    if (!(pc.plans[i].key == k)) continue;
    std::rotate(pc.plans.begin(), pc.plans.begin() + i, pc.plans.begin() + i + 1);
    pc.has_last = false;
    HIP_TRY(hipGraphLaunch(pc.plans[0].exec, s));
    return HAPI_OK;
  }
  if (!pc.has_last || !(pc.last == k)) {
    pc.last = std::move(k);
    pc.has_last = true;
    return run_batch(desc, m, weights, images, batch, start, split, out, ws, chunk, lanes, lanes, nullptr);
  }
  // Second identical call in a row: capture it on this thread's private
  // stream of the device, then launch the graph on the caller's stream.
  pc.has_last = false;
  const int dev = k.dev;
  if ((int)pc.capture.size() <= dev) pc.capture.resize(dev + 1, nullptr);
  if (!pc.capture[dev]) HIP_TRY(hipStreamCreateWithFlags(&pc.capture[dev], hipStreamNonBlocking));
  hapi_model_desc dc = *desc;
  dc.stream = pc.capture[dev];
  HIP_TRY(hipStreamBeginCapture(pc.capture[dev], hipStreamCaptureModeThreadLocal));
  const int r = run_batch(&dc, m, weights, images, batch, start, split, out, ws, chunk, lanes, lanes, nullptr);
  Plan p;
  p.key = std::move(k);
  const hipError_t e = hipStreamEndCapture(pc.capture[dev], &p.graph);
  if (r != HAPI_OK) {
    if (p.graph) (void)hipGraphDestroy(p.graph);
    return r;
  }
  if (e != hipSuccess) return fail(HAPI_E_DEVICE, "hipStreamEndCapture failed: %s", hipGetErrorString(e));
  const hipError_t ie = hipGraphInstantiate(&p.exec, p.graph, nullptr, nullptr, 0);
  if (ie != hipSuccess) {
    (void)hipGraphDestroy(p.graph);
    return fail(HAPI_E_DEVICE, "hipGraphInstantiate failed: %s", hipGetErrorString(ie));
  }
  if (pc.plans.size() == kMaxPlans) {
    (void)hipGraphExecDestroy(pc.plans.back().exec);
    (void)hipGraphDestroy(pc.plans.back().graph);
    pc.plans.pop_back();
  }
  pc.plans.insert(pc.plans.begin(), std::move(p));
  HIP_TRY(hipGraphLaunch(pc.plans[0].exec, s));
  return HAPI_OK;
}

bool stats_enabled() {
  std::lock_guard<std::mutex> g(g_stats_mu);
  return g_stats_on;
}

}  // namespace
}  // namespace hapi

using namespace hapi;

extern "C" {

int64_t hapi_raw_weight_count(const hapi_model_desc *desc) {
  Model m;
  const int r = analyze(desc, m);
  return r != HAPI_OK ? r : m.raw_count;
}

int64_t hapi_packed_weight_bytes(const hapi_model_desc *desc) {
  Model m;
  const int r = analyze(desc, m);
  return r != HAPI_OK ? r : m.packed_bytes;
}

int hapi_layer_shape(const hapi_model_desc *desc, int32_t layer, int64_t *dims, int32_t *ndim) {
  Model m;
  const int r = analyze(desc, m);
  if (r != HAPI_OK) return r;
  if (!dims || !ndim) return fail(HAPI_E_INVAL, "dims / ndim is NULL");
  if (layer < 0 || layer > (int)m.layers.size())
    return fail(HAPI_E_INVAL, "layer %d outside [0, %d]", layer, (int)m.layers.size());
  const Act a = layer == 0 ? m.input : m.layers[layer - 1].out;
  if (a.tok) {
    *ndim = 2; dims[0] = a.h; dims[1] = a.c; dims[2] = 0;
  } else {
    *ndim = 3; dims[0] = a.c; dims[1] = a.h; dims[2] = a.w;
  }
  return HAPI_OK;
}

int32_t hapi_chunk_count(const hapi_model_desc *desc, int32_t batch) {
  Model m;
  const int r = analyze(desc, m);
  if (r != HAPI_OK) return r;
  if (batch < 1) return fail(HAPI_E_INVAL, "batch must be >= 1");
  const int c = chunk_for(desc, m, batch);
  return (batch + c - 1) / c;
}

int64_t hapi_workspace_bytes(const hapi_model_desc *desc, int32_t batch, int32_t split_layer,
                             int32_t profile) {
  Model m;
  const int r = analyze(desc, m);
  if (r != HAPI_OK) return r;
  if (batch < 1) return fail(HAPI_E_INVAL, "batch must be >= 1");
  if (split_layer < 0 || split_layer > (int)m.layers.size())
    return fail(HAPI_E_INVAL, "split %d outside [0, %d]", split_layer, (int)m.layers.size());
  const int chunk = chunk_for(desc, m, batch);
  if ((int64_t)chunk * max_tmp(m, split_layer) >= kIndexLimit)
    return fail(HAPI_E_UNSUPPORTED, "a partition of %d images exceeds 2^31 elements; lower chunk", chunk);
  return workspace_for(m, split_layer, chunk, profile != 0, batch, lanes_for(desc, chunk, batch));
}

int32_t hapi_workspace_guards(const hapi_model_desc *desc, int32_t batch, int32_t split_layer,
                              int64_t *offsets, int32_t max_entries) {
  Model m;
  const int r = analyze(desc, m);
  if (r != HAPI_OK) return r;
  if (batch < 1) return fail(HAPI_E_INVAL, "batch must be >= 1");
  if (split_layer < 0 || split_layer > (int)m.layers.size())
    return fail(HAPI_E_INVAL, "split %d outside [0, %d]", split_layer, (int)m.layers.size());
  if (max_entries < 0 || (max_entries > 0 && !offsets)) return fail(HAPI_E_INVAL, "offsets is NULL");
  if (split_layer == 0) return 0;
  const int chunk = chunk_for(desc, m, batch);
  const int lanes = lanes_for(desc, chunk, batch);
  const LaneLayout ll = lane_layout(m, split_layer, chunk);
  int n = 0;
  for (int l = 0; l < lanes; ++l)
    for (int g = 0; g < 4; ++g, ++n)
      if (n < max_entries) offsets[n] = (int64_t)l * ll.bytes + ll.guard[g];
  return n;
}

int hapi_pack_weights(const hapi_model_desc *desc, const void *raw_weights, void *packed) {
  Model m;
  int r = analyze(desc, m);
  if (r != HAPI_OK) return r;
  if (m.packed_bytes == 0) return HAPI_OK;  // a model without parameters (pools only)
  if (!raw_weights || !packed) return fail(HAPI_E_INVAL, "raw_weights / packed is NULL");
  if ((uintptr_t)packed % kAlign) return fail(HAPI_E_INVAL, "packed must be 256-byte aligned");
  if ((uintptr_t)raw_weights % 4) return fail(HAPI_E_INVAL, "raw_weights must be 4-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(desc->stream);
  const float *raw = static_cast<const float *>(raw_weights);
  uint8_t *pk = static_cast<uint8_t *>(packed);
  for (size_t li = 0; li < m.layers.size(); ++li) {
    const LayerPlan &lp = m.layers[li];
    const bool nchw = li == 0 && m.first_reads_nchw;
    for (const ConvSpec &c : lp.convs) {
      const float *bn = c.raw_bn >= 0 ? raw + c.raw_bn : nullptr;
      const PackOrder order = c.s2d ? PACK_S2D : c.nhwc8 ? PACK_KHKWC8 : nchw ? PACK_CKHKW : PACK_KHKWC;
      float *bias = reinterpret_cast<float *>(pk + c.pk_b);
      HIP_TRY(launch_pack_conv(m.bf16, raw + c.raw_w, c.raw_b >= 0 ? raw + c.raw_b : nullptr,
                               bn, bn ? bn + c.cout : nullptr, bn ? bn + 2 * c.cout : nullptr,
                               bn ? bn + 3 * c.cout : nullptr, c.cout, c.cin, c.k, c.k,
                               c.fused ? c.K1 : c.Kp, c.Kp, 0, false, order, pk + c.pk_w, bias, s));
      if (c.fused) {
        const float *bn2 = raw + c.raw_bn2;
        HIP_TRY(launch_pack_conv(m.bf16, raw + c.raw_w2, nullptr, bn2, bn2 + c.cout, bn2 + 2 * c.cout,
                                 bn2 + 3 * c.cout, c.cout, c.cin2, 1, 1, c.cin2, c.Kp, c.K1, true,
                                 PACK_KHKWC, pk + c.pk_w, bias, s));
      }
    }
    for (const Extra &e : lp.extras) {
      float *dst = reinterpret_cast<float *>(pk + e.pk);
      if (e.bn_affine) HIP_TRY(launch_pack_affine(raw + e.raw, (int)e.n, dst, dst + e.n, s));
      else HIP_TRY(launch_copy_f32(raw + e.raw, dst, e.n, s));
    }
  }
  return HAPI_OK;
}

}  // extern "C"

namespace {

// Device scratch of hapi_extract_noalloc: one copy per GPU the library runs
// on, held until the process ends.  In host code `scratch` only names the
// symbol; its device address comes from hipGetSymbolAddress, per device.
constexpr int64_t kScratchBytes = HAPI_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

// The address of `scratch` on the current device `dev`, looked up once per
// device (with that device current) and kept; null on failure.
uint8_t *scratch_on(int dev) {
  static std::mutex mu;
  static uint8_t *ptr[64] = {};
  if (dev < 0 || dev >= 64) {
    fail(HAPI_E_DEVICE, "device %d outside the %d the static scratch supports", dev, 64);
    return nullptr;
  }
  std::lock_guard<std::mutex> g(mu);
  if (!ptr[dev]) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      fail(HAPI_E_DEVICE, "hipGetSymbolAddress(scratch) failed: %s", hipGetErrorString(e));
      return nullptr;
    }
    ptr[dev] = static_cast<uint8_t *>(p);
  }
  return ptr[dev];
}

// use_scratch: the workspace is the library's static scratch (desc->workspace
// and desc->workspace_bytes are ignored); partitions run one at a time on
// desc->stream with direct launches, so the call creates no HIP object.
int extract_range(const hapi_model_desc *desc, const void *weights, const void *images,
                  int32_t batch, int32_t start_layer, int32_t split_layer, void *out,
                  bool use_scratch = false) {
  Model m;
  int r = analyze(desc, m);
  if (r != HAPI_OK) return r;
  if (!images || !out) return fail(HAPI_E_INVAL, "images / out is NULL");
  if (batch < 1) return fail(HAPI_E_INVAL, "batch must be >= 1");
  if (split_layer < 0 || split_layer > (int)m.layers.size())
    return fail(HAPI_E_INVAL, "split %d outside [0, %d]", split_layer, (int)m.layers.size());
  if (start_layer < 0 || start_layer > split_layer)
    return fail(HAPI_E_INVAL, "start layer %d outside [0, %d]", start_layer, split_layer);
  hipStream_t s = static_cast<hipStream_t>(desc->stream);
  if (split_layer == start_layer) {  // nothing to run: the input is the result
    const int64_t bytes = (int64_t)batch * act_at(m, start_layer).elems() * m.esz;
    HIP_TRY(timed(s, F_COPY, 0.0, 2.0 * bytes, [&] { return launch_copy(images, out, bytes, s); }));
    return HAPI_OK;
  }
  if (!weights && m.packed_bytes > 0) return fail(HAPI_E_INVAL, "weights is NULL");
  if ((uintptr_t)weights % kAlign) return fail(HAPI_E_INVAL, "weights must be 256-byte aligned");
  if ((uintptr_t)images % m.esz || (uintptr_t)out % m.esz)
    return fail(HAPI_E_INVAL, "images / out are not aligned to the element size");
  const int chunk = chunk_for(desc, m, batch);
  if ((int64_t)chunk * max_tmp(m, split_layer) >= kIndexLimit)
    return fail(HAPI_E_UNSUPPORTED, "a partition of %d images exceeds 2^31 elements; lower chunk", chunk);
  if (use_scratch) {
    const int64_t need = workspace_for(m, split_layer, chunk, false, batch, 1);
    if (need > kScratchBytes)
      return fail(HAPI_E_NOMEM, "%lld workspace bytes needed, the static scratch holds %lld; "
                  "use hapi_extract with a caller workspace", (long long)need, (long long)kScratchBytes);
    int dev = -1, cur = -1;
    HIP_TRY(hipStreamGetDevice(s, &dev));
    HIP_TRY(hipGetDevice(&cur));
    if (dev != cur) return fail(HAPI_E_INVAL, "desc->stream belongs to device %d, current device is %d", dev, cur);
    uint8_t *ws = scratch_on(dev);
    if (!ws) return HAPI_E_DEVICE;
    return run_batch(desc, m, weights, images, batch, start_layer, split_layer, out, ws, chunk, 1, 1, nullptr);
  }
  const int lanes = lanes_for(desc, chunk, batch);
  const int64_t need = workspace_for(m, split_layer, chunk, false, batch, lanes);
  if (!desc->workspace || (int64_t)desc->workspace_bytes < need)
    return fail(HAPI_E_NOMEM, "workspace of %zu bytes, %lld needed", desc->workspace_bytes,
                (long long)need);
  if ((uintptr_t)desc->workspace % kAlign) return fail(HAPI_E_INVAL, "workspace must be 256-byte aligned");
  if (desc->direct == 0 && !stats_enabled())
    return run_planned(desc, m, weights, images, batch, start_layer, split_layer, out,
                       static_cast<uint8_t *>(desc->workspace), chunk, lanes);
  return run_batch(desc, m, weights, images, batch, start_layer, split_layer, out,
                   static_cast<uint8_t *>(desc->workspace), chunk, lanes, lanes, nullptr);
}

}  // namespace

extern "C" {

int hapi_extract(const hapi_model_desc *desc, const void *weights, const void *images,
                 int32_t batch, int32_t split_layer, void *out) {
  return extract_range(desc, weights, images, batch, 0, split_layer, out);
}

int hapi_extract_range(const hapi_model_desc *desc, const void *weights, const void *input,
                       int32_t batch, int32_t start_layer, int32_t end_layer, void *out) {
  return extract_range(desc, weights, input, batch, start_layer, end_layer, out);
}

int hapi_extract_noalloc(const hapi_model_desc *desc, const void *weights, const void *images,
                         int32_t batch, int32_t split_layer, void *out) {
  return extract_range(desc, weights, images, batch, 0, split_layer, out, true);
}

int hapi_profile_memory(const hapi_model_desc *desc, int32_t batch, int64_t *bytes) {
  Model m;
  const int r = analyze(desc, m);
  if (r != HAPI_OK) return r;
  if (batch < 1) return fail(HAPI_E_INVAL, "batch must be >= 1");
  if (!bytes) return fail(HAPI_E_INVAL, "bytes is NULL");
  const int n = (int)m.layers.size();
  const int chunk = chunk_for(desc, m, batch);
  if ((int64_t)chunk * max_tmp(m, n) >= kIndexLimit)
    return fail(HAPI_E_UNSUPPORTED, "a partition of %d images exceeds 2^31 elements; lower chunk", chunk);
  const int64_t images = (int64_t)batch * m.input.elems() * m.esz;
  for (int k = 0; k <= n; ++k) {
    const int64_t weights = k == 0 ? 0 : m.layers[k - 1].pk_end;
    const int64_t out = (int64_t)batch * act_at(m, k).elems() * m.esz;
    bytes[k] = weights + images + out + workspace_for(m, k, chunk, false, batch, lanes_for(desc, chunk, batch));
  }
  return HAPI_OK;
}

int hapi_profile_layers(const hapi_model_desc *desc, int32_t batch, int64_t *out_bytes,
                        float *out_us) {
  Model m;
  int r = analyze(desc, m);
  if (r != HAPI_OK) return r;
  if (batch < 1) return fail(HAPI_E_INVAL, "batch must be >= 1");
  if (!out_bytes && !out_us) return fail(HAPI_E_INVAL, "out_bytes and out_us are both NULL");
  const int n = (int)m.layers.size();
  if (out_bytes) {
    out_bytes[0] = (int64_t)batch * m.input.elems() * m.esz;
    for (int k = 1; k <= n; ++k) out_bytes[k] = (int64_t)batch * m.layers[k - 1].out.elems() * m.esz;
  }
  if (!out_us) return HAPI_OK;

  const int chunk = chunk_for(desc, m, batch);
  if ((int64_t)chunk * max_tmp(m, n) >= kIndexLimit)
    return fail(HAPI_E_UNSUPPORTED, "a partition of %d images exceeds 2^31 elements; lower chunk", chunk);
  const int64_t need = workspace_for(m, n, chunk, true, batch, 1);
  if (!desc->workspace || (int64_t)desc->workspace_bytes < need)
    return fail(HAPI_E_NOMEM, "workspace of %zu bytes, %lld needed", desc->workspace_bytes,
                (long long)need);
  if ((uintptr_t)desc->workspace % kAlign) return fail(HAPI_E_INVAL, "workspace must be 256-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(desc->stream);
  uint8_t *ws = static_cast<uint8_t *>(desc->workspace);
  uint8_t *pk = ws + lane_layout(m, n, chunk).bytes;
  uint8_t *img = pk + align_up(m.packed_bytes);
  // Synthetic model and inputs: small pseudo-random values in every parameter.
  for (const LayerPlan &lp : m.layers) {
    for (const ConvSpec &c : lp.convs) {
      HIP_TRY(launch_fill_pattern(m.bf16, pk + c.pk_w, (int64_t)c.cout * c.Kp, 0x1234u + (uint32_t)c.pk_w,
                                  1.0f / std::sqrt((float)c.K), s));
      HIP_TRY(launch_fill_pattern(false, pk + c.pk_b, c.cout, 0x77u + (uint32_t)c.pk_b, 0.05f, s));
    }
    for (const Extra &e : lp.extras)
      HIP_TRY(launch_fill_pattern(false, pk + e.pk, e.bn_affine ? 2 * e.n : e.n, 0x99u + (uint32_t)e.pk,
                                  0.05f, s));
  }
  HIP_TRY(launch_fill_pattern(m.bf16, img, (int64_t)batch * m.input.elems(), 0xabcdu, 1.0f, s));

  constexpr int kWarm = 5, kRuns = 20;
  std::vector<hipEvent_t> ev;
  std::vector<std::vector<float>> t(n, std::vector<float>());
  std::vector<float> acc(n);
  const int nchunks = (batch + chunk - 1) / chunk;
  const int per_pass = 2 * n * nchunks;
  // Partitions run one after another on desc->stream (each layer is timed
  // alone), with the tile choice of an extraction of this batch.
  const int route = lanes_for(desc, chunk, batch);
  ev.resize(per_pass);
  for (auto &e : ev) HIP_TRY(hipEventCreate(&e));
  int rc = HAPI_OK;
  for (int it = 0; it < kWarm + kRuns && rc == HAPI_OK; ++it) {
    int idx = 0;
    auto cb = [&](int layer, bool begin) {
      (void)layer;
      (void)begin;
      (void)hipEventRecord(ev[idx++], s);
    };
    rc = run_batch(desc, m, pk, img, batch, 0, n, nullptr, ws, chunk, 1, route, cb);
    if (rc != HAPI_OK) break;
    if (hipEventSynchronize(ev[idx - 1]) != hipSuccess) {
      rc = fail(HAPI_E_DEVICE, "hipEventSynchronize failed");
      break;
    }
    if (it < kWarm) continue;
    std::fill(acc.begin(), acc.end(), 0.0f);
    for (int ci = 0; ci < nchunks; ++ci)
      for (int k = 0; k < n; ++k) {
        float ms = 0.0f;
        (void)hipEventElapsedTime(&ms, ev[ci * 2 * n + 2 * k], ev[ci * 2 * n + 2 * k + 1]);
        acc[k] += ms;
      }
    for (int k = 0; k < n; ++k) t[k].push_back(acc[k]);
  }
  for (auto &e : ev) (void)hipEventDestroy(e);
  if (rc != HAPI_OK) return rc;
  out_us[0] = 0.0f;
  for (int k = 0; k < n; ++k) {
    std::vector<float> v = t[k];
    std::nth_element(v.begin(), v.begin() + v.size() / 2, v.end());
    out_us[k + 1] = v[v.size() / 2] * 1000.0f;
  }
  return HAPI_OK;
}

int hapi_stats_enable(int32_t enable) {
  std::lock_guard<std::mutex> g(g_stats_mu);
  for (StatRec &r : g_recs) {
    g_pool.push_back(r.a);
    g_pool.push_back(r.b);
  }
  g_recs.clear();
  g_stats_on = enable != 0;
  return HAPI_OK;
}

int hapi_stats_collect(hapi_kernel_stat *out, int32_t max_entries) {
  std::lock_guard<std::mutex> g(g_stats_mu);
  if (!out || max_entries < 0) return fail(HAPI_E_INVAL, "out is NULL");
  hapi_kernel_stat acc[F_COUNT];
  std::memset(acc, 0, sizeof acc);
  for (int f = 0; f < F_COUNT; ++f) std::snprintf(acc[f].name, sizeof acc[f].name, "%s", kFamily[f]);
  // Launch intervals relative to the first recorded start, per family, for
  // the time at least one launch of the family was running (launches of
  // partitions in flight on different streams overlap).
  std::vector<std::pair<float, float>> iv[F_COUNT];
  for (StatRec &r : g_recs) {
    if (hipEventSynchronize(r.b) != hipSuccess) return fail(HAPI_E_DEVICE, "hipEventSynchronize failed");
    float ms = 0.0f, t0 = 0.0f;
    (void)hipEventElapsedTime(&ms, r.a, r.b);
    (void)hipEventElapsedTime(&t0, g_recs.front().a, r.a);
    acc[r.fam].launches += 1;
    acc[r.fam].total_ms += ms;
    acc[r.fam].flops += r.flops;
    acc[r.fam].bytes += r.bytes;
    iv[r.fam].emplace_back(t0, t0 + ms);
  }
  for (int f = 0; f < F_COUNT; ++f) {
    std::sort(iv[f].begin(), iv[f].end());
    double busy = 0.0, lo = 0.0, hi = -1e30;
    for (const auto &x : iv[f]) {
      if (x.first > hi) {
        if (hi > lo) busy += hi - lo;
        lo = x.first;
        hi = x.second;
      } else {
        hi = std::max(hi, (double)x.second);
      }
    }
    if (!iv[f].empty() && hi > lo) busy += hi - lo;
    acc[f].busy_ms = busy;
  }
  int nout = 0;
  for (int f = 0; f < F_COUNT; ++f) {
    if (acc[f].launches == 0) continue;
    if (nout < max_entries) out[nout] = acc[f];
    ++nout;
  }
  return nout;
}

const char *hapi_last_error(void) { return g_err.c_str(); }

}  // extern "C"
