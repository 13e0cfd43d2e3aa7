// Host-only stand-ins for the library's kernel launchers, so that the host
// runtime (api.cpp, split.cpp) links into a sanitizer build without device
// code.  The sanitizer driver only calls entry points that launch nothing;
// any launch reaching these fails loudly.
#include "internal.h"

namespace hapi {
namespace {
hipError_t none() { return hipErrorNotSupported; }
}  // namespace
hipError_t launch_conv_bf16(const ConvArgs &, Loader, hipStream_t) { return none(); }
hipError_t launch_conv_f32(const ConvArgs &, Loader, hipStream_t) { return none(); }
hipError_t launch_f32_split_reduce(const ConvArgs &, hipStream_t) { return none(); }
hipError_t launch_maxpool(bool, const void *, void *, int, int, int, int, int, int, int, int, int, hipStream_t) {
  return none();
}
hipError_t launch_avgpool(bool, const void *, void *, int, int, int, int, int, int, int, int, hipStream_t) {
  return none();
}
hipError_t launch_nhwc_to_nchw(bool, const void *, void *, int, int, int, hipStream_t) { return none(); }
hipError_t launch_nchw_to_nhwc(bool, const void *, void *, int, int, int, hipStream_t) { return none(); }
hipError_t launch_copy(const void *, void *, size_t, hipStream_t) { return none(); }
hipError_t launch_fill_pattern(bool, void *, int64_t, uint32_t, float, hipStream_t) { return none(); }
hipError_t launch_tokens(const void *, const float *, const float *, void *, int, int, int, hipStream_t) {
  return none();
}
hipError_t launch_layernorm(const void *, const float *, const float *, void *, int64_t, int, float, hipStream_t) {
  return none();
}
hipError_t launch_attention(const void *, void *, int, int, int, int, hipStream_t) { return none(); }
hipError_t launch_pack_conv(bool, const float *, const float *, const float *, const float *, const float *,
                            const float *, int, int, int, int, int, int, int, bool, PackOrder, void *, float *,
                            hipStream_t) {
  return none();
}
hipError_t launch_nchw_to_nhwc8(const void *, void *, int, int, int, int, hipStream_t) { return none(); }
hipError_t launch_space_to_depth(const void *, void *, int, int, int, int, int, int, int, hipStream_t) {
  return none();
}
bool conv3x3_c64_supported(int, int, int, int, int, int, int, int, int, int) { return false; }
hipError_t launch_conv3x3_c64(const void *, const void *, int, const float *, const void *, int, void *, int, int,
                              int, int, bool, int, hipStream_t, const void *, int, const float *, bool) {
  return none();
}
bool conv3x3_c64_pool_supported(int, int, int) { return false; }
bool conv3x3_c64_expand_supported(int, int, int, int, int) { return false; }
bool conv_first_supported(const ConvArgs &) { return false; }
bool bottleneck_link_supported(int, int, int, int, int) { return false; }
hipError_t launch_bottleneck_link(const void *, const void *, const float *, const void *, void *, const void *,
                                  const float *, void *, int, int, int, int, hipStream_t) {
  return none();
}
hipError_t launch_conv_first(const ConvArgs &, hipStream_t) { return none(); }
int cu_count() { return 256; }
bool stem_pool_supported(int, int, int, int, int, int, int, int) { return false; }
hipError_t launch_stem_pool_bf16(const void *, const void *, int, const float *, void *, int, int, int, int, int, int,
                                 int, int, int, hipStream_t) {
  return none();
}
hipError_t launch_copy_f32(const float *, float *, int64_t, hipStream_t) { return none(); }
hipError_t launch_channel_copy(const void *, void *, int64_t, int, int, int, int, hipStream_t) { return none(); }
hipError_t launch_affine(const void *, const float *, const float *, void *, int64_t, int, int, bool, hipStream_t) {
  return none();
}
hipError_t launch_pack_affine(const float *, int, float *, float *, hipStream_t) { return none(); }
}  // namespace hapi
