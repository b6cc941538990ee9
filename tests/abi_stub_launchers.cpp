// Stand-ins for the kernel launchers, linked only into the sanitizer build of
// the C ABI layer that the CPU tests load (tests/test_abi_sanitized.py).
// The ABI checks there never reach a launch; if one did, it fails loudly.
#include "launch.hpp"

namespace vidax {
namespace {
hipError_t no_launch() { return hipErrorInvalidDeviceFunction; }
}  // namespace

hipError_t launch_rope3d(const uint16_t*, uint16_t*, int, int, int, const RopeParams&, hipStream_t) {
  return no_launch();
}
hipError_t launch_attn_bwd(const uint16_t*, const uint16_t*, const uint16_t*, const uint16_t*, const uint16_t*,
                           const float*, float*, size_t, uint16_t*, uint16_t*, uint16_t*, int, int, int, int, float,
                           const int32_t*, hipStream_t) {
  return no_launch();
}
int device_cu_count() { return 256; }
hipError_t launch_attn_bwd_noalloc(const uint16_t*, const uint16_t*, const uint16_t*, const uint16_t*,
                                   const uint16_t*, const float*, uint16_t*, uint16_t*, uint16_t*, int, int, int,
                                   int, float, const int32_t*, hipStream_t) {
  return no_launch();
}
hipError_t launch_qk_norm(const uint16_t*, uint16_t*, const float*, float, int, int, int, const RopeParams&,
                          hipStream_t) {
  return no_launch();
}
hipError_t launch_attn_naive(const uint16_t*, const uint16_t*, const uint16_t*, uint16_t*, float*, int, int, int,
                             int, float, const int32_t*, const RopeParams&, hipStream_t) {
  return no_launch();
}
bool attn_rope_supported(const RopeParams& rp) {
  if (!rp.enabled) return true;
  if (rp.pair_mode != 0) return false;
  if (rp.gw > kAttnGridHWMax || rp.gh > kAttnGridHWMax || rp.gt > kAttnGridTMax) return false;
  const long entries =
      (long)(rp.gt + 1) * (rp.dt / 2) + (long)(rp.gh + 1) * (rp.dh / 2) + (long)(rp.gw + 1) * (rp.dw / 2);
  return entries <= kAttnTableMax;
}
hipError_t launch_na3d_fwd(const uint16_t*, const uint16_t*, const uint16_t*, uint16_t*, float*, int, int, int, int,
                           int, int, int, int, int, float, hipStream_t) {
  return no_launch();
}
hipError_t launch_attn_fwd(const uint16_t*, const uint16_t*, const uint16_t*, uint16_t*, float*, int, int, int, int,
                           float, const int32_t*, const RopeParams&, hipStream_t) {
  return no_launch();
}
hipError_t launch_xattn_fwd(const uint16_t*, const uint16_t*, const uint16_t*, uint16_t*, float*, int, int, int, int,
                            float, const int32_t*, int, hipStream_t) {
  return no_launch();
}
hipError_t launch_qkv_proj(const uint16_t*, const uint16_t*, const float*, const float*, const float*, float,
                           uint16_t*, uint16_t*, uint16_t*, int, int, int, int, const RopeParams&, hipStream_t) {
  return no_launch();
}
}  // namespace vidax
