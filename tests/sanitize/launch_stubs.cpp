// launch_stubs.cpp -- host-only stand-ins for the kernel launchers of
// libviscache, for the sanitizer build of its host code (no GPU, no device
// code).  Each stub reads every host byte the real launcher would copy into
// its kernel arguments, so an out-of-bounds plan is caught by the address
// sanitizer, then reports a failed launch; the driver expects VC_ERR_HIP
// from every call that passes the host checks.
#include <cstring>

#include "../../paper_2608_24063_amd/csrc/vc_internal.h"

namespace vc {

volatile uint32_t g_sink;

static hipError_t touch(const void *p, size_t bytes) {
  uint32_t acc = 0;
  const uint8_t *b = static_cast<const uint8_t *>(p);
  for (size_t i = 0; i < bytes; ++i) acc += b[i];
  g_sink = acc;
  return hipErrorInvalidValue;
}

hipError_t launch_upload(uint8_t *, const uint8_t *src, size_t bytes, hipStream_t) { return touch(src, bytes); }
hipError_t launch_score_stats(const PrunePlan &p, uint32_t *, const uint8_t *src, uint32_t words, hipStream_t) {
  if (words > kChunkWords) return hipErrorInvalidValue;
  (void)touch(&p, sizeof(p));
  return touch(src, (size_t)words * 4);
}
hipError_t launch_score_colsum(const PrunePlan &p, hipStream_t) { return touch(&p, sizeof(p)); }
hipError_t launch_score_global(const PrunePlan &p, hipStream_t) { return touch(&p, sizeof(p)); }
hipError_t launch_pscore(const PrunePlan &p, uint32_t *, const uint8_t *src, uint32_t words, hipStream_t) {
  if (words > kChunkWords) return hipErrorInvalidValue;
  (void)touch(&p, sizeof(p));
  return touch(src, (size_t)words * 4);
}
hipError_t launch_pscore_reduce(const PrunePlan &p, hipStream_t) { return touch(&p, sizeof(p)); }
hipError_t launch_select(const PrunePlan &p, hipStream_t) { return touch(&p, sizeof(p)); }
hipError_t launch_fuse(const PrunePlan &p, hipStream_t) { return touch(&p, sizeof(p)); }
hipError_t launch_append(int32_t, int32_t, uint16_t *, uint16_t *, const int64_t *, const int32_t *, int32_t *,
                         const uint16_t *, const uint16_t *, hipStream_t) {
  return hipErrorInvalidValue;
}
hipError_t launch_decode(const DecodePlan &p, hipStream_t) { return touch(&p, sizeof(p)); }
hipError_t launch_decode_step(const DecodePlan &p, hipStream_t) { return touch(&p, sizeof(p)); }
hipError_t launch_decode_step_q4(const DecodePlan &p, hipStream_t) { return touch(&p, sizeof(p)); }
hipError_t launch_decode_planned(const DecodePlan &p, bool, hipStream_t) { return touch(&p, sizeof(p)); }
hipError_t noalloc_scratch(uint8_t **out, hipStream_t) {
  *out = nullptr;
  return hipErrorInvalidValue;
}
hipError_t launch_quant_rows(int32_t, int64_t, const uint16_t *, uint8_t *, float2 *, hipStream_t) {
  return hipErrorInvalidValue;
}

}  // namespace vc
