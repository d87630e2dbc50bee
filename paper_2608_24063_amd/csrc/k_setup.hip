// k_setup.hip -- moves the host-built prune plan (layer pointer table, budgets,
// offsets) into the device workspace.  The plan travels as kernel arguments,
// at most kUploadBytes per launch, so no host buffer has to outlive the call
// and nothing is copied through pageable memory.
#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

constexpr int kUploadWords = 480;  // 1920-byte payload per launch

struct UploadChunk {
  uint32_t words;
  uint32_t pad;
  uint32_t data[kUploadWords];
};

__global__ __launch_bounds__(256) void k_upload(uint32_t *dst, UploadChunk c) {
  for (uint32_t i = threadIdx.x; i < c.words; i += 256) dst[i] = c.data[i];
}

}  // namespace

hipError_t launch_upload(uint8_t *dst, const uint8_t *src, size_t bytes, uint32_t * /*zero*/,
                         size_t /*zero_words*/, hipStream_t st) {
  // `bytes` is a multiple of 4 (the plan is built from 4- and 8-byte fields).
  const size_t words = bytes / 4;
  for (size_t w0 = 0; w0 < words; w0 += kUploadWords) {
    UploadChunk c;
    c.words = (uint32_t)((words - w0) < (size_t)kUploadWords ? (words - w0) : kUploadWords);
    c.pad = 0;
    __builtin_memcpy(c.data, src + w0 * 4, (size_t)c.words * 4);
    hipLaunchKernelGGL(k_upload, dim3(1), dim3(256), 0, st, reinterpret_cast<uint32_t *>(dst) + w0, c);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace vc
