// k_setup.hip -- moves the host-built prune plan (layer pointer table, budgets,
// offsets, fusion unit records) into the device workspace.  The plan travels
// as kernel arguments, so no host buffer has to outlive the call and nothing
// is copied through pageable memory.  Its first 30 KB ride with the score
// statistics launch; this kernel carries the rest (no launch for the shapes
// seen in practice).
#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

template <uint32_t W>
__global__ __launch_bounds__(256) void k_upload(uint32_t *dst, UploadChunk<W> c) {
  const uint32_t i0 = blockIdx.x * 1024;
  const uint32_t i1 = min(c.words, i0 + 1024);
  for (uint32_t i = i0 + threadIdx.x; i < i1; i += 256) dst[i] = c.data[i];
}

template <uint32_t W>
hipError_t upload_chunk(uint32_t *dst, const uint8_t *src, uint32_t words, hipStream_t st) {
  UploadChunk<W> c;
  c.words = words;
  c.pad = 0;
  __builtin_memcpy(c.data, src, (size_t)words * 4);
  hipLaunchKernelGGL(k_upload<W>, dim3((words + 1023) / 1024), dim3(256), 0, st, dst, c);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_upload(uint8_t *dst, const uint8_t *src, size_t bytes, hipStream_t st) {
  // `bytes` is a multiple of 4 (the plan is built from 4- and 8-byte fields).
  const size_t words = bytes / 4;
  for (size_t w0 = 0; w0 < words; w0 += kChunkWords) {
    const uint32_t n = (uint32_t)((words - w0) < (size_t)kChunkWords ? (words - w0) : kChunkWords);
    uint32_t *d = reinterpret_cast<uint32_t *>(dst) + w0;
    const uint8_t *s = src + w0 * 4;
    const hipError_t e = n <= kChunkWordsSmall ? upload_chunk<kChunkWordsSmall>(d, s, n, st)
                         : n <= kChunkWordsMid ? upload_chunk<kChunkWordsMid>(d, s, n, st)
                                               : upload_chunk<kChunkWords>(d, s, n, st);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace vc
