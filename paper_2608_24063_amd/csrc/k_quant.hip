// k_quant.hip -- 4-bit cache rows: each row's channels in groups of 32, a
// group keeping fp32 (scale, lo) = ((max - min) / 15, min) and 4-bit codes
// clamp(rint((x - lo) / scale), 0, 15).  Every step is IEEE fp32 (correctly
// rounded division), so the integer codes are fixed bit for bit.  This is the
// reading taken of the 4-bit KV-cache quantisation the paper combines with
// the pruned cache (it names the quantisers but does not define them).
#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

// One thread per (row, group): the group's 32 bf16 values are consecutive, so
// thread i reads values [32 i, 32 i + 32) and writes code bytes [16 i, 16 i + 16)
// and meta[i].
__global__ __launch_bounds__(256) void k_quant_rows(int64_t total, const uint16_t *src, uint8_t *codes,
                                                    float2 *meta) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const uint16_t *x = src + i * 32;
  float v[32];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const u32x4 w = ld16(x + 8 * j);
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      v[8 * j + 2 * k] = bf16_lo(ws[k]);
      v[8 * j + 2 * k + 1] = bf16_hi(ws[k]);
    }
  }
  float lo = v[0], hi = v[0];
#pragma unroll
  for (int c = 1; c < 32; ++c) {
    lo = v[c] < lo ? v[c] : lo;
    hi = v[c] > hi ? v[c] : hi;
  }
  lo = lo + 0.f;  // -0 -> +0, so the stored offset does not depend on which zero came first
  const float scale = __fdiv_rn(hi - lo, 15.f);
  uint32_t word[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int c = 0; c < 32; ++c) {
    uint32_t code = 0u;
    if (scale > 0.f) {
      const float t = rintf(__fdiv_rn(v[c] - lo, scale));
      code = (uint32_t)fminf(fmaxf(t, 0.f), 15.f);
    }
    word[c / 8] |= code << (4 * (c % 8));
  }
  st16(codes + i * 16, u32x4{word[0], word[1], word[2], word[3]});
  stg(meta + i, make_float2(scale, lo));
}

}  // namespace

hipError_t launch_quant_rows(int32_t d, int64_t rows, const uint16_t *src, uint8_t *codes, float2 *meta,
                             hipStream_t st) {
  const int64_t total = rows * (d / 32);
  if (total == 0) return hipSuccess;
  const int64_t grid = (total + 255) / 256;
  hipLaunchKernelGGL(k_quant_rows, dim3((uint32_t)grid), dim3(256), 0, st, total, src, codes, meta);
  return hipGetLastError();
}

}  // namespace vc
