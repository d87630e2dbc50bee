// k_select.hip -- keep / drop partition of PruneKV (Algorithm 1, Step 1 and
// Step 3): one ranking per (layer, sequence, kv head) ordered by score
// descending then token index ascending; the first k tokens are kept, the next
// n_surv - k are dropped (their values get fused), the rest are discarded.
//
// One 1024-thread workgroup per unit.  Scores are non-negative fp32, so their
// bit patterns order like the values.  The k-th largest bit pattern is found
// exactly by a 31-step bisection over the bit positions (both cuts in the same
// loop), ties at the threshold go to the lowest indices, and a block-wide
// prefix sum compacts kept and dropped indices in ascending token order.
#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

constexpr int kWaves = kSelectThreads / 64;

// Exclusive prefix over the block of four counters; returns the totals too.
__device__ __forceinline__ void block_scan4(uint32_t v[4], uint32_t excl[4], uint32_t tot[4],
                                            uint32_t (*sh)[4]) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  uint32_t inc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint32_t x = v[j];
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      uint32_t y = __shfl_up(x, off, 64);
      if (lane >= off) x += y;
    }
    inc[j] = x;
  }
  if (lane == 63) {
#pragma unroll
    for (int j = 0; j < 4; ++j) sh[w][j] = inc[j];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint32_t before = 0, all = 0;
    for (int i = 0; i < kWaves; ++i) {
      uint32_t t = sh[i][j];
      if (i < w) before += t;
      all += t;
    }
    excl[j] = before + inc[j] - v[j];
    tot[j] = all;
  }
  __syncthreads();
}

__device__ __forceinline__ uint32_t wave_sum(uint32_t x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

__global__ __launch_bounds__(kSelectThreads) void k_select(PrunePlan p) {
  __shared__ uint32_t red[2][kWaves][2];
  __shared__ uint32_t scan_sh[kWaves][4];

  const int u = blockIdx.x;  // ((l * B) + b) * Hkv + g, l < h
  const int g = u % p.Hkv;
  const int b = (u / p.Hkv) % p.B;
  const int l = u / (p.Hkv * p.B);
  const int n = p.nb[b];
  const int k = p.kk[b * p.L + l];
  const int nsv = p.ns[b * p.L + l];
  const int r = nsv - k;
  if (nsv == 0) return;

  const float *S = p.mode ? p.gs + p.toff[b]
                          : p.S + (int64_t)l * p.Ntot * p.Hkv + (int64_t)p.toff[b] * p.Hkv +
                                (int64_t)g * n;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int per = (n + kSelectThreads - 1) / kSelectThreads;  // <= kSelectPerThread
  const int v0 = tid * per;
  const int cnt = max(0, min(per, n - v0));

  // Bit patterns of non-negative floats order like the values.  A set sign
  // bit (only possible from non-finite inputs) is mapped to the top of the
  // 31-bit range so every count below stays consistent.
  uint32_t key[kSelectPerThread];
#pragma unroll
  for (int i = 0; i < kSelectPerThread; ++i) {
    const uint32_t x = (i < cnt) ? __float_as_uint(S[v0 + i]) : 0u;
    key[i] = (x & 0x80000000u) ? 0x7FFFFFFFu : x;
  }

  // Bisection for the k-th and n_surv-th largest keys.
  uint32_t tk = 0, ts = 0;
  for (int bit = 30, it = 0; bit >= 0; --bit, ++it) {
    const uint32_t ck = tk | (1u << bit), cs = ts | (1u << bit);
    uint32_t nk = 0, nsu = 0;
#pragma unroll
    for (int i = 0; i < kSelectPerThread; ++i)
      if (i < cnt) {
        nk += key[i] >= ck;
        nsu += key[i] >= cs;
      }
    nk = wave_sum(nk);
    nsu = wave_sum(nsu);
    if (lane == 0) {
      red[it & 1][w][0] = nk;
      red[it & 1][w][1] = nsu;
    }
    __syncthreads();
    uint32_t tnk = 0, tns = 0;
#pragma unroll
    for (int i = 0; i < kWaves; ++i) {
      tnk += red[it & 1][i][0];
      tns += red[it & 1][i][1];
    }
    if (tnk >= (uint32_t)k) tk = ck;
    if (tns >= (uint32_t)nsv) ts = cs;
  }

  // Counts above and at each threshold; ties fill in ascending index order.
  uint32_t c4[4] = {0, 0, 0, 0};
#pragma unroll
  for (int i = 0; i < kSelectPerThread; ++i)
    if (i < cnt) {
      c4[0] += key[i] > tk;
      c4[1] += key[i] == tk;
      c4[2] += key[i] > ts;
      c4[3] += key[i] == ts;
    }
  uint32_t ex[4], tot[4];
  block_scan4(c4, ex, tot, scan_sh);
  const uint32_t need_k = k > 0 ? (uint32_t)k - tot[0] : 0u;
  const uint32_t need_s = (uint32_t)nsv - tot[2];
  uint32_t ek = ex[1], es = ex[3];

  uint32_t keepmask = 0, dropmask = 0;
#pragma unroll
  for (int i = 0; i < kSelectPerThread; ++i)
    if (i < cnt) {
      const uint32_t x = key[i];
      bool kp = false, sv;
      if (k > 0) {
        kp = x > tk || (x == tk && ek < need_k);
        if (x == tk) ++ek;
      }
      sv = x > ts || (x == ts && es < need_s);
      if (x == ts) ++es;
      if (kp) keepmask |= 1u << i;
      else if (sv) dropmask |= 1u << i;
    }

  uint32_t c2[4] = {(uint32_t)__popc(keepmask), (uint32_t)__popc(dropmask), 0, 0};
  block_scan4(c2, ex, tot, scan_sh);

  int32_t *idx = reinterpret_cast<int32_t *>(p.lp[LP_IDX * p.L + l]) + p.orow[l * (p.B + 1) + b] +
                 (int64_t)g * k;
  int32_t *drop = reinterpret_cast<int32_t *>(p.lp[LP_DROP * p.L + l]) +
                  p.drow[l * (p.B + 1) + b] + (int64_t)g * r;
  uint32_t pk = ex[0], pd = ex[1];
#pragma unroll
  for (int i = 0; i < kSelectPerThread; ++i) {
    if ((keepmask & (1u << i)) && pk < (uint32_t)k) idx[pk++] = v0 + i;
    if ((dropmask & (1u << i)) && pd < (uint32_t)r) drop[pd++] = v0 + i;
  }
}

}  // namespace

hipError_t launch_select(const PrunePlan &p, hipStream_t st) {
  const uint32_t grid = (uint32_t)p.h * p.B * p.Hkv;
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(k_select, dim3(grid), dim3(kSelectThreads), 0, st, p);
  return hipGetLastError();
}

}  // namespace vc
