// k_select.hip -- keep / drop partition of PruneKV (Algorithm 1, Step 1 and
// Step 3): one ranking per (layer, sequence, kv head) ordered by score
// descending then token index ascending; the first k tokens are kept, the next
// n_surv - k are dropped (their values get fused), the rest are discarded.
//
// One workgroup per unit; each thread holds a contiguous run of PER scores in
// registers.  Scores are non-negative fp32, so their bit patterns order like
// the values.  The k-th largest bit pattern is found exactly by a 31-step
// bisection over the bit positions (both cuts in the same loop; counts come
// from wave ballots and scalar popcounts), ties at the threshold go to the
// lowest indices, and a block-wide prefix sum compacts kept and dropped
// indices in ascending token order.
#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

// Exclusive prefix over the block of four counters per thread, plus totals.
template <int THREADS>
__device__ __forceinline__ void block_scan4(const uint32_t v[4], uint32_t excl[4], uint32_t tot[4],
                                            uint4 *sh) {
  const int tid = threadIdx.x, lane = tid & 63;
  sh[tid] = make_uint4(v[0], v[1], v[2], v[3]);
  __syncthreads();
  if (tid < 64) {
    constexpr int per = THREADS / 64;
    uint4 run = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int i = 0; i < per; ++i) {
      const uint4 x = sh[lane * per + i];
      run.x += x.x; run.y += x.y; run.z += x.z; run.w += x.w;
    }
    uint4 inc = run;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t a = __shfl_up(inc.x, off, 64), b = __shfl_up(inc.y, off, 64);
      const uint32_t c = __shfl_up(inc.z, off, 64), d = __shfl_up(inc.w, off, 64);
      if (lane >= off) { inc.x += a; inc.y += b; inc.z += c; inc.w += d; }
    }
    uint4 base = make_uint4(inc.x - run.x, inc.y - run.y, inc.z - run.z, inc.w - run.w);
#pragma unroll
    for (int i = 0; i < per; ++i) {
      const uint4 x = sh[lane * per + i];
      sh[lane * per + i] = base;
      base.x += x.x; base.y += x.y; base.z += x.z; base.w += x.w;
    }
    if (lane == 63) sh[THREADS] = inc;
  }
  __syncthreads();
  const uint4 e = sh[tid], t = sh[THREADS];
  excl[0] = e.x; excl[1] = e.y; excl[2] = e.z; excl[3] = e.w;
  tot[0] = t.x; tot[1] = t.y; tot[2] = t.z; tot[3] = t.w;
  __syncthreads();
}

__device__ __forceinline__ uint32_t count_wave(bool pred) {
  return (uint32_t)__builtin_popcountll(__builtin_amdgcn_ballot_w64(pred));
}

template <int THREADS, int PER>
__global__ __launch_bounds__(THREADS) void k_select(PrunePlan p) {
  constexpr int kWaves = THREADS / 64;
  __shared__ uint32_t red[2][kWaves][2];
  __shared__ uint4 scan_sh[THREADS + 1];

  const int u = blockIdx.x;  // ((l * B) + b) * Hkv + g, l < h
  const int g = u % p.Hkv;
  const int b = (u / p.Hkv) % p.B;
  const int l = u / (p.Hkv * p.B);
  const int nsv = ldg(p.ns + b * p.L + l);
  if (nsv == 0) return;
  const int n = ldg(p.nb + b);
  const int k = ldg(p.kk + b * p.L + l);
  const int r = nsv - k;
  const int64_t toff = ldg(p.toff + b);

  const float *S = p.mode ? p.gs + toff
                          : p.S + (int64_t)l * p.Ntot * p.Hkv + toff * p.Hkv + (int64_t)g * n;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int per = (n + THREADS - 1) / THREADS;  // <= PER
  const int v0 = tid * per;
  const int cnt = max(0, min(per, n - v0));

  // Bit patterns of non-negative floats order like the values.  A set sign
  // bit (only possible from non-finite inputs) is mapped to the top of the
  // 31-bit range so every count below stays consistent.  Slots past the
  // thread's run hold 0, which no bisection candidate (>= 1) counts.
  uint32_t key[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const uint32_t x = (i < cnt) ? __float_as_uint(ldg(S + v0 + i)) : 0u;
    key[i] = (x & 0x80000000u) ? 0x7FFFFFFFu : x;
  }

  // Bisection for the k-th and n_surv-th largest keys.
  uint32_t tk = 0, ts = 0;
  for (int bit = 30, it = 0; bit >= 0; --bit, ++it) {
    const uint32_t ck = tk | (1u << bit), cs = ts | (1u << bit);
    uint32_t nk = 0, nsu = 0;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      nk += count_wave(key[i] >= ck);
      nsu += count_wave(key[i] >= cs);
    }
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
  for (int i = 0; i < PER; ++i)
    if (i < cnt) {
      c4[0] += key[i] > tk;
      c4[1] += key[i] == tk;
      c4[2] += key[i] > ts;
      c4[3] += key[i] == ts;
    }
  uint32_t ex[4], tot[4];
  block_scan4<THREADS>(c4, ex, tot, scan_sh);
  const uint32_t need_k = k > 0 ? (uint32_t)k - tot[0] : 0u;
  const uint32_t need_s = (uint32_t)nsv - tot[2];
  uint32_t ek = ex[1], es = ex[3];

  uint32_t keepmask[(PER + 31) / 32], dropmask[(PER + 31) / 32];
#pragma unroll
  for (int j = 0; j < (PER + 31) / 32; ++j) keepmask[j] = dropmask[j] = 0u;
  uint32_t nkeep = 0, ndrop = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i)
    if (i < cnt) {
      const uint32_t x = key[i];
      bool kp = false;
      if (k > 0) {
        kp = x > tk || (x == tk && ek < need_k);
        if (x == tk) ++ek;
      }
      const bool sv = x > ts || (x == ts && es < need_s);
      if (x == ts) ++es;
      if (kp) { keepmask[i / 32] |= 1u << (i % 32); ++nkeep; }
      else if (sv) { dropmask[i / 32] |= 1u << (i % 32); ++ndrop; }
    }

  const uint32_t c2[4] = {nkeep, ndrop, 0, 0};
  block_scan4<THREADS>(c2, ex, tot, scan_sh);

  int32_t *idx = reinterpret_cast<int32_t *>(ldg(p.lp + LP_IDX * p.L + l)) +
                 ldg(p.orow + l * (p.B + 1) + b) + (int64_t)g * k;
  int32_t *drop = reinterpret_cast<int32_t *>(ldg(p.lp + LP_DROP * p.L + l)) +
                  ldg(p.drow + l * (p.B + 1) + b) + (int64_t)g * r;
  uint32_t pk = ex[0], pd = ex[1];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    if ((keepmask[i / 32] >> (i % 32)) & 1u) {
      if (pk < (uint32_t)k) stg(idx + pk, (int32_t)(v0 + i));
      ++pk;
    }
    if ((dropmask[i / 32] >> (i % 32)) & 1u) {
      if (pd < (uint32_t)r) stg(drop + pd, (int32_t)(v0 + i));
      ++pd;
    }
  }
}

}  // namespace

hipError_t launch_select(const PrunePlan &p, hipStream_t st) {
  const uint32_t grid = (uint32_t)p.h * p.B * p.Hkv;
  if (grid == 0) return hipSuccess;
  // Smallest block that holds the longest sequence in registers.
  if (p.nmax <= 256 * 16)
    hipLaunchKernelGGL((k_select<256, 16>), dim3(grid), dim3(256), 0, st, p);
  else if (p.nmax <= 256 * 32)
    hipLaunchKernelGGL((k_select<256, 32>), dim3(grid), dim3(256), 0, st, p);
  else if (p.nmax <= 512 * 32)
    hipLaunchKernelGGL((k_select<512, 32>), dim3(grid), dim3(512), 0, st, p);
  else
    hipLaunchKernelGGL((k_select<1024, 32>), dim3(grid), dim3(1024), 0, st, p);
  return hipGetLastError();
}

}  // namespace vc
