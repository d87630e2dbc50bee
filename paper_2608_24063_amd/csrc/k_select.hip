// k_select.hip -- keep / drop partition of PruneKV (Algorithm 1, Step 1 and
// Step 3): one ranking per (layer, sequence, kv head) ordered by score
// descending then token index ascending; the first k tokens are kept, the next
// n_surv - k are dropped (their values get fused), the rest are discarded.
//
// One workgroup per unit (256 to 1024 threads, by the longest sequence); each
// thread holds a contiguous run of up to PER scores in registers.  Scores are
// non-negative fp32, so their bit patterns order like the values.  The k-th
// and n_surv-th largest bit patterns are found exactly by a most-significant-
// digit radix select over the 31 value bits (digits of 8, 8, 8 and 7 bits,
// both cuts in the same passes): each wave counts the digits of the keys that
// still match a cut's prefix into its own LDS histogram, and two waves scan
// the summed histograms for the bin holding the wanted rank.  Ties at a
// threshold go to the lowest indices, and block-wide prefix sums (DPP wave
// scans) compact kept and dropped indices in ascending token order.
#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

// Exclusive prefix over the block of four counters per thread, plus totals.
template <int kWaves>
__device__ __forceinline__ void block_scan4(const uint32_t v[4], uint32_t excl[4], uint32_t tot[4],
                                            uint32_t (*wt)[kWaves]) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  uint32_t inc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    inc[c] = wave_incl_scan(v[c]);
    if (lane == 63) wt[c][w] = inc[c];
  }
  __syncthreads();
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    uint32_t before = 0, all = 0;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) {
      const uint32_t x = wt[c][q];
      before += q < w ? x : 0u;
      all += x;
    }
    excl[c] = before + inc[c] - v[c];
    tot[c] = all;
  }
  __syncthreads();
}

// One radix pass for both cuts: digits of `wd` bits at bit `sh`.  On entry
// pre[c] holds the cut's value bits above the digit and rank[c] the wanted
// rank (1-based, descending) among the keys sharing them; on exit the digit
// is fixed and the rank is relative to it.  A rank of 0 (nothing wanted)
// stays 0.
template <int kWaves, int PER>
__device__ __forceinline__ void radix_pass(const uint32_t (&key)[PER], int cnt, int sh, int wd, uint32_t (&pre)[2],
                                           uint32_t (&rank)[2], uint32_t (*hist)[2][256], uint32_t (*res)[2]) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  // This wave's histogram (the previous pass's scans finished before the
  // barrier that ended it).
#pragma unroll
  for (int i = 0; i < 8; ++i) (&hist[w][0][0])[lane + 64 * i] = 0u;
  __builtin_amdgcn_wave_barrier();
  const int top = sh + wd;
  const uint32_t dm = (1u << wd) - 1u;
  const uint32_t p0 = top >= 31 ? 0u : pre[0] >> top, p1 = top >= 31 ? 0u : pre[1] >> top;
  // While both cuts share their prefix (always in the first pass), one
  // histogram serves both.
  const bool same = p0 == p1;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    if (i < cnt) {
      const uint32_t hi = top >= 31 ? 0u : key[i] >> top;
      const uint32_t dg = (key[i] >> sh) & dm;
      if (hi == p0) atomicAdd(&hist[w][0][dg], 1u);
      if (!same && hi == p1) atomicAdd(&hist[w][1][dg], 1u);
    }
  }
  __syncthreads();
  if (w < 2) {
    // Wave c scans cut c: lane l owns bins 255-4l .. 252-4l (descending).
    const int c = w, hc = same ? 0 : w;
    uint32_t b4[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int q = 0; q < kWaves; ++q) {
      const uint4 h = *reinterpret_cast<const uint4 *>(&hist[q][hc][252 - 4 * lane]);
      b4[0] += h.w;
      b4[1] += h.z;
      b4[2] += h.y;
      b4[3] += h.x;
    }
    const uint32_t tot = (b4[0] + b4[1]) + (b4[2] + b4[3]);
    const uint32_t incl = wave_incl_scan(tot);
    const uint32_t excl = incl - tot;
    const uint32_t r = rank[c];
    const uint64_t hit = __builtin_amdgcn_ballot_w64(r > 0 && excl < r && r <= incl);
    if (hit) {
      const int src = __builtin_ctzll(hit);
      if (lane == src) {
        uint32_t cum = excl, dg = 0u, nr = 0u;
#pragma unroll
        for (int j = 3; j >= 0; --j) {  // pick the first bin (descending) that reaches the rank
          const uint32_t j2 = 3 - j;
          if (cum < r && r <= cum + b4[j2] && nr == 0u) {
            dg = 255u - 4u * lane - j2;
            nr = r - cum;
          }
          cum += b4[j2];
        }
        res[c][0] = dg;
        res[c][1] = nr;
      }
    } else if (lane == 0) {
      res[c][0] = 0u;
      res[c][1] = 0u;
    }
  }
  __syncthreads();
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    pre[c] |= res[c][0] << sh;
    rank[c] = res[c][1];
  }
}

template <int kThreads, int PER>
__global__ __launch_bounds__(kThreads) void k_select(PrunePlan p) {
  constexpr int kWaves = kThreads / 64;
  __shared__ __attribute__((aligned(16))) uint32_t hist[kWaves][2][256];  // per-wave digit counts per cut
  __shared__ uint32_t res[2][2];                                          // per cut: digit, rank within it
  __shared__ uint32_t wt[4][kWaves];

  const int u = blockIdx.x;  // ((l * B) + b) * Hkv + g, l < h
  const int g = u % p.Hkv;
  const int b = (u / p.Hkv) % p.B;
  const int l = u / (p.Hkv * p.B);
  // Every parameter of the unit, output pointers included, in one batch of
  // loads.  There is no early exit: a unit with n_surv = 0 (k = 0) finds no
  // kept or dropped token below and writes nothing, and without the branch
  // the loads are not deferred behind the first one.
  const int nsv = ldg(p.ns + b * p.L + l);
  const int n = ldg(p.nb + b);
  const int k = ldg(p.kk + b * p.L + l);
  const int64_t toff = ldg(p.toff + b);
  const uint64_t idx_base = ldg(p.lp + LP_IDX * p.L + l), drop_base = ldg(p.lp + LP_DROP * p.L + l);
  const int64_t orow = ldg(p.orow + l * (p.B + 1) + b), drow = ldg(p.drow + l * (p.B + 1) + b);
  const int r = nsv - k;

  const float *S = p.mode ? p.gs + toff
                          : p.S + (int64_t)l * p.Ntot * p.Hkv + toff * p.Hkv + (int64_t)g * n;
  const int tid = threadIdx.x;
  const int per = (n + kThreads - 1) / kThreads;  // <= PER
  const int v0 = tid * per;
  const int cnt = max(0, min(per, n - v0));

  // Bit patterns of non-negative floats order like the values.  A set sign
  // bit (only possible from non-finite inputs) is mapped to the top of the
  // 31-bit range so every count below stays consistent.  Slots past the
  // thread's run hold 0 and are never counted.
  uint32_t key[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const uint32_t x = (i < cnt) ? __float_as_uint(ldg(S + v0 + i)) : 0u;
    key[i] = (x & 0x80000000u) ? 0x7FFFFFFFu : x;
  }

  // Thresholds: the k-th and n_surv-th largest bit patterns (none wanted:
  // above every key).
  uint32_t pre[2] = {0u, 0u}, rank[2] = {(uint32_t)k, (uint32_t)nsv};
  radix_pass<kWaves, PER>(key, cnt, 23, 8, pre, rank, hist, res);
  radix_pass<kWaves, PER>(key, cnt, 15, 8, pre, rank, hist, res);
  radix_pass<kWaves, PER>(key, cnt, 7, 8, pre, rank, hist, res);
  radix_pass<kWaves, PER>(key, cnt, 0, 7, pre, rank, hist, res);
  const uint32_t tk = k > 0 ? pre[0] : 0xFFFFFFFFu, ts = nsv > 0 ? pre[1] : 0xFFFFFFFFu;

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
  uint32_t ex[4], tot4[4];
  block_scan4<kWaves>(c4, ex, tot4, wt);
  const uint32_t need_k = k > 0 ? (uint32_t)k - tot4[0] : 0u;
  const uint32_t need_s = (uint32_t)nsv - tot4[2];
  uint32_t ek = ex[1], es = ex[3];

  uint32_t keepmask = 0u, dropmask = 0u;
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
      if (kp) { keepmask |= 1u << i; ++nkeep; }
      else if (sv) { dropmask |= 1u << i; ++ndrop; }
    }

  const uint32_t c2[4] = {nkeep, ndrop, 0, 0};
  block_scan4<kWaves>(c2, ex, tot4, wt);

  int32_t *idx = reinterpret_cast<int32_t *>(idx_base) + orow + (int64_t)g * k;
  int32_t *drop = reinterpret_cast<int32_t *>(drop_base) + drow + (int64_t)g * r;
  uint32_t pk = ex[0], pd = ex[1];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    if ((keepmask >> i) & 1u) {
      if (pk < (uint32_t)k) stg(idx + pk, (int32_t)(v0 + i));
      ++pk;
    }
    if ((dropmask >> i) & 1u) {
      if (pd < (uint32_t)r) stg(drop + pd, (int32_t)(v0 + i));
      ++pd;
    }
  }
}

}  // namespace

hipError_t launch_select(const PrunePlan &p, hipStream_t st) {
  const uint32_t grid = (uint32_t)p.h * p.B * p.Hkv;
  if (grid == 0) return hipSuccess;
  // 256 threads hold up to 8 scores each, then 512 and 1024 threads up to 16,
  // then 1024 threads up to 32.  Fewer scores per thread shorten each radix
  // pass; more waves lengthen the histogram scans, so 512 threads beat both
  // 256 and 1024 at 3136 keys (measured).
  if (p.nmax <= 256 * 8)
    hipLaunchKernelGGL((k_select<256, 16>), dim3(grid), dim3(256), 0, st, p);
  else if (p.nmax <= 512 * 16)
    hipLaunchKernelGGL((k_select<512, 16>), dim3(grid), dim3(512), 0, st, p);
  else if (p.nmax <= 1024 * 16)
    hipLaunchKernelGGL((k_select<1024, 16>), dim3(grid), dim3(1024), 0, st, p);
  else
    hipLaunchKernelGGL((k_select<1024, 32>), dim3(grid), dim3(1024), 0, st, p);
  return hipGetLastError();
}

}  // namespace vc
