// k_pscore.hip -- prefill scores of PruneKV: Eq. (token_score) with every token
// of the prefill as a query.  The sequence of unit (layer, sequence b, kv head
// g) is the n visual tokens followed by the W text tokens; the query of token
// i of each query head of the group attends tokens 0..i (causal
// self-attention) over the visual keys and then the text keys, and
//   S[v] = sum over heads h and tokens i >= v of softmax_j(bf16(q_hi) . k_j / sqrt(d))[v]
// for the visual keys v.
//
// Row r of a unit is (head r / N, token r % N), N = n + W; rows come in
// groups of 256.  Each of the C workgroups of a unit owns the groups c, c + C,
// c + 2C, ... (round robin, so every workgroup gets a similar mix of short and
// long causal prefixes).  A group's 256 queries stay in registers as bf16
// while the keys up to its last position stream through LDS twice:
//   pass A: Z^T = K Q^T on the matrix cores; a lane holds one row and keeps its
//           running max and sum, which end as the row's log-sum-exp;
//   pass B: Z = Q K^T over the visual keys only; a lane holds one key of each
//           16-key block and adds exp2(z - lse) over its rows; the waves' sums
//           meet in LDS and go into the workgroup's own column partial.
// Queries are read once and the unit's keys (a few MB at most) come from L2;
// nothing of size rows x keys is stored.  A second kernel adds the C partials
// of each key in a fixed order, so the scores are deterministic.
#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

constexpr float kNegInf = -__builtin_inff();
constexpr float kInf = __builtin_inff();
constexpr float kFloor = -1e30f;  // finite start of the running maxima

__device__ __forceinline__ void unit_coords(const PrunePlan &p, int u, int &ls, int &b, int &g) {
  g = u % p.Hkv;
  b = (u / p.Hkv) % p.B;
  ls = u / (p.Hkv * p.B);
}

// Key j of the unit's sequence: visual key j < n, else text key j - n.
__device__ __forceinline__ const uint16_t *key_row(const uint16_t *Kv, const uint16_t *Kt, int n, int j, int D) {
  return j < n ? Kv + (int64_t)j * D : Kt + (int64_t)(j - n) * D;
}

#define VC_LDS __attribute__((address_space(3)))

// A 64-key tile in LDS, filled by direct global-to-LDS loads (no registers):
// each 16-byte load instruction of a wave writes 1 KB of LDS, lane i bytes
// [16i, 16i + 16).  Key row r keeps its 16-byte chunk c at slot c ^ sw(r), so
// the 16 rows that one operand read touches fall on 16 distinct bank groups.
template <int D>
struct KTile {
  static constexpr int kSlots = D / 8;                // 16-byte chunks per row
  static constexpr int kLoadsPerWave = 64 * D * 2 / 1024 / 4;
  static constexpr int kRowsPerLoad = 1024 / (D * 2);

  __device__ static __forceinline__ int sw(int r) { return (r * kSlots / 16) & (kSlots - 1); }

  // This wave's share of the tile of keys key0 .. key0+63; keys at or past
  // kend repeat key kend - 1 (valid memory; callers mask or discard them).
  __device__ static __forceinline__ void issue(const uint16_t *Kv, const uint16_t *Kt, int n, int key0, int kend,
                                               uint16_t *buf, int w, int lane) {
#pragma unroll
    for (int j = 0; j < kLoadsPerWave; ++j) {
      const int ld = w * kLoadsPerWave + j;
      const int r = ld * kRowsPerLoad + lane / kSlots;
      const int c = (lane % kSlots) ^ sw(r);
      const uint16_t *src = key_row(Kv, Kt, n, min(key0 + r, kend - 1), D) + c * 8;
      __builtin_amdgcn_global_load_lds((const VC_GLOBAL void *)src, (VC_LDS void *)(buf + ld * 512), 16, 0, 0);
    }
  }

  // Operand of keys kb*16 + lr, k-elements 32*s + 8*lg .. + 8.
  __device__ static __forceinline__ bf16x8 operand(const uint16_t *buf, int kb, int s, int lr, int lg) {
    const int r = kb * 16 + lr;
    return as_bf16x8(*reinterpret_cast<const u32x4 *>(buf + r * D + ((4 * s + lg) ^ sw(r)) * 8));
  }
};

// Barrier after which the tile loads this wave issued have landed in LDS
// (s_waitcnt vmcnt(0), then the workgroup barrier).
__device__ __forceinline__ void tile_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0); expcnt and lgkmcnt left alone
  __syncthreads();
}

// Scheduling hint: one matrix instruction, then `v` vector instructions,
// `n` times.
template <int n, int v>
__device__ __forceinline__ void interleave_mfma_valu() {
#pragma unroll
  for (int i = 0; i < n; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, v, 0);
  }
}

// Token position of the row `off` (< 64) rows after a row at position base.
__device__ __forceinline__ int run_pos(int base, int off, int N) {
  if (N >= 64) {
    const int p = base + off;  // off < 64 <= N: wraps at most once
    return p >= N ? p - N : p;
  }
  return (base + off) % N;
}

__device__ __forceinline__ int wave_min(int x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x = min(x, shfl_xor(x, m));
  return x;
}

template <int D, uint32_t CW>
__global__ __launch_bounds__(256, 2) void k_pscore(PrunePlan p, uint32_t *plan_dst, UploadChunk<CW> c) {
  constexpr int KS = D / 32;
  using KT = KTile<D>;
  // The two key tiles are separate LDS variables: the compiler then knows
  // that a direct load into one does not write the other, and does not drain
  // the next tile's loads before reading the current one.
  __shared__ __attribute__((aligned(16))) uint16_t kt0[64 * D];
  __shared__ __attribute__((aligned(16))) uint16_t kt1[64 * D];
  __shared__ __attribute__((aligned(16))) float lse[kStatsRows];  // per row: max*sc + log2(sum); +inf: none
  __shared__ float cs[2][4][64];     // per key tile: the four waves' column sums

  for (uint32_t i = blockIdx.x * 256 + threadIdx.x; i < c.words; i += gridDim.x * 256) plan_dst[i] = c.data[i];

  const uint32_t lb = xcd_block(blockIdx.x, gridDim.x);
  const int ch = lb % p.pwg;  // this workgroup's share: groups ch, ch + C, ...
  const int u = lb / p.pwg;
  int ls, b, g;
  unit_coords(p, u, ls, b, g);
  auto u64 = [&](int w) { return (uint64_t)c.data[w] | ((uint64_t)c.data[w + 1] << 32); };
  const int n = (int)c.data[p.w_nb + b];
  const int64_t toff = (int64_t)u64(p.w_toff + 2 * b);
  const int N = n + p.W;
  const int Ru = p.G * N;  // rows of this unit
  const int ngroups = (Ru + kStatsRows - 1) / kStatsRows;
  if (ch >= ngroups || n == 0) return;  // whole workgroup exits together; the reduction skips it
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const float sc = p.sc;

  const uint16_t *Kv = reinterpret_cast<const uint16_t *>(u64(p.w_lp + 2 * (LP_K_IN * p.L + ls))) +
                       (toff * p.Hkv + (int64_t)g * n) * D;
  const uint16_t *Kt = reinterpret_cast<const uint16_t *>(u64(p.w_lp + 2 * (LP_K_TEXT * p.L + ls))) +
                       ((int64_t)b * p.Hkv + g) * p.W * D;
  // Queries of the unit: rows (head g*G + hh, token i), packed over sequences.
  const float *Q = reinterpret_cast<const float *>(u64(p.w_lp + 2 * (LP_Q * p.L + ls))) +
                   (((toff + (int64_t)b * p.W) * p.Hq) + (int64_t)g * p.G * N) * D;
  // This workgroup's column partial over the unit's visual keys.  Thread
  // tid < 64 owns keys tid + 64j: it clears them here and is the only thread
  // that adds to them, so its own program order orders every update.
  float *cp = p.pcol + ((int64_t)u * p.pwg + ch) * p.nmax;
  if (tid < 64)
    for (int j = tid; j < n; j += 64) stg(cp + j, 0.f);

  for (int q = ch; q < ngroups; q += p.pwg) {
    const int r0 = q * kStatsRows;
    const int r1 = min(Ru, r0 + kStatsRows);
    // Keys the group needs: tokens 0 .. the largest position of its rows.
    const int kend = (r0 / N == (r1 - 1) / N) ? (r1 - 1) % N + 1 : N;
    const int row0 = r0 + w * 64;
    const bool active = row0 < r1;  // wave-uniform
    const int base = row0 % N;

    // The wave's 64 queries as bf16 operands (zero for rows past the group).
    bf16x8 bq[4][KS];
    int pos[4];  // pass A: position of this lane's row per 16-row block (-1: none)
#pragma unroll
    for (int qb = 0; qb < 4; ++qb) {
      const int row = row0 + qb * 16 + lr;
      const bool ok = row < r1;
      pos[qb] = ok ? run_pos(base, qb * 16 + lr, N) : -1;
      const int rc = min(row, Ru - 1);
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const float *src = Q + (int64_t)rc * D + 32 * s + 8 * lg;
        const u32x4 a = ld16(src), e = ld16(src + 4);
        u32x4 pk = {pack_bf16(__uint_as_float(a.x), __uint_as_float(a.y)),
                    pack_bf16(__uint_as_float(a.z), __uint_as_float(a.w)),
                    pack_bf16(__uint_as_float(e.x), __uint_as_float(e.y)),
                    pack_bf16(__uint_as_float(e.z), __uint_as_float(e.w))};
        if (!ok) pk = u32x4{0, 0, 0, 0};
        bq[qb][s] = as_bf16x8(pk);
      }
    }
    // Smallest position among the wave's rows (-1 if a row is missing): key
    // tiles wholly at or before it need no causal mask in either pass.
    const int wmin = __builtin_amdgcn_readfirstlane(wave_min(min(min(pos[0], pos[1]), min(pos[2], pos[3]))));

    // ---------------- pass A: row statistics over keys 0 .. kend-1
    const int ntA = (kend + 63) / 64;
    float m[4], sum[4];
#pragma unroll
    for (int qb = 0; qb < 4; ++qb) { m[qb] = kFloor; sum[qb] = 0.f; }
    KT::issue(Kv, Kt, n, 0, kend, kt0, w, lane);
    tile_barrier();
    auto stepA = [&](auto par, int t) {
      constexpr int PAR = decltype(par)::value;
      const int tb = t * 64;
      // The other buffer was last read in tile t - 1, before the last barrier.
      if (t + 1 < ntA) KT::issue(Kv, Kt, n, tb + 64, kend, PAR ? kt0 : kt1, w, lane);
      if (active) {
        const uint16_t *kl = PAR ? kt1 : kt0;
        // Two halves of 32 keys (operands of one half in registers at a time);
        // each half updates the rows' running max and sum.  Tiles wholly at or
        // before every row of the wave take the copy without the causal mask,
        // so no branch separates a block's products from the softmax they
        // overlap with.
        auto tileA = [&](auto intr) {
          constexpr bool INTERIOR = decltype(intr)::value;
#pragma unroll
          for (int kh = 0; kh < 2; ++kh) {
            bf16x8 a[2][KS];
#pragma unroll
            for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
              for (int s = 0; s < KS; ++s) a[k2][s] = KT::operand(kl, 2 * kh + k2, s, lr, lg);
            // The products of block qb + 1 are issued ahead of the softmax of
            // block qb, so the matrix and vector work overlap.
            auto prod = [&](int qb, f32x4 (&acc)[2]) {
#pragma unroll
              for (int s = 0; s < KS; ++s)
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2)
                  acc[k2] = mfma_bf16(a[k2][s], bq[qb][s], s == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : acc[k2]);
            };
            f32x4 cur[2], nxt[2];
            prod(0, cur);
#pragma unroll
            for (int qb = 0; qb < 4; ++qb) {
              if (INTERIOR && qb + 1 < 4) prod(qb + 1, nxt);
              f32x4 (&acc)[2] = cur;
              if constexpr (!INTERIOR) {
                // Keys past the row's token (this covers keys past kend too).
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
                  for (int i = 0; i < 4; ++i)
                    if (tb + (2 * kh + k2) * 16 + 4 * lg + i > pos[qb]) acc[k2][i] = kNegInf;
              }
              // Exponentials against the running max as it stands; only when
              // they grow past 2^96 (the row's first keys, or a logit far above
              // the earlier ones) is the max raised and the half redone.
              float part = 0.f;
#pragma unroll
              for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
                for (int i = 0; i < 4; ++i) part += fast_exp2(fmaf(acc[k2][i], sc, -m[qb]));
              if (part <= 0x1p96f) {
                sum[qb] += part;
              } else {
                float tm = kNegInf;
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
                  for (int i = 0; i < 4; ++i) tm = fmaxf(tm, acc[k2][i]);
                const float mnew = fmaxf(m[qb], tm * sc);
                part = 0.f;
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
                  for (int i = 0; i < 4; ++i) part += fast_exp2(fmaf(acc[k2][i], sc, -mnew));
                sum[qb] = fmaf(sum[qb], fast_exp2(m[qb] - mnew), part);
                m[qb] = mnew;
              }
              if (qb + 1 < 4) {
                if constexpr (INTERIOR) {
                  interleave_mfma_valu<2 * KS, 3>();
#pragma unroll
                  for (int k2 = 0; k2 < 2; ++k2) cur[k2] = nxt[k2];
                } else {
                  prod(qb + 1, cur);
                }
              }
            }
          }
        };
        if (tb + 63 <= wmin)  // wave-uniform
          tileA(std::true_type{});
        else
          tileA(std::false_type{});
      }
      tile_barrier();
    };
    {
      int t = 0;
      for (; t + 1 < ntA; t += 2) {
        stepA(std::integral_constant<int, 0>{}, t);
        stepA(std::integral_constant<int, 1>{}, t + 1);
      }
      if (t < ntA) stepA(std::integral_constant<int, 0>{}, t);
    }
    // Combine the four lane groups of each row; publish max*sc + log2(sum).
    if (active) {
#pragma unroll
      for (int qb = 0; qb < 4; ++qb) {
#pragma unroll
        for (int mask = 16; mask <= 32; mask <<= 1) {
          const float mo = shfl_xor(m[qb], mask), so = shfl_xor(sum[qb], mask);
          const float M = fmaxf(m[qb], mo);
          sum[qb] = sum[qb] * fast_exp2(m[qb] - M) + so * fast_exp2(mo - M);
          m[qb] = M;
        }
        if (lg == 0) lse[w * 64 + qb * 16 + lr] = sum[qb] > 0.f ? m[qb] + __builtin_amdgcn_logf(sum[qb]) : kInf;
      }
    }

    // ---------------- pass B: column sums over the visual keys 0 .. min(kend, n)-1
    const int kendB = min(kend, n);
    const int ntB = (kendB + 63) / 64;
    KT::issue(Kv, Kt, n, 0, kendB, kt0, w, lane);
    tile_barrier();  // also publishes lse
    float pend = 0.f;  // tid < 64: the column partial of the tile in flight, read ahead
    auto stepB = [&](auto par, int t) {
      constexpr int PAR = decltype(par)::value;
      const int tb = t * 64;
      if (t + 1 < ntB) KT::issue(Kv, Kt, n, tb + 64, kendB, PAR ? kt0 : kt1, w, lane);
      if (tid < 64) {
        // The previous tile's column sums are complete since the last barrier.
        if (t > 0 && tb - 64 + tid < n) {
          constexpr int pb = PAR ^ 1;
          stg(cp + tb - 64 + tid, pend + ((cs[pb][0][tid] + cs[pb][1][tid]) + (cs[pb][2][tid] + cs[pb][3][tid])));
        }
        pend = tb + tid < n ? ldg(cp + tb + tid) : 0.f;
      }
      float col[4] = {0.f, 0.f, 0.f, 0.f};
      if (active) {
        const uint16_t *kl = PAR ? kt1 : kt0;
        const bool interior = tb + 63 <= wmin;  // wave-uniform
#pragma unroll
        for (int kh = 0; kh < 2; ++kh) {
          bf16x8 a[2][KS];
#pragma unroll
          for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
            for (int s = 0; s < KS; ++s) a[k2][s] = KT::operand(kl, 2 * kh + k2, s, lr, lg);
#pragma unroll
          for (int qb = 0; qb < 4; ++qb) {
            f32x4 acc[2];
#pragma unroll
            for (int s = 0; s < KS; ++s)
#pragma unroll
              for (int k2 = 0; k2 < 2; ++k2)
                acc[k2] = mfma_bf16(bq[qb][s], a[k2][s], s == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : acc[k2]);
            // This lane's rows in the Z layout: 4*lg + i of the 16-row block.
            const float4 l4 = *reinterpret_cast<const float4 *>(&lse[w * 64 + qb * 16 + 4 * lg]);
            const float rl[4] = {l4.x, l4.y, l4.z, l4.w};
            if (interior) {
#pragma unroll
              for (int k2 = 0; k2 < 2; ++k2)
#pragma unroll
                for (int i = 0; i < 4; ++i) col[2 * kh + k2] += fast_exp2(fmaf(acc[k2][i], sc, -rl[i]));
            } else {
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const int off = qb * 16 + 4 * lg + i;
                const int pr = row0 + off < r1 ? run_pos(base, off, N) : -1;
#pragma unroll
                for (int k2 = 0; k2 < 2; ++k2) {
                  const float e = fast_exp2(fmaf(acc[k2][i], sc, -rl[i]));
                  col[2 * kh + k2] += tb + (2 * kh + k2) * 16 + lr <= pr ? e : 0.f;
                }
              }
            }
          }
        }
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          col[kb] += shfl_xor(col[kb], 16);
          col[kb] += shfl_xor(col[kb], 32);
        }
      }
      if (lg == 0) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) cs[PAR][w][kb * 16 + lr] = col[kb];
      }
      tile_barrier();
    };
    {
      int t = 0;
      for (; t + 1 < ntB; t += 2) {
        stepB(std::integral_constant<int, 0>{}, t);
        stepB(std::integral_constant<int, 1>{}, t + 1);
      }
      if (t < ntB) stepB(std::integral_constant<int, 0>{}, t);
    }
    if (tid < 64 && (ntB - 1) * 64 + tid < n) {
      const int pb = (ntB - 1) & 1;
      stg(cp + (ntB - 1) * 64 + tid, pend + ((cs[pb][0][tid] + cs[pb][1][tid]) + (cs[pb][2][tid] + cs[pb][3][tid])));
    }
    // The next group writes kt0, lse and cs only after barriers that every
    // read above precedes.
  }
}

// S[v] of each unit: its workgroups' column partials added in workgroup order.
__global__ __launch_bounds__(256) void k_pscore_reduce(PrunePlan p) {
  const int per = (p.nmax + 255) / 256;
  const int u = blockIdx.x / per;
  const int v = (blockIdx.x % per) * 256 + threadIdx.x;
  int ls, b, g;
  unit_coords(p, u, ls, b, g);
  const int n = ldg(p.nb + b);
  if (v >= n) return;
  const int ngroups = (p.G * (n + p.W) + kStatsRows - 1) / kStatsRows;
  const int C = min(p.pwg, ngroups);
  const float *cp = p.pcol + (int64_t)u * p.pwg * p.nmax + v;
  float s = 0.f;
  for (int c = 0; c < C; ++c) s += ldg(cp + (int64_t)c * p.nmax);
  const int64_t toff = ldg(p.toff + b);
  stg(p.S + (int64_t)ls * p.Ntot * p.Hkv + toff * p.Hkv + (int64_t)g * n + v, s);
}

template <uint32_t CW>
hipError_t pscore_with_chunk(const PrunePlan &p, uint32_t grid, uint32_t *dst, const uint8_t *src, uint32_t words,
                             hipStream_t st) {
  UploadChunk<CW> c;
  c.words = words;
  c.pad = 0;
  __builtin_memcpy(c.data, src, (size_t)words * 4);
  if (p.d == 128)
    hipLaunchKernelGGL((k_pscore<128, CW>), dim3(grid), dim3(256), 0, st, p, dst, c);
  else
    hipLaunchKernelGGL((k_pscore<64, CW>), dim3(grid), dim3(256), 0, st, p, dst, c);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_pscore(const PrunePlan &p, uint32_t *dst, const uint8_t *src, uint32_t words, hipStream_t st) {
  const int units = p.Ls * p.B * p.Hkv;
  const uint32_t grid = (uint32_t)units * p.pwg;
  if (grid == 0 || words > kChunkWords) return hipErrorInvalidValue;
  return words <= kChunkWordsSmall ? pscore_with_chunk<kChunkWordsSmall>(p, grid, dst, src, words, st)
         : words <= kChunkWordsMid ? pscore_with_chunk<kChunkWordsMid>(p, grid, dst, src, words, st)
                                   : pscore_with_chunk<kChunkWords>(p, grid, dst, src, words, st);
}

hipError_t launch_pscore_reduce(const PrunePlan &p, hipStream_t st) {
  const int units = p.Ls * p.B * p.Hkv;
  const uint32_t grid = (uint32_t)units * ((p.nmax + 255) / 256);
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(k_pscore_reduce, dim3(grid), dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace vc
