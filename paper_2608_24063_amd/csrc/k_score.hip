// k_score.hip -- window scores of PruneKV (Eq. (token_score), window reading):
//   S[v] = sum over the G*W window rows r of softmax_v(bf16(q_r) . k_v / sqrt(d)).
// Two passes over the keys, both on the bf16 matrix cores:
//   stats : per row r, the max m_r and sum_v exp(z_rv - m_r) over a key split
//   colsum: combines the splits, then S[v] = sum_r exp(z_rv - m_r) / sum_r
// and, for the shared ranking, a fixed-order fp64 sum over layers and heads.
#include <type_traits>

#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

constexpr float kNegInf = -__builtin_inff();
// Running maxima are kept already multiplied by the exp2 scale, so every
// rescale factor is exp2 of a plain difference of two floats (no product that
// the compiler could contract into an inexact fma).  They start at a finite
// floor, so rescaling never computes (-inf) - (-inf): exp2(floor - real max)
// underflows to 0 and exp2(floor - floor) is 1.
constexpr float kFloor = -1e30f;

// Interleave hints for the scheduler: alternate one matrix instruction with
// `v` vector instructions, `n` times.
template <int n, int v>
__device__ __forceinline__ void interleave_mfma_valu() {
#pragma unroll
  for (int i = 0; i < n; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, v, 0);
  }
}

#define VC_LDS_AS __attribute__((address_space(3)))

// A 64-row tile of bf16 rows in LDS, filled by direct global-to-LDS loads
// (no staging registers): each 16-byte load instruction of a wave writes
// 1 KB of LDS, lane i bytes [16i, 16i + 16).  Row r keeps its 16-byte chunk c
// at slot c ^ sw(r), so the 16 rows one operand read touches fall on 16
// distinct bank groups.
template <int D>
struct RowTileLds {
  static constexpr int kSlots = D / 8;                 // 16-byte chunks per row
  static constexpr int kLoadsPerWave = 64 * D * 2 / 1024 / 4;
  static constexpr int kRowsPerLoad = 1024 / (D * 2);
  __device__ static __forceinline__ int sw(int r) { return (r * kSlots / 16) & (kSlots - 1); }
  // This wave's share of rows r0 .. r0 + 63; rows at or past rmax repeat
  // row rmax - 1 (callers give them no weight).
  __device__ static __forceinline__ void issue(const uint16_t *src, int r0, int rmax, uint16_t *buf, int w,
                                               int lane) {
#pragma unroll
    for (int j = 0; j < kLoadsPerWave; ++j) {
      const int ld = w * kLoadsPerWave + j;
      const int r = ld * kRowsPerLoad + lane / kSlots;
      const int c = (lane % kSlots) ^ sw(r);
      const uint16_t *s = src + (int64_t)min(r0 + r, rmax - 1) * D + c * 8;
      __builtin_amdgcn_global_load_lds((const VC_GLOBAL void *)s, (VC_LDS_AS void *)(buf + ld * 512), 16, 0, 0);
    }
  }
  // Operand of rows rb*16 + lr, k-elements 32*s + 8*lg .. + 8.
  __device__ static __forceinline__ bf16x8 operand(const uint16_t *buf, int rb, int s, int lr, int lg) {
    const int r = rb * 16 + lr;
    return as_bf16x8(*reinterpret_cast<const u32x4 *>(buf + r * D + ((4 * s + lg) ^ sw(r)) * 8));
  }
};

// Barrier after which the direct loads this wave issued have landed in LDS.
__device__ __forceinline__ void lds_fill_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0); expcnt and lgkmcnt left alone
  __syncthreads();
}

// The same, leaving this wave's newest N (< 16) vector memory operations in
// flight: the direct loads of later tiles, when nothing else was issued after
// them.  A plain s_barrier, not __syncthreads(): the latter's release fence
// counts those loads as pending LDS writes and waits for all of them.  The
// wait here covers what the fence would: the older direct loads (vmcnt) and
// every LDS access of this wave (lgkmcnt); the empty asm statements keep the
// compiler from moving memory accesses across the barrier.
template <int N>
__device__ __forceinline__ void lds_fill_barrier_but() {
  static_assert(N >= 0 && N < 16, "vmcnt field");
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0x0070 | N);  // vmcnt(N) lgkmcnt(0); expcnt left alone
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

__device__ __forceinline__ void unit_coords(const PrunePlan &p, int u, int &ls, int &b, int &g) {
  g = u % p.Hkv;
  b = (u / p.Hkv) % p.B;
  ls = u / (p.Hkv * p.B);
}

// ---------------------------------------------------------------------------
// Pass 1: row statistics.  Workgroup = (unit, 256-row query group, key split).
// Wave w owns query rows qg*256 + w*64 + [0, 64) as MFMA B operands and all
// four waves share each 64-key tile of K in LDS (A operands; direct loads into
// a ring of three chunk-swizzled tiles, two ahead of the one in use), so the
// product is Z^T (keys x queries): lane l sees query l%16 of each 16-row block
// and keys 4*(l/16)+i, and keeps a running (max, sum) per query in registers.
// ---------------------------------------------------------------------------
// Softmax statistics of one 16-row query block (lane's row: qb*16 + l%16)
// over the 64 keys of a tile.
template <bool MASK>
__device__ __forceinline__ void stats_rows(f32x4 (&acc)[4], float &m, float &sum, int tb, int k1,
                                           int lg, float sc) {
  if (MASK) {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (tb + kb * 16 + 4 * lg + i >= k1) acc[kb][i] = kNegInf;
  }
  // Exponentials against the running max as it stands; only when they grow
  // past 2^96 (a logit far above every earlier one, or the first tile) is
  // the max raised and the tile redone.
  float part = 0.f;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int i = 0; i < 4; ++i) part += fast_exp2(fmaf(acc[kb][i], sc, -m));
  if (part <= 0x1p96f) {
    sum += part;
  } else {
    float tm = acc[0][0];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) tm = fmaxf(tm, acc[kb][i]);
    const float mnew = fmaxf(m, tm * sc);  // scaled running max
    part = 0.f;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int i = 0; i < 4; ++i) part += fast_exp2(fmaf(acc[kb][i], sc, -mnew));
    sum = fmaf(sum, fast_exp2(m - mnew), part);
    m = mnew;
  }
}

// One 64-key tile against the wave's four 16-row query blocks.  The K tile's
// operands are read from LDS once; the matrix work of block qb+1 is issued
// ahead of the softmax work of block qb so the two units overlap.
template <int D, bool MASK>
__device__ __forceinline__ void stats_tile(const uint16_t *kl, const bf16x8 (&bq)[4][D / 32],
                                           float (&m)[4], float (&sum)[4], int tb, int k1, int lr,
                                           int lg, float sc) {
  constexpr int KS = D / 32;
  bf16x8 a[4][KS];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int s = 0; s < KS; ++s) a[kb][s] = RowTileLds<D>::operand(kl, kb, s, lr, lg);
  f32x4 cur[4], nxt[4];
#pragma unroll
  for (int s = 0; s < KS; ++s)
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) cur[kb] = mfma_bf16(a[kb][s], bq[0][s], s == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : cur[kb]);
#pragma unroll
  for (int qb = 0; qb < 4; ++qb) {
    if (qb + 1 < 4) {
#pragma unroll
      for (int s = 0; s < KS; ++s)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
          nxt[kb] = mfma_bf16(a[kb][s], bq[qb + 1][s], s == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : nxt[kb]);
    }
    stats_rows<MASK>(cur, m[qb], sum[qb], tb, k1, lg, sc);
    if (qb + 1 < 4) interleave_mfma_valu<4 * KS, 4>();
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) cur[kb] = nxt[kb];
  }
}

// A 64-bit table entry of the plan chunk (two words, low first).
template <uint32_t CW>
__device__ __forceinline__ uint64_t chunk_u64(const UploadChunk<CW> &c, int w) {
  return (uint64_t)c.data[w] | ((uint64_t)c.data[w + 1] << 32);
}

// The plan's first chunk arrives with this launch: the grid copies it into
// the workspace for the later kernels, and every workgroup reads its own
// tables (layer pointers, token offsets, lengths) from the argument itself.
template <int D, uint32_t CW>
__global__ __launch_bounds__(256, 2) void k_score_stats(PrunePlan p, uint32_t *plan_dst, UploadChunk<CW> c) {
  constexpr int KS = D / 32;
  // K tiles through a ring of three LDS buffers (direct loads, chunk
  // swizzled), two in flight ahead of the one in use.
  // Separate LDS variables, so the compiler knows a direct load into one
  // tile does not write the others and leaves the later tiles in flight.
  __shared__ __attribute__((aligned(16))) uint16_t kt0[kKeyTile * D];
  __shared__ __attribute__((aligned(16))) uint16_t kt1[kKeyTile * D];
  __shared__ __attribute__((aligned(16))) uint16_t kt2[kKeyTile * D];
  auto ktile = [&](auto i) -> uint16_t * {
    constexpr int I = decltype(i)::value;
    return I == 0 ? kt0 : I == 1 ? kt1 : kt2;
  };
  using KT = RowTileLds<D>;

  for (uint32_t i = blockIdx.x * 256 + threadIdx.x; i < c.words; i += gridDim.x * 256) plan_dst[i] = c.data[i];

  const uint32_t lb = xcd_block(blockIdx.x, gridDim.x);
  const int qg = lb % p.nqg;
  const int ks = (lb / p.nqg) % p.nks;
  const int u = lb / (p.nqg * p.nks);
  int ls, b, g;
  unit_coords(p, u, ls, b, g);
  const int n = (int)c.data[p.w_nb + b];
  const int64_t toff = (int64_t)chunk_u64(c, p.w_toff + 2 * b);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const float sc = p.sc;

  // Key splits are whole tiles, so only the last split of a unit can end in
  // a partial tile.
  const int span = ((n + p.nks - 1) / p.nks + kKeyTile - 1) & ~(kKeyTile - 1);
  const int k0 = min(n, ks * span), k1 = min(n, k0 + span);

  const uint16_t *K = reinterpret_cast<const uint16_t *>(chunk_u64(c, p.w_lp + 2 * (LP_K_IN * p.L + ls))) +
                      (toff * p.Hkv + (int64_t)g * n) * D;
  const int64_t qoff = ((int64_t)b * p.Hq + (int64_t)g * p.G) * p.W * D;
  const float *Q = reinterpret_cast<const float *>(chunk_u64(c, p.w_lp + 2 * (LP_Q * p.L + ls))) + qoff;
  uint16_t *Qb = p.qbf + (int64_t)ls * p.B * p.Hq * p.W * D + qoff;

  // Query rows -> bf16 B operands (round to nearest even), zero past R.  All
  // loads of a half (two 16-row blocks) are issued before any is used (rows
  // clamped rather than branched on), so the prologue costs two round trips
  // instead of one per load pair.
  const int row0 = qg * kStatsRows + w * 64;
  const bool active = row0 < p.R;  // wave-uniform: waves of padding rows only stage tiles
  bf16x8 bq[4][KS];
#pragma unroll
  for (int hq = 0; hq < 2; ++hq) {
    u32x4 raw[2][KS][2];
#pragma unroll
    for (int qq = 0; qq < 2; ++qq) {
      const int rc = min(row0 + (2 * hq + qq) * 16 + lr, p.R - 1);
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const float *src = Q + (int64_t)rc * D + 32 * s + 8 * lg;
        raw[qq][s][0] = ld16(src);
        raw[qq][s][1] = ld16(src + 4);
      }
    }
#pragma unroll
    for (int qq = 0; qq < 2; ++qq) {
      const int qb = 2 * hq + qq;
      const int row = row0 + qb * 16 + lr;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const u32x4 a = raw[qq][s][0], c = raw[qq][s][1];
        u32x4 pk = {pack_bf16(__uint_as_float(a.x), __uint_as_float(a.y)),
                    pack_bf16(__uint_as_float(a.z), __uint_as_float(a.w)),
                    pack_bf16(__uint_as_float(c.x), __uint_as_float(c.y)),
                    pack_bf16(__uint_as_float(c.z), __uint_as_float(c.w))};
        if (row >= p.R) pk = u32x4{0, 0, 0, 0};
        bq[qb][s] = as_bf16x8(pk);
      }
    }
  }
  // The first key split also leaves the bf16 queries for the column pass.
  if (ks == 0) {
#pragma unroll
    for (int qb = 0; qb < 4; ++qb) {
      const int row = row0 + qb * 16 + lr;
      if (row < p.R) {
#pragma unroll
        for (int s = 0; s < KS; ++s) st16(Qb + (int64_t)row * D + 32 * s + 8 * lg, as_u32x4(bq[qb][s]));
      }
    }
  }

  float m[4], sum[4];
#pragma unroll
  for (int qb = 0; qb < 4; ++qb) { m[qb] = kFloor; sum[qb] = 0.f; }

  const int ntiles = (k1 - k0 + kKeyTile - 1) / kKeyTile;
  // Tile t lives in buffer t % 3: it is requested at step t - 2 (into the
  // buffer tile t - 3 left, which every wave is past) and waited for at the
  // end of step t - 1, with tile t + 1's loads left in flight.  Tiles past
  // the end re-read the last key and are never used.
  if (ntiles > 0) {
    KT::issue(K, k0, k1, kt0, w, lane);
    KT::issue(K, min(k0 + kKeyTile, k1 - 1), k1, kt1, w, lane);
    lds_fill_barrier_but<KT::kLoadsPerWave>();
  }
  auto step = [&](auto par, int t) {
    constexpr int PAR = decltype(par)::value;
    const int tb = k0 + t * kKeyTile;
    KT::issue(K, min(tb + 2 * kKeyTile, k1 - 1), k1, ktile(std::integral_constant<int, (PAR + 2) % 3>{}), w, lane);
    if (active) {
      if (tb + kKeyTile <= k1)
        stats_tile<D, false>(ktile(par), bq, m, sum, tb, k1, lr, lg, sc);
      else
        stats_tile<D, true>(ktile(par), bq, m, sum, tb, k1, lr, lg, sc);
    }
    lds_fill_barrier_but<KT::kLoadsPerWave>();
  };
  int t = 0;
  for (; t + 2 < ntiles; t += 3) {
    step(std::integral_constant<int, 0>{}, t);
    step(std::integral_constant<int, 1>{}, t + 1);
    step(std::integral_constant<int, 2>{}, t + 2);
  }
  if (t < ntiles) step(std::integral_constant<int, 0>{}, t);
  if (t + 1 < ntiles) step(std::integral_constant<int, 1>{}, t + 1);
  if (ntiles > 0) lds_fill_barrier();  // every load in flight lands before the workgroup's LDS is released

  if (!active) return;

  // Combine the four lane groups that share a query row, then store.
#pragma unroll
  for (int qb = 0; qb < 4; ++qb) {
#pragma unroll
    for (int mask = 16; mask <= 32; mask <<= 1) {
      const float mo = shfl_xor(m[qb], mask), so = shfl_xor(sum[qb], mask);
      const float M = fmaxf(m[qb], mo);
      sum[qb] = sum[qb] * fast_exp2(m[qb] - M) + so * fast_exp2(mo - M);
      m[qb] = M;
    }
    const int row = row0 + qb * 16 + lr;
    if (lg == 0 && row < p.R) {
      const float mc = m[qb] <= kFloor ? kNegInf : m[qb];
      stg(p.part + ((int64_t)u * p.nks + ks) * p.R + row, make_float2(mc, sum[qb]));
    }
  }
}

// ---------------------------------------------------------------------------
// Pass 2: column sums.  Workgroup = (unit, 256-key chunk).  Wave w owns keys
// chunk*256 + w*64 + [0, 64) as B operands; the G*W query rows (bf16 copies
// written by pass 1) stream through LDS 64 rows at a time as A operands (direct
// global-to-LDS loads into a chunk-swizzled tile, one tile ahead), so the
// product is Z (queries x keys): lane l sees key l%16 of each 16-key block and
// rows 4*(l/16)+i, and accumulates exp2(z*sc - m_r) / sum_r per key.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256, 3) void k_score_colsum(PrunePlan p) {
  constexpr int KS = D / 32;
  constexpr int kMaxR = 1024;
  __shared__ __attribute__((aligned(16))) uint16_t qt0[64 * D];  // separate variables: see the statistics pass
  __shared__ __attribute__((aligned(16))) uint16_t qt1[64 * D];
  __shared__ __attribute__((aligned(16))) float2 rs[kMaxR];
  using QT = RowTileLds<D>;

  const uint32_t lb = xcd_block(blockIdx.x, gridDim.x);
  const int c = lb % p.ncol;
  const int u = lb / p.ncol;
  int ls, b, g;
  unit_coords(p, u, ls, b, g);
  const int n = ldg(p.nb + b);
  if (c * kColKeys >= n) return;  // whole workgroup exits together
  const int64_t toff = ldg(p.toff + b);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const float sc = p.sc;
  const int R = p.R;
  const int Rpad = (R + 63) & ~63;

  const uint16_t *K = reinterpret_cast<const uint16_t *>(ldg(p.lp + LP_K_IN * p.L + ls)) +
                      (toff * p.Hkv + (int64_t)g * n) * D;
  const uint16_t *Qb = p.qbf + (int64_t)ls * p.B * p.Hq * p.W * D +
                       ((int64_t)b * p.Hq + (int64_t)g * p.G) * p.W * D;

  // Keys of this wave as B operands.
  const int key0 = c * kColKeys + w * 64;
  const bool active = key0 < n;  // wave-uniform
  bf16x8 bk[4][KS];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    const int key = key0 + kb * 16 + lr;
#pragma unroll
    for (int s = 0; s < KS; ++s)
      bk[kb][s] = as_bf16x8(key < n ? ld16(K + (int64_t)key * D + 32 * s + 8 * lg) : u32x4{0, 0, 0, 0});
  }
  QT::issue(Qb, 0, R, qt0, w, lane);

  // Row statistics: merge the key splits of pass 1.  Rows past R get a
  // reference of +inf so they contribute exp2(-inf) = 0.
  // All partials of a row are loaded in one batch (nks <= kMaxSplits).
  for (int r = tid; r < Rpad; r += 256) {
    float2 st = make_float2(__builtin_inff(), 0.f);
    if (r < R) {
      const float2 *pr = p.part + (int64_t)u * p.nks * R + r;
      float2 q[kMaxSplits];
#pragma unroll
      for (int k = 0; k < kMaxSplits; ++k)
        q[k] = k < p.nks ? ldg(pr + (int64_t)k * R) : make_float2(kNegInf, 0.f);
      float M = kNegInf;
#pragma unroll
      for (int k = 0; k < kMaxSplits; ++k) M = fmaxf(M, q[k].x);
      float s = 0.f;
      if (M != kNegInf) {
#pragma unroll
        for (int k = 0; k < kMaxSplits; ++k)
          if (q[k].x != kNegInf) s += q[k].y * fast_exp2(q[k].x - M);
      }
      st = make_float2(M == kNegInf ? __builtin_inff() : M, s > 0.f ? 1.f / s : 0.f);
    }
    rs[r] = st;
  }
  lds_fill_barrier();

  float col[4] = {0.f, 0.f, 0.f, 0.f};
  const int ntiles = Rpad / 64;
  auto step = [&](auto par, int t) {
    constexpr int PAR = decltype(par)::value;
    if (t + 1 < ntiles) QT::issue(Qb, (t + 1) * 64, R, PAR ? qt0 : qt1, w, lane);
    if (active) {
      const uint16_t *ql = PAR ? qt1 : qt0;
      // Two halves of two query blocks x four key blocks: eight accumulation
      // chains at a time, every operand read from LDS feeding four products.
#pragma unroll
      for (int qh = 0; qh < 2; ++qh) {
        f32x4 acc[2][4];
#pragma unroll
        for (int s = 0; s < KS; ++s) {
          bf16x8 a[2];
#pragma unroll
          for (int q2 = 0; q2 < 2; ++q2) a[q2] = QT::operand(ql, 2 * qh + q2, s, lr, lg);
#pragma unroll
          for (int q2 = 0; q2 < 2; ++q2)
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
              acc[q2][kb] = mfma_bf16(a[q2], bk[kb][s], s == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : acc[q2][kb]);
        }
#pragma unroll
        for (int q2 = 0; q2 < 2; ++q2) {
          const int qb = 2 * qh + q2;
          const int rbase = t * 64 + qb * 16 + 4 * lg;
          const f32x4 s01 = *reinterpret_cast<const f32x4 *>(&rs[rbase]);
          const f32x4 s23 = *reinterpret_cast<const f32x4 *>(&rs[rbase + 2]);
          const float mr[4] = {s01.x, s01.z, s23.x, s23.z}, ir[4] = {s01.y, s01.w, s23.y, s23.w};
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              col[kb] = fmaf(fast_exp2(fmaf(acc[q2][kb][i], sc, -mr[i])), ir[i], col[kb]);
        }
      }
    }
    lds_fill_barrier();
  };
  int t = 0;
  for (; t + 1 < ntiles; t += 2) {
    step(std::integral_constant<int, 0>{}, t);
    step(std::integral_constant<int, 1>{}, t + 1);
  }
  if (t < ntiles) step(std::integral_constant<int, 0>{}, t);
  if (!active) return;

  float *S = p.S + (int64_t)ls * p.Ntot * p.Hkv + toff * p.Hkv + (int64_t)g * n;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    float v = col[kb];
    v += shfl_xor(v, 16);
    v += shfl_xor(v, 32);
    const int key = key0 + kb * 16 + lr;
    if (lg == 0 && key < n) stg(S + key, v);
  }
}

// Shared ranking: s[v] = sum over all layers and kv heads of S, accumulated
// in fp64 in a fixed order: wave w sums the w-th quarter of the (layer,
// head) pairs in order, loading 16 at a time, and the quarters are added in
// order.  A workgroup covers 64 consecutive tokens, so every load of a wave
// reads one contiguous run.
__global__ __launch_bounds__(256) void k_score_global(PrunePlan p) {
  __shared__ double part[4][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int64_t t = (int64_t)blockIdx.x * 64 + lane;
  const bool in = t < p.Ntot;
  const int64_t tc = in ? t : p.Ntot - 1;
  // Sequence of token tc: the number of later sequence starts at or before it
  // (independent loads; empty sequences are passed over).
  int b = 0;
  for (int bb = 1; bb < p.B; ++bb) b += ldg(p.toff + bb) <= tc ? 1 : 0;
  const int64_t toff = ldg(p.toff + b);
  const int64_t v = tc - toff;
  const int n = ldg(p.nb + b);
  const float *S = p.S + toff * p.Hkv + v;
  const int npair = p.Ls * p.Hkv;
  const int q0 = npair * w / 4, q1 = npair * (w + 1) / 4;
  double acc = 0.0;
  for (int q = q0; q < q1; q += 16) {
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int qq = min(q + i, q1 - 1);
      const int l = qq / p.Hkv, g = qq - l * p.Hkv;
      x[i] = ldg(S + (int64_t)l * p.Ntot * p.Hkv + (int64_t)g * n);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i)
      if (q + i < q1) acc += (double)x[i];
  }
  part[w][lane] = acc;
  __syncthreads();
  if (w == 0 && in) stg(p.gs + t, (float)(((part[0][lane] + part[1][lane]) + part[2][lane]) + part[3][lane]));
}

}  // namespace

namespace {
template <uint32_t CW>
hipError_t stats_with_chunk(const PrunePlan &p, uint32_t grid, uint32_t *dst, const uint8_t *src, uint32_t words,
                            hipStream_t st) {
  UploadChunk<CW> c;
  c.words = words;
  c.pad = 0;
  __builtin_memcpy(c.data, src, (size_t)words * 4);
  if (p.d == 128)
    hipLaunchKernelGGL((k_score_stats<128, CW>), dim3(grid), dim3(256), 0, st, p, dst, c);
  else
    hipLaunchKernelGGL((k_score_stats<64, CW>), dim3(grid), dim3(256), 0, st, p, dst, c);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_score_stats(const PrunePlan &p, uint32_t *dst, const uint8_t *src, uint32_t words,
                              hipStream_t st) {
  const int units = p.Ls * p.B * p.Hkv;
  const uint32_t grid = (uint32_t)units * p.nqg * p.nks;
  if (grid == 0 || words > kChunkWords) return hipErrorInvalidValue;
  return words <= kChunkWordsSmall ? stats_with_chunk<kChunkWordsSmall>(p, grid, dst, src, words, st)
         : words <= kChunkWordsMid ? stats_with_chunk<kChunkWordsMid>(p, grid, dst, src, words, st)
                                   : stats_with_chunk<kChunkWords>(p, grid, dst, src, words, st);
}

hipError_t launch_score_colsum(const PrunePlan &p, hipStream_t st) {
  const int units = p.Ls * p.B * p.Hkv;
  const uint32_t grid = (uint32_t)units * p.ncol;
  if (grid == 0) return hipSuccess;
  if (p.d == 128)
    hipLaunchKernelGGL(k_score_colsum<128>, dim3(grid), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(k_score_colsum<64>, dim3(grid), dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_score_global(const PrunePlan &p, hipStream_t st) {
  const uint32_t grid = (uint32_t)((p.Ntot + 63) / 64);
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(k_score_global, dim3(grid), dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace vc
