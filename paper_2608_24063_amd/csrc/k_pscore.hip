// k_pscore.hip -- prefill scores of PruneKV: Eq. (token_score) with every token
// of the prefill as a query.  The sequence of unit (layer, sequence b, kv head
// g) is the n visual tokens followed by the W text tokens; the query of token
// i of each query head of the group attends tokens 0..i (causal
// self-attention) over the visual keys and then the text keys, and
//   S[v] = sum over heads h and tokens i >= v of softmax_j(bf16(q_hi) . k_j / sqrt(d))[v]
// for the visual keys v.  Two passes on the bf16 matrix cores, as for the
// window scores:
//   stats : workgroup = (unit, 256 query rows); the rows' queries stay in
//           registers and the keys up to the rows' last position stream
//           through LDS (Z^T = K Q^T: a lane holds one row and keeps its
//           running max and sum);
//   colsum: workgroup = (unit, 256 visual keys); the keys stay in registers
//           and the query rows that can reach them (position >= the chunk's
//           first key) stream through LDS with their row statistics
//           (Z = Q K^T: a lane holds one key and sums its column in order).
// Row r of a unit is (head r / N, token r % N), N = n + W.
#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

constexpr float kNegInf = -__builtin_inff();
constexpr float kFloor = -1e30f;  // finite start of the running maxima

template <int D>
constexpr int kPitch = D + 16;  // LDS row pitch (16-byte aligned, conflict-free operand reads)

__device__ __forceinline__ void unit_coords(const PrunePlan &p, int u, int &ls, int &b, int &g) {
  g = u % p.Hkv;
  b = (u / p.Hkv) % p.B;
  ls = u / (p.Hkv * p.B);
}

// Key j of the unit's sequence: visual key j < n, else text key j - n.
__device__ __forceinline__ const uint16_t *key_row(const uint16_t *Kv, const uint16_t *Kt, int n, int j, int D) {
  return j < n ? Kv + (int64_t)j * D : Kt + (int64_t)(j - n) * D;
}

// 64 keys x D bf16 staged through registers into LDS; keys past kend read
// key kend - 1 (callers mask them).  All 256 threads take part.
template <int D>
struct KeyTile {
  static constexpr int kChunks = 64 * D / 8 / 256;
  u32x4 v[kChunks];
  __device__ __forceinline__ void load(const uint16_t *Kv, const uint16_t *Kt, int n, int k0, int kend, int tid) {
#pragma unroll
    for (int i = 0; i < kChunks; ++i) {
      const int c = tid + i * 256;
      const int row = c / (D / 8), col = c % (D / 8);
      v[i] = ld16(key_row(Kv, Kt, n, min(k0 + row, kend - 1), D) + col * 8);
    }
  }
  __device__ __forceinline__ void store(uint16_t *lds, int tid) const {
#pragma unroll
    for (int i = 0; i < kChunks; ++i) {
      const int c = tid + i * 256;
      *reinterpret_cast<u32x4 *>(lds + (c / (D / 8)) * kPitch<D> + (c % (D / 8)) * 8) = v[i];
    }
  }
};

// ---------------------------------------------------------------------------
// Pass 1: row statistics.  Wave w holds rows r0 + 64w + [0, 64): lane l sees
// row r0 + 64w + 16qb + l%16 and keys 4*(l/16) + i of each 16-key block.
// ---------------------------------------------------------------------------
template <int D, uint32_t CW>
__global__ __launch_bounds__(256, 2) void k_pscore_stats(PrunePlan p, uint32_t *plan_dst, UploadChunk<CW> c) {
  constexpr int KS = D / 32, P = kPitch<D>;
  __shared__ __attribute__((aligned(16))) uint16_t kt[2][64 * P];

  for (uint32_t i = blockIdx.x * 256 + threadIdx.x; i < c.words; i += gridDim.x * 256) plan_dst[i] = c.data[i];

  const uint32_t lb = xcd_block(blockIdx.x, gridDim.x);
  const int qg = lb % p.nqg;
  const int u = lb / p.nqg;
  int ls, b, g;
  unit_coords(p, u, ls, b, g);
  auto u64 = [&](int w) { return (uint64_t)c.data[w] | ((uint64_t)c.data[w + 1] << 32); };
  const int n = (int)c.data[p.w_nb + b];
  const int64_t toff = (int64_t)u64(p.w_toff + 2 * b);
  const int N = n + p.W;
  const int Ru = p.G * N;  // rows of this unit
  const int r0 = qg * kStatsRows;
  if (r0 >= Ru) return;  // whole workgroup exits together
  const int r1 = min(Ru, r0 + kStatsRows);
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

  // Keys this workgroup needs: tokens 0 .. the largest position of its rows.
  const int kend = (r0 / N == (r1 - 1) / N) ? (r1 - 1) % N + 1 : N;
  const int ntiles = (kend + 63) / 64;

  const int row0 = r0 + w * 64;
  const bool active = row0 < r1;  // wave-uniform
  bf16x8 bq[4][KS];
  int pos[4];  // this lane's token position per query block (-1: no row)
#pragma unroll
  for (int qb = 0; qb < 4; ++qb) {
    const int row = row0 + qb * 16 + lr;
    const bool ok = row < r1;
    pos[qb] = ok ? row % N : -1;
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

  float m[4], sum[4];
#pragma unroll
  for (int qb = 0; qb < 4; ++qb) { m[qb] = kFloor; sum[qb] = 0.f; }

  KeyTile<D> tr;
  if (ntiles > 0) {
    tr.load(Kv, Kt, n, 0, kend, tid);
    tr.store(kt[0], tid);
  }
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int tb = t * 64;
    if (t + 1 < ntiles) tr.load(Kv, Kt, n, tb + 64, kend, tid);
    if (active) {
      const uint16_t *kl = kt[t & 1];
      bf16x8 a[4][KS];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int s = 0; s < KS; ++s)
          a[kb][s] = as_bf16x8(*reinterpret_cast<const u32x4 *>(kl + (kb * 16 + lr) * P + 32 * s + 8 * lg));
#pragma unroll
      for (int qb = 0; qb < 4; ++qb) {
        f32x4 acc[4];
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
            acc[kb] = mfma_bf16(a[kb][s], bq[qb][s], s == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : acc[kb]);
        // Causal mask (keys past the row's token, and past kend).
        float tm = kNegInf;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int j = tb + kb * 16 + 4 * lg + i;
            if (j > pos[qb] || j >= kend) acc[kb][i] = kNegInf;
            tm = fmaxf(tm, acc[kb][i]);
          }
        const float mnew = fmaxf(m[qb], tm * sc);
        float part = 0.f;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) part += fast_exp2(fmaf(acc[kb][i], sc, -mnew));
        sum[qb] = fmaf(sum[qb], fast_exp2(m[qb] - mnew), part);
        m[qb] = mnew;
      }
    }
    if (t + 1 < ntiles) tr.store(kt[(t + 1) & 1], tid);
    __syncthreads();
  }
  if (!active) return;

  // Combine the four lane groups of each row, then store (max*sc, sum).
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
    if (lg == 0 && row < r1) stg(p.part + (int64_t)u * p.Rmax + row, make_float2(m[qb], sum[qb]));
  }
}

// ---------------------------------------------------------------------------
// Pass 2: column sums.  Wave w holds visual keys v0 + 64w + [0, 64) as B
// operands; the rows that can attend them (every head's tokens v0 .. N-1)
// stream 64 at a time: queries to bf16 in LDS, (max, 1/sum) beside them.
// Lane l sees key 16kb + l%16 of its wave and rows 4*(l/16) + i of each
// 16-row block, and adds exp2(z*sc - m_r) / sum_r for rows at or after its key.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256, 2) void k_pscore_colsum(PrunePlan p) {
  constexpr int KS = D / 32, P = kPitch<D>;
  constexpr int kQChunks = 64 * D / 4 / 256;  // fp32 16-byte chunks per thread per tile
  __shared__ __attribute__((aligned(16))) uint16_t qt[2][64 * P];
  __shared__ __attribute__((aligned(16))) float2 rs[2][64];
  __shared__ int rpos[2][64];

  const uint32_t lb = xcd_block(blockIdx.x, gridDim.x);
  const int ch = lb % p.nkc;
  const int u = lb / p.nkc;
  int ls, b, g;
  unit_coords(p, u, ls, b, g);
  const int n = ldg(p.nb + b);
  const int v0 = ch * kPColKeys;
  if (v0 >= n) return;  // whole workgroup exits together
  const int64_t toff = ldg(p.toff + b);
  const int N = n + p.W;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const float sc = p.sc;

  const uint16_t *Kv = reinterpret_cast<const uint16_t *>(ldg(p.lp + LP_K_IN * p.L + ls)) +
                       (toff * p.Hkv + (int64_t)g * n) * D;
  const float *Q = reinterpret_cast<const float *>(ldg(p.lp + LP_Q * p.L + ls)) +
                   (((toff + (int64_t)b * p.W) * p.Hq) + (int64_t)g * p.G * N) * D;
  const float2 *part = p.part + (int64_t)u * p.Rmax;

  // Keys of this wave as B operands (zero past n).
  const int key0 = v0 + w * 64;
  bf16x8 bk[4][KS];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    const int key = key0 + kb * 16 + lr;
#pragma unroll
    for (int s = 0; s < KS; ++s)
      bk[kb][s] = as_bf16x8(key < n ? ld16(Kv + (int64_t)key * D + 32 * s + 8 * lg) : u32x4{0, 0, 0, 0});
  }

  // Row list: for every head, tokens v0 .. N-1 (earlier tokens attend none
  // of these keys).
  const int per = N - v0;
  const int nrows = p.G * per;
  const int ntiles = (nrows + 63) / 64;
  auto row_of = [&](int e) { return (e / per) * N + v0 + e % per; };

  // Stage a tile: queries (fp32 -> bf16 pairs in registers), then LDS.
  u32x4 qr[kQChunks];
  float2 st = make_float2(0.f, 0.f);
  int sp = -1;
  auto load = [&](int t) {
#pragma unroll
    for (int i = 0; i < kQChunks; ++i) {
      const int cidx = tid + i * 256;
      const int rr = cidx / (D / 4), col = cidx % (D / 4);
      const int e = min(t * 64 + rr, nrows - 1);
      qr[i] = ld16(Q + (int64_t)row_of(e) * D + col * 4);
    }
    if (tid < 64) {
      const int e = t * 64 + tid;
      if (e < nrows) {
        const int r = row_of(e);
        const float2 ms = ldg(part + r);
        st = make_float2(ms.x, ms.y > 0.f ? 1.f / ms.y : 0.f);
        sp = r % N;
      } else {
        st = make_float2(__builtin_inff(), 0.f);  // padding rows add exp2(-inf) * 0 = 0
        sp = -1;
      }
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < kQChunks; ++i) {
      const int cidx = tid + i * 256;
      const int rr = cidx / (D / 4), col = cidx % (D / 4);
      const u32x4 a = qr[i];
      *reinterpret_cast<u32x2 *>(qt[buf] + rr * P + col * 4) =
          u32x2{pack_bf16(__uint_as_float(a.x), __uint_as_float(a.y)), pack_bf16(__uint_as_float(a.z), __uint_as_float(a.w))};
    }
    if (tid < 64) {
      rs[buf][tid] = st;
      rpos[buf][tid] = sp;
    }
  };

  float col[4] = {0.f, 0.f, 0.f, 0.f};
  if (ntiles > 0) {
    load(0);
    store(0);
  }
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) load(t + 1);
    const uint16_t *ql = qt[buf];
    // The tile's 16 terms per key are summed apart and then added to the
    // column: a long run of rows adds to the large running sum once a tile.
    float ts[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int qb = 0; qb < 4; ++qb) {
      bf16x8 a[KS];
#pragma unroll
      for (int s = 0; s < KS; ++s)
        a[s] = as_bf16x8(*reinterpret_cast<const u32x4 *>(ql + (qb * 16 + lr) * P + 32 * s + 8 * lg));
      f32x4 acc[4];
#pragma unroll
      for (int s = 0; s < KS; ++s)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
          acc[kb] = mfma_bf16(a[s], bk[kb][s], s == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : acc[kb]);
      const int rb = qb * 16 + 4 * lg;
      float mr[4], ir[4];
      int pr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float2 x = rs[buf][rb + i];
        mr[i] = x.x;
        ir[i] = x.y;
        pr[i] = rpos[buf][rb + i];
      }
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        const int key = key0 + kb * 16 + lr;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = fast_exp2(fmaf(acc[kb][i], sc, -mr[i])) * ir[i];
          ts[kb] += pr[i] >= key ? e : 0.f;
        }
      }
    }
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) col[kb] += ts[kb];
    if (t + 1 < ntiles) store(buf ^ 1);  // read last in tile t - 1, before that tile's barrier
    __syncthreads();
  }

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

template <uint32_t CW>
hipError_t pstats_with_chunk(const PrunePlan &p, uint32_t grid, uint32_t *dst, const uint8_t *src, uint32_t words,
                             hipStream_t st) {
  UploadChunk<CW> c;
  c.words = words;
  c.pad = 0;
  __builtin_memcpy(c.data, src, (size_t)words * 4);
  if (p.d == 128)
    hipLaunchKernelGGL((k_pscore_stats<128, CW>), dim3(grid), dim3(256), 0, st, p, dst, c);
  else
    hipLaunchKernelGGL((k_pscore_stats<64, CW>), dim3(grid), dim3(256), 0, st, p, dst, c);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_pscore_stats(const PrunePlan &p, uint32_t *dst, const uint8_t *src, uint32_t words,
                               hipStream_t st) {
  const int units = p.Ls * p.B * p.Hkv;
  const uint32_t grid = (uint32_t)units * p.nqg;
  if (grid == 0 || words > kChunkWords) return hipErrorInvalidValue;
  return words <= kChunkWordsSmall ? pstats_with_chunk<kChunkWordsSmall>(p, grid, dst, src, words, st)
         : words <= kChunkWordsMid ? pstats_with_chunk<kChunkWordsMid>(p, grid, dst, src, words, st)
                                   : pstats_with_chunk<kChunkWords>(p, grid, dst, src, words, st);
}

hipError_t launch_pscore_colsum(const PrunePlan &p, hipStream_t st) {
  const int units = p.Ls * p.B * p.Hkv;
  const uint32_t grid = (uint32_t)units * p.nkc;
  if (grid == 0) return hipSuccess;
  if (p.d == 128)
    hipLaunchKernelGGL(k_pscore_colsum<128>, dim3(grid), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(k_pscore_colsum<64>, dim3(grid), dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace vc
