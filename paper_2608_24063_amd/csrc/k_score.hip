// k_score.hip -- window scores of PruneKV (Eq. (token_score), window reading):
//   S[v] = sum over the G*W window rows r of softmax_v(bf16(q_r) . k_v / sqrt(d)).
// Two passes over the keys, both on the bf16 matrix cores:
//   stats : per row r, the max m_r and sum_v exp(z_rv - m_r) over a key split
//   colsum: combines the splits, then S[v] = sum_r exp(z_rv - m_r) / sum_r
// and, for the shared ranking, a fixed-order fp64 sum over layers and heads.
#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

constexpr float kNegInf = -__builtin_inff();

// Stage a tile of 64 rows x D bf16 (rows [r0, r0+64) of `src`, rows >= rmax
// read as zero) into registers; the whole workgroup participates.
template <int D>
struct TileRegs {
  static constexpr int kChunks = 64 * D / 8 / 256;  // 16-byte chunks per thread
  u32x4 v[kChunks];
  __device__ __forceinline__ void load(const uint16_t *src, int64_t r0, int64_t rmax, int tid) {
#pragma unroll
    for (int i = 0; i < kChunks; ++i) {
      int c = tid + i * 256;
      int row = c / (D / 8), col = c % (D / 8);
      int64_t gr = r0 + row;
      if (gr < rmax)
        v[i] = *reinterpret_cast<const u32x4 *>(src + gr * D + col * 8);
      else
        v[i] = u32x4{0, 0, 0, 0};
    }
  }
  __device__ __forceinline__ void store(uint16_t *lds, int tid) const {
    constexpr int P = D + 8;
#pragma unroll
    for (int i = 0; i < kChunks; ++i) {
      int c = tid + i * 256;
      int row = c / (D / 8), col = c % (D / 8);
      *reinterpret_cast<u32x4 *>(lds + row * P + col * 8) = v[i];
    }
  }
};

__device__ __forceinline__ void unit_coords(const PrunePlan &p, int u, int &ls, int &b, int &g) {
  g = u % p.Hkv;
  b = (u / p.Hkv) % p.B;
  ls = u / (p.Hkv * p.B);
}

// Merge two (max, sum) pairs whose sums are relative to exp2(max * sc).
__device__ __forceinline__ void merge_stats(float &m, float &s, float mo, float so, float sc) {
  float M = fmaxf(m, mo);
  if (M == kNegInf) return;  // both empty
  float Mc = M * sc;
  float a = (m == kNegInf) ? 0.f : s * fast_exp2(m * sc - Mc);
  float c = (mo == kNegInf) ? 0.f : so * fast_exp2(mo * sc - Mc);
  m = M;
  s = a + c;
}

// ---------------------------------------------------------------------------
// Pass 1: row statistics.  Workgroup = (unit, 256-row query group, key split).
// Wave w owns query rows qg*256 + w*64 + [0, 64) as MFMA B operands and all
// four waves share each 64-key tile of K staged in LDS (A operands), so the
// product is Z^T (keys x queries): lane l sees query l%16 of each 16-row block
// and keys 4*(l/16)+i, and keeps running (max, sum) per query in registers.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256, 2) void k_score_stats(PrunePlan p) {
  constexpr int KS = D / 32;
  constexpr int P = D + 8;
  __shared__ __attribute__((aligned(16))) uint16_t kt[2][kKeyTile * P];

  const uint32_t lb = xcd_block(blockIdx.x, gridDim.x);
  const int qg = lb % p.nqg;
  const int ks = (lb / p.nqg) % p.nks;
  const int u = lb / (p.nqg * p.nks);
  int ls, b, g;
  unit_coords(p, u, ls, b, g);
  const int n = p.nb[b];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const float sc = p.sc;

  const int span = ((n + p.nks - 1) / p.nks + 15) & ~15;
  const int k0 = min(n, ks * span), k1 = min(n, k0 + span);

  const uint16_t *K = reinterpret_cast<const uint16_t *>(p.lp[LP_K_IN * p.L + ls]) +
                      ((int64_t)p.toff[b] * p.Hkv + (int64_t)g * n) * D;
  const int64_t qoff = ((int64_t)b * p.Hq + (int64_t)g * p.G) * p.W * D;
  const float *Q = reinterpret_cast<const float *>(p.lp[LP_Q * p.L + ls]) + qoff;
  uint16_t *Qb = p.qbf + (int64_t)ls * p.B * p.Hq * p.W * D + qoff;

  // Query rows -> bf16 B operands (round to nearest even), zero past R.
  const int row0 = qg * kStatsRows + w * 64;
  bf16x8 bq[4][KS];
#pragma unroll
  for (int qb = 0; qb < 4; ++qb) {
    const int row = row0 + qb * 16 + lr;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      u32x4 pk = {0, 0, 0, 0};
      if (row < p.R) {
        const float4 *src = reinterpret_cast<const float4 *>(Q + (int64_t)row * D + 32 * s + 8 * lg);
        float4 x0 = src[0], x1 = src[1];
        pk = u32x4{pack_bf16(x0.x, x0.y), pack_bf16(x0.z, x0.w), pack_bf16(x1.x, x1.y),
                   pack_bf16(x1.z, x1.w)};
        if (ks == 0) *reinterpret_cast<u32x4 *>(Qb + (int64_t)row * D + 32 * s + 8 * lg) = pk;
      }
      bq[qb][s] = as_bf16x8(pk);
    }
  }

  float m[4], sum[4];
#pragma unroll
  for (int qb = 0; qb < 4; ++qb) { m[qb] = kNegInf; sum[qb] = 0.f; }

  const int ntiles = (k1 - k0 + kKeyTile - 1) / kKeyTile;
  TileRegs<D> tr;
  if (ntiles > 0) {
    tr.load(K, k0, k1, tid);
    tr.store(kt[0], tid);
  }
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    const int tb = k0 + t * kKeyTile;
    if (t + 1 < ntiles) tr.load(K, tb + kKeyTile, k1, tid);
    const uint16_t *kl = kt[t & 1];
    f32x4 acc[4][4];
#pragma unroll
    for (int kb = 0; kb < 4; ++kb)
#pragma unroll
      for (int qb = 0; qb < 4; ++qb) acc[kb][qb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) {
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        bf16x8 a = as_bf16x8(*reinterpret_cast<const u32x4 *>(kl + (kb * 16 + lr) * P + 32 * s + 8 * lg));
#pragma unroll
        for (int qb = 0; qb < 4; ++qb) acc[kb][qb] = mfma_bf16(a, bq[qb][s], acc[kb][qb]);
      }
    }
    const bool full = tb + kKeyTile <= k1;
#pragma unroll
    for (int qb = 0; qb < 4; ++qb) {
      float tm = kNegInf;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float z = acc[kb][qb][i];
          if (!full && tb + kb * 16 + 4 * lg + i >= k1) z = kNegInf;
          acc[kb][qb][i] = z;
          tm = fmaxf(tm, z);
        }
      if (tm > m[qb]) {
        if (m[qb] != kNegInf) sum[qb] *= fast_exp2(m[qb] * sc - tm * sc);
        m[qb] = tm;
      }
      if (m[qb] != kNegInf) {
        const float mc = m[qb] * sc;
        float acc_s = 0.f;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) acc_s += fast_exp2(fmaf(acc[kb][qb][i], sc, -mc));
        sum[qb] += acc_s;
      }
    }
    if (t + 1 < ntiles) tr.store(kt[(t + 1) & 1], tid);
    __syncthreads();
  }

  // Combine the four lane groups that share a query row, then store.
#pragma unroll
  for (int qb = 0; qb < 4; ++qb) {
#pragma unroll
    for (int mask = 16; mask <= 32; mask <<= 1) {
      float mo = shfl_xor(m[qb], mask), so = shfl_xor(sum[qb], mask);
      merge_stats(m[qb], sum[qb], mo, so, sc);
    }
    const int row = row0 + qb * 16 + lr;
    if (lg == 0 && row < p.R) {
      float mc = m[qb] == kNegInf ? kNegInf : m[qb] * sc;
      p.part[((int64_t)u * p.nks + ks) * p.R + row] = make_float2(mc, sum[qb]);
    }
  }
}

// ---------------------------------------------------------------------------
// Pass 2: column sums.  Workgroup = (unit, 256-key chunk).  Wave w owns keys
// chunk*256 + w*64 + [0, 64) as B operands; the G*W query rows (bf16 copies
// written by pass 1) stream through LDS 64 rows at a time as A operands, so the
// product is Z (queries x keys): lane l sees key l%16 of each 16-key block and
// rows 4*(l/16)+i, and accumulates exp2(z*sc - m_r) / sum_r per key.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256, 2) void k_score_colsum(PrunePlan p) {
  constexpr int KS = D / 32;
  constexpr int P = D + 8;
  constexpr int kMaxR = 1024;
  __shared__ __attribute__((aligned(16))) uint16_t qt[2][64 * P];
  __shared__ __attribute__((aligned(16))) float2 rs[kMaxR + 64];

  const uint32_t lb = xcd_block(blockIdx.x, gridDim.x);
  const int c = lb % p.ncol;
  const int u = lb / p.ncol;
  int ls, b, g;
  unit_coords(p, u, ls, b, g);
  const int n = p.nb[b];
  if (c * kColKeys >= n) return;  // whole workgroup exits together
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const float sc = p.sc;
  const int R = p.R;

  // Row statistics: merge the key splits of pass 1.  Rows past R get a
  // reference of +inf so they contribute exp2(-inf) = 0.
  const int Rpad = (R + 63) & ~63;
  for (int r = tid; r < Rpad; r += 256) {
    float2 st = make_float2(__builtin_inff(), 0.f);
    if (r < R) {
      float M = kNegInf;
      for (int k = 0; k < p.nks; ++k) M = fmaxf(M, p.part[((int64_t)u * p.nks + k) * R + r].x);
      float s = 0.f;
      if (M != kNegInf)
        for (int k = 0; k < p.nks; ++k) {
          float2 q = p.part[((int64_t)u * p.nks + k) * R + r];
          if (q.x != kNegInf) s += q.y * fast_exp2(q.x - M);
        }
      st = make_float2(M == kNegInf ? __builtin_inff() : M, s > 0.f ? 1.f / s : 0.f);
    }
    rs[r] = st;
  }

  const uint16_t *K = reinterpret_cast<const uint16_t *>(p.lp[LP_K_IN * p.L + ls]) +
                      ((int64_t)p.toff[b] * p.Hkv + (int64_t)g * n) * D;
  const uint16_t *Qb = p.qbf + (int64_t)ls * p.B * p.Hq * p.W * D +
                       ((int64_t)b * p.Hq + (int64_t)g * p.G) * p.W * D;

  const int key0 = c * kColKeys + w * 64;
  bf16x8 bk[4][KS];
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    const int key = key0 + kb * 16 + lr;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      u32x4 v = {0, 0, 0, 0};
      if (key < n) v = *reinterpret_cast<const u32x4 *>(K + (int64_t)key * D + 32 * s + 8 * lg);
      bk[kb][s] = as_bf16x8(v);
    }
  }
  float col[4] = {0.f, 0.f, 0.f, 0.f};

  const int ntiles = Rpad / 64;
  TileRegs<D> tr;
  tr.load(Qb, 0, R, tid);
  tr.store(qt[0], tid);
  __syncthreads();
  for (int t = 0; t < ntiles; ++t) {
    if (t + 1 < ntiles) tr.load(Qb, (t + 1) * 64, R, tid);
    const uint16_t *ql = qt[t & 1];
#pragma unroll
    for (int qb = 0; qb < 4; ++qb) {
      f32x4 acc[4];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) acc[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        bf16x8 a = as_bf16x8(*reinterpret_cast<const u32x4 *>(ql + (qb * 16 + lr) * P + 32 * s + 8 * lg));
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) acc[kb] = mfma_bf16(a, bk[kb][s], acc[kb]);
      }
      const int rbase = t * 64 + qb * 16 + 4 * lg;
      float mr[4], ir[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float2 st = rs[rbase + i];
        mr[i] = st.x;
        ir[i] = st.y;
      }
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          col[kb] = fmaf(fast_exp2(fmaf(acc[kb][i], sc, -mr[i])), ir[i], col[kb]);
    }
    if (t + 1 < ntiles) tr.store(qt[(t + 1) & 1], tid);
    __syncthreads();
  }

  float *S = p.S + (int64_t)ls * p.Ntot * p.Hkv + (int64_t)p.toff[b] * p.Hkv + (int64_t)g * n;
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    float v = col[kb];
    v += shfl_xor(v, 16);
    v += shfl_xor(v, 32);
    const int key = key0 + kb * 16 + lr;
    if (lg == 0 && key < n) S[key] = v;
  }
}

// Shared ranking: s[v] = sum over all layers and kv heads of S, in fixed
// (layer, head) order, accumulated in fp64.
__global__ __launch_bounds__(256) void k_score_global(PrunePlan p) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= p.Ntot) return;
  int b = 0;
  while (b + 1 < p.B && p.toff[b + 1] <= t) ++b;
  const int64_t v = t - p.toff[b];
  const int n = p.nb[b];
  double acc = 0.0;
  for (int l = 0; l < p.Ls; ++l) {
    const float *S = p.S + (int64_t)l * p.Ntot * p.Hkv + (int64_t)p.toff[b] * p.Hkv;
    for (int g = 0; g < p.Hkv; ++g) acc += (double)S[(int64_t)g * n + v];
  }
  p.gs[t] = (float)acc;
}

}  // namespace

hipError_t launch_score_stats(const PrunePlan &p, hipStream_t st) {
  const int units = p.Ls * p.B * p.Hkv;
  const uint32_t grid = (uint32_t)units * p.nqg * p.nks;
  if (grid == 0) return hipSuccess;
  if (p.d == 128)
    hipLaunchKernelGGL(k_score_stats<128>, dim3(grid), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(k_score_stats<64>, dim3(grid), dim3(256), 0, st, p);
  return hipGetLastError();
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
  const uint32_t grid = (uint32_t)((p.Ntot + 255) / 256);
  if (grid == 0) return hipSuccess;
  hipLaunchKernelGGL(k_score_global, dim3(grid), dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace vc
