// k_decode.hip -- decode over the (compressed) cache (Sec. 2, "VLLM
// Decoding"): append one K/V row per (layer, sequence, kv head) and attend one
// query per query head over all cached rows.
//
// Attention is split over rows: workgroup = (unit, split of split_rows rows),
// and each of its four waves takes 32-row tiles in turn.  The G query heads of
// a kv head form one 16-column MFMA block (heads >= G are zero), so each K/V
// row is read once for all of them:
//   S^T = K Q^T   A = K rows straight from HBM, B = Q (registers)
//   O^T = V^T P^T A = V^T (per-wave transposed LDS tile), B = P^T (registers)
// Partial (max, sum, O) per split go to the workspace; a second kernel merges
// them in split order.
#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

constexpr float kNegInf = -__builtin_inff();
constexpr float kFloor = -1e30f;
constexpr int kRowTile = 32;

__global__ __launch_bounds__(64) void k_append(int32_t units, int32_t d, uint16_t *k_pool,
                                               uint16_t *v_pool, const int64_t *row_off,
                                               const int32_t *cap, int32_t *len,
                                               const uint16_t *k_new, const uint16_t *v_new) {
  const int u = blockIdx.x;
  const int t = threadIdx.x;
  const int L0 = ldg(len + u);
  const bool room = L0 < ldg(cap + u);
  const int chunks = d / 8;
  if (room) {
    const int64_t dst = (ldg(row_off + u) + L0) * d;
    for (int c = t; c < 2 * chunks; c += 64) {
      const bool isv = c >= chunks;
      const int cc = isv ? c - chunks : c;
      const uint16_t *src = (isv ? v_new : k_new) + (int64_t)u * d + cc * 8;
      uint16_t *dp = (isv ? v_pool : k_pool) + dst + cc * 8;
      st16(dp, ld16(src));
    }
  }
  __syncthreads();  // every thread has read len before it moves
  if (t == 0 && room) stg(len + u, L0 + 1);
}

__device__ __forceinline__ bf16x8 load_split8(const uint16_t *row, int c) {
  u32x2 a = *reinterpret_cast<const u32x2 *>(row + c);
  u32x2 b = *reinterpret_cast<const u32x2 *>(row + c + 16);
  return as_bf16x8(u32x4{a.x, a.y, b.x, b.y});
}

template <int D>
__global__ __launch_bounds__(256, 2) void k_decode_attn(DecodePlan p) {
  constexpr int KS = D / 32;
  constexpr int MB = D / 16;
  constexpr int PT = kRowTile + 8;
  __shared__ __attribute__((aligned(16))) uint16_t vt[4][D * PT];
  __shared__ float2 wml[4][16];
  __shared__ __attribute__((aligned(16))) float wo[4][16][D + 4];

  const uint32_t lb = xcd_block(blockIdx.x, gridDim.x);
  const int split = lb % p.nsplit;
  const int u = lb / p.nsplit;
  const int len = min(ldg(p.len + u), ldg(p.cap + u));
  const int r0 = split * p.split_rows;
  if (r0 >= len && split > 0) return;  // uniform: nothing for this split
  const int r1 = min(len, r0 + p.split_rows);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int g = u % p.Hkv;
  const int lb_ = u / p.Hkv;  // l * B + b
  const int64_t roff = ldg(p.row_off + u);
  const uint16_t *Kp = p.k_pool + roff * D;
  const uint16_t *Vp = p.v_pool + roff * D;

  // Query heads g*G + lr as B operands (natural k order: 8 consecutive d).
  bf16x8 bq[KS];
  const uint16_t *q = p.q + ((int64_t)lb_ * p.Hq + (int64_t)g * p.G + lr) * D;
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    u32x4 v = {0, 0, 0, 0};
    if (lr < p.G) v = ld16(q + 32 * s + 8 * lg);
    bq[s] = as_bf16x8(v);
  }

  f32x4 O[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) O[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Running max per head, pre-multiplied by the exp2 scale; starts at a finite
  // floor so rescaling never forms (-inf) - (-inf).
  float mrow = kFloor, lsum = 0.f;
  const float sc = p.sc;
  uint16_t *myvt = vt[w];

  const int ntiles = (r1 - r0 + kRowTile - 1) / kRowTile;
  for (int t = w; t < ntiles; t += 4) {
    const int t0 = r0 + t * kRowTile;
    // K rows -> A operands; S^T for 2 blocks of 16 rows.
    f32x4 acc[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
      const int row = t0 + rb * 16 + lr;
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        u32x4 a = {0, 0, 0, 0};
        if (row < r1) a = ld16(Kp + (int64_t)row * D + 32 * s + 8 * lg);
        acc[rb] = mfma_bf16(as_bf16x8(a), bq[s], acc[rb]);
      }
    }
    // V rows -> transposed per-wave LDS tile [d][32 rows].
    {
      const int pp = lane & 15;  // rows 2pp, 2pp+1
#pragma unroll
      for (int it = 0; it < D / 32; ++it) {
        const int c = (lane >> 4) + 4 * it;  // 16-byte chunk of the row
        const int ra = t0 + 2 * pp, rb2 = ra + 1;
        u32x4 va = {0, 0, 0, 0}, vb = {0, 0, 0, 0};
        if (ra < r1) va = ld16(Vp + (int64_t)ra * D + c * 8);
        if (rb2 < r1) vb = ld16(Vp + (int64_t)rb2 * D + c * 8);
        const uint32_t ea[4] = {va.x, va.y, va.z, va.w}, eb[4] = {vb.x, vb.y, vb.z, vb.w};
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
          uint32_t lo = (ea[qq] & 0xFFFFu) | (eb[qq] << 16);
          uint32_t hi = (ea[qq] >> 16) | (eb[qq] & 0xFFFF0000u);
          *reinterpret_cast<uint32_t *>(myvt + (c * 8 + 2 * qq) * PT + 2 * pp) = lo;
          *reinterpret_cast<uint32_t *>(myvt + (c * 8 + 2 * qq + 1) * PT + 2 * pp) = hi;
        }
      }
    }
    // Online softmax per head (lane column); lane groups share the max.
    float tm = kNegInf;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (t0 + rb * 16 + 4 * lg + i >= r1) acc[rb][i] = kNegInf;
        tm = fmaxf(tm, acc[rb][i]);
      }
    tm = fmaxf(tm, shfl_xor(tm, 16));
    tm = fmaxf(tm, shfl_xor(tm, 32));
    const float mc = fmaxf(mrow, tm * sc);
    const float alpha = fast_exp2(mrow - mc);
    mrow = mc;
    lsum *= alpha;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) O[mb] *= alpha;
    float pr[2][4];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pr[rb][i] = fast_exp2(fmaf(acc[rb][i], sc, -mc));
        lsum += pr[rb][i];
      }
    // Probabilities as a bf16 hi + lo pair keep the product at fp32 accuracy.
    const u32x4 hi = {pack_bf16(pr[0][0], pr[0][1]), pack_bf16(pr[0][2], pr[0][3]),
                      pack_bf16(pr[1][0], pr[1][1]), pack_bf16(pr[1][2], pr[1][3])};
    const u32x4 lo = {pack_bf16(pr[0][0] - bf16_lo(hi.x), pr[0][1] - bf16_hi(hi.x)),
                      pack_bf16(pr[0][2] - bf16_lo(hi.y), pr[0][3] - bf16_hi(hi.y)),
                      pack_bf16(pr[1][0] - bf16_lo(hi.z), pr[1][1] - bf16_hi(hi.z)),
                      pack_bf16(pr[1][2] - bf16_lo(hi.w), pr[1][3] - bf16_hi(hi.w))};
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0): this wave's LDS writes landed
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const bf16x8 a = load_split8(myvt + (mb * 16 + lr) * PT, 4 * lg);
      O[mb] = mfma_bf16(a, as_bf16x8(hi), O[mb]);
      O[mb] = mfma_bf16(a, as_bf16x8(lo), O[mb]);
    }
    __builtin_amdgcn_wave_barrier();  // reads done before the next tile's writes
  }

  // Merge the four waves, then store this split's partial.
  lsum += shfl_xor(lsum, 16);
  lsum += shfl_xor(lsum, 32);
  if (lg == 0) wml[w][lr] = make_float2(mrow <= kFloor ? kNegInf : mrow, lsum);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int i = 0; i < 4; ++i) wo[w][lr][mb * 16 + 4 * lg + i] = O[mb][i];
  __syncthreads();
  const int64_t pbase = ((int64_t)u * p.nsplit + split) * 16;
  for (int e = tid; e < 16 * D; e += 256) {
    const int h = e / D, x = e % D;
    float M = kNegInf;
#pragma unroll
    for (int i = 0; i < 4; ++i) M = fmaxf(M, wml[i][h].x);
    float o = 0.f, s = 0.f;
    if (M != kNegInf) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float2 ml = wml[i][h];
        if (ml.x != kNegInf) {
          const float f = fast_exp2(ml.x - M);
          o += f * wo[i][h][x];
          s += f * ml.y;
        }
      }
    }
    stg(p.part_o + (pbase + h) * D + x, o);
    if (x == 0) stg(p.part_ml + pbase + h, make_float2(M, s));
  }
}

// Merge split partials in split order; out = O / sum (zeros for empty caches).
template <int D>
__global__ __launch_bounds__(256) void k_decode_combine(DecodePlan p) {
  const int u = blockIdx.x;
  const int len = min(ldg(p.len + u), ldg(p.cap + u));
  const int ns = len > 0 ? min(p.nsplit, (len + p.split_rows - 1) / p.split_rows) : 1;
  const int g = u % p.Hkv;
  const int lb_ = u / p.Hkv;
  const float sc = p.sc;
  for (int e = threadIdx.x; e < p.G * D; e += 256) {
    const int h = e / D, x = e % D;
    float M = kNegInf;
    for (int s = 0; s < ns; ++s) M = fmaxf(M, ldg(p.part_ml + ((int64_t)u * p.nsplit + s) * 16 + h).x);
    float o = 0.f, sum = 0.f;
    if (M != kNegInf) {
      for (int s = 0; s < ns; ++s) {
        const int64_t pb = ((int64_t)u * p.nsplit + s) * 16 + h;
        const float2 ml = ldg(p.part_ml + pb);
        if (ml.x == kNegInf) continue;
        const float f = fast_exp2(ml.x - M);
        o += f * ldg(p.part_o + pb * D + x);
        sum += f * ml.y;
      }
    }
    stg(p.out + ((int64_t)lb_ * p.Hq + (int64_t)g * p.G + h) * D + x, sum > 0.f ? o / sum : 0.f);
  }
}

}  // namespace

hipError_t launch_append(int32_t units, int32_t d, uint16_t *k_pool, uint16_t *v_pool,
                         const int64_t *row_off, const int32_t *cap, int32_t *len,
                         const uint16_t *k_new, const uint16_t *v_new, hipStream_t st) {
  if (units == 0) return hipSuccess;
  hipLaunchKernelGGL(k_append, dim3(units), dim3(64), 0, st, units, d, k_pool, v_pool, row_off,
                     cap, len, k_new, v_new);
  return hipGetLastError();
}

hipError_t launch_decode(const DecodePlan &p, hipStream_t st) {
  const int units = p.L * p.B * p.Hkv;
  if (units == 0) return hipSuccess;
  const uint32_t grid = (uint32_t)units * p.nsplit;
  if (p.d == 128) {
    hipLaunchKernelGGL(k_decode_attn<128>, dim3(grid), dim3(256), 0, st, p);
    hipLaunchKernelGGL(k_decode_combine<128>, dim3(units), dim3(256), 0, st, p);
  } else {
    hipLaunchKernelGGL(k_decode_attn<64>, dim3(grid), dim3(256), 0, st, p);
    hipLaunchKernelGGL(k_decode_combine<64>, dim3(units), dim3(256), 0, st, p);
  }
  return hipGetLastError();
}

}  // namespace vc
