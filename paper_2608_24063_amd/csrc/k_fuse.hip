// k_fuse.hip -- key pruning and value fusion of PruneKV (Sec. 3.2, "Asymmetric
// Key-Value Update"; Algorithm 1, Step 3):
//   K_new = K[kept]                                   (bit copy)
//   Phi   = row-softmax(V_k V_d^T / tau)              (Eq. (redistribution))
//   V_new = mu V_k + (1 - mu) Phi V_d                 (Eq. (weight_fusion))
// Phi is never stored: it is attention with queries V_k and keys = values =
// V_d, computed flash-style with an online softmax over 64-row tiles of V_d.
//
// Workgroup = (layer, sequence, kv head, 64 kept rows); wave w owns 16 kept
// rows.  Both contractions run on the bf16 matrix cores in transposed form:
//   S^T = V_d V_k^T     A = V_d rows (LDS, row-major), B = V_k (registers)
//   O^T = V_d^T P^T     A = V_d^T (LDS, transposed),  B = P^T (registers)
// so the scores' accumulator layout (lane: kept row l%16, dropped rows
// 4*(l/16)+i) is directly the B operand of the second product, and each lane
// ends holding kept row l%16, columns 16*mb + 4*(l/16) + i -- the same columns
// it loaded of V_k, which the mu-blend reuses.  With fp32 output the
// probabilities enter the second product as a bf16 hi + lo pair.
#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

constexpr float kNegInf = -__builtin_inff();

// 8 bf16 at d = {c, c+1, c+2, c+3, c+16, ..., c+19}: the k-element order shared
// by both operands of S^T for lane group lg at k-step s (c = 32 s + 4 lg).
__device__ __forceinline__ bf16x8 load_split8(const uint16_t *row, int c) {
  u32x2 a = *reinterpret_cast<const u32x2 *>(row + c);
  u32x2 b = *reinterpret_cast<const u32x2 *>(row + c + 16);
  return as_bf16x8(u32x4{a.x, a.y, b.x, b.y});
}

template <int D>
__global__ __launch_bounds__(256, 2) void k_fuse(PrunePlan p) {
  constexpr int KS = D / 32;
  constexpr int MB = D / 16;
  constexpr int PR = D + 8;           // row-major pitch (bf16)
  constexpr int PT = kDropTile + 8;   // transposed pitch (bf16)
  __shared__ __attribute__((aligned(16))) uint16_t vr[kDropTile * PR];
  __shared__ __attribute__((aligned(16))) uint16_t vt[D * PT];
  __shared__ int32_t kidx[kFuseRows];
  __shared__ int32_t didx[kDropTile];

  const uint32_t lb = xcd_block(blockIdx.x, gridDim.x);
  const int tile = lb % p.nfuse;
  const int u = lb / p.nfuse;
  const int g = u % p.Hkv;
  const int b = (u / p.Hkv) % p.B;
  const int l = u / (p.Hkv * p.B);
  const int n = p.nb[b];
  const int k = p.kk[b * p.L + l];
  const int r = p.ns[b * p.L + l] - k;
  const int j0 = tile * kFuseRows;
  if (j0 >= k) return;
  const int nrows = min(kFuseRows, k - j0);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;

  const int64_t orow = p.orow[l * (p.B + 1) + b] + (int64_t)g * k;
  const int32_t *idx = reinterpret_cast<const int32_t *>(p.lp[LP_IDX * p.L + l]) + orow;
  const int32_t *drop = reinterpret_cast<const int32_t *>(p.lp[LP_DROP * p.L + l]) +
                        p.drow[l * (p.B + 1) + b] + (int64_t)g * r;
  const int64_t ioff = ((int64_t)p.toff[b] * p.Hkv + (int64_t)g * n) * D;
  const uint16_t *Kin = reinterpret_cast<const uint16_t *>(p.lp[LP_K_IN * p.L + l]) + ioff;
  const uint16_t *Vin = reinterpret_cast<const uint16_t *>(p.lp[LP_V_IN * p.L + l]) + ioff;
  uint16_t *Kout = reinterpret_cast<uint16_t *>(p.lp[LP_K_OUT * p.L + l]) + orow * D;

  // Token indices come from the selection kernel; clamping keeps every
  // gathered row inside the unit even if they were corrupted.
  if (tid < nrows) kidx[tid] = min(max(idx[j0 + tid], 0), n - 1);
  __syncthreads();

  // Key pruning: bit copies of the kept rows.
  for (int c = tid; c < nrows * (D / 8); c += 256) {
    const int row = c / (D / 8), col = c % (D / 8);
    *reinterpret_cast<u32x4 *>(Kout + (int64_t)(j0 + row) * D + col * 8) =
        *reinterpret_cast<const u32x4 *>(Kin + (int64_t)kidx[row] * D + col * 8);
  }

  // Kept values of this lane's row, in the split k-element order.
  const int krow = w * 16 + lr;
  const bool kvalid = krow < nrows;
  bf16x8 bvk[KS];
#pragma unroll
  for (int s = 0; s < KS; ++s)
    bvk[s] = kvalid ? load_split8(Vin + (int64_t)kidx[krow] * D, 32 * s + 4 * lg)
                    : as_bf16x8(u32x4{0, 0, 0, 0});

  f32x4 O[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) O[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  float mrow = kNegInf, lsum = 0.f;
  const float tc = p.tc;

  const int ntiles = (r + kDropTile - 1) / kDropTile;
  for (int dt = 0; dt < ntiles; ++dt) {
    const int d0 = dt * kDropTile;
    const int nd = min(kDropTile, r - d0);
    __syncthreads();  // previous tile fully consumed
    if (tid < kDropTile) didx[tid] = tid < nd ? min(max(drop[d0 + tid], 0), n - 1) : -1;
    __syncthreads();
    // Stage the dropped rows: row-major copy and transposed copy.
    {
      const int pp = tid & 31, c0 = tid >> 5;
#pragma unroll
      for (int it = 0; it < D / 64; ++it) {
        const int c = c0 + 8 * it;
        const int ra = 2 * pp, rb = 2 * pp + 1;
        u32x4 va = {0, 0, 0, 0}, vb = {0, 0, 0, 0};
        if (didx[ra] >= 0) va = *reinterpret_cast<const u32x4 *>(Vin + (int64_t)didx[ra] * D + c * 8);
        if (didx[rb] >= 0) vb = *reinterpret_cast<const u32x4 *>(Vin + (int64_t)didx[rb] * D + c * 8);
        *reinterpret_cast<u32x4 *>(vr + ra * PR + c * 8) = va;
        *reinterpret_cast<u32x4 *>(vr + rb * PR + c * 8) = vb;
        const uint32_t ea[4] = {va.x, va.y, va.z, va.w}, eb[4] = {vb.x, vb.y, vb.z, vb.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          uint32_t lo = (ea[q] & 0xFFFFu) | (eb[q] << 16);
          uint32_t hi = (ea[q] >> 16) | (eb[q] & 0xFFFF0000u);
          *reinterpret_cast<uint32_t *>(vt + (c * 8 + 2 * q) * PT + ra) = lo;
          *reinterpret_cast<uint32_t *>(vt + (c * 8 + 2 * q + 1) * PT + ra) = hi;
        }
      }
    }
    __syncthreads();

    // S^T = V_d V_k^T for 64 dropped x 16 kept rows.
    f32x4 acc[4];
#pragma unroll
    for (int db = 0; db < 4; ++db) acc[db] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int db = 0; db < 4; ++db)
        acc[db] = mfma_bf16(load_split8(vr + (db * 16 + lr) * PR, 32 * s + 4 * lg), bvk[s], acc[db]);

    // Online softmax over dropped rows; the four lane groups of a kept row
    // share one running max.
    float tm = kNegInf;
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (db * 16 + 4 * lg + i >= nd) acc[db][i] = kNegInf;
        tm = fmaxf(tm, acc[db][i]);
      }
    tm = fmaxf(tm, shfl_xor(tm, 16));
    tm = fmaxf(tm, shfl_xor(tm, 32));
    const float mnew = fmaxf(mrow, tm);
    const float alpha = (mrow == kNegInf) ? 0.f : fast_exp2(mrow * tc - mnew * tc);
    mrow = mnew;
    lsum *= alpha;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) O[mb] *= alpha;
    const float mc = mnew * tc;
    float pr[4][4];
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pr[db][i] = fast_exp2(fmaf(acc[db][i], tc, -mc));
        lsum += pr[db][i];
      }

    // O^T += V_d^T P^T, two 32-row k-steps.
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      const float *p0 = pr[2 * t2], *p1 = pr[2 * t2 + 1];
      u32x4 hi = {pack_bf16(p0[0], p0[1]), pack_bf16(p0[2], p0[3]), pack_bf16(p1[0], p1[1]),
                  pack_bf16(p1[2], p1[3])};
      bf16x8 bph = as_bf16x8(hi);
      bf16x8 bpl;
      if (p.v_fp32) {
        u32x4 lo = {pack_bf16(p0[0] - bf16_lo(hi.x), p0[1] - bf16_hi(hi.x)),
                    pack_bf16(p0[2] - bf16_lo(hi.y), p0[3] - bf16_hi(hi.y)),
                    pack_bf16(p1[0] - bf16_lo(hi.z), p1[1] - bf16_hi(hi.z)),
                    pack_bf16(p1[2] - bf16_lo(hi.w), p1[3] - bf16_hi(hi.w))};
        bpl = as_bf16x8(lo);
      }
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        bf16x8 a = load_split8(vt + (mb * 16 + lr) * PT, 32 * t2 + 4 * lg);
        O[mb] = mfma_bf16(a, bph, O[mb]);
        if (p.v_fp32) O[mb] = mfma_bf16(a, bpl, O[mb]);
      }
    }
  }

  if (!kvalid) return;
  lsum += shfl_xor(lsum, 16);
  lsum += shfl_xor(lsum, 32);
  const float mu = p.mu, omu = 1.f - p.mu;
  const float inv = (r > 0 && lsum > 0.f) ? 1.f / lsum : 0.f;
  const int64_t orow_j = orow + j0 + krow;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const u32x4 kv = as_u32x4(bvk[mb / 2]);
    const uint32_t w0 = (mb & 1) ? kv.z : kv.x, w1 = (mb & 1) ? kv.w : kv.y;
    float vk[4] = {bf16_lo(w0), bf16_hi(w0), bf16_lo(w1), bf16_hi(w1)};
    float o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = (r > 0) ? mu * vk[i] + omu * (O[mb][i] * inv) : vk[i];
    const int64_t off = orow_j * D + mb * 16 + 4 * lg;
    if (p.v_fp32) {
      *reinterpret_cast<float4 *>(reinterpret_cast<float *>(p.lp[LP_V_OUT * p.L + l]) + off) =
          make_float4(o[0], o[1], o[2], o[3]);
    } else {
      *reinterpret_cast<u32x2 *>(reinterpret_cast<uint16_t *>(p.lp[LP_V_OUT * p.L + l]) + off) =
          u32x2{pack_bf16(o[0], o[1]), pack_bf16(o[2], o[3])};
    }
  }
}

}  // namespace

hipError_t launch_fuse(const PrunePlan &p, hipStream_t st) {
  const uint32_t grid = (uint32_t)p.h * p.B * p.Hkv * p.nfuse;
  if (grid == 0) return hipSuccess;
  if (p.d == 128)
    hipLaunchKernelGGL(k_fuse<128>, dim3(grid), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(k_fuse<64>, dim3(grid), dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace vc
