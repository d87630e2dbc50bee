// k_decode.hip -- decode over the (compressed) cache (Sec. 2, "VLLM
// Decoding"): append one K/V row per (layer, sequence, kv head) and attend one
// query per query head over all cached rows.
//
// Attention is split over rows: workgroup = (unit, split of split_rows rows),
// and each of its four waves takes 32-row tiles in turn, the next tile's rows
// in flight while the current one is processed.  The G query heads of
// a kv head form one 16-column MFMA block (heads >= G are zero), so each K/V
// row is read once for all of them:
//   S^T = K Q^T   A = K rows straight from HBM, B = Q (registers)
//   O^T = V^T P^T A = V^T (per-wave LDS tile, transposing reads), B = P^T
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

// gfx950 transposing LDS read: within each group of 16 lanes, lane 4a+b gets
// element b of the 8-byte chunks addressed by lanes a, a+4, a+8 and a+12.
__device__ __forceinline__ u32x2 lds_read_tr16(const uint16_t *p) {
  typedef short v4i16 __attribute__((ext_vector_type(4)));
  const v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16 *)(p));
  return __builtin_bit_cast(u32x2, v);
}

// K and V of one 32-row tile in registers.  K: lane (lr, lg) holds row
// rb*16 + lr, elements 32 s + 8 lg .. + 7 (the S^T A operand).  V: lane holds
// 16-byte chunk lane % 16 of rows lane / 16 + 4 it (staged to LDS row-major).
template <int D>
struct RowTile {
  static constexpr int KS = D / 32;
  static constexpr int kVIt = 32 * D / 8 / 64;  // 16-byte V chunks per lane
  u32x4 k[2][KS];
  u32x4 v[kVIt];
  // Row `nrow` (if >= 0) is not in the pool yet: it comes from knew / vnew.
  __device__ __forceinline__ void load(const uint16_t *Kp, const uint16_t *Vp, int t0, int r1, int lr, int lg,
                                       int lane, int nrow, const uint16_t *knew, const uint16_t *vnew) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const int row = min(t0 + rb * 16 + lr, r1 - 1);
      const uint16_t *src = row == nrow ? knew : Kp + (int64_t)row * D;
#pragma unroll
      for (int s = 0; s < KS; ++s) k[rb][s] = ld16(src + 32 * s + 8 * lg);
    }
    constexpr int kCpr = D / 8;  // chunks per row
#pragma unroll
    for (int it = 0; it < kVIt; ++it) {
      const int c = lane + 64 * it;
      const int row = min(t0 + c / kCpr, r1 - 1);
      const uint16_t *src = row == nrow ? vnew : Vp + (int64_t)row * D;
      v[it] = ld16(src + (c % kCpr) * 8);
    }
  }
};

// Partials of the fused step are exchanged between workgroups that may sit
// on different XCDs (separate L2s): they are written and read with
// device-coherent accesses instead of fences that would write back and
// invalidate a whole L2.
template <bool COHERENT>
__device__ __forceinline__ void st_part(float *p, float v) {
  if (COHERENT)
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  else
    stg(p, v);
}
template <bool COHERENT>
__device__ __forceinline__ float ld_part(const float *p) {
  if (COHERENT) return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return ldg(p);
}

template <int D>
struct DecodeSmem {
  static constexpr int PR = D + 16;  // V tile row pitch: conflict-free transposing reads
  uint16_t vt[4][kRowTile * PR] __attribute__((aligned(16)));
  float2 wml[4][16];
  float wo[4][16][D + 4] __attribute__((aligned(16)));
  uint32_t last;
};

// Attention of the query heads of unit u over cache rows [r0, r1) (row nrow,
// if >= 0, read from knew / vnew); writes the split's partial (max, sum, O).
// Where a split's result goes: its partial (plain or device-coherent stores),
// or, for a unit with a single split, the normalised output itself.
enum SplitOut { kPartial = 0, kPartialCoherent = 1, kOutput = 2 };

template <int D, int OUT>
__device__ __forceinline__ void attend_split(const DecodePlan &p, DecodeSmem<D> &sm, int u, int split, int r0,
                                             int r1, int nrow, const uint16_t *knew, const uint16_t *vnew) {
  constexpr int KS = D / 32;
  constexpr int MB = D / 16;
  constexpr int PR = DecodeSmem<D>::PR;
  auto &vt = sm.vt;
  auto &wml = sm.wml;
  auto &wo = sm.wo;
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
  const int tr_row = 4 * lg + (lr >> 2), tr_col = 4 * (lr & 3);

  // Wave w takes tiles w, w+4, ...; the next tile's rows are in flight while
  // the current one is processed.
  const int ntiles = r1 > r0 ? (r1 - r0 + kRowTile - 1) / kRowTile : 0;
  RowTile<D> cur, nxt;
  if (w < ntiles) cur.load(Kp, Vp, r0 + w * kRowTile, r1, lr, lg, lane, nrow, knew, vnew);
  for (int t = w; t < ntiles; t += 4) {
    const int t0 = r0 + t * kRowTile;
    if (t + 4 < ntiles) nxt.load(Kp, Vp, t0 + 4 * kRowTile, r1, lr, lg, lane, nrow, knew, vnew);
    // S^T = K Q^T for 2 blocks of 16 rows.
    f32x4 acc[2];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS; ++s) acc[rb] = mfma_bf16(as_bf16x8(cur.k[rb][s]), bq[s], acc[rb]);
    }
    // V rows -> per-wave LDS tile, row-major (read back transposed below).
    {
      constexpr int kCpr = D / 8;
#pragma unroll
      for (int it = 0; it < RowTile<D>::kVIt; ++it) {
        const int c = lane + 64 * it;
        *reinterpret_cast<u32x4 *>(myvt + (c / kCpr) * PR + (c % kCpr) * 8) = cur.v[it];
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
    // O^T += V^T P^T: A = V^T (16 d x 32 rows) from transposing reads.
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const uint16_t *base = myvt + tr_row * PR + 16 * mb + tr_col;
      const u32x2 lo4 = lds_read_tr16(base), hi4 = lds_read_tr16(base + 16 * PR);
      const bf16x8 a = as_bf16x8(u32x4{lo4.x, lo4.y, hi4.x, hi4.y});
      O[mb] = mfma_bf16(a, as_bf16x8(hi), O[mb]);
      O[mb] = mfma_bf16(a, as_bf16x8(lo), O[mb]);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // reads done before the next tile's writes
    __builtin_amdgcn_wave_barrier();
    cur = nxt;
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
    if (OUT == kOutput) {
      // The merge of a single split: its factor is exp2(0) = 1 exactly.
      if (h < p.G) stg(p.out + ((int64_t)lb_ * p.Hq + (int64_t)g * p.G + h) * D + x, s > 0.f ? o / s : 0.f);
      continue;
    }
    st_part<OUT == kPartialCoherent>(p.part_o + (pbase + h) * D + x, o);
    if (x == 0) {
      float *ml = reinterpret_cast<float *>(p.part_ml + pbase + h);
      st_part<OUT == kPartialCoherent>(ml, M);
      st_part<OUT == kPartialCoherent>(ml + 1, s);
    }
  }
}

template <int D>
__global__ __launch_bounds__(256, 2) void k_decode_attn(DecodePlan p) {
  __shared__ DecodeSmem<D> sm;
  const uint32_t lb = xcd_block(blockIdx.x, gridDim.x);
  const int split = lb % p.nsplit;
  const int u = lb / p.nsplit;
  const int len = min(ldg(p.len + u), ldg(p.cap + u));
  const int r0 = split * p.split_rows;
  if (r0 >= len && split > 0) return;  // uniform: nothing for this split
  attend_split<D, kPartial>(p, sm, u, split, r0, min(len, r0 + p.split_rows), -1, nullptr, nullptr);
}

// Merge the split partials of unit u in split order; out = O / sum (zeros
// for an empty cache).  Every partial of an output element is loaded in one
// batch.
template <int D, bool COHERENT>
__device__ __forceinline__ void merge_splits(const DecodePlan &p, int u, int ns) {
  const int g = u % p.Hkv;
  const int lb_ = u / p.Hkv;
  for (int e = threadIdx.x; e < p.G * D; e += 256) {
    const int h = e / D, x = e % D;
    float2 ml[kMaxDecodeSplits];
    float po[kMaxDecodeSplits];
#pragma unroll
    for (int s = 0; s < kMaxDecodeSplits; ++s) {
      const int64_t pb = ((int64_t)u * p.nsplit + s) * 16 + h;
      const float *mlp = reinterpret_cast<const float *>(p.part_ml + pb);
      ml[s] = s < ns ? make_float2(ld_part<COHERENT>(mlp), ld_part<COHERENT>(mlp + 1)) : make_float2(kNegInf, 0.f);
      po[s] = s < ns ? ld_part<COHERENT>(p.part_o + pb * D + x) : 0.f;
    }
    float M = kNegInf;
#pragma unroll
    for (int s = 0; s < kMaxDecodeSplits; ++s) M = fmaxf(M, ml[s].x);
    float o = 0.f, sum = 0.f;
    if (M != kNegInf) {
#pragma unroll
      for (int s = 0; s < kMaxDecodeSplits; ++s) {
        if (ml[s].x == kNegInf) continue;
        const float f = fast_exp2(ml[s].x - M);
        o += f * po[s];
        sum += f * ml[s].y;
      }
    }
    stg(p.out + ((int64_t)lb_ * p.Hq + (int64_t)g * p.G + h) * D + x, sum > 0.f ? o / sum : 0.f);
  }
}

// One decode step in one launch: append (the split holding the new row takes
// it from k_new / v_new and writes it to the pool), attention per split, and
// the merge done by the last split of each unit to arrive, which also
// advances len and re-arms the unit's counter.
template <int D>
__global__ __launch_bounds__(256, 2) void k_decode_step(DecodePlan p) {
  __shared__ DecodeSmem<D> sm;
  const uint32_t lb = xcd_block(blockIdx.x, gridDim.x);
  const int split = lb % p.nsplit;
  const int u = lb / p.nsplit;
  const int len0 = ldg(p.len + u), cap = ldg(p.cap + u);
  const bool room = len0 < cap;
  const int len = room ? len0 + 1 : min(len0, cap);  // rows attended this step
  // Rows past nsplit * split_rows (a length beyond max_rows) are not attended.
  const int ns = min(p.nsplit, max(1, (len + p.split_rows - 1) / p.split_rows));
  // Every launched split of the unit arrives at the counter below, so every
  // read of len above happens before the last arriver advances it.
  if (split < ns) {  // uniform
    const int r0 = split * p.split_rows, r1 = min(len, r0 + p.split_rows);
    const int nrow = room ? len0 : -1;
    const uint16_t *knew = p.k_new + (int64_t)u * D, *vnew = p.v_new + (int64_t)u * D;
    if (room && nrow >= r0 && nrow < r1 && threadIdx.x < 2 * (D / 8)) {
      const int c = threadIdx.x, cc = c % (D / 8);
      const int64_t dst = (ldg(p.row_off + u) + nrow) * D + cc * 8;
      if (c < D / 8)
        st16(p.k_pool_w + dst, ld16(knew + cc * 8));
      else
        st16(p.v_pool_w + dst, ld16(vnew + cc * 8));
    }
    if (ns == 1)
      attend_split<D, kOutput>(p, sm, u, split, r0, r1, nrow, knew, vnew);
    else
      attend_split<D, kPartialCoherent>(p, sm, u, split, r0, r1, nrow, knew, vnew);
  }
  if (p.nsplit == 1) {  // the only workgroup of the unit: nothing to merge or count
    if (threadIdx.x == 0 && room) stg(p.len_w + u, len);
    return;
  }
  // The partial's device-coherent stores complete before the arrival is
  // counted; the last arriver reads every partial with device-coherent loads.
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (threadIdx.x == 0)
    sm.last = __hip_atomic_fetch_add(p.arrive + u, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
              (uint32_t)(p.nsplit - 1);
  __syncthreads();
  if (!sm.last) return;
  if (ns > 1) merge_splits<D, true>(p, u, ns);
  if (threadIdx.x == 0) {
    __hip_atomic_store(p.arrive + u, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (room) stg(p.len_w + u, len);
  }
}

// Merge split partials of each unit (second kernel of the two-call path).
template <int D>
__global__ __launch_bounds__(256) void k_decode_combine(DecodePlan p) {
  const int u = blockIdx.x;
  const int len = min(ldg(p.len + u), ldg(p.cap + u));
  merge_splits<D, false>(p, u, len > 0 ? min(p.nsplit, (len + p.split_rows - 1) / p.split_rows) : 1);
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

hipError_t launch_decode_step(const DecodePlan &p, hipStream_t st) {
  const int units = p.L * p.B * p.Hkv;
  if (units == 0) return hipSuccess;
  const uint32_t grid = (uint32_t)units * p.nsplit;
  if (p.d == 128)
    hipLaunchKernelGGL(k_decode_step<128>, dim3(grid), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(k_decode_step<64>, dim3(grid), dim3(256), 0, st, p);
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
