// k_fuse.hip -- key pruning and value fusion of PruneKV (Sec. 3.2, "Asymmetric
// Key-Value Update"; Algorithm 1, Step 3):
//   K_new = K[kept]                                   (bit copy)
//   Phi   = row-softmax(V_k V_d^T / tau)              (Eq. (redistribution))
//   V_new = mu V_k + (1 - mu) Phi V_d                 (Eq. (weight_fusion))
// Phi is never stored: it is attention with queries V_k and keys = values =
// V_d, computed flash-style with an online softmax over 64-row tiles of V_d.
//
// Both contractions run on the bf16 matrix cores in transposed form:
//   S^T = V_d V_k^T     A = V_d rows (LDS, direct reads),     B = V_k (registers)
//   O^T = V_d^T P^T     A = V_d^T (LDS, transposing reads),   B = P^T (registers)
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

// Row pitch of the staged dropped tile: 32 bytes of padding.  Measured on
// gfx950, this keeps the transposing reads conflict-free and costs the direct
// 8-byte reads one extra cycle in three; a single row-major copy serves both.
template <int D>
constexpr int kPitchRow = D + 16;

// 8 bf16 at d = {c..c+3, c+16..c+19} of one staged row: the k-element order
// shared by both operands of S^T for lane group lg at k-step s (c = 32 s + 4 lg).
__device__ __forceinline__ bf16x8 load_split8_lds(const uint16_t *row, int c) {
  const u32x2 a = *reinterpret_cast<const u32x2 *>(row + c);
  const u32x2 b = *reinterpret_cast<const u32x2 *>(row + c + 16);
  return as_bf16x8(u32x4{a.x, a.y, b.x, b.y});
}

// gfx950 transposing LDS read: within each group of 16 lanes, lane 4a+b gets
// element b of the 8-byte chunks addressed by lanes a, a+4, a+8 and a+12.
__device__ __forceinline__ u32x2 lds_read_tr16(const uint16_t *p) {
  typedef short v4i16 __attribute__((ext_vector_type(4)));
  const v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16 *)(p));
  return __builtin_bit_cast(u32x2, v);
}

// Rows of one 64-row dropped tile between their global load and their LDS
// store: thread t owns rows 2*(t%32) and 2*(t%32)+1 and the 16-byte chunks
// (t/32) + 8*it of both.
template <int D>
struct DropRegs {
  static constexpr int kIt = D / 64;
  u32x4 a[kIt], b[kIt];
  __device__ __forceinline__ void load(const uint16_t *V, int ia, int ib, int c0) {
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int c = c0 + 8 * it;
      a[it] = ia >= 0 ? ld16(V + (int64_t)ia * D + c * 8) : u32x4{0, 0, 0, 0};
      b[it] = ib >= 0 ? ld16(V + (int64_t)ib * D + c * 8) : u32x4{0, 0, 0, 0};
    }
  }
  __device__ __forceinline__ void store(uint16_t *vr, int pp, int c0) const {
    constexpr int PR = kPitchRow<D>;
    const int ra = 2 * pp;
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
      const int c = c0 + 8 * it;
      *reinterpret_cast<u32x4 *>(vr + ra * PR + c * 8) = a[it];
      *reinterpret_cast<u32x4 *>(vr + (ra + 1) * PR + c * 8) = b[it];
    }
  }
};

// Workgroup = (layer, sequence, kv head, 128 kept rows); wave w owns kept rows
// w*32 + nb*16 + [0, 16) for nb = 0, 1, so every operand read from LDS feeds
// two matrix instructions.  Dropped tiles are double-buffered in LDS.
template <int D>
__global__ __launch_bounds__(256, 2) void k_fuse(PrunePlan p) {
  constexpr int KS = D / 32;
  constexpr int MB = D / 16;
  constexpr int PR = kPitchRow<D>;
  constexpr int NB = 2;
  __shared__ __attribute__((aligned(16))) uint16_t vr[2][kDropTile * PR];
  __shared__ int32_t kidx[kFuseRows];

  const uint32_t lb = xcd_block(blockIdx.x, gridDim.x);
  const int tile = lb % p.nfuse;
  const int u = lb / p.nfuse;
  const int g = u % p.Hkv;
  const int b = (u / p.Hkv) % p.B;
  const int l = u / (p.Hkv * p.B);
  const int k = ldg(p.kk + b * p.L + l);
  const int j0 = tile * kFuseRows;
  if (j0 >= k) return;
  const int n = ldg(p.nb + b);
  const int r = ldg(p.ns + b * p.L + l) - k;
  const int nrows = min(kFuseRows, k - j0);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;

  const int64_t orow = ldg(p.orow + l * (p.B + 1) + b) + (int64_t)g * k;
  const int32_t *idx = reinterpret_cast<const int32_t *>(ldg(p.lp + LP_IDX * p.L + l)) + orow;
  const int32_t *drop = reinterpret_cast<const int32_t *>(ldg(p.lp + LP_DROP * p.L + l)) +
                        ldg(p.drow + l * (p.B + 1) + b) + (int64_t)g * r;
  const int64_t ioff = (ldg(p.toff + b) * p.Hkv + (int64_t)g * n) * D;
  const uint16_t *Kin = reinterpret_cast<const uint16_t *>(ldg(p.lp + LP_K_IN * p.L + l)) + ioff;
  const uint16_t *Vin = reinterpret_cast<const uint16_t *>(ldg(p.lp + LP_V_IN * p.L + l)) + ioff;
  uint16_t *Kout = reinterpret_cast<uint16_t *>(ldg(p.lp + LP_K_OUT * p.L + l)) + orow * D;

  // Token indices come from the selection kernel; clamping keeps every
  // gathered row inside the unit even if they were corrupted.
  if (tid < nrows) kidx[tid] = min(max(ldg(idx + j0 + tid), 0), n - 1);

  // Dropped-tile pipeline: indices one tile ahead of the rows, rows one tile
  // ahead of the matrix work.
  const int ntiles = (r + kDropTile - 1) / kDropTile;
  const int pp = tid & 31, c0 = tid >> 5;
  auto drop_idx = [&](int dt, int row) -> int {
    const int j = dt * kDropTile + row;
    return j < r ? min(max(ldg(drop + j), 0), n - 1) : -1;
  };
  DropRegs<D> dr;
  int ia = -1, ib = -1;
  if (ntiles > 0) {
    dr.load(Vin, drop_idx(0, 2 * pp), drop_idx(0, 2 * pp + 1), c0);
    if (ntiles > 1) { ia = drop_idx(1, 2 * pp); ib = drop_idx(1, 2 * pp + 1); }
    dr.store(vr[0], pp, c0);
    if (ntiles > 1) dr.load(Vin, ia, ib, c0);
    if (ntiles > 2) { ia = drop_idx(2, 2 * pp); ib = drop_idx(2, 2 * pp + 1); }
  }
  __syncthreads();

  // Key pruning: bit copies of the kept rows.
  for (int c = tid; c < nrows * (D / 8); c += 256) {
    const int row = c / (D / 8), col = c % (D / 8);
    st16(Kout + (int64_t)(j0 + row) * D + col * 8, ld16(Kin + (int64_t)kidx[row] * D + col * 8));
  }

  // Kept values of this lane's rows, in the split k-element order.
  bf16x8 bvk[NB][KS];
  bool kvalid[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int krow = w * 32 + nb * 16 + lr;
    kvalid[nb] = krow < nrows;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const uint16_t *row = Vin + (int64_t)kidx[kvalid[nb] ? krow : 0] * D + 32 * s + 4 * lg;
      const u32x2 x = ld8(row), y = ld8(row + 16);
      bvk[nb][s] = kvalid[nb] ? as_bf16x8(u32x4{x.x, x.y, y.x, y.y}) : as_bf16x8(u32x4{0, 0, 0, 0});
    }
  }

  f32x4 O[NB][MB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) O[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Running maxima kept pre-multiplied by log2(e)/tau: every rescale factor is
  // exp2 of a plain difference (exp2(floor - max) = 0 on the first tile).
  float mrow[NB] = {-1e30f, -1e30f}, lsum[NB] = {0.f, 0.f};
  const float tc = p.tc;
  // Transposing-read address of this lane inside a staged tile: group lane j
  // points at row j/4 (plus the k-step base) and column 4*(j%4) (plus 16*mb).
  const int tr_row = 4 * lg + (lr >> 2), tr_col = 4 * (lr & 3);

  for (int dt = 0; dt < ntiles; ++dt) {
    const uint16_t *vt = vr[dt & 1];
    const int nd = min(kDropTile, r - dt * kDropTile);

    // S^T = V_d V_k^T for 64 dropped x 32 kept rows.
    f32x4 acc[NB][4];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int db = 0; db < 4; ++db) acc[nb][db] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s)
#pragma unroll
      for (int db = 0; db < 4; ++db) {
        const bf16x8 a = load_split8_lds(vt + (db * 16 + lr) * PR, 32 * s + 4 * lg);
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) acc[nb][db] = mfma_bf16(a, bvk[nb][s], acc[nb][db]);
      }

    // Online softmax over dropped rows; the four lane groups of a kept row
    // share one running max.
    float pr[NB][4][4];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      if (nd < kDropTile) {
#pragma unroll
        for (int db = 0; db < 4; ++db)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            if (db * 16 + 4 * lg + i >= nd) acc[nb][db][i] = kNegInf;
      }
      float tm = acc[nb][0][0];
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) tm = fmaxf(tm, acc[nb][db][i]);
      tm = fmaxf(tm, shfl_xor(tm, 16));
      tm = fmaxf(tm, shfl_xor(tm, 32));
      const float mc = fmaxf(mrow[nb], tm * tc);
      const float alpha = fast_exp2(mrow[nb] - mc);
      mrow[nb] = mc;
      lsum[nb] *= alpha;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) O[nb][mb] *= alpha;
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          pr[nb][db][i] = fast_exp2(fmaf(acc[nb][db][i], tc, -mc));
          lsum[nb] += pr[nb][db][i];
        }
    }

    // O^T += V_d^T P^T, two 32-row k-steps; V_d^T comes from transposing reads.
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      bf16x8 bph[NB], bpl[NB];
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const float *p0 = pr[nb][2 * t2], *p1 = pr[nb][2 * t2 + 1];
        const u32x4 hi = {pack_bf16(p0[0], p0[1]), pack_bf16(p0[2], p0[3]), pack_bf16(p1[0], p1[1]),
                          pack_bf16(p1[2], p1[3])};
        bph[nb] = as_bf16x8(hi);
        if (p.v_fp32) {
          const u32x4 lo = {pack_bf16(p0[0] - bf16_lo(hi.x), p0[1] - bf16_hi(hi.x)),
                            pack_bf16(p0[2] - bf16_lo(hi.y), p0[3] - bf16_hi(hi.y)),
                            pack_bf16(p1[0] - bf16_lo(hi.z), p1[1] - bf16_hi(hi.z)),
                            pack_bf16(p1[2] - bf16_lo(hi.w), p1[3] - bf16_hi(hi.w))};
          bpl[nb] = as_bf16x8(lo);
        }
      }
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const uint16_t *base = vt + (32 * t2 + tr_row) * PR + 16 * mb + tr_col;
        const u32x2 lo4 = lds_read_tr16(base), hi4 = lds_read_tr16(base + 16 * PR);
        const bf16x8 a = as_bf16x8(u32x4{lo4.x, lo4.y, hi4.x, hi4.y});
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
          O[nb][mb] = mfma_bf16(a, bph[nb], O[nb][mb]);
          if (p.v_fp32) O[nb][mb] = mfma_bf16(a, bpl[nb], O[nb][mb]);
        }
      }
    }

    // Stage tile dt+1 into the other buffer, then fetch tile dt+2.
    if (dt + 1 < ntiles) dr.store(vr[(dt + 1) & 1], pp, c0);
    if (dt + 2 < ntiles) dr.load(Vin, ia, ib, c0);
    if (dt + 3 < ntiles) { ia = drop_idx(dt + 3, 2 * pp); ib = drop_idx(dt + 3, 2 * pp + 1); }
    __syncthreads();
  }

  const float mu = p.mu, omu = 1.f - p.mu;
  void *vout = reinterpret_cast<void *>(ldg(p.lp + LP_V_OUT * p.L + l));
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float ls = lsum[nb];
    ls += shfl_xor(ls, 16);
    ls += shfl_xor(ls, 32);
    if (!kvalid[nb]) continue;
    const float inv = (r > 0 && ls > 0.f) ? 1.f / ls : 0.f;
    const int64_t orow_j = orow + j0 + w * 32 + nb * 16 + lr;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const u32x4 kv = as_u32x4(bvk[nb][mb / 2]);
      const uint32_t w0 = (mb & 1) ? kv.z : kv.x, w1 = (mb & 1) ? kv.w : kv.y;
      const float vk[4] = {bf16_lo(w0), bf16_hi(w0), bf16_lo(w1), bf16_hi(w1)};
      float o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = (r > 0) ? mu * vk[i] + omu * (O[nb][mb][i] * inv) : vk[i];
      const int64_t off = orow_j * D + mb * 16 + 4 * lg;
      if (p.v_fp32)
        st16(reinterpret_cast<float *>(vout) + off,
             u32x4{__float_as_uint(o[0]), __float_as_uint(o[1]), __float_as_uint(o[2]), __float_as_uint(o[3])});
      else
        st8(reinterpret_cast<uint16_t *>(vout) + off, u32x2{pack_bf16(o[0], o[1]), pack_bf16(o[2], o[3])});
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
