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
//
// Pipeline per workgroup: dropped-row indices are fetched four tiles ahead,
// the rows themselves three tiles ahead into two register sets, and staged
// into one of two LDS buffers one tile ahead; LDS operands of the matrix
// products are read one k-step ahead.  The running row maximum is only
// raised when a tile's logits exceed it by more than 2^kSlack, so most tiles
// skip the cross-lane reduction and the rescale of the accumulators.
#include <type_traits>

#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

constexpr float kNegInf = -__builtin_inff();
// Probabilities are allowed to reach 2^kSlack before the running maximum is
// raised (and the accumulators rescaled); fp32 has ample range for that.
constexpr float kSlack = 8.f;

// Staged dropped tile: rows of D bf16 at a pitch of D + 16 elements.  On
// gfx950 (LDS serves 64 banks x 4 bytes per pass) this pitch keeps all three
// access patterns below conflict-free at full rate (measured): 16-byte writes
// of one row per 16 lanes, 16-byte reads of 16 rows x 4 chunks (the S^T A
// operand), and transposing 8-byte reads of 4 rows x 32 bytes per 16 lanes
// (the O^T A operand).
template <int D>
constexpr int kPitchRow = D + 16;

__device__ __forceinline__ bf16x8 lds16(const uint16_t *p) {
  return as_bf16x8(*reinterpret_cast<const u32x4 *>(p));
}

// gfx950 transposing LDS read: within each group of 16 lanes, lane 4a+b gets
// element b of the 8-byte chunks addressed by lanes a, a+4, a+8 and a+12.
__device__ __forceinline__ u32x2 lds_read_tr16(const uint16_t *p) {
  typedef short v4i16 __attribute__((ext_vector_type(4)));
  const v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) v4i16 *)(p));
  return __builtin_bit_cast(u32x2, v);
}

// Rows of one 64-row dropped tile between their global load and their LDS
// store: thread t owns 16-byte chunk t % kCpr of rows t / kCpr + kRpp * it,
// so every 16 lanes move whole rows (coalesced in HBM, conflict-free in LDS).
template <int D>
struct DropRegs {
  static constexpr int kCpr = D / 8;             // 16-byte chunks per row
  static constexpr int kRpp = 256 / kCpr;        // rows per pass of the block
  static constexpr int kIt = kDropTile / kRpp;   // rows per thread
  u32x4 v[kIt];
  __device__ __forceinline__ void load(const uint16_t *V, const int (&row)[kIt], int chunk) {
#pragma unroll
    for (int it = 0; it < kIt; ++it) v[it] = ld16(V + (int64_t)row[it] * D + chunk * 8);
  }
  __device__ __forceinline__ void store(uint16_t *vr, int row0, int chunk) const {
    constexpr int PR = kPitchRow<D>;
#pragma unroll
    for (int it = 0; it < kIt; ++it) *reinterpret_cast<u32x4 *>(vr + (row0 + kRpp * it) * PR + chunk * 8) = v[it];
  }
};

template <int D>
struct FuseState {
  static constexpr int KS = D / 32, MB = D / 16, NB = 2;
  bf16x8 bvk[NB][KS];  // kept values, B operand of S^T (elements 32 s + 8 lg ..)
  f32x4 O[NB][MB];     // O^T accumulators
  float mrow[NB];      // running max of the scaled logits (x log2(e)/tau)
  float lsum[NB];      // this lane's share of the running denominator
};

// One 64-row dropped tile: S^T, online softmax, O^T.  MASK: the tile has
// fewer than 64 valid rows (nd).
template <int D, bool VFP32, bool MASK>
__device__ __forceinline__ void fuse_tile(FuseState<D> &st, const uint16_t *vt, int nd, float tc, int lr,
                                          int lg) {
  constexpr int KS = D / 32, MB = D / 16, NB = 2, PR = kPitchRow<D>;

  // S^T = V_d V_k^T for 64 dropped x 32 kept rows; A operands one k-step ahead.
  f32x4 acc[NB][4];
  bf16x8 a[2][4];
  // k-step s, lane group lg: elements 32 s + 8 lg .. + 7 of the row.
#pragma unroll
  for (int db = 0; db < 4; ++db) a[0][db] = lds16(vt + (db * 16 + lr) * PR + 8 * lg);
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    if (s + 1 < KS) {
#pragma unroll
      for (int db = 0; db < 4; ++db)
        a[(s + 1) & 1][db] = lds16(vt + (db * 16 + lr) * PR + 32 * (s + 1) + 8 * lg);
    }
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        acc[nb][db] = mfma_bf16(a[s & 1][db], st.bvk[nb][s], s == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : acc[nb][db]);
    __builtin_amdgcn_sched_barrier(0);
  }

  // Transposed V_d operands of the first half of O^T, read while the
  // softmax runs on the vector unit.
  const int tr_row = 4 * lg + (lr >> 2), tr_col = 4 * (lr & 3);
  const uint16_t *tbase = vt + tr_row * PR + tr_col;
  constexpr int kPre = 4;
  bf16x8 at[2 * MB];
#pragma unroll
  for (int q = 0; q < kPre; ++q) {
    const uint16_t *b0 = tbase + (32 * (q / MB)) * PR + 16 * (q % MB);
    const u32x2 lo4 = lds_read_tr16(b0), hi4 = lds_read_tr16(b0 + 16 * PR);
    at[q] = as_bf16x8(u32x4{lo4.x, lo4.y, hi4.x, hi4.y});
  }
  __builtin_amdgcn_sched_barrier(0);

  // Online softmax over dropped rows.  The four lane groups of a kept row
  // share one running max, raised (wave-uniformly) only when some logit
  // exceeds it by more than 2^kSlack.
  float tm[NB];
  bool grow = false;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    if (MASK) {
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (db * 16 + 4 * lg + i >= nd) acc[nb][db][i] = kNegInf;
    }
    float m = acc[nb][0][0];
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) m = fmaxf(m, acc[nb][db][i]);
    tm[nb] = m * tc;
    grow |= tm[nb] > st.mrow[nb] + kSlack;
  }
  if (__builtin_amdgcn_ballot_w64(grow) != 0) {
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      float m = tm[nb];
      m = fmaxf(m, shfl_xor(m, 16));
      m = fmaxf(m, shfl_xor(m, 32));
      const float mc = fmaxf(st.mrow[nb], m);
      const float alpha = fast_exp2(st.mrow[nb] - mc);
      st.mrow[nb] = mc;
      st.lsum[nb] *= alpha;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) st.O[nb][mb] *= alpha;
    }
  }
  bf16x8 bph[NB][2], bpl[NB][2];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float pr[4][4];
#pragma unroll
    for (int db = 0; db < 4; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pr[db][i] = fast_exp2(fmaf(acc[nb][db][i], tc, -st.mrow[nb]));
        st.lsum[nb] += pr[db][i];
      }
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      const float *p0 = pr[2 * t2], *p1 = pr[2 * t2 + 1];
      const u32x4 hi = {pack_bf16(p0[0], p0[1]), pack_bf16(p0[2], p0[3]), pack_bf16(p1[0], p1[1]),
                        pack_bf16(p1[2], p1[3])};
      bph[nb][t2] = as_bf16x8(hi);
      if (VFP32) {
        const u32x4 lo = {pack_bf16(p0[0] - bf16_lo(hi.x), p0[1] - bf16_hi(hi.x)),
                          pack_bf16(p0[2] - bf16_lo(hi.y), p0[3] - bf16_hi(hi.y)),
                          pack_bf16(p1[0] - bf16_lo(hi.z), p1[1] - bf16_hi(hi.z)),
                          pack_bf16(p1[2] - bf16_lo(hi.w), p1[3] - bf16_hi(hi.w))};
        bpl[nb][t2] = as_bf16x8(lo);
      }
    }
  }
  __builtin_amdgcn_sched_barrier(0);

  // O^T += V_d^T P^T over two 32-row k-steps, operands kPre reads ahead.
#pragma unroll
  for (int q = 0; q < 2 * MB; ++q) {
    if (q + kPre < 2 * MB) {
      const int qn = q + kPre;
      const uint16_t *b0 = tbase + (32 * (qn / MB)) * PR + 16 * (qn % MB);
      const u32x2 lo4 = lds_read_tr16(b0), hi4 = lds_read_tr16(b0 + 16 * PR);
      at[qn] = as_bf16x8(u32x4{lo4.x, lo4.y, hi4.x, hi4.y});
    }
    const int t2 = q / MB, mb = q % MB;
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
      st.O[nb][mb] = mfma_bf16(at[q], bph[nb][t2], st.O[nb][mb]);
      if (VFP32) st.O[nb][mb] = mfma_bf16(at[q], bpl[nb][t2], st.O[nb][mb]);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Workgroup = (fusion unit, 128 kept rows); wave w owns kept rows
// w*32 + nb*16 + [0, 16) for nb = 0, 1, so every operand read from LDS feeds
// two matrix instructions.
template <int D>
using DropTiles = uint16_t[2][kDropTile * kPitchRow<D>];

// One fusion job: kept rows [128 tile, 128 tile + 128) of the unit of rank
// `rank` in the fusion unit list.
template <int D, bool VFP32>
__device__ __forceinline__ void fuse_job(const PrunePlan &p, int rank, int tile, DropTiles<D> &vr) {
  constexpr int KS = D / 32, MB = D / 16, NB = 2;
  const u32x4 *rec = reinterpret_cast<const u32x4 *>(p.funit + rank);
  const u32x4 r0 = ld16(rec), r1 = ld16(rec + 1), r2 = ld16(rec + 2), r3 = ld16(rec + 3);
  auto ptr = [](uint32_t lo, uint32_t hi) { return (uint64_t)lo | ((uint64_t)hi << 32); };
  const int k = (int)r3.x, r = (int)r3.y, n = (int)r3.z;
  const int j0 = tile * kFuseRows;  // < k: the host lists only non-empty jobs
  const uint16_t *Kin = reinterpret_cast<const uint16_t *>(ptr(r0.x, r0.y));
  const uint16_t *Vin = reinterpret_cast<const uint16_t *>(ptr(r0.z, r0.w));
  uint16_t *Kout = reinterpret_cast<uint16_t *>(ptr(r1.x, r1.y)) + (int64_t)j0 * D;
  void *vout = reinterpret_cast<void *>(ptr(r1.z, r1.w));
  const int32_t *kept = reinterpret_cast<const int32_t *>(ptr(r2.x, r2.y)) + j0;
  const int32_t *drop = reinterpret_cast<const int32_t *>(ptr(r2.z, r2.w));
  const int nrows = min(kFuseRows, k - j0);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;

  // Token indices come from the selection kernel; clamping keeps every
  // gathered row inside the unit even if they were corrupted.
  auto clampi = [&](int v) { return min(max(v, 0), n - 1); };
  auto kept_idx = [&](int row) { return ldg(kept + min(row, nrows - 1)); };

  // Every index this thread needs before the first tile, in one batch:
  // kept rows of its key-copy chunks and of its lanes' value operands, and
  // dropped rows of tiles 0..3.  Dropped indices are read raw and clamped
  // one tile later, so no wait on them lands right behind the row loads;
  // tiles past the end re-read the last tile (never consumed).
  constexpr int kCpr = D / 8;                          // 16-byte chunks per row
  constexpr int kChunks = kFuseRows * kCpr / 256;      // key-copy chunks per thread
  int kc_idx[kChunks];
#pragma unroll
  for (int i = 0; i < kChunks; ++i) kc_idx[i] = kept_idx((tid + 256 * i) / kCpr);
  int kv_idx[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) kv_idx[nb] = kept_idx(w * 32 + nb * 16 + lr);
  const int ntiles = (r + kDropTile - 1) / kDropTile;
  using Regs = DropRegs<D>;
  constexpr int kIt = Regs::kIt;
  const int row0 = tid / Regs::kCpr, chunk = tid % Regs::kCpr;
  auto raw_idx = [&](int dt, int (&o)[kIt]) {
    const int base = min(dt, ntiles - 1) * kDropTile + row0;
#pragma unroll
    for (int it = 0; it < kIt; ++it) o[it] = ldg(drop + min(base + Regs::kRpp * it, r - 1));
  };
  auto clamp_rows = [&](const int (&in)[kIt], int (&o)[kIt]) {
#pragma unroll
    for (int it = 0; it < kIt; ++it) o[it] = clampi(in[it]);
  };
  int di[4][kIt];
  if (ntiles > 0) {
#pragma unroll
    for (int t = 0; t < 4; ++t) raw_idx(t, di[t]);
  }

  // Row loads: key copies, kept values, dropped tiles 0 and 1.
  u32x4 kc[kChunks];
#pragma unroll
  for (int i = 0; i < kChunks; ++i) kc[i] = ld16(Kin + (int64_t)clampi(kc_idx[i]) * D + ((tid + 256 * i) % kCpr) * 8);
  FuseState<D> st;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
    for (int s = 0; s < KS; ++s) st.bvk[nb][s] = as_bf16x8(ld16(Vin + (int64_t)clampi(kv_idx[nb]) * D + 32 * s + 8 * lg));
  }
  Regs set0, set1;
  int pend[kIt];  // raw indices of the next tile to load
  if (ntiles > 0) {
    int rr[kIt];
    clamp_rows(di[0], rr);
    set0.load(Vin, rr, chunk);
    clamp_rows(di[1], rr);
    set1.load(Vin, rr, chunk);
  }

  // Key pruning: bit copies of the kept rows.
#pragma unroll
  for (int i = 0; i < kChunks; ++i) {
    const int c = tid + 256 * i;
    if (c / kCpr < nrows) st16(Kout + (int64_t)(c / kCpr) * D + (c % kCpr) * 8, kc[i]);
  }
  if (ntiles > 0) {
    set0.store(vr[0], row0, chunk);
    int rr[kIt];
    clamp_rows(di[2], rr);
    set0.load(Vin, rr, chunk);
#pragma unroll
    for (int it = 0; it < kIt; ++it) pend[it] = di[3][it];
  }
  bool kvalid[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    kvalid[nb] = w * 32 + nb * 16 + lr < nrows;
    if (!kvalid[nb]) {
#pragma unroll
      for (int s = 0; s < KS; ++s) st.bvk[nb][s] = as_bf16x8(u32x4{0, 0, 0, 0});
    }
  }
  __syncthreads();

#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) st.O[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    // Running maxima are pre-multiplied by log2(e)/tau; the finite floor makes
    // the first tile's rescale factor exp2(floor - max) = 0.
    st.mrow[nb] = -1e30f;
    st.lsum[nb] = 0.f;
  }
  const float tc = p.tc;

  // End of tile t (parity PAR): stage tile t+1 from its register set into
  // the other LDS buffer, refill that set with tile t+3, fetch indices of
  // tile t+4, and synchronise.
  auto advance = [&](auto par, int t) {
    constexpr int PAR = decltype(par)::value;
    Regs &nx = PAR ? set0 : set1;
    nx.store(vr[PAR ^ 1], row0, chunk);
    int nxt[kIt], rr[kIt];
    raw_idx(t + 4, nxt);
    clamp_rows(pend, rr);
    nx.load(Vin, rr, chunk);
#pragma unroll
    for (int it = 0; it < kIt; ++it) pend[it] = nxt[it];
    __syncthreads();
  };
  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;
  const int nfull = r / kDropTile;
  int t = 0;
  for (; t + 1 < nfull; t += 2) {
    fuse_tile<D, VFP32, false>(st, vr[0], kDropTile, tc, lr, lg);
    advance(P0{}, t);
    fuse_tile<D, VFP32, false>(st, vr[1], kDropTile, tc, lr, lg);
    advance(P1{}, t + 1);
  }
  if (t < nfull) {
    fuse_tile<D, VFP32, false>(st, vr[0], kDropTile, tc, lr, lg);
    advance(P0{}, t);
    ++t;
  }
  if (t < ntiles) {  // partial last tile
    const int nd = r - t * kDropTile;
    fuse_tile<D, VFP32, true>(st, vr[t & 1], nd, tc, lr, lg);
  }

  const float mu = p.mu, omu = 1.f - p.mu;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float ls = st.lsum[nb];
    ls += shfl_xor(ls, 16);
    ls += shfl_xor(ls, 32);
    if (!kvalid[nb]) continue;
    const float inv = (r > 0 && ls > 0.f) ? 1.f / ls : 0.f;
    const int64_t orow_j = j0 + w * 32 + nb * 16 + lr;
    // Kept values at this lane's output columns 16 mb + 4 lg + i (L2-hot).
    const uint16_t *vrow = Vin + (int64_t)clampi(kv_idx[nb]) * D + 4 * lg;
    u32x2 kvv[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) kvv[mb] = ld8(vrow + 16 * mb);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const uint32_t w0 = kvv[mb].x, w1 = kvv[mb].y;
      const float vk[4] = {bf16_lo(w0), bf16_hi(w0), bf16_lo(w1), bf16_hi(w1)};
      float o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = (r > 0) ? mu * vk[i] + omu * (st.O[nb][mb][i] * inv) : vk[i];
      const int64_t off = orow_j * D + mb * 16 + 4 * lg;
      if (VFP32)
        st16(reinterpret_cast<float *>(vout) + off,
             u32x4{__float_as_uint(o[0]), __float_as_uint(o[1]), __float_as_uint(o[2]), __float_as_uint(o[3])});
      else
        st8(reinterpret_cast<uint16_t *>(vout) + off, u32x2{pack_bf16(o[0], o[1]), pack_bf16(o[2], o[3])});
    }
  }
}

// Persistent workgroups: block b walks the job list the host packed for it
// (block b runs on XCD b % 8, which holds the L2 lines of its units).  Wave w
// owns kept rows w*32 + nb*16 + [0, 16) of a job for nb = 0, 1, so every
// operand read from LDS feeds two matrix instructions.
template <int D, bool VFP32>
__global__ __launch_bounds__(256, 2) void k_fuse(PrunePlan p) {
  __shared__ __attribute__((aligned(16))) DropTiles<D> vr;
  const int j0 = ldg(p.fwoff + blockIdx.x), j1 = ldg(p.fwoff + blockIdx.x + 1);
  for (int j = j0; j < j1; ++j) {
    const int code = ldg(p.fwjob + j);
    fuse_job<D, VFP32>(p, code >> 8, code & 255, vr);
    __syncthreads();  // the next job restages the LDS tiles
  }
}

template <int D>
hipError_t launch_fuse_d(const PrunePlan &p, hipStream_t st, uint32_t grid) {
  if (p.v_fp32)
    hipLaunchKernelGGL((k_fuse<D, true>), dim3(grid), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL((k_fuse<D, false>), dim3(grid), dim3(256), 0, st, p);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_fuse(const PrunePlan &p, hipStream_t st) {
  if (p.nfunits == 0 || p.nfwg <= 0) return hipSuccess;
  const uint32_t grid = (uint32_t)p.nfwg;
  return p.d == 128 ? launch_fuse_d<128>(p, st, grid) : launch_fuse_d<64>(p, st, grid);
}

}  // namespace vc
