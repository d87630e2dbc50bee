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
// ends holding kept row l%16, columns 16*mb + 4*(l/16) + i; the mu-blend
// takes V_k at those columns from its operand registers through LDS.  With
// fp32 output the probabilities enter the second product as a bf16 hi + lo
// pair.
//
// Pipeline per workgroup: dropped-row indices are fetched four tiles ahead,
// the rows themselves three tiles ahead into two register sets, and staged
// into one of two LDS buffers one tile ahead.  A tile is processed as two
// halves of 32 dropped rows, which are the two k-steps of the second product:
// the scores of the second half are issued before the softmax of the first,
// and the first half's products with V_d^T before the softmax of the second,
// so matrix and vector work can overlap.  The running row maximum is lazy: a
// half's probabilities are taken against the maximum as it stands, and only
// when their sum on some lane passes 2^64 (always on a job's first half) is
// the maximum raised, the accumulators rescaled and the half redone.
#include <type_traits>

#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

constexpr float kNegInf = -__builtin_inff();
// A half tile's probabilities against a stale maximum may sum to this much
// before the maximum is raised: fp32 keeps the accumulators finite (at most
// 2^15 dropped rows of values below 2^16 in magnitude).
constexpr float kGrowLimit = 0x1p64f;

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

__device__ __forceinline__ uint32_t uni(uint32_t x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ uint64_t uni64(uint32_t lo, uint32_t hi) {
  return (uint64_t)uni(lo) | ((uint64_t)uni(hi) << 32);
}
// Address `off` bytes past a wave-uniform base (32-bit offset arithmetic).
template <typename T>
__device__ __forceinline__ T *boff(uint64_t base, uint32_t off) {
  return reinterpret_cast<T *>(base + off);
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
  __device__ __forceinline__ void load(uint64_t V, const int (&row)[kIt], int chunk) {
#pragma unroll
    for (int it = 0; it < kIt; ++it) v[it] = ld16(boff<const uint16_t>(V, (uint32_t)row[it] * (D * 2) + 16u * chunk));
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

// S^T of one half tile (dropped rows 32 h .. 32 h + 31) for both kept
// blocks; each operand read from LDS feeds two matrix instructions.
template <int D>
__device__ __forceinline__ void scores_half(const FuseState<D> &st, const uint16_t *vt, int h, int lr, int lg,
                                            f32x4 (&acc)[2][2]) {
  constexpr int KS = D / 32, PR = kPitchRow<D>;
#pragma unroll
  for (int s = 0; s < KS; ++s) {
    bf16x8 a[2];
#pragma unroll
    for (int d2 = 0; d2 < 2; ++d2) a[d2] = lds16(vt + (32 * h + 16 * d2 + lr) * PR + 32 * s + 8 * lg);
#pragma unroll
    for (int d2 = 0; d2 < 2; ++d2)
#pragma unroll
      for (int nb = 0; nb < 2; ++nb)
        acc[nb][d2] = mfma_bf16(a[d2], st.bvk[nb][s], s == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : acc[nb][d2]);
  }
}

// Online softmax of one half tile: probabilities against the running max
// (raised lazily), the denominators, and the bf16 B operands of O^T (with
// VFP32, also the low parts).  MASK: rows at or past nd are not dropped rows.
template <int D, bool VFP32, bool MASK>
__device__ __forceinline__ void softmax_half(FuseState<D> &st, f32x4 (&acc)[2][2], int h, int nd, float tc, int lg,
                                             bf16x8 (&ph)[2], bf16x8 (&pl)[2]) {
  constexpr int MB = D / 16;
  if (MASK) {
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
      for (int d2 = 0; d2 < 2; ++d2)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (32 * h + 16 * d2 + 4 * lg + i >= nd) acc[nb][d2][i] = kNegInf;
  }
  float pr[2][2][4], part[2];
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    part[nb] = 0.f;
#pragma unroll
    for (int d2 = 0; d2 < 2; ++d2)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pr[nb][d2][i] = fast_exp2(fmaf(acc[nb][d2][i], tc, -st.mrow[nb]));
        part[nb] += pr[nb][d2][i];
      }
  }
  const bool grow = !(part[0] <= kGrowLimit && part[1] <= kGrowLimit);
  if (__builtin_amdgcn_ballot_w64(grow) != 0) {
    // Raise each kept row's max to cover this half (the four lane groups of
    // a row agree on it), rescale what is accumulated, redo the half.
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      float m = kNegInf;
#pragma unroll
      for (int d2 = 0; d2 < 2; ++d2)
#pragma unroll
        for (int i = 0; i < 4; ++i) m = fmaxf(m, acc[nb][d2][i]);
      m *= tc;
      m = fmaxf(m, shfl_xor(m, 16));
      m = fmaxf(m, shfl_xor(m, 32));
      const float mc = fmaxf(st.mrow[nb], m);
      const float alpha = fast_exp2(st.mrow[nb] - mc);
      st.mrow[nb] = mc;
      st.lsum[nb] *= alpha;
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) st.O[nb][mb] *= alpha;
      part[nb] = 0.f;
#pragma unroll
      for (int d2 = 0; d2 < 2; ++d2)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          pr[nb][d2][i] = fast_exp2(fmaf(acc[nb][d2][i], tc, -mc));
          part[nb] += pr[nb][d2][i];
        }
    }
  }
#pragma unroll
  for (int nb = 0; nb < 2; ++nb) {
    st.lsum[nb] += part[nb];
    const float *p0 = pr[nb][0], *p1 = pr[nb][1];
    const u32x4 hi = {pack_bf16(p0[0], p0[1]), pack_bf16(p0[2], p0[3]), pack_bf16(p1[0], p1[1]),
                      pack_bf16(p1[2], p1[3])};
    ph[nb] = as_bf16x8(hi);
    if (VFP32) {
      const u32x4 lo = {pack_bf16(p0[0] - bf16_lo(hi.x), p0[1] - bf16_hi(hi.x)),
                        pack_bf16(p0[2] - bf16_lo(hi.y), p0[3] - bf16_hi(hi.y)),
                        pack_bf16(p1[0] - bf16_lo(hi.z), p1[1] - bf16_hi(hi.z)),
                        pack_bf16(p1[2] - bf16_lo(hi.w), p1[3] - bf16_hi(hi.w))};
      pl[nb] = as_bf16x8(lo);
    }
  }
}

// O^T += V_d^T P^T for the k-step of one half tile: lane lr of lane group lg
// reads dropped rows 32 h + 4 lg + (lr >> 2) and (+16), value columns
// 16 mb + 4 (lr & 3) .. + 3, through the transposing read.
template <int D, bool VFP32>
__device__ __forceinline__ void values_half(FuseState<D> &st, const uint16_t *vt, int h, int lr, int lg,
                                            const bf16x8 (&ph)[2], const bf16x8 (&pl)[2]) {
  constexpr int MB = D / 16, PR = kPitchRow<D>;
  const uint16_t *tb = vt + (32 * h + 4 * lg + (lr >> 2)) * PR + 4 * (lr & 3);
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const u32x2 lo4 = lds_read_tr16(tb + 16 * mb), hi4 = lds_read_tr16(tb + 16 * PR + 16 * mb);
    const bf16x8 at = as_bf16x8(u32x4{lo4.x, lo4.y, hi4.x, hi4.y});
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) {
      st.O[nb][mb] = mfma_bf16(at, ph[nb], st.O[nb][mb]);
      if (VFP32) st.O[nb][mb] = mfma_bf16(at, pl[nb], st.O[nb][mb]);
    }
  }
}

// One 64-row dropped tile (nd valid rows).
template <int D, bool VFP32, bool MASK>
__device__ __forceinline__ void fuse_tile(FuseState<D> &st, const uint16_t *vt, int nd, float tc, int lr, int lg) {
  f32x4 accA[2][2], accB[2][2];
  bf16x8 phA[2], plA[2], phB[2], plB[2];
  scores_half<D>(st, vt, 0, lr, lg, accA);
  scores_half<D>(st, vt, 1, lr, lg, accB);
  softmax_half<D, VFP32, MASK>(st, accA, 0, nd, tc, lg, phA, plA);
  values_half<D, VFP32>(st, vt, 0, lr, lg, phA, plA);
  softmax_half<D, VFP32, MASK>(st, accB, 1, nd, tc, lg, phB, plB);
  values_half<D, VFP32>(st, vt, 1, lr, lg, phB, plB);
}

// Workgroup = (fusion unit, 128 kept rows); wave w owns kept rows
// w*32 + nb*16 + [0, 16) for nb = 0, 1, so every operand read from LDS feeds
// two matrix instructions.
template <int D>
using DropTiles = uint16_t[2][kDropTile * kPitchRow<D>];

// One fusion job: kept rows [128 tile, 128 tile + 128) of the unit whose
// record is `rec`.  `next()` is called once the job's tiles are done (it
// starts fetching the next job's record while this one blends and stores).
template <int D, bool VFP32, typename Next>
__device__ __forceinline__ void fuse_job(const PrunePlan &p, const u32x4 (&rec)[4], int tile, DropTiles<D> &vr,
                                         Next &&next) {
  constexpr int KS = D / 32, MB = D / 16, NB = 2;
  constexpr uint32_t kRowBytes = D * 2;
  const uint64_t Kin = uni64(rec[0].x, rec[0].y), Vin = uni64(rec[0].z, rec[0].w);
  const uint64_t Kout = uni64(rec[1].x, rec[1].y), Vout = uni64(rec[1].z, rec[1].w);
  const uint64_t kept = uni64(rec[2].x, rec[2].y), drop = uni64(rec[2].z, rec[2].w);
  const int k = (int)uni(rec[3].x), r = (int)uni(rec[3].y), n = (int)uni(rec[3].z);
  const int j0 = tile * kFuseRows;  // < k: the host lists only non-empty jobs
  const int nrows = min(kFuseRows, k - j0);
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;

  // Token indices come from the selection kernel; clamping keeps every
  // gathered row inside the unit even if they were corrupted.
  auto clampi = [&](int v) { return min(max(v, 0), n - 1); };
  auto kept_idx = [&](int row) { return ldg(boff<const int32_t>(kept, 4u * (uint32_t)(j0 + min(row, nrows - 1)))); };

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
    for (int it = 0; it < kIt; ++it)
      o[it] = ldg(boff<const int32_t>(drop, 4u * (uint32_t)min(base + Regs::kRpp * it, r - 1)));
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
  for (int i = 0; i < kChunks; ++i)
    kc[i] = ld16(boff<const uint16_t>(Kin, (uint32_t)clampi(kc_idx[i]) * kRowBytes + 16u * ((tid + 256 * i) % kCpr)));
  FuseState<D> st;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
    for (int s = 0; s < KS; ++s)
      st.bvk[nb][s] = as_bf16x8(
          ld16(boff<const uint16_t>(Vin, (uint32_t)clampi(kv_idx[nb]) * kRowBytes + 2u * (32 * s + 8 * lg))));
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
    if (c / kCpr < nrows)
      st16(boff<uint16_t>(Kout, (uint32_t)(j0 + c / kCpr) * kRowBytes + 16u * (c % kCpr)), kc[i]);
  }
  // The previous job's waves may still read their kept values from the
  // tile buffers (below): nothing is staged before every wave is past them.
  __syncthreads();
  if (ntiles > 0) {
    set0.store(vr[0], row0, chunk);
    int rr[kIt];
    clamp_rows(di[2], rr);
    set0.load(Vin, rr, chunk);
#pragma unroll
    for (int it = 0; it < kIt; ++it) pend[it] = di[3][it];
  }
  // Rows past the job's end get zero operands.  The select reads every
  // kept-value register here, after the wait for tile 0 (loaded after them),
  // so no wait on these loads is left for the tile loop, where it would
  // stall on the newest prefetches instead.
  bool kvalid[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    kvalid[nb] = w * 32 + nb * 16 + lr < nrows;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const u32x4 v = as_u32x4(st.bvk[nb][s]);
      st.bvk[nb][s] = as_bf16x8(kvalid[nb] ? v : u32x4{0, 0, 0, 0});
    }
  }
  __syncthreads();

#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) st.O[nb][mb] = f32x4{0.f, 0.f, 0.f, 0.f};
    // Running maxima are pre-multiplied by log2(e)/tau; the finite floor makes
    // the first half tile raise them (its probabilities overflow the limit).
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
  next();

  // Every wave is past its last tile (the take synchronises), so the tile
  // buffers are free: each wave moves its kept values from the operand
  // layout (row l % 16, columns 32 s + 8 lg ..) to the output layout
  // (columns 16 mb + 4 lg ..) through its own 32 rows of a 128-row table,
  // instead of reading them from memory again.  At a pitch of D + 8
  // elements the 16-byte writes and the 8-byte reads are conflict-free.
  constexpr int PR = D + 8;
  static_assert(128 * PR <= 2 * kDropTile * kPitchRow<D>, "the kept-value table fits the tile buffers");
  uint16_t *kvt = &vr[0][0];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int s = 0; s < KS; ++s)
      *reinterpret_cast<u32x4 *>(kvt + (w * 32 + nb * 16 + lr) * PR + 32 * s + 8 * lg) = as_u32x4(st.bvk[nb][s]);
  u32x2 kvv[NB][MB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
      kvv[nb][mb] = *reinterpret_cast<const u32x2 *>(kvt + (w * 32 + nb * 16 + lr) * PR + 16 * mb + 4 * lg);

  const float mu = p.mu, omu = 1.f - p.mu;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    float ls = st.lsum[nb];
    ls += shfl_xor(ls, 16);
    ls += shfl_xor(ls, 32);
    if (!kvalid[nb]) continue;
    const float inv = (r > 0 && ls > 0.f) ? 1.f / ls : 0.f;
    const uint32_t orow_j = (uint32_t)(j0 + w * 32 + nb * 16 + lr);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) {
      const uint32_t w0 = kvv[nb][mb].x, w1 = kvv[nb][mb].y;
      const float vk[4] = {bf16_lo(w0), bf16_hi(w0), bf16_lo(w1), bf16_hi(w1)};
      float o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = (r > 0) ? mu * vk[i] + omu * (st.O[nb][mb][i] * inv) : vk[i];
      const uint32_t col = (uint32_t)(mb * 16 + 4 * lg);
      if (VFP32)
        st16(boff<float>(Vout, (orow_j * D + col) * 4u),
             u32x4{__float_as_uint(o[0]), __float_as_uint(o[1]), __float_as_uint(o[2]), __float_as_uint(o[3])});
      else
        st8(boff<uint16_t>(Vout, (orow_j * D + col) * 2u), u32x2{pack_bf16(o[0], o[1]), pack_bf16(o[2], o[3])});
    }
  }
}

// Persistent workgroups, the same number on every XCD: block b runs on XCD
// x = b % 8 and works through that XCD's queue (its units' dropped rows stay
// in that L2).  It starts on job b / 8 of the queue and then takes the next
// untaken job each time it finishes one (one device-scope atomic per job,
// issued while the finished job blends and stores), so the XCD's workgroups
// stay busy until its queue is empty.  Every index is handed out once.
template <int D, bool VFP32>
__global__ __launch_bounds__(256, 2) void k_fuse(PrunePlan p) {
  __shared__ __attribute__((aligned(16))) DropTiles<D> vr;
  __shared__ int s_code;
  const int x = (int)(blockIdx.x % kXcds);
  const int q0 = ldg(p.fwoff + x), qlen = ldg(p.fwoff + x + 1) - q0;
  auto take = [&]() -> int {
    __syncthreads();  // every thread has read the previous code
    if (threadIdx.x == 0) {
      const int i = __hip_atomic_fetch_add(p.fcnt + x, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      s_code = i < qlen ? ldg(p.fwjob + q0 + i) : -1;
    }
    __syncthreads();
    return s_code;
  };
  auto fetch = [&](int code, u32x4 (&rec)[4]) {
    const u32x4 *rp = reinterpret_cast<const u32x4 *>(p.funit + (code >> 8));
#pragma unroll
    for (int i = 0; i < 4; ++i) rec[i] = ld16(rp + i);
  };
  const int first = (int)(blockIdx.x / kXcds);
  int code = first < qlen ? ldg(p.fwjob + q0 + first) : -1;
  u32x4 rec[4] = {};
  if (code >= 0) fetch(code, rec);
  while (code >= 0) {
    int ncode = -1;
    u32x4 nrec[4] = {};
    fuse_job<D, VFP32>(p, rec, code & 255, vr, [&]() {
      ncode = take();
      if (ncode >= 0) fetch(ncode, nrec);
    });
    code = ncode;
#pragma unroll
    for (int i = 0; i < 4; ++i) rec[i] = nrec[i];
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
