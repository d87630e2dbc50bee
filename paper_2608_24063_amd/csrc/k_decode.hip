// k_decode.hip -- decode over the (compressed) cache (Sec. 2, "VLLM
// Decoding"): append one K/V row per (layer, sequence, kv head) and attend one
// query per query head over all cached rows.
//
// Work is balanced over rows, not units: the 32-row tiles of every unit's
// capacity are split into pieces of nearly equal size, a number of pieces
// proportional to the capacity, one workgroup per piece, so a pruned cache,
// whose units differ widely in length, still spreads evenly over the chip.
// The cut comes either from a piece table the host builds once per cache
// (capacities do not change between steps) or, in the calls without one,
// from every workgroup deriving it from the capacities (wave sums over the
// units).  Inside a piece each of the four waves takes a contiguous run of
// 32-row tiles, the next tile's rows in flight while the current one is
// processed.  The G query heads of a kv head form one 16-column MFMA block
// (heads >= G are zero), so each K/V row is read once for all of them.  A
// unit in one piece is normalised and written directly; the pieces of a split
// unit leave partial (max, sum, O) results that are merged in row order.
#include <mutex>

#include "vc_device.h"
#include "vc_internal.h"

namespace vc {

namespace {

constexpr float kNegInf = -__builtin_inff();
constexpr float kFloor = -1e30f;
constexpr int kRowTile = kDecodeTileRows;

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
// 16-byte chunk lane % (d/8) of rows lane / (d/8) + (64 / (d/8)) it (staged to
// LDS row-major).
template <int D>
struct RowTile {
  static constexpr int KS = D / 32;
  static constexpr int kCpr = D / 8;             // 16-byte chunks per row
  static constexpr int kVIt = 32 * D / 8 / 64;   // 16-byte V chunks per lane
  u32x4 k[2][KS];
  u32x4 v[kVIt];
  // bf16 rows t0 .. t0 + 31 of the unit's pool block, each row index clamped
  // to lim - 1 (a row that exists in the block; clamped rows are masked).
  __device__ __forceinline__ void load(const uint16_t *Kp, const uint16_t *Vp, int t0, int lim, int lr, int lg,
                                       int lane) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const uint16_t *src = Kp + (int64_t)min(t0 + rb * 16 + lr, lim - 1) * D;
#pragma unroll
      for (int s = 0; s < KS; ++s) k[rb][s] = ld16(src + 32 * s + 8 * lg);
    }
#pragma unroll
    for (int it = 0; it < kVIt; ++it) {
      const int c = lane + 64 * it;
      v[it] = ld16(Vp + (int64_t)min(t0 + c / kCpr, lim - 1) * D + (c % kCpr) * 8);
    }
  }
  // Rows of a bf16 tile whose pool contents are not this step's: row `nrow`
  // (the row appended by this launch, not yet in the pool when the tile was
  // read) takes K and V from the staged copy nk / nv in LDS, and rows at or
  // past `e` (the wave's last row) get zero values, so that whatever the pool
  // held there (possibly not finite) meets only zero probabilities.  Their
  // scores are masked separately.
  __device__ __forceinline__ void patch(int t0, int e, int nrow, const uint16_t *nk, const uint16_t *nv, int lr,
                                        int lg, int lane) {
    const bool h0 = t0 + lr == nrow, h1 = t0 + 16 + lr == nrow;
    if (h0 || h1) {
#pragma unroll
      for (int s = 0; s < KS; ++s) {
        const u32x4 x = *reinterpret_cast<const u32x4 *>(nk + 32 * s + 8 * lg);
        if (h0) k[0][s] = x;
        if (h1) k[1][s] = x;
      }
    }
    const u32x4 xv = *reinterpret_cast<const u32x4 *>(nv + (lane % kCpr) * 8);
    const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int it = 0; it < kVIt; ++it) {
      const int row = t0 + (lane + 64 * it) / kCpr;
      v[it] = row == nrow ? xv : (row >= e ? zero : v[it]);
    }
  }
  // 4-bit rows t0.. of the unit's quantised block Kc/Km, Vc/Vm, row indices
  // clamped to lim - 1.  K: lane (lr, lg) takes the codes of channels
  // 32 lg .. 32 lg + 31 (d = 128; 16 lg .. 16 lg + 15 for d = 64) of its row,
  // all in one group, into k[rb][0] and the group's (scale, lo) into k[rb][1];
  // the products then pair them with the query in the same channel order.
  // V: lane takes whole groups (row, group) = lane + 64 it, codes in v[2 it],
  // (scale, lo) in v[2 it + 1].
  static constexpr int kG = D / 32;         // groups per row
  static constexpr int kVG = 32 * kG / 64;  // V groups per lane
  __device__ __forceinline__ void load_q(const uint8_t *Kc, const float2 *Km, const uint8_t *Vc, const float2 *Vm,
                                         int t0, int lim, int lr, int lg, int lane) {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const int64_t row = min(t0 + rb * 16 + lr, lim - 1);
      const float2 m = ldg(Km + row * kG + lg * kG / 4);
      if (D == 128) {
        k[rb][0] = ld16(Kc + row * (D / 2) + 16 * lg);
      } else {
        const u32x2 c = ld8(Kc + row * (D / 2) + 8 * lg);
        k[rb][0] = u32x4{c.x, c.y, 0u, 0u};
      }
      k[rb][1] = u32x4{__float_as_uint(m.x), __float_as_uint(m.y), 0u, 0u};
    }
#pragma unroll
    for (int it = 0; it < kVG; ++it) {
      const int gi = lane + 64 * it;
      const int64_t row = min(t0 + gi / kG, lim - 1);
      const int grp = gi % kG;
      const float2 m = ldg(Vm + row * kG + grp);
      v[2 * it] = ld16(Vc + row * (D / 2) + 16 * grp);
      v[2 * it + 1] = u32x4{__float_as_uint(m.x), __float_as_uint(m.y), 0u, 0u};
    }
    // Every member defined on both load paths (a tile of either kind then
    // stays in registers instead of a stack copy).
    const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int s = 2; s < KS; ++s) k[rb][s] = zero;
#pragma unroll
    for (int it = 2 * kVG; it < kVIt; ++it) v[it] = zero;
  }
  // bf16(fma(code, scale, lo)) of the 8 codes of one word, in channel order.
  static __device__ __forceinline__ u32x4 deq8(uint32_t w, float sc, float lo) {
    const uint32_t e = w & 0x0F0F0F0Fu, o = (w >> 4) & 0x0F0F0F0Fu;  // even / odd channels, one per byte
    float f[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      f[2 * j] = fmaf((float)((e >> (8 * j)) & 0xFFu), sc, lo);
      f[2 * j + 1] = fmaf((float)((o >> (8 * j)) & 0xFFu), sc, lo);
    }
    return u32x4{pack_bf16(f[0], f[1]), pack_bf16(f[2], f[3]), pack_bf16(f[4], f[5]), pack_bf16(f[6], f[7])};
  }
  // K of a 4-bit tile into bf16 operands: k[rb][s] = chunk lg * KS + s.
  __device__ __forceinline__ void unpack_k() {
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
      const u32x4 c = k[rb][0];
      const float sc = __uint_as_float(k[rb][1].x), lo = __uint_as_float(k[rb][1].y);
      const uint32_t w[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
      for (int s = 0; s < KS; ++s) k[rb][s] = deq8(w[s], sc, lo);
    }
  }
};

// Partials exchanged inside one launch may cross XCDs (separate L2s): they
// are written and read with device-coherent accesses instead of fences that
// would write back and invalidate a whole L2.
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
  static constexpr int kVtBytes = kRowTile * PR * 2;
  static constexpr int kWoBytes = 16 * (D + 4) * 4;
  static constexpr int kWaveBytes = kVtBytes > kWoBytes ? kVtBytes : kWoBytes;
  // Per wave: its V tile while it walks the rows, then its partial O (written
  // after the wave's last tile, so the two uses never overlap in time).
  uint8_t wave[4][kWaveBytes] __attribute__((aligned(16)));
  // The query heads, row-major, for the 4-bit tiles' operands (their channel
  // order differs from the bf16 tiles'; read from here instead of holding a
  // second copy in registers).  Rows padded by 16 bytes.
  static constexpr int QP = D + 8;
  uint16_t qh[16][QP] __attribute__((aligned(16)));
  // The K and V row the launch appends to this unit (the fused step), one
  // copy per wave (K then V), so that no barrier waits for it.
  uint16_t newrow[4][2 * D] __attribute__((aligned(16)));
  float2 wml[4][16];
  float2 mlb[128];  // (max, sum) pairs of a batch of partials being merged
  uint32_t flag[1];
};

__device__ __forceinline__ uint16_t *wave_vt(uint8_t *w) { return reinterpret_cast<uint16_t *>(w); }

// Rows of a unit attended by this launch and the index of the row appended
// by it (-1 if none).  The fused step appends where there is room.
template <bool STEP>
__device__ __forceinline__ void unit_rows(int len0, int cap, int max_rows, int &rows, int &nrow) {
  len0 = max(len0, 0);
  const bool room = STEP && len0 < cap;
  rows = room ? len0 + 1 : min(len0, cap);
  nrow = room ? len0 : -1;
  rows = max(min(rows, max_rows), 0);
}
__device__ __forceinline__ uint32_t unit_tiles(int rows) {
  return rows > 0 ? (uint32_t)(rows + kRowTile - 1) / kRowTile : 1u;
}

// Sum over the 64 lanes of a wave, in every lane.
__device__ __forceinline__ uint32_t wave_sum(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_scan(x), 63);
}

// ceil(a / b) by a reciprocal, 1 <= b, a + b < 2^32: the rounded product is
// off by at most one, which the integer check corrects.  With `small`
// (a + b < 2^20) single precision is close enough; else double.
struct Recip {
  uint32_t b;
  float f;
  double d;
};
__device__ __forceinline__ Recip recip(uint32_t b, bool small) {
  Recip r;
  r.b = b;
  r.f = small ? __builtin_amdgcn_rcpf((float)b) : 0.f;
  r.d = small ? 0.0 : 1.0 / (double)b;
  return r;
}
__device__ __forceinline__ uint32_t ceil_div(uint32_t a, const Recip &r, bool small) {
  const uint32_t x = a + r.b - 1;
  uint32_t q = small ? (uint32_t)((float)x * r.f) : (uint32_t)((double)x * r.d);
  if ((uint64_t)q * r.b > x) --q;
  else if ((uint64_t)(q + 1) * r.b <= x) ++q;
  return q;
}

// floor(a / b) for a < 2^52, 1 <= b < 2^31 (the reciprocal's error
// corrected as above; single precision where a < 2^20).
__device__ __forceinline__ uint64_t floor_div64(uint64_t a, uint32_t b) {
  const bool small = a < (1u << 20);
  uint64_t q = small ? (uint64_t)(uint32_t)((float)(uint32_t)a * __builtin_amdgcn_rcpf((float)b))
                     : (uint64_t)((double)a * (1.0 / (double)b));
  if (q * b > a) --q;
  else if ((q + 1) * b <= a) ++q;
  return q;
}

// The cut.  The tiles of every unit's capacity (cap rows, at most max_rows)
// are split into np_u = ceil(tiles_u / c) pieces of nearly equal tile
// counts, one workgroup each, pieces numbered in unit order.  Capacities do
// not change during a call, so every workgroup derives the same cut, and a
// unit's length is read only by its own pieces, the last of which advances it
// (no grid-wide ordering is needed).  The piece bound c is the smallest of
// four multiples of 4 tiles (from T / grid up, at least kMinPiece: below
// that, splitting a unit saves less than the merge of its pieces costs) whose
// piece count fits the grid, so the four waves of a workgroup get equal
// numbers of tiles; if none
// fits, c = T / (grid - U) (rounded up to a multiple of 4) always does, since
// the pieces then number at most T / c + U.  Each wave computes the whole cut
// by itself (lane l takes units 64 k + l of each 256-unit chunk), so no
// barrier is needed; the result, this workgroup's piece, is the same in every
// wave.
constexpr uint32_t kMinPiece = kDecodeMinPiece;

struct Piece {
  int32_t u, j, np, p0, nt, len0, cap;  // u = -1: no piece
  int64_t roff;                         // the unit's first pool row
};

template <bool STEP>
__device__ __forceinline__ Piece cut(const DecodePlan &p, uint32_t i) {
  constexpr int kChunk = 256;  // units per pass: 64 lanes x 4
  const int lane = threadIdx.x & 63;
  const int nch = (p.units + kChunk - 1) / kChunk;
  uint32_t tl[4];
  int2 lc[4];
  int64_t ro[4];
  // 64-unit groups of chunk c that hold units (uniform).
  auto groups = [&](int c) { return min(4, (p.units - c * kChunk + 63) / 64); };
  // All loads are issued before any is used (indices clamped rather than
  // branched on), so they cost one round trip; the row offsets come along so
  // that the piece's own is at hand without another.
  auto load = [&](int c) {
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int uc = min(c * kChunk + k * 64 + lane, p.units - 1);
      lc[k] = make_int2(ldg(p.len + uc), ldg(p.cap + uc));
      ro[k] = ldg(p.row_off + uc);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const bool in = c * kChunk + k * 64 + lane < p.units;
      tl[k] = in ? unit_tiles(max(min(lc[k].y, p.max_rows), 0)) : 0u;
    }
  };
  if (nch == 1) load(0);  // one chunk: its values stay in registers
  uint32_t T = 0;
  for (int c = 0; c < nch; ++c) {
    if (nch > 1) load(c);
    T += wave_sum(tl[0] + tl[1] + tl[2] + tl[3]);
  }
  const uint32_t N = gridDim.x;  // > U (host)
  const uint32_t c0 = max(kMinPiece, (T / N + (T % N != 0) + 3u) & ~3u);
  const bool small = T + c0 + 16u < (1u << 20);
  Recip rc[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) rc[q] = recip(c0 + 4u * q, small);
  uint32_t P[4] = {0u, 0u, 0u, 0u};
  for (int c = 0; c < nch; ++c) {
    if (nch > 1) load(c);
    const int K = groups(c);
    uint32_t v[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (k < K) {  // uniform (a guard, not a break: the loop unrolls, the arrays stay in registers)
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] += tl[k] ? ceil_div(tl[k], rc[q], small) : 0u;
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) P[q] += wave_sum(v[q]);
  }
  const uint32_t free_ = N - (uint32_t)p.units;
  uint32_t cb = ((T / free_ + (T % free_ != 0)) + 3u) & ~3u;
#pragma unroll
  for (int q = 3; q >= 0; --q)
    if (P[q] <= N) cb = c0 + 4u * q;
  const bool small_b = T + cb < (1u << 20);
  const Recip rcb = recip(cb, small_b);
  // Pieces per unit in unit order: lane l's units 64k + l are interleaved,
  // so the prefix runs over k (outer) and lanes (inner) of each chunk.
  Piece pc{-1, 0, 0, 0, 0, 0, 0, 0};
  uint32_t base = 0;
  for (int c = 0; c < nch; ++c) {
    if (nch > 1) load(c);
    const int K = groups(c);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      if (k < K) {  // uniform
        const uint32_t n = tl[k] ? ceil_div(tl[k], rcb, small_b) : 0u;
        const uint32_t inc = wave_incl_scan(n);
        const uint32_t a = base + inc - n;
        const uint64_t hit = __builtin_amdgcn_ballot_w64(n > 0 && i >= a && i < a + n);
        if (hit) {
          const int src = __builtin_ctzll(hit);
          const int u = c * kChunk + k * 64 + src;
          pc.u = u;
          pc.np = __builtin_amdgcn_readlane((int)n, src);
          pc.p0 = __builtin_amdgcn_readlane((int)a, src);
          pc.j = (int)i - pc.p0;
          pc.nt = __builtin_amdgcn_readlane((int)tl[k], src);
          pc.len0 = __builtin_amdgcn_readlane(lc[k].x, src);
          pc.cap = __builtin_amdgcn_readlane(lc[k].y, src);
          const uint32_t rlo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)ro[k], src);
          const uint32_t rhi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(ro[k] >> 32), src);
          pc.roff = (int64_t)(((uint64_t)rhi << 32) | rlo);
        }
        base += (uint32_t)__builtin_amdgcn_readlane((int)inc, 63);
      }
    }
  }
  return pc;
}

// Where a piece's result goes: its partial (plain or device-coherent stores),
// or, for a unit attended by one workgroup, the normalised output itself.
enum PieceOut { kPartial = 0, kPartialCoherent = 1, kOutput = 2 };

// The query heads g*G + lr of unit u as MFMA B operands in natural channel
// order (8 consecutive channels per lane group); heads >= G are zero.  With
// 4-bit tiles (Q4), wave 0 also writes them row-major to LDS, from where
// those tiles read them in their own channel order (chunk lg * KS + s in
// block s); a barrier must follow before the first tile.
template <int D, bool Q4>
struct QueryOps {
  static constexpr int KS = D / 32;
  // With 4-bit tiles the bf16 tiles read the query from LDS too (nat), which
  // keeps the kernel within its registers.
  bf16x8 bq[Q4 ? 1 : KS];
  const uint16_t *row0;  // the group's first query row (a readable row of d values)
  // (Every lane loads, from a head clamped into the group, so no load sits
  // in a divergent branch, where the wait for it could not be counted
  // exactly and would drain every load in flight.)
  __device__ __forceinline__ void load(const DecodePlan &p, DecodeSmem<D> &sm, int u, int w, int lr, int lg) {
    const int g = u % p.Hkv;
    const int lb_ = u / p.Hkv;  // l * B + b
    row0 = p.q + ((int64_t)lb_ * p.Hq + (int64_t)g * p.G) * D;
    const uint16_t *q = row0 + (int64_t)min(lr, p.G - 1) * D;
    const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const u32x4 x = ld16(q + 32 * s + 8 * lg);
      const u32x4 v = lr < p.G ? x : zero;
      if (Q4) {
        if (w == 0) *reinterpret_cast<u32x4 *>(&sm.qh[lr][32 * s + 8 * lg]) = v;
      } else {
        bq[Q4 ? 0 : s] = as_bf16x8(v);
      }
    }
  }
  // Block s of the bf16 tiles' B operand (natural channel order).
  __device__ __forceinline__ bf16x8 nat(const DecodeSmem<D> &sm, int s, int lr, int lg) const {
    if (Q4) return as_bf16x8(*reinterpret_cast<const u32x4 *>(&sm.qh[lr][32 * s + 8 * lg]));
    return bq[Q4 ? 0 : s];
  }
  // Block s of the 4-bit tiles' B operand.
  static __device__ __forceinline__ bf16x8 perm(const DecodeSmem<D> &sm, int s, int lr, int lg) {
    return as_bf16x8(*reinterpret_cast<const u32x4 *>(&sm.qh[lr][8 * (lg * KS + s)]));
  }
};

// Where a unit's rows live: its bf16 pool block and, for 4-bit tiles (rows
// below nq, a multiple of the tile), its quantised block.
template <int D>
struct UnitRows {
  const uint16_t *Kp, *Vp;
  const uint8_t *Kc, *Vc;
  const float2 *Km, *Vm;
  int nq;
};

// One wave's share of a piece: rows [a, e) of the unit, a tile at a time
// from a (a multiple of the tile), with the next tile's rows in flight while
// the current one is processed.  `cur` and `nxt` hold the rows of the first
// two tiles, read by the caller with row indices clamped to spec - 1; a tile
// that has rows below e at or past spec is read again (with the rows known,
// so only when the early bound fell short).  The wave's running (max, sum,
// O) of the G heads come back in mrow, lsum and O.
//   S^T = K Q^T   A = K rows straight from HBM, B = Q (registers)
//   O^T = V^T P^T A = V^T (per-wave LDS tile, transposing reads), B = P^T
template <int D, bool Q4>
__device__ __forceinline__ void wave_rows(const DecodePlan &p, DecodeSmem<D> &sm, const QueryOps<D, Q4> &qo,
                                          const UnitRows<D> &ur, RowTile<D> &cur, RowTile<D> &nxt, int a, int e,
                                          int spec, int nrow, f32x4 (&O)[D / 16], float &mrow, float &lsum) {
  constexpr int KS = D / 32;
  constexpr int MB = D / 16;
  constexpr int PR = DecodeSmem<D>::PR;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int lr = lane & 15, lg = lane >> 4;
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) O[mb] = f32x4{0.f, 0.f, 0.f, 0.f};
  // Running max per head, pre-multiplied by the exp2 scale; starts at a finite
  // floor so rescaling never forms (-inf) - (-inf).
  mrow = kFloor;
  lsum = 0.f;
  const float sc = p.sc;
  uint16_t *myvt = wave_vt(sm.wave[w]);
  const int tr_row = 4 * lg + (lr >> 2), tr_col = 4 * (lr & 3);
  const int nq = Q4 ? ur.nq : 0;
  if (a < e && min(a + kRowTile, e) > spec) cur.load(ur.Kp, ur.Vp, a, e, lr, lg, lane);  // (bf16 only)
  for (int t0 = a; t0 < e; t0 += kRowTile) {
    const int tn = t0 + kRowTile;
    // The second tile is in nxt already, unless its early read fell short.
    if (tn < e && (t0 > a || min(tn + kRowTile, e) > spec)) {
      if (Q4 && tn < nq)
        nxt.load_q(ur.Kc, ur.Km, ur.Vc, ur.Vm, tn, e, lr, lg, lane);
      else
        nxt.load(ur.Kp, ur.Vp, tn, e, lr, lg, lane);
    }
    const bool qt = Q4 && t0 < nq;  // wave-uniform
    if (!qt && (tn > e || (nrow >= t0 && nrow < tn)))  // wave-uniform
      cur.patch(t0, e, nrow, sm.newrow[w], sm.newrow[w] + D, lr, lg, lane);
    // S^T = K Q^T for 2 blocks of 16 rows.
    f32x4 acc[2];
    if (qt) {
      cur.unpack_k();
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s)
          acc[rb] = mfma_bf16(as_bf16x8(cur.k[rb][s]), QueryOps<D, Q4>::perm(sm, s, lr, lg), acc[rb]);
      }
    } else {
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KS; ++s) acc[rb] = mfma_bf16(as_bf16x8(cur.k[rb][s]), qo.nat(sm, s, lr, lg), acc[rb]);
      }
    }
    // V rows -> per-wave LDS tile, row-major (read back transposed below);
    // 4-bit groups are read back on the way.
    if (qt) {
      constexpr int kG = RowTile<D>::kG;
#pragma unroll
      for (int it = 0; it < RowTile<D>::kVG; ++it) {
        const int gi = lane + 64 * it;
        const u32x4 c = cur.v[2 * it];
        const float vs = __uint_as_float(cur.v[2 * it + 1].x), vl = __uint_as_float(cur.v[2 * it + 1].y);
        uint16_t *dst = myvt + (gi / kG) * PR + (gi % kG) * 32;
        *reinterpret_cast<u32x4 *>(dst) = RowTile<D>::deq8(c.x, vs, vl);
        *reinterpret_cast<u32x4 *>(dst + 8) = RowTile<D>::deq8(c.y, vs, vl);
        *reinterpret_cast<u32x4 *>(dst + 16) = RowTile<D>::deq8(c.z, vs, vl);
        *reinterpret_cast<u32x4 *>(dst + 24) = RowTile<D>::deq8(c.w, vs, vl);
      }
    } else {
      constexpr int kCpr = RowTile<D>::kCpr;
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
        if (t0 + rb * 16 + 4 * lg + i >= e) acc[rb][i] = kNegInf;
        tm = fmaxf(tm, acc[rb][i]);
      }
    tm = max_halves(fmaxf(tm, swap16(tm)));
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
      const bf16x8 av = as_bf16x8(u32x4{lo4.x, lo4.y, hi4.x, hi4.y});
      O[mb] = mfma_bf16(av, as_bf16x8(hi), O[mb]);
      O[mb] = mfma_bf16(av, as_bf16x8(lo), O[mb]);
    }
    __builtin_amdgcn_s_waitcnt(0xc07f);  // reads done before the next tile's writes
    __builtin_amdgcn_wave_barrier();
    cur = nxt;
  }
}

// Merges the four waves' (max, sum, O) of a piece and stores the result:
// the partial of slot `slot`, or (OUT == kOutput, the unit's only piece) the
// normalised output.  Each wave's O goes into its own V tile area, which it
// no longer reads.
template <int D, int OUT>
__device__ __forceinline__ void finish_piece(const DecodePlan &p, DecodeSmem<D> &sm, int u, int slot,
                                             const f32x4 (&O)[D / 16], float mrow, float lsum) {
  constexpr int MB = D / 16;
  auto &wml = sm.wml;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  lsum = sum_halves(lsum + swap16(lsum));
  if (lg == 0) wml[w][lr] = make_float2(mrow <= kFloor ? kNegInf : mrow, lsum);
  {
    float(*wo)[D + 4] = reinterpret_cast<float(*)[D + 4]>(sm.wave[w]);
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i) wo[lr][mb * 16 + 4 * lg + i] = O[mb][i];
  }
  __syncthreads();
  // Thread t takes channel x = t mod d of heads h0 + (256 / d) k, h0 = t / d,
  // k < 16 d / 256; all its LDS reads are issued before any is used (one
  // wave per SIMD here, so their latency is not hidden otherwise).  Heads at
  // or past G are neither output nor merged: they are skipped.
  constexpr int kEl = 16 * D / 256;
  constexpr int kHs = 256 / D;
  const int x = tid % D, h0 = __builtin_amdgcn_readfirstlane(tid / D);  // h0 is the same across a wave
  float2 ml[kEl][4];
  float wv[kEl][4];
#pragma unroll
  for (int k = 0; k < kEl; ++k)
    if (h0 + kHs * k < p.G) {  // wave-uniform
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        ml[k][i] = wml[i][h0 + kHs * k];
        wv[k][i] = reinterpret_cast<const float(*)[D + 4]>(sm.wave[i])[h0 + kHs * k][x];
      }
    }
  const int g = u % p.Hkv;
  const int lb_ = u / p.Hkv;
  const int64_t pbase = (int64_t)slot * 16;
#pragma unroll
  for (int k = 0; k < kEl; ++k) {
    const int h = h0 + kHs * k;
    if (h >= p.G) continue;
    float M = kNegInf;
#pragma unroll
    for (int i = 0; i < 4; ++i) M = fmaxf(M, ml[k][i].x);
    float o = 0.f, s = 0.f;
    if (M != kNegInf) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if (ml[k][i].x != kNegInf) {
          const float f = fast_exp2(ml[k][i].x - M);
          o += f * wv[k][i];
          s += f * ml[k][i].y;
        }
      }
    }
    if (OUT == kOutput) {
      // The merge of a single piece: its factor is exp2(0) = 1 exactly.
      stg(p.out + ((int64_t)lb_ * p.Hq + (int64_t)g * p.G + h) * D + x, s > 0.f ? o / s : 0.f);
      continue;
    }
    st_part<OUT == kPartialCoherent>(p.part_o + (pbase + h) * D + x, o);
    if (x == 0) {
      float *mlp = reinterpret_cast<float *>(p.part_ml + pbase + h);
      st_part<OUT == kPartialCoherent>(mlp, M);
      st_part<OUT == kPartialCoherent>(mlp + 1, s);
    }
  }
  __syncthreads();  // LDS free for the next piece
}

// The first two tiles of a wave's rows [a, lim): bf16 rows, or 4-bit ones
// below nq (Q4).  Without 4-bit rows the loads are branch-free: a tile past
// lim reads row 0 of `dummy` (any readable row of d values) instead, and is
// never used.  (A load under a branch makes the compiler's wait for the
// loads issued before it, the appended row's, drain every load in flight.)
template <int D, bool Q4>
__device__ __forceinline__ void first_tiles(const UnitRows<D> &ur, const uint16_t *dummy, RowTile<D> &cur,
                                            RowTile<D> &nxt, int a, int lim, int lr, int lg, int lane) {
  if (!Q4) {
    const bool ok0 = a < lim, ok1 = a + kRowTile < lim;
    cur.load(ok0 ? ur.Kp : dummy, ok0 ? ur.Vp : dummy, ok0 ? a : 0, ok0 ? lim : 1, lr, lg, lane);
    nxt.load(ok1 ? ur.Kp : dummy, ok1 ? ur.Vp : dummy, ok1 ? a + kRowTile : 0, ok1 ? lim : 1, lr, lg, lane);
    return;
  }
  const int nq = ur.nq;
  if (a < lim) {
    if (a < nq)
      cur.load_q(ur.Kc, ur.Km, ur.Vc, ur.Vm, a, lim, lr, lg, lane);
    else
      cur.load(ur.Kp, ur.Vp, a, lim, lr, lg, lane);
  }
  const int a1 = a + kRowTile;
  if (a1 < lim) {
    if (a1 < nq)
      nxt.load_q(ur.Kc, ur.Km, ur.Vc, ur.Vm, a1, lim, lr, lg, lane);
    else
      nxt.load(ur.Kp, ur.Vp, a1, lim, lr, lg, lane);
  }
}

// The four waves' shares of a piece of nt tiles starting at row r0: wave w
// takes tiles [floor(w nt / 4), floor((w + 1) nt / 4)), contiguous, so the
// loads of a piece differ by at most one tile between waves.
__device__ __forceinline__ void wave_share(int r0, int nt, int w, int &a, int &b) {
  a = r0 + kRowTile * ((w * nt) >> 2);
  b = r0 + kRowTile * (((w + 1) * nt) >> 2);
}

// Merge the np partials of unit u (slots slot0 .. slot0+np-1, in row order);
// out = O / sum, zeros for an empty cache.  Thread t combines elements
// e = t + 256 k (head e / d, channel e % d) with a running maximum, eight
// pieces at a time: the (max, sum) pairs of a batch (all 16 heads) go
// through LDS (mlb, 128 pairs), and every load of a batch is issued before
// any is used, under uniform bounds (no load in a divergent branch), so a
// batch costs one round trip.
template <int D, bool COHERENT>
__device__ __forceinline__ void merge_pieces(const DecodePlan &p, float2 *mlb, int u, int slot0, int np) {
  constexpr int kBatch = 8;
  constexpr int kEl = 16 * D / 256;
  const int tid = threadIdx.x;
  const int g = u % p.Hkv;
  const int lb_ = u / p.Hkv;
  const int GD = p.G * D;
  const int nel = (GD + 255) / 256;  // element slots in use (uniform)
  float M[kEl], o[kEl], sum[kEl];
#pragma unroll
  for (int k = 0; k < kEl; ++k) {
    M[k] = kNegInf;
    o[k] = 0.f;
    sum[k] = 0.f;
  }
  for (int j0 = 0; j0 < np; j0 += kBatch) {
    const int nb = min(kBatch, np - j0);  // pieces in this batch (uniform)
    // Pair (piece j0 + t / 16, head t % 16) for t < 16 nb; the other
    // threads read pair 0 again and drop it.
    const int tp = tid < 16 * nb ? tid : 0;
    const float *mlp = reinterpret_cast<const float *>(p.part_ml + (int64_t)(slot0 + j0) * 16) + 2 * tp;
    const float m0 = ld_part<COHERENT>(mlp), s0 = ld_part<COHERENT>(mlp + 1);
    // Branch-free: pieces past the batch's end read its last piece again
    // and are dropped below; each load is a uniform base plus the lane's
    // 32-bit element offset.
    float po[kEl][kBatch];
#pragma unroll
    for (int k = 0; k < kEl; ++k) {
      if (k < nel) {  // uniform
#pragma unroll
        for (int b = 0; b < kBatch; ++b) {
          const float *base = p.part_o + (int64_t)(slot0 + j0 + min(b, nb - 1)) * 16 * D;
          po[k][b] = ld_part<COHERENT>(base + min(tid + 256 * k, GD - 1));
        }
      }
    }
    __syncthreads();  // the previous batch's pairs are read
    if (tid < kBatch * 16) mlb[tid] = tid < 16 * nb ? make_float2(m0, s0) : make_float2(kNegInf, 0.f);
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kEl; ++k) {
      if (k >= nel) continue;
      const int h = min(tid + 256 * k, GD - 1) / D;
      float Mc = M[k];
#pragma unroll
      for (int b = 0; b < kBatch; ++b) Mc = fmaxf(Mc, mlb[b * 16 + h].x);
      if (Mc == kNegInf) continue;
      if (M[k] != kNegInf && M[k] != Mc) {
        const float f = fast_exp2(M[k] - Mc);
        o[k] *= f;
        sum[k] *= f;
      }
      M[k] = Mc;
#pragma unroll
      for (int b = 0; b < kBatch; ++b) {
        const float2 ml = mlb[b * 16 + h];
        if (b >= nb || ml.x == kNegInf) continue;
        const float f = fast_exp2(ml.x - Mc);
        o[k] += f * po[k][b];
        sum[k] += f * ml.y;
      }
    }
  }
#pragma unroll
  for (int k = 0; k < kEl; ++k) {
    const int e = tid + 256 * k;
    if (k < nel && e < GD)
      stg(p.out + ((int64_t)lb_ * p.Hq + (int64_t)g * p.G) * D + e, sum[k] > 0.f ? o[k] / sum[k] : 0.f);
  }
}

// The end of a piece in the fused step.  A unit in one piece advances its
// length.  The pieces of a split unit: their partials' device-coherent stores
// complete before the arrival is counted; the last arriver reads every
// partial with device-coherent loads, merges them, advances the length
// (every piece read it before arriving) and re-arms the unit's counter.
template <int D>
__device__ __forceinline__ void arrive_and_merge(const DecodePlan &p, DecodeSmem<D> &sm, int u, int p0, int np,
                                                 int nrow) {
  const int tid = threadIdx.x;
  if (np == 1) {
    if (tid == 0 && nrow >= 0) stg(p.len_w + u, nrow + 1);
    return;
  }
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  if (tid == 0)
    sm.flag[0] = __hip_atomic_fetch_add(p.arrive + u, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                 (uint32_t)(np - 1);
  __syncthreads();
  if (!sm.flag[0]) return;
  merge_pieces<D, true>(p, sm.mlb, u, p0, np);
  if (tid == 0) {
    __hip_atomic_store(p.arrive + u, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (nrow >= 0) stg(p.len_w + u, nrow + 1);
  }
}

// The appended K/V row of unit u, 16-byte chunk c = tid mod 2 (d/8) (K
// chunks first; every thread loads one, so the load sits in no branch):
// read from k_new / v_new ...
template <int D>
__device__ __forceinline__ u32x4 load_new_chunk(const DecodePlan &p, int u, int tid) {
  const int c = tid % (2 * (D / 8));
  const int cc = c % (D / 8);
  return ld16((c < D / 8 ? p.k_new : p.v_new) + (int64_t)u * D + cc * 8);
}
// ... then staged in the wave's own LDS copy (every lane writes its chunk;
// lanes holding the same chunk write the same bytes), from where the wave
// patches it into the tile that holds it, and written to the pool by the
// first wave of the unit's first piece.
template <int D>
__device__ __forceinline__ void stage_new_chunk(const DecodePlan &p, DecodeSmem<D> &sm, int w, int tid, u32x4 x,
                                                int64_t roff, int nrow, bool first) {
  const int c = tid % (2 * (D / 8));
  *reinterpret_cast<u32x4 *>(sm.newrow[w] + c * 8) = x;
  if (first && nrow >= 0 && tid < 2 * (D / 8)) {
    const int cc = c % (D / 8);
    st16((c >= D / 8 ? p.v_pool_w : p.k_pool_w) + (roff + nrow) * D + cc * 8, x);
  }
}

// Decode attention over the cut (STEP: the fused step, which also appends
// the new rows, merges each split unit in the last of its workgroups to
// finish, and advances the unit's length there).
template <int D, bool STEP, bool Q4 = false>
__device__ __forceinline__ void decode_body(const DecodePlan &p) {
  __shared__ DecodeSmem<D> sm;
  // Pieces follow the dispatch order, so the workgroups left without a piece
  // are spread over all XCDs.
  const uint32_t i = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lg = lane >> 4;
  const Piece pc = cut<STEP>(p, i);
  const int u = pc.u, np = pc.np, p0 = pc.p0;
  if (u < 0) return;
  int rows, nrow;
  unit_rows<STEP>(pc.len0, pc.cap, p.max_rows, rows, nrow);
  // Piece j of np covers tiles [j nt / np, (j + 1) nt / np) of the unit
  // (nt < 2^26 since rows fit int32, so the products stay below 2^52).
  const int t0 = (int)floor_div64((uint64_t)pc.j * (uint32_t)pc.nt, (uint32_t)np);
  const int t1 = (int)floor_div64((uint64_t)(pc.j + 1) * (uint32_t)pc.nt, (uint32_t)np);
  int a, b;
  wave_share(t0 * kRowTile, t1 - t0, w, a, b);
  const int e = min(b, rows);
  const u32x4 nrc = STEP ? load_new_chunk<D>(p, u, tid) : u32x4{0u, 0u, 0u, 0u};
  QueryOps<D, Q4> qo;
  qo.load(p, sm, u, w, lr, lg);
  UnitRows<D> ur{};
  ur.Kp = p.k_pool + pc.roff * D;
  ur.Vp = p.v_pool + pc.roff * D;
  if (Q4) {
    // The unit's 4-bit rows: a multiple of the tile, within its length.
    ur.nq = max(min(ldg(p.nq + u) & ~(kRowTile - 1), max(pc.len0, 0) & ~(kRowTile - 1)), 0);
    const int64_t qoff = ldg(p.qoff + u);
    ur.Kc = p.qk + qoff * (D / 2);
    ur.Vc = p.qv + qoff * (D / 2);
    ur.Km = p.qkm + qoff * (D / 32);
    ur.Vm = p.qvm + qoff * (D / 32);
  }
  RowTile<D> cur, nxt;
  first_tiles<D, Q4>(ur, qo.row0, cur, nxt, a, e, lr, lg, lane);
  if (STEP) {
    stage_new_chunk<D>(p, sm, w, tid, nrc, pc.roff, nrow, pc.j == 0);
  } else if (pc.j == 0 && tid == 0) {
    stg(reinterpret_cast<int32_t *>(p.pinfo + u), p0);
    stg(reinterpret_cast<int32_t *>(p.pinfo + u) + 1, np);
  }
  if (Q4) __syncthreads();  // the query rows in LDS
  f32x4 O[D / 16];
  float mrow, lsum;
  wave_rows<D, Q4>(p, sm, qo, ur, cur, nxt, a, e, e, nrow, O, mrow, lsum);
  if (np == 1)
    finish_piece<D, kOutput>(p, sm, u, 0, O, mrow, lsum);
  else
    finish_piece<D, STEP ? kPartialCoherent : kPartial>(p, sm, u, (int)i, O, mrow, lsum);
  if (STEP) arrive_and_merge<D>(p, sm, u, p0, np, nrow);
}

// The fused step over a piece table built on the host.  Workgroup i reads
// its record (unit, piece, rows [r0, r1) of the unit's capacity, the unit's
// first pool row); the unit's length, its query heads, the appended row and
// the first tile of each wave (rows up to the piece's end, as far as the
// capacity goes) are then all requested at once, so the length costs no
// round trip of its own: tiles read before the length was known are patched
// where the length says their rows are not this step's (the appended row,
// rows past the end).  4-bit caches read their first tile after the length,
// since its kind depends on it.  A table whose header does not match the
// call's shape and row bound leaves NaN in every output.
template <int D, bool Q4>
__device__ __forceinline__ void planned_body(const DecodePlan &p) {
  __shared__ DecodeSmem<D> sm;
  const int i = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane & 15, lg = lane >> 4;
  const int32_t *hdr = p.plan;
  const int32_t *rec = p.plan + kDecodePlanHdrWords + (int64_t)kDecodePlanRecWords * i;
  // Header and record in one round trip (both loads unconditional; the
  // host checked that the table has a record for every workgroup).
  const int h0 = ldg(hdr), h1 = ldg(hdr + 1), h2 = ldg(hdr + 2), h3 = ldg(hdr + 3), h4 = ldg(hdr + 4);
  const int u = ldg(rec), jn = ldg(rec + 1), p0 = ldg(rec + 2);
  const int r0 = ldg(rec + 3), r1 = ldg(rec + 4), rs = ldg(rec + 5);
  const int j = jn & 0xFFFF, np = jn >> 16;
  const int64_t roff = (int64_t)(((uint64_t)(uint32_t)ldg(rec + 7) << 32) | (uint32_t)ldg(rec + 6));
  // (The record's unit takes part in the check, which keeps its load beside
  // the header's instead of behind the branch.)
  const bool ok = (h0 == kDecodePlanMagic) & (h1 == p.units) & (h2 == p.nwg) & (h3 == D) & (h4 == p.max_rows) &
                  (u < p.units);
  if (!ok) {
    if (i < p.units) {
      const int g = i % p.Hkv, lb_ = i / p.Hkv;
      float *o = p.out + ((int64_t)lb_ * p.Hq + (int64_t)g * p.G) * D;
      for (int x = tid; x < p.G * D; x += 256) stg(o + x, __builtin_nanf(""));
    }
    return;
  }
  if (u < 0) return;
  int a, b;
  wave_share(r0, (r1 - r0 + kRowTile - 1) / kRowTile, w, a, b);
  b = min(b, r1);
  // The appended row first: staging it waits for it (and for any load
  // issued before it), not for the query or the tiles.
  // The length and capacity as vector loads (an opaque zero offset keeps
  // them off the scalar path, whose wait would also hold back the tile
  // requests behind them), ahead of the tiles' requests.
  int z;
  asm volatile("v_mov_b32 %0, 0" : "=v"(z));
  const int len_v = ldg(p.len + u + z), cap_v = ldg(p.cap + u + z);
  const u32x4 nrc = load_new_chunk<D>(p, u, tid);
  __builtin_amdgcn_sched_barrier(0);
  QueryOps<D, Q4> qo;
  qo.load(p, sm, u, w, lr, lg);
  UnitRows<D> ur{};
  ur.Kp = p.k_pool + roff * D;
  ur.Vp = p.v_pool + roff * D;
  int nq0 = 0;
  int64_t qoff = 0;
  if (Q4) {
    nq0 = ldg(p.nq + u);
    qoff = ldg(p.qoff + u);
  }
  // Rows read before the length is known: up to the piece's early bound.
  const int spec = Q4 ? 0 : min(b, rs);
  RowTile<D> cur, nxt;
  if (!Q4) first_tiles<D, false>(ur, qo.row0, cur, nxt, a, spec, lr, lg, lane);
  __builtin_amdgcn_sched_barrier(0);
  const int len0 = __builtin_amdgcn_readfirstlane(len_v), capd = __builtin_amdgcn_readfirstlane(cap_v);
  int rows, nrow;
  unit_rows<true>(len0, capd, p.max_rows, rows, nrow);
  const int e = min(b, rows);
  stage_new_chunk<D>(p, sm, w, tid, nrc, roff, nrow, j == 0);
  if (Q4) {
    __syncthreads();  // the query rows in LDS
    ur.nq = max(min(nq0 & ~(kRowTile - 1), max(len0, 0) & ~(kRowTile - 1)), 0);
    ur.Kc = p.qk + qoff * (D / 2);
    ur.Vc = p.qv + qoff * (D / 2);
    ur.Km = p.qkm + qoff * (D / 32);
    ur.Vm = p.qvm + qoff * (D / 32);
    first_tiles<D, true>(ur, qo.row0, cur, nxt, a, e, lr, lg, lane);
  }
  f32x4 O[D / 16];
  float mrow, lsum;
  wave_rows<D, Q4>(p, sm, qo, ur, cur, nxt, a, e, Q4 ? e : spec, nrow, O, mrow, lsum);
  if (np == 1)
    finish_piece<D, kOutput>(p, sm, u, 0, O, mrow, lsum);
  else
    finish_piece<D, kPartialCoherent>(p, sm, u, p0 + j, O, mrow, lsum);
  arrive_and_merge<D>(p, sm, u, p0, np, nrow);
}

template <int D>
__global__ __launch_bounds__(256, 2) void k_decode_attn(DecodePlan p) {
  decode_body<D, false>(p);
}

// One decode step in one launch: append, attention and the merge of split
// units.
template <int D>
__global__ __launch_bounds__(256, 2) void k_decode_step(DecodePlan p) {
  decode_body<D, true>(p);
}

// The fused step over a cache with a 4-bit prefix.
template <int D>
__global__ __launch_bounds__(256, 2) void k_decode_step_q4(DecodePlan p) {
  decode_body<D, true, true>(p);
}

// The fused step over a host-built piece table (bf16 rows, or a 4-bit prefix).
template <int D, bool Q4>
__global__ __launch_bounds__(256, 2) void k_decode_planned(DecodePlan p) {
  planned_body<D, Q4>(p);
}

// Merge the pieces of each split unit (second kernel of the two-call path).
template <int D>
__global__ __launch_bounds__(256) void k_decode_combine(DecodePlan p) {
  const int u = blockIdx.x;
  const int slot0 = ldg(reinterpret_cast<const int32_t *>(p.pinfo + u));
  const int np = ldg(reinterpret_cast<const int32_t *>(p.pinfo + u) + 1);
  __shared__ float2 mlb[128];
  if (np > 1) merge_pieces<D, false>(p, mlb, u, slot0, np);
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
  if (p.units == 0 || p.nwg < 1) return hipSuccess;
  if (p.d == 128)
    hipLaunchKernelGGL(k_decode_step<128>, dim3(p.nwg), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(k_decode_step<64>, dim3(p.nwg), dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_decode_step_q4(const DecodePlan &p, hipStream_t st) {
  if (p.units == 0 || p.nwg < 1) return hipSuccess;
  if (p.d == 128)
    hipLaunchKernelGGL(k_decode_step_q4<128>, dim3(p.nwg), dim3(256), 0, st, p);
  else
    hipLaunchKernelGGL(k_decode_step_q4<64>, dim3(p.nwg), dim3(256), 0, st, p);
  return hipGetLastError();
}

hipError_t launch_decode_planned(const DecodePlan &p, bool q4, hipStream_t st) {
  if (p.units == 0 || p.nwg < 1) return hipSuccess;
  if (p.d == 128) {
    if (q4)
      hipLaunchKernelGGL((k_decode_planned<128, true>), dim3(p.nwg), dim3(256), 0, st, p);
    else
      hipLaunchKernelGGL((k_decode_planned<128, false>), dim3(p.nwg), dim3(256), 0, st, p);
  } else {
    if (q4)
      hipLaunchKernelGGL((k_decode_planned<64, true>), dim3(p.nwg), dim3(256), 0, st, p);
    else
      hipLaunchKernelGGL((k_decode_planned<64, false>), dim3(p.nwg), dim3(256), 0, st, p);
  }
  return hipGetLastError();
}

// ---- scratch of the allocation-free decode step ---------------------------
// One copy of this array per device, allocated when the code object is loaded
// and held until the process ends: the arrival counters of split units at
// the front (kNoAllocCounterBytes, zero between calls), the pieces' partial
// results behind them.  Host code never passes the array's name to a
// kernel (on the host it names a stand-in, not device memory); it uses the
// device address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) uint8_t scratch[kNoAllocBytes];

namespace {
__global__ __launch_bounds__(256) void k_clear_words(uint32_t *p, uint32_t n) {
  for (uint32_t i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0u;
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
uint8_t *g_scratch[kMaxDevices];
}  // namespace

hipError_t noalloc_scratch(uint8_t **out, hipStream_t st) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void *ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!ptr) return hipErrorInvalidSymbol;
    // The counters start at zero (the array is zero when loaded; clear them
    // anyway before the first call on this device uses them), and every
    // call leaves them at zero.
    hipLaunchKernelGGL(k_clear_words, dim3(kNoAllocCounterBytes / 4 / 256), dim3(256), 0, st,
                       static_cast<uint32_t *>(ptr), (uint32_t)(kNoAllocCounterBytes / 4));
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    g_scratch[dev] = static_cast<uint8_t *>(ptr);
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

hipError_t launch_decode(const DecodePlan &p, hipStream_t st) {
  if (p.units == 0 || p.nwg < 1) return hipSuccess;
  if (p.d == 128) {
    hipLaunchKernelGGL(k_decode_attn<128>, dim3(p.nwg), dim3(256), 0, st, p);
    hipLaunchKernelGGL(k_decode_combine<128>, dim3(p.units), dim3(256), 0, st, p);
  } else {
    hipLaunchKernelGGL(k_decode_attn<64>, dim3(p.nwg), dim3(256), 0, st, p);
    hipLaunchKernelGGL(k_decode_combine<64>, dim3(p.units), dim3(256), 0, st, p);
  }
  return hipGetLastError();
}

}  // namespace vc
