// vc_decode_plan.cpp -- host: the piece table of a planned decode step
// (Sec. 2, decoding).  Capacities do not change from step to step, so the cut
// of the caches' rows into workgroup pieces is made once per cache here,
// instead of by every workgroup of every step.
//
// The cut works in 32-row tiles of each unit's capacity (at most max_rows
// rows).  A piece of n tiles is shared by the four waves of its workgroup,
// each taking floor or ceil of n / 4 consecutive tiles, so what bounds a
// step is the largest per-wave share m.  The table takes the smallest m (at
// least 2 tiles: below that a split saves less than the merge of its pieces
// costs) for which splitting every unit into ceil(tiles / 4m) pieces fits
// the launch's workgroups; workgroups left over then split further the units
// that need the fewest extra pieces to bring their share below m.  With more
// units than resident slots whose units past the first round are short, no
// unit is cut (see below).  Pieces are dealt to workgroups longest first, so
// a launch with more pieces than resident slots starts its longest ones
// first, and consecutive workgroups (which the hardware spreads over the
// XCDs) carry similar loads.
#include <algorithm>
#include <cstdint>
#include <functional>
#include <numeric>
#include <vector>

#include "vc_internal.h"
#include "viscache.h"

namespace vc {

namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Rows past the length at planning time that the early reads still cover.
constexpr int64_t kSpecRows = 64;

// Per-wave share (tiles) of a unit of t tiles cut into np pieces.
int64_t wave_share(int64_t t, int64_t np) { return ceil_div(ceil_div(t, np), 4); }

}  // namespace

int decode_plan_build(int32_t units, const int32_t *cap, const int64_t *row_off, const int32_t *len_hint,
                      int64_t max_rows, int32_t nwg, int32_t d, int32_t *out) {
  if (units < 1 || nwg <= units || max_rows < 0) return VC_ERR_ARG;
  const int64_t U = units;
  if (len_hint)
    for (int64_t u = 0; u < U; ++u)
      if (len_hint[u] < 0) return VC_ERR_ARG;
  // Blocks: non-negative, and no two units' rows overlap.
  for (int64_t u = 0; u < U; ++u)
    if (cap[u] < 0 || row_off[u] < 0 || row_off[u] > INT64_MAX - cap[u]) return VC_ERR_ARG;
  // Row indices of a piece, rounded up to whole tiles, stay within int32.
  for (int64_t u = 0; u < U; ++u)
    if (cap[u] > INT32_MAX - 2 * kDecodeTileRows) return VC_ERR_UNSUPPORTED;
  {
    std::vector<int64_t> ord;
    ord.reserve((size_t)U);
    for (int64_t u = 0; u < U; ++u)
      if (cap[u] > 0) ord.push_back(u);
    std::sort(ord.begin(), ord.end(), [&](int64_t a, int64_t b) { return row_off[a] < row_off[b]; });
    for (size_t k = 1; k < ord.size(); ++k)
      if (row_off[ord[k]] < row_off[ord[k - 1]] + cap[ord[k - 1]]) return VC_ERR_ARG;
  }
  const int64_t kTile = kDecodeTileRows;
  std::vector<int64_t> capb((size_t)U), t((size_t)U);
  int64_t tmax = 0;
  for (int64_t u = 0; u < U; ++u) {
    capb[u] = std::min<int64_t>(cap[u], max_rows);
    t[u] = ceil_div(capb[u], kTile);
    tmax = std::max(tmax, t[u]);
  }
  auto pieces = [&](int64_t m) {
    int64_t P = 0;
    for (int64_t u = 0; u < U; ++u) P += std::max<int64_t>(1, ceil_div(t[u], 4 * m));
    return P;
  };
  // Smallest share m with a cut that fits (P(m) does not grow with m; at
  // m_hi every unit is one piece, and nwg > units).
  const int64_t m_lo = kDecodeMinPiece / 4;
  int64_t lo = m_lo, hi = std::max(m_lo, ceil_div(tmax, 4));
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo) / 2;
    if (pieces(mid) <= nwg)
      hi = mid;
    else
      lo = mid + 1;
  }
  int64_t m = lo;
  // More units than resident slots: if the units past the first round are
  // at most a quarter of the longest (they fill the gaps the first round
  // leaves), cut none, since a split only adds its merge; otherwise the
  // longest would wait for a second round whole, and the cut above
  // shortens them.
  bool cut_none = false;
  if (U > kDecodeSlots) {
    std::vector<int64_t> ts(t);
    std::nth_element(ts.begin(), ts.begin() + kDecodeSlots, ts.end(), std::greater<int64_t>());
    cut_none = 4 * ts[(size_t)kDecodeSlots] <= tmax;
    if (cut_none) m = std::max(m, ceil_div(tmax, 4));
  }
  std::vector<int64_t> np((size_t)U);
  int64_t P = 0;
  for (int64_t u = 0; u < U; ++u) {
    np[u] = std::max<int64_t>(1, ceil_div(t[u], 4 * m));
    P += np[u];
  }
  // Leftover workgroups: bring the units whose share is m below it, those
  // needing the fewest extra pieces first (not when no unit is to be cut).
  if (!cut_none && m > m_lo && P < nwg) {
    std::vector<std::pair<int64_t, int64_t>> need;  // (extra pieces, unit)
    for (int64_t u = 0; u < U; ++u)
      if (wave_share(t[u], np[u]) >= m) need.emplace_back(ceil_div(t[u], 4 * (m - 1)) - np[u], u);
    std::stable_sort(need.begin(), need.end(),
                     [](const std::pair<int64_t, int64_t> &a, const std::pair<int64_t, int64_t> &b) {
                       return a.first < b.first;
                     });
    for (const auto &x : need) {
      if (P + x.first > nwg) break;
      np[x.second] += x.first;
      P += x.first;
    }
  }
  for (int64_t u = 0; u < U; ++u)
    if (np[u] > 0xFFFF) return VC_ERR_UNSUPPORTED;  // (at most nwg - units + 1; cannot happen)
  // Pieces in unit order (their partial slots), then dealt longest first.
  struct Pc {
    int32_t u, j, np, p0, r0, r1, rs, tiles;
  };
  std::vector<Pc> pcs;
  pcs.reserve((size_t)P);
  int64_t slot = 0;
  for (int64_t u = 0; u < U; ++u) {
    for (int64_t j = 0; j < np[u]; ++j) {
      const int64_t T0 = j * t[u] / np[u], T1 = (j + 1) * t[u] / np[u];
      Pc pc;
      pc.u = (int32_t)u;
      pc.j = (int32_t)j;
      pc.np = (int32_t)np[u];
      pc.p0 = (int32_t)slot;
      pc.r0 = (int32_t)(T0 * kTile);
      pc.r1 = (int32_t)std::min<int64_t>(T1 * kTile, capb[u]);
      pc.rs = pc.r1;
      if (len_hint)
        pc.rs = (int32_t)std::max<int64_t>(pc.r0, std::min<int64_t>(pc.r1, (int64_t)len_hint[u] + kSpecRows));
      pc.tiles = (int32_t)(T1 - T0);
      pcs.push_back(pc);
    }
    slot += np[u];
  }
  std::stable_sort(pcs.begin(), pcs.end(), [](const Pc &a, const Pc &b) { return a.tiles > b.tiles; });
  int32_t *h = out;
  h[0] = kDecodePlanMagic;
  h[1] = units;
  h[2] = nwg;
  h[3] = d;
  h[4] = (int32_t)std::min<int64_t>(max_rows, INT32_MAX);
  h[5] = (int32_t)P;
  h[6] = 0;
  h[7] = 0;
  for (int64_t i = 0; i < nwg; ++i) {
    int32_t *r = out + kDecodePlanHdrWords + kDecodePlanRecWords * i;
    if (i < P) {
      const Pc &pc = pcs[(size_t)i];
      const uint64_t ro = (uint64_t)row_off[pc.u];
      r[0] = pc.u;
      r[1] = pc.j | (pc.np << 16);
      r[2] = pc.p0;
      r[3] = pc.r0;
      r[4] = pc.r1;
      r[5] = pc.rs;
      r[6] = (int32_t)(uint32_t)(ro & 0xFFFFFFFFu);
      r[7] = (int32_t)(uint32_t)(ro >> 32);
    } else {
      r[0] = -1;
      for (int k = 1; k < kDecodePlanRecWords; ++k) r[k] = 0;
    }
  }
  return VC_OK;
}

}  // namespace vc
