// vc_api.cpp -- the C ABI of libviscache (include/viscache.h): argument
// checks, budgets, workspace layout, and the launch sequence of one PruneKV
// call (Algorithm 1) and of one decode step.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <vector>

#include "../../include/viscache.h"
#include "vc_budget.h"
#include "vc_internal.h"

using namespace vc;

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

// Everything derived from (shape, params) on the host.
struct Layout {
  int32_t B, L, Hq, Hkv, d, W, G, R, h, Ls, mode, vfp32;
  int32_t nqg, nks, ncol, nmax;
  int32_t prefill, pwg;
  int64_t Ntot;
  std::vector<int32_t> n, k, ns;       // n[B], k[B*L], ns[B*L]
  std::vector<int32_t> funit;          // fusion units, longest drop list first
  std::vector<int32_t> fwoff, fwjob;   // fusion job queues per XCD (CSR): job = rank << 8 | tile
  std::vector<int32_t> fcnt0;          // jobs of each queue handed out at launch
  int32_t nfwg = 0;                    // persistent fusion workgroups
  std::vector<int64_t> toff, orow, drow;
  // workspace regions (byte offsets)
  size_t off_plan, plan_bytes, off_qbf, off_part, off_S, off_gs, off_drop, total;
  // offsets inside the plan blob
  size_t p_lp, p_nb, p_toff, p_kk, p_ns, p_orow, p_drow, p_funit, p_fwoff, p_fwjob, p_fcnt;
};

vc_status check_shape(const vc_shape *s) {
  if (!s || !s->n_vis) return VC_ERR_ARG;
  if (s->B < 1 || s->L < 2 || s->Hq < 1 || s->Hkv < 1 || s->W < 1) return VC_ERR_SHAPE;
  if (s->Hq % s->Hkv != 0) return VC_ERR_SHAPE;
  if (s->d != 64 && s->d != 128) return VC_ERR_UNSUPPORTED;
  for (int32_t b = 0; b < s->B; ++b)
    if (s->n_vis[b] < 0 || s->n_vis[b] > kMaxTokens) return s->n_vis[b] < 0 ? VC_ERR_SHAPE : VC_ERR_UNSUPPORTED;
  // The layer pointers, token offsets and lengths must fit the plan's first
  // chunk (L = 128 layers leave room for about 1800 sequences).
  if (sizeof(uint64_t) * (LP_COUNT * (size_t)s->L + s->B + 1) + sizeof(int32_t) * (size_t)s->B + 8 >
      sizeof(uint32_t) * (size_t)kChunkWords)
    return VC_ERR_UNSUPPORTED;
  return VC_OK;
}

vc_status check_params(const vc_params *p, int32_t L) {
  if (!p) return VC_ERR_ARG;
  if (!(p->retention > 0.0 && p->retention <= 1.0)) return VC_ERR_BUDGET;
  if (!(p->m > 0.0 && p->m <= 1.0)) return VC_ERR_BUDGET;
  if (p->h != 0 && (p->h < 2 || p->h > L)) return VC_ERR_BUDGET;
  if (!(p->tau > 0.f) || !std::isfinite(p->tau)) return VC_ERR_ARG;
  if (!(p->mu >= 0.f && p->mu <= 1.f)) return VC_ERR_ARG;
  if (p->rank_mode != VC_RANK_LAYER_HEAD && p->rank_mode != VC_RANK_GLOBAL) return VC_ERR_ARG;
  if (p->v_out_fp32 != 0 && p->v_out_fp32 != 1) return VC_ERR_ARG;
  if (p->schedule < VC_SCHED_PARABOLIC || p->schedule > VC_SCHED_GEOMETRIC) return VC_ERR_ARG;
  if (p->drop_all != 0 && p->drop_all != 1) return VC_ERR_ARG;
  if (p->score_queries != VC_SCORE_WINDOW && p->score_queries != VC_SCORE_PREFILL) return VC_ERR_ARG;
  return VC_OK;
}

vc_status make_layout(const vc_shape *s, const vc_params *p, Layout &y) {
  vc_status st = check_shape(s);
  if (st != VC_OK) return st;
  st = check_params(p, s->L);
  if (st != VC_OK) return st;
  y.B = s->B; y.L = s->L; y.Hq = s->Hq; y.Hkv = s->Hkv; y.d = s->d; y.W = s->W;
  y.G = s->Hq / s->Hkv;
  y.R = y.G * y.W;
  y.mode = p->rank_mode;
  y.vfp32 = p->v_out_fp32;
  y.prefill = p->score_queries == VC_SCORE_PREFILL;
  if (!y.prefill && (int64_t)y.R > 1024) return VC_ERR_UNSUPPORTED;
  y.n.assign(s->n_vis, s->n_vis + s->B);
  y.k.assign((size_t)y.B * y.L, 0);
  y.ns.assign((size_t)y.B * y.L, 0);
  y.h = 0;
  for (int32_t b = 0; b < y.B; ++b) {
    int32_t nsv = 0, hu = 0;
    if (!budget_one(y.L, y.n[b], p->retention, p->h, p->m, p->schedule, p->drop_all, &y.k[(size_t)b * y.L],
                    &nsv, &hu))
      return VC_ERR_BUDGET;
    for (int32_t l = 0; l < y.L; ++l) y.ns[(size_t)b * y.L + l] = nsv;
    y.h = hu;
  }
  y.Ls = y.mode == VC_RANK_GLOBAL ? y.L : y.h;
  y.toff.assign(y.B + 1, 0);
  for (int32_t b = 0; b < y.B; ++b) y.toff[b + 1] = y.toff[b] + y.n[b];
  y.Ntot = y.toff[y.B];
  y.orow.assign((size_t)y.L * (y.B + 1), 0);
  y.drow.assign((size_t)y.L * (y.B + 1), 0);
  for (int32_t l = 0; l < y.L; ++l)
    for (int32_t b = 0; b < y.B; ++b) {
      const int32_t kk = y.k[(size_t)b * y.L + l];
      const int32_t rr = l < y.h ? y.ns[(size_t)b * y.L + l] - kk : 0;
      y.orow[(size_t)l * (y.B + 1) + b + 1] = y.orow[(size_t)l * (y.B + 1) + b] + (int64_t)y.Hkv * kk;
      y.drow[(size_t)l * (y.B + 1) + b + 1] = y.drow[(size_t)l * (y.B + 1) + b] + (int64_t)y.Hkv * rr;
    }
  y.nmax = *std::max_element(y.n.begin(), y.n.end());
  const int64_t units = (int64_t)y.Ls * y.B * y.Hkv;
  int64_t rows = y.R;  // query rows of the longest unit
  y.pwg = 0;
  if (y.prefill) {
    // Every prefill token queries: a unit has G * (n_b + W) rows, in groups
    // of 256.  Each of a unit's pwg workgroups owns every pwg-th group.  The
    // groups per workgroup are chosen so that all units together make about
    // eight rounds of the resident slots: small workgroups of near-equal
    // size let the dispatcher balance groups whose causal prefixes differ
    // (two groups per workgroup ran 19% faster than three to four on the 7B
    // shape), at the price of more column partials to add up.
    rows = (int64_t)y.G * ((int64_t)y.nmax + y.W);
    if (rows > (int64_t(1) << 26)) return VC_ERR_UNSUPPORTED;
    const int64_t groups = (rows + kStatsRows - 1) / kStatsRows;
    const int64_t per_wg = std::max<int64_t>(1, (groups * units + 4 * kScoreSlots) / (8 * kScoreSlots));
    y.pwg = (int32_t)std::min<int64_t>(groups, (groups + per_wg - 1) / per_wg);
  }
  y.nqg = (int32_t)((rows + kStatsRows - 1) / kStatsRows);
  const int64_t base = std::max<int64_t>(1, units * y.nqg);
  // Key splits so that the statistics pass runs in one round of resident
  // workgroups: a second, partial round costs a full workgroup time for a
  // fraction of the work.  A grid of more than one round takes two splits:
  // halving every workgroup halves the granularity of the last round
  // (measured on the batched shape: statistics 1.80 -> 1.64 ms, the column
  // pass unchanged; neutral on the 72B shape).
  int64_t nks = base > kScoreSlots ? 2 : std::max<int64_t>(1, kScoreSlots / base);
  nks = std::min<int64_t>(nks, kMaxSplits);
  nks = std::min<int64_t>(nks, std::max(1, (y.nmax + kKeyTile - 1) / kKeyTile));
  y.nks = y.prefill ? 1 : (int32_t)std::max<int64_t>(1, nks);
  y.ncol = std::max(1, (y.nmax + kColKeys - 1) / kColKeys);
  // A launch holds at most 2^32 - 1 threads: 256-thread workgroups per
  // (unit, row group, key split) and per (unit, key chunk) for the window
  // scores; per (unit, share) and per (unit, 256 keys) for the prefill scores.
  const int64_t per_unit = y.prefill ? std::max<int64_t>(y.pwg, (y.nmax + 255) / 256)
                                     : std::max<int64_t>((int64_t)y.nqg * y.nks, y.ncol);
  if (units * per_unit > (int64_t(1) << 24) - 1) return VC_ERR_UNSUPPORTED;
  // Fusion units (layer < h with kept rows), ordered by dropped-row count,
  // descending: every workgroup of a unit walks all of its dropped tiles, so
  // dispatching the longest chains first bounds the tail.
  y.funit.clear();
  for (int32_t l = 0; l < y.h; ++l)
    for (int32_t b = 0; b < y.B; ++b)
      if (y.k[(size_t)b * y.L + l] > 0)
        for (int32_t g = 0; g < y.Hkv; ++g) y.funit.push_back((l * y.B + b) * y.Hkv + g);
  // A fusion job is one int32, unit rank << 8 | 128-row tile (a unit has at
  // most 32768 / 128 = 256 tiles), so the ranks must stay below 2^23.
  if (y.funit.size() >= (size_t(1) << 23)) return VC_ERR_UNSUPPORTED;
  auto drops = [&](int32_t u) {
    const int32_t l = u / (y.Hkv * y.B), b = (u / y.Hkv) % y.B;
    return y.ns[(size_t)b * y.L + l] - y.k[(size_t)b * y.L + l];
  };
  std::stable_sort(y.funit.begin(), y.funit.end(),
                   [&](int32_t a, int32_t c) { return drops(a) > drops(c); });
  // Fusion jobs (unit, 128 kept rows) in one queue per XCD.  Units are dealt
  // to XCDs largest first, each to the XCD with the least work so far (all
  // jobs of a unit share its dropped rows in that XCD's L2); each queue lists
  // its jobs longest first.  Cost of a job: its dropped tiles plus a job's
  // fixed start-up and wind-down, in tile units.  The persistent workgroups
  // of an XCD (block b runs on XCD b % 8) start on the first jobs of its
  // queue and take the rest one by one as they finish, so the work balances
  // itself at run time.
  {
    constexpr int32_t kFuseSlots = 512;  // resident fusion workgroups (256 CUs x 2)
    constexpr int64_t kJobStart = 4;
    struct Job { int32_t cost; int32_t code; };
    std::vector<std::vector<Job>> xj(kXcdsHost);
    std::vector<int64_t> xload(kXcdsHost, 0);
    int64_t njobs = 0;
    for (size_t rk = 0; rk < y.funit.size(); ++rk) {
      const int32_t u = y.funit[rk];
      const int32_t l = u / (y.Hkv * y.B), b = (u / y.Hkv) % y.B;
      const int32_t kk = y.k[(size_t)b * y.L + l];
      const int32_t rr = y.ns[(size_t)b * y.L + l] - kk;
      const int32_t cost = (rr + kDropTile - 1) / kDropTile;
      const int32_t nj = (kk + kFuseRows - 1) / kFuseRows;
      const int32_t x = (int32_t)(std::min_element(xload.begin(), xload.end()) - xload.begin());
      xload[x] += (int64_t)nj * (kJobStart + cost);
      for (int32_t t = 0; t < nj; ++t) xj[x].push_back({cost, (int32_t)(rk << 8) | t});
      njobs += nj;
    }
    y.fwoff.assign(kXcdsHost + 1, 0);
    y.fwjob.clear();
    y.fwjob.reserve((size_t)njobs);
    size_t longest = 0;
    for (int32_t x = 0; x < kXcdsHost; ++x) {
      auto &jl = xj[x];
      // Units come longest drop list first, so the jobs usually are in order.
      auto longer = [](const Job &a, const Job &c) { return a.cost > c.cost; };
      if (!std::is_sorted(jl.begin(), jl.end(), longer)) std::stable_sort(jl.begin(), jl.end(), longer);
      for (const Job &j : jl) y.fwjob.push_back(j.code);
      y.fwoff[(size_t)x + 1] = (int32_t)y.fwjob.size();
      longest = std::max(longest, jl.size());
    }
    y.nfwg = (int32_t)std::min<int64_t>(kFuseSlots / kXcdsHost, (int64_t)longest) * kXcdsHost;
    // Jobs already handed out per queue: each of the XCD's workgroups starts
    // on one of the first jobs.
    y.fcnt0.assign(kXcdsHost, 0);
    for (int32_t x = 0; x < kXcdsHost; ++x)
      y.fcnt0[(size_t)x] = std::min<int32_t>(y.nfwg / kXcdsHost, (int32_t)xj[x].size());
  }

  // Plan blob.
  size_t o = 0;
  // The score statistics kernel reads the first three tables from the
  // plan's first chunk, so they come first (check_shape bounds their size).
  y.p_lp = o; o += sizeof(uint64_t) * LP_COUNT * y.L;
  y.p_toff = o; o += sizeof(int64_t) * (y.B + 1);
  y.p_nb = o; o += sizeof(int32_t) * y.B;
  o = (o + 7) & ~size_t(7);
  y.p_orow = o; o += sizeof(int64_t) * y.L * (y.B + 1);
  y.p_drow = o; o += sizeof(int64_t) * y.L * (y.B + 1);
  y.p_kk = o; o += sizeof(int32_t) * y.B * y.L;
  y.p_ns = o; o += sizeof(int32_t) * y.B * y.L;
  o = (o + 15) & ~size_t(15);
  y.p_funit = o; o += sizeof(FuseUnit) * y.funit.size();
  y.p_fwoff = o; o += sizeof(int32_t) * y.fwoff.size();
  y.p_fcnt = o; o += sizeof(int32_t) * kXcdsHost;  // queue counters, reset by every plan upload
  y.p_fwjob = o; o += sizeof(int32_t) * y.fwjob.size();
  o = (o + 7) & ~size_t(7);
  y.plan_bytes = o;

  size_t w = 0;
  y.off_plan = w; w = align_up(w + y.plan_bytes);
  y.off_qbf = w;  // bf16 window queries (the prefill passes convert their queries in registers)
  w = align_up(w + (y.prefill ? 0 : sizeof(uint16_t) * (size_t)y.Ls * y.B * y.Hq * y.W * y.d));
  y.off_part = w;  // window row statistics, or the prefill column partials
  w = align_up(w + (y.prefill ? sizeof(float) * (size_t)units * y.pwg * y.nmax
                              : sizeof(float2) * (size_t)units * y.nks * y.R));
  y.off_S = w; w = align_up(w + sizeof(float) * (size_t)y.Ls * y.Ntot * y.Hkv);
  y.off_gs = w; w = align_up(w + (y.mode == VC_RANK_GLOBAL ? sizeof(float) * (size_t)y.Ntot : 0));
  y.off_drop = w;
  for (int32_t l = 0; l < y.h; ++l) w = align_up(w + sizeof(int32_t) * (size_t)y.drow[(size_t)l * (y.B + 1) + y.B]);
  y.total = std::max<size_t>(w, kAlign);
  return VC_OK;
}

// The last layout of the calling thread, reused while the shape (with its
// lengths) and the parameters are unchanged: a serving loop that prunes
// many requests of one shape, or queries sizes before pruning, plans once.
struct LayoutKey {
  int32_t B = 0, L = 0, Hq = 0, Hkv = 0, d = 0, W = 0;
  std::vector<int32_t> n;
  double retention = 0, m = 0;
  float tau = 0, mu = 0;
  int32_t h = 0, rank_mode = 0, v_out_fp32 = 0, schedule = 0, drop_all = 0, score_queries = 0;
  bool same(const vc_shape *s, const vc_params *p) const {
    return B == s->B && L == s->L && Hq == s->Hq && Hkv == s->Hkv && d == s->d && W == s->W &&
           std::equal(n.begin(), n.end(), s->n_vis) && retention == p->retention && m == p->m && tau == p->tau &&
           mu == p->mu && h == p->h && rank_mode == p->rank_mode && v_out_fp32 == p->v_out_fp32 &&
           schedule == p->schedule && drop_all == p->drop_all && score_queries == p->score_queries;
  }
  void set(const vc_shape *s, const vc_params *p) {
    B = s->B; L = s->L; Hq = s->Hq; Hkv = s->Hkv; d = s->d; W = s->W;
    n.assign(s->n_vis, s->n_vis + s->B);
    retention = p->retention; m = p->m; tau = p->tau; mu = p->mu; h = p->h; rank_mode = p->rank_mode;
    v_out_fp32 = p->v_out_fp32; schedule = p->schedule; drop_all = p->drop_all; score_queries = p->score_queries;
  }
};

struct LayoutCache {
  bool valid = false;
  LayoutKey key;
  Layout y;
};

// The layout of (shape, params): the cached one when the key matches, else
// a fresh one (cached when valid).  nullptr with *st set on an error.
const Layout *get_layout(const vc_shape *s, const vc_params *p, vc_status *st) {
  thread_local LayoutCache cache;
  *st = VC_OK;
  if (s && p && s->n_vis && s->B >= 1 && cache.valid && cache.key.B == s->B && cache.key.same(s, p))
    return &cache.y;
  Layout y;
  *st = make_layout(s, p, y);
  if (*st != VC_OK) return nullptr;
  cache.key.set(s, p);
  cache.y = std::move(y);
  cache.valid = true;
  return &cache.y;
}

}  // namespace

extern "C" {

void viscache_default_params(vc_params *p, double retention) {
  if (!p) return;
  p->retention = retention;
  p->h = 0;
  p->m = 0.75;
  p->tau = 1.0f;
  p->mu = 0.7f;
  p->rank_mode = VC_RANK_LAYER_HEAD;
  p->v_out_fp32 = 0;
  p->schedule = VC_SCHED_PARABOLIC;
  p->drop_all = 0;
  p->score_queries = VC_SCORE_WINDOW;
}

vc_status viscache_budget(const vc_shape *shape, const vc_params *params, int32_t *k,
                          int32_t *n_surv, int32_t *h_out) {
  if (!k || !n_surv) return VC_ERR_ARG;
  vc_status st;
  const Layout *yp = get_layout(shape, params, &st);
  if (!yp) return st;
  const Layout &y = *yp;
  std::memcpy(k, y.k.data(), sizeof(int32_t) * y.k.size());
  std::memcpy(n_surv, y.ns.data(), sizeof(int32_t) * y.ns.size());
  if (h_out) *h_out = y.h;
  return VC_OK;
}

vc_status viscache_out_rows(const vc_shape *shape, const vc_params *params, int64_t *rows) {
  if (!rows) return VC_ERR_ARG;
  vc_status st;
  const Layout *yp = get_layout(shape, params, &st);
  if (!yp) return st;
  const Layout &y = *yp;
  std::memcpy(rows, y.orow.data(), sizeof(int64_t) * y.orow.size());
  return VC_OK;
}

size_t viscache_prune_workspace_bytes(const vc_shape *shape, const vc_params *params) {
  vc_status st;
  const Layout *yp = get_layout(shape, params, &st);
  return yp ? yp->total : 0;
}

vc_status viscache_prune_score_offsets(const vc_shape *shape, const vc_params *params,
                                       size_t *scores_off, size_t *shared_off) {
  if (!scores_off || !shared_off) return VC_ERR_ARG;
  vc_status st;
  const Layout *yp = get_layout(shape, params, &st);
  if (!yp) return st;
  const Layout &y = *yp;
  *scores_off = y.off_S;
  *shared_off = y.mode == VC_RANK_GLOBAL ? y.off_gs : (size_t)-1;
  return VC_OK;
}

vc_status viscache_prune(const vc_shape *shape, const vc_params *params, const vc_prune_io *io,
                         void *workspace, size_t workspace_bytes, void *stream) {
  return viscache_prune_staged(shape, params, io, workspace, workspace_bytes, stream, nullptr);
}

vc_status viscache_prune_staged(const vc_shape *shape, const vc_params *params, const vc_prune_io *io,
                                void *workspace, size_t workspace_bytes, void *stream,
                                void *const *events) {
  vc_status st;
  const Layout *yp = get_layout(shape, params, &st);
  if (!yp) return st;
  const Layout &y = *yp;
  if (!io || !io->k_in || !io->v_in || !io->q_win || !io->k_out || !io->v_out || !io->idx_out)
    return VC_ERR_ARG;
  if (!workspace || workspace_bytes < y.total) return VC_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return VC_ERR_WORKSPACE;
  for (int32_t l = 0; l < y.Ls; ++l)
    if (y.Ntot > 0 && (!io->k_in[l] || !io->q_win[l])) return VC_ERR_ARG;
  if (y.prefill && y.W > 0 && y.Ntot > 0) {
    if (!io->k_text) return VC_ERR_ARG;
    for (int32_t l = 0; l < y.Ls; ++l)
      if (!io->k_text[l]) return VC_ERR_ARG;
  }
  for (int32_t l = 0; l < y.h; ++l) {
    const int64_t rows = y.orow[(size_t)l * (y.B + 1) + y.B];
    if (rows > 0 && (!io->v_in[l] || !io->k_out[l] || !io->v_out[l] || !io->idx_out[l]))
      return VC_ERR_ARG;
  }
  if (y.Ntot == 0) return VC_OK;  // nothing to score or keep

  uint8_t *ws = static_cast<uint8_t *>(workspace);
  hipStream_t hs = static_cast<hipStream_t>(stream);

  // Host copy of the plan.
  std::vector<uint8_t> blob(y.plan_bytes, 0);
  auto lp = reinterpret_cast<uint64_t *>(blob.data() + y.p_lp);
  for (int32_t l = 0; l < y.L; ++l) {
    lp[LP_K_IN * y.L + l] = reinterpret_cast<uint64_t>(io->k_in[l]);
    lp[LP_V_IN * y.L + l] = reinterpret_cast<uint64_t>(io->v_in[l]);
    lp[LP_Q * y.L + l] = reinterpret_cast<uint64_t>(io->q_win[l]);
    lp[LP_K_OUT * y.L + l] = l < y.h ? reinterpret_cast<uint64_t>(io->k_out[l]) : 0;
    lp[LP_V_OUT * y.L + l] = l < y.h ? reinterpret_cast<uint64_t>(io->v_out[l]) : 0;
    lp[LP_IDX * y.L + l] = l < y.h ? reinterpret_cast<uint64_t>(io->idx_out[l]) : 0;
    lp[LP_K_TEXT * y.L + l] = (y.prefill && io->k_text) ? reinterpret_cast<uint64_t>(io->k_text[l]) : 0;
  }
  size_t doff = y.off_drop;
  for (int32_t l = 0; l < y.h; ++l) {
    const size_t rows = (size_t)y.drow[(size_t)l * (y.B + 1) + y.B];
    uint64_t dp = reinterpret_cast<uint64_t>(ws + doff);
    if (io->drop_out && io->drop_out[l]) dp = reinterpret_cast<uint64_t>(io->drop_out[l]);
    lp[LP_DROP * y.L + l] = dp;
    doff = align_up(doff + sizeof(int32_t) * rows);
  }
  std::memcpy(blob.data() + y.p_toff, y.toff.data(), sizeof(int64_t) * y.toff.size());
  std::memcpy(blob.data() + y.p_orow, y.orow.data(), sizeof(int64_t) * y.orow.size());
  std::memcpy(blob.data() + y.p_drow, y.drow.data(), sizeof(int64_t) * y.drow.size());
  std::memcpy(blob.data() + y.p_nb, y.n.data(), sizeof(int32_t) * y.n.size());
  std::memcpy(blob.data() + y.p_kk, y.k.data(), sizeof(int32_t) * y.k.size());
  std::memcpy(blob.data() + y.p_ns, y.ns.data(), sizeof(int32_t) * y.ns.size());
  std::memcpy(blob.data() + y.p_fwoff, y.fwoff.data(), sizeof(int32_t) * y.fwoff.size());
  std::memcpy(blob.data() + y.p_fcnt, y.fcnt0.data(), sizeof(int32_t) * y.fcnt0.size());
  if (!y.fwjob.empty()) std::memcpy(blob.data() + y.p_fwjob, y.fwjob.data(), sizeof(int32_t) * y.fwjob.size());
  {
    // Fusion unit records: absolute row addresses, so the fusion kernel
    // needs one dependent load before its index loads.
    FuseUnit *fr = reinterpret_cast<FuseUnit *>(blob.data() + y.p_funit);
    const size_t vsz = y.vfp32 ? 4 : 2;
    for (size_t i = 0; i < y.funit.size(); ++i) {
      const int32_t u = y.funit[i];
      const int32_t g = u % y.Hkv, b = (u / y.Hkv) % y.B, l = u / (y.Hkv * y.B);
      const int32_t kk = y.k[(size_t)b * y.L + l], nn = y.n[b];
      const int32_t rr = y.ns[(size_t)b * y.L + l] - kk;
      const int64_t in_row = y.toff[b] * y.Hkv + (int64_t)g * nn;
      const int64_t out_row = y.orow[(size_t)l * (y.B + 1) + b] + (int64_t)g * kk;
      const int64_t drop_row = y.drow[(size_t)l * (y.B + 1) + b] + (int64_t)g * rr;
      FuseUnit f{};
      f.k_in = lp[LP_K_IN * y.L + l] + (uint64_t)(in_row * y.d * 2);
      f.v_in = lp[LP_V_IN * y.L + l] + (uint64_t)(in_row * y.d * 2);
      f.k_out = lp[LP_K_OUT * y.L + l] + (uint64_t)(out_row * y.d * 2);
      f.v_out = lp[LP_V_OUT * y.L + l] + (uint64_t)(out_row * y.d * vsz);
      f.kept = lp[LP_IDX * y.L + l] + (uint64_t)(out_row * 4);
      f.drop = lp[LP_DROP * y.L + l] + (uint64_t)(drop_row * 4);
      f.k = kk;
      f.r = rr;
      f.n = nn;
      fr[i] = f;
    }
  }

  PrunePlan pl{};
  pl.B = y.B; pl.L = y.L; pl.Hq = y.Hq; pl.Hkv = y.Hkv; pl.d = y.d; pl.W = y.W; pl.G = y.G;
  pl.R = y.R; pl.h = y.h; pl.Ls = y.Ls; pl.mode = y.mode; pl.v_fp32 = y.vfp32;
  pl.nqg = y.nqg; pl.nks = y.nks; pl.ncol = y.ncol; pl.nmax = y.nmax;
  pl.pwg = y.pwg;
  pl.nfunits = (int32_t)y.funit.size();
  pl.nfwg = y.nfwg;
  pl.sc = (float)(1.4426950408889634 / std::sqrt((double)y.d));
  pl.tc = (float)(1.4426950408889634 / (double)params->tau);
  pl.mu = params->mu;
  pl.Ntot = y.Ntot;
  pl.w_lp = (int32_t)(y.p_lp / 4);
  pl.w_toff = (int32_t)(y.p_toff / 4);
  pl.w_nb = (int32_t)(y.p_nb / 4);
  uint8_t *pb = ws + y.off_plan;
  pl.lp = reinterpret_cast<const uint64_t *>(pb + y.p_lp);
  pl.nb = reinterpret_cast<const int32_t *>(pb + y.p_nb);
  pl.toff = reinterpret_cast<const int64_t *>(pb + y.p_toff);
  pl.kk = reinterpret_cast<const int32_t *>(pb + y.p_kk);
  pl.ns = reinterpret_cast<const int32_t *>(pb + y.p_ns);
  pl.orow = reinterpret_cast<const int64_t *>(pb + y.p_orow);
  pl.drow = reinterpret_cast<const int64_t *>(pb + y.p_drow);
  pl.funit = reinterpret_cast<const FuseUnit *>(pb + y.p_funit);
  pl.fwoff = reinterpret_cast<const int32_t *>(pb + y.p_fwoff);
  pl.fwjob = reinterpret_cast<const int32_t *>(pb + y.p_fwjob);
  pl.fcnt = reinterpret_cast<int32_t *>(pb + y.p_fcnt);
  pl.qbf = reinterpret_cast<uint16_t *>(ws + y.off_qbf);
  pl.part = reinterpret_cast<float2 *>(ws + y.off_part);
  pl.pcol = reinterpret_cast<float *>(ws + y.off_part);
  pl.S = reinterpret_cast<float *>(ws + y.off_S);
  pl.gs = y.mode == VC_RANK_GLOBAL ? reinterpret_cast<float *>(ws + y.off_gs) : nullptr;

  auto mark = [&](int i) {
    return events && events[i] ? hipEventRecord(static_cast<hipEvent_t>(events[i]), hs) : hipSuccess;
  };
  // The plan's first chunk travels with the score statistics launch; only a
  // plan larger than one chunk needs upload launches for the rest.
  const size_t first = std::min(blob.size(), sizeof(uint32_t) * (size_t)kChunkWords);
  if (mark(0) != hipSuccess) return VC_ERR_HIP;
  if (blob.size() > first && launch_upload(pb + first, blob.data() + first, blob.size() - first, hs) != hipSuccess)
    return VC_ERR_HIP;
  if (mark(1) != hipSuccess) return VC_ERR_HIP;
  if ((y.prefill ? launch_pscore(pl, reinterpret_cast<uint32_t *>(pb), blob.data(), (uint32_t)(first / 4), hs)
                 : launch_score_stats(pl, reinterpret_cast<uint32_t *>(pb), blob.data(), (uint32_t)(first / 4), hs)) !=
      hipSuccess)
    return VC_ERR_HIP;
  if (mark(2) != hipSuccess) return VC_ERR_HIP;
  if ((y.prefill ? launch_pscore_reduce(pl, hs) : launch_score_colsum(pl, hs)) != hipSuccess) return VC_ERR_HIP;
  if (mark(3) != hipSuccess) return VC_ERR_HIP;
  if (y.mode == VC_RANK_GLOBAL && launch_score_global(pl, hs) != hipSuccess) return VC_ERR_HIP;
  if (mark(4) != hipSuccess) return VC_ERR_HIP;
  if (launch_select(pl, hs) != hipSuccess) return VC_ERR_HIP;
  if (mark(5) != hipSuccess) return VC_ERR_HIP;
  if (launch_fuse(pl, hs) != hipSuccess) return VC_ERR_HIP;
  if (mark(6) != hipSuccess) return VC_ERR_HIP;
  return VC_OK;
}

// ---- decode ----------------------------------------------------------------

namespace {

vc_status check_decode(const vc_decode_shape *s) {
  if (!s) return VC_ERR_ARG;
  if (s->B < 1 || s->L < 1 || s->Hq < 1 || s->Hkv < 1) return VC_ERR_SHAPE;
  if (s->Hq % s->Hkv != 0) return VC_ERR_SHAPE;
  if ((int64_t)s->L * s->B * s->Hq > INT32_MAX) return VC_ERR_SHAPE;
  if (s->Hq / s->Hkv > 16) return VC_ERR_UNSUPPORTED;
  if (s->d != 64 && s->d != 128) return VC_ERR_UNSUPPORTED;
  return VC_OK;
}

// Workspace layout of the decode calls: partial O and (max, sum) per piece
// (workgroup), then the (first piece, pieces) table of the units; the fused
// step adds one arrival counter per unit.
struct DecodeWs {
  size_t o, ml, pinfo, arrive, base, step;
};
DecodeWs decode_ws(int64_t units, int64_t nwg, int d) {
  const size_t slots = (size_t)nwg;
  DecodeWs w{};
  w.o = 0;
  w.ml = align_up(sizeof(float) * slots * 16 * (size_t)d);
  w.pinfo = w.ml + align_up(sizeof(float2) * slots * 16);
  w.arrive = w.pinfo + align_up(sizeof(int2) * (size_t)units);
  w.base = w.arrive;
  w.step = w.arrive + align_up(sizeof(uint32_t) * (size_t)units);
  return w;
}

// Plan of a decode call, or a status if it cannot run.
vc_status decode_plan(const vc_decode_shape *s, const vc_cache *c, const void *q, float *out, float scale,
                      int64_t max_rows, DecodePlan &p) {
  vc_status st = check_decode(s);
  if (st != VC_OK) return st;
  if (!c || !c->k_pool || !c->v_pool || !c->row_off || !c->cap || !c->len || !q || !out) return VC_ERR_ARG;
  if (!(scale > 0.f) || !std::isfinite(scale) || max_rows < 0) return VC_ERR_ARG;
  const int64_t units = (int64_t)s->L * s->B * s->Hkv;
  const int32_t nwg = decode_grid(units, max_rows);
  if (nwg < 1) return VC_ERR_UNSUPPORTED;
  p = DecodePlan{};
  p.B = s->B; p.L = s->L; p.Hq = s->Hq; p.Hkv = s->Hkv; p.d = s->d; p.G = s->Hq / s->Hkv;
  p.units = (int32_t)units;
  p.max_rows = (int32_t)std::min<int64_t>(max_rows, INT32_MAX);
  p.nwg = nwg;
  p.sc = scale * 1.4426950408889634f;
  p.k_pool = static_cast<const uint16_t *>(c->k_pool);
  p.v_pool = static_cast<const uint16_t *>(c->v_pool);
  p.row_off = c->row_off;
  p.cap = c->cap;
  p.len = c->len;
  p.q = static_cast<const uint16_t *>(q);
  p.out = out;
  return VC_OK;
}

void decode_bind_ws(DecodePlan &p, uint8_t *ws) {
  const DecodeWs w = decode_ws(p.units, p.nwg, p.d);
  p.part_o = reinterpret_cast<float *>(ws + w.o);
  p.part_ml = reinterpret_cast<float2 *>(ws + w.ml);
  p.pinfo = reinterpret_cast<int2 *>(ws + w.pinfo);
  p.arrive = reinterpret_cast<uint32_t *>(ws + w.arrive);
}
}  // namespace

size_t viscache_decode_workspace_bytes(const vc_decode_shape *s, int64_t max_rows) {
  if (check_decode(s) != VC_OK || max_rows < 0) return 0;
  const int64_t units = (int64_t)s->L * s->B * s->Hkv;
  const int32_t nwg = decode_grid(units, max_rows);
  if (nwg < 1) return 0;
  return decode_ws(units, nwg, s->d).base;
}

vc_status viscache_append_kv(const vc_decode_shape *s, const vc_cache *c, const void *k_new,
                             const void *v_new, void *stream) {
  vc_status st = check_decode(s);
  if (st != VC_OK) return st;
  if (!c || !c->k_pool || !c->v_pool || !c->row_off || !c->cap || !c->len || !k_new || !v_new)
    return VC_ERR_ARG;
  const int32_t units = s->L * s->B * s->Hkv;
  if (launch_append(units, s->d, static_cast<uint16_t *>(c->k_pool), static_cast<uint16_t *>(c->v_pool),
                    c->row_off, c->cap, c->len, static_cast<const uint16_t *>(k_new),
                    static_cast<const uint16_t *>(v_new), static_cast<hipStream_t>(stream)) != hipSuccess)
    return VC_ERR_HIP;
  return VC_OK;
}

vc_status viscache_decode_attn(const vc_decode_shape *s, const vc_cache *c, const void *q, float *out,
                               float scale, int64_t max_rows, void *workspace, size_t workspace_bytes,
                               void *stream) {
  DecodePlan p;
  const vc_status st = decode_plan(s, c, q, out, scale, max_rows, p);
  if (st != VC_OK) return st;
  const size_t need = viscache_decode_workspace_bytes(s, max_rows);
  if (!workspace || workspace_bytes < need) return VC_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return VC_ERR_WORKSPACE;
  decode_bind_ws(p, static_cast<uint8_t *>(workspace));
  p.arrive = nullptr;
  if (launch_decode(p, static_cast<hipStream_t>(stream)) != hipSuccess) return VC_ERR_HIP;
  return VC_OK;
}

size_t viscache_decode_step_workspace_bytes(const vc_decode_shape *s, int64_t max_rows) {
  if (check_decode(s) != VC_OK || max_rows < 0) return 0;
  const int64_t units = (int64_t)s->L * s->B * s->Hkv;
  const int32_t nwg = decode_grid(units, max_rows);
  if (nwg < 1) return 0;
  return decode_ws(units, nwg, s->d).step;
}

vc_status viscache_decode_step(const vc_decode_shape *s, const vc_cache *c, const void *k_new,
                               const void *v_new, const void *q, float *out, float scale, int64_t max_rows,
                               void *workspace, size_t workspace_bytes, void *stream) {
  DecodePlan p;
  const vc_status st = decode_plan(s, c, q, out, scale, max_rows, p);
  if (st != VC_OK) return st;
  if (!k_new || !v_new) return VC_ERR_ARG;
  const size_t need = viscache_decode_step_workspace_bytes(s, max_rows);
  if (!workspace || workspace_bytes < need) return VC_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return VC_ERR_WORKSPACE;
  decode_bind_ws(p, static_cast<uint8_t *>(workspace));
  p.k_pool_w = static_cast<uint16_t *>(c->k_pool);
  p.v_pool_w = static_cast<uint16_t *>(c->v_pool);
  p.len_w = c->len;
  p.k_new = static_cast<const uint16_t *>(k_new);
  p.v_new = static_cast<const uint16_t *>(v_new);
  if (launch_decode_step(p, static_cast<hipStream_t>(stream)) != hipSuccess) return VC_ERR_HIP;
  return VC_OK;
}

vc_status viscache_decode_step_q4(const vc_decode_shape *s, const vc_cache *c, const vc_qcache *qc,
                                  const void *k_new, const void *v_new, const void *q, float *out, float scale,
                                  int64_t max_rows, void *workspace, size_t workspace_bytes, void *stream) {
  DecodePlan p;
  const vc_status st = decode_plan(s, c, q, out, scale, max_rows, p);
  if (st != VC_OK) return st;
  if (!k_new || !v_new || !qc || !qc->k_codes || !qc->k_meta || !qc->v_codes || !qc->v_meta || !qc->qrow_off ||
      !qc->nq)
    return VC_ERR_ARG;
  if ((reinterpret_cast<uintptr_t>(qc->k_codes) | reinterpret_cast<uintptr_t>(qc->v_codes)) % 4 != 0 ||
      (reinterpret_cast<uintptr_t>(qc->k_meta) | reinterpret_cast<uintptr_t>(qc->v_meta)) % 8 != 0)
    return VC_ERR_ARG;
  const size_t need = viscache_decode_step_workspace_bytes(s, max_rows);
  if (!workspace || workspace_bytes < need) return VC_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return VC_ERR_WORKSPACE;
  decode_bind_ws(p, static_cast<uint8_t *>(workspace));
  p.k_pool_w = static_cast<uint16_t *>(c->k_pool);
  p.v_pool_w = static_cast<uint16_t *>(c->v_pool);
  p.len_w = c->len;
  p.k_new = static_cast<const uint16_t *>(k_new);
  p.v_new = static_cast<const uint16_t *>(v_new);
  p.qk = static_cast<const uint8_t *>(qc->k_codes);
  p.qv = static_cast<const uint8_t *>(qc->v_codes);
  p.qkm = static_cast<const float2 *>(qc->k_meta);
  p.qvm = static_cast<const float2 *>(qc->v_meta);
  p.qoff = qc->qrow_off;
  p.nq = qc->nq;
  if (launch_decode_step_q4(p, static_cast<hipStream_t>(stream)) != hipSuccess) return VC_ERR_HIP;
  return VC_OK;
}

vc_status viscache_decode_step_noalloc(const vc_decode_shape *s, const vc_cache *c, const void *k_new,
                                       const void *v_new, const void *q, float *out, float scale, int64_t max_rows,
                                       void *stream) {
  DecodePlan p;
  const vc_status st = decode_plan(s, c, q, out, scale, max_rows, p);
  if (st != VC_OK) return st;
  if (!k_new || !v_new) return VC_ERR_ARG;
  // The scratch holds the counters of at most kNoAllocUnits units and the
  // partial results of the launch's pieces (as in decode_ws, without the
  // two-call path's piece table).
  const size_t o_bytes = align_up(sizeof(float) * (size_t)p.nwg * 16 * (size_t)p.d);
  const size_t ml_bytes = align_up(sizeof(float2) * (size_t)p.nwg * 16);
  if (p.units > kNoAllocUnits || kNoAllocCounterBytes + o_bytes + ml_bytes > kNoAllocBytes)
    return VC_ERR_WORKSPACE;
  hipStream_t hs = static_cast<hipStream_t>(stream);
  uint8_t *ws = nullptr;
  if (noalloc_scratch(&ws, hs) != hipSuccess) return VC_ERR_HIP;
  p.arrive = reinterpret_cast<uint32_t *>(ws);
  p.part_o = reinterpret_cast<float *>(ws + kNoAllocCounterBytes);
  p.part_ml = reinterpret_cast<float2 *>(ws + kNoAllocCounterBytes + o_bytes);
  p.pinfo = nullptr;
  p.k_pool_w = static_cast<uint16_t *>(c->k_pool);
  p.v_pool_w = static_cast<uint16_t *>(c->v_pool);
  p.len_w = c->len;
  p.k_new = static_cast<const uint16_t *>(k_new);
  p.v_new = static_cast<const uint16_t *>(v_new);
  if (launch_decode_step(p, hs) != hipSuccess) return VC_ERR_HIP;
  return VC_OK;
}

size_t viscache_decode_plan_bytes(const vc_decode_shape *s, int64_t max_rows) {
  if (check_decode(s) != VC_OK || max_rows < 0) return 0;
  const int64_t units = (int64_t)s->L * s->B * s->Hkv;
  const int32_t nwg = decode_grid(units, max_rows);
  if (nwg < 1) return 0;
  return decode_plan_table_bytes(nwg);
}

vc_status viscache_decode_plan(const vc_decode_shape *s, const int32_t *cap, const int64_t *row_off,
                               const int32_t *len_hint, int64_t max_rows, void *plan, size_t plan_bytes) {
  vc_status st = check_decode(s);
  if (st != VC_OK) return st;
  if (!cap || !row_off || !plan || max_rows < 0) return VC_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(plan) % alignof(int32_t) != 0) return VC_ERR_ARG;
  const size_t need = viscache_decode_plan_bytes(s, max_rows);
  if (need == 0) return VC_ERR_UNSUPPORTED;
  if (plan_bytes < need) return VC_ERR_WORKSPACE;
  const int64_t units = (int64_t)s->L * s->B * s->Hkv;
  return (vc_status)decode_plan_build((int32_t)units, cap, row_off, len_hint, max_rows, decode_grid(units, max_rows),
                                      s->d, static_cast<int32_t *>(plan));
}

vc_status viscache_decode_step_planned(const vc_decode_shape *s, const vc_cache *c, const vc_qcache *qc,
                                       const void *plan, size_t plan_bytes, const void *k_new, const void *v_new,
                                       const void *q, float *out, float scale, int64_t max_rows, void *workspace,
                                       size_t workspace_bytes, void *stream) {
  DecodePlan p;
  const vc_status st = decode_plan(s, c, q, out, scale, max_rows, p);
  if (st != VC_OK) return st;
  if (!k_new || !v_new || !plan) return VC_ERR_ARG;
  if (reinterpret_cast<uintptr_t>(plan) % 16 != 0 || plan_bytes < decode_plan_table_bytes(p.nwg)) return VC_ERR_ARG;
  if (qc) {
    if (!qc->k_codes || !qc->k_meta || !qc->v_codes || !qc->v_meta || !qc->qrow_off || !qc->nq) return VC_ERR_ARG;
    if ((reinterpret_cast<uintptr_t>(qc->k_codes) | reinterpret_cast<uintptr_t>(qc->v_codes)) % 4 != 0 ||
        (reinterpret_cast<uintptr_t>(qc->k_meta) | reinterpret_cast<uintptr_t>(qc->v_meta)) % 8 != 0)
      return VC_ERR_ARG;
  }
  const size_t need = viscache_decode_step_workspace_bytes(s, max_rows);
  if (!workspace || workspace_bytes < need) return VC_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0) return VC_ERR_WORKSPACE;
  decode_bind_ws(p, static_cast<uint8_t *>(workspace));
  p.k_pool_w = static_cast<uint16_t *>(c->k_pool);
  p.v_pool_w = static_cast<uint16_t *>(c->v_pool);
  p.len_w = c->len;
  p.k_new = static_cast<const uint16_t *>(k_new);
  p.v_new = static_cast<const uint16_t *>(v_new);
  p.plan = static_cast<const int32_t *>(plan);
  if (qc) {
    p.qk = static_cast<const uint8_t *>(qc->k_codes);
    p.qv = static_cast<const uint8_t *>(qc->v_codes);
    p.qkm = static_cast<const float2 *>(qc->k_meta);
    p.qvm = static_cast<const float2 *>(qc->v_meta);
    p.qoff = qc->qrow_off;
    p.nq = qc->nq;
  }
  if (launch_decode_planned(p, qc != nullptr, static_cast<hipStream_t>(stream)) != hipSuccess) return VC_ERR_HIP;
  return VC_OK;
}

vc_status viscache_quantize_rows(int32_t d, int64_t rows, const void *src, void *codes, void *meta, void *stream) {
  if (d != 64 && d != 128) return VC_ERR_UNSUPPORTED;
  if (rows < 0) return VC_ERR_ARG;
  if (rows == 0) return VC_OK;
  if (!src || !codes || !meta || (reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(codes)) % 16 != 0 ||
      reinterpret_cast<uintptr_t>(meta) % 8 != 0)
    return VC_ERR_ARG;
  if (rows * (d / 32) > (int64_t)INT32_MAX * 256) return VC_ERR_UNSUPPORTED;
  if (launch_quant_rows(d, rows, static_cast<const uint16_t *>(src), static_cast<uint8_t *>(codes),
                        static_cast<float2 *>(meta), static_cast<hipStream_t>(stream)) != hipSuccess)
    return VC_ERR_HIP;
  return VC_OK;
}

const char *viscache_strerror(vc_status s) {
  switch (s) {
    case VC_OK: return "ok";
    case VC_ERR_ARG: return "invalid argument";
    case VC_ERR_SHAPE: return "invalid shape";
    case VC_ERR_BUDGET: return "no valid budget for these retention parameters";
    case VC_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
    case VC_ERR_UNSUPPORTED: return "shape not supported by the kernels";
    case VC_ERR_HIP: return "HIP launch failed";
  }
  return "unknown status";
}

}  // extern "C"
