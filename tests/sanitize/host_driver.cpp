// host_driver.cpp -- runs the host code of libviscache (argument checks,
// budgets, plan layout and packing, decode planning) and every oracle
// function under the address and undefined-behaviour sanitizers, on the CPU.
// Device pointers are fake, well-aligned addresses that the host code only
// stores; the launchers are stubs (launch_stubs.cpp) that report a failed
// launch, so a call that passes every host check returns VC_ERR_HIP.
//
// Usage: host_driver CASES_FILE.  Each line of CASES_FILE is one prune
// shape: B L Hq Hkv d W rr h m rank_mode v_out_fp32 schedule drop_all
// score_queries n_0 .. n_{B-1}.  Prints "case <i> <status>" per line, then
// "oracle ok" and "done"; exits non-zero on any inconsistency.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <fstream>
#include <sstream>
#include <string>
#include <vector>

#include "../../include/viscache.h"

extern "C" {
#include "../../oracle/oracle.h"
}

static int g_fail = 0;
#define CHECK(c, ...)                                   \
  do {                                                  \
    if (!(c)) {                                         \
      std::fprintf(stderr, "FAIL %s:%d: ", __FILE__, __LINE__); \
      std::fprintf(stderr, __VA_ARGS__);                \
      std::fprintf(stderr, "\n");                       \
      ++g_fail;                                         \
    }                                                   \
  } while (0)

static void *fake(uintptr_t i) { return reinterpret_cast<void *>((uintptr_t)0x7f0000000000ull + (i << 20)); }

static int run_case(int idx, const std::vector<double> &v) {
  const int B = (int)v[0], L = (int)v[1], Hq = (int)v[2], Hkv = (int)v[3], d = (int)v[4], W = (int)v[5];
  std::vector<int32_t> n(B);
  for (int b = 0; b < B; ++b) n[b] = (int32_t)v[14 + b];
  vc_shape s{B, L, Hq, Hkv, d, W, n.data()};
  vc_params p;
  viscache_default_params(&p, v[6]);
  p.h = (int32_t)v[7];
  p.m = v[8];
  p.rank_mode = (int32_t)v[9];
  p.v_out_fp32 = (int32_t)v[10];
  p.schedule = (int32_t)v[11];
  p.drop_all = (int32_t)v[12];
  p.score_queries = (int32_t)v[13];
  std::vector<int32_t> k((size_t)B * L), ns((size_t)B * L);
  int32_t h = 0;
  const vc_status st = viscache_budget(&s, &p, k.data(), ns.data(), &h);
  std::printf("case %d %d\n", idx, (int)st);
  if (st != VC_OK) {
    CHECK(viscache_prune_workspace_bytes(&s, &p) == 0, "case %d: workspace size of a refused shape", idx);
    return 0;
  }
  // Budgets against the oracle, sequence by sequence.
  for (int b = 0; b < B; ++b) {
    std::vector<int32_t> kk(L);
    int32_t nsv = 0, ho = 0;
    const int rc = orc_budget(L, n[b], p.retention, p.h, p.m, p.schedule, p.drop_all, kk.data(), &nsv, &ho,
                              nullptr, nullptr);
    CHECK(rc == 0, "case %d: oracle refuses b=%d", idx, b);
    CHECK(ho == h, "case %d: h %d vs %d", idx, h, ho);
    for (int l = 0; l < L; ++l) {
      CHECK(kk[l] == k[(size_t)b * L + l], "case %d: k b=%d l=%d", idx, b, l);
      CHECK(nsv == ns[(size_t)b * L + l], "case %d: n_surv b=%d", idx, b);
    }
  }
  // Output rows: per layer, prefix sums of Hkv * k over sequences.
  std::vector<int64_t> rows((size_t)L * (B + 1));
  CHECK(viscache_out_rows(&s, &p, rows.data()) == VC_OK, "case %d: out_rows", idx);
  for (int l = 0; l < L; ++l) {
    CHECK(rows[(size_t)l * (B + 1)] == 0, "case %d: first row offset", idx);
    for (int b = 0; b < B; ++b)
      CHECK(rows[(size_t)l * (B + 1) + b + 1] - rows[(size_t)l * (B + 1) + b] == (int64_t)Hkv * k[(size_t)b * L + l],
            "case %d: out rows l=%d b=%d", idx, l, b);
  }
  const size_t ws = viscache_prune_workspace_bytes(&s, &p);
  CHECK(ws > 0 && ws % 256 == 0, "case %d: workspace size %zu", idx, ws);
  size_t so = 0, go = 0;
  CHECK(viscache_prune_score_offsets(&s, &p, &so, &go) == VC_OK && so < ws, "case %d: score offsets", idx);
  // The whole planning path up to the first launch, with fake buffers.
  std::vector<const void *> kin(L), vin(L), kt(L);
  std::vector<const float *> qw(L);
  std::vector<void *> ko(L), vo(L);
  std::vector<int32_t *> io_idx(L), io_drop(L);
  for (int l = 0; l < L; ++l) {
    kin[l] = fake(8 * l);
    vin[l] = fake(8 * l + 1);
    qw[l] = static_cast<const float *>(fake(8 * l + 2));
    ko[l] = fake(8 * l + 3);
    vo[l] = fake(8 * l + 4);
    io_idx[l] = static_cast<int32_t *>(fake(8 * l + 5));
    io_drop[l] = static_cast<int32_t *>(fake(8 * l + 6));
    kt[l] = fake(8 * l + 7);
  }
  vc_prune_io io{kin.data(), vin.data(), qw.data(), ko.data(), vo.data(), io_idx.data(), io_drop.data(), kt.data()};
  int64_t ntot = 0;
  for (int b = 0; b < B; ++b) ntot += n[b];
  void *wsp = fake(1u << 20);
  const vc_status pr = viscache_prune(&s, &p, &io, wsp, ws, nullptr);
  CHECK(pr == (ntot > 0 ? VC_ERR_HIP : VC_OK), "case %d: prune status %d", idx, (int)pr);
  CHECK(viscache_prune(&s, &p, &io, wsp, ws - 1, nullptr) == VC_ERR_WORKSPACE, "case %d: short workspace", idx);
  CHECK(viscache_prune(&s, &p, nullptr, wsp, ws, nullptr) == VC_ERR_ARG, "case %d: null io", idx);
  // Decode planning over caches of this shape (the visual rows, the window
  // and 128 generated rows).
  int32_t nmax = 0;
  for (int b = 0; b < B; ++b) nmax = n[b] > nmax ? n[b] : nmax;
  vc_decode_shape ds{B, L, Hq, Hkv, d};
  const int64_t max_rows = (int64_t)nmax + W + 128;
  const size_t dws = viscache_decode_step_workspace_bytes(&ds, max_rows);
  const size_t aws = viscache_decode_workspace_bytes(&ds, max_rows);
  vc_cache c{fake(900), fake(901), static_cast<const int64_t *>(fake(902)), static_cast<const int32_t *>(fake(903)),
             static_cast<int32_t *>(fake(904))};
  if (Hq / Hkv <= 16) {
    CHECK(dws > 0 && aws > 0 && aws <= dws, "case %d: decode workspace %zu %zu", idx, aws, dws);
    CHECK(viscache_decode_step(&ds, &c, fake(905), fake(906), fake(907), static_cast<float *>(fake(908)),
                               0.088f, max_rows, fake(909), dws, nullptr) == VC_ERR_HIP,
          "case %d: decode step", idx);
    CHECK(viscache_decode_attn(&ds, &c, fake(907), static_cast<float *>(fake(908)), 0.088f, max_rows, fake(909),
                               aws, nullptr) == VC_ERR_HIP,
          "case %d: decode attn", idx);
    CHECK(viscache_decode_step(&ds, &c, fake(905), fake(906), fake(907), static_cast<float *>(fake(908)),
                               0.088f, max_rows, fake(909), dws - 1, nullptr) == VC_ERR_WORKSPACE,
          "case %d: decode short workspace", idx);
    // Allocation-free step: refused beyond its scratch, else it reaches the
    // (stub) scratch lookup.
    const bool fits = (int64_t)L * B * Hkv <= VC_DECODE_NOALLOC_UNITS &&
                      dws <= (size_t)VC_DECODE_NOALLOC_BYTES - 4 * (size_t)VC_DECODE_NOALLOC_UNITS;
    const vc_status na = viscache_decode_step_noalloc(&ds, &c, fake(905), fake(906), fake(907),
                                                      static_cast<float *>(fake(908)), 0.088f, max_rows, nullptr);
    CHECK(na == VC_ERR_HIP || (!fits && na == VC_ERR_WORKSPACE), "case %d: decode noalloc status %d", idx, (int)na);
    // Piece table of caches holding the retained visual rows, the window and
    // 128 generated rows per unit (every fifth unit empty), then the planned
    // step up to its (stub) launch.
    const int64_t units = (int64_t)L * B * Hkv;
    std::vector<int32_t> cap((size_t)units);
    std::vector<int64_t> off((size_t)units);
    int64_t o = 0;
    for (int64_t u = 0; u < units; ++u) {
      const int b = (int)((u / Hkv) % B);
      cap[u] = u % 5 == 4 ? 0 : (int32_t)(n[b] * p.retention) + W + 128;
      off[u] = o;
      o += cap[u];
    }
    const size_t pb = viscache_decode_plan_bytes(&ds, max_rows);
    CHECK(pb > 0, "case %d: plan bytes", idx);
    std::vector<int32_t> plan(pb / 4 + 1);
    std::vector<int32_t> hint((size_t)units);
    for (int64_t u = 0; u < units; ++u) hint[u] = cap[u] > 128 ? cap[u] - 128 : 0;
    CHECK(viscache_decode_plan(&ds, cap.data(), off.data(), nullptr, max_rows, plan.data(), pb) == VC_OK,
          "case %d: plan without hint", idx);
    const vc_status ps = viscache_decode_plan(&ds, cap.data(), off.data(), hint.data(), max_rows, plan.data(), pb);
    CHECK(ps == VC_OK, "case %d: plan status %d", idx, (int)ps);
    if (ps == VC_OK) {
      // Every unit's min(cap, max_rows) rows are covered once, in order, by
      // its pieces, whose slots are p0 .. p0 + np - 1.
      const int32_t nwg = plan[2], P = plan[5];
      CHECK(plan[1] == units && P >= units && P <= nwg, "case %d: plan header", idx);
      std::vector<int64_t> covered((size_t)units, 0), seen((size_t)units, 0);
      for (int32_t i = 0; i < nwg; ++i) {
        const int32_t *r = plan.data() + 8 + 8 * (size_t)i;
        if (i >= P) {
          CHECK(r[0] == -1, "case %d: record %d past the pieces", idx, i);
          continue;
        }
        const int32_t j = r[1] & 0xFFFF, npc = r[1] >> 16;
        CHECK(r[0] >= 0 && r[0] < units && j < npc && r[3] <= r[5] && r[5] <= r[4], "case %d: record %d", idx, i);
        if (!(r[0] >= 0 && r[0] < units)) continue;
        covered[r[0]] += r[4] - r[3];
        seen[r[0]] += 1;
        CHECK(r[6] == (int32_t)(uint32_t)off[r[0]] && r[7] == (int32_t)(off[r[0]] >> 32), "case %d: offset", idx);
      }
      for (int64_t u = 0; u < units; ++u) {
        const int64_t want = cap[u] < max_rows ? cap[u] : max_rows;
        CHECK(covered[u] == want && seen[u] >= 1, "case %d: unit %lld covered %lld of %lld", idx, (long long)u,
              (long long)covered[u], (long long)want);
      }
    }
    CHECK(viscache_decode_plan(&ds, cap.data(), off.data(), hint.data(), max_rows, plan.data(), pb - 4) ==
              VC_ERR_WORKSPACE,
          "case %d: short plan buffer", idx);
    if (units > 1 && cap[0] > 0) {
      std::vector<int64_t> bad(off);
      bad[1] = bad[0] + cap[0] - 1;  // overlaps unit 0's block
      if (cap[1] > 0)
        CHECK(viscache_decode_plan(&ds, cap.data(), bad.data(), nullptr, max_rows, plan.data(), pb) == VC_ERR_ARG,
              "case %d: overlapping blocks accepted", idx);
    }
    CHECK(viscache_decode_step_planned(&ds, &c, nullptr, fake(910), pb, fake(905), fake(906), fake(907),
                                       static_cast<float *>(fake(908)), 0.088f, max_rows, fake(909), dws,
                                       nullptr) == VC_ERR_HIP,
          "case %d: planned step", idx);
    CHECK(viscache_decode_step_planned(&ds, &c, nullptr, fake(910), pb - 32, fake(905), fake(906), fake(907),
                                       static_cast<float *>(fake(908)), 0.088f, max_rows, fake(909), dws,
                                       nullptr) == VC_ERR_ARG,
          "case %d: planned step, short table", idx);
  } else {
    CHECK(dws == 0, "case %d: decode group above 16 accepted", idx);
    CHECK(viscache_decode_plan_bytes(&ds, max_rows) == 0, "case %d: plan bytes for a group above 16", idx);
  }
  return 0;
}

// Deterministic inputs for the oracle functions.
static uint64_t g_state = 0x9E3779B97F4A7C15ull;
static double uni() {
  g_state = g_state * 6364136223846793005ull + 1442695040888963407ull;
  return (double)(g_state >> 11) * (1.0 / 9007199254740992.0);
}
static uint16_t bf16_of(double x) {
  float f = (float)x;
  uint32_t u;
  std::memcpy(&u, &f, 4);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

static void run_oracle() {
  // Budgets over a sweep, every schedule, both survivor rules.
  for (int L : {2, 3, 4, 28, 80})
    for (int n : {0, 1, 7, 512, 3136, 23040})
      for (double rr : {0.05, 0.19, 0.28, 0.5625, 1.0})
        for (int sched = 0; sched < 4; ++sched)
          for (int da = 0; da < 2; ++da) {
            std::vector<int32_t> k(L);
            std::vector<double> b(L);
            int32_t ns = 0, h = 0;
            double q = 0;
            const int rc = orc_budget(L, n, rr, rr == 1.0 ? L : 0, rr == 1.0 ? 1.0 : 0.75, sched, da, k.data(), &ns,
                                      &h, b.data(), &q);
            if (rc == 0) {
              long long sum = 0;
              for (int l = 0; l < L; ++l) sum += k[l];
              CHECK(sum == (long long)std::floor(rr * L * n + 0.5), "oracle budget sum L=%d n=%d", L, n);
            }
          }
  // One small unit through every function.
  const int n = 300, d = 64, R = 24, T = 7, G = 3;
  std::vector<uint16_t> K((size_t)n * d), V((size_t)n * d), Kt((size_t)T * d);
  std::vector<float> Q((size_t)R * d), Qp((size_t)G * (n + T) * d);
  for (auto &x : K) x = bf16_of(2.0 * uni() - 1.0);
  for (auto &x : V) x = bf16_of(4.0 * uni() - 2.0);
  for (auto &x : Kt) x = bf16_of(2.0 * uni() - 1.0);
  for (auto &x : Q) x = (float)(3.0 * uni() - 1.5);
  for (auto &x : Qp) x = (float)(3.0 * uni() - 1.5);
  std::vector<double> S(n), Sp(n), St(T);
  orc_scores_unit(n, d, R, K.data(), Q.data(), S.data());
  double tot = 0;
  for (double x : S) tot += x;
  CHECK(std::fabs(tot - R) < 1e-9 * R, "oracle scores sum %g", tot);
  orc_scores_unit_prefill(n, T, d, G, K.data(), Kt.data(), Qp.data(), Sp.data(), St.data());
  std::vector<float> s32(n);
  for (int v = 0; v < n; ++v) s32[v] = (float)S[v];
  const int k = 90, nsv = 160;
  std::vector<int32_t> kept(k), drop(nsv - k);
  orc_select(n, s32.data(), k, nsv, kept.data(), drop.data());
  std::vector<uint16_t> Ko((size_t)k * d);
  orc_gather(d, k, kept.data(), K.data(), Ko.data());
  std::vector<double> Vo((size_t)k * d);
  orc_fuse(d, k, nsv - k, V.data(), kept.data(), drop.data(), 1.0, 0.7, Vo.data());
  orc_fuse(d, k, 0, V.data(), kept.data(), nullptr, 1.0, 0.7, Vo.data());
  orc_fuse(d, 0, nsv - k, V.data(), nullptr, drop.data(), 1.0, 0.7, Vo.data());
  std::vector<double> o(d);
  orc_attend(d, n, K.data(), K.data(), V.data(), 0.125, o.data());
  orc_attend(d, 0, K.data(), K.data(), V.data(), 0.125, o.data());
  std::vector<uint8_t> codes((size_t)n * d / 2);
  std::vector<float> meta((size_t)n * (d / 32) * 2);
  std::vector<uint16_t> back((size_t)n * d);
  orc_quant_rows(n, d, V.data(), codes.data(), meta.data());
  orc_dequant_rows(n, d, codes.data(), meta.data(), back.data());
  std::vector<int32_t> kp(k), dp(nsv - k);
  std::vector<uint16_t> Kp((size_t)k * d);
  std::vector<double> Vp((size_t)k * d);
  std::vector<float> S32(n);
  orc_prune_unit(n, d, R, K.data(), V.data(), Q.data(), k, nsv, 1.0, 0.7, kp.data(), dp.data(), Kp.data(),
                 Vp.data(), S32.data());
  CHECK(std::memcmp(kp.data(), kept.data(), sizeof(int32_t) * k) == 0, "oracle prune_unit kept set");
  std::printf("oracle ok\n");
}

int main(int argc, char **argv) {
  if (argc != 2) {
    std::fprintf(stderr, "usage: %s CASES_FILE\n", argv[0]);
    return 2;
  }
  std::ifstream in(argv[1]);
  std::string line;
  int idx = 0;
  while (std::getline(in, line)) {
    if (line.empty()) continue;
    std::istringstream ss(line);
    std::vector<double> v;
    double x;
    while (ss >> x) v.push_back(x);
    if (v.size() < 15 || v.size() != 14 + (size_t)v[0]) {
      std::fprintf(stderr, "bad case line %d\n", idx);
      return 2;
    }
    run_case(idx++, v);
  }
  run_oracle();
  std::printf("done %d cases, %d failures\n", idx, g_fail);
  return g_fail ? 1 : 0;
}
