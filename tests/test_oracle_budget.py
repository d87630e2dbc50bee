"""Pins for the oracle's layer budgets (Sec. 3.2 Eq. (parabolic) and its
normalisation; Sec. 4 Implementation Details for RR = p*q*(h/L)*m and the
defaults; Appendix B Algorithm 1 Step 1 for the top-q cut)."""
import json
import math
import os

import numpy as np
import pytest

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def test_parabola_endpoints_from_paper(orc):
    # With h = 2 and m = 0.75 the normalisation target h*m = 1.5 equals the raw
    # sum 1 + 0.5, so the normalised proportions are the raw ones.
    g = GOLD["parabola_endpoints"]
    r = orc.budget(L=2, n=1000, rr=0.375, h=2, m=0.75)
    assert r["b"][0] == g["b_first"]
    assert r["b"][1] == g["b_last"]


@pytest.mark.parametrize("h", [2, 3, 5, 21, 48, 60])
def test_endpoint_ratio_and_concave_decay(orc, h):
    # b_1 / b_h = 1 / 0.5 for every h (no clipping at m = 0.75), and the decay
    # is slow early and steep late: successive drops grow.
    r = orc.budget(L=80, n=4096, rr=0.01, h=h, m=0.75)
    b = r["b"][:h]
    assert b[-1] / b[0] == pytest.approx(GOLD["parabola_endpoints"]["b_last"], rel=1e-14)
    drops = -np.diff(b)
    assert np.all(drops > 0)
    assert np.all(np.diff(drops) > 0)


@pytest.mark.parametrize("L,h,m", [(4, 3, 0.75), (28, 21, 0.75), (80, 60, 0.75), (28, 21, 0.95),
                                   (28, 28, 1.0), (10, 2, 0.6), (64, 48, 0.9)])
def test_normalisation_target(orc, L, h, m):
    # sum_{l<=h} b_l = h*m, every proportion in (0, 1], zero beyond h.
    r = orc.budget(L=L, n=5000, rr=0.9 * (h / L) * m, h=h, m=m)
    b = r["b"]
    assert b[:h].sum() == pytest.approx(h * m, rel=1e-12)
    assert np.all(b[:h] > 0) and np.all(b[:h] <= 1.0)
    assert np.all(b[h:] == 0)


def test_defaults_and_truncation_64(orc):
    d = GOLD["defaults"]
    t = GOLD["truncation_64_layers"]
    r = orc.budget(L=t["L"], n=1000, rr=0.2)
    assert r["h"] == t["h"] == round(d["h_over_L"] * t["L"])
    assert orc.budget(L=28, n=10, rr=0.2)["h"] == 21
    assert orc.budget(L=80, n=10, rr=0.2)["h"] == 60
    assert orc.budget(L=4, n=10, rr=0.2)["h"] == 3


def test_retention_composition_from_paper(orc):
    # RR = p*q*(h/L)*m.  This build has no frame filter (p = 1), so the token
    # ratio it derives from RR must be p*q of the paper's rows.
    g = GOLD["retention_examples"]
    for row in g["rows"]:
        rr = row["p"] * row["q"] * g["h_over_L"] * g["m"]
        assert round(100 * rr) == row["rr_percent"]
        r = orc.budget(L=64, n=10000, rr=rr, m=g["m"])
        assert r["q"] == pytest.approx(row["p"] * row["q"], rel=1e-12)


SWEEP_L = [2, 3, 4, 8, 28, 36, 64, 80]
SWEEP_N = [0, 1, 7, 64, 512, 3136, 12544]
SWEEP_RR = [0.05, 0.19, 0.22, 0.25, 0.28, 0.40, 0.5625]


@pytest.mark.parametrize("L", SWEEP_L)
def test_integer_budget_invariants(orc, L):
    for n in SWEEP_N:
        for rr in SWEEP_RR:
            h = int(math.floor(0.75 * L + 0.5))
            if h < 2 or rr / ((h / L) * 0.75) > 1 + 1e-9:
                with pytest.raises(ValueError):
                    orc.budget(L=L, n=n, rr=rr)
                continue
            r = orc.budget(L=L, n=n, rr=rr)
            k, ns = r["k"], r["n_surv"]
            T = math.floor(rr * L * n + 0.5)
            assert int(k.sum()) == T  # totals match the stated overall retention
            assert np.all(np.diff(k) <= 0)  # non-increasing with depth
            assert np.all(k[h:] == 0)  # layers past h fully evicted
            assert 0 <= k[0] <= ns <= n
            # largest-remainder apportionment: within one token of the exact share
            b = r["b"][:h]
            x = T * b / b.sum()
            assert np.all(np.abs(k[:h] - x) < 1.0)


def test_keep_all(orc):
    for L, n in [(2, 5), (4, 512), (28, 3136)]:
        r = orc.budget(L=L, n=n, rr=1.0, h=L, m=1.0)
        assert np.all(r["k"] == n)
        assert r["n_surv"] == n and r["q"] == 1.0


def test_remainder_ties_go_to_lower_layer(orc):
    # m = 1 clips every proportion to 1, so all layers get the same share
    # T/h = 14/3 and the two leftover tokens go to layers 1 and 2.
    r = orc.budget(L=4, n=7, rr=0.5, h=3, m=1.0)
    assert list(r["k"]) == [5, 5, 4, 0]


def test_water_filling_clips_at_one(orc):
    # m = 0.95 asks for more than the scaled parabola can give below 1.
    r = orc.budget(L=28, n=3136, rr=0.5, h=21, m=0.95)
    b = r["b"][:21]
    assert b[0] == 1.0 and np.sum(b == 1.0) >= 2
    free = b[b < 1.0]
    assert b.sum() == pytest.approx(21 * 0.95, rel=1e-12)
    assert np.all(np.diff(free) < 0)


@pytest.mark.parametrize("kw", [dict(L=28, n=100, rr=0.6), dict(L=28, n=100, rr=0.2, h=1),
                                dict(L=28, n=100, rr=0.2, h=29), dict(L=28, n=100, rr=0.0),
                                dict(L=28, n=100, rr=0.2, m=0.0), dict(L=1, n=100, rr=0.2),
                                dict(L=28, n=-1, rr=0.2)])
def test_invalid_parameters(orc, kw):
    with pytest.raises(ValueError):
        orc.budget(**kw)


def test_workload_budgets(orc, sg):
    # The five seeded workloads: the per-sequence totals equal round(RR*L*n).
    for w in sg.WORKLOADS.values():
        for n in w.n_vis():
            r = orc.budget(L=w.L, n=int(n), rr=w.retention)
            assert int(r["k"].sum()) == math.floor(w.retention * w.L * int(n) + 0.5)


# ---- alternative schedules of the budget ablation and the fuse-all reading ----

def test_fixed_schedule_is_uniform(orc):
    # "Uniform budget per layer": every proportion equals m, and the integer
    # budgets of layers 1..h differ by at most one token.
    for L, n, rr in [(28, 3136, 0.28), (80, 8192, 0.22), (4, 512, 0.25)]:
        r = orc.budget(L=L, n=n, rr=rr, schedule=orc.SCHEDULES["fixed"])
        h = r["h"]
        assert np.allclose(r["b"][:h], 0.75, rtol=0, atol=1e-15)
        k = r["k"][:h]
        assert k.max() - k.min() <= 1
        assert k.sum() == math.floor(rr * L * n + 0.5)


@pytest.mark.parametrize("h", [3, 21, 60])
def test_arithmetic_schedule_is_linear_from_one_to_half(orc, h):
    # Endpoints 1 and 1/2 make the mean exactly 0.75, so at m = 0.75 the
    # normalisation leaves the line unchanged: equal steps, b_1 = 1, b_h = 1/2.
    r = orc.budget(L=80, n=8192, rr=0.01, h=h, m=0.75, schedule=orc.SCHEDULES["arithmetic"])
    b = r["b"][:h]
    assert b[0] == pytest.approx(1.0, abs=1e-15) and b[-1] == pytest.approx(0.5, abs=1e-15)
    steps = np.diff(b)
    assert np.allclose(steps, steps[0], rtol=0, atol=1e-14) and steps[0] < 0
    # Integer budgets follow: successive differences vary by at most one token
    # around a constant step.
    r = orc.budget(L=28, n=3136, rr=0.28, schedule=orc.SCHEDULES["arithmetic"])
    dk = np.diff(r["k"][:r["h"]].astype(np.int64))
    assert dk.max() - dk.min() <= 2 and np.all(dk <= 0)


def test_geometric_schedule_water_fills_four_blocks(orc):
    # Four equal depth blocks with ratio 1/2 give raw 1, 1/2, 1/4, 1/8 (mean
    # 15/32 < 0.75): scaling to the mean 0.75 holds blocks 0 and 1 at 1 and
    # leaves 2/3 and 1/3 for blocks 2 and 3 (the sum is h*m exactly).
    h = 20
    r = orc.budget(L=28, n=4000, rr=0.05, h=h, m=0.75, schedule=orc.SCHEDULES["geometric"])
    b = r["b"][:h].reshape(4, 5)
    for j, want in enumerate([1.0, 1.0, 2.0 / 3.0, 1.0 / 3.0]):
        assert np.allclose(b[j], want, rtol=0, atol=1e-15)
    assert b.sum() == pytest.approx(h * 0.75, rel=1e-14)


@pytest.mark.parametrize("schedule", ["parabolic", "fixed", "arithmetic", "geometric"])
def test_schedules_keep_the_integer_invariants(orc, schedule):
    s = orc.SCHEDULES[schedule]
    for L in [2, 4, 28, 80]:
        for n in [0, 1, 64, 3136, 12544]:
            for rr in [0.05, 0.19, 0.28]:
                try:
                    r = orc.budget(L=L, n=n, rr=rr, schedule=s)
                except ValueError:
                    continue
                k, h = r["k"], r["h"]
                assert k.sum() == math.floor(rr * L * n + 0.5)
                assert np.all(np.diff(k[:h].astype(np.int64)) <= 0)  # non-increasing
                assert np.all(k[h:] == 0)
                assert k.max() <= r["n_surv"] <= n


def test_drop_all_fuses_every_non_kept_token(orc):
    # drop_all: the survivor count is n, whatever q, and the kept budgets are
    # those of the default reading.
    for L, n, rr in [(28, 3136, 0.28), (4, 512, 0.25), (28, 12544, 0.19)]:
        a = orc.budget(L=L, n=n, rr=rr)
        b = orc.budget(L=L, n=n, rr=rr, drop_all=True)
        assert b["n_surv"] == n and a["n_surv"] < n
        assert np.array_equal(a["k"], b["k"])
