"""Pins for the oracle's selection (Alg. 1 Steps 1 and 3: one ranking, the
top-q survivors and the top-b_l keep set), key pruning, and value fusion
(Sec. 3.2 Eq. (redistribution) and Eq. (weight_fusion))."""
import json
import os

import numpy as np
import pytest
from scipy.special import softmax

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_values.json")))


def _bf16(x):
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def _f(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# ---------------------------------------------------------------- selection
@pytest.mark.parametrize("n,k,ns", [(1, 1, 1), (10, 3, 7), (100, 0, 40), (100, 40, 40),
                                    (257, 100, 180), (500, 500, 500)])
def test_select_brute_force(orc, n, k, ns):
    rng = np.random.default_rng(n + k)
    s = rng.integers(0, 20, n).astype(np.float32) / 7  # many exact ties
    kept, drop = orc.select(s, k, ns)
    order = np.lexsort((np.arange(n), -s.astype(np.float64)))  # score desc, index asc
    np.testing.assert_array_equal(kept, np.sort(order[:k]))
    np.testing.assert_array_equal(drop, np.sort(order[k:ns]))
    assert np.all(np.diff(kept) > 0) and np.all(np.diff(drop) > 0)
    assert not set(kept) & set(drop)


def test_select_all_equal_takes_lowest_indices(orc):
    kept, drop = orc.select(np.full(50, 0.25, np.float32), 12, 30)
    np.testing.assert_array_equal(kept, np.arange(12))
    np.testing.assert_array_equal(drop, np.arange(12, 30))


def test_select_nesting(orc):
    # One ranking: a smaller budget keeps a subset of a larger one (the layer
    # budgets decrease with depth under a shared ranking).
    rng = np.random.default_rng(2)
    s = rng.random(300).astype(np.float32)
    prev = None
    for k in [250, 200, 120, 60, 1]:
        kept, _ = orc.select(s, k, 260)
        if prev is not None:
            assert set(kept) <= set(prev)
        prev = kept


def test_gather_is_bit_copy(orc):
    rng = np.random.default_rng(4)
    K = rng.integers(0, 2 ** 16, (40, 64), dtype=np.uint16)
    kept = np.array([0, 3, 7, 39], np.int32)
    np.testing.assert_array_equal(orc.gather(K, kept), K[kept])
    np.testing.assert_array_equal(orc.gather(K, np.arange(40, dtype=np.int32)), K)


# ------------------------------------------------------------------- fusion
def _vals(rng, n, d, scale=1.0):
    return _bf16(rng.standard_normal((n, d)).astype(np.float32) * scale)


def _split(n, k, r, rng):
    perm = rng.permutation(n)
    return np.sort(perm[:k]).astype(np.int32), np.sort(perm[k:k + r]).astype(np.int32)


def test_mu_one_is_plain_pruning(orc):
    rng = np.random.default_rng(1)
    V = _vals(rng, 30, 64)
    kept, drop = _split(30, 10, 15, rng)
    out = orc.fuse(V, kept, drop, tau=1.0, mu=GOLD["mu_limits"]["mu_pruning"])
    np.testing.assert_array_equal(out, _f(V[kept]))


def test_brute_force_and_mu_zero(orc):
    rng = np.random.default_rng(7)
    for n, k, r, d in [(12, 4, 6, 64), (40, 9, 20, 128), (16, 1, 15, 64)]:
        V = _vals(rng, n, d, 0.4)
        kept, drop = _split(n, k, r, rng)
        Vk, Vd = _f(V[kept]), _f(V[drop])
        for tau, mu in [(1.0, 0.7), (3.0, 0.2), (0.5, GOLD["mu_limits"]["mu_replace"])]:
            Phi = softmax(Vk @ Vd.T / tau, axis=1)  # each kept row absorbs the drops
            ref = mu * Vk + (1 - mu) * (Phi @ Vd)
            np.testing.assert_allclose(orc.fuse(V, kept, drop, tau, mu), ref, rtol=1e-12, atol=1e-13)


def test_single_drop_is_absorbed_whole(orc):
    rng = np.random.default_rng(8)
    V = _vals(rng, 10, 64, 5.0)
    kept, drop = np.array([1, 4, 6], np.int32), np.array([8], np.int32)
    out = orc.fuse(V, kept, drop, 1.0, 0.7)
    mu = 0.7
    np.testing.assert_array_equal(out, mu * _f(V[kept]) + (1 - mu) * _f(V[8])[None, :])


def test_equal_drops_fuse_to_that_row(orc):
    rng = np.random.default_rng(9)
    V = _vals(rng, 20, 64)
    V[10:] = V[10]
    kept, drop = np.arange(5, dtype=np.int32), np.arange(10, 20, dtype=np.int32)
    out = orc.fuse(V, kept, drop, 1.0, 0.0)
    np.testing.assert_allclose(out, np.repeat(_f(V[10:11]), 5, axis=0), rtol=1e-14)


def test_temperature_limits(orc):
    rng = np.random.default_rng(10)
    V = _vals(rng, 30, 64)
    kept, drop = _split(30, 6, 20, rng)
    Vk, Vd = _f(V[kept]), _f(V[drop])
    hot = orc.fuse(V, kept, drop, 1e30, 0.0)  # flat Phi: the mean of the drops
    np.testing.assert_allclose(hot, np.repeat(Vd.mean(0, keepdims=True), 6, 0), rtol=1e-12)
    cold = orc.fuse(V, kept, drop, 1e-6, 0.0)  # one-hot Phi: the best-matching drop
    best = np.argmax(Vk @ Vd.T, axis=1)
    np.testing.assert_allclose(cold, Vd[best], rtol=1e-12, atol=1e-300)


def test_fused_rows_stay_in_the_drop_box_and_ignore_drop_order(orc):
    rng = np.random.default_rng(12)
    V = _vals(rng, 60, 64, 2.0)
    kept, drop = _split(60, 15, 30, rng)
    F = orc.fuse(V, kept, drop, 1.0, 0.0)
    Vd = _f(V[drop])
    assert np.all(F >= Vd.min(0) - 1e-12) and np.all(F <= Vd.max(0) + 1e-12)
    F2 = orc.fuse(V, kept, drop[::-1].copy(), 1.0, 0.0)
    np.testing.assert_allclose(F, F2, rtol=1e-12, atol=1e-14)


def test_empty_drop_or_keep(orc):
    rng = np.random.default_rng(13)
    V = _vals(rng, 8, 64)
    kept = np.arange(8, dtype=np.int32)
    out = orc.fuse(V, kept, np.zeros(0, np.int32), 1.0, 0.7)
    np.testing.assert_array_equal(out, _f(V))  # nothing dropped: values unchanged
    assert orc.fuse(V, np.zeros(0, np.int32), np.arange(3, dtype=np.int32)).shape == (0, 64)


# ------------------------------------------------------------------ decode
def test_attend(orc):
    rng = np.random.default_rng(14)
    d = 128
    K, V, q = _vals(rng, 33, d), _vals(rng, 33, d), _vals(rng, 1, d)[0]
    out = orc.attend(q, K, V, d ** -0.5)
    w = softmax(_f(K) @ _f(q) * d ** -0.5)
    np.testing.assert_allclose(out, w @ _f(V), rtol=1e-12, atol=1e-14)
    np.testing.assert_array_equal(orc.attend(q, K[:1], V[:1], 0.1), _f(V[0]))
    Ke = np.repeat(K[:1], 10, 0)
    np.testing.assert_allclose(orc.attend(q, Ke, V[:10], 0.1), _f(V[:10]).mean(0), rtol=1e-13)


# --------------------------------------------------------------- whole unit
def _numpy_unit(K, V, Q, k, ns, tau, mu):
    d = K.shape[1]
    Qb = _f(_bf16(Q))
    S = softmax(Qb @ _f(K).T / np.sqrt(d), axis=1).sum(0).astype(np.float32)
    order = np.lexsort((np.arange(len(S)), -S.astype(np.float64)))
    kept, drop = np.sort(order[:k]), np.sort(order[k:ns])
    Vk, Vd = _f(V[kept]), _f(V[drop])
    if len(drop) and len(kept):
        Vn = mu * Vk + (1 - mu) * softmax(Vk @ Vd.T / tau, axis=1) @ Vd
    else:
        Vn = Vk
    return kept, drop, K[kept], Vn


@pytest.mark.parametrize("n,k,ns,rows", [(16, 5, 9, 4), (12, 12, 12, 2), (16, 1, 16, 8), (9, 0, 4, 3)])
def test_unit_brute_force(orc, n, k, ns, rows):
    rng = np.random.default_rng(n * 3 + k)
    K, V = _vals(rng, n, 64), _vals(rng, n, 64)
    Q = rng.standard_normal((rows, 64)).astype(np.float32)
    got = orc.prune_unit(K, V, Q, k, ns, 1.0, 0.7)
    kept, drop, Ko, Vn = _numpy_unit(K, V, Q, k, ns, 1.0, 0.7)
    np.testing.assert_array_equal(got["kept"], kept)
    np.testing.assert_array_equal(got["drop"], drop)
    np.testing.assert_array_equal(got["K_out"], Ko)
    np.testing.assert_allclose(got["V_out"], Vn, rtol=1e-12, atol=1e-13)


def test_unit_keep_all_returns_cache(orc):
    rng = np.random.default_rng(21)
    K, V = _vals(rng, 40, 64), _vals(rng, 40, 64)
    got = orc.prune_unit(K, V, rng.standard_normal((6, 64)).astype(np.float32), 40, 40)
    np.testing.assert_array_equal(got["kept"], np.arange(40))
    np.testing.assert_array_equal(got["K_out"], K)
    np.testing.assert_array_equal(got["V_out"], _f(V))


def test_select_with_every_token_surviving_drops_the_complement(orc):
    # The fuse-all reading (n_surv = n): the dropped set is exactly the tokens
    # outside the kept set, in ascending order.
    rng = np.random.default_rng(11)
    for n, k in [(64, 10), (300, 1), (300, 299), (5, 0)]:
        s = rng.random(n).astype(np.float32)
        kept, drop = orc.select(s, k, n)
        assert len(kept) == k and len(drop) == n - k
        assert np.array_equal(np.sort(np.concatenate([kept, drop])), np.arange(n))
        assert np.all(np.diff(drop) > 0)
        top = np.argsort(-s.astype(np.float64), kind="stable")[:k]
        assert set(kept.tolist()) == set(top.tolist())
