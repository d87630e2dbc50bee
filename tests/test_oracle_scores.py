"""Pins for the oracle's window scores (Sec. 3.2 Eq. (token_score), read as the
attention that the trailing window queries give each visual key, summed over
the query rows of a KV-head group; see the design notes for the reading)."""
import numpy as np
import pytest
from scipy.special import expit, softmax


def _bf16(x):
    """Round float32 to bf16 (nearest even), returned as bits."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def _f(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _rand(rng, shape, scale=1.0):
    return _bf16(rng.standard_normal(shape).astype(np.float32) * scale)


@pytest.mark.parametrize("n,d,rows", [(1, 64, 3), (5, 64, 1), (37, 64, 8), (200, 128, 20)])
def test_rows_are_distributions(orc, n, d, rows):
    # Every query row's softmax sums to one, so the scores sum to the row count.
    rng = np.random.default_rng(n * 7 + rows)
    K = _rand(rng, (n, d), 2.0)
    Q = _f(_rand(rng, (rows, d), 2.0)).astype(np.float32)
    S = orc.scores_unit(K, Q)
    assert S.sum() == pytest.approx(rows, rel=1e-12)
    assert np.all(S > 0)


def test_identical_keys_give_uniform_scores(orc):
    rng = np.random.default_rng(3)
    K = np.repeat(_rand(rng, (1, 64)), 50, axis=0)
    Q = _f(_rand(rng, (6, 64), 3.0)).astype(np.float32)
    S = orc.scores_unit(K, Q)
    np.testing.assert_allclose(S, 6 / 50, rtol=1e-13)


@pytest.mark.parametrize("d", [64, 128])
def test_two_keys_sigmoid_closed_form(orc, d):
    # One query, two keys: the first key's weight is the logistic function of
    # the logit difference (q.k0 - q.k1)/sqrt(d).
    rng = np.random.default_rng(d)
    K = _rand(rng, (2, d))
    q = _f(_rand(rng, (1, d)))
    S = orc.scores_unit(K, q.astype(np.float32))
    diff = (q[0] @ (_f(K[0]) - _f(K[1]))) / np.sqrt(d)
    assert S[0] == pytest.approx(expit(diff), rel=1e-12)
    assert S[1] == pytest.approx(expit(-diff), rel=1e-12)


@pytest.mark.parametrize("n,d,rows", [(16, 64, 4), (9, 128, 7), (64, 64, 16)])
def test_brute_force_small(orc, n, d, rows):
    # Library softmax over a float64 matmul on tiny units.
    rng = np.random.default_rng(n + d + rows)
    K = _rand(rng, (n, d), 1.5)
    Qb = _rand(rng, (rows, d), 1.5)
    S = orc.scores_unit(K, _f(Qb).astype(np.float32))
    logits = (_f(Qb) @ _f(K).T) / np.sqrt(d)
    ref = softmax(logits, axis=1).sum(axis=0)
    np.testing.assert_allclose(S, ref, rtol=1e-12)


def test_query_enters_in_bf16(orc):
    # A query perturbed below half a bf16 ulp rounds to the same bf16 value, so
    # the scores are unchanged; perturbed across it they change.
    rng = np.random.default_rng(11)
    K = _rand(rng, (40, 64))
    q = _f(_rand(rng, (2, 64))).astype(np.float32)
    ulp = np.abs(q) * 2.0 ** -8
    S0 = orc.scores_unit(K, q)
    S1 = orc.scores_unit(K, (q + 0.25 * ulp).astype(np.float32))
    np.testing.assert_array_equal(S0, S1)
    S2 = orc.scores_unit(K, (q + 1.5 * ulp).astype(np.float32))
    assert not np.array_equal(S0, S2)


def test_large_logits_are_stable(orc):
    # Outlier-scale keys (x8) give logits in the hundreds: still finite, still
    # a distribution per row.
    rng = np.random.default_rng(5)
    K = _rand(rng, (30, 128), 24.0)
    Q = _f(_rand(rng, (3, 128), 24.0)).astype(np.float32)
    S = orc.scores_unit(K, Q)
    assert np.all(np.isfinite(S)) and S.sum() == pytest.approx(3, rel=1e-12)


def test_global_ranking_sum(orc):
    # Shared ranking: the sum over L layer-units of row-count-sum scores.
    rng = np.random.default_rng(9)
    units = [orc.scores_unit(_rand(rng, (20, 64)), _f(_rand(rng, (4, 64))).astype(np.float32))
             for _ in range(5)]
    s = orc.global_scores(units)
    assert s.dtype == np.float32
    assert float(s.astype(np.float64).sum()) == pytest.approx(20.0, rel=1e-6)
    np.testing.assert_array_equal(s, np.sum(units, axis=0).astype(np.float32))


# --- Prefill scoring: Eq. (token_score) with every prefill token as a query -----
# The sequence is n visual tokens then T text tokens; query i attends keys
# 0..i (causal); the score sums A_{i,v} over heads and queries.

def _prefill_inputs(rng, n, T, d, G, scale=1.5):
    K = _rand(rng, (n, d), scale)
    Kt = _rand(rng, (T, d), scale)
    Q = _f(_rand(rng, (G, n + T, d), scale)).astype(np.float32)
    return K, Kt, Q


@pytest.mark.parametrize("n,T,d,G", [(1, 0, 64, 1), (7, 3, 64, 2), (40, 9, 128, 3), (64, 16, 64, 4)])
def test_prefill_rows_are_distributions(orc, n, T, d, G):
    # Every query's causal softmax sums to one: visual plus text columns hold
    # the G*(n+T) rows' whole mass.
    rng = np.random.default_rng(n + 31 * T + d + G)
    K, Kt, Q = _prefill_inputs(rng, n, T, d, G)
    S, St = orc.scores_unit_prefill(K, Kt, Q, with_text=True)
    assert S.sum() + St.sum() == pytest.approx(G * (n + T), rel=1e-12)
    assert np.all(S > 0)


@pytest.mark.parametrize("n,T,G", [(1, 0, 1), (5, 0, 2), (12, 4, 3), (33, 7, 2)])
def test_prefill_identical_keys_harmonic(orc, n, T, G):
    # All keys equal: query i spreads weight 1/(i+1) over its i+1 keys, so
    # visual key v scores G * (H_{n+T} - H_v), H_k the k-th harmonic number.
    rng = np.random.default_rng(n * 5 + T)
    K = np.repeat(_rand(rng, (1, 64)), n, axis=0)
    Kt = np.repeat(K[:1], T, axis=0)
    Q = _f(_rand(rng, (G, n + T, 64), 2.0)).astype(np.float32)
    S = orc.scores_unit_prefill(K, Kt, Q)
    H = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, n + T + 1))])
    np.testing.assert_allclose(S, G * (H[n + T] - H[:n]), rtol=1e-13)


def test_prefill_first_token_sees_only_itself(orc):
    # One visual token and no text: its only query attends only it.
    rng = np.random.default_rng(2)
    K, Kt, Q = _prefill_inputs(rng, 1, 0, 64, 3)
    assert orc.scores_unit_prefill(K, Kt, Q)[0] == pytest.approx(3.0, rel=1e-15)


def test_prefill_visual_queries_ignore_text(orc):
    # Causality: visual tokens precede the text, so appending text tokens adds
    # only the text queries' attention; with the text scored alone the two
    # parts account for the text rows' mass.
    rng = np.random.default_rng(17)
    n, T, d, G = 20, 6, 64, 2
    K, Kt, Q = _prefill_inputs(rng, n, T, d, G)
    S0 = orc.scores_unit_prefill(K, Kt[:0], np.ascontiguousarray(Q[:, :n]))
    S, St = orc.scores_unit_prefill(K, Kt, Q, with_text=True)
    assert np.all(S - S0 >= -1e-12)
    assert (S - S0).sum() + St.sum() == pytest.approx(G * T, rel=1e-12)
    # changing a text key changes the visual scores only through text queries
    Kt2 = Kt.copy()
    Kt2[-1] = _rand(rng, (1, d), 3.0)[0]
    S2 = orc.scores_unit_prefill(K, Kt2, Q)
    assert not np.allclose(S, S2)
    Q3 = Q.copy()
    Q3[:, n:] = 0.0  # text queries with zero logits: uniform over their keys
    S3 = orc.scores_unit_prefill(K, Kt, Q3)
    uniform = G * sum(1.0 / (i + 1) for i in range(n, n + T))
    np.testing.assert_allclose(S3 - S0, uniform, rtol=1e-12)


@pytest.mark.parametrize("n,T,d,G", [(9, 4, 64, 2), (16, 0, 128, 1), (5, 11, 64, 3)])
def test_prefill_brute_force_small(orc, n, T, d, G):
    # Library softmax of the causally masked logit matrix on tiny units.
    rng = np.random.default_rng(100 + n + T + d + G)
    K, Kt, Q = _prefill_inputs(rng, n, T, d, G)
    keys = np.concatenate([_f(K), _f(Kt).reshape(-1, d)], axis=0)
    N = n + T
    ref = np.zeros(n)
    for h in range(G):
        q = _f(_bf16(Q[h]))
        logits = (q @ keys.T) / np.sqrt(d)
        logits[np.triu_indices(N, 1)] = -np.inf
        ref += softmax(logits, axis=1)[:, :n].sum(axis=0)
    np.testing.assert_allclose(orc.scores_unit_prefill(K, Kt, Q), ref, rtol=1e-12)
