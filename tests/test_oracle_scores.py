"""Pins of the oracle's score functions (softmax, H2O, SnapKV, max-pool).

Each test checks the oracle against something other than itself: closed
forms, invariants the definitions fix, a library routine, or the independent
pure-Python loops of ``oracle.brute``.
"""

import math

import numpy as np
import pytest
import scipy.ndimage
import scipy.special

import oracle as O
from oracle import brute


def _rng(seed=0):
    return np.random.default_rng(seed)


def test_softmax_rows_sum_to_one_and_first_row_is_one_hot():
    r = _rng(1)
    N, d = 40, 16
    q = r.standard_normal((N, d))
    k = r.standard_normal((N, d))
    p = O.causal_softmax(O.causal_logits(q, np.arange(N), k, 0.25))
    assert np.all(np.abs(p.sum(axis=1) - 1.0) < 1e-12)
    assert p[0, 0] == 1.0 and np.all(p[0, 1:] == 0.0)
    assert np.all(np.triu(p, 1) == 0.0)                      # causal


def test_softmax_matches_scipy_on_causal_rows():
    r = _rng(2)
    N, d = 30, 8
    q = r.standard_normal((N, d))
    k = r.standard_normal((N, d))
    scale = 1 / math.sqrt(d)
    p = O.causal_softmax(O.causal_logits(q, np.arange(N), k, scale))
    for i in range(N):
        ref = scipy.special.softmax(scale * (k[:i + 1] @ q[i]))
        np.testing.assert_allclose(p[i, :i + 1], ref, rtol=1e-13, atol=1e-15)


def test_two_token_softmax_is_logistic():
    """With keys k0 = 0 and k1 = b*e1, a query a*e1 at position 1 puts
    logistic(scale*a*b) on key 1 (sign, scale and operand order all matter)."""
    d = 4
    a, b = 1.5, 2.0
    q_win = np.zeros((1, 1, d))
    q_win[0, 0, 0] = a
    k = np.zeros((2, d))
    k[1, 0] = b
    s = O.snapkv_mass(q_win, k)                 # W = 1: the query at position 1
    p1 = 1.0 / (1.0 + math.exp(-0.5 * a * b))   # scale 1/sqrt(4) = 0.5
    assert abs(p1 - 0.8175744761936437) < 1e-15
    np.testing.assert_allclose(s, [1 - p1, p1], rtol=1e-14)
    s2 = O.snapkv_mass(q_win, k, scale=1.0)
    p2 = 1.0 / (1.0 + math.exp(-a * b))
    np.testing.assert_allclose(s2, [1 - p2, p2], rtol=1e-14)


def test_logit_uses_query_rows_against_key_rows():
    """A non-square case where a transposed operand would give wrong mass:
    queries along e2 must pick the key that is large along e2."""
    d = 3
    q_win = np.zeros((1, 2, d))
    q_win[0, :, 1] = 4.0
    k = np.zeros((5, d))
    k[1, 1] = 3.0      # strongly matched by the queries
    k[2, 0] = 3.0      # matched only under a wrong axis
    s = O.snapkv_mass(q_win, k, scale=1.0)
    assert np.argmax(s[:3]) == 1
    assert s[1] > 1.9


def test_h2o_total_mass_equals_query_count():
    r = _rng(3)
    G, N, d = 3, 50, 16
    q = r.standard_normal((G, N, d))
    k = r.standard_normal((N, d))
    s = O.h2o_mass(q, k)
    assert abs(s.sum() - G * N) < 1e-9
    # the last key is seen only by the last query of each head
    qq = np.concatenate([q[h] for h in range(G)])
    del qq
    last = sum(O.causal_softmax(O.causal_logits(q[h][-1:], np.array([N - 1]), k,
                                                1 / math.sqrt(d)))[0, -1] for h in range(G))
    assert abs(s[-1] - last) < 1e-12


def test_snapkv_total_mass_equals_window_queries():
    r = _rng(4)
    G, W, N, d = 4, 7, 60, 16
    s = O.snapkv_mass(r.standard_normal((G, W, d)), r.standard_normal((N, d)))
    assert abs(s.sum() - G * W) < 1e-10


def _harmonic(n):
    return sum(1.0 / i for i in range(1, n + 1))


def test_equal_keys_closed_form_h2o():
    """All keys equal: p[i, t] = 1/(i+1), so s(t) = G (H_N - H_t)."""
    r = _rng(5)
    G, N, d = 2, 33, 8
    q = r.standard_normal((G, N, d))
    k = np.tile(r.standard_normal(d), (N, 1))
    s = O.h2o_mass(q, k)
    ref = np.array([G * (_harmonic(N) - _harmonic(t)) for t in range(N)])
    np.testing.assert_allclose(s, ref, rtol=1e-12)


@pytest.mark.parametrize("W", [1, 5, 33])
def test_equal_keys_closed_form_snapkv(W):
    """All keys equal: s(t) = G * sum_{i=max(t, N-W)}^{N-1} 1/(i+1)."""
    r = _rng(6)
    G, N, d = 3, 33, 8
    q = r.standard_normal((G, W, d))
    k = np.zeros((N, d))
    s = O.snapkv_mass(q, k)
    ref = np.array([G * sum(1.0 / (i + 1) for i in range(max(t, N - W), N)) for t in range(N)])
    np.testing.assert_allclose(s, ref, rtol=1e-12, atol=1e-15)


def test_snapkv_with_full_window_equals_h2o():
    r = _rng(7)
    G, N, d = 2, 41, 16
    q = r.standard_normal((G, N, d))
    k = r.standard_normal((N, d))
    np.testing.assert_allclose(O.snapkv_mass(q, k), O.h2o_mass(q, k), rtol=1e-12)
    sc = O.snapkv_score(q[None, None], k[None, None, None], 1, pool_kernel=1)
    np.testing.assert_allclose(sc[0, 0, 0], O.h2o_mass(q, k), rtol=1e-12)


def test_key_shift_invariance():
    """Adding one vector to every key shifts each query's logits by a constant."""
    r = _rng(8)
    G, W, N, d = 2, 6, 45, 16
    q = r.standard_normal((G, W, d))
    k = r.standard_normal((N, d))
    c = 3.0 * r.standard_normal(d)
    np.testing.assert_allclose(O.snapkv_mass(q, k + c), O.snapkv_mass(q, k), rtol=1e-9, atol=1e-13)
    qf = r.standard_normal((G, N, d))
    np.testing.assert_allclose(O.h2o_mass(qf, k + c), O.h2o_mass(qf, k), rtol=1e-9, atol=1e-13)


def test_gqa_groups_are_contiguous_and_summed():
    """Query heads 0,1 belong to KV head 0 and heads 2,3 to KV head 1."""
    d, N, W = 4, 8, 2
    q = np.zeros((1, 1, 4, W, d))
    q[0, 0, 0:2, :, 0] = 6.0     # group 0 looks along e0
    q[0, 0, 2:4, :, 1] = 6.0     # group 1 looks along e1
    k = np.zeros((1, 1, 2, N, d))
    for j in range(2):
        k[0, 0, j, 3, 0] = 3.0
        k[0, 0, j, 5, 1] = 3.0
    s = O.snapkv_score(q, k, n_kv_heads=2, pool_kernel=1, scale=1.0)
    assert np.argmax(s[0, 0, 0]) == 3 and np.argmax(s[0, 0, 1]) == 5
    # the mass of the two heads of a group is summed: total G*W per KV head
    np.testing.assert_allclose(s[0, 0].sum(axis=1), [2 * W, 2 * W], rtol=1e-12)
    assert s[0, 0, 0, 3] > 0.99 * 2 * W


def test_h2o_wrapper_groups_heads_contiguously_and_sums_them():
    """oracle.h2o_score: query heads 0,1 read KV head 0 and heads 2,3 KV head 1
    (contiguous groups), and the mass of a group's heads is summed.  Heads 0,1
    look along e0, heads 2,3 along e1; KV head 0 has one key large along e0
    (t = 3), KV head 1 one key large along e1 (t = 5).  With contiguous groups
    each head of a group puts nearly all its mass on that key from the first
    query that sees it, so s(3) and s(5) approach G * (N - t); a strided
    grouping (heads 0,2 | 1,3) halves them, a swapped one moves the argmax."""
    N, d, G = 10, 4, 2
    q = np.zeros((1, 1, 4, N, d))
    q[0, 0, 0:2, :, 0] = 6.0
    q[0, 0, 2:4, :, 1] = 6.0
    k = np.zeros((1, 1, 2, N, d))
    k[0, 0, 0, 3, 0] = 3.0
    k[0, 0, 1, 5, 1] = 3.0
    s = O.h2o_score(q, k, n_kv_heads=2, scale=1.0)
    assert s.shape == (1, 1, 2, N)
    assert np.argmax(s[0, 0, 0]) == 3 and np.argmax(s[0, 0, 1]) == 5
    assert s[0, 0, 0, 3] > 0.999 * G * (N - 3)
    assert s[0, 0, 1, 5] > 0.999 * G * (N - 5)
    # every query row's probabilities sum to 1: total mass G * N per KV head
    np.testing.assert_allclose(s[0, 0].sum(axis=1), [G * N, G * N], rtol=1e-12)
    # keys before the spike share each query's mass uniformly: key 0 of KV
    # head 0 gets 1, 1/2, 1/3 from queries 0..2 of each of the two heads
    np.testing.assert_allclose(s[0, 0, 0, 0], G * (1 + 1 / 2 + 1 / 3), rtol=1e-6)


@pytest.mark.parametrize("seed", range(4))
def test_brute_force_agreement(seed):
    r = _rng(100 + seed)
    G, W, N, d = 2, 4, 19, 6
    q = r.standard_normal((G, W, d))
    k = r.standard_normal((N, d))
    np.testing.assert_allclose(O.snapkv_mass(q, k),
                               brute.snapkv_loops(q.tolist(), k.tolist()), rtol=1e-12)
    qf = r.standard_normal((G, N, d))
    np.testing.assert_allclose(O.h2o_mass(qf, k, row_block=5),
                               brute.h2o_loops(qf.tolist(), k.tolist()), rtol=1e-12)
    s = r.random(N)
    for kern in (1, 3, 5, 7):
        np.testing.assert_array_equal(O.maxpool_prefix(s, W, kern), brute.pool_loops(s.tolist(), W, kern))


def test_pool_kernel_one_is_identity():
    s = _rng(9).random(50)
    np.testing.assert_array_equal(O.maxpool_prefix(s, 10, 1), s)


@pytest.mark.parametrize("kern", [3, 5, 7, 15])
@pytest.mark.parametrize("W", [0, 1, 16])
def test_pool_matches_scipy_on_prefix(kern, W):
    s = _rng(10 + kern + W).random(64)
    N = s.shape[0]
    out = O.maxpool_prefix(s, W, kern)
    ref = scipy.ndimage.maximum_filter1d(s[:N - W], size=kern, mode="constant", cval=-np.inf)
    np.testing.assert_array_equal(out[:N - W], ref)
    np.testing.assert_array_equal(out[N - W:], s[N - W:])       # window unpooled


def test_pool_rejects_even_kernel():
    with pytest.raises(ValueError):
        O.maxpool_prefix(np.zeros(8), 2, 4)


def test_window_lse_is_the_softmax_normaliser():
    """The window rows' log-sum-exp matches scipy's logsumexp over the causal
    keys, and exp(x - lse) rows sum to 1 and equal the oracle's softmax."""
    from scipy.special import logsumexp
    r = np.random.default_rng(700)
    G, W, N, d = 3, 5, 40, 16
    q, k = r.standard_normal((G, W, d)), r.standard_normal((N, d))
    lse = O.window_lse(q, k)
    pos = np.arange(N - W, N)
    for h in range(G):
        x = O.causal_logits(q[h], pos, k, 1.0 / np.sqrt(d))
        for i in range(W):
            assert np.isclose(lse[h, i], logsumexp(x[i, :pos[i] + 1]), rtol=1e-13, atol=1e-13)
        p = np.exp(x - lse[h][:, None])
        assert np.allclose(p.sum(axis=1), 1.0, atol=1e-12)
        assert np.allclose(p, O.causal_softmax(x), atol=1e-13)
