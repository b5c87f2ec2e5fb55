"""Pins of the oracle's one-shot Quest analogue (§4.1 "Query-aware baseline").

The page bound is pinned by pure-Python loops, by its defining property (no
key of a page scores above the page's bound, and the bound is reached when a
page holds one distinct key), a one-channel closed form, and the page
geometry (ragged last page, window outside every page).  The selection it
drives is pinned against a page-level selection written independently.
"""

import math

import numpy as np
import pytest

import oracle as O
from oracle import brute


def _rand(r, *shape):
    return r.standard_normal(shape)


@pytest.mark.parametrize("seed", range(6))
def test_quest_equals_loops(seed):
    r = np.random.default_rng(500 + seed)
    G, W, N, d = int(r.integers(1, 5)), int(r.integers(1, 6)), int(r.integers(1, 60)), int(r.choice([1, 3, 8]))
    W = min(W, N)
    page = int(r.choice([1, 4, 16]))
    q, k = _rand(r, G, W, d), _rand(r, N, d)
    ref = brute.quest_loops(q.tolist(), k.tolist(), page)
    got = O.quest_mass(q, k, page)
    assert np.array_equal(np.isinf(got), np.isinf(ref))
    fin = ~np.isinf(got)
    assert np.allclose(got[fin], np.array(ref)[fin], rtol=1e-12, atol=1e-12)


def test_bound_dominates_every_key_and_is_tight_for_one_key():
    r = np.random.default_rng(510)
    G, W, N, d, page = 4, 8, 200, 32, 16
    q, k = _rand(r, G, W, d), _rand(r, N, d)
    s = O.quest_mass(q, k, page)
    qbar = q.mean(axis=1)
    exact = np.sum(qbar @ k.T, axis=0)            # sum_h <qbar_h, k_t>
    P = N - W
    assert np.all(exact[:P] <= s[:P] + 1e-12)
    assert np.all(np.isinf(s[P:]))
    # a page of one repeated key: the bound is that key's score
    k2 = k.copy()
    k2[16:32] = k2[20]
    s2 = O.quest_mass(q, k2, page)
    assert np.allclose(s2[16:32], exact[20], rtol=1e-12)


def test_one_channel_closed_form_and_sign():
    # d = 1, one head, W = 1: bound = max(q * kmin, q * kmax)
    k = np.array([[-2.0], [0.5], [3.0], [1.0], [-1.0], [9.0]])
    for qv, expect in [(2.0, [6.0, 6.0, 6.0, 2.0, 2.0]), (-1.5, [3.0, 3.0, 3.0, 1.5, 1.5])]:
        q = np.array([[[qv]]])
        s = O.quest_mass(q, k, 3)
        # pages {0,1,2} and {3,4}; row 5 is the window
        assert s[:5].tolist() == expect and math.isinf(s[5])


def test_mean_query_and_head_sum():
    r = np.random.default_rng(520)
    W, N, d = 6, 50, 8
    q, k = _rand(r, 2, W, d), _rand(r, N, d)
    both = O.quest_mass(q, k, 8)
    each = O.quest_mass(q[:1], k, 8) + O.quest_mass(q[1:], k, 8)
    fin = ~np.isinf(both)
    assert np.allclose(both[fin], each[fin], rtol=1e-12)
    # every window row equal to the mean gives the same scores
    qm = np.repeat(q.mean(axis=1, keepdims=True), W, axis=1)
    assert np.allclose(O.quest_mass(qm, k, 8)[fin], both[fin], rtol=1e-12)


@pytest.mark.parametrize("seed", range(8))
def test_selection_keeps_whole_pages_in_bound_order(seed):
    """One bucket: the per-bucket top-k over page-constant scores takes pages
    in bound order (lower page first on ties), the last one cut at K_p."""
    r = np.random.default_rng(530 + seed)
    G, W, N, d, page = 2, 4, int(r.integers(20, 300)), 8, 16
    q, k = _rand(r, G, W, d), _rand(r, N, d)
    if seed % 2:
        k[16:32] = k[0:16]                      # two pages with equal bounds
    s = O.quest_mass(q, k, page)
    B = float(r.choice([0.1, 0.3, 0.5]))
    roles = np.zeros(N, dtype=np.int8)
    quota, kept = O.role_allocate(roles, 1, [1.0], B, W)
    got = O.select_keep(s, roles, quota, W)
    P = N - W
    K_p = int(quota[0])
    n_pages = (P + page - 1) // page
    bounds = [s[j * page] for j in range(n_pages)]
    order = sorted(range(n_pages), key=lambda j: (-bounds[j], j))
    take = []
    for j in order:
        for t in range(j * page, min((j + 1) * page, P)):
            if len(take) < K_p:
                take.append(t)
    ref = sorted(take + list(range(P, N)))
    assert got.tolist() == ref and len(got) == kept


def test_quest_wrapper_groups_heads_contiguously_and_sums_them():
    """oracle.quest_score: query heads 0,1 read KV head 0 and heads 2,3 KV
    head 1, and the bounds of a group's heads are summed.  Heads 0,1 have mean
    window query 2*e0, heads 2,3 mean 2*e1; pages of 2 tokens, N = 10, W = 2
    (four pages).  KV head 0: keys zero except t = 2 (3 along e0, page 1) and
    t = 5 (5 along e1, page 2); KV head 1: t = 1 (4 along e0, page 0) and t = 6
    (2 along e1, page 3).  With contiguous groups only the channel a group
    looks along counts: KV head 0 scores page 1 at 2 heads * 2 * 3 = 12, KV
    head 1 page 3 at 2 * 2 * 2 = 8, every other page 0 and the window +inf.
    A strided grouping (heads 0,2 | 1,3) would score page 2 of KV head 0 at
    10 and page 1 at 6."""
    N, W, d, page = 10, 2, 4, 2
    q = np.zeros((1, 1, 4, W, d))
    q[0, 0, 0:2, :, 0] = 2.0
    q[0, 0, 2:4, :, 1] = 2.0
    k = np.zeros((1, 1, 2, N, d))
    k[0, 0, 0, 2, 0] = 3.0
    k[0, 0, 0, 5, 1] = 5.0
    k[0, 0, 1, 1, 0] = 4.0
    k[0, 0, 1, 6, 1] = 2.0
    s = O.quest_score(q, k, n_kv_heads=2, page=page)
    inf = np.inf
    assert s[0, 0, 0].tolist() == [0, 0, 12, 12, 0, 0, 0, 0, inf, inf]
    assert s[0, 0, 1].tolist() == [0, 0, 0, 0, 0, 0, 8, 8, inf, inf]
