"""Pins of the oracle's other policies over the partition-and-allocate
container: fair eviction (§4.1 "Fair-eviction baseline") and the No-X
counterfactual (§4 "Counterfactual", Table 2).

Fair eviction is pinned by its closed form in exact rational arithmetic (the
same retention rate K_p / P for every bucket, rounded up per bucket); No-X by
exhaustive subset search on tiny inputs and by its definition written without
buckets.
"""

import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
from oracle import brute

BUDGETS = [0.01, 0.05, 0.07, 0.1, 0.2, 0.33, 0.5, 0.9]


def _K(budget, N):
    """K = min(N, ceil(B*N)) with B read as the decimal it is written as."""
    return min(N, math.ceil(Fraction(str(budget)) * N))


@pytest.mark.parametrize("seed", range(4))
def test_fair_closed_form_exact(seed):
    r = np.random.default_rng(300 + seed)
    for _ in range(300):
        N = int(r.integers(1, 400))
        W = int(r.integers(0, N + 1))
        R = int(r.integers(1, 9))
        B = float(r.choice(BUDGETS))
        # skewed populations, some buckets empty
        p = r.dirichlet(np.full(R, 0.5))
        roles = r.choice(R, N, p=p).astype(np.int8)
        q, kept = O.fair_allocate(roles, R, B, W)
        P = N - W
        n = [int(np.sum(roles[:P] == b)) for b in range(R)]
        Kp = max(0, _K(B, N) - W)
        if P == 0:
            assert list(q) == [0] * R and kept == W
            continue
        expect = [(c * Kp + P - 1) // P for c in n]      # ceil(n_r K_p / P)
        assert list(q) == expect
        assert kept == W + sum(expect)
        assert 0 <= sum(expect) - Kp <= R - 1
        for c, qq in zip(n, q):
            if c:
                # the same rate for every bucket, up to one token of rounding
                assert Fraction(Kp, P) <= Fraction(int(qq), c) < Fraction(Kp, P) + Fraction(1, c)
                assert qq <= c


def test_fair_equal_populations_is_the_uniform_role_policy():
    r = np.random.default_rng(310)
    for _ in range(100):
        R = int(r.integers(1, 6))
        per = int(r.integers(1, 40))
        W = int(r.integers(0, 10))
        pre = np.repeat(np.arange(R, dtype=np.int8), per)
        r.shuffle(pre)
        roles = np.concatenate([pre, r.integers(0, R, W).astype(np.int8)])
        B = float(r.choice(BUDGETS))
        qf, kf = O.fair_allocate(roles, R, B, W)
        qu, ku = O.role_allocate(roles, R, [1.0] * R, B, W)
        assert np.array_equal(qf, qu) and kf == ku


def test_fair_edge_cases():
    roles = np.array([0, 1, 1, 2, 0, 1, 2, 2, 0, 1], dtype=np.int8)
    # full budget keeps every token
    q, kept = O.fair_allocate(roles, 3, 1.0, 2)
    assert kept == 10 and list(q) == [2, 3, 3]
    # the window is the whole sequence: nothing to allocate
    q, kept = O.fair_allocate(roles, 3, 0.3, 10)
    assert kept == 10 and list(q) == [0, 0, 0]
    # K < W: the window alone
    q, kept = O.fair_allocate(roles, 3, 0.1, 4)
    assert kept == 4 and list(q) == [0, 0, 0]
    # a hand-worked case: N=10, W=2, B=0.5 -> K=5, K_p=3, P=8, n=(2,3,3)
    # q = ceil(6/8), ceil(9/8), ceil(9/8) = 1, 2, 2
    q, kept = O.fair_allocate(roles, 3, 0.5, 2)
    assert list(q) == [1, 2, 2] and kept == 7
    with pytest.raises(ValueError):
        O.fair_allocate(roles, 2, 0.5, 2)


def test_role_map():
    r = np.random.default_rng(320)
    roles = r.integers(0, 5, (3, 50)).astype(np.int8)
    bmap = [2, 0, 0, 1, 2]
    out = O.role_map(roles, bmap)
    assert out.dtype == np.int8 and out.shape == roles.shape
    for b in range(3):
        for t in range(50):
            assert out[b, t] == bmap[roles[b, t]]
    with pytest.raises(ValueError):
        O.role_map(np.array([0, 5], dtype=np.int8), bmap)
    assert O.no_role_policy(1, 4) == ([0, 1, 0, 0], [1.0, 0.0])
    with pytest.raises(ValueError):
        O.no_role_policy(4, 4)


@pytest.mark.parametrize("seed", range(40))
def test_no_role_equals_exhaustive_search(seed):
    """No-X three ways on tiny inputs: its definition, the bucket composition
    (map, allocate with alpha = (1, 0), select) and exhaustive subset search."""
    r = np.random.default_rng(330 + seed)
    N = int(r.integers(3, 15))
    W = int(r.integers(0, 4))
    n_roles = int(r.integers(2, 5))
    x = int(r.integers(0, n_roles))
    roles = r.integers(0, n_roles, N).astype(np.int8)
    s = r.choice([0.25, 0.5, 0.75, -0.0, 0.0, np.nan], N) if seed % 2 else r.random(N)
    B = float(r.choice([0.2, 0.3, 0.5, 0.7, 0.9]))
    Kp = max(0, _K(B, N) - W)
    allowed = [t for t in range(N - W) if roles[t] != x]
    ref = brute.select_exhaustive(s.tolist(), [0 if t in allowed else 1 for t in range(N)],
                                  [min(Kp, len(allowed)), 0], W)
    assert O.no_role_keep(s, roles, x, B, W).tolist() == ref
    bucket_of, alpha = O.no_role_policy(x, n_roles)
    buckets = O.role_map(roles, bucket_of)
    q, kept = O.role_allocate(buckets, 2, alpha, B, W)
    assert list(q) == [min(Kp, len(allowed)), 0]
    got = O.select_keep(s, buckets, q, W)
    assert got.tolist() == ref and len(got) == kept


def test_no_role_bans_only_the_role_and_fills_the_budget():
    r = np.random.default_rng(380)
    N, W = 400, 16
    roles = r.integers(0, 4, N).astype(np.int8)
    s = r.random(N)
    s[roles == 1] += 10.0                # the banned role carries the most mass
    for B in (0.05, 0.2, 0.5, 0.9):
        idx = O.no_role_keep(s, roles, 1, B, W)
        pre = idx[idx < N - W]
        assert not np.any(roles[pre] == 1)
        allowed = int(np.sum(roles[:N - W] != 1))
        assert len(pre) == min(max(0, _K(B, N) - W), allowed)
        assert idx[-W:].tolist() == list(range(N - W, N))
    # B >= 1 is the full cache whatever the policy
    assert O.no_role_keep(s, roles, 1, 1.0, W).tolist() == list(range(N))
