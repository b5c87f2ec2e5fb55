"""Pins of the oracle's role allocation and per-role selection.

Hand-worked allocations live in tests/golden/allocation_worked_examples.txt;
the selection is pinned by exhaustive search over subsets on tiny inputs and
by NumPy's lexsort.
"""

import math
import os

import numpy as np
import pytest

import oracle as O
from oracle import brute

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load_examples():
    rows = []
    with open(os.path.join(GOLDEN, "allocation_worked_examples.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            t = line.split()
            name, N, W, B = t[0], int(t[1]), int(t[2]), float(t[3])
            alpha = [float(x) for x in t[4:8]]
            n = [int(x) for x in t[8:12]]
            quota = [int(x) for x in t[12:16]]
            kept = int(t[16])
            rows.append((name, N, W, B, alpha, n, quota, kept))
    return rows


def _roles_from_counts(n, W, seed=0):
    """A prefix holding n[r] tokens of role r (shuffled) followed by W window
    tokens of role 3."""
    pre = np.concatenate([np.full(c, r, dtype=np.int8) for r, c in enumerate(n)])
    np.random.default_rng(seed).shuffle(pre)
    return np.concatenate([pre, np.full(W, 3, dtype=np.int8)])


@pytest.mark.parametrize("ex", _load_examples(), ids=lambda e: e[0])
def test_worked_examples(ex):
    name, N, W, B, alpha, n, quota, kept = ex
    roles = _roles_from_counts(n, W)
    assert roles.shape[0] == N
    q, k = O.role_allocate(roles, 4, alpha, B, W)
    assert list(q) == quota, name
    assert k == kept, name


def test_binary64_guard():
    assert 0.07 * 100 > 7.0                    # the product binary64 actually gives
    assert O.ceil_guarded(0.07 * 100) == 7
    assert O.ceil_guarded(7.2) == 8
    assert O.ceil_guarded(0.0) == 0


def _random_case(r):
    N = int(r.integers(1, 400))
    W = int(r.integers(0, N + 1))
    R = int(r.integers(1, 9))
    roles = r.integers(0, R, N).astype(np.int8)
    alpha = r.random(R)
    alpha[r.random(R) < 0.3] = 0.0
    if alpha.sum() == 0:
        alpha[0] = 1.0
    B = float(r.choice([0.01, 0.05, 0.1, 0.2, 0.33, 0.5, 0.75, 0.9, 0.999, 1.0]))
    return N, W, R, roles, alpha, B


def test_allocation_properties_on_random_grid():
    r = np.random.default_rng(11)
    for _ in range(3000):
        N, W, R, roles, alpha, B = _random_case(r)
        q, kept = O.role_allocate(roles, R, alpha, B, W)
        n = O.role_counts(roles, R, W)
        assert kept == W + q.sum()
        assert np.all(q >= 0) and np.all(q <= n)
        if B >= 1.0:
            assert kept == N and np.array_equal(q, n)
            continue
        K = min(N, math.ceil(B * N - 1e-9))
        Kp = max(0, K - W)
        assert np.all(q[alpha == 0] == 0)
        pos = alpha > 0
        # the whole prefix budget is used unless every positive bucket is full
        assert q.sum() >= min(Kp, n[pos].sum())
        # ceilings can overshoot K by at most one per bucket minus one
        if Kp > 0:
            assert kept <= K + R - 1
        # with no bucket exceeding its population the quota is the literal ceiling
        open_ = pos & (n > 0)
        tot = alpha[open_].sum()
        shares = np.array([math.ceil(a / tot * Kp - 1e-9) if o else 0
                           for a, o in zip(alpha, open_)])
        if Kp > 0 and np.all(shares[open_] <= n[open_]):
            assert np.array_equal(q, shares)


def test_full_budget_general_path_keeps_everything():
    """A budget that rounds to K = N with every weight positive keeps all tokens
    through the water-filling path itself (no special case involved)."""
    r = np.random.default_rng(12)
    for _ in range(200):
        N = int(r.integers(10, 300))
        W = int(r.integers(0, N // 2))
        R = 4
        roles = r.integers(0, R, N).astype(np.int8)
        alpha = r.random(R) + 0.01
        q, kept = O.role_allocate(roles, R, alpha, 1.0 - 1e-12, W)
        assert kept == N


def test_allocation_rejects_bad_arguments():
    roles = np.array([0, 1, 2, 3, 0], dtype=np.int8)
    with pytest.raises(ValueError):
        O.role_allocate(roles, 4, [0.25, 0, 0.7, 0.05], 0.0, 1)
    with pytest.raises(ValueError):
        O.role_allocate(roles, 4, [0.25, 0, 0.7, 0.05], 0.5, 6)
    with pytest.raises(ValueError):
        O.role_allocate(roles, 3, [0.25, 0, 0.7], 0.5, 1)          # label 3 >= R
    with pytest.raises(ValueError):
        O.role_allocate(roles, 4, [0.25, -0.1, 0.7, 0.05], 0.5, 1)
    with pytest.raises(ValueError):
        O.role_allocate(roles, 4, [0, 0, 0, 0], 0.5, 1)


# ---------------------------------------------------------------------------
# Selection
# ---------------------------------------------------------------------------

def _tie_scores(r, N):
    s = r.integers(0, 4, N).astype(np.float64) / 4.0      # many exact ties
    s[r.random(N) < 0.1] = -0.0
    s[r.random(N) < 0.1] = -np.inf
    s[r.random(N) < 0.1] = np.nan
    return s


@pytest.mark.parametrize("seed", range(40))
def test_selection_equals_exhaustive_search(seed):
    r = np.random.default_rng(200 + seed)
    N = int(r.integers(4, 15))
    W = int(r.integers(0, 4))
    R = int(r.integers(1, 4))
    roles = r.integers(0, R, N).astype(np.int8)
    s = _tie_scores(r, N) if seed % 2 else r.random(N)
    n = O.role_counts(roles, R, W)
    quota = [int(r.integers(0, c + 1)) for c in n]
    got = O.select_keep(s, roles, quota, W)
    ref = brute.select_exhaustive(s.tolist(), roles.tolist(), quota, W)
    assert got.tolist() == ref
    assert len(got) == W + sum(quota)


def test_selection_tie_rule_lower_index_and_nan_last():
    s = np.array([0.5, 0.5, np.nan, 0.5, -0.0, 0.0, 0.9, 0.1])
    roles = np.zeros(8, dtype=np.int8)
    # prefix = first 6 tokens, window = last 2
    assert O.select_keep(s, roles, [2], 2).tolist() == [0, 1, 6, 7]
    assert O.select_keep(s, roles, [3], 2).tolist() == [0, 1, 3, 6, 7]
    assert O.select_keep(s, roles, [5], 2).tolist() == [0, 1, 3, 4, 5, 6, 7]
    assert O.select_keep(s, roles, [6], 2).tolist() == [0, 1, 2, 3, 4, 5, 6, 7]


def test_selection_ranks_nan_below_minus_infinity():
    """NaN ranks strictly below -inf (not equal to it): with the boundary
    inside a run of -inf and NaN scores, every -inf is taken before any NaN,
    whatever their positions; NaNs among themselves go lowest index first."""
    s = np.array([np.nan, -np.inf, np.nan, -np.inf, 1.0, np.nan])
    roles = np.zeros(6, dtype=np.int8)
    assert O.select_keep(s, roles, [1], 0).tolist() == [4]
    assert O.select_keep(s, roles, [2], 0).tolist() == [1, 4]
    assert O.select_keep(s, roles, [3], 0).tolist() == [1, 3, 4]
    assert O.select_keep(s, roles, [4], 0).tolist() == [0, 1, 3, 4]
    assert O.select_keep(s, roles, [5], 0).tolist() == [0, 1, 2, 3, 4]
    for q in range(7):
        assert O.select_keep(s, roles, [q], 0).tolist() == brute.select_exhaustive(s.tolist(), [0] * 6, [q], 0)
    # two buckets with the boundary of each between -inf and NaN
    roles2 = np.array([0, 1, 1, 0, 0, 1], dtype=np.int8)
    assert O.select_keep(s, roles2, [2, 1], 0).tolist() == [1, 3, 4]
    # the No-X definition ranks the same way
    assert O.no_role_keep(s, np.zeros(6, dtype=np.int8), 1, 0.5, 0).tolist() == [1, 3, 4]


def test_neutral_single_bucket_is_plain_snapkv():
    """One bucket with weight 1: the top-K_p prefix tokens by score (lower index
    first on ties) plus the window, at budget B."""
    r = np.random.default_rng(13)
    for _ in range(50):
        N = int(r.integers(20, 200))
        W = int(r.integers(0, 10))
        B = float(r.choice([0.05, 0.1, 0.3, 0.6]))
        s = np.round(r.random(N), 2)
        roles = np.zeros(N, dtype=np.int8)
        q, kept = O.role_allocate(roles, 1, [1.0], B, W)
        K = min(N, math.ceil(B * N - 1e-9))
        Kp = max(0, K - W)
        assert q[0] == Kp
        got = O.select_keep(s, roles, q, W)
        order = sorted(range(N - W), key=lambda t: (-s[t], t))
        ref = sorted(order[:Kp] + list(range(N - W, N)))
        assert got.tolist() == ref


def test_alpha_key_zero_keeps_no_prefix_key():
    r = np.random.default_rng(14)
    N, W = 300, 16
    roles = r.integers(0, 4, N).astype(np.int8)
    s = r.random(N)
    s[roles == 1] += 10.0                       # KEY tokens carry the most mass
    q, kept = O.role_allocate(roles, 4, [0.25, 0.0, 0.70, 0.05], 0.3, W)
    idx = O.select_keep(s, roles, q, W)
    pre = idx[idx < N - W]
    assert not np.any(roles[pre] == 1)
    assert len(idx) == kept


def test_out_of_range_labels_never_kept():
    s = np.arange(10, dtype=np.float64)
    roles = np.array([0, 5, 0, 5, 0, 5, 0, 5, 0, 0], dtype=np.int8)
    idx = O.select_keep(s, roles, [2], 2)
    assert idx.tolist() == [4, 6, 8, 9]


def test_compaction_is_a_bit_copy():
    r = np.random.default_rng(15)
    kv = r.integers(0, 65536, (50, 8)).astype(np.uint16)     # bf16 bit patterns
    idx = np.array([0, 3, 4, 17, 49])
    out = O.kv_compact(kv, idx)
    for m, t in enumerate(idx):
        assert out[m].tobytes() == kv[t].tobytes()
