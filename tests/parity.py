"""Comparison rules between the HIP path and the oracle.

Scores: |gpu - oracle| <= RTOL * |oracle| + floor for every entry, with
RTOL = 1e-3 (float32 accumulation of bfloat16 products) and floor =
1e-6 * mean(oracle) for entries that are exactly zero or underflow.

Kept sets: equal, except pairs of candidates of one bucket whose oracle scores
lie within RTOL of that bucket's boundary score (near-ties at the k-th
boundary); such pairs are counted and returned, never silently accepted.
"""

from __future__ import annotations

import numpy as np

RTOL = 1e-3
FLOOR_FRAC = 1e-6

# Figures the GPU tests record (near-tie counts, worst error ratios); the
# conftest prints them in pytest's terminal summary so that they reach the
# records of a passing run too.
REPORT: dict = {}


def report(key: str, value) -> None:
    """Record one figure under `key` (numbers under one key are summed)."""
    if isinstance(value, (int, float)) and isinstance(REPORT.get(key), (int, float)):
        REPORT[key] += value
    else:
        REPORT[key] = value


def check_scores(gpu: np.ndarray, orc: np.ndarray, what: str = "score"):
    gpu = np.asarray(gpu, dtype=np.float64)
    orc = np.asarray(orc, dtype=np.float64)
    assert gpu.shape == orc.shape, (gpu.shape, orc.shape)
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite values"
    floor = FLOOR_FRAC * float(np.mean(np.abs(orc)))
    err = np.abs(gpu - orc)
    bound = RTOL * np.abs(orc) + floor
    bad = err > bound
    if np.any(bad):
        i = np.unravel_index(np.argmax(err / bound), err.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} entries out of tolerance; "
                             f"worst at {i}: gpu={gpu[i]!r} oracle={orc[i]!r}")
    return float(np.max(err / np.maximum(np.abs(orc), floor)))


def check_kept_set(idx_gpu, idx_orc, score_orc, roles, W: int, quota):
    """Compare the kept sets of one segment; returns the number of near-tie
    pairs accepted.  idx_* are ascending index arrays."""
    g = np.asarray(idx_gpu, dtype=np.int64)
    o = np.asarray(idx_orc, dtype=np.int64)
    assert np.all(np.diff(g) > 0), "gpu indices not strictly ascending"
    assert len(g) == len(o), (len(g), len(o))
    if np.array_equal(g, o):
        return 0
    N = len(score_orc)
    roles = np.asarray(roles)
    gs, os_ = set(g.tolist()), set(o.tolist())
    only_g = sorted(gs - os_)
    only_o = sorted(os_ - gs)
    assert all(t < N - W for t in only_g + only_o), "window mismatch"
    ties = 0
    for r in range(len(quota)):
        a = [t for t in only_g if roles[t] == r]
        b = [t for t in only_o if roles[t] == r]
        assert len(a) == len(b), f"bucket {r}: counts differ"
        if not a:
            continue
        cand = np.array([t for t in range(N - W) if roles[t] == r])
        s = np.asarray(score_orc, dtype=np.float64)[cand]
        q = int(quota[r])
        boundary = np.sort(s)[::-1][q - 1]
        for t in a + b:
            assert abs(score_orc[t] - boundary) <= RTOL * max(abs(boundary), abs(score_orc[t])), (
                f"bucket {r}: token {t} (oracle score {score_orc[t]!r}) is not a near-tie of the "
                f"boundary {boundary!r}")
        ties += len(a)
    return ties


# Decode outputs: o = sum_t p_t v_t is checked against the oracle entry by
# entry with a bound proportional to sum_t p_t |v_t| (the magnitude the float32
# sums actually carry, not |o|, which cancels).  Float32 logits of bfloat16
# products are off by about 1e-6 of their magnitude; the factor (1 + xmax / 16)
# widens the bound for large logits x (natural-log units), whose absolute
# rounding error, and hence the relative error of exp(x), grows with |x|.
DEC_RTOL = 1e-4


def check_decode(gpu: np.ndarray, orc: np.ndarray, orc_abs: np.ndarray, xmax: float,
                 what: str = "decode"):
    gpu = np.asarray(gpu, dtype=np.float64)
    orc = np.asarray(orc, dtype=np.float64)
    assert gpu.shape == orc.shape, (gpu.shape, orc.shape)
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite values"
    bound = DEC_RTOL * (1.0 + xmax / 16.0) * np.asarray(orc_abs, dtype=np.float64) + 1e-30
    err = np.abs(gpu - orc)
    bad = err > bound
    if np.any(bad):
        i = np.unravel_index(np.argmax(err / bound), err.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} entries out of tolerance; "
                             f"worst at {i}: gpu={gpu[i]!r} oracle={orc[i]!r} bound={bound[i]!r}")
    return float(np.max(err / bound))
