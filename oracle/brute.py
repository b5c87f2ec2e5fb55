"""Pure-Python loop versions of the scores and the selection, for tiny inputs.

TEST INFRASTRUCTURE ONLY.  A second, independent reading of the same
definitions as ``oracle.reference`` (no NumPy arithmetic, only ``math``), used
by the tests to pin the vectorised oracle.  Quadratic or exponential cost:
keep N small.
"""

from __future__ import annotations

import itertools
import math


def _dot(a, b):
    return sum(float(x) * float(y) for x, y in zip(a, b))


def mass_loops(q_heads, q_positions, k, scale):
    """s(t) = sum over heads h, query rows i (at position q_positions[i]) of the
    causal softmax probability p_h[i, t] (§2).  q_heads[h][i] is a d-vector."""
    N = len(k)
    s = [0.0] * N
    for rows in q_heads:
        for q, pos in zip(rows, q_positions):
            logits = [scale * _dot(q, k[t]) for t in range(pos + 1)]
            m = max(logits)
            w = [math.exp(x - m) for x in logits]
            z = sum(w)
            for t in range(pos + 1):
                s[t] += w[t] / z
    return s


def snapkv_loops(q_win, k, scale=None):
    """q_win[h][i] for the last W positions; see ``oracle.reference.snapkv_mass``."""
    d = len(k[0])
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    N, W = len(k), len(q_win[0])
    return mass_loops(q_win, list(range(N - W, N)), k, scale)


def h2o_loops(q, k, scale=None):
    """q[h][i] for every position i; see ``oracle.reference.h2o_mass``."""
    d = len(k[0])
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    return mass_loops(q, list(range(len(k))), k, scale)


def pool_loops(s, W, kernel):
    """Max over the in-prefix neighbours within kernel//2 (§4, Algorithm 1)."""
    N = len(s)
    P = N - W
    h = kernel // 2
    out = list(s)
    for t in range(P):
        best = -math.inf
        for u in range(t - h, t + h + 1):
            if 0 <= u < P and s[u] > best:
                best = s[u]
        out[t] = best
    return out


def _rank(score, idx):
    """Sort key of a candidate, best first: every number before every NaN
    (NaN ranks below -inf), then the larger score, then the lower index."""
    if math.isnan(score):
        return (1, 0.0, idx)
    return (0, -score, idx)


def _better(a_score, a_idx, b_score, b_idx):
    """True when candidate a outranks b (see _rank)."""
    return _rank(a_score, a_idx) < _rank(b_score, b_idx)


def select_exhaustive(score, roles, quota, W):
    """Kept set found by enumerating every quota[r]-subset of each bucket and
    taking the one that is best under the ranking order: compare the subsets'
    members sorted best-first, element by element (a lexicographic maximum).
    Exponential: for N <= 16 only."""
    N = len(score)
    keep = set(range(N - W, N))
    for r, q in enumerate(quota):
        cand = [t for t in range(N - W) if roles[t] == r]
        if q <= 0 or not cand:
            continue
        q = min(q, len(cand))
        best = None
        for sub in itertools.combinations(cand, q):
            ordered = sorted(sub, key=lambda t: _rank(score[t], t))
            if best is None or _lex_better(ordered, best, score):
                best = ordered
        keep.update(best)
    return sorted(keep)


def _lex_better(a, b, score):
    for x, y in zip(a, b):
        if x == y:
            continue
        return _better(score[x], x, score[y], y)
    return False


def decode_loops(q_heads, k, v, keep, scale=None):
    """Decode through a keep-set with loops: for each head, the softmax of the
    scaled dot products over the kept positions only, then the weighted sum of
    their value rows (Algorithm 1, last step)."""
    d = len(q_heads[0])
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    keep = sorted(set(int(t) for t in keep))
    out = []
    for q in q_heads:
        if not keep:
            out.append([0.0] * d)
            continue
        logits = [scale * _dot(q, k[t]) for t in keep]
        m = max(logits)
        w = [math.exp(x - m) for x in logits]
        z = sum(w)
        out.append([sum(w[i] * float(v[t][c]) for i, t in enumerate(keep)) / z for c in range(d)])
    return out


def quest_loops(q_win, k, page):
    """Page bounds of the one-shot Quest analogue with loops (§4.1 "Query-aware
    baseline"): q_win[h][i] window rows of head h, k the key rows; returns the
    score of every position (window positions: +inf)."""
    G, W, d = len(q_win), len(q_win[0]), len(k[0])
    N = len(k)
    P = N - W
    qbar = [[sum(float(q_win[h][i][c]) for i in range(W)) / W for c in range(d)] for h in range(G)]
    out = [math.inf] * N
    for start in range(0, P, page):
        rows = list(range(start, min(start + page, P)))
        bound = 0.0
        for h in range(G):
            for c in range(d):
                lo = min(float(k[t][c]) for t in rows)
                hi = max(float(k[t][c]) for t in rows)
                bound += max(qbar[h][c] * lo, qbar[h][c] * hi)
        for t in rows:
            out[t] = bound
    return out
