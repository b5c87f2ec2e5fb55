"""NumPy float64 definitions of the role-conditional eviction hot path.

TEST INFRASTRUCTURE ONLY (see the package docstring): never imported by the
product path.

Notation (paper §2, §4 and Algorithm 1):
  N   cached tokens, W observation window (last W prefill queries),
  G   query heads per KV head (grouped-query attention),
  P   candidate prefix [0, N-W); the window [N-W, N) is always kept,
  B   budget (fraction of the N tokens that may stay in the cache),
  R   number of role buckets, alpha[r] the per-bucket weight.

Readings taken where the paper is silent (each one is restated in the function
that uses it):
  R1  softmax scale defaults to 1/sqrt(d);
  R2  query head h reads KV head h // G (contiguous groups) and the mass of the
      G heads of a group is summed;
  R3  the window queries sit at positions N-W .. N-1 and are causal inside the
      window (query at position i sees keys t <= i);
  R4  the max-pool is stride 1, same length, padded with -inf and runs over the
      candidate prefix only; window scores are left unpooled;
  R5  the window is inside the budget: K = min(N, ceil(B*N)), K_p = max(0, K-W);
  R6  the bucket quotas split K_p (the n_kv of the per-bucket ceiling with the
      window taken out);
  R7  every ceiling is taken as ceil(x - 1e-9) so that binary64 products such
      as 0.07*100 = 7.000000000000001 round to the intended integer;
  R8  alpha is renormalised over the buckets that take part (alpha > 0 and at
      least one candidate token);
  R9  "redistribute unused budget from saturated buckets": a bucket whose
      ceiling share exceeds its population keeps its whole population and the
      budget it cannot use is re-split, by the same proportional-ceiling rule,
      over the buckets still open; repeated until no bucket overflows;
  R10 budget left once every positive-weight bucket is full stays unspent; a
      budget B >= 1 is the full-cache baseline and keeps all N tokens;
  R12 equal scores: the lower token index wins;
  R13 -0.0 ranks equal to +0.0 and NaN ranks below every number;
  R17 the No-X counterfactual (§4 "Counterfactual", Table 2) keeps the same
      K_p prefix slots as the other policies, filled by score from the prefix
      tokens whose role is not X; when fewer such tokens exist the slots left
      stay empty;
  R18 fair eviction (§4.1 "Fair-eviction baseline") retains every bucket at the
      same rate: bucket r keeps ceil(n_r * K_p / P) of its n_r candidates, the
      ceiling of R7 as for the role policy;
  R20 the one-shot Quest analogue (§4.1 "Query-aware baseline") scores pages of
      16 consecutive prefix tokens (the last one ragged; the window belongs to
      no page) by Quest's per-channel key bound against each head's mean
      window query, summed over the G heads of the group (as R2 sums their
      mass); every token carries its page's bound, window tokens +inf, and the
      same per-bucket top-k then keeps whole pages in bound order (the lower
      index first on ties), the last one cut at the budget;
  R21 the linear role probe (§6 "Deployment: a linear role probe") scores
      role r of token t as b[r] + sum over offsets o = -2..2 of
      W[o + 2, id(t + o), r], skipping positions outside the sequence and ids
      outside the vocabulary; the sum is taken in float32 in offset order
      (b first), the precision the probe is stored in, and the label is the
      argmax, the lowest role on ties.
"""

from __future__ import annotations

import math

import numpy as np

__all__ = [
    "CEIL_GUARD",
    "ceil_guarded",
    "causal_logits",
    "causal_softmax",
    "snapkv_mass",
    "window_lse",
    "h2o_mass",
    "maxpool_prefix",
    "snapkv_score",
    "quest_page_bounds",
    "quest_mass",
    "quest_score",
    "h2o_score",
    "role_counts",
    "role_allocate",
    "role_allocate_batch",
    "role_map",
    "no_role_policy",
    "no_role_keep",
    "fair_allocate",
    "fair_allocate_batch",
    "rank_key",
    "select_keep",
    "kv_compact",
    "PROBE_OFFSETS",
    "probe_logits",
    "probe_roles",
    "decode_attention",
    "masked_decode_attention",
    "decode_attention_batch",
    "per_role_mean_mass",
    "retention_rate",
    "retained_snr_db",
]

CEIL_GUARD = 1e-9


def ceil_guarded(x: float) -> int:
    """Integer ceiling with the binary64 guard of reading R7."""
    return int(math.ceil(float(x) - CEIL_GUARD))


# ---------------------------------------------------------------------------
# Scores: causal softmax, H2O accumulated mass, SnapKV windowed mass, pool
# ---------------------------------------------------------------------------

def causal_logits(q_rows: np.ndarray, q_pos: np.ndarray, k: np.ndarray,
                  scale: float) -> np.ndarray:
    """Scaled logits x[r, t] = scale * <q_r, k_t> for keys t <= q_pos[r].

    Entries with t > q_pos[r] (future keys) are -inf: the prefill attention the
    scores are read from is causal (§2, p_t(q) is the attention probability a
    query q puts on key t).  float64 throughout.
    """
    q = np.asarray(q_rows, dtype=np.float64)
    kk = np.asarray(k, dtype=np.float64)
    x = scale * (q @ kk.T)
    t = np.arange(kk.shape[0])
    x = np.where(t[None, :] <= np.asarray(q_pos)[:, None], x, -np.inf)
    return x


def causal_softmax(x: np.ndarray) -> np.ndarray:
    """Row softmax of causal logits (masked entries, -inf, get probability 0).

    p[r, t] = exp(x[r, t] - m_r) / sum_u exp(x[r, u] - m_r), m_r = max_u x[r, u],
    the probability p_t(q) of §2 for query row r.
    """
    m = np.max(x, axis=1, keepdims=True)
    e = np.exp(x - m)
    return e / np.sum(e, axis=1, keepdims=True)


def snapkv_mass(q_win: np.ndarray, k: np.ndarray, scale: float | None = None) -> np.ndarray:
    """SnapKV windowed mass of one KV head (§2; §4 "SnapKV mechanism";
    Algorithm 1, windowed-mass step).

    q_win : [G, W, d] the last W prefill queries of the G query heads that
            share this KV head (readings R2, R3);
    k     : [N, d] the cached keys.
    Returns s[N] with s(t) = sum over heads h and window queries i >= t of
    p_h[i, t].  Summed over the G heads (R2).
    """
    q_win = np.asarray(q_win, dtype=np.float64)
    G, W, d = q_win.shape
    N = k.shape[0]
    if scale is None:
        scale = 1.0 / math.sqrt(d)                       # R1
    pos = np.arange(N - W, N)                            # R3
    s = np.zeros(N, dtype=np.float64)
    for h in range(G):
        p = causal_softmax(causal_logits(q_win[h], pos, k, scale))
        s += p.sum(axis=0)
    return s


def window_lse(q_win: np.ndarray, k: np.ndarray, scale: float | None = None) -> np.ndarray:
    """Natural-log log-sum-exp of every window row over its causal keys, the
    statistic a prefill attention kernel returns per query row: [G, W] with
    lse[h, i] = log sum_{t <= N-W+i} exp(scale <q_h[i], k_t>).  With it,
    p_h[i, t] = exp(x - lse) (§2)."""
    q_win = np.asarray(q_win, dtype=np.float64)
    G, W, d = q_win.shape
    N = k.shape[0]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    pos = np.arange(N - W, N)
    out = np.zeros((G, W), dtype=np.float64)
    for h in range(G):
        x = causal_logits(q_win[h], pos, k, scale)
        m = np.max(x, axis=1, keepdims=True)
        out[h] = (m + np.log(np.sum(np.exp(x - m), axis=1, keepdims=True)))[:, 0]
    return out


def h2o_mass(q: np.ndarray, k: np.ndarray, scale: float | None = None,
             row_block: int = 2048) -> np.ndarray:
    """H2O heavy-hitter score of one KV head: s(t) = sum_q p_t(q) over every
    prefill query (§2, H2O family), summed over the G query heads (R2).

    q : [G, N, d] all prefill queries of the group, k : [N, d].
    Rows are processed in blocks only to bound memory; each row's softmax is
    the full causal row.
    """
    q = np.asarray(q, dtype=np.float64)
    G, N, d = q.shape
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    s = np.zeros(N, dtype=np.float64)
    for h in range(G):
        for r0 in range(0, N, row_block):
            pos = np.arange(r0, min(N, r0 + row_block))
            p = causal_softmax(causal_logits(q[h, pos], pos, k, scale))
            s += p.sum(axis=0)
    return s


def maxpool_prefix(s: np.ndarray, W: int, kernel: int) -> np.ndarray:
    """1-D max-pool along the KV axis (§4 "SnapKV mechanism", kernel 7;
    Algorithm 1, pooling step), reading R4.

    For t in the prefix P = [0, N-W): s~(t) = max{ s(u) : u in P, |u-t| <= kernel//2 }.
    Window positions keep their raw score.
    """
    if kernel < 1 or kernel % 2 == 0:
        raise ValueError("pool kernel must be odd and >= 1")
    s = np.asarray(s, dtype=np.float64)
    N = s.shape[0]
    P = N - W
    out = s.copy()
    h = kernel // 2
    for t in range(P):
        lo, hi = max(0, t - h), min(P, t + h + 1)
        out[t] = np.max(s[lo:hi])
    return out


def snapkv_score(q_win: np.ndarray, k: np.ndarray, n_kv_heads: int,
                 pool_kernel: int, scale: float | None = None) -> np.ndarray:
    """Pooled SnapKV score for whole tensors.

    q_win [L, B, Hq, W, d], k [L, B, Hkv, N, d] -> score [L, B, Hkv, N]
    (pooled on the prefix, raw on the window).  Query head h belongs to KV head
    h // G with G = Hq / Hkv (R2).
    """
    L, Bt, Hq, W, d = q_win.shape
    N = k.shape[3]
    G = Hq // n_kv_heads
    out = np.zeros((L, Bt, n_kv_heads, N), dtype=np.float64)
    for l in range(L):
        for b in range(Bt):
            for j in range(n_kv_heads):
                s = snapkv_mass(q_win[l, b, j * G:(j + 1) * G], k[l, b, j], scale)
                out[l, b, j] = maxpool_prefix(s, W, pool_kernel)
    return out


def h2o_score(q: np.ndarray, k: np.ndarray, n_kv_heads: int,
              scale: float | None = None) -> np.ndarray:
    """H2O score for whole tensors: q [L, B, Hq, N, d], k [L, B, Hkv, N, d]
    -> [L, B, Hkv, N].  No window and no pool (reading R14: W = 0, kernel 1)."""
    L, Bt, Hq, N, d = q.shape
    G = Hq // n_kv_heads
    out = np.zeros((L, Bt, n_kv_heads, N), dtype=np.float64)
    for l in range(L):
        for b in range(Bt):
            for j in range(n_kv_heads):
                out[l, b, j] = h2o_mass(q[l, b, j * G:(j + 1) * G], k[l, b, j], scale)
    return out


def quest_page_bounds(q_mean: np.ndarray, k: np.ndarray, page: int) -> np.ndarray:
    """Quest's page bound (§4.1 "Query-aware baseline"; R20) for the pages of
    the key rows k [P, d]: page j covers rows [j*page, min((j+1)*page, P)).
    For each head h, sum_c max(qbar_h[c] * kmin_j[c], qbar_h[c] * kmax_j[c])
    with kmin/kmax the per-channel minimum and maximum of the page's keys,
    summed over the heads.  q_mean [G, d].  No score of a key of the page,
    sum_h <qbar_h, k_t>, exceeds its page's bound."""
    q_mean = np.asarray(q_mean, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    P = k.shape[0]
    n_pages = (P + page - 1) // page
    out = np.zeros(n_pages, dtype=np.float64)
    for j in range(n_pages):
        rows = k[j * page:min((j + 1) * page, P)]
        kmin = rows.min(axis=0)
        kmax = rows.max(axis=0)
        out[j] = float(np.sum(np.maximum(q_mean * kmin[None, :], q_mean * kmax[None, :])))
    return out


def quest_mass(q_win: np.ndarray, k: np.ndarray, page: int = 16) -> np.ndarray:
    """Token scores of the one-shot Quest analogue for one KV head (R20):
    q_win [G, W, d] window queries, k [N, d].  Prefix token t gets the bound
    of page t // page; window tokens get +inf (always kept)."""
    q_win = np.asarray(q_win, dtype=np.float64)
    N = np.asarray(k).shape[0]
    W = q_win.shape[1]
    P = N - W
    q_mean = q_win.mean(axis=1)                       # each head's mean window query
    s = np.full(N, np.inf, dtype=np.float64)
    if P > 0:
        bounds = quest_page_bounds(q_mean, np.asarray(k)[:P], page)
        s[:P] = bounds[np.arange(P) // page]
    return s


def quest_score(q_win: np.ndarray, k: np.ndarray, n_kv_heads: int, page: int = 16) -> np.ndarray:
    """quest_mass for whole tensors: q_win [L, B, Hq, W, d], k [L, B, Hkv, N, d]
    -> [L, B, Hkv, N]."""
    L, Bt, Hq, W, d = q_win.shape
    N = k.shape[3]
    G = Hq // n_kv_heads
    out = np.zeros((L, Bt, n_kv_heads, N), dtype=np.float64)
    for l in range(L):
        for b in range(Bt):
            for j in range(n_kv_heads):
                out[l, b, j] = quest_mass(q_win[l, b, j * G:(j + 1) * G], k[l, b, j], page)
    return out


# ---------------------------------------------------------------------------
# Role-conditional allocation (§4.1, Algorithm 1 per-bucket top-k and
# redistribution steps)
# ---------------------------------------------------------------------------

def role_counts(roles: np.ndarray, R: int, W: int) -> np.ndarray:
    """n_r: number of candidate-prefix tokens (t < N-W) carrying role r."""
    roles = np.asarray(roles)
    N = roles.shape[0]
    pre = roles[:N - W]
    return np.array([int(np.sum(pre == r)) for r in range(R)], dtype=np.int64)


def role_allocate(roles: np.ndarray, R: int, alpha, budget: float, W: int):
    """Per-bucket quotas for one sample (§4.1 role policy; Algorithm 1).

    Returns (quota[R], kept) where quota[r] tokens of bucket r are kept from
    the candidate prefix and kept = W + sum(quota) counts the window too.
    Readings R5-R10.
    """
    roles = np.asarray(roles)
    N = int(roles.shape[0])
    alpha = [float(a) for a in alpha]
    if len(alpha) != R:
        raise ValueError("alpha must have R entries")
    if not (0 <= W <= N):
        raise ValueError("need 0 <= W <= N")
    if budget <= 0:
        raise ValueError("budget must be > 0")
    if np.any(roles < 0) or np.any(roles >= R):
        raise ValueError("role label outside [0, R)")
    if any(a < 0 for a in alpha) or sum(alpha) <= 0:
        raise ValueError("alpha must be >= 0 with a positive sum")
    n = role_counts(roles, R, W)
    if budget >= 1.0:                                  # R10: full-cache baseline
        return n.copy(), N
    K = min(N, ceil_guarded(budget * N))               # R5
    rem = max(0, K - W)                                # R5/R6
    quota = np.zeros(R, dtype=np.int64)
    open_ = [r for r in range(R) if alpha[r] > 0 and n[r] > 0]   # R8
    while rem > 0 and open_:
        total = sum(alpha[r] for r in open_)
        share = {r: ceil_guarded(alpha[r] / total * rem) for r in open_}
        full = [r for r in open_ if share[r] > n[r]]   # R9: cannot use its share
        if not full:
            for r in open_:
                quota[r] = share[r]
            break
        for r in full:
            quota[r] = n[r]
            rem -= int(n[r])
        open_ = [r for r in open_ if r not in full]
        rem = max(rem, 0)
    return quota, int(W + quota.sum())


def role_allocate_batch(roles: np.ndarray, R: int, alpha, budget: float, W: int):
    """role_allocate for every sample of roles [B, N]: (quota[B, R], kept[B], k_cap)."""
    roles = np.asarray(roles)
    Bt = roles.shape[0]
    quota = np.zeros((Bt, R), dtype=np.int64)
    kept = np.zeros(Bt, dtype=np.int64)
    for b in range(Bt):
        quota[b], kept[b] = role_allocate(roles[b], R, alpha, budget, W)
    return quota, kept, int(kept.max()) if Bt else 0


# ---------------------------------------------------------------------------
# Other policies over the same partition-and-allocate container: the No-X
# counterfactual (§4 "Counterfactual", Table 2) and fair eviction (§4.1)
# ---------------------------------------------------------------------------

def role_map(roles: np.ndarray, bucket_of) -> np.ndarray:
    """Bucket labels: token t goes to bucket bucket_of[roles[t]]."""
    roles = np.asarray(roles)
    bucket_of = [int(x) for x in bucket_of]
    if np.any(roles < 0) or np.any(roles >= len(bucket_of)):
        raise ValueError("role label outside the map")
    out = np.empty(roles.shape, dtype=np.int8)
    for r, b in enumerate(bucket_of):
        out[roles == r] = b
    return out


def no_role_policy(x: int, n_roles: int):
    """No-X as a two-bucket policy: role x alone in bucket 1 with weight 0,
    every other role in bucket 0 with weight 1.  Returns (bucket_of, alpha)."""
    if not 0 <= x < n_roles:
        raise ValueError("banned role outside [0, n_roles)")
    bucket_of = [1 if r == x else 0 for r in range(n_roles)]
    return bucket_of, [1.0, 0.0]


def no_role_keep(score: np.ndarray, roles: np.ndarray, x: int, budget: float,
                 W: int) -> np.ndarray:
    """Kept indices of one segment under No-X, from the definition (R17): the
    window, plus the K_p best-scoring prefix tokens whose role is not x (score
    descending, index ascending; NaN below every number), ascending."""
    score = np.asarray(score, dtype=np.float64)
    roles = np.asarray(roles)
    N = score.shape[0]
    if budget >= 1.0:
        return np.arange(N, dtype=np.int64)
    K = min(N, ceil_guarded(budget * N))
    K_p = max(0, K - W)
    nan = np.isnan(score)
    allowed = [t for t in range(N - W) if roles[t] != x]
    allowed.sort(key=lambda t: (1, 0.0, t) if nan[t] else (0, -score[t], t))
    kept = allowed[:K_p] + list(range(N - W, N))
    return np.array(sorted(kept), dtype=np.int64)


def fair_allocate(roles: np.ndarray, R: int, budget: float, W: int):
    """Fair-eviction quotas of one sample (R18): (quota[R], kept)."""
    roles = np.asarray(roles)
    N = int(roles.shape[0])
    if not (0 <= W <= N):
        raise ValueError("need 0 <= W <= N")
    if budget <= 0:
        raise ValueError("budget must be > 0")
    if np.any(roles < 0) or np.any(roles >= R):
        raise ValueError("role label outside [0, R)")
    n = role_counts(roles, R, W)
    if budget >= 1.0:
        return n.copy(), N
    if n.sum() == 0:                       # no candidate prefix: the window alone
        return np.zeros(R, dtype=np.int64), W
    # the weight of a bucket is its own population: the same rate everywhere
    return role_allocate(roles, R, [float(c) for c in n], budget, W)


def fair_allocate_batch(roles: np.ndarray, R: int, budget: float, W: int):
    """fair_allocate for every sample of roles [B, N]: (quota[B, R], kept[B], k_cap)."""
    roles = np.asarray(roles)
    Bt = roles.shape[0]
    quota = np.zeros((Bt, R), dtype=np.int64)
    kept = np.zeros(Bt, dtype=np.int64)
    for b in range(Bt):
        quota[b], kept[b] = fair_allocate(roles[b], R, budget, W)
    return quota, kept, int(kept.max()) if Bt else 0


# ---------------------------------------------------------------------------
# Selection and compaction
# ---------------------------------------------------------------------------

def rank_key(score: np.ndarray):
    """Ranking keys (R13): (is_nan, value) with NaN values replaced by 0.
    Candidates are ordered by is_nan ascending (every number, -inf included,
    before every NaN), then by value descending, then by index ascending.
    -0.0 already compares equal to +0.0 in IEEE arithmetic, so equal values
    fall back to the index."""
    s = np.asarray(score, dtype=np.float64)
    nan = np.isnan(s)
    return nan, np.where(nan, 0.0, s)


def select_keep(score: np.ndarray, roles: np.ndarray, quota, W: int) -> np.ndarray:
    """Kept token indices of one (layer, batch, KV head), ascending.

    Within bucket r the candidate tokens (t < N-W, role r) are ranked by score
    descending, then index ascending (R12), and the first quota[r] are kept
    (Algorithm 1, per-bucket top-k).  The window [N-W, N) is always kept.
    Labels outside [0, len(quota)) are never kept.
    """
    score = np.asarray(score)
    roles = np.asarray(roles)
    N = score.shape[0]
    nan, key = rank_key(score)
    keep = [np.arange(N - W, N)]
    t_all = np.arange(N - W)
    for r, q in enumerate(quota):
        cand = t_all[roles[:N - W] == r]
        if q <= 0 or cand.size == 0:
            continue
        order = np.lexsort((cand, -key[cand], nan[cand]))      # last key is primary
        keep.append(cand[order[:int(q)]])
    return np.sort(np.concatenate(keep)).astype(np.int64)


def kv_compact(kv: np.ndarray, idx: np.ndarray) -> np.ndarray:
    """Compacted rows kv[idx] of one (layer, batch, KV head): a pure copy,
    the dense cache a compacting implementation keeps (§6, systems cost)."""
    return np.asarray(kv)[np.asarray(idx)]


# ---------------------------------------------------------------------------
# Linear role probe (§6 "Deployment: a linear role probe"): role labels from a
# multinomial logistic regression over the token ids at t-2 .. t+2
# ---------------------------------------------------------------------------

PROBE_OFFSETS = (-2, -1, 0, 1, 2)


def probe_logits(ids: np.ndarray, weight: np.ndarray, bias: np.ndarray) -> np.ndarray:
    """Float32 logits [n, R] of one sequence of token ids (R21): weight
    [5, V, R] holds one table per offset of PROBE_OFFSETS, bias [R].  Each
    logit is accumulated in float32, bias first, then the offsets in order."""
    ids = np.asarray(ids, dtype=np.int64)
    weight = np.asarray(weight, dtype=np.float32)
    bias = np.asarray(bias, dtype=np.float32)
    n = ids.shape[0]
    V, R = weight.shape[1], weight.shape[2]
    out = np.empty((n, R), dtype=np.float32)
    for t in range(n):
        acc = bias.copy()
        for j, o in enumerate(PROBE_OFFSETS):
            p = t + o
            if 0 <= p < n and 0 <= ids[p] < V:
                acc = (acc + weight[j, ids[p]]).astype(np.float32)
        out[t] = acc
    return out


def probe_roles(ids: np.ndarray, weight: np.ndarray, bias: np.ndarray) -> np.ndarray:
    """Role label of every token of ids [B, N] (or [N]): the argmax of its
    float32 logits, the lowest role on ties.  int8, same shape as ids."""
    ids = np.asarray(ids)
    flat = ids.reshape(-1, ids.shape[-1])
    out = np.empty(flat.shape, dtype=np.int8)
    for b in range(flat.shape[0]):
        out[b] = np.argmax(probe_logits(flat[b], weight, bias), axis=1)   # first maximum
    return out.reshape(ids.shape)


# ---------------------------------------------------------------------------
# Decoding through the keep-set (Algorithm 1, last step; §3 "Setup"; §6
# "Systems cost": a compacting implementation attends over the kept rows only)
# ---------------------------------------------------------------------------

def _softmax_rows(x: np.ndarray) -> np.ndarray:
    """Row softmax; a row whose entries are all -inf gets probability 0 everywhere."""
    m = np.max(x, axis=1, keepdims=True)
    m = np.where(np.isneginf(m), 0.0, m)
    e = np.exp(x - m)
    z = np.sum(e, axis=1, keepdims=True)
    return np.divide(e, z, out=np.zeros_like(e), where=z > 0)


def decode_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
                     scale: float | None = None) -> np.ndarray:
    """One decode query per head over the rows of a cache (one KV head).

    q [G, d] (the G query heads of the group), k, v [n, d]; returns [G, d]
    with o_h = sum_t softmax_t(scale <q_h, k_t>) v_t.  An empty cache (n = 0)
    gives zeros.  Applied to the compacted rows K[idx], V[idx] this is the
    decode of a compacting implementation.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    G, d = q.shape
    if k.shape[0] == 0:
        return np.zeros((G, d), dtype=np.float64)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    x = scale * (q @ k.T)
    return _softmax_rows(x) @ v


def masked_decode_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, keep,
                            scale: float | None = None) -> np.ndarray:
    """Decode through a keep-mask over the full cache, the form the paper's
    harness uses: the logit of every position outside ``keep`` is set to -inf
    and the softmax runs over all N positions.  q [G, d], k, v [N, d]."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    d = q.shape[1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    mask = np.zeros(k.shape[0], dtype=bool)
    mask[np.asarray(keep, dtype=np.int64)] = True
    x = scale * (q @ k.T)
    x[:, ~mask] = -np.inf
    return _softmax_rows(x) @ v


def decode_attention_batch(q: np.ndarray, k_c: np.ndarray, v_c: np.ndarray,
                           count: np.ndarray, scale: float | None = None) -> np.ndarray:
    """decode_attention for whole tensors: q [L, B, Hq, d], k_c, v_c
    [L, B, Hkv, k_cap, d], count [L, B, Hkv] (rows in use, clamped to
    [0, k_cap]) -> [L, B, Hq, d].  Query head h reads KV head h // G (R2)."""
    L, Bt, Hq, d = q.shape
    Hkv, k_cap = k_c.shape[2], k_c.shape[3]
    G = Hq // Hkv
    out = np.zeros((L, Bt, Hq, d), dtype=np.float64)
    for l in range(L):
        for b in range(Bt):
            for j in range(Hkv):
                n = int(min(max(int(count[l, b, j]), 0), k_cap))
                out[l, b, j * G:(j + 1) * G] = decode_attention(
                    q[l, b, j * G:(j + 1) * G], k_c[l, b, j, :n], v_c[l, b, j, :n], scale)
    return out


# ---------------------------------------------------------------------------
# Diagnostics (§3): per-role mass, retention rate, retained-state SNR
# ---------------------------------------------------------------------------

def per_role_mean_mass(score: np.ndarray, roles: np.ndarray, R: int,
                       upto: int | None = None) -> np.ndarray:
    """Mean per-token mass of each role (§3 "Mass concentration", Fig. 1).
    Only positions t < upto are counted (default: all).  NaN for empty roles."""
    s = np.asarray(score, dtype=np.float64)
    roles = np.asarray(roles)
    n = s.shape[0] if upto is None else upto
    out = np.full(R, np.nan)
    for r in range(R):
        m = roles[:n] == r
        if np.any(m):
            out[r] = float(np.mean(s[:n][m]))
    return out


def retention_rate(idx: np.ndarray, roles: np.ndarray, R: int,
                   upto: int | None = None) -> np.ndarray:
    """Fraction of each role's tokens that are kept (§3 "Retention bias",
    Table 1).  Only positions t < upto are counted (default: all)."""
    roles = np.asarray(roles)
    n = roles.shape[0] if upto is None else upto
    kept = np.zeros(roles.shape[0], dtype=bool)
    kept[np.asarray(idx)] = True
    out = np.full(R, np.nan)
    for r in range(R):
        m = roles[:n] == r
        if np.any(m):
            out[r] = float(np.mean(kept[:n][m]))
    return out


def retained_snr_db(signal_energy: float, noise_energy: float) -> float:
    """Retained-state SNR of §3: 10 log10 of the per-token energy of the
    answer-carrying role over that of the structural role."""
    return 10.0 * math.log10(signal_energy / noise_energy)
