"""The whole eviction step (one pass of the hot path) over resident tensors.

score (SnapKV windowed + pooled, H2O, or the one-shot Quest page bound)  ->
role allocation (host)  ->
per-role top-k  ->  K/V compaction.  Buffers are allocated once by
``EvictBuffers`` so that repeated steps allocate nothing.

``Policy`` names how the budget is split over buckets: the role-conditional
weights of §4.1, fair eviction (§4.1, the same rate for every bucket) or the
No-X counterfactual of §4 (one role banned from the prefix).
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import binding as kb


@dataclass(frozen=True)
class Policy:
    """A split of the prefix budget over R buckets.

    alpha      per-bucket weights (role-conditional policy), or None for fair
               eviction, where every sample weights each bucket by its own
               candidate count.
    bucket_of  map from role label to bucket, or None when the role labels are
               the buckets.  The step itself takes bucket labels: relabel the
               roles once with ``buckets`` and keep the result resident.
    """
    R: int
    alpha: tuple | None = None
    bucket_of: tuple | None = None

    @staticmethod
    def role(alpha) -> "Policy":
        a = tuple(float(x) for x in alpha)
        return Policy(len(a), a)

    @staticmethod
    def fair(R: int) -> "Policy":
        return Policy(int(R), None)

    @staticmethod
    def no_role(x: int, n_roles: int) -> "Policy":
        """No-X: role x alone in bucket 1 with weight 0, the rest in bucket 0."""
        if not 0 <= x < n_roles:
            raise ValueError("banned role outside [0, n_roles)")
        return Policy(2, (1.0, 0.0), tuple(1 if r == x else 0 for r in range(n_roles)))

    def buckets(self, roles_host: np.ndarray) -> np.ndarray:
        """Bucket labels of roles [B, N] (host int8)."""
        if self.bucket_of is None:
            return np.asarray(roles_host, dtype=np.int8)
        return kb.role_map(roles_host, self.bucket_of)

    def allocate(self, buckets_host: np.ndarray, budget: float, W: int):
        """(quota [B, R], kept [B], k_cap) for bucket labels [B, N]."""
        if self.alpha is None:
            return kb.role_allocate_fair(buckets_host, self.R, budget, W)
        return kb.role_allocate(buckets_host, self.R, self.alpha, budget, W)


# The probe's roles (§6: KEY, VALUE, DELIM, HEADER, PROSE, WS) in the
# allocation's four buckets (SINK 0, KEY 1, VALUE 2, OTHER 3): delimiters and
# whitespace are the sink bucket, headers join the keys, prose is OTHER.
PROBE_TO_BUCKET = (1, 2, 0, 1, 3, 0)


def probe_buckets(ids, weight, bias, bucket_of=PROBE_TO_BUCKET):
    """Bucket labels from the linear role probe on the device: returns (host
    int8 [B, N], device int8 [B, N]).  The host copy feeds the allocation."""
    labels = kb.role_probe(ids, weight, bias)
    buckets = kb.role_map(labels.cpu().numpy(), bucket_of)
    import torch
    return buckets, torch.from_numpy(buckets).to(ids.device)


def as_policy(policy) -> Policy:
    """A Policy, or a plain weight sequence read as the role-conditional policy."""
    return policy if isinstance(policy, Policy) else Policy.role(policy)


@dataclass
class EvictBuffers:
    score: object
    ws_score: object
    ws_topk: object
    quota_host: object   # pinned int32 [B, R]
    quota_dev: object
    idx: object
    count: object
    k_out: object
    v_out: object
    k_cap: int
    copy_done: object = None   # event after the last quota upload from quota_host
    hist: object = None        # per-tile role histograms of the fused SnapKV epilogue, [L, words per layer]


def alloc_buffers(k, n_q_heads: int, W: int, R: int, k_cap: int, scorer: str = "snapkv",
                  with_v: bool = True, fused: bool = False) -> EvictBuffers:
    """Buffers of repeated eviction steps.  fused (SnapKV only): the score's
    pool epilogue counts the top-k's first digit per role bucket
    (snapkv_score_hist / topk_select_hist) and the histograms live here.  Off
    by default: on the 32-layer N = 32768 step the counting adds more to the
    pool (about 100 us) than it takes off the top-k (about 25 us)."""
    import torch
    L, B, Hkv, N, d = k.shape
    dev = k.device
    if scorer == "snapkv":
        wsb = kb.snapkv_workspace_size(L, B, n_q_heads, Hkv, N, W, d)
    elif scorer == "quest":
        wsb = kb.quest_workspace_size(L, B, n_q_heads, Hkv, d)
    else:
        wsb = kb.h2o_workspace_size(L, B, n_q_heads, Hkv, N, d)
    return EvictBuffers(
        score=torch.empty((L, B, Hkv, N), dtype=torch.float32, device=dev),
        ws_score=torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev),
        ws_topk=torch.empty(kb.topk_workspace_size(L, B, Hkv, N, R), dtype=torch.uint8, device=dev),
        quota_host=torch.zeros((B, R), dtype=torch.int32).pin_memory(),
        quota_dev=torch.zeros((B, R), dtype=torch.int32, device=dev),
        idx=torch.full((L, B, Hkv, k_cap), -1, dtype=torch.int32, device=dev),
        count=torch.zeros((L, B, Hkv), dtype=torch.int32, device=dev),
        k_out=torch.zeros((L, B, Hkv, k_cap, d), dtype=k.dtype, device=dev),
        v_out=torch.zeros((L, B, Hkv, k_cap, d), dtype=k.dtype, device=dev) if with_v else None,
        k_cap=k_cap,
        hist=(torch.empty((L, kb.role_hist_size(1, B, Hkv, N, R) // 4), dtype=torch.int32, device=dev)
              if fused and scorer == "snapkv" else None),
    )


def _fused(bufs, scorer, lse_win):
    return bufs.hist is not None and scorer == "snapkv" and lse_win is None


def _score(q, k, bufs, scorer, pool_k, scale, page, l0, l1, stream=None, lse_win=None, roles_dev=None, R=0):
    """Score layers [l0, l1) into bufs.score[l0:l1] on ``stream`` (None: current);
    with the fused role epilogue also their role histograms."""
    if _fused(bufs, scorer, lse_win):
        kb.snapkv_score_hist(q[l0:l1], k[l0:l1], roles_dev, R, pool_k, scale, score=bufs.score[l0:l1],
                             hist=bufs.hist[l0:l1], workspace=bufs.ws_score, stream=stream)
    elif scorer == "snapkv" and lse_win is not None:
        kb.snapkv_score_lse(q[l0:l1], k[l0:l1], lse_win[l0:l1], pool_k, scale, score=bufs.score[l0:l1],
                            workspace=bufs.ws_score, stream=stream)
    elif scorer == "snapkv":
        kb.snapkv_score(q[l0:l1], k[l0:l1], pool_k, scale, score=bufs.score[l0:l1],
                        workspace=bufs.ws_score, stream=stream)
    elif scorer == "quest":
        kb.quest_score(q[l0:l1], k[l0:l1], page, score=bufs.score[l0:l1], workspace=bufs.ws_score,
                       stream=stream)
    else:
        kb.h2o_score(q[l0:l1], k[l0:l1], scale, score=bufs.score[l0:l1], workspace=bufs.ws_score,
                     stream=stream)


def _select(k, v, roles_dev, bufs, W, R, l0, l1, stream=None, events=None, fused=False):
    """Top-k and compaction of layers [l0, l1) on ``stream`` (None: current);
    ``events``, three torch.cuda.Event, are recorded before the top-k, between
    the two calls and after the compaction.  fused: the score call counted the
    first digit (bufs.hist)."""
    if events is not None:
        events[0].record(stream)
    if fused:
        kb.topk_select_hist(bufs.score[l0:l1], roles_dev, bufs.quota_dev, bufs.hist[l0:l1], W, R, bufs.k_cap,
                            idx_out=bufs.idx[l0:l1], count_out=bufs.count[l0:l1], workspace=bufs.ws_topk,
                            stream=stream)
    else:
        kb.topk_select(bufs.score[l0:l1], roles_dev, bufs.quota_dev, W, R, bufs.k_cap,
                       idx_out=bufs.idx[l0:l1], count_out=bufs.count[l0:l1], workspace=bufs.ws_topk,
                       stream=stream)
    if events is not None:
        events[1].record(stream)
    kb.kv_compact(k[l0:l1], None if v is None else v[l0:l1], bufs.idx[l0:l1], bufs.count[l0:l1],
                  k_out=bufs.k_out[l0:l1], v_out=None if bufs.v_out is None else bufs.v_out[l0:l1],
                  stream=stream)
    if events is not None:
        events[2].record(stream)


def _upload_quotas(policy, roles_host, budget, W, bufs):
    """Work out the quotas on the host and queue their upload (pinned host
    buffer to device) on the current stream; returns (quota, kept)."""
    import torch
    quota, kept, k_cap = policy.allocate(roles_host, budget, W)
    if k_cap > bufs.k_cap:
        raise ValueError(f"buffers hold {bufs.k_cap} rows, the allocation keeps {k_cap}")
    if bufs.copy_done is None:
        bufs.copy_done = torch.cuda.Event()
    bufs.copy_done.synchronize()          # the previous upload has left quota_host
    bufs.quota_host.numpy()[...] = quota
    bufs.quota_dev.copy_(bufs.quota_host, non_blocking=True)
    bufs.copy_done.record()
    return quota, kept


def evict(q, k, v, roles_host: np.ndarray, roles_dev, policy, budget: float, W: int,
          pool_k: int, bufs: EvictBuffers, scorer: str = "snapkv", scale: float = 0.0,
          score_events=None, page: int = 16, chunks: int = 1, side_stream=None, lse_win=None,
          select_events=None):
    """One eviction step; returns (quota [B, R] host, kept [B] host).

    q is the window queries [L, B, Hq, W, d] (SnapKV; Quest, which scores
    pages of ``page`` tokens and ignores pool_k) or all queries [L, B, Hq, N, d]
    (H2O, which uses W = 0 and no pool).  roles_host / roles_dev are the bucket
    labels [B, N] of ``policy`` (a Policy, or the weights of the
    role-conditional policy).  ``score_events``, a pair of torch.cuda.Event,
    brackets the score calls on the launch stream, and ``select_events``, three
    events, bracket the top-k and the compaction (unchunked steps only).
    ``lse_win`` (SnapKV only),
    the window rows' log-sum-exp [L, B, Hq, W] as the prefill attention
    returned it, lets the score read K once.

    The score does not depend on the quotas: it is queued first, and the host
    works the quotas out from the labels and queues their upload while the
    device scores (the top-k, queued after the upload, uses them), so the host
    allocation adds nothing to the step's device time.  A ValueError for
    buffers too small for the allocation is therefore raised after the score
    was queued.  With ``chunks`` > 1 and a ``side_stream``, the quotas come
    first; the layers are then scored in that many chunks on the current stream
    while the top-k and compaction of each scored chunk run on the side stream,
    overlapping the scoring of the next; the current stream waits for the side
    stream before returning."""
    import torch
    policy = as_policy(policy)
    R = policy.R
    L = k.shape[0]
    main = torch.cuda.current_stream()
    fused = _fused(bufs, scorer, lse_win)
    if chunks <= 1 or side_stream is None:
        if score_events is not None:
            score_events[0].record(main)
        _score(q, k, bufs, scorer, pool_k, scale, page, 0, L, stream=main, lse_win=lse_win, roles_dev=roles_dev,
               R=R)
        if score_events is not None:
            score_events[1].record(main)
        quota, kept = _upload_quotas(policy, roles_host, budget, W, bufs)
        _select(k, v, roles_dev, bufs, W, R, 0, L, stream=main, events=select_events, fused=fused)
        return quota, kept
    quota, kept = _upload_quotas(policy, roles_host, budget, W, bufs)
    side_stream.wait_stream(main)         # the quota upload and earlier work
    per = (L + chunks - 1) // chunks
    if score_events is not None:
        score_events[0].record(main)
    for l0 in range(0, L, per):
        l1 = min(L, l0 + per)
        _score(q, k, bufs, scorer, pool_k, scale, page, l0, l1, stream=main, lse_win=lse_win, roles_dev=roles_dev,
               R=R)
        done = torch.cuda.Event()
        done.record(main)
        side_stream.wait_event(done)
        _select(k, v, roles_dev, bufs, W, R, l0, l1, stream=side_stream, fused=fused)
    if score_events is not None:
        score_events[1].record(main)
    main.wait_stream(side_stream)
    return quota, kept


class StepGraph:
    """The device part of an eviction step (quota upload, score, top-k,
    compaction) captured as a HIP graph and replayed, for callers that run the
    step inside captured work (serving loops, launch-bound small shapes).

    The score is one graph; the selection (quota upload, top-k, compaction)
    is captured twice, each copy uploading the quotas from its own pinned host
    buffer, and replays alternate between the two.  A replay queues the score
    graph, works the quotas out on the host while the device scores, writes
    them into its buffer once the replay before last (the previous user of
    that buffer) has finished, and queues its selection graph.  The inputs,
    labels and buffers are the tensors given here (refill them in place
    between replays).  The library launches no memset and allocates nothing,
    so the graphs hold only kernel nodes and the one copy."""

    def __init__(self, q, k, v, roles_dev, policy, W: int, pool_k: int, bufs: EvictBuffers,
                 scorer: str = "snapkv", scale: float = 0.0, page: int = 16, lse_win=None):
        import torch
        self.policy = as_policy(policy)
        self.W = W
        self.bufs = bufs
        L = k.shape[0]
        R = self.policy.R
        self.quota_host = [bufs.quota_host, torch.zeros_like(bufs.quota_host).pin_memory()]

        fused = _fused(bufs, scorer, lse_win)

        def score():
            _score(q, k, bufs, scorer, pool_k, scale, page, 0, L, lse_win=lse_win, roles_dev=roles_dev, R=R)

        def select(src):
            bufs.quota_dev.copy_(src, non_blocking=True)
            _select(k, v, roles_dev, bufs, W, R, 0, L, fused=fused)

        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            score()                     # one eager run on the capture stream first
            select(self.quota_host[0])
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        self.score_graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.score_graph, stream=side):
            score()
        self.graphs = []
        for src in self.quota_host:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                select(src)
            self.graphs.append(g)
        self.done = [torch.cuda.Event(), torch.cuda.Event()]
        for e in self.done:
            e.record()
        self.turn = 0

    def replay(self, roles_host: np.ndarray, budget: float):
        """Replay the captured step on the current stream for these bucket
        labels and budget, allocating on the host while the device scores;
        returns (quota, kept).  A ValueError for buffers too small for the
        allocation is raised after the score was queued."""
        self.score_graph.replay()
        quota, kept, k_cap = self.policy.allocate(roles_host, budget, self.W)
        if k_cap > self.bufs.k_cap:
            raise ValueError(f"buffers hold {self.bufs.k_cap} rows, the allocation keeps {k_cap}")
        i = self.turn
        self.done[i].synchronize()      # the replay before last has read this buffer
        self.quota_host[i].numpy()[...] = quota
        self.graphs[i].replay()
        self.done[i].record()
        self.turn = 1 - i
        return quota, kept
