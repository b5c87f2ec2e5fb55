"""Role-conditional KV-cache eviction on MI355X (gfx950).

The hot path runs in libkve.so (HIP); this package is its thin Python binding:

  snapkv_score   SnapKV windowed score + GQA sum + prefix max-pool
  snapkv_score_lse  the same with the window rows' log-sum-exp supplied (one read of K)
  h2o_score      H2O accumulated score (baseline scorer)
  quest_score    one-shot Quest page-bound score (query-aware baseline scorer)
  role_allocate  per-bucket quotas with redistribution (host)
  role_allocate_fair  equal retention rate per bucket (host)
  role_map       relabel roles into buckets, e.g. the No-X counterfactual (host)
  role_probe     role labels from the linear probe over token ids (device)
  topk_select    per-role top-k with the window kept, ascending indices
  snapkv_score_hist / topk_select_hist  the same two calls with the role
                 histograms counted in the score's pool epilogue (fused)
  kv_compact     dense K/V cache of the kept rows
  snapkv_score_strided, kv_compact_strided, h2o_score_strided, quest_score_strided
                 the same on strided views (e.g. a token-major cache)
  decode_attention  one decode query per head over the compacted cache
  pipeline.evict the whole step over resident tensors
"""

from .binding import (EXPORTED, KveError, decode_attention, decode_workspace_size, snapkv_score_noalloc,  # noqa: F401
                      role_hist_size, snapkv_score_hist, topk_select_hist,
                      h2o_score, h2o_workspace_size, kv_compact, last_error, quest_score, source_hash,
                      quest_workspace_size, role_allocate,
                      role_allocate_fair, role_map, role_probe, snapkv_score, snapkv_score_lse, snapkv_workspace_size,
                      topk_select, topk_workspace_size, Strides, snapkv_score_strided, kv_compact_strided,
                      h2o_score_strided, quest_score_strided)
from . import pipeline  # noqa: F401

__all__ = ["snapkv_score", "snapkv_score_strided", "kv_compact_strided", "Strides", "h2o_score", "h2o_score_strided", "quest_score_strided", "role_allocate", "role_allocate_fair", "role_map",
           "topk_select", "kv_compact", "snapkv_workspace_size", "h2o_workspace_size", "KveError",
           "last_error", "pipeline", "decode_attention", "decode_workspace_size", "quest_score",
           "quest_workspace_size", "role_probe", "snapkv_score_lse", "topk_workspace_size", "source_hash",
           "snapkv_score_noalloc", "role_hist_size", "snapkv_score_hist", "topk_select_hist"]
