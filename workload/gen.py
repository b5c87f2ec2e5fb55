"""Workload definitions and seeded input generation.

Inputs stand in for the paper's schema-dense corpora (indented JSON, deeper
nesting, markdown tables with delimiter bursts; §3 Setup).  No corpus item,
prompt or answer is reproduced: only token-role label sequences with the
corpora's role mix and run structure, and random Q/K/V of the model shapes.

Recipe
------
* roles: a seeded cycle  [SINK run][KEY run][SINK run][VALUE run]  with prose
  (OTHER) runs of mean 8 inserted between cycles, a BOS position (SINK) at
  t=0, an OTHER instruction prefix of 8 tokens and a trailing OTHER question of
  max(W, 16) tokens (so the observation window lands on the question).  Run
  lengths are 1 + Poisson(mean - 1), with means solved from the target mix.
  The "table" pattern adds SINK bursts of 128-384 tokens carrying 5% of the
  tokens.
* Q, K, V: iid N(0, 1) drawn in float32 by torch from a per-(workload, tensor,
  layer) seed, rounded to the workload dtype by round-to-nearest-even.  The
  queries of one KV group also share a random offset of norm ``q_mean`` (3 by
  default), as the queries of a real attention head share a common direction:
  without it the projection of iid queries on any fixed direction is too
  noisy for a key bias to make sinks draw 10-30x the content mass.
* sink bias: for every (layer, batch, KV head) let qbar be the mean of the
  group's queries (the window queries for SnapKV, all queries for H2O) and u
  its direction.  Every SINK key gets beta*u added before rounding, with
  beta = 2c / (scale*|qbar|): this raises the mean query's logit on sink keys
  by 2c standard deviations of the unbiased logits (N(0,1) entries with the
  1/sqrt(d) scale give unit-variance logits).  c is fixed per workload so that
  a sink token draws 10-30x the mean mass of a content token.
"""

from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass

import numpy as np

SINK, KEY, VALUE, OTHER = 0, 1, 2, 3
ROLE_NAMES = ("SINK", "KEY", "VALUE", "OTHER")
NUM_ROLES = 4

PREFIX_LEN = 8
PROSE_MEAN = 8.0
BURST_LO, BURST_HI = 128, 384

__all__ = [
    "SINK", "KEY", "VALUE", "OTHER", "ROLE_NAMES", "NUM_ROLES",
    "Workload", "WORKLOADS", "get_workload", "default_alpha",
    "role_pattern", "make_roles", "make_inputs", "tensor_seed",
]


@dataclass(frozen=True)
class Workload:
    name: str
    L: int
    B: int
    Hq: int
    Hkv: int
    N: int
    W: int
    d: int
    pool_k: int
    dtype: str                      # "bf16" or "f32"
    mix: tuple                      # target fractions (SINK, KEY, VALUE, OTHER)
    budgets: tuple
    pattern: str = "json"           # "json" or "table"
    scorer: str = "snapkv"          # "snapkv", "h2o" or "quest" (window queries, as snapkv)
    sink_c: float = 1.6             # sink-bias multiplier c
    burst_frac: float = 0.0
    q_mean: float = 3.0             # norm of the query offset shared by a KV group

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    "tiny": Workload("tiny", L=1, B=1, Hq=2, Hkv=1, N=512, W=16, d=64, pool_k=5,
                     dtype="f32", mix=(0.35, 0.20, 0.30, 0.15), budgets=(0.10,),
                     sink_c=1.6),
    "layer8k": Workload("layer8k", L=1, B=1, Hq=32, Hkv=8, N=8192, W=32, d=128, pool_k=7,
                        dtype="bf16", mix=(0.35, 0.20, 0.30, 0.15),
                        budgets=(0.05, 0.10, 0.20, 0.50), sink_c=1.6),
    "stack32k": Workload("stack32k", L=32, B=4, Hq=32, Hkv=8, N=32768, W=32, d=128, pool_k=7,
                         dtype="bf16", mix=(0.40, 0.25, 0.25, 0.10), budgets=(0.05,),
                         sink_c=1.6),
    "h2o16k": Workload("h2o16k", L=1, B=1, Hq=32, Hkv=8, N=16384, W=0, d=128, pool_k=1,
                       dtype="bf16", mix=(0.35, 0.20, 0.30, 0.15), budgets=(0.10,),
                       scorer="h2o", sink_c=1.6),
    "long128k": Workload("long128k", L=32, B=1, Hq=32, Hkv=8, N=131072, W=64, d=128, pool_k=7,
                         dtype="bf16", mix=(0.40, 0.15, 0.35, 0.10), budgets=(0.05, 0.20),
                         pattern="table", sink_c=1.6, burst_frac=0.05),
}


def get_workload(name: str) -> Workload:
    return WORKLOADS[name]


def default_alpha(alpha_key: float = 0.0):
    """Role weights over (SINK, KEY, VALUE, OTHER): the paper's policy with
    delimiters and whitespace merged into SINK (0.20 + 0.05), KEY and HEADER
    into KEY (the tuned alpha_KEY), VALUE 0.70 and PROSE as OTHER 0.05 (§4.1)."""
    return [0.25, float(alpha_key), 0.70, 0.05]


def tensor_seed(base: int, *parts) -> int:
    """64-bit seed for one tensor stream, derived with numpy's SeedSequence."""
    words = [int(base)] + [int(p) if isinstance(p, (int, np.integer)) else
                           int.from_bytes(str(p).encode()[:8].ljust(8, b"\0"), "little")
                           for p in parts]
    st = np.random.SeedSequence(words).generate_state(2, dtype=np.uint32)
    return int(st[0]) | (int(st[1] & 0x7FFFFFFF) << 32)


def _run(rng, mean: float) -> int:
    return 1 + int(rng.poisson(max(mean - 1.0, 0.0)))


def role_pattern(N: int, W: int, mix, rng, pattern: str = "json",
                 burst_frac: float = 0.0) -> np.ndarray:
    """int8 role labels of one sample (see the module docstring)."""
    fS, fK, fV, fO = (float(x) for x in mix)
    q_len = min(max(W, 16), max(N - PREFIX_LEN - 1, 0))
    head = [SINK] + [OTHER] * min(PREFIX_LEN, max(N - 1 - q_len, 0))
    body_len = N - len(head) - q_len
    fixed_other = len(head) - 1 + q_len
    # body fractions: remove the fixed OTHER tokens and the bursts from the targets
    other_body = max(fO * N - fixed_other, 0.0)
    burst_body = burst_frac * N
    sink_body = max(fS * N - 1 - burst_body, 0.0)
    mu_k = 2.0
    mu_v = mu_k * fV / fK
    mu_s = max(mu_k * sink_body / (fK * N), 2.0)
    o_per_cycle = mu_k * other_body / (fK * N)
    p_prose = min(o_per_cycle / PROSE_MEAN, 1.0)
    cyc_tokens = mu_k + mu_v + mu_s + o_per_cycle
    p_burst = 0.0
    if burst_frac > 0:
        p_burst = cyc_tokens * burst_frac / (1.0 - burst_frac) / ((BURST_LO + BURST_HI) / 2.0)
    body = []
    while len(body) < body_len:
        body += [SINK] * _run(rng, mu_s / 2)
        body += [KEY] * _run(rng, mu_k)
        body += [SINK] * _run(rng, mu_s / 2)
        body += [VALUE] * _run(rng, mu_v)
        if rng.random() < p_prose:
            body += [OTHER] * _run(rng, PROSE_MEAN)
        if p_burst and rng.random() < p_burst:
            body += [SINK] * int(rng.integers(BURST_LO, BURST_HI + 1))
    seq = head + body[:body_len] + [OTHER] * q_len
    return np.asarray(seq[:N], dtype=np.int8)


def make_roles(wl: Workload, seed: int = 0) -> np.ndarray:
    """Role labels [B, N] (int8) for a workload, one seeded stream per sample."""
    out = np.zeros((wl.B, wl.N), dtype=np.int8)
    for b in range(wl.B):
        rng = np.random.default_rng(tensor_seed(seed, wl.name, "roles", b))
        out[b] = role_pattern(wl.N, wl.W, wl.mix, rng, wl.pattern, wl.burst_frac)
    return out


def _torch_dtype(torch, name):
    return {"bf16": torch.bfloat16, "f32": torch.float32}[name]


def make_inputs(wl: Workload, device="cpu", seed: int = 0, layers=None,
                with_v: bool = True, roles=None):
    """Generate the tensors of a workload on ``device`` (torch).

    Returns a dict with
      roles  int8  [B, N]             (host numpy and device tensor),
      q      [L, B, Hq, W, d]         (window queries, SnapKV) or
             [L, B, Hq, N, d]         (all queries, H2O),
      k, v   [L, B, Hkv, N, d]        in the workload dtype.
    ``layers`` selects a subset of layer indices (each layer has its own seed
    stream, so a subset reproduces the same bits as the full stack).
    """
    import torch

    dt = _torch_dtype(torch, wl.dtype)
    layers = list(range(wl.L)) if layers is None else list(layers)
    if roles is None:
        roles = make_roles(wl, seed)
    roles_t = torch.from_numpy(np.ascontiguousarray(roles)).to(device)
    sink = (roles_t == SINK)                                   # [B, N]
    rows = wl.N if wl.scorer == "h2o" else wl.W
    scale = 1.0 / math.sqrt(wl.d)
    Ls = len(layers)
    q = torch.empty((Ls, wl.B, wl.Hq, rows, wl.d), dtype=dt, device=device)
    k = torch.empty((Ls, wl.B, wl.Hkv, wl.N, wl.d), dtype=dt, device=device)
    v = torch.empty_like(k) if with_v else None
    for li, layer in enumerate(layers):
        g = torch.Generator(device=device)
        g.manual_seed(tensor_seed(seed, wl.name, "q", layer))
        q32 = torch.randn((wl.B, wl.Hq, rows, wl.d), generator=g, device=device)
        if wl.q_mean > 0:
            off = torch.randn((wl.B, wl.Hkv, 1, 1, wl.d), generator=g, device=device)
            off = wl.q_mean * off / off.norm(dim=-1, keepdim=True)
            q32 = (q32.reshape(wl.B, wl.Hkv, wl.G, rows, wl.d) + off).reshape(q32.shape)
        q[li] = q32.to(dt)
        del q32
        g.manual_seed(tensor_seed(seed, wl.name, "k", layer))
        k32 = torch.randn((wl.B, wl.Hkv, wl.N, wl.d), generator=g, device=device)
        if rows > 0:
            qg = q[li].float().reshape(wl.B, wl.Hkv, wl.G * rows, wl.d)
            qbar = qg.mean(dim=2)                                   # [B, Hkv, d]
            nrm = qbar.norm(dim=-1, keepdim=True).clamp_min(1e-12)
            u = qbar / nrm
            beta = 2.0 * wl.sink_c / (scale * nrm)                  # [B, Hkv, 1]
            bias = (beta * u)[:, :, None, :]                        # [B, Hkv, 1, d]
            k32 += bias * sink[:, None, :, None].to(k32.dtype)
            del qg
        k[li] = k32.to(dt)
        del k32
        if with_v:
            g.manual_seed(tensor_seed(seed, wl.name, "v", layer))
            v[li] = torch.randn((wl.B, wl.Hkv, wl.N, wl.d), generator=g, device=device).to(dt)
    return {"roles": roles, "roles_t": roles_t, "q": q, "k": k, "v": v,
            "layers": layers, "workload": wl}
