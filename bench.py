"""Benchmark of the role-conditional eviction step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload stack32k] [--budget 0.05]

A step is one pass of the whole hot path over one batch already resident in
HBM: SnapKV windowed score with GQA sum and max-pool (every layer and KV
head), role allocation, per-role top-k and K/V compaction.  The default
workload is the 32-layer Llama-3-8B-shaped stack (32 query / 8 KV heads,
d=128, N=32768, W=32, pool 7, batch 4, B=0.05) on synthetic inputs.

Prints one JSON line.  ``value`` is prefill tokens scored and compressed per
second (a token counts once it has passed through all layers and KV heads) at
``ms_per_step``, the median of the K timed steps, each run after 512 MiB have
been written to a scratch buffer so that no cache holds the previous step's
data (``loop`` gives the mean of K back-to-back steps as well); ``roofline``
refers to the SnapKV score call, timed with HIP events on the stream it is
launched on (mean over the timed steps); ``long128k`` times the 131072-token
32-layer stack at B = 0.05 and 0.20 the same way; ``read_ceilings`` gives the
streaming HBM read rate and the last-level-cache re-read rate of a plain read
kernel; ``near_ties`` counts, on the last timed step's scores, the selection
boundaries a relative score change of 1e-3 could move; ``cpu_baseline`` times the float64 CPU oracle on a
bounded sample of the same workload; ``policies`` gives the step time of the
same workload under fair eviction and the No-KEY counterfactual, which reuse
every kernel with other quotas; ``decode`` times one decode query per head over
the compacted cache of every layer against the same kernel over the full
cache; ``quest`` times the one-shot Quest page-bound scorer on the same
inputs, alone and as the score of the whole step; ``probe`` times the linear
role probe labelling the batch's tokens (random weights of the paper's size);
``prefill_lse`` times the score and the step when the window rows' log-sum-exp
comes from the prefill attention (as such kernels return it per query row):
K is then read once.  ``--lse`` makes that the main line (for profiling it).

``roofline.traffic`` is the measured HBM traffic of one score call, read from
the counter summary in profiles/ (rocprofv3 FETCH_SIZE and WRITE_SIZE,
scaled by what the same counters read for a plain device copy of known
size); it is null when the kernel sources differ from the ones that summary
was taken on.  ``python bench.py --calibrate-copy`` runs only that copy.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "prefill tokens scored+compressed/s per GPU; % HBM peak (SnapKV), % MFMA (H2O)"
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "snapkv_score_stack32k_traffic.md")
# the same for the score with the window statistics supplied (pass 2 + pool)
TRAFFIC_SUMMARY_LSE = os.path.join(ROOT, "profiles", "snapkv_score_lse_stack32k_traffic.md")
# the score on the 128K-token workload (kernel times, matrix-core counters, traffic)
TRAFFIC_SUMMARY_LONG = os.path.join(ROOT, "profiles", "long128k_score_profile.md")
# sources of the kernels one score call launches
SCORE_SOURCES = ("paper_2607_13205_amd/csrc/snapkv.hip", "paper_2607_13205_amd/csrc/kve_stream.h",
                 "paper_2607_13205_amd/csrc/kve_device.h", "paper_2607_13205_amd/csrc/kve_snap_plan.h")
# untimed calls before each leg's timed ones: after a leg's set-up (new buffers,
# host work) the latency-bound kernels and the clock take some 10 steps to settle
LEG_WARMUP = 10
COPY_BYTES = 1 << 30
HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="stack32k")
    ap.add_argument("--budget", type=float, default=None)
    ap.add_argument("--alpha-key", type=float, default=0.0)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the oracle baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-h2o", action="store_true", help="skip the H2O scorer leg")
    ap.add_argument("--no-quest", action="store_true", help="skip the Quest scorer timings")
    ap.add_argument("--no-lse", action="store_true", help="skip the supplied-statistics timings")
    ap.add_argument("--lse", action="store_true",
                    help="main line with the window rows' log-sum-exp supplied (one read of K)")
    ap.add_argument("--no-probe", action="store_true", help="skip the role-probe timing")
    ap.add_argument("--chunks", type=int, default=1,
                    help="layer chunks of the step: each scored chunk's top-k and compaction run on a "
                         "second stream while the next chunk is scored (1: no overlap)")
    ap.add_argument("--no-decode", action="store_true",
                    help="skip the decode timings over the compacted and the full cache")
    ap.add_argument("--no-policies", action="store_true",
                    help="skip the fair-eviction and No-KEY step timings")
    ap.add_argument("--no-graph", action="store_true",
                    help="skip the step timing through a captured HIP graph")
    ap.add_argument("--no-long", action="store_true", help="skip the long128k legs")
    ap.add_argument("--no-fused", action="store_true", help="skip the fused role-epilogue step")
    ap.add_argument("--no-ceilings", action="store_true", help="skip the read-ceiling probes")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain device copy of 1 GiB (5 times), for counter calibration")
    return ap.parse_args()


def score_sources_sha() -> str:
    h = hashlib.sha256()
    for rel in SCORE_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(wl_name: str, summary: str = TRAFFIC_SUMMARY):
    """HBM bytes per score call from the committed counter summary, or None when
    it is missing, covers another workload, or was taken on other sources."""
    try:
        with open(summary) as f:
            text = f.read()
    except OSError:
        return None
    fields = {}
    for line in text.splitlines():
        line = line.strip().strip("`")
        if line.startswith("- ") and ":" in line:
            key, val = line[2:].split(":", 1)
            fields[key.strip()] = val.strip().strip("`")
    if fields.get("workload") != wl_name or fields.get("sources_sha256") != score_sources_sha():
        return None
    try:
        return int(fields["traffic_bytes_per_call"])
    except (KeyError, ValueError):
        return None


def calibrate_copy():
    import torch
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes_read": COPY_BYTES, "bytes_written": COPY_BYTES, "repeats": 5}))


def snapkv_algorithmic_bytes(wl, elem=2):
    """Bytes the score call must move at least once: K and the window
    queries read, the float32 score written."""
    segs = wl.L * wl.B * wl.Hkv
    return (segs * wl.N * wl.d * elem                     # K
            + wl.L * wl.B * wl.Hq * wl.W * wl.d * elem    # Q window
            + segs * wl.N * 4)                            # score


def step_algorithmic_bytes(wl, kept, elem=2):
    """Whole step: score call + score read by the select + role labels + kept
    indices written + kept K and V rows read and written."""
    segs_per_b = wl.L * wl.Hkv
    kept_rows = sum(int(k) for k in kept) * segs_per_b
    return (snapkv_algorithmic_bytes(wl, elem)
            + wl.L * wl.B * wl.Hkv * wl.N * 4             # score read
            + wl.B * wl.N                                 # roles
            + kept_rows * 4                               # indices
            + kept_rows * wl.d * elem * 4)                # K,V read + write


def cpu_baseline(wl, inp, budget, alpha, target_s):
    """Time the oracle on whole (layer, sample) units of the workload until about
    target_s seconds have been spent (at least one unit)."""
    import numpy as np

    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:  # pragma: no cover
        threads = 1
    quota, kept, _ = O.role_allocate_batch(inp["roles"], 4, alpha, budget, wl.W)
    units = 0
    t0 = time.perf_counter()
    order = [(l, b) for l in range(len(inp["layers"])) for b in range(wl.B)]
    for (l, b) in order:
        roles = inp["roles"][b]
        for j in range(wl.Hkv):
            q = inp["q"][l, b, j * wl.G:(j + 1) * wl.G].double().cpu().numpy()
            k = inp["k"][l, b, j].double().cpu().numpy()
            v = inp["v"][l, b, j].cpu()
            s = O.maxpool_prefix(O.snapkv_mass(q, k), wl.W, wl.pool_k)
            idx = O.select_keep(s, roles, quota[b], wl.W)
            O.kv_compact(k, idx)
            O.kv_compact(v.float().numpy(), idx)
        units += 1
        if time.perf_counter() - t0 >= target_s:
            break
    el = time.perf_counter() - t0
    # one unit is N tokens through one layer of one sample; a prefill token
    # needs all L layers
    tokens_per_s = units * wl.N / wl.L / el
    return {"value": tokens_per_s, "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{units} (layer, sample) units of {wl.name} ({wl.Hkv} KV heads, N={wl.N}) "
                      f"in {el:.1f} s: float64 score, pool, selection and compaction",
            "host_cpus": os.cpu_count(), "cpu_model": _cpu_model()}


def _cpu_model():
    """The host CPU's model name as /proc/cpuinfo gives it (None elsewhere)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def h2o_leg(K, WL, steps):
    """H2O scorer on the 16k-token workload: MFMA fraction on the causal flops."""
    import torch
    wl = WL.get_workload("h2o16k")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    score = torch.empty((wl.L, wl.B, wl.Hkv, wl.N), dtype=torch.float32, device="cuda")
    ws = torch.empty(K.h2o_workspace_size(wl.L, wl.B, wl.Hq, wl.Hkv, wl.N, wl.d),
                     dtype=torch.uint8, device="cuda")
    for _ in range(LEG_WARMUP):
        K.h2o_score(inp["q"], inp["k"], score=score, workspace=ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        K.h2o_score(inp["q"], inp["k"], score=score, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    causal = wl.L * wl.B * wl.Hq * wl.N * (wl.N + 1) / 2 * 2 * wl.d
    tf2 = 2 * causal / (ms * 1e-3) / 1e12
    del inp, ws
    torch.cuda.empty_cache()
    return {"workload": "h2o16k: 1 layer, 32q/8kv heads, d=128, N=16384, bf16",
            "ms": round(ms, 4), "tflops_2pass": round(tf2, 1),
            "mfma_frac_2pass": round(tf2 / BF16_MFMA_PEAK_TFLOPS, 4),
            "mfma_frac_1pass": round(tf2 / 2 / BF16_MFMA_PEAK_TFLOPS, 4)}


def policy_leg(WL, pipeline, wl, inp, budget, W, pool, steps):
    """Step time (HIP events) of the same workload under fair eviction and the
    No-KEY counterfactual: same kernels, other bucket labels and quotas."""
    import torch
    Policy = pipeline.Policy
    out = {}
    for name, pol in (("fair", Policy.fair(4)), ("no_key", Policy.no_role(WL.KEY, 4))):
        buckets = pol.buckets(inp["roles"])
        buckets_t = torch.from_numpy(buckets).to(inp["k"].device)
        _, kept, k_cap = pol.allocate(buckets, budget, W)
        bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, W, pol.R, k_cap, scorer=wl.scorer)

        def step():
            pipeline.evict(inp["q"], inp["k"], inp["v"], buckets, buckets_t, pol, budget, W, pool,
                           bufs, scorer=wl.scorer)

        out[name] = {"ms_per_step": round(_median_calls(step, steps), 4), "k_cap": k_cap,
                     "kept_mean": round(float(kept.mean()), 1)}
        del bufs
        torch.cuda.empty_cache()
    return out


def fused_leg(pipeline, wl, inp, alpha, budget, W, pool, k_cap, steps):
    """The same step with the fused role epilogue (the score's pool step counts
    the top-k's first digit per bucket): flushed median step, mean score and
    top-k times, as for the main line."""
    import torch
    bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, W, 4, k_cap, fused=True)
    run = lambda e, s_: pipeline.evict(inp["q"], inp["k"], inp["v"], inp["roles"], inp["roles_t"], alpha,  # noqa: E731
                                       budget, W, pool, bufs, score_events=e, select_events=s_)
    for _ in range(LEG_WARMUP):
        run(None, None)
    t = flushed_steps(run, steps)
    del bufs
    torch.cuda.empty_cache()
    return {"calls": "kve_snapkv_score_hist + kve_topk_select_hist", "ms_per_step": round(t["median_ms"], 4),
            "score_ms": round(t["score_ms"], 4), "topk_ms": round(t["topk_ms"], 4),
            "compact_ms": round(t["compact_ms"], 4)}


def graph_leg(pipeline, inp, alpha, budget, W, pool, bufs, scorer, steps, lse_win=None):
    """Step time with the device part captured once as a HIP graph and replayed
    (the host allocation runs between the score graph and the selection graph,
    while the device scores), and whether the replays give
    the eager step's kept indices and counts."""
    import torch
    idx0, cnt0 = bufs.idx.clone(), bufs.count.clone()
    g = pipeline.StepGraph(inp["q"], inp["k"], inp["v"], inp["roles_t"], alpha, W, pool, bufs, scorer=scorer,
                           lse_win=lse_win)
    ms = _median_calls(lambda: g.replay(inp["roles"], budget), steps)
    torch.cuda.synchronize()
    same = bool(torch.equal(bufs.idx, idx0) and torch.equal(bufs.count, cnt0))
    return {"ms_per_step": round(ms, 4), "matches_eager": same,
            "launch": "two HIP graph replays per step (the score; the quota copy, top-k and "
                      "compaction), the host allocation between them while the device scores"}


def select_figures(wl, inp, bufs, ms_topk, ms_compact):
    """Achieved rates of the top-k and the compaction inside the timed steps.
    Top-k algorithmic bytes: every score read once, the labels once per layer
    (1/Hkv byte per token and head), the kept indices written; compaction: the
    kept K and V rows read and written."""
    import torch
    L, B, Hkv, N, d = inp["k"].shape
    elem = inp["k"].element_size()
    kept = int(torch.clamp(bufs.count, 0, bufs.k_cap).sum().item())
    topk_bytes = L * B * Hkv * N * 4 + L * B * N + kept * 4
    compact_bytes = kept * d * elem * (2 if bufs.v_out is not None else 1) * 2
    gbs_t = topk_bytes / (ms_topk * 1e-3) / 1e9
    gbs_c = compact_bytes / (ms_compact * 1e-3) / 1e9
    return {"topk_ms": round(ms_topk, 4), "topk_algorithmic_bytes": topk_bytes,
            "topk_GBs": round(gbs_t, 1), "topk_hbm_frac": round(gbs_t / HBM_PEAK_GBS, 4),
            "compact_ms": round(ms_compact, 4), "compact_bytes": compact_bytes,
            "compact_GBs": round(gbs_c, 1), "compact_hbm_frac": round(gbs_c / HBM_PEAK_GBS, 4)}


def flushed_steps(run, steps, with_select=True):
    """Time `steps` eviction steps one by one, 512 MiB written to a scratch
    buffer before each (outside its events) so that neither the L2s nor the
    256 MB last-level cache hold anything of the previous step.  run(score_ev,
    select_ev) runs one step recording the given events.  Returns the median,
    minimum and maximum step time and the mean score time of those steps, and
    (with_select) the median top-k and compaction times of as many further steps
    run the same way with events around those two calls as well: an event
    between two kernels leaves the device idle for a few microseconds, so the
    timed steps carry only the events around the score (ms)."""
    import statistics
    import torch
    scratch = torch.empty(512 << 20, dtype=torch.uint8, device="cuda")
    mk = lambda n: tuple(torch.cuda.Event(enable_timing=True) for _ in range(n))  # noqa: E731
    step_ev = [mk(2) for _ in range(steps)]
    score_ev = [mk(2) for _ in range(steps)]
    sel_ev = [mk(3) for _ in range(steps)]
    torch.cuda.synchronize()
    for i in range(steps):
        scratch.fill_(i & 0xff)
        step_ev[i][0].record()
        run(score_ev[i], None)
        step_ev[i][1].record()
        torch.cuda.synchronize()
    if with_select:
        for i in range(steps):
            scratch.fill_(i & 0xff)
            run(mk(2), sel_ev[i])
            torch.cuda.synchronize()
    del scratch
    times = [a.elapsed_time(b) for a, b in step_ev]
    out = {"median_ms": statistics.median(times), "min_ms": min(times), "max_ms": max(times),
           "score_ms": sum(a.elapsed_time(b) for a, b in score_ev) / steps}
    if with_select:  # medians: a host pause before a launch would otherwise land in a mean
        out["topk_ms"] = statistics.median(a.elapsed_time(b) for a, b, _ in sel_ev)
        out["compact_ms"] = statistics.median(b.elapsed_time(c) for _, b, c in sel_ev)
    return out


def loop_leg(step, steps, tokens):
    """The same step back to back with nothing in between (the caches keep what
    the previous step left): the mean over `steps` steps."""
    ms = _time_calls(step, steps)
    return {"ms_per_step": round(ms, 4), "tokens_per_s": round(tokens / (ms * 1e-3), 1),
            "protocol": "mean of back-to-back steps, no cache flush"}


def long_leg(K, WL, pipeline, alpha, steps):
    """long128k (32 layers, batch 1, N = 131072, W = 64, 256 window rows per KV
    head) at B = 0.05 and 0.20: the flushed median step and the mean score
    call, with the score's HBM fraction on algorithmic bytes and its
    matrix-core fraction on the two passes' products (2 x 2.2 TFLOP)."""
    import torch
    wl = WL.get_workload("long128k")
    inp = WL.make_inputs(wl, device="cuda")
    torch.cuda.synchronize()
    res = {"workload": f"long128k: {wl.L} layers, batch {wl.B}, {wl.Hq}q/{wl.Hkv}kv heads, d={wl.d}, "
                       f"N={wl.N}, W={wl.W}, pool {wl.pool_k}, role mix {wl.mix}, table pattern"}
    segs = wl.L * wl.B * wl.Hkv
    flops_2pass = 2 * segs * (wl.G * wl.W) * wl.N * wl.d * 2
    for budget in wl.budgets:
        _, kept, k_cap = K.role_allocate(inp["roles"], 4, alpha, budget, wl.W)
        bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, wl.W, 4, k_cap)

        def run(e=None, s_=None):
            pipeline.evict(inp["q"], inp["k"], inp["v"], inp["roles"], inp["roles_t"], alpha, budget, wl.W,
                           wl.pool_k, bufs, score_events=e, select_events=s_)

        for _ in range(LEG_WARMUP):
            run()
        t = flushed_steps(run, steps)
        sb = snapkv_algorithmic_bytes(wl)
        stb = step_algorithmic_bytes(wl, kept)
        gbs = sb / (t["score_ms"] * 1e-3) / 1e9
        tf = flops_2pass / (t["score_ms"] * 1e-3) / 1e12
        traffic = measured_traffic(wl.name, TRAFFIC_SUMMARY_LONG)
        res[f"B={budget}"] = {
            "ms_per_step": round(t["median_ms"], 4), "tokens_per_s": round(wl.B * wl.N / (t["median_ms"] * 1e-3), 1),
            "step_hbm_frac": round(stb / (t["median_ms"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "score_ms": round(t["score_ms"], 4), "score_hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
            "score_tflops_2pass": round(tf, 1), "score_mfma_frac_2pass": round(tf / BF16_MFMA_PEAK_TFLOPS, 4),
            "score_traffic": traffic,
            "score_traffic_GBs": None if traffic is None else round(traffic / (t["score_ms"] * 1e-3) / 1e9, 1),
            "topk_ms": round(t["topk_ms"], 4), "compact_ms": round(t["compact_ms"], 4), "k_cap": k_cap}
        del bufs
        torch.cuda.empty_cache()
    del inp
    torch.cuda.empty_cache()
    return res


def copy_ceiling(repeats=5):
    """A plain 1 GiB device-to-device copy (the runtime's copy kernel): bytes read
    and written per second, the practical ceiling of a read-and-write kernel."""
    import torch
    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    ms = _time_calls(lambda: dst.copy_(src), repeats)
    gbs = 2 * COPY_BYTES / (ms * 1e-3) / 1e9
    del src, dst
    torch.cuda.empty_cache()
    return {"bytes_moved": 2 * COPY_BYTES, "ms": round(ms, 4), "GBs": round(gbs, 1),
            "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}


def read_ceilings(K, repeats=10):
    """Read rates of the probe kernel (kve_read_probe): a 4 GiB buffer streamed
    once with non-temporal loads (the HBM streaming-read ceiling the score
    passes are held to), and a 128 MiB buffer read again and again with cached
    loads (it fits in the 256 MB last-level cache but not in the 32 MB of L2:
    the rate at which that cache serves a second read of the same data)."""
    import torch
    blocks = 32768   # the fastest of 1024 .. 32768 workgroups in a sweep
    out = {"kernel": f"kve_read_probe (16-byte loads, 8 in flight per thread, {blocks} workgroups of 256)"}
    big = torch.empty(4 << 30, dtype=torch.uint8, device="cuda")
    big.fill_(1)
    sink = torch.empty(blocks, dtype=torch.float32, device="cuda")
    ms = _time_calls(lambda: K.binding.read_probe(big, True, blocks, sink), repeats)
    gbs = big.numel() / (ms * 1e-3) / 1e9
    out["stream_read"] = {"bytes": big.numel(), "ms": round(ms, 4), "GBs": round(gbs, 1),
                          "hbm_frac": round(gbs / HBM_PEAK_GBS, 4)}
    del big
    torch.cuda.empty_cache()
    small = torch.empty(128 << 20, dtype=torch.uint8, device="cuda")
    small.fill_(1)
    ms = _time_calls(lambda: K.binding.read_probe(small, False, blocks, sink), 4 * repeats)
    gbs = small.numel() / (ms * 1e-3) / 1e9
    out["llc_reread"] = {"bytes": small.numel(), "ms": round(ms, 4), "GBs": round(gbs, 1),
                         "note": "128 MiB read repeatedly: served by the last-level cache"}
    del small, sink
    torch.cuda.empty_cache()
    return out


def near_ties(score, roles, quota, W, rtol=1e-3):
    """Selection boundaries that a relative score change of rtol could move,
    from the step's own float32 scores (untimed): per (segment, bucket) with a
    proper cut (0 < quota < population), the dropped candidates whose score is
    within rtol of the bucket's boundary (quota-th best) score.  These are the
    places where a kept set computed from scores within the parity tolerance
    (the float64 oracle's) may legitimately differ."""
    import numpy as np
    L, B, H, N = score.shape
    P = N - W
    n_cuts = n_cut_ties = n_seg_ties = n_cand = n_equal = 0
    for b in range(B):
        rb = roles[b, :P]
        masks = [rb == r for r in range(quota.shape[1])]
        for l in range(L):
            for j in range(H):
                s = score[l, b, j, :P]
                seg_has = False
                for r, m in enumerate(masks):
                    q = int(quota[b, r])
                    cand = s[m]
                    if q <= 0 or q >= cand.size:
                        continue
                    n_cuts += 1
                    part = np.partition(cand, cand.size - q)
                    bnd = float(part[cand.size - q])          # q-th largest
                    dropped = part[:cand.size - q]
                    # dropped candidates equal to the boundary score are exact ties,
                    # decided by the index rule alike on every side; the others within
                    # rtol are the near-ties
                    n_equal += int(np.count_nonzero(dropped == bnd))
                    close = int(np.count_nonzero((dropped >= bnd - rtol * abs(bnd)) & (dropped != bnd)))
                    if close:
                        n_cand += close
                        n_cut_ties += 1
                        seg_has = True
                if seg_has:
                    n_seg_ties += 1
    return {"rtol": rtol, "bucket_cuts": n_cuts, "cuts_with_near_ties": n_cut_ties,
            "segments_with_near_ties": n_seg_ties, "segments": L * B * H,
            "dropped_candidates_within_rtol_of_boundary": n_cand,
            "dropped_candidates_equal_to_boundary": n_equal}


def _optional_leg(name, fn):
    """Run an optional leg of the bench; a failure becomes an error entry in the
    output line instead of ending the run (the main step is already timed)."""
    try:
        return fn()
    except Exception as e:  # noqa: BLE001 - reported, not hidden
        print(f"[bench] {name} leg failed: {e!r}", file=sys.stderr, flush=True)
        return {"error": f"{type(e).__name__}: {e}"}


def _median_calls(fn, steps):
    """Median time (ms) of `steps` single calls of fn, each bracketed by HIP
    events and followed by a synchronisation (after LEG_WARMUP untimed calls): one
    host-side stall moves a mean of back-to-back calls, not this median."""
    import statistics
    import torch
    for _ in range(LEG_WARMUP):
        fn()
    torch.cuda.synchronize()
    times = []
    for _ in range(steps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fn()
        e1.record()
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1))
    return statistics.median(times)


def _time_calls(fn, steps):
    import torch
    for _ in range(LEG_WARMUP):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def decode_leg(K, wl, inp, bufs, steps):
    """One decode query per head over the compacted cache of every layer
    (HIP events around the decode call), and the same kernel over the full,
    uncompressed cache: the 1 - B saving of a compacting implementation."""
    import torch
    L, B, Hkv, N, d = inp["k"].shape
    elem = inp["k"].element_size()
    g = torch.Generator(device="cuda")
    g.manual_seed(2024)
    q = (3.0 * torch.randn((L, B, wl.Hq, d), generator=g, device="cuda")).to(inp["k"].dtype)
    out = torch.empty((L, B, wl.Hq, d), dtype=torch.float32, device="cuda")
    ws = torch.empty(K.decode_workspace_size(L, B, wl.Hq, Hkv, bufs.k_cap, d), dtype=torch.uint8,
                     device="cuda")
    ms_c = _time_calls(lambda: K.decode_attention(q, bufs.k_out, bufs.v_out, bufs.count, out=out,
                                                  workspace=ws), steps)
    rows = int(torch.clamp(bufs.count, 0, bufs.k_cap).sum().item())
    small = L * B * wl.Hq * d * (elem + 4)                     # q read, out written
    bytes_c = rows * d * elem * 2 + small
    full = torch.full((L, B, Hkv), N, dtype=torch.int32, device="cuda")
    ws_f = torch.empty(K.decode_workspace_size(L, B, wl.Hq, Hkv, N, d), dtype=torch.uint8, device="cuda")
    ms_f = _time_calls(lambda: K.decode_attention(q, inp["k"], inp["v"], full, out=out, workspace=ws_f),
                       steps)
    bytes_f = L * B * Hkv * N * d * elem * 2 + small
    gbs_c = bytes_c / (ms_c * 1e-3) / 1e9
    gbs_f = bytes_f / (ms_f * 1e-3) / 1e9
    return {"kernel": "kve_decode_attention (split + combine), all layers in one call",
            "ms": round(ms_c, 4), "kept_rows": rows, "algorithmic_bytes": bytes_c,
            "achieved_GBs": round(gbs_c, 1), "hbm_frac": round(gbs_c / HBM_PEAK_GBS, 4),
            "ms_full_cache": round(ms_f, 4), "full_cache_GBs": round(gbs_f, 1),
            "full_cache_hbm_frac": round(gbs_f / HBM_PEAK_GBS, 4),
            "speedup_vs_full_cache": round(ms_f / ms_c, 2)}


def quest_leg(K, pipeline, wl, inp, budget, alpha, steps):
    """The one-shot Quest page-bound score (pages of 16) on the same inputs:
    the score call alone (HBM-bound: K read once, one float per token written)
    and the whole step with it as the score."""
    import torch
    L, B, Hkv, N, d = inp["k"].shape
    elem = inp["k"].element_size()
    score = torch.empty((L, B, Hkv, N), dtype=torch.float32, device="cuda")
    ws = torch.empty(K.quest_workspace_size(L, B, wl.Hq, Hkv, d), dtype=torch.uint8, device="cuda")
    ms = _time_calls(lambda: K.quest_score(inp["q"], inp["k"], 16, score=score, workspace=ws), steps)
    qbytes = L * B * wl.Hq * wl.W * d * elem
    nbytes = L * B * Hkv * (N - wl.W) * d * elem + qbytes + L * B * Hkv * N * 4
    gbs = nbytes / (ms * 1e-3) / 1e9
    del score, ws
    _, _, k_cap = K.role_allocate(inp["roles"], 4, alpha, budget, wl.W)
    bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, wl.W, 4, k_cap, scorer="quest")
    ms_step = _median_calls(lambda: pipeline.evict(inp["q"], inp["k"], inp["v"], inp["roles"], inp["roles_t"],
                                                   alpha, budget, wl.W, 1, bufs, scorer="quest"), steps)
    del bufs
    torch.cuda.empty_cache()
    return {"kernel": "kve_quest_score (mean query + page bounds), page 16", "ms": round(ms, 4),
            "algorithmic_bytes": nbytes, "achieved_GBs": round(gbs, 1),
            "hbm_frac": round(gbs / HBM_PEAK_GBS, 4), "ms_per_step": round(ms_step, 4),
            "tokens_per_s": round(B * N / (ms_step * 1e-3), 1)}


def probe_leg(K, wl, steps):
    """The linear role probe over the batch's B x N token ids: 5 tables of a
    128256-id vocabulary x 6 roles (3.85 M float32 parameters, random)."""
    import torch
    V, R = 128256, 6
    g = torch.Generator(device="cuda")
    g.manual_seed(77)
    weight = 0.1 * torch.randn((5, V, R), generator=g, device="cuda")
    bias = 0.1 * torch.randn((R,), generator=g, device="cuda")
    ids = torch.randint(0, V, (wl.B, wl.N), generator=g, device="cuda", dtype=torch.int32)
    out = torch.empty((wl.B, wl.N), dtype=torch.int8, device="cuda")
    ms = _time_calls(lambda: K.role_probe(ids, weight, bias, out=out), steps)
    return {"kernel": "kve_role_probe", "tokens": wl.B * wl.N, "us": round(ms * 1000, 2),
            "tokens_per_s": round(wl.B * wl.N / (ms * 1e-3), 1)}


def window_lse(q, k, wl):
    """The window rows' natural-log log-sum-exp [L, B, Hq, W], float32, layer by
    layer with torch: the statistic a prefill attention kernel returns per
    query row (input preparation, outside every timed region)."""
    import torch
    L = k.shape[0]
    out = torch.empty((L, wl.B, wl.Hq, wl.W), dtype=torch.float32, device=k.device)
    pos = torch.arange(wl.N - wl.W, wl.N, device=k.device)
    mask = torch.arange(wl.N, device=k.device)[None, :] <= pos[:, None]
    scale = 1.0 / math.sqrt(wl.d)
    for l in range(L):
        qf = q[l].float().reshape(wl.B, wl.Hkv, wl.G * wl.W, wl.d)
        kf = k[l].float().transpose(-1, -2).contiguous()
        x = (torch.matmul(qf, kf) * scale).reshape(wl.B, wl.Hkv, wl.G, wl.W, wl.N)
        out[l] = torch.logsumexp(x.masked_fill(~mask, float("-inf")), dim=-1).reshape(wl.B, wl.Hq, wl.W)
        del qf, kf, x
    torch.cuda.empty_cache()
    return out


def lse_leg(K, pipeline, wl, inp, lse, budget, alpha, steps):
    """Score call and whole step with the window rows' statistics supplied."""
    import torch
    L, B, Hkv, N, d = inp["k"].shape
    score = torch.empty((L, B, Hkv, N), dtype=torch.float32, device="cuda")
    ws = torch.empty(K.snapkv_workspace_size(L, B, wl.Hq, Hkv, N, wl.W, d), dtype=torch.uint8, device="cuda")
    ms = _time_calls(lambda: K.snapkv_score_lse(inp["q"], inp["k"], lse, wl.pool_k, score=score, workspace=ws),
                     steps)
    nbytes = snapkv_algorithmic_bytes(wl)
    del score, ws
    _, _, k_cap = K.role_allocate(inp["roles"], 4, alpha, budget, wl.W)
    bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, wl.W, 4, k_cap)
    ms_step = _median_calls(lambda: pipeline.evict(inp["q"], inp["k"], inp["v"], inp["roles"], inp["roles_t"],
                                                   alpha, budget, wl.W, wl.pool_k, bufs, lse_win=lse), steps)
    del bufs
    torch.cuda.empty_cache()
    gbs = nbytes / (ms * 1e-3) / 1e9
    return {"kernel": "kve_snapkv_score_lse (window statistics supplied; pass 2 + pool)", "ms": round(ms, 4),
            "achieved_GBs": round(gbs, 1), "hbm_frac": round(gbs / HBM_PEAK_GBS, 4),
            "ms_per_step": round(ms_step, 4), "tokens_per_s": round(wl.B * wl.N / (ms_step * 1e-3), 1)}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only; --gpus {args.gpus} is not supported "
              "(the eviction path shards by layer or KV head with no exchange between GPUs, so "
              "one GPU's throughput times the GPU count is the whole job's)",
              file=sys.stderr)
        sys.exit(2)
    import torch

    if args.calibrate_copy:
        calibrate_copy()
        return
    import workload as WL
    from paper_2607_13205_amd.build import ensure_built
    ensure_built()
    import paper_2607_13205_amd as K
    from paper_2607_13205_amd import pipeline

    wl = WL.get_workload(args.workload)
    budget = args.budget if args.budget is not None else wl.budgets[0]
    alpha = WL.default_alpha(args.alpha_key)
    torch.cuda.set_device(0)
    print(f"[bench] generating {wl.name} inputs on the GPU", file=sys.stderr, flush=True)
    inp = WL.make_inputs(wl, device="cuda")
    torch.cuda.synchronize()
    scorer = wl.scorer
    W = 0 if scorer == "h2o" else wl.W
    pool = 1 if scorer == "h2o" else wl.pool_k
    lse = None
    if scorer == "snapkv" and (args.lse or not args.no_lse):
        print("[bench] window-row statistics for the supplied-lse runs (untimed)", file=sys.stderr, flush=True)
        lse = window_lse(inp["q"], inp["k"], wl)
    main_lse = lse if args.lse else None
    _, kept, k_cap = K.role_allocate(inp["roles"], 4, alpha, budget, W)
    bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, W, 4, k_cap, scorer=scorer)

    side = torch.cuda.Stream() if args.chunks > 1 else None

    def step():
        pipeline.evict(inp["q"], inp["k"], inp["v"], inp["roles"], inp["roles_t"], alpha, budget,
                       W, pool, bufs, scorer=scorer, chunks=args.chunks, side_stream=side, lse_win=main_lse)

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # timed region: K steps, each after 512 MiB written to a scratch buffer
    # (outside its events) so that no cache holds the previous step's data;
    # HIP events on the launch stream around each step, the score call, the
    # top-k and the compaction
    timed = flushed_steps(lambda e, s_: pipeline.evict(
        inp["q"], inp["k"], inp["v"], inp["roles"], inp["roles_t"], alpha, budget, W, pool, bufs,
        scorer=scorer, score_events=e, chunks=args.chunks, side_stream=side, lse_win=main_lse,
        select_events=s_ if args.chunks <= 1 else None), args.steps, with_select=args.chunks <= 1)
    ms_step = timed["median_ms"]
    ms_score = timed["score_ms"]
    ms_topk, ms_compact = timed.get("topk_ms"), timed.get("compact_ms")
    tokens = wl.B * wl.N
    value = tokens / (ms_step * 1e-3)
    score_bytes = snapkv_algorithmic_bytes(wl)
    achieved = score_bytes / (ms_score * 1e-3) / 1e9
    step_bytes = step_algorithmic_bytes(wl, kept)
    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: {wl.L} layers, batch {wl.B}, {wl.Hq}q/{wl.Hkv}kv heads, "
                        f"d={wl.d}, N={wl.N}, W={wl.W}, pool {wl.pool_k}, B={budget}, "
                        f"alpha_KEY={args.alpha_key}, role mix {wl.mix}"
                        + (", window-row log-sum-exp supplied (K read once)" if args.lse else ""),
            "global_batch": wl.B, "seq_len": wl.N, "parallelism": "none (1 GPU)",
            "layer_tokens_per_s": round(value * wl.L, 1),
            "k_cap": k_cap, "layer_chunks": args.chunks,
            "ms_per_step_is": "median of the timed steps, 512 MiB written before each one (outside its events)",
            "step_ms_min_max": [round(timed["min_ms"], 4), round(timed["max_ms"], 4)],
            "step_algorithmic_GBs": round(step_bytes / (ms_step * 1e-3) / 1e9, 1),
            "step_hbm_frac": round(step_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        },
        "roofline": {
            "kernel": ("kve_snapkv_score_lse (pass 2 + pool)" if args.lse
                       else "kve_snapkv_score (score passes + pool)"),
            "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(wl.name, TRAFFIC_SUMMARY_LSE if args.lse else
                                        TRAFFIC_SUMMARY_LONG if wl.name == "long128k" else TRAFFIC_SUMMARY),
            "ms": round(ms_score, 4), "ms_is": "mean of the score call over the timed steps",
            "algorithmic_bytes": score_bytes,
        },
    }
    if ms_topk is not None:
        out["select"] = select_figures(wl, inp, bufs, ms_topk, ms_compact)
    if scorer != "h2o":
        print("[bench] near-ties of the last timed step (untimed)", file=sys.stderr, flush=True)
        out["near_ties"] = _optional_leg("near_ties", lambda: near_ties(
            bufs.score.cpu().numpy(), inp["roles"], bufs.quota_host.numpy().copy(), W))
    out["loop"] = _optional_leg("loop", lambda: loop_leg(step, args.steps, tokens))
    out["copy_ceiling"] = _optional_leg("copy_ceiling", copy_ceiling)
    if not args.no_ceilings:
        print("[bench] read ceilings", file=sys.stderr, flush=True)
        out["read_ceilings"] = _optional_leg("read_ceilings", lambda: read_ceilings(K))
    if scorer == "snapkv" and not args.lse and args.chunks <= 1 and not args.no_fused:
        print("[bench] fused role epilogue", file=sys.stderr, flush=True)
        out["fused_epilogue"] = _optional_leg("fused_epilogue", lambda: fused_leg(
            pipeline, wl, inp, alpha, budget, W, pool, k_cap, max(5, args.steps // 2)))
    if not args.no_graph and args.chunks <= 1:
        print("[bench] step through a HIP graph", file=sys.stderr, flush=True)
        out["graph"] = _optional_leg("graph", lambda: graph_leg(
            pipeline, inp, alpha, budget, W, pool, bufs, scorer, max(3, args.steps // 2), lse_win=main_lse))
    if not args.no_decode and scorer == "snapkv":
        print("[bench] decode over the compacted and the full cache", file=sys.stderr, flush=True)
        out["decode"] = _optional_leg("decode", lambda: decode_leg(K, wl, inp, bufs, max(3, args.steps // 2)))
    del bufs
    torch.cuda.empty_cache()
    if lse is not None and not args.lse and not args.no_lse:
        print("[bench] supplied window statistics", file=sys.stderr, flush=True)
        out["prefill_lse"] = _optional_leg("prefill_lse", lambda: lse_leg(
            K, pipeline, wl, inp, lse, budget, alpha, max(3, args.steps // 2)))
    if not args.no_quest and scorer == "snapkv":
        print("[bench] Quest scorer", file=sys.stderr, flush=True)
        out["quest"] = _optional_leg("quest", lambda: quest_leg(
            K, pipeline, wl, inp, budget, alpha, max(3, args.steps // 2)))
    if not args.no_probe:
        out["probe"] = _optional_leg("probe", lambda: probe_leg(K, wl, max(3, args.steps // 2)))
    if not args.no_policies:
        print("[bench] fair-eviction and No-KEY steps", file=sys.stderr, flush=True)
        out["policies"] = _optional_leg("policies", lambda: policy_leg(
            WL, pipeline, wl, inp, budget, W, pool, max(3, args.steps // 2)))
    if not args.no_long and wl.name == "stack32k" and not args.lse:
        print("[bench] long128k legs", file=sys.stderr, flush=True)
        out["long128k"] = _optional_leg("long128k", lambda: long_leg(
            K, WL, pipeline, alpha, max(5, args.steps // 2)))
    if not args.no_h2o and wl.name != "h2o16k":
        print("[bench] H2O leg", file=sys.stderr, flush=True)
        out["h2o"] = _optional_leg("h2o", lambda: h2o_leg(K, WL, max(3, args.steps // 2)))
    if not args.no_cpu_baseline:
        print("[bench] CPU oracle baseline", file=sys.stderr, flush=True)
        out["cpu_baseline"] = _optional_leg("cpu_baseline", lambda: cpu_baseline(
            wl, inp, budget, alpha, args.cpu_seconds))
    print(json.dumps(out), flush=True)
    # nothing left in flight, device and pinned host memory handed back before
    # the interpreter and the runtime shut down
    del inp, lse
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


if __name__ == "__main__":
    main()
