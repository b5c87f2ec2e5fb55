"""Parity of the HIP path (through the C ABI) with the CPU oracle on MI355X.

Every input comes from the seeded generators in ``workload``; the oracle gets
the exact bits the GPU received (bf16 upcast exactly to float64).
"""

from __future__ import annotations

import math

import numpy as np
import pytest

import oracle as O
import workload as WL
from tests.parity import check_decode, check_kept_set, check_scores, report

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def K():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_13205_amd.build import ensure_built
    ensure_built()
    import paper_2607_13205_amd as K
    return K


def f64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def custom(name, L, B, Hq, Hkv, N, W, d, pool_k, dtype, scorer="snapkv"):
    return WL.Workload(name, L=L, B=B, Hq=Hq, Hkv=Hkv, N=N, W=W, d=d, pool_k=pool_k, dtype=dtype,
                       mix=(0.35, 0.20, 0.30, 0.15), budgets=(0.1,), scorer=scorer)


def note(msg):
    print(msg, flush=True)


def run_snapkv(K, q, k, pool_k, scale=0.0):
    """Score with an explicit workspace filled with NaN bytes: no result may
    depend on what the workspace held before the call."""
    L, B, Hq, W, d = q.shape
    Hkv, N = k.shape[2], k.shape[3]
    ws = torch.full((K.snapkv_workspace_size(L, B, Hq, Hkv, N, W, d),), 0xFF, dtype=torch.uint8, device=k.device)
    score = K.snapkv_score(q, k, pool_k, scale, workspace=ws)
    torch.cuda.synchronize()
    return score


SNAP_CASES = [
    WL.get_workload("tiny"),
    custom("ragged", 2, 2, 8, 2, 1000, 24, 128, 7, "bf16"),
    custom("rowgroups", 1, 1, 8, 2, 700, 64, 64, 3, "bf16"),
    custom("w1", 1, 1, 4, 4, 300, 1, 128, 7, "bf16"),
    custom("wfull", 1, 1, 2, 1, 96, 96, 64, 1, "f32"),
    custom("f32d128", 1, 2, 4, 2, 333, 16, 128, 15, "f32"),
    custom("bigpool", 1, 1, 4, 1, 450, 8, 128, 31, "bf16"),
    custom("n1", 1, 1, 2, 1, 1, 1, 64, 5, "bf16"),
    custom("g8", 1, 1, 16, 2, 513, 20, 128, 7, "bf16"),
    custom("rounds", 8, 2, 8, 4, 2000, 16, 128, 7, "bf16"),
    custom("wide", 1, 1, 8, 1, 3000, 64, 128, 7, "bf16"),
    # 32 vsegs x 141 chunks: 71 ranges of two 64-key chunks, the last a single ragged chunk of 40 keys
    custom("multirange", 2, 2, 8, 8, 9000, 16, 128, 7, "bf16"),
    custom("f32multirange", 2, 2, 8, 4, 9000, 8, 64, 5, "f32"),
    # wide pools across many one-chunk ranges of 64 keys (half-widths 64 and 65)
    custom("pool129", 1, 2, 8, 4, 5000, 16, 128, 129, "bf16"),
    custom("pool131", 1, 2, 8, 4, 5000, 16, 128, 131, "bf16"),
    # a last range of 6 keys, shorter than the half-width 7
    custom("shorttail", 1, 1, 4, 2, 1030, 8, 64, 15, "bf16"),
    # 300 window rows: two 256-row groups, the second with 44 rows and 212 padding rows
    custom("rows300", 1, 2, 12, 2, 3000, 50, 128, 7, "bf16"),
    # 160 window rows (one 256-row group): ranges of three chunks and a last range of one
    # chunk of 10 keys, so that the second wave group of the 256-row kernels has nothing to do
    custom("rows160tail", 1, 1, 4, 1, 394, 40, 128, 7, "bf16"),
    # kernel 7 on rows too short for the register path: every key taken one by one
    custom("short7", 1, 2, 4, 2, 20, 4, 128, 7, "bf16"),
    # the most window rows a KV head may have (G*W = 1024): four 256-row groups
    # (bf16, four planes of column sums) and eight 128-row groups (float32)
    custom("rows1024", 1, 1, 16, 1, 1500, 64, 128, 7, "bf16"),
    custom("rows1024_f32", 1, 1, 16, 1, 700, 64, 64, 5, "f32"),
    # three KV heads in two layers and two samples (segments not a power of two)
    custom("kv3", 2, 2, 12, 3, 1000, 16, 128, 7, "bf16"),
]


@pytest.mark.parametrize("wl", SNAP_CASES, ids=lambda w: w.name)
def test_snapkv_score_matches_oracle(K, wl):
    note(f"snapkv parity {wl}")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    score = run_snapkv(K, inp["q"], inp["k"], wl.pool_k)
    ref = O.snapkv_score(f64(inp["q"]), f64(inp["k"]), wl.Hkv, wl.pool_k)
    check_scores(f64(score), ref, wl.name)


def test_snapkv_score_layer8k_all_segments(K):
    wl = WL.get_workload("layer8k")
    note("snapkv parity layer8k (8 segments)")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    score = run_snapkv(K, inp["q"], inp["k"], wl.pool_k)
    ref = O.snapkv_score(f64(inp["q"]), f64(inp["k"]), wl.Hkv, wl.pool_k)
    check_scores(f64(score), ref, wl.name)


def test_snapkv_explicit_scale(K):
    wl = custom("scale", 1, 1, 4, 2, 256, 8, 64, 5, "bf16")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    score = run_snapkv(K, inp["q"], inp["k"], wl.pool_k, scale=0.05)
    ref = O.snapkv_score(f64(inp["q"]), f64(inp["k"]), wl.Hkv, wl.pool_k, scale=0.05)
    check_scores(f64(score), ref, "scale")


# Logit spikes: every 97th key row scaled by 40, so that (with N(0, 1) inputs)
# many rows meet a key whose logit lies more than 64, and some more than 128,
# log2 units above the running reference of their range: the row sums leave
# [0, 2^64] (or overflow) after the first chunk, and the kernels raise their
# reference from the chunk's logits taken again.  One-set and two-set row
# groups and float32.
SPIKE_CASES = [
    custom("spike_rows128", 1, 2, 8, 2, 3000, 16, 128, 7, "bf16"),
    custom("spike_rows256", 1, 2, 8, 2, 5000, 64, 128, 7, "bf16"),
    custom("spike_f32", 1, 1, 4, 2, 2000, 16, 128, 5, "f32"),
]


@pytest.mark.parametrize("wl", SPIKE_CASES, ids=lambda w: w.name)
def test_snapkv_score_logit_spikes_match_oracle(K, wl):
    note(f"snapkv parity with logit spikes {wl}")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    k = inp["k"].clone()
    k[:, :, :, 40::97, :] *= 40
    q = inp["q"]
    ref = O.snapkv_score(f64(q), f64(k), wl.Hkv, wl.pool_k)
    # the case does what it is for: some window row meets a logit more than 128
    # log2 units above its largest over the keys before the first spike
    # (float64, from the same rounded inputs)
    qq = f64(q).reshape(wl.L, wl.B, wl.Hkv, wl.G * wl.W, wl.d)
    logit2 = np.matmul(qq, np.swapaxes(f64(k), -1, -2)) * (wl.d ** -0.5) * math.log2(math.e)
    span = float((logit2.max(axis=-1) - logit2[..., :40].max(axis=-1)).max())
    assert span > 128, span
    score = run_snapkv(K, q, k, wl.pool_k)
    check_scores(f64(score), ref, wl.name)


# Strided views: the window queries as the last W rows of all prefill queries,
# the keys from a token-major cache [L, B, N, Hkv, d] (optionally with padded
# rows), through kve_snapkv_score_strided: the same arithmetic in the same order
# as on dense copies, so the scores must be bit-identical; the dense scores are
# checked against the oracle as well.
STRIDED_CASES = [
    custom("strided_bf16", 2, 2, 8, 2, 1000, 24, 128, 7, "bf16"),
    custom("strided_rows256", 1, 2, 8, 2, 3000, 64, 128, 7, "bf16"),   # 256-row groups
    custom("strided_f32", 1, 2, 4, 2, 333, 16, 64, 5, "f32"),
]


def _strided_views(q_win, k, pad):
    """(q view, k view): q_win as the tail of a [L, B, Hq, N, d] tensor, k as a
    permuted token-major tensor whose rows are d + pad elements apart."""
    L, B, Hq, W, d = q_win.shape
    N, Hkv = k.shape[3], k.shape[2]
    q_full = torch.full((L, B, Hq, N, d), float("nan"), dtype=q_win.dtype, device=q_win.device)
    q_full[:, :, :, N - W:, :] = q_win
    k_tm = torch.full((L, B, N, Hkv, d + pad), float("nan"), dtype=k.dtype, device=k.device)
    k_tm[..., :d] = k.permute(0, 1, 3, 2, 4)
    return q_full[:, :, :, N - W:, :], k_tm[..., :d].permute(0, 1, 3, 2, 4)


@pytest.mark.parametrize("wl", STRIDED_CASES, ids=lambda w: w.name)
@pytest.mark.parametrize("pad", [0, 8])
def test_snapkv_strided_views_match_dense(K, wl, pad):
    note(f"snapkv strided views {wl} pad={pad}")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    qv, kv = _strided_views(inp["q"], inp["k"], pad)
    assert not qv.is_contiguous() and not kv.is_contiguous()
    dense = run_snapkv(K, inp["q"], inp["k"], wl.pool_k)
    strided = K.snapkv_score_strided(qv, kv, wl.pool_k)
    torch.cuda.synchronize()
    assert torch.equal(strided, dense)
    check_scores(f64(dense), O.snapkv_score(f64(inp["q"]), f64(inp["k"]), wl.Hkv, wl.pool_k), wl.name)


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("f32", 64)])
def test_kv_compact_strided_views_match_dense(K, dtype, d):
    rng = np.random.default_rng(5)
    L, B, Hkv, N, k_cap = 2, 2, 3, 300, 48
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    kk = torch.randn((L, B, Hkv, N, d)).to(tdt).cuda()
    vv = torch.randn((L, B, Hkv, N, d)).to(tdt).cuda()
    idx = np.full((L, B, Hkv, k_cap), -1, dtype=np.int32)
    cnt = rng.integers(0, k_cap + 1, (L, B, Hkv)).astype(np.int32)
    for s in np.ndindex(L, B, Hkv):
        idx[s][:cnt[s]] = np.sort(rng.choice(N, cnt[s], replace=False))
    idx_d, cnt_d = torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda()
    ko, vo = K.kv_compact(kk, vv, idx_d, cnt_d)
    # K token-major with padded rows, V token-major with dense rows: different row strides
    k_tm = torch.zeros((L, B, N, Hkv, d + 16), dtype=tdt, device="cuda")
    k_tm[..., :d] = kk.permute(0, 1, 3, 2, 4)
    v_tm = vv.permute(0, 1, 3, 2, 4).contiguous()
    ks, vs = K.kv_compact_strided(k_tm[..., :d].permute(0, 1, 3, 2, 4), v_tm.permute(0, 1, 3, 2, 4), idx_d, cnt_d)
    torch.cuda.synchronize()
    assert torch.equal(ks, ko) and torch.equal(vs, vo)
    # keys only, through the dispatching wrapper
    k_only, v_none = K.kv_compact(k_tm[..., :d].permute(0, 1, 3, 2, 4), None, idx_d, cnt_d)
    torch.cuda.synchronize()
    assert v_none is None and torch.equal(k_only, ko)


H2O_CASES = [
    custom("h2o_small", 1, 1, 4, 2, 300, 0, 128, 1, "bf16", scorer="h2o"),
    custom("h2o_f32", 1, 1, 2, 1, 200, 0, 64, 1, "f32", scorer="h2o"),
    custom("h2o_ragged", 2, 1, 8, 2, 513, 0, 128, 1, "bf16", scorer="h2o"),
    custom("h2o_n1", 1, 1, 2, 2, 1, 0, 64, 1, "bf16", scorer="h2o"),
    # G = 8: 16 positions per row block; G = 3: 42 positions and 2 padding rows
    custom("h2o_g8", 1, 1, 16, 2, 700, 0, 128, 1, "bf16", scorer="h2o"),
    custom("h2o_g3", 1, 2, 6, 2, 333, 0, 64, 1, "bf16", scorer="h2o"),
    custom("h2o_g1_f32", 1, 1, 2, 2, 260, 0, 128, 1, "f32", scorer="h2o"),
    # three KV heads (neither a divisor nor a multiple of the eight XCDs pass 1
    # spreads its heads over) in two layers and two samples
    custom("h2o_kv3", 2, 2, 6, 3, 400, 0, 128, 1, "bf16", scorer="h2o"),
]


@pytest.mark.parametrize("wl", H2O_CASES, ids=lambda w: w.name)
def test_h2o_score_matches_oracle(K, wl):
    note(f"h2o parity {wl}")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    score = K.h2o_score(inp["q"], inp["k"])
    torch.cuda.synchronize()
    ref = O.h2o_score(f64(inp["q"]), f64(inp["k"]), wl.Hkv)
    check_scores(f64(score), ref, wl.name)
    # total mass: every query row distributes exactly G*N per KV head in sum
    tot = f64(score).sum(axis=-1)
    np.testing.assert_allclose(tot, wl.G * wl.N, rtol=1e-4)


@pytest.mark.parametrize("wl", [custom("h2o_spike", 1, 1, 8, 2, 700, 0, 128, 1, "bf16", scorer="h2o"),
                                custom("h2o_spike_f32", 1, 1, 4, 2, 500, 0, 64, 1, "f32", scorer="h2o")],
                         ids=lambda w: w.name)
def test_h2o_score_logit_spikes_match_oracle(K, wl):
    """Every 97th key row scaled by 40: causal rows meet logits far above the
    running reference of their first chunks, so the row sums of pass 1 leave
    [0, 2^64] (or overflow) and raise their reference part way."""
    note(f"h2o parity with logit spikes {wl}")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    k = inp["k"].clone()
    k[:, :, :, 40::97, :] *= 40
    q = inp["q"]
    qq = f64(q).reshape(wl.L, wl.B, wl.Hkv, wl.G * wl.N, wl.d)
    logit2 = np.matmul(qq, np.swapaxes(f64(k), -1, -2)) * (wl.d ** -0.5) * math.log2(math.e)
    assert float((logit2.max(axis=-1) - logit2[..., :40].max(axis=-1)).max()) > 128
    score = K.h2o_score(q, k)
    torch.cuda.synchronize()
    ref = O.h2o_score(f64(q), f64(k), wl.Hkv)
    check_scores(f64(score), ref, wl.name)


def _token_major(x, pad):
    """x [L, B, H, T, d] as a view of a token-major tensor [L, B, T, H, d + pad]
    (NaN in the padding, which must never be read)."""
    L, B, H, T, d = x.shape
    tm = torch.full((L, B, T, H, d + pad), float("nan"), dtype=x.dtype, device=x.device)
    tm[..., :d] = x.permute(0, 1, 3, 2, 4)
    return tm[..., :d].permute(0, 1, 3, 2, 4)


@pytest.mark.parametrize("wl", [H2O_CASES[0], H2O_CASES[1], H2O_CASES[5]], ids=lambda w: w.name)
@pytest.mark.parametrize("pad", [0, 8])
def test_h2o_strided_views_match_dense(K, wl, pad):
    """Token-major queries and keys through kve_h2o_score_strided: the same
    arithmetic in the same order as the dense call, so bit-identical scores."""
    note(f"h2o strided views {wl} pad={pad}")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    qv, kv = _token_major(inp["q"], pad), _token_major(inp["k"], pad)
    assert not qv.is_contiguous()  # (k with one KV head and no padding is dense either way)
    dense = K.h2o_score(inp["q"], inp["k"])
    strided = K.h2o_score_strided(qv, kv)
    torch.cuda.synchronize()
    assert torch.equal(strided, dense)


def test_h2o_full_size_one_kv_head(K):
    """The 16k-token H2O workload at its real shape; the oracle recomputes the
    scores of one KV head (4 query heads x 16384 rows) in float64."""
    wl = WL.get_workload("h2o16k")
    note("h2o parity h2o16k (full size, KV head 5 checked)")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    score = K.h2o_score(inp["q"], inp["k"])
    torch.cuda.synchronize()
    j = 5
    q = f64(inp["q"][0, 0, j * wl.G:(j + 1) * wl.G])
    k = f64(inp["k"][0, 0, j])
    ref = O.h2o_mass(q, k, row_block=1024)
    check_scores(f64(score[0, 0, j]), ref, "h2o16k head 5")
    np.testing.assert_allclose(f64(score).sum(axis=-1), wl.G * wl.N, rtol=1e-4)


def _random_selection_case(rng, N, R_labels, R):
    s = rng.random(N).astype(np.float32)
    s[rng.random(N) < 0.2] = 0.5                         # exact ties
    s[rng.random(N) < 0.05] = -0.0
    s[rng.random(N) < 0.05] = np.nan
    roles = rng.integers(-1, R_labels, N).astype(np.int8)
    return s, roles


def _topk_check(K, score, roles, quota, W, R, roles_dev=None, score_dev=None):
    """Run the GPU top-k on host arrays and compare every segment with the oracle."""
    L, B, Hkv, N = score.shape
    kept = [W + sum(min(max(int(quota[b, r]), 0), int(np.sum(roles[b, :N - W] == r)))
                    for r in range(R)) for b in range(B)]
    k_cap = max(kept)
    sd = torch.from_numpy(score).cuda() if score_dev is None else score_dev
    rd = torch.from_numpy(roles).cuda() if roles_dev is None else roles_dev
    idx, cnt = K.topk_select(sd, rd, torch.from_numpy(quota).cuda(), W, R, k_cap)
    torch.cuda.synchronize()
    idx, cnt = idx.cpu().numpy(), cnt.cpu().numpy()
    for l in range(L):
        for b in range(B):
            for j in range(Hkv):
                ref = O.select_keep(score[l, b, j], roles[b], quota[b], W)
                assert cnt[l, b, j] == len(ref) == kept[b], (l, b, j)
                assert idx[l, b, j, :len(ref)].tolist() == ref.tolist(), (l, b, j)


# N per bucket count: ragged lengths take the one-load-per-position path, the
# multiples of 16 the 16-byte span loads
TOPK_N = {"ragged": [7, 300, 1000, 4097, 70001, 33, 2049, 65],
          "aligned": [16, 304, 1024, 4096, 70000, 48, 2048, 64]}


@pytest.mark.parametrize("layout", ["ragged", "aligned"])
@pytest.mark.parametrize("R", range(1, 9))  # the kernel is instantiated per bucket count
def test_topk_select_bit_exact_with_oracle(K, R, layout):
    rng = np.random.default_rng(R + (100 if layout == "aligned" else 0))
    L, B, Hkv = 2, 2, 3
    N = TOPK_N[layout][R - 1]
    W = int(rng.integers(0, min(N, 40)))
    score = np.zeros((L, B, Hkv, N), dtype=np.float32)
    roles = np.zeros((B, N), dtype=np.int8)
    for b in range(B):
        _, roles[b] = _random_selection_case(rng, N, R + 1, R)
    for l in range(L):
        for b in range(B):
            for j in range(Hkv):
                score[l, b, j], _ = _random_selection_case(rng, N, R, R)
    quota = rng.integers(-2, N // max(R, 1) + 3, (B, R)).astype(np.int32)
    _topk_check(K, score, roles, quota, W, R)


@pytest.mark.parametrize("R,N", [(4, 301), (4, 304), (8, 1000), (1, 4096)])
def test_topk_many_segments_take_the_four_wave_workgroups(K, R, N):
    """512 segments and more use four-wave workgroups (fewer use sixteen waves)."""
    rng = np.random.default_rng(60 + R + N)
    L, B, Hkv = 4, 4, 32
    W = 20
    score = np.zeros((L, B, Hkv, N), dtype=np.float32)
    roles = np.zeros((B, N), dtype=np.int8)
    for b in range(B):
        _, roles[b] = _random_selection_case(rng, N, R + 1, R)
    for l in range(L):
        for b in range(B):
            for j in range(Hkv):
                score[l, b, j], _ = _random_selection_case(rng, N, R, R)
    quota = rng.integers(-1, N // R + 2, (B, R)).astype(np.int32)
    _topk_check(K, score, roles, quota, W, R)


@pytest.mark.parametrize("N,W", [(1, 0), (1, 1), (2, 0), (2, 1), (3, 3), (17, 0), (17, 5), (16, 16)])
def test_topk_very_short_rows(K, N, W):
    """Rows shorter than one 16-position span, a row that is all window, and a
    call that keeps nothing (k_cap 0, empty index output)."""
    rng = np.random.default_rng(70 + 31 * N + W)
    L, B, Hkv, R = 1, 2, 3, 3
    score = np.zeros((L, B, Hkv, N), dtype=np.float32)
    roles = np.zeros((B, N), dtype=np.int8)
    for b in range(B):
        _, roles[b] = _random_selection_case(rng, N, R + 1, R)
        for j in range(Hkv):
            score[0, b, j], _ = _random_selection_case(rng, N, R, R)
    quota = rng.integers(0, 3, (B, R)).astype(np.int32)
    _topk_check(K, score, roles, quota, W, R)
    if W == 0:
        # nothing kept at all: zero quotas, k_cap 0
        zero = np.zeros((B, R), dtype=np.int32)
        idx, cnt = K.topk_select(torch.from_numpy(score).cuda(), torch.from_numpy(roles).cuda(),
                                 torch.from_numpy(zero).cuda(), W, R, 0)
        torch.cuda.synchronize()
        assert idx.shape[-1] == 0 and not cnt.cpu().numpy().any()


def test_topk_misaligned_rows_take_the_per_position_loads(K):
    """N a multiple of 16 but the score and label rows not 16-byte aligned."""
    rng = np.random.default_rng(41)
    L, B, Hkv, N, R, W = 1, 2, 2, 4096, 4, 32
    score = rng.random((L, B, Hkv, N)).astype(np.float32)
    roles = rng.integers(0, R, (B, N)).astype(np.int8)
    quota = rng.integers(0, N // R, (B, R)).astype(np.int32)
    sbuf = torch.empty(L * B * Hkv * N + 1, dtype=torch.float32, device="cuda")
    sbuf[1:] = torch.from_numpy(score.ravel()).cuda()
    rbuf = torch.empty(B * N + 3, dtype=torch.int8, device="cuda")
    rbuf[3:] = torch.from_numpy(roles.ravel()).cuda()
    sd, rd = sbuf[1:].view(L, B, Hkv, N), rbuf[3:].view(B, N)
    assert sd.data_ptr() % 16 and rd.data_ptr() % 16
    _topk_check(K, score, roles, quota, W, R, roles_dev=rd, score_dev=sd)


@pytest.mark.parametrize("case", ["all_equal", "all_nan", "two_values", "window_only", "no_window",
                                  "one_bin", "inf", "nan_below_neginf"])
def test_topk_degenerate_inputs(K, case):
    """Every key in the threshold's bin, every key tied, no prefix, no window."""
    rng = np.random.default_rng(50)
    L, B, Hkv, N, R = 1, 2, 2, 2048, 3
    W = 16
    score = rng.random((L, B, Hkv, N)).astype(np.float32)
    roles = rng.integers(0, R, (B, N)).astype(np.int8)
    quota = np.array([[100, 0, 700], [1, 2000, 5]], dtype=np.int32)
    if case == "all_equal":
        score[:] = 0.25
    elif case == "all_nan":
        score[:] = np.nan
    elif case == "two_values":
        score[:] = np.where(rng.random(score.shape) < 0.5, 1.0, -0.0).astype(np.float32)
    elif case == "window_only":
        W = N
    elif case == "no_window":
        W = 0
    elif case == "one_bin":
        # distinct keys that all share the top 11 bits (one quarter binade)
        score[:] = (1.0 + rng.random(score.shape) * 0.24).astype(np.float32)
    elif case == "inf":
        score[rng.random(score.shape) < 0.3] = np.inf
        score[rng.random(score.shape) < 0.3] = -np.inf
    elif case == "nan_below_neginf":
        # about 10% finite, 45% -inf, 45% NaN: the quotas put bucket boundaries
        # inside the -inf run and inside the NaN run (NaN ranks below -inf)
        u = rng.random(score.shape)
        score[u < 0.45] = -np.inf
        score[u > 0.55] = np.nan
        quota = np.array([[400, 0, 350], [1, 2000, 380]], dtype=np.int32)
    _topk_check(K, score, roles, quota, W, R)


def test_topk_reports_truncation(K):
    N, W = 100, 4
    score = torch.rand((1, 1, 1, N)).cuda()
    roles = torch.zeros((1, N), dtype=torch.int8).cuda()
    quota = torch.tensor([[50]], dtype=torch.int32).cuda()
    idx, cnt = K.topk_select(score, roles, quota, W, 1, 20)
    torch.cuda.synchronize()
    assert int(cnt[0, 0, 0]) == 54
    ref = O.select_keep(score[0, 0, 0].cpu().numpy(), np.zeros(N, dtype=np.int8), [50], W)
    assert idx[0, 0, 0].cpu().numpy().tolist() == ref[:20].tolist()


@pytest.mark.parametrize("dtype,d", [("bf16", 128), ("bf16", 64), ("f32", 64), ("f32", 128)])
def test_kv_compact_bit_exact(K, dtype, d):
    rng = np.random.default_rng(3)
    L, B, Hkv, N, k_cap = 2, 2, 3, 257, 40
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    kk = torch.randn((L, B, Hkv, N, d)).to(tdt).cuda()
    vv = torch.randn((L, B, Hkv, N, d)).to(tdt).cuda()
    idx = np.full((L, B, Hkv, k_cap), -1, dtype=np.int32)
    cnt = rng.integers(0, k_cap + 1, (L, B, Hkv)).astype(np.int32)
    for s in np.ndindex(L, B, Hkv):
        idx[s][:cnt[s]] = np.sort(rng.choice(N, cnt[s], replace=False))
    idx[0, 0, 0, 0] = N + 5                 # out-of-range entry: skipped
    cnt[1, 1, 2] = k_cap + 7                # count above capacity: clamped
    idx[1, 1, 2] = np.arange(k_cap)
    ko, vo = K.kv_compact(kk, vv, torch.from_numpy(idx).cuda(), torch.from_numpy(cnt).cuda())
    torch.cuda.synchronize()
    bits = torch.int16 if dtype == "bf16" else torch.int32
    kbits, vbits = kk.view(bits).cpu().numpy(), vv.view(bits).cpu().numpy()
    kob, vob = ko.view(bits).cpu().numpy(), vo.view(bits).cpu().numpy()
    for s in np.ndindex(L, B, Hkv):
        c = min(cnt[s], k_cap)
        for m in range(k_cap):
            t = idx[s][m]
            if m < c and 0 <= t < N:
                assert np.array_equal(kob[s][m], O.kv_compact(kbits[s], [t])[0])
                assert np.array_equal(vob[s][m], O.kv_compact(vbits[s], [t])[0])
            else:
                assert not kob[s][m].any() and not vob[s][m].any()


def test_step_graph_replays_match_eager_steps(K):
    """The step captured as a HIP graph, replayed at several budgets with eager
    steps and synchronisations in between, gives the eager step's quotas,
    scores, kept indices, counts and compacted rows bit for bit."""
    from paper_2607_13205_amd import pipeline
    wl = WL.get_workload("layer8k")
    note("step graph layer8k")
    inp = WL.make_inputs(wl, device="cuda")
    alpha = WL.default_alpha(0.0)
    budgets = [0.05, 0.20, 0.10, 0.05, 0.50]
    cap = max(K.role_allocate(inp["roles"], 4, alpha, b, wl.W)[2] for b in budgets)
    bufs_g = pipeline.alloc_buffers(inp["k"], wl.Hq, wl.W, 4, cap)
    bufs_e = pipeline.alloc_buffers(inp["k"], wl.Hq, wl.W, 4, cap)
    g = pipeline.StepGraph(inp["q"], inp["k"], inp["v"], inp["roles_t"], alpha, wl.W, wl.pool_k, bufs_g)
    for b in budgets:
        qg, kg = g.replay(inp["roles"], b)
        torch.cuda.synchronize()
        qe, ke = pipeline.evict(inp["q"], inp["k"], inp["v"], inp["roles"], inp["roles_t"], alpha, b,
                                wl.W, wl.pool_k, bufs_e)
        torch.cuda.synchronize()
        assert np.array_equal(qg, qe) and np.array_equal(kg, ke)
        for name in ("score", "idx", "count", "k_out", "v_out"):
            assert torch.equal(getattr(bufs_g, name), getattr(bufs_e, name)), (b, name)
    # and the last replay against the oracle's kept sets for two segments
    ref_q, _, _ = O.role_allocate_batch(inp["roles"], 4, alpha, budgets[-1], wl.W)
    assert np.array_equal(ref_q, qg)
    s_all = O.snapkv_score(f64(inp["q"]), f64(inp["k"]), wl.Hkv, wl.pool_k)
    for (l, b, j) in [(0, 0, 0), (0, 0, 7)]:
        s_ref = s_all[l, b, j]
        ref = O.select_keep(s_ref, inp["roles"][b], qg[b], wl.W)
        got = bufs_g.idx[l, b, j, :int(bufs_g.count[l, b, j])].cpu().numpy()
        check_kept_set(got, ref, s_ref, inp["roles"][b], wl.W, qg[b])


def check_quest_or_scores(gpu, ref, W, what):
    """Scores of any scorer; the Quest window entries are +inf on both sides."""
    N = len(ref)
    if np.isinf(ref[N - W:]).all() and W > 0:
        assert np.isinf(gpu[N - W:]).all() and (gpu[N - W:] > 0).all(), f"{what}: window not +inf"
        if N - W > 0:
            check_scores(gpu[:N - W], ref[:N - W], what)
        return
    check_scores(gpu, ref, what)


def _pipeline_check(K, wl, inp, budget, policy, segs=None, chunks=1):
    """Run the whole step on the GPU and check scores, kept sets and compacted
    rows of the given segments against the oracle.  ``policy`` is a Policy or
    the weights of the role-conditional policy."""
    from paper_2607_13205_amd import pipeline
    policy = pipeline.as_policy(policy)
    W = 0 if wl.scorer == "h2o" else wl.W
    pool = 1 if wl.scorer == "h2o" else wl.pool_k
    R = policy.R
    buckets = policy.buckets(inp["roles"])
    buckets_t = inp["roles_t"] if policy.bucket_of is None else torch.from_numpy(buckets).cuda()
    _, _, k_cap = policy.allocate(buckets, budget, W)
    bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, W, R, k_cap, scorer=wl.scorer)
    side = torch.cuda.Stream() if chunks > 1 else None
    quota, kept = pipeline.evict(inp["q"], inp["k"], inp["v"], buckets, buckets_t, policy,
                                 budget, W, pool, bufs, scorer=wl.scorer, chunks=chunks, side_stream=side)
    torch.cuda.synchronize()
    ob = inp["roles"] if policy.bucket_of is None else O.role_map(inp["roles"], policy.bucket_of)
    assert np.array_equal(buckets, ob)
    if policy.alpha is None:
        qo, ko, _ = O.fair_allocate_batch(ob, R, budget, W)
    else:
        qo, ko, _ = O.role_allocate_batch(ob, R, list(policy.alpha), budget, W)
    assert np.array_equal(quota, qo) and np.array_equal(kept, ko)
    if segs is None:
        segs = list(np.ndindex(len(inp["layers"]), wl.B, wl.Hkv))
    ties = 0
    for (l, b, j) in segs:
        kseg = f64(inp["k"][l, b, j])
        if wl.scorer == "h2o":
            s_ref = O.h2o_mass(f64(inp["q"][l, b, j * wl.G:(j + 1) * wl.G]), kseg, row_block=1024)
        elif wl.scorer == "quest":
            s_ref = O.quest_mass(f64(inp["q"][l, b, j * wl.G:(j + 1) * wl.G]), kseg, 16)
        else:
            s_ref = O.maxpool_prefix(O.snapkv_mass(f64(inp["q"][l, b, j * wl.G:(j + 1) * wl.G]), kseg),
                                     W, pool)
        check_quest_or_scores(f64(bufs.score[l, b, j]), s_ref, W, f"{wl.name} seg {(l, b, j)}")
        roles = ob[b]
        idx_ref = O.select_keep(s_ref, roles, qo[b], W)
        if policy.bucket_of is not None and policy.alpha == (1.0, 0.0) and sum(policy.bucket_of) == 1:
            # No-X: the bucket composition is the definition's kept set
            x = list(policy.bucket_of).index(1)
            assert np.array_equal(idx_ref, O.no_role_keep(s_ref, inp["roles"][b], x, budget, W))
        n = int(bufs.count[l, b, j])
        assert n == kept[b]
        idx_gpu = bufs.idx[l, b, j, :n].cpu().numpy()
        ties += check_kept_set(idx_gpu, idx_ref, s_ref, roles, W, qo[b])
        # the oracle's selection on the GPU's own float32 scores is bit-exact
        idx_same = O.select_keep(bufs.score[l, b, j].cpu().numpy(), roles, qo[b], W)
        assert np.array_equal(idx_gpu, idx_same)
        # compaction: row m is the input row idx_gpu[m], bit for bit
        bits = torch.int16 if inp["k"].dtype == torch.bfloat16 else torch.int32
        kin = inp["k"][l, b, j].view(bits).cpu().numpy()
        vin = inp["v"][l, b, j].view(bits).cpu().numpy()
        assert np.array_equal(bufs.k_out[l, b, j, :n].view(bits).cpu().numpy(), O.kv_compact(kin, idx_gpu))
        assert np.array_equal(bufs.v_out[l, b, j, :n].view(bits).cpu().numpy(), O.kv_compact(vin, idx_gpu))
    return ties


@pytest.mark.parametrize("name,budget", [("tiny", 0.10), ("layer8k", 0.05), ("layer8k", 0.10),
                                         ("layer8k", 0.20), ("layer8k", 0.50)])
def test_pipeline_small_workloads(K, name, budget):
    wl = WL.get_workload(name)
    note(f"pipeline {name} B={budget}")
    inp = WL.make_inputs(wl, device="cuda")
    ties = _pipeline_check(K, wl, inp, budget, WL.default_alpha(0.0))
    report(f"near-tie pairs vs oracle, {name} B={budget} (every segment)", ties)


@pytest.mark.parametrize("scorer", ["snapkv", "quest", "h2o"])
def test_pipeline_on_strided_views_matches_dense(K, scorer):
    """The whole step on a token-major cache (keys [L, B, N, Hkv, d] with padded
    rows, values [L, B, N, Hkv, d]) and, for SnapKV and Quest, the window
    queries as the tail of all prefill queries: the same scores, kept indices,
    counts and compacted rows as on dense tensors."""
    from paper_2607_13205_amd import pipeline
    h2o = scorer == "h2o"
    wl = custom(f"views_{scorer}", 2, 2, 8, 2, 1200, 0 if h2o else 24, 128, 1 if h2o else 7, "bf16", scorer=scorer)
    note(f"pipeline on strided views {wl}")
    inp = WL.make_inputs(wl, device="cuda")
    if h2o:
        qv, kv = _token_major(inp["q"], 0), _token_major(inp["k"], 8)
    else:
        qv, kv = _strided_views(inp["q"], inp["k"], 8)
    vv = _token_major(inp["v"], 0)
    policy = pipeline.as_policy(WL.default_alpha(0.0))
    _, _, k_cap = policy.allocate(inp["roles"], 0.1, wl.W)
    out = []
    for q, k, v in ((inp["q"], inp["k"], inp["v"]), (qv, kv, vv)):
        bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, wl.W, policy.R, k_cap, scorer=scorer)
        pipeline.evict(q, k, v, inp["roles"], inp["roles_t"], policy, 0.1, wl.W, wl.pool_k, bufs, scorer=scorer)
        torch.cuda.synchronize()
        out.append(bufs)
    d, s = out
    assert torch.equal(d.score, s.score) and torch.equal(d.count, s.count) and torch.equal(d.idx, s.idx)
    assert torch.equal(d.k_out, s.k_out) and torch.equal(d.v_out, s.v_out)


def test_pipeline_alpha_key_nonzero_and_neutral(K):
    wl = WL.get_workload("layer8k").with_(Hq=8, Hkv=2)
    inp = WL.make_inputs(wl, device="cuda")
    _pipeline_check(K, wl, inp, 0.1, WL.default_alpha(0.02))
    # neutral policy: one bucket with weight 1 is plain SnapKV at budget B
    roles1 = np.zeros_like(inp["roles"])
    inp1 = dict(inp, roles=roles1, roles_t=torch.from_numpy(roles1).cuda())
    from paper_2607_13205_amd import pipeline
    _, _, k_cap = K.role_allocate(roles1, 1, [1.0], 0.1, wl.W)
    bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, wl.W, 1, k_cap)
    pipeline.evict(inp1["q"], inp1["k"], inp1["v"], roles1, inp1["roles_t"], [1.0], 0.1, wl.W,
                   wl.pool_k, bufs)
    torch.cuda.synchronize()
    for j in range(wl.Hkv):
        s = bufs.score[0, 0, j].cpu().numpy()
        K_ = math.ceil(0.1 * wl.N - 1e-9)
        order = sorted(range(wl.N - wl.W), key=lambda t: (-s[t], t))
        ref = sorted(order[:K_ - wl.W] + list(range(wl.N - wl.W, wl.N)))
        n = int(bufs.count[0, 0, j])
        assert bufs.idx[0, 0, j, :n].cpu().numpy().tolist() == ref


def test_pipeline_h2o_small(K):
    wl = custom("h2o_pipe", 1, 1, 8, 2, 700, 0, 128, 1, "bf16", scorer="h2o")
    inp = WL.make_inputs(wl, device="cuda")
    _pipeline_check(K, wl, inp, 0.1, WL.default_alpha(0.0))


def _policy(name):
    from paper_2607_13205_amd.pipeline import Policy
    return {"fair": Policy.fair(4), "no_key": Policy.no_role(WL.KEY, 4),
            "no_sink": Policy.no_role(WL.SINK, 4), "no_value": Policy.no_role(WL.VALUE, 4)}[name]


@pytest.mark.parametrize("pol,budget", [("no_key", 0.1), ("no_key", 0.5), ("no_sink", 0.3),
                                        ("no_value", 0.75), ("fair", 0.1)])
def test_pipeline_h2o_policies(K, pol, budget):
    """The counterfactual No-X conditions over the H2O score (§4), and fair
    eviction, through the same allocator, top-k and compaction."""
    wl = custom("h2o_pol", 1, 2, 8, 2, 1500, 0, 128, 1, "bf16", scorer="h2o")
    note(f"pipeline h2o {pol} B={budget}")
    inp = WL.make_inputs(wl, device="cuda")
    _pipeline_check(K, wl, inp, budget, _policy(pol))


@pytest.mark.parametrize("pol,budget", [("fair", 0.05), ("fair", 0.2), ("no_key", 0.1)])
def test_pipeline_snapkv_policies(K, pol, budget):
    wl = WL.get_workload("layer8k")
    note(f"pipeline layer8k {pol} B={budget}")
    inp = WL.make_inputs(wl, device="cuda")
    _pipeline_check(K, wl, inp, budget, _policy(pol))


@pytest.mark.parametrize("chunks", [2, 3])
def test_pipeline_layer_chunks_on_two_streams(K, chunks):
    """Scoring chunks of layers on one stream while the top-k and compaction of
    the scored chunks run on a second stream gives the oracle's result."""
    wl = WL.get_workload("layer8k").with_(L=5, Hq=8, Hkv=2, N=4000)
    note(f"pipeline in {chunks} layer chunks")
    inp = WL.make_inputs(wl, device="cuda")
    _pipeline_check(K, wl, inp, 0.1, WL.default_alpha(0.0), chunks=chunks)


def test_determinism(K):
    wl = WL.get_workload("layer8k")
    inp = WL.make_inputs(wl, device="cuda")
    from paper_2607_13205_amd import pipeline
    alpha = WL.default_alpha(0.0)
    outs = []
    for _ in range(2):
        _, _, k_cap = K.role_allocate(inp["roles"], 4, alpha, 0.1, wl.W)
        bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, wl.W, 4, k_cap)
        pipeline.evict(inp["q"], inp["k"], inp["v"], inp["roles"], inp["roles_t"], alpha, 0.1,
                       wl.W, wl.pool_k, bufs)
        torch.cuda.synchronize()
        outs.append((bufs.score.clone(), bufs.idx.clone(), bufs.k_out.clone()))
    assert torch.equal(outs[0][0], outs[1][0])
    assert torch.equal(outs[0][1], outs[1][1])
    assert torch.equal(outs[0][2].view(torch.int16), outs[1][2].view(torch.int16))


@pytest.mark.parametrize("name,budget,segs,pol", [
    ("stack32k", 0.05, [(9, 1, 4)], "fair"),
    ("stack32k", 0.05, [(3, 0, 1), (30, 3, 6)], "role4chunks"),
    ("h2o16k", 0.10, [(0, 0, 3)], "no_key"),
])
def test_pipeline_full_size_sampled(K, name, budget, segs, pol):
    """Real shapes under the other policies and the chunked two-stream step;
    the oracle recomputes a few sampled (layer, sample, KV head) segments (the
    role policy is checked on every segment below)."""
    wl = WL.get_workload(name)
    note(f"pipeline full size {name} B={budget} {pol}: generating inputs")
    inp = WL.make_inputs(wl, device="cuda")
    torch.cuda.synchronize()
    note("  running and checking sampled segments")
    policy = WL.default_alpha(0.0) if pol.startswith("role") else _policy(pol)
    ties = _pipeline_check(K, wl, inp, budget, policy, segs=segs, chunks=4 if pol == "role4chunks" else 1)
    report(f"near-tie pairs vs oracle, {name} B={budget} {pol} ({len(segs)} sampled segments)", ties)
    del inp
    torch.cuda.empty_cache()


# one oracle segment per layer for the score check; h2o16k (one layer, an
# O(N^2) oracle) checks three of its eight KV heads
FULL_CASES = [("stack32k", 0.05), ("long128k", 0.05), ("long128k", 0.20), ("h2o16k", 0.10)]


@pytest.mark.parametrize("name,budget", FULL_CASES)
def test_pipeline_full_size_every_segment(K, name, budget):
    """The benchmark's launch configuration at full size, role policy.  Every
    segment: the kept set equals the oracle's selection on the GPU's own
    float32 scores bit for bit, the count equals the allocation's, and every
    compacted K and V row is the input row it names, bit for bit.  One segment
    per layer (three heads of h2o16k): the scores are the float64 oracle's to
    the tolerance and the kept set the oracle's, apart from near-ties, which
    are counted and reported.  Checked layer by layer to bound host memory."""
    from paper_2607_13205_amd import pipeline
    wl = WL.get_workload(name)
    note(f"full size every segment {name} B={budget}: generating inputs")
    inp = WL.make_inputs(wl, device="cuda")
    torch.cuda.synchronize()
    alpha = WL.default_alpha(0.0)
    W = 0 if wl.scorer == "h2o" else wl.W
    pool = 1 if wl.scorer == "h2o" else wl.pool_k
    _, _, k_cap = K.role_allocate(inp["roles"], 4, alpha, budget, W)
    bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, W, 4, k_cap, scorer=wl.scorer)
    quota, kept = pipeline.evict(inp["q"], inp["k"], inp["v"], inp["roles"], inp["roles_t"], alpha, budget, W,
                                 pool, bufs, scorer=wl.scorer)
    torch.cuda.synchronize()
    qo, ko, _ = O.role_allocate_batch(inp["roles"], 4, alpha, budget, W)
    assert np.array_equal(quota, qo) and np.array_equal(kept, ko)
    L = len(inp["layers"])
    if wl.scorer == "h2o":
        oracle_segs = {(0, 0, 0), (0, 0, 4), (0, 0, 7)}
    else:
        oracle_segs = {(l, l % wl.B, (3 * l + 1) % wl.Hkv) for l in range(L)}
    bits = torch.int16 if inp["k"].dtype == torch.bfloat16 else torch.int32
    ties = exact = 0
    for l in range(L):
        note(f"  layer {l}")
        sc = bufs.score[l].cpu().numpy()
        idx = bufs.idx[l].cpu().numpy()
        cnt = bufs.count[l].cpu().numpy()
        kin = inp["k"][l].view(bits).cpu().numpy()
        vin = inp["v"][l].view(bits).cpu().numpy()
        kout = bufs.k_out[l].view(bits).cpu().numpy()
        vout = bufs.v_out[l].view(bits).cpu().numpy()
        for b, j in np.ndindex(wl.B, wl.Hkv):
            n = int(cnt[b, j])
            assert n == kept[b], (l, b, j)
            idx_gpu = idx[b, j, :n]
            assert np.array_equal(idx_gpu, O.select_keep(sc[b, j], inp["roles"][b], qo[b], W)), (l, b, j)
            assert np.array_equal(kout[b, j, :n], O.kv_compact(kin[b, j], idx_gpu)), (l, b, j)
            assert np.array_equal(vout[b, j, :n], O.kv_compact(vin[b, j], idx_gpu)), (l, b, j)
            if (l, b, j) in oracle_segs:
                kseg = f64(inp["k"][l, b, j])
                qg = f64(inp["q"][l, b, j * wl.G:(j + 1) * wl.G])
                if wl.scorer == "h2o":
                    s_ref = O.h2o_mass(qg, kseg, row_block=1024)
                else:
                    s_ref = O.maxpool_prefix(O.snapkv_mass(qg, kseg), W, pool)
                check_scores(sc[b, j].astype(np.float64), s_ref, f"{name} seg {(l, b, j)}")
                idx_ref = O.select_keep(s_ref, inp["roles"][b], qo[b], W)
                t = check_kept_set(idx_gpu, idx_ref, s_ref, inp["roles"][b], W, qo[b])
                ties += t
                exact += int(t == 0)
        del sc, idx, cnt, kin, vin, kout, vout
    if wl.scorer == "snapkv":
        # decode one new query per head over the compacted cache of every layer
        # (one call, the benchmark's launch configuration) = decode through the
        # keep-mask over the full cache, on the oracle segments
        note("  decode over the compacted cache")
        g = torch.Generator(device="cuda")
        g.manual_seed(4321)
        qd = (3.0 * torch.randn((L, wl.B, wl.Hq, wl.d), generator=g, device="cuda")).to(inp["k"].dtype)
        out = K.decode_attention(qd, bufs.k_out, bufs.v_out, bufs.count).cpu().numpy()
        worst = 0.0
        for (l, b, j) in sorted(oracle_segs):
            n = int(bufs.count[l, b, j])
            sel = bufs.idx[l, b, j, :n].cpu().numpy()
            qs = f64(qd[l, b, j * wl.G:(j + 1) * wl.G])
            kf, vf = f64(inp["k"][l, b, j]), f64(inp["v"][l, b, j])
            ref = O.masked_decode_attention(qs, kf, vf, sel)
            ref_abs = O.masked_decode_attention(qs, kf, np.abs(vf), sel)
            xmax = float(np.max(np.abs(qs @ kf[sel].T))) / math.sqrt(wl.d)
            worst = max(worst, check_decode(out[l, b, j * wl.G:(j + 1) * wl.G], ref, ref_abs, xmax,
                                            f"{name} decode seg {(l, b, j)}"))
        report(f"decode worst err/bound, full size {name} B={budget} ({len(oracle_segs)} segments)", round(worst, 4))
    report(f"full size {name} B={budget}: segments with kept sets and compacted rows checked", L * wl.B * wl.Hkv)
    report(f"full size {name} B={budget}: oracle-score segments (identical kept set / near-tie pairs)",
           f"{len(oracle_segs)} ({exact} / {ties})")
    del inp, bufs
    torch.cuda.empty_cache()


def _window_lse_oracle(inp, wl):
    """The oracle's window-row log-sum-exp of every segment, float32 [L, B, Hq, W]."""
    L = inp["k"].shape[0]
    out = np.zeros((L, wl.B, wl.Hq, wl.W), dtype=np.float32)
    for l, b, j in np.ndindex(L, wl.B, wl.Hkv):
        out[l, b, j * wl.G:(j + 1) * wl.G] = O.window_lse(f64(inp["q"][l, b, j * wl.G:(j + 1) * wl.G]),
                                                          f64(inp["k"][l, b, j]))
    return out


@pytest.mark.parametrize("wl", [WL.get_workload("tiny")] + [c for c in SNAP_CASES if c.name in
                                ("ragged", "g8", "multirange", "f32d128", "wfull", "shorttail", "pool129", "rows300")],
                         ids=lambda w: w.name)
def test_snapkv_score_lse_matches_oracle(K, wl):
    """With the window rows' statistics supplied (one read of K), the score is
    the oracle's."""
    note(f"snapkv with supplied lse {wl.name}")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    lse = torch.from_numpy(_window_lse_oracle(inp, wl)).cuda()
    ws = torch.full((K.snapkv_workspace_size(wl.L, wl.B, wl.Hq, wl.Hkv, wl.N, wl.W, wl.d),), 0xFF,
                    dtype=torch.uint8, device="cuda")
    sc = K.snapkv_score_lse(inp["q"], inp["k"], lse, wl.pool_k, workspace=ws)
    torch.cuda.synchronize()
    ref = O.snapkv_score(f64(inp["q"]), f64(inp["k"]), wl.Hkv, wl.pool_k)
    for idx in np.ndindex(wl.L, wl.B, wl.Hkv):
        check_scores(f64(sc[idx]), ref[idx], f"{wl.name} lse seg {idx}")


def test_pipeline_with_supplied_lse_full_size(K):
    """stack32k's launch configuration with the statistics supplied (computed
    here in float32 by torch, standing in for a prefill attention kernel); the
    oracle recomputes sampled segments end to end."""
    from paper_2607_13205_amd import pipeline
    wl = WL.get_workload("stack32k")
    note("pipeline stack32k with supplied lse")
    inp = WL.make_inputs(wl, device="cuda")
    lse = window_lse_torch(inp["q"], inp["k"], wl)
    alpha = WL.default_alpha(0.0)
    _, _, k_cap = K.role_allocate(inp["roles"], 4, alpha, 0.05, wl.W)
    bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, wl.W, 4, k_cap)
    quota, kept = pipeline.evict(inp["q"], inp["k"], inp["v"], inp["roles"], inp["roles_t"], alpha, 0.05, wl.W,
                                 wl.pool_k, bufs, lse_win=lse)
    torch.cuda.synchronize()
    for (l, b, j) in [(0, 0, 0), (20, 3, 6)]:
        kseg = f64(inp["k"][l, b, j])
        s_ref = O.maxpool_prefix(O.snapkv_mass(f64(inp["q"][l, b, j * wl.G:(j + 1) * wl.G]), kseg), wl.W, wl.pool_k)
        check_scores(f64(bufs.score[l, b, j]), s_ref, f"stack32k lse seg {(l, b, j)}")
        n = int(bufs.count[l, b, j])
        idx_ref = O.select_keep(s_ref, inp["roles"][b], quota[b], wl.W)
        check_kept_set(bufs.idx[l, b, j, :n].cpu().numpy(), idx_ref, s_ref, inp["roles"][b], wl.W, quota[b])
    del inp
    torch.cuda.empty_cache()


def window_lse_torch(q, k, wl):
    """Window-row log-sum-exp [L, B, Hq, W] in float32 on the device, layer by
    layer (test input only, as a prefill attention kernel would return it)."""
    L = k.shape[0]
    out = torch.empty((L, wl.B, wl.Hq, wl.W), dtype=torch.float32, device=k.device)
    pos = torch.arange(wl.N - wl.W, wl.N, device=k.device)
    t = torch.arange(wl.N, device=k.device)
    mask = t[None, :] <= pos[:, None]                                   # [W, N]
    scale = 1.0 / math.sqrt(wl.d)
    for l in range(L):
        qf = q[l].float().reshape(wl.B, wl.Hkv, wl.G * wl.W, wl.d)
        kf = k[l].float().transpose(-1, -2).contiguous()                 # [B, Hkv, d, N]
        x = torch.matmul(qf, kf) * scale                                # [B, Hkv, G*W, N]
        x = x.reshape(wl.B, wl.Hkv, wl.G, wl.W, wl.N).masked_fill(~mask, float("-inf"))
        out[l] = torch.logsumexp(x, dim=-1).reshape(wl.B, wl.Hq, wl.W)
    return out


# ---------------------------------------------------------------------------
# Decode through the keep-set over the compacted cache
# ---------------------------------------------------------------------------

def _decode_ref(q, kc, vc, count, scale=None):
    """Oracle output, the same with |v| (the bound's magnitude) and the largest
    |logit| in natural-log units, for q [L, B, Hq, d], caches [L, B, Hkv, k_cap, d]."""
    ref = O.decode_attention_batch(q, kc, vc, count, scale)
    ref_abs = O.decode_attention_batch(q, kc, np.abs(vc), count, scale)
    L, B, Hq, d = q.shape
    Hkv, k_cap = kc.shape[2], kc.shape[3]
    G = Hq // Hkv
    s = 1.0 / math.sqrt(d) if scale is None else scale
    xmax = 0.0
    for l, b, j in np.ndindex(L, B, Hkv):
        n = int(min(max(int(count[l, b, j]), 0), k_cap))
        if n:
            xmax = max(xmax, float(np.max(np.abs(s * q[l, b, j * G:(j + 1) * G] @ kc[l, b, j, :n].T))))
    return ref, ref_abs, xmax


DECODE_CASES = [
    # name, L, B, Hq, Hkv, k_cap, d, dtype, q gain
    ("g4", 2, 2, 8, 2, 300, 128, "bf16", 3.0),
    ("g1", 1, 2, 4, 4, 77, 128, "bf16", 3.0),
    ("g8", 1, 1, 16, 2, 513, 128, "bf16", 3.0),
    ("g3", 1, 2, 6, 2, 129, 128, "bf16", 3.0),
    ("g6d64", 2, 1, 12, 2, 1000, 64, "bf16", 3.0),
    ("kcap1", 1, 1, 8, 2, 1, 128, "bf16", 3.0),
    ("splits", 1, 2, 8, 1, 7000, 128, "bf16", 3.0),
    ("hot", 1, 2, 8, 2, 2000, 128, "bf16", 25.0),
    ("f32", 1, 2, 8, 2, 260, 128, "f32", 3.0),
    ("f32d64g8", 1, 1, 8, 1, 333, 64, "f32", 3.0),
]


@pytest.mark.parametrize("case", DECODE_CASES, ids=lambda c: c[0])
def test_decode_matches_oracle(K, case):
    """Ragged counts (0, 1, k_cap, above k_cap, in between), rows at and beyond
    the count filled with NaN (they must never be read into the result), and a
    workspace filled with NaN bytes."""
    name, L, B, Hq, Hkv, k_cap, d, dt, gain = case
    note(f"decode {name}")
    tdt = torch.bfloat16 if dt == "bf16" else torch.float32
    g = torch.Generator(device="cpu")
    g.manual_seed(1234 + len(name))
    q = (gain * torch.randn((L, B, Hq, d), generator=g)).to(tdt)
    kc = torch.randn((L, B, Hkv, k_cap, d), generator=g).to(tdt)
    vc = torch.randn((L, B, Hkv, k_cap, d), generator=g).to(tdt)
    r = np.random.default_rng(77)
    count = r.integers(0, k_cap + 1, (L, B, Hkv)).astype(np.int32)
    flat = count.reshape(-1)
    specials = [0, 1, k_cap, k_cap + 5, -3]
    for i in range(min(len(flat), len(specials))):
        flat[i] = specials[i]
    count = flat.reshape(count.shape)
    for idx in np.ndindex(L, B, Hkv):
        n = int(min(max(int(count[idx]), 0), k_cap))
        kc[idx][n:] = float("nan")
        vc[idx][n:] = float("nan")
    qd, kd, vd = q.cuda(), kc.cuda(), vc.cuda()
    cd = torch.from_numpy(count).cuda()
    ws = torch.full((K.decode_workspace_size(L, B, Hq, Hkv, k_cap, d),), 0xFF, dtype=torch.uint8, device="cuda")
    out = K.decode_attention(qd, kd, vd, cd, workspace=ws)
    torch.cuda.synchronize()
    kc64, vc64 = f64(kc), f64(vc)
    kc64 = np.nan_to_num(kc64, nan=0.0)
    vc64 = np.nan_to_num(vc64, nan=0.0)
    ref, ref_abs, xmax = _decode_ref(f64(q), kc64, vc64, count)
    r = check_decode(out.cpu().numpy(), ref, ref_abs, xmax, f"decode {name}")
    report(f"decode worst err/bound {name}", round(r, 4))
    # empty segments give zeros
    for idx in np.ndindex(L, B, Hkv):
        if min(max(int(count[idx]), 0), k_cap) == 0:
            G = Hq // Hkv
            assert not out[idx[0], idx[1], idx[2] * G:(idx[2] + 1) * G].any()


def test_decode_explicit_scale_and_repeat(K):
    L, B, Hq, Hkv, k_cap, d = 1, 2, 8, 2, 400, 128
    g = torch.Generator(device="cpu")
    g.manual_seed(99)
    q = torch.randn((L, B, Hq, d), generator=g).to(torch.bfloat16)
    kc = torch.randn((L, B, Hkv, k_cap, d), generator=g).to(torch.bfloat16)
    vc = torch.randn((L, B, Hkv, k_cap, d), generator=g).to(torch.bfloat16)
    count = np.full((L, B, Hkv), k_cap, dtype=np.int32)
    cd = torch.from_numpy(count).cuda()
    out1 = K.decode_attention(q.cuda(), kc.cuda(), vc.cuda(), cd, scale=0.3)
    out2 = K.decode_attention(q.cuda(), kc.cuda(), vc.cuda(), cd, scale=0.3)
    torch.cuda.synchronize()
    assert torch.equal(out1, out2)
    ref, ref_abs, xmax = _decode_ref(f64(q), f64(kc), f64(vc), count, scale=0.3)
    check_decode(out1.cpu().numpy(), ref, ref_abs, xmax, "decode scale 0.3")


def _decode_after_eviction(K, wl, inp, budget, segs):
    """Evict with the role policy, decode one new query per head over the
    compacted cache, and compare with decoding through the keep-mask over the
    full cache (the paper's harness form) for the sampled segments."""
    from paper_2607_13205_amd import pipeline
    W = wl.W
    alpha = WL.default_alpha(0.0)
    _, _, k_cap = K.role_allocate(inp["roles"], 4, alpha, budget, W)
    bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, W, 4, k_cap)
    pipeline.evict(inp["q"], inp["k"], inp["v"], inp["roles"], inp["roles_t"], alpha, budget, W,
                   wl.pool_k, bufs)
    g = torch.Generator(device="cuda")
    g.manual_seed(4321)
    L = inp["k"].shape[0]
    qd = (3.0 * torch.randn((L, wl.B, wl.Hq, wl.d), generator=g, device="cuda")).to(inp["k"].dtype)
    out = K.decode_attention(qd, bufs.k_out, bufs.v_out, bufs.count)
    torch.cuda.synchronize()
    G = wl.G
    for (l, b, j) in segs:
        n = int(bufs.count[l, b, j])
        idx = bufs.idx[l, b, j, :n].cpu().numpy()
        qs = f64(qd[l, b, j * G:(j + 1) * G])
        kf, vf = f64(inp["k"][l, b, j]), f64(inp["v"][l, b, j])
        ref = O.masked_decode_attention(qs, kf, vf, idx)
        ref_abs = O.masked_decode_attention(qs, kf, np.abs(vf), idx)
        xmax = float(np.max(np.abs(qs @ kf[idx].T))) / math.sqrt(wl.d)
        check_decode(out[l, b, j * G:(j + 1) * G].cpu().numpy(), ref, ref_abs, xmax,
                     f"{wl.name} decode seg {(l, b, j)}")
    return bufs, out


def test_decode_after_eviction_layer8k(K):
    wl = WL.get_workload("layer8k")
    inp = WL.make_inputs(wl, device="cuda")
    _decode_after_eviction(K, wl, inp, 0.1, list(np.ndindex(len(inp["layers"]), wl.B, wl.Hkv)))


# ---------------------------------------------------------------------------
# One-shot Quest analogue
# ---------------------------------------------------------------------------

QUEST_CASES = [
    # name, L, B, Hq, Hkv, N, W, d, dtype, page
    ("q16", 2, 2, 8, 2, 1000, 24, 128, "bf16", 16),
    ("g1", 1, 1, 4, 4, 300, 8, 128, "bf16", 16),
    ("g8", 1, 1, 16, 2, 513, 20, 128, "bf16", 16),
    ("g3d64", 1, 2, 6, 2, 700, 16, 64, "bf16", 16),
    ("page1", 1, 1, 8, 2, 200, 8, 128, "bf16", 1),
    ("page37", 1, 1, 8, 2, 900, 8, 128, "bf16", 37),
    ("wfull", 1, 1, 4, 1, 64, 64, 128, "bf16", 16),
    ("f32", 1, 2, 8, 2, 333, 16, 128, "f32", 16),
    ("f32d64", 1, 1, 8, 1, 500, 9, 64, "f32", 8),
    ("kv3", 2, 2, 12, 3, 700, 13, 128, "bf16", 16),
    ("long", 2, 1, 8, 2, 20000, 32, 128, "bf16", 16),
]


@pytest.mark.parametrize("case", [QUEST_CASES[0], QUEST_CASES[3], QUEST_CASES[7]], ids=lambda c: c[0])
@pytest.mark.parametrize("pad", [0, 8])
def test_quest_strided_views_match_dense(K, case, pad):
    """The window queries as the tail of all prefill queries and the keys
    token-major through kve_quest_score_strided: bit-identical to the dense call."""
    name, L, B, Hq, Hkv, N, W, d, dt, page = case
    note(f"quest strided views {name} pad={pad}")
    wl = custom(name, L, B, Hq, Hkv, N, W, d, 1, dt, scorer="quest")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    qv, kv = _strided_views(inp["q"], inp["k"], pad)
    dense = K.quest_score(inp["q"], inp["k"], page)
    strided = K.quest_score_strided(qv, kv, page)
    torch.cuda.synchronize()
    assert torch.equal(strided, dense)


@pytest.mark.parametrize("case", QUEST_CASES, ids=lambda c: c[0])
def test_quest_score_matches_oracle(K, case):
    name, L, B, Hq, Hkv, N, W, d, dt, page = case
    note(f"quest {name}")
    wl = custom(name, L, B, Hq, Hkv, N, W, d, 1, dt, scorer="quest")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    ws = torch.full((K.quest_workspace_size(L, B, Hq, Hkv, d),), 0xFF, dtype=torch.uint8, device="cuda")
    sc = torch.full((L, B, Hkv, N), float("nan"), device="cuda")
    K.quest_score(inp["q"], inp["k"], page, score=sc, workspace=ws)
    torch.cuda.synchronize()
    ref = O.quest_score(f64(inp["q"]), f64(inp["k"]), Hkv, page)
    got = sc.cpu().numpy().astype(np.float64)
    for idx in np.ndindex(L, B, Hkv):
        check_quest_or_scores(got[idx], ref[idx], W, f"quest {name} seg {idx}")
        # every token of a page carries the same bits
        P = N - W
        for p0 in range(0, P, page):
            assert np.all(got[idx][p0:min(p0 + page, P)] == got[idx][p0])


@pytest.mark.parametrize("budget,pol", [(0.1, "role"), (0.3, "role"), (0.1, "neutral")])
def test_pipeline_quest(K, budget, pol):
    wl = custom("quest_pipe", 2, 2, 8, 2, 3000, 32, 128, 1, "bf16", scorer="quest")
    note(f"pipeline quest B={budget} {pol}")
    inp = WL.make_inputs(wl, device="cuda")
    if pol == "neutral":
        from paper_2607_13205_amd.pipeline import Policy
        roles1 = np.zeros_like(inp["roles"])
        inp = dict(inp, roles=roles1, roles_t=torch.from_numpy(roles1).cuda())
        policy = Policy(1, (1.0,))
    else:
        policy = WL.default_alpha(0.0)
    _pipeline_check(K, wl, inp, budget, policy)


def test_quest_full_size_one_layer(K):
    """stack32k's shape (one layer of the 32): the launch configuration of a
    whole-stack call at a quarter of the depth is the same per segment."""
    wl = WL.get_workload("stack32k")
    note("quest stack32k layer 5")
    inp = WL.make_inputs(wl, device="cuda", layers=[5], with_v=False)
    sc = K.quest_score(inp["q"], inp["k"], 16)
    torch.cuda.synchronize()
    for (b, j) in [(0, 0), (3, 7)]:
        ref = O.quest_mass(f64(inp["q"][0, b, j * wl.G:(j + 1) * wl.G]), f64(inp["k"][0, b, j]), 16)
        check_quest_or_scores(sc[0, b, j].cpu().numpy().astype(np.float64), ref, wl.W, f"quest stack32k {(b, j)}")


def test_quest_full_size_all_layers(K):
    """The Quest leg's launch configuration: all 32 layers of stack32k in one
    call; sampled segments against the oracle."""
    wl = WL.get_workload("stack32k")
    note("quest stack32k, all layers in one call (sampled segments)")
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    sc = K.quest_score(inp["q"], inp["k"], 16)
    torch.cuda.synchronize()
    for (l, b, j) in [(0, 0, 0), (13, 1, 4), (31, 3, 7)]:
        ref = O.quest_mass(f64(inp["q"][l, b, j * wl.G:(j + 1) * wl.G]), f64(inp["k"][l, b, j]), 16)
        check_quest_or_scores(sc[l, b, j].cpu().numpy().astype(np.float64), ref, wl.W,
                              f"quest stack32k {(l, b, j)}")


# ---------------------------------------------------------------------------
# Linear role probe
# ---------------------------------------------------------------------------

def _probe_tables(V, R, seed):
    g = torch.Generator(device="cpu")
    g.manual_seed(seed)
    weight = (0.1 * torch.randn((5, V, R), generator=g)).float()
    bias = (0.1 * torch.randn((R,), generator=g)).float()
    return weight, bias


@pytest.mark.parametrize("B,N,V,R", [(4, 3000, 128256, 6), (3, 1, 50, 6), (2, 2, 50, 3), (1, 5, 7, 8),
                                     (2, 777, 1000, 1), (1, 4100, 32000, 5)])
def test_role_probe_bit_exact(K, B, N, V, R):
    """Labels are decided in float32 in the same order on both sides, so they
    agree bit for bit; out-of-vocabulary ids add nothing."""
    note(f"probe B={B} N={N} V={V} R={R}")
    weight, bias = _probe_tables(V, R, 7 + N)
    r = np.random.default_rng(N)
    ids = r.integers(0, V, (B, N)).astype(np.int32)
    ids[r.random((B, N)) < 0.02] = -5
    ids[r.random((B, N)) < 0.02] = V + 3
    out = K.role_probe(torch.from_numpy(ids).cuda(), weight.cuda(), bias.cuda())
    torch.cuda.synchronize()
    ref = O.probe_roles(ids, weight.numpy(), bias.numpy())
    assert np.array_equal(out.cpu().numpy(), ref)


def test_probe_drives_the_pipeline(K):
    """Probe labels on the device, mapped to the four buckets, feed the
    allocation and the selection like parser labels."""
    from paper_2607_13205_amd import pipeline
    wl = WL.get_workload("layer8k").with_(Hq=8, Hkv=2)
    inp = WL.make_inputs(wl, device="cuda")
    weight, bias = _probe_tables(32000, 6, 3)
    ids = np.random.default_rng(5).integers(0, 32000, (wl.B, wl.N)).astype(np.int32)
    buckets, buckets_t = pipeline.probe_buckets(torch.from_numpy(ids).cuda(), weight.cuda(), bias.cuda())
    ref = O.role_map(O.probe_roles(ids, weight.numpy(), bias.numpy()), pipeline.PROBE_TO_BUCKET)
    assert np.array_equal(buckets, ref)
    inp = dict(inp, roles=buckets, roles_t=buckets_t)
    _pipeline_check(K, wl, inp, 0.1, WL.default_alpha(0.02))


def test_role_probe_full_size(K):
    """stack32k's batch (4 x 32768 tokens) with a Llama-3-sized vocabulary;
    the oracle recomputes the first and the last sequence."""
    B, N, V, R = 4, 32768, 128256, 6
    weight, bias = _probe_tables(V, R, 11)
    ids = np.random.default_rng(9).integers(0, V, (B, N)).astype(np.int32)
    out = K.role_probe(torch.from_numpy(ids).cuda(), weight.cuda(), bias.cuda())
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    for b in (0, B - 1):
        assert np.array_equal(got[b], O.probe_roles(ids[b], weight.numpy(), bias.numpy()))


# ---------------------------------------------------------------------------
# Fused role epilogue: the score's pool step counts the top-k's first digit
# ---------------------------------------------------------------------------

def _host_role_hist(score, roles, W, R):
    """Histogram [L, B, Hkv, R, 2048] of the candidates' top 11 key bits,
    counted on the host from the scores (order-preserving key: -0 as +0, every
    NaN below -inf)."""
    L, B, H, N = score.shape
    bits = np.ascontiguousarray(score, dtype=np.float32).view(np.uint32).copy()
    bits[bits == 0x80000000] = 0
    key = np.where(bits & 0x80000000, ~bits, bits | 0x80000000).astype(np.uint32)
    key[np.isnan(score)] = 0
    digit = (key >> 21).astype(np.int64)
    out = np.zeros((L, B, H, R, 2048), dtype=np.int64)
    P = N - W
    for l, b, j in np.ndindex(L, B, H):
        lab = roles[b, :P].astype(np.int64)
        ok = (lab >= 0) & (lab < R)
        np.add.at(out[l, b, j], (lab[ok], digit[l, b, j, :P][ok]), 1)
    return out


def _decode_tile_records(words, L, B, H, N, R):
    """The per-segment histograms [L, B, H, R, 2048] the tile records add up to
    (the record layout of include/kve.h), and which segments had a tile whose
    bins overflowed its window."""
    tiles = (N + 4095) // 4096
    tw = 4 + R * 256
    rec = words.view(np.uint32).reshape(L, B, H, tiles, tw)
    out = np.zeros((L, B, H, R, 2048), dtype=np.int64)
    over = np.zeros((L, B, H), dtype=bool)
    for l, b, j, t in np.ndindex(L, B, H, tiles):
        lo, ov = int(rec[l, b, j, t, 0]), int(rec[l, b, j, t, 1])
        if ov:
            over[l, b, j] = True
            continue
        if lo == 0xFFFFFFFF:
            continue
        body = rec[l, b, j, t, 4:].reshape(R, 256)
        cnt = np.stack([body & 0xFFFF, body >> 16], axis=-1).reshape(R, 512).astype(np.int64)
        hi = min(2048, lo + 512)
        out[l, b, j, :, lo:hi] += cnt[:, :hi - lo]
    return out, over


FUSED_CASES = [
    # name, L, B, Hq, Hkv, N, W, d, pool, dtype, R, budget
    ("tiny_f32", 1, 1, 2, 1, 512, 16, 64, 5, "f32", 4, 0.10),
    ("layer8k", 1, 1, 32, 8, 8192, 32, 128, 7, "bf16", 4, 0.05),
    ("ragged_pool1", 2, 2, 8, 2, 3001, 24, 128, 1, "bf16", 4, 0.20),
    ("ragged_pool7", 2, 2, 8, 2, 5003, 32, 128, 7, "bf16", 3, 0.10),
    ("r1", 2, 1, 8, 2, 4096, 32, 128, 7, "bf16", 1, 0.10),
    ("r8_labels_out_of_range", 1, 2, 8, 2, 6000, 16, 128, 7, "bf16", 8, 0.30),
    ("overflow", 1, 1, 4, 1, 4096, 16, 128, 7, "bf16", 4, 0.10),
]


@pytest.mark.parametrize("case", FUSED_CASES, ids=lambda c: c[0])
def test_fused_role_epilogue_matches_unfused(K, case):
    """kve_snapkv_score_hist + kve_topk_select_hist against kve_snapkv_score +
    kve_topk_select: scores, kept indices and counts bit for bit, and the
    histograms equal to the host's count over the GPU's scores."""
    name, L, B, Hq, Hkv, N, W, d, pool, dt, R, budget = case
    note(f"fused role epilogue {name}")
    wl = custom(name, L, B, Hq, Hkv, N, W, d, pool, dt)
    inp = WL.make_inputs(wl, device="cuda", with_v=False)
    if name == "overflow":
        # every window query along one direction, one key far along it: that key
        # takes all the mass (pooled score near G*W = 64, about bin 1560) while
        # the keys beyond its pool window score exactly 0 (bin 1024) in the same
        # tile: the bins span more than the 512-bin window
        u = torch.zeros(d, device="cuda")
        u[0] = 1.0
        inp["q"][:] = (4.0 * u).to(inp["q"].dtype)
        inp["k"][:] = (0.01 * torch.randn_like(inp["k"], dtype=torch.float32)).to(inp["k"].dtype)
        inp["k"][0, 0, 0, 1000] = (400.0 * u).to(inp["k"].dtype)
    rng = np.random.default_rng(11)
    roles = rng.integers(0, R, (B, N)).astype(np.int8)
    if name.startswith("r8"):
        roles[rng.random((B, N)) < 0.1] = -3      # labels outside [0, R): never counted, never kept
        roles[rng.random((B, N)) < 0.05] = 9
    rd = torch.from_numpy(roles).cuda()
    alpha = [1.0 / R] * R
    clean = np.where((roles >= 0) & (roles < R), roles, 0).astype(np.int8)
    quota, kept, k_cap = K.role_allocate(clean, R, alpha, budget, W)
    qd = torch.from_numpy(quota).cuda()
    ws = torch.full((K.snapkv_workspace_size(L, B, Hq, Hkv, N, W, d),), 0xFF, dtype=torch.uint8, device="cuda")
    hist = torch.full((K.role_hist_size(L, B, Hkv, N, R) // 4,), 12345, dtype=torch.int32, device="cuda")  # stale
    s_f, h_f = K.snapkv_score_hist(inp["q"], inp["k"], rd, R, pool, hist=hist, workspace=ws)
    i_f, c_f = K.topk_select_hist(s_f, rd, qd, h_f, W, R, k_cap)
    s_u = K.snapkv_score(inp["q"], inp["k"], pool)
    i_u, c_u = K.topk_select(s_u, rd, qd, W, R, k_cap)
    torch.cuda.synchronize()
    assert torch.equal(s_f.view(torch.int32), s_u.view(torch.int32)), "fused scores differ"
    assert torch.equal(c_f, c_u), "fused counts differ"
    cnt = c_u.cpu().numpy()
    fi, ui = i_f.cpu().numpy(), i_u.cpu().numpy()
    for idx in np.ndindex(L, B, Hkv):
        n = int(cnt[idx])
        assert np.array_equal(fi[idx][:n], ui[idx][:n]), idx
    ref = _host_role_hist(s_u.cpu().numpy(), roles, W, R)
    got, over = _decode_tile_records(h_f.cpu().numpy(), L, B, Hkv, N, R)
    assert np.array_equal(got[~over], ref[~over]), "histogram differs from the host count"
    report(f"fused epilogue {name}: segments counted in the top-k's own sweep (a tile overflowed)",
           int(over.sum()))
    if name == "overflow":
        assert over.any()


def test_fused_pipeline_matches_unfused_stack32k(K):
    """The step with the fused epilogue against the same step with the
    separate calls (the default): every index, count and compacted row."""
    from paper_2607_13205_amd import pipeline
    wl = WL.get_workload("stack32k")
    note("fused vs unfused pipeline stack32k")
    inp = WL.make_inputs(wl, device="cuda")
    alpha = WL.default_alpha(0.0)
    _, _, k_cap = K.role_allocate(inp["roles"], 4, alpha, 0.05, wl.W)
    res = []
    for fused in (True, False):
        bufs = pipeline.alloc_buffers(inp["k"], wl.Hq, wl.W, 4, k_cap, fused=fused)
        assert (bufs.hist is not None) == fused
        pipeline.evict(inp["q"], inp["k"], inp["v"], inp["roles"], inp["roles_t"], alpha, 0.05, wl.W, wl.pool_k, bufs)
        torch.cuda.synchronize()
        res.append(bufs)
    a, b = res
    assert torch.equal(a.score.view(torch.int32), b.score.view(torch.int32))
    assert torch.equal(a.count, b.count) and torch.equal(a.idx, b.idx)
    assert torch.equal(a.k_out.view(torch.int16), b.k_out.view(torch.int16))
    assert torch.equal(a.v_out.view(torch.int16), b.v_out.view(torch.int16))
    del inp, res, a, b
    torch.cuda.empty_cache()
