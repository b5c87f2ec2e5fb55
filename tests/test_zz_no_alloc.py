"""kve_snapkv_score_noalloc: the SnapKV score with its workspace in the
library's static device scratch array, called through the C ABI and compared
with kve_snapkv_score (the same kernels with a caller's workspace) and with
the oracle, on two calls in a row, the second with a smaller input."""

import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle as O  # noqa: E402
import workload as WL  # noqa: E402
from tests.parity import check_scores  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def K():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_13205_amd.build import ensure_built
    ensure_built()
    import paper_2607_13205_amd as K
    return K


def _noalloc(K, q, k, W, pool_k):
    """One call of kve_snapkv_score_noalloc through the C ABI."""
    L, B, Hq, _, d = q.shape
    Hkv, N = k.shape[2], k.shape[3]
    score = torch.full((L, B, Hkv, N), float("nan"), dtype=torch.float32, device=k.device)
    dt = 0 if k.dtype == torch.bfloat16 else 1
    st = K.binding.LIB.kve_snapkv_score_noalloc(
        ctypes.c_void_p(q.data_ptr()), ctypes.c_void_p(k.data_ptr()), dt, L, B, Hq, Hkv, N, W, d,
        ctypes.c_float(0.0), pool_k, ctypes.c_void_p(score.data_ptr()),
        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, K.last_error()
    return score


def _with_workspace(K, q, k, pool_k):
    return K.snapkv_score(q, k, pool_k)


def test_noalloc_matches_the_workspace_entry_point_on_two_calls(K):
    """A layer8k-shaped call (two layers, 8 KV heads, N = 8192, bf16), then a
    smaller fp32 call (the tiny workload) on the same scratch array: each
    equals kve_snapkv_score bit for bit and the oracle to its tolerance."""
    big = WL.Workload("noalloc_big", L=2, B=1, Hq=32, Hkv=8, N=8192, W=32, d=128, pool_k=7, dtype="bf16",
                      mix=WL.get_workload("layer8k").mix, budgets=(0.05,))
    small = WL.get_workload("tiny")
    for wl in (big, small):
        print(f"noalloc case {wl.name}: L={wl.L} Hq={wl.Hq} Hkv={wl.Hkv} N={wl.N} W={wl.W} {wl.dtype}", flush=True)
        inp = WL.make_inputs(wl, device="cuda:0", with_v=False)
        s_na = _noalloc(K, inp["q"], inp["k"], wl.W, wl.pool_k)
        s_ws = _with_workspace(K, inp["q"], inp["k"], wl.pool_k)
        torch.cuda.synchronize()
        a, b = s_na.cpu().numpy(), s_ws.cpu().numpy()
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32)), wl.name
        # the oracle on one segment per layer (all of them for the small case)
        q64 = inp["q"].double().cpu().numpy()
        k64 = inp["k"].double().cpu().numpy()
        G = wl.Hq // wl.Hkv
        for l in range(wl.L):
            j = (3 * l) % wl.Hkv
            ref = O.maxpool_prefix(O.snapkv_mass(q64[l, 0, j * G:(j + 1) * G], k64[l, 0, j]), wl.W, wl.pool_k)
            check_scores(a[l, 0, j], ref, f"noalloc {wl.name} layer {l} head {j}")


def test_noalloc_rejects_shapes_above_the_scratch_size(K):
    """16 layers of a batch-4, N = 32768 stack need more than the 64 MiB array:
    a clear error, nothing launched, the output untouched."""
    lib = K.binding.LIB
    cap = int(lib.kve_snapkv_scratch_bytes())
    assert cap == 64 << 20
    assert K.snapkv_workspace_size(16, 4, 32, 8, 32768, 32, 128) > cap
    assert K.snapkv_workspace_size(15, 4, 32, 8, 32768, 32, 128) <= cap
    out = torch.zeros(16, dtype=torch.float32, device="cuda")
    dummy = ctypes.c_void_p(out.data_ptr())
    st = lib.kve_snapkv_score_noalloc(dummy, dummy, 0, 16, 4, 32, 8, 32768, 32, 128, ctypes.c_float(0.0), 7,
                                      dummy, ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 3 and "static scratch" in K.last_error()
    torch.cuda.synchronize()
    assert torch.count_nonzero(out).item() == 0
