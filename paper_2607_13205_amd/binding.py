"""Thin ctypes binding of libkve.so (argument marshalling only).

Every step of the eviction path runs in the HIP library; this module only
checks tensor shapes against the C ABI, allocates outputs and workspaces with
torch when the caller does not pass them, and forwards raw device pointers and
the current HIP stream.  There is no fallback: the first call into the
library (any entry point below) raises ImportError if libkve.so is missing.
The library is opened on first use, so that the package (and its build
module) can be imported before the library is built.
"""

from __future__ import annotations

import ctypes
import os

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libkve.so")

KVE_OK = 0
KVE_ERR_INVALID_ARG = 1
KVE_ERR_UNSUPPORTED = 2
KVE_ERR_WORKSPACE = 3
KVE_ERR_HIP = 4
DTYPE_BF16 = 0
DTYPE_F32 = 1

#: every symbol include/kve.h declares
EXPORTED = (
    "kve_version", "kve_last_error", "kve_source_hash",
    "kve_snapkv_workspace_size", "kve_snapkv_score", "kve_snapkv_score_lse",
    "kve_snapkv_score_noalloc", "kve_snapkv_scratch_bytes",
    "kve_h2o_workspace_size", "kve_h2o_score", "kve_h2o_score_strided",
    "kve_role_allocate", "kve_role_allocate_fair", "kve_role_map", "kve_role_probe",
    "kve_topk_workspace_size", "kve_topk_select",
    "kve_role_hist_size", "kve_snapkv_score_hist", "kve_topk_select_hist",
    "kve_kv_compact", "kve_snapkv_score_strided", "kve_kv_compact_strided",
    "kve_decode_workspace_size", "kve_decode_attention",
    "kve_quest_workspace_size", "kve_quest_score", "kve_quest_score_strided",
    "kve_read_probe",
)


class Strides(ctypes.Structure):
    """kve_strides_t: element strides of a [layer, batch, head, token] view of
    rows of d contiguous elements."""
    _fields_ = [("layer", ctypes.c_int64), ("batch", ctypes.c_int64), ("head", ctypes.c_int64),
                ("token", ctypes.c_int64)]


class KveError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"kve status {status}: {message}")
        self.status = status


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(
            f"{_LIB_PATH} is missing: build it with `python -m paper_2607_13205_amd.build` "
            "(or __graft_entry__.build()); there is no non-HIP fallback")
    lib = ctypes.CDLL(_LIB_PATH)
    c_int, c_size, c_void, c_float, c_double = (ctypes.c_int, ctypes.c_size_t, ctypes.c_void_p,
                                                ctypes.c_float, ctypes.c_double)
    sig = {
        "kve_version": (c_int, []),
        "kve_last_error": (ctypes.c_char_p, []),
        "kve_source_hash": (ctypes.c_char_p, []),
        "kve_snapkv_workspace_size": (c_size, [c_int] * 7),
        "kve_snapkv_score": (c_int, [c_void, c_void, c_int] + [c_int] * 7 +
                             [c_float, c_int, c_void, c_void, c_size, c_void]),
        "kve_snapkv_score_lse": (c_int, [c_void, c_void, c_void, c_int] + [c_int] * 7 +
                                 [c_float, c_int, c_void, c_void, c_size, c_void]),
        "kve_snapkv_score_noalloc": (c_int, [c_void, c_void, c_int] + [c_int] * 7 +
                                     [c_float, c_int, c_void, c_void]),
        "kve_snapkv_scratch_bytes": (c_size, []),
        "kve_h2o_workspace_size": (c_size, [c_int] * 6),
        "kve_h2o_score": (c_int, [c_void, c_void, c_int] + [c_int] * 6 +
                          [c_float, c_void, c_void, c_size, c_void]),
        "kve_h2o_score_strided": (c_int, [c_void, c_void, c_void, c_void, c_int] + [c_int] * 6 +
                                  [c_float, c_void, c_void, c_size, c_void]),
        "kve_role_allocate": (c_int, [c_void, c_int, c_int, c_int, c_void, c_double, c_int,
                                      c_void, c_void, c_void]),
        "kve_role_allocate_fair": (c_int, [c_void, c_int, c_int, c_int, c_double, c_int,
                                           c_void, c_void, c_void]),
        "kve_role_map": (c_int, [c_void, c_size, c_void, c_int, c_void]),
        "kve_role_probe": (c_int, [c_void, c_int, c_int, c_void, c_void, c_int, c_int, c_void, c_void]),
        "kve_topk_workspace_size": (c_size, [c_int] * 5),
        "kve_topk_select": (c_int, [c_void, c_void, c_void] + [c_int] * 7 +
                            [c_void, c_void, c_void, c_size, c_void]),
        "kve_role_hist_size": (c_size, [c_int] * 5),
        "kve_snapkv_score_hist": (c_int, [c_void, c_void, c_int] + [c_int] * 7 +
                                  [c_float, c_int, c_void, c_int, c_void, c_void, c_void, c_size, c_void]),
        "kve_topk_select_hist": (c_int, [c_void, c_void, c_void, c_void] + [c_int] * 7 +
                                 [c_void, c_void, c_void, c_size, c_void]),
        "kve_kv_compact": (c_int, [c_void, c_void, c_int, c_void, c_void] + [c_int] * 6 +
                           [c_void, c_void, c_void]),
        "kve_snapkv_score_strided": (c_int, [c_void, c_void, c_void, c_void, c_int] + [c_int] * 7 +
                                     [c_float, c_int, c_void, c_void, c_size, c_void]),
        "kve_kv_compact_strided": (c_int, [c_void, c_void, c_void, c_void, c_int, c_void, c_void] +
                                   [c_int] * 6 + [c_void, c_void, c_void]),
        "kve_decode_workspace_size": (c_size, [c_int] * 6),
        "kve_quest_workspace_size": (c_size, [c_int] * 5),
        "kve_quest_score": (c_int, [c_void, c_void, c_int] + [c_int] * 8 + [c_void, c_void, c_size, c_void]),
        "kve_quest_score_strided": (c_int, [c_void, c_void, c_void, c_void, c_int] + [c_int] * 8 +
                                    [c_void, c_void, c_size, c_void]),
        "kve_read_probe": (c_int, [c_void, c_size, c_int, c_void, c_int, c_void]),
        "kve_decode_attention": (c_int, [c_void, c_void, c_void, c_void, c_int] + [c_int] * 6 +
                                 [c_float, c_void, c_void, c_size, c_void]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


class _Lib:
    """libkve.so, opened on first attribute access."""

    _cdll = None

    def __getattr__(self, name):
        if _Lib._cdll is None:
            _Lib._cdll = _load()
        return getattr(_Lib._cdll, name)


LIB = _Lib()


def last_error() -> str:
    return LIB.kve_last_error().decode()


def source_hash() -> str:
    """SHA-256 of the sources the loaded library was built from."""
    return LIB.kve_source_hash().decode()


def _check(status: int):
    if status != KVE_OK:
        raise KveError(status, last_error())


# ---------------------------------------------------------------------------
# torch plumbing
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return DTYPE_BF16
    if t.dtype == torch.float32:
        return DTYPE_F32
    raise TypeError(f"unsupported dtype {t.dtype} (bfloat16 or float32)")


def _dev(t, name):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _view(t, name):
    """(pointer, Strides) of a 5-D device tensor whose last dimension is
    contiguous, for the strided entry points."""
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dim() != 5 or (t.shape[4] > 1 and t.stride(4) != 1):
        raise ValueError(f"{name} must be 5-D with a contiguous last dimension")
    st = Strides(*(int(t.stride(i)) for i in range(4)))
    return ctypes.c_void_p(t.data_ptr()), st


def _stream(stream=None):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _workspace(size, device, workspace=None):
    """(tensor, bytes) of the caller's workspace, or of one allocated here of
    size() bytes (the size is only computed when allocating: the library checks
    a caller's workspace itself)."""
    torch = _torch()
    if workspace is not None:
        return workspace, workspace.numel() * workspace.element_size()
    nbytes = size()
    if nbytes == 0:
        return None, 0
    return torch.empty(int(nbytes), dtype=torch.uint8, device=device), int(nbytes)


def _ptr(t):
    return ctypes.c_void_p(0 if t is None else t.data_ptr())


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------

def snapkv_workspace_size(L, B, Hq, Hkv, N, W, d) -> int:
    return int(LIB.kve_snapkv_workspace_size(L, B, Hq, Hkv, N, W, d))


def snapkv_score(q_win, k, pool_k: int, scale: float = 0.0, score=None, workspace=None,
                 stream=None):
    """Pooled SnapKV score [L, B, Hkv, N] (float32) of q_win [L, B, Hq, W, d]
    and k [L, B, Hkv, N, d]; see kve_snapkv_score in include/kve.h."""
    torch = _torch()
    L, B, Hq, W, d = q_win.shape
    Lk, Bk, Hkv, N, dk = k.shape
    if (L, B, d) != (Lk, Bk, dk) or q_win.dtype != k.dtype:
        raise ValueError("q_win and k disagree in L, B, d or dtype")
    if not (q_win.is_contiguous() and k.is_contiguous()):
        return snapkv_score_strided(q_win, k, pool_k, scale, score, workspace, stream)
    if score is None:
        score = torch.empty((L, B, Hkv, N), dtype=torch.float32, device=k.device)
    ws, wsb = _workspace(lambda: snapkv_workspace_size(L, B, Hq, Hkv, N, W, d), k.device, workspace)
    _check(LIB.kve_snapkv_score(_dev(q_win, "q_win"), _dev(k, "k"), _dtype_code(k),
                                L, B, Hq, Hkv, N, W, d, float(scale), int(pool_k),
                                _dev(score, "score"), _ptr(ws), wsb, _stream(stream)))
    return score


def snapkv_score_strided(q_win, k, pool_k: int, scale: float = 0.0, score=None, workspace=None,
                         stream=None):
    """snapkv_score on views: q_win [L, B, Hq, W, d] and k [L, B, Hkv, N, d]
    may have any strides with a contiguous last dimension (e.g. q_full[..., -W:, :]
    or a token-major cache permuted to [L, B, Hkv, N, d]); see
    kve_snapkv_score_strided in include/kve.h."""
    torch = _torch()
    L, B, Hq, W, d = q_win.shape
    Lk, Bk, Hkv, N, dk = k.shape
    if (L, B, d) != (Lk, Bk, dk) or q_win.dtype != k.dtype:
        raise ValueError("q_win and k disagree in L, B, d or dtype")
    if score is None:
        score = torch.empty((L, B, Hkv, N), dtype=torch.float32, device=k.device)
    ws, wsb = _workspace(lambda: snapkv_workspace_size(L, B, Hq, Hkv, N, W, d), k.device, workspace)
    qp, qs = _view(q_win, "q_win")
    kp, ks = _view(k, "k")
    _check(LIB.kve_snapkv_score_strided(qp, ctypes.byref(qs), kp, ctypes.byref(ks), _dtype_code(k),
                                        L, B, Hq, Hkv, N, W, d, float(scale), int(pool_k),
                                        _dev(score, "score"), _ptr(ws), wsb, _stream(stream)))
    return score


def snapkv_score_lse(q_win, k, lse_win, pool_k: int, scale: float = 0.0, score=None, workspace=None,
                     stream=None):
    """snapkv_score with the window rows' natural-log log-sum-exp supplied
    (float32 [L, B, Hq, W], as a prefill attention kernel returns it): K is
    read once."""
    torch = _torch()
    L, B, Hq, W, d = q_win.shape
    Lk, Bk, Hkv, N, dk = k.shape
    if (L, B, d) != (Lk, Bk, dk) or q_win.dtype != k.dtype:
        raise ValueError("q_win and k disagree in L, B, d or dtype")
    if tuple(lse_win.shape) != (L, B, Hq, W) or lse_win.dtype != torch.float32:
        raise ValueError("lse_win must be float32 [L, B, Hq, W]")
    if score is None:
        score = torch.empty((L, B, Hkv, N), dtype=torch.float32, device=k.device)
    ws, wsb = _workspace(lambda: snapkv_workspace_size(L, B, Hq, Hkv, N, W, d), k.device, workspace)
    _check(LIB.kve_snapkv_score_lse(_dev(q_win, "q_win"), _dev(k, "k"), _dev(lse_win, "lse_win"), _dtype_code(k),
                                    L, B, Hq, Hkv, N, W, d, float(scale), int(pool_k), _dev(score, "score"),
                                    _ptr(ws), wsb, _stream(stream)))
    return score


def snapkv_score_noalloc(q_win, k, pool_k: int, scale: float = 0.0, score=None, stream=None):
    """snapkv_score with the workspace taken from the library's static device
    scratch array (kve_snapkv_score_noalloc): the library allocates nothing."""
    torch = _torch()
    L, B, Hq, W, d = q_win.shape
    Lk, Bk, Hkv, N, dk = k.shape
    if (L, B, d) != (Lk, Bk, dk) or q_win.dtype != k.dtype:
        raise ValueError("q_win and k disagree in L, B, d or dtype")
    if score is None:
        score = torch.empty((L, B, Hkv, N), dtype=torch.float32, device=k.device)
    _check(LIB.kve_snapkv_score_noalloc(_dev(q_win, "q_win"), _dev(k, "k"), _dtype_code(k),
                                        L, B, Hq, Hkv, N, W, d, float(scale), int(pool_k),
                                        _dev(score, "score"), _stream(stream)))
    return score


def h2o_workspace_size(L, B, Hq, Hkv, N, d) -> int:
    return int(LIB.kve_h2o_workspace_size(L, B, Hq, Hkv, N, d))


def h2o_score(q, k, scale: float = 0.0, score=None, workspace=None, stream=None):
    """H2O score [L, B, Hkv, N] of q [L, B, Hq, N, d] and k [L, B, Hkv, N, d]."""
    torch = _torch()
    L, B, Hq, N, d = q.shape
    Lk, Bk, Hkv, Nk, dk = k.shape
    if (L, B, N, d) != (Lk, Bk, Nk, dk) or q.dtype != k.dtype:
        raise ValueError("q and k disagree in L, B, N, d or dtype")
    if not (q.is_contiguous() and k.is_contiguous()):
        return h2o_score_strided(q, k, scale, score, workspace, stream)
    if score is None:
        score = torch.empty((L, B, Hkv, N), dtype=torch.float32, device=k.device)
    ws, wsb = _workspace(lambda: h2o_workspace_size(L, B, Hq, Hkv, N, d), k.device, workspace)
    _check(LIB.kve_h2o_score(_dev(q, "q"), _dev(k, "k"), _dtype_code(k), L, B, Hq, Hkv, N, d,
                             float(scale), _dev(score, "score"), _ptr(ws), wsb, _stream(stream)))
    return score


def h2o_score_strided(q, k, scale: float = 0.0, score=None, workspace=None, stream=None):
    """h2o_score on views: q [L, B, Hq, N, d] and k [L, B, Hkv, N, d] with any
    strides and a contiguous last dimension; see kve_h2o_score_strided."""
    torch = _torch()
    L, B, Hq, N, d = q.shape
    Lk, Bk, Hkv, Nk, dk = k.shape
    if (L, B, N, d) != (Lk, Bk, Nk, dk) or q.dtype != k.dtype:
        raise ValueError("q and k disagree in L, B, N, d or dtype")
    if score is None:
        score = torch.empty((L, B, Hkv, N), dtype=torch.float32, device=k.device)
    ws, wsb = _workspace(lambda: h2o_workspace_size(L, B, Hq, Hkv, N, d), k.device, workspace)
    qp, qs = _view(q, "q")
    kp, ks = _view(k, "k")
    _check(LIB.kve_h2o_score_strided(qp, ctypes.byref(qs), kp, ctypes.byref(ks), _dtype_code(k), L, B, Hq, Hkv,
                                     N, d, float(scale), _dev(score, "score"), _ptr(ws), wsb, _stream(stream)))
    return score


def quest_workspace_size(L, B, Hq, Hkv, d) -> int:
    return int(LIB.kve_quest_workspace_size(L, B, Hq, Hkv, d))


def quest_score(q_win, k, page: int = 16, score=None, workspace=None, stream=None):
    """One-shot Quest page-bound scores [L, B, Hkv, N] (window tokens +inf)."""
    torch = _torch()
    L, B, Hq, W, d = q_win.shape
    Lk, Bk, Hkv, N, dk = k.shape
    if (L, B, d) != (Lk, Bk, dk) or q_win.dtype != k.dtype:
        raise ValueError("q_win and k disagree in L, B, d or dtype")
    if not (q_win.is_contiguous() and k.is_contiguous()):
        return quest_score_strided(q_win, k, page, score, workspace, stream)
    if score is None:
        score = torch.empty((L, B, Hkv, N), dtype=torch.float32, device=k.device)
    ws, wsb = _workspace(lambda: quest_workspace_size(L, B, Hq, Hkv, d), k.device, workspace)
    _check(LIB.kve_quest_score(_dev(q_win, "q_win"), _dev(k, "k"), _dtype_code(k), L, B, Hq, Hkv, N, W, d,
                               int(page), _dev(score, "score"), _ptr(ws), wsb, _stream(stream)))
    return score


def quest_score_strided(q_win, k, page: int = 16, score=None, workspace=None, stream=None):
    """quest_score on views (any strides, contiguous last dimension); see
    kve_quest_score_strided."""
    torch = _torch()
    L, B, Hq, W, d = q_win.shape
    Lk, Bk, Hkv, N, dk = k.shape
    if (L, B, d) != (Lk, Bk, dk) or q_win.dtype != k.dtype:
        raise ValueError("q_win and k disagree in L, B, d or dtype")
    if score is None:
        score = torch.empty((L, B, Hkv, N), dtype=torch.float32, device=k.device)
    ws, wsb = _workspace(lambda: quest_workspace_size(L, B, Hq, Hkv, d), k.device, workspace)
    qp, qs = _view(q_win, "q_win")
    kp, ks = _view(k, "k")
    _check(LIB.kve_quest_score_strided(qp, ctypes.byref(qs), kp, ctypes.byref(ks), _dtype_code(k), L, B, Hq, Hkv,
                                       N, W, d, int(page), _dev(score, "score"), _ptr(ws), wsb, _stream(stream)))
    return score


def role_allocate(roles, R: int, alpha, budget: float, W: int):
    """Host role allocation.  roles: int8 array [B, N] (host).  Returns
    (quota int32 [B, R], kept int32 [B], k_cap)."""
    roles = np.ascontiguousarray(np.asarray(roles, dtype=np.int8))
    if roles.ndim == 1:
        roles = roles[None]
    B, N = roles.shape
    alpha = np.ascontiguousarray(np.asarray(alpha, dtype=np.float64))
    quota = np.zeros((B, R), dtype=np.int32)
    kept = np.zeros(B, dtype=np.int32)
    kcap = ctypes.c_int32(0)
    _check(LIB.kve_role_allocate(roles.ctypes.data_as(ctypes.c_void_p), B, N, int(R),
                                 alpha.ctypes.data_as(ctypes.c_void_p), float(budget), int(W),
                                 quota.ctypes.data_as(ctypes.c_void_p),
                                 kept.ctypes.data_as(ctypes.c_void_p), ctypes.byref(kcap)))
    return quota, kept, int(kcap.value)


def role_allocate_fair(roles, R: int, budget: float, W: int):
    """Fair-eviction quotas (every bucket kept at the same rate), host.
    roles: int8 array [B, N] (host).  Returns (quota int32 [B, R], kept int32 [B], k_cap)."""
    roles = np.ascontiguousarray(np.asarray(roles, dtype=np.int8))
    if roles.ndim == 1:
        roles = roles[None]
    B, N = roles.shape
    quota = np.zeros((B, R), dtype=np.int32)
    kept = np.zeros(B, dtype=np.int32)
    kcap = ctypes.c_int32(0)
    _check(LIB.kve_role_allocate_fair(roles.ctypes.data_as(ctypes.c_void_p), B, N, int(R),
                                      float(budget), int(W),
                                      quota.ctypes.data_as(ctypes.c_void_p),
                                      kept.ctypes.data_as(ctypes.c_void_p), ctypes.byref(kcap)))
    return quota, kept, int(kcap.value)


def role_map(roles, bucket_of):
    """Bucket labels out[i] = bucket_of[roles[i]] (host int8 arrays of any shape)."""
    roles = np.ascontiguousarray(np.asarray(roles, dtype=np.int8))
    bmap = np.ascontiguousarray(np.asarray(bucket_of, dtype=np.int8))
    if bmap.ndim != 1 or bmap.size == 0:
        raise ValueError("bucket_of must be a non-empty 1-D sequence")
    out = np.empty_like(roles)
    _check(LIB.kve_role_map(roles.ctypes.data_as(ctypes.c_void_p), roles.size,
                            bmap.ctypes.data_as(ctypes.c_void_p), int(bmap.size),
                            out.ctypes.data_as(ctypes.c_void_p)))
    return out


def topk_workspace_size(L, B, Hkv, N, R) -> int:
    return int(LIB.kve_topk_workspace_size(L, B, Hkv, N, R))


def topk_select(score, roles, quota, W: int, R: int, k_cap: int, idx_out=None, count_out=None,
                workspace=None, stream=None):
    """Ascending kept indices [L, B, Hkv, k_cap] and per-segment counts [L, B, Hkv]."""
    torch = _torch()
    L, B, Hkv, N = score.shape
    if tuple(roles.shape) != (B, N) or roles.dtype != torch.int8:
        raise ValueError("roles must be int8 [B, N]")
    if tuple(quota.shape) != (B, R) or quota.dtype != torch.int32:
        raise ValueError("quota must be int32 [B, R]")
    if idx_out is None:
        idx_out = torch.full((L, B, Hkv, max(k_cap, 0)), -1, dtype=torch.int32, device=score.device)
    if count_out is None:
        count_out = torch.empty((L, B, Hkv), dtype=torch.int32, device=score.device)
    ws, wsb = _workspace(lambda: topk_workspace_size(L, B, Hkv, N, R), score.device, workspace)
    _check(LIB.kve_topk_select(_dev(score, "score"), _dev(roles, "roles"), _dev(quota, "quota"),
                               L, B, Hkv, N, int(W), int(R), int(k_cap),
                               _dev(idx_out, "idx_out"), _dev(count_out, "count_out"),
                               _ptr(ws), wsb, _stream(stream)))
    return idx_out, count_out


def role_hist_size(L, B, Hkv, N, R) -> int:
    return int(LIB.kve_role_hist_size(L, B, Hkv, N, R))


def snapkv_score_hist(q_win, k, roles, R: int, pool_k: int, scale: float = 0.0, score=None, hist=None,
                      workspace=None, stream=None):
    """snapkv_score with the fused role epilogue: also the per-tile role
    histograms of the pooled scores (kve_snapkv_score_hist; an int32 tensor of
    role_hist_size / 4 words).  Returns (score, hist)."""
    torch = _torch()
    L, B, Hq, W, d = q_win.shape
    Lk, Bk, Hkv, N, dk = k.shape
    if (L, B, d) != (Lk, Bk, dk) or q_win.dtype != k.dtype:
        raise ValueError("q_win and k disagree in L, B, d or dtype")
    if tuple(roles.shape) != (B, N) or roles.dtype != torch.int8:
        raise ValueError("roles must be int8 [B, N]")
    if score is None:
        score = torch.empty((L, B, Hkv, N), dtype=torch.float32, device=k.device)
    if hist is None:
        hist = torch.empty((role_hist_size(L, B, Hkv, N, R) // 4,), dtype=torch.int32, device=k.device)
    ws, wsb = _workspace(lambda: snapkv_workspace_size(L, B, Hq, Hkv, N, W, d), k.device, workspace)
    _check(LIB.kve_snapkv_score_hist(_dev(q_win, "q_win"), _dev(k, "k"), _dtype_code(k),
                                     L, B, Hq, Hkv, N, W, d, float(scale), int(pool_k), _dev(roles, "roles"), int(R),
                                     _dev(score, "score"), _dev(hist, "hist"), _ptr(ws), wsb, _stream(stream)))
    return score, hist


def topk_select_hist(score, roles, quota, hist, W: int, R: int, k_cap: int, idx_out=None, count_out=None,
                     workspace=None, stream=None):
    """topk_select with the first digit's counts from snapkv_score_hist."""
    torch = _torch()
    L, B, Hkv, N = score.shape
    if tuple(roles.shape) != (B, N) or roles.dtype != torch.int8:
        raise ValueError("roles must be int8 [B, N]")
    if tuple(quota.shape) != (B, R) or quota.dtype != torch.int32:
        raise ValueError("quota must be int32 [B, R]")
    if hist.numel() * 4 < role_hist_size(L, B, Hkv, N, R) or hist.dtype != torch.int32:
        raise ValueError("hist must be int32 with role_hist_size / 4 words")
    if idx_out is None:
        idx_out = torch.full((L, B, Hkv, max(k_cap, 0)), -1, dtype=torch.int32, device=score.device)
    if count_out is None:
        count_out = torch.empty((L, B, Hkv), dtype=torch.int32, device=score.device)
    ws, wsb = _workspace(lambda: topk_workspace_size(L, B, Hkv, N, R), score.device, workspace)
    _check(LIB.kve_topk_select_hist(_dev(score, "score"), _dev(roles, "roles"), _dev(quota, "quota"),
                                    _dev(hist, "hist"), L, B, Hkv, N, int(W), int(R), int(k_cap),
                                    _dev(idx_out, "idx_out"), _dev(count_out, "count_out"),
                                    _ptr(ws), wsb, _stream(stream)))
    return idx_out, count_out


def kv_compact(k, v, idx, count, k_out=None, v_out=None, stream=None):
    """Compacted K (and V) [L, B, Hkv, k_cap, d]."""
    torch = _torch()
    L, B, Hkv, N, d = k.shape
    k_cap = idx.shape[-1]
    if tuple(idx.shape[:3]) != (L, B, Hkv) or idx.dtype != torch.int32:
        raise ValueError("idx must be int32 [L, B, Hkv, k_cap]")
    if tuple(count.shape) != (L, B, Hkv) or count.dtype != torch.int32:
        raise ValueError("count must be int32 [L, B, Hkv]")
    if v is not None and (v.shape != k.shape or v.dtype != k.dtype):
        raise ValueError("v must match k")
    if k_out is None:
        k_out = torch.zeros((L, B, Hkv, k_cap, d), dtype=k.dtype, device=k.device)
    if v is not None and v_out is None:
        v_out = torch.zeros_like(k_out)
    if not (k.is_contiguous() and (v is None or v.is_contiguous())):
        return kv_compact_strided(k, v, idx, count, k_out, v_out, stream)
    _check(LIB.kve_kv_compact(_dev(k, "k"), None if v is None else _dev(v, "v"), _dtype_code(k),
                              _dev(idx, "idx"), _dev(count, "count"), L, B, Hkv, N, d, int(k_cap),
                              _dev(k_out, "k_out"), None if v is None else _dev(v_out, "v_out"),
                              _stream(stream)))
    return k_out, v_out


def kv_compact_strided(k, v, idx, count, k_out=None, v_out=None, stream=None):
    """kv_compact reading k and v [L, B, Hkv, N, d] as views (any strides with
    a contiguous last dimension); outputs dense.  See kve_kv_compact_strided."""
    torch = _torch()
    L, B, Hkv, N, d = k.shape
    k_cap = idx.shape[-1]
    if tuple(idx.shape[:3]) != (L, B, Hkv) or idx.dtype != torch.int32:
        raise ValueError("idx must be int32 [L, B, Hkv, k_cap]")
    if tuple(count.shape) != (L, B, Hkv) or count.dtype != torch.int32:
        raise ValueError("count must be int32 [L, B, Hkv]")
    if v is not None and (v.shape != k.shape or v.dtype != k.dtype):
        raise ValueError("v must match k")
    if k_out is None:
        k_out = torch.zeros((L, B, Hkv, k_cap, d), dtype=k.dtype, device=k.device)
    if v is not None and v_out is None:
        v_out = torch.zeros_like(k_out)
    kp, ks = _view(k, "k")
    vp, vs = (None, None) if v is None else _view(v, "v")
    _check(LIB.kve_kv_compact_strided(kp, ctypes.byref(ks), vp, None if v is None else ctypes.byref(vs),
                                      _dtype_code(k), _dev(idx, "idx"), _dev(count, "count"), L, B, Hkv, N,
                                      d, int(k_cap), _dev(k_out, "k_out"),
                                      None if v is None else _dev(v_out, "v_out"), _stream(stream)))
    return k_out, v_out


def decode_workspace_size(L, B, Hq, Hkv, k_cap, d) -> int:
    return int(LIB.kve_decode_workspace_size(L, B, Hq, Hkv, k_cap, d))


def decode_attention(q, k_c, v_c, count, scale: float = 0.0, out=None, workspace=None, stream=None):
    """Decode over the first count rows of a compacted cache: q [L, B, Hq, d],
    k_c, v_c [L, B, Hkv, k_cap, d], count int32 [L, B, Hkv] -> float32 [L, B, Hq, d]."""
    torch = _torch()
    L, B, Hq, d = q.shape
    Lk, Bk, Hkv, k_cap, dk = k_c.shape
    if (L, B, d) != (Lk, Bk, dk) or v_c.shape != k_c.shape or q.dtype != k_c.dtype or v_c.dtype != k_c.dtype:
        raise ValueError("q, k_c and v_c disagree in L, B, d, shape or dtype")
    if tuple(count.shape) != (L, B, Hkv) or count.dtype != torch.int32:
        raise ValueError("count must be int32 [L, B, Hkv]")
    if out is None:
        out = torch.empty((L, B, Hq, d), dtype=torch.float32, device=k_c.device)
    ws, wsb = _workspace(lambda: decode_workspace_size(L, B, Hq, Hkv, k_cap, d), k_c.device, workspace)
    _check(LIB.kve_decode_attention(_dev(q, "q"), _dev(k_c, "k_c"), _dev(v_c, "v_c"), _dev(count, "count"),
                                    _dtype_code(k_c), L, B, Hq, Hkv, k_cap, d, float(scale),
                                    _dev(out, "out"), _ptr(ws), wsb, _stream(stream)))
    return out


def role_probe(ids, weight, bias, out=None, stream=None):
    """Probe role labels int8 [B, N] from token ids int32 [B, N], weight
    float32 [5, V, R] and bias float32 [R] (all device tensors)."""
    torch = _torch()
    if ids.dim() != 2 or ids.dtype != torch.int32:
        raise ValueError("ids must be int32 [B, N]")
    if weight.dim() != 3 or weight.shape[0] != 5 or weight.dtype != torch.float32:
        raise ValueError("weight must be float32 [5, V, R]")
    B, N = ids.shape
    V, R = weight.shape[1], weight.shape[2]
    if tuple(bias.shape) != (R,) or bias.dtype != torch.float32:
        raise ValueError("bias must be float32 [R]")
    if out is None:
        out = torch.empty((B, N), dtype=torch.int8, device=ids.device)
    _check(LIB.kve_role_probe(_dev(ids, "ids"), B, N, _dev(weight, "weight"), _dev(bias, "bias"), V, R,
                              _dev(out, "out"), _stream(stream)))
    return out


def read_probe(buf, nontemporal: bool = True, blocks: int = 4096, sink=None, stream=None):
    """Stream every byte of the device tensor `buf` once (kve_read_probe);
    returns the sink tensor (one float per workgroup)."""
    torch = _torch()
    nbytes = buf.numel() * buf.element_size()
    if sink is None:
        sink = torch.empty(blocks, dtype=torch.float32, device=buf.device)
    _check(LIB.kve_read_probe(_dev(buf, "buf"), nbytes, int(bool(nontemporal)), _dev(sink, "sink"), int(blocks),
                              _stream(stream)))
    return sink
