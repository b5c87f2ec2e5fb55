"""Pins of the oracle's decode through the keep-set (Algorithm 1, last step;
§3 "Setup"; §6 "Systems cost").

The compacted form (attention over K[idx], V[idx]) must equal the masked form
over the full cache that the paper's harness uses; both are pinned against
scipy's softmax, pure-Python loops and closed forms.
"""

import math

import numpy as np
import pytest
from scipy.special import softmax

import oracle as O
from oracle import brute


def _rand(r, *shape):
    return r.standard_normal(shape)


def test_full_keep_set_is_softmax_attention():
    r = np.random.default_rng(400)
    for G, n, d in [(1, 1, 8), (4, 37, 16), (8, 200, 64), (3, 5, 128)]:
        q, k, v = _rand(r, G, d), _rand(r, n, d), _rand(r, n, d)
        ref = softmax(q @ k.T / math.sqrt(d), axis=1) @ v
        assert np.allclose(O.decode_attention(q, k, v), ref, rtol=1e-12, atol=1e-12)
        assert np.allclose(O.masked_decode_attention(q, k, v, np.arange(n)), ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", range(10))
def test_compacted_equals_masked_full_cache(seed):
    r = np.random.default_rng(410 + seed)
    G, N, d = int(r.integers(1, 9)), int(r.integers(1, 300)), int(r.choice([16, 64, 128]))
    q, k, v = 3 * _rand(r, G, d), _rand(r, N, d), _rand(r, N, d)
    keep = np.sort(r.choice(N, int(r.integers(1, N + 1)), replace=False))
    compact = O.decode_attention(q, k[keep], v[keep])
    masked = O.masked_decode_attention(q, k, v, keep)
    assert np.allclose(compact, masked, rtol=1e-12, atol=1e-13)
    # the kept rows' order does not matter
    perm = r.permutation(len(keep))
    assert np.allclose(O.decode_attention(q, k[keep[perm]], v[keep[perm]]), compact, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("seed", range(6))
def test_decode_equals_loops(seed):
    r = np.random.default_rng(430 + seed)
    G, N, d = int(r.integers(1, 5)), int(r.integers(1, 20)), int(r.choice([2, 4, 8]))
    q, k, v = _rand(r, G, d), _rand(r, N, d), _rand(r, N, d)
    keep = sorted(r.choice(N, int(r.integers(0, N + 1)), replace=False).tolist())
    ref = np.array(brute.decode_loops(q.tolist(), k.tolist(), v.tolist(), keep))
    assert np.allclose(O.masked_decode_attention(q, k, v, keep) if keep else
                       O.decode_attention(q, k[:0], v[:0]), ref, rtol=1e-12, atol=1e-12)
    assert np.allclose(O.decode_attention(q, k[keep], v[keep]), ref, rtol=1e-12, atol=1e-12)


def test_closed_forms():
    r = np.random.default_rng(440)
    d = 16
    q, k, v = _rand(r, 3, d), _rand(r, 2, d), _rand(r, 2, d)
    # one row: the output is that row
    assert np.allclose(O.decode_attention(q, k[:1], v[:1]), np.repeat(v[:1], 3, axis=0), rtol=0, atol=1e-15)
    # equal keys: the mean of the value rows
    kk = np.repeat(k[:1], 5, axis=0)
    vv = _rand(r, 5, d)
    assert np.allclose(O.decode_attention(q, kk, vv), np.repeat(vv.mean(0, keepdims=True), 3, axis=0))
    # two keys: a logistic weight on the scaled logit difference (sign, scale, operand order)
    s = 0.37
    w = 1.0 / (1.0 + np.exp(-s * (q @ (k[0] - k[1]))))
    ref = w[:, None] * v[0] + (1 - w[:, None]) * v[1]
    assert np.allclose(O.decode_attention(q, k, v, scale=s), ref, rtol=1e-13, atol=1e-14)
    # empty cache: zeros; huge logits stay finite
    assert not O.decode_attention(q, k[:0], v[:0]).any()
    out = O.decode_attention(1e4 * q, k, v)
    assert np.all(np.isfinite(out))


def test_batch_grouping_and_counts():
    r = np.random.default_rng(450)
    L, B, Hq, Hkv, k_cap, d = 2, 2, 8, 2, 12, 8
    G = Hq // Hkv
    q = _rand(r, L, B, Hq, d)
    kc, vc = _rand(r, L, B, Hkv, k_cap, d), _rand(r, L, B, Hkv, k_cap, d)
    count = np.array([[[12, 5], [0, 20]], [[1, -3], [7, 12]]])
    out = O.decode_attention_batch(q, kc, vc, count)
    for l in range(L):
        for b in range(B):
            for h in range(Hq):
                j = h // G                      # contiguous groups
                n = min(max(count[l, b, j], 0), k_cap)
                ref = brute.decode_loops([q[l, b, h].tolist()], kc[l, b, j].tolist(),
                                         vc[l, b, j].tolist(), range(n))[0]
                assert np.allclose(out[l, b, h], ref, rtol=1e-12, atol=1e-12)
