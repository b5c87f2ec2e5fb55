"""Pins of the oracle's linear role probe (§6 "Deployment: a linear role
probe"): hand-worked logits with weights exact in float32, the centre-token
and neighbour rules, sequence edges, out-of-vocabulary ids, ties, and the
float32 result against a float64 recomputation."""

import numpy as np

import oracle as O


def _tables(V, R, fill=0.0):
    return np.full((5, V, R), fill, dtype=np.float32), np.zeros(R, dtype=np.float32)


def test_hand_worked_example():
    # V = 4 ids, R = 3 roles; small integers are exact in float32
    W, b = _tables(4, 3)
    b[:] = [0.5, 0.0, 0.25]
    W[2, 1] = [0, 2, 0]        # centre id 1 votes role 1
    W[2, 2] = [0, 0, 3]        # centre id 2 votes role 2
    W[0, 3] = [4, 0, 0]        # an id 3 two tokens back votes role 0
    W[4, 3] = [0, 0, 1]        # an id 3 two tokens ahead adds to role 2
    ids = np.array([1, 2, 3, 1, 2])
    # t0: b + W2[1]                 = [0.5, 2, 0.25]   -> 1
    # t1: b + W2[2]                 = [0.5, 0, 3.25]   -> 2
    # t2: b + W2[3]                 = [0.5, 0, 0.25]   -> 0
    # t3: b + W2[1]                 = [0.5, 2, 0.25]   -> 1
    # t4: b + W0[3] + W2[2]         = [4.5, 0, 3.25]   -> 0
    # (t0 also sees W4[ids[2] = 3] = [0, 0, 1]: [0.5, 2, 1.25] -> 1)
    lg = O.probe_logits(ids, W, b)
    assert lg.dtype == np.float32
    assert lg[0].tolist() == [0.5, 2.0, 1.25]
    assert lg[4].tolist() == [4.5, 0.0, 3.25]
    assert O.probe_roles(ids, W, b).tolist() == [1, 2, 0, 1, 0]


def test_centre_token_rule_and_edges():
    r = np.random.default_rng(600)
    V, R = 50, 6
    f = r.integers(0, R, V)
    W, b = _tables(V, R)
    W[2, np.arange(V), f] = 1.0               # only the centre token decides
    ids = r.integers(0, V, (3, 40))
    assert np.array_equal(O.probe_roles(ids, W, b), f[ids].astype(np.int8))
    # a neighbour table shifts the decision; positions outside the sequence add nothing
    W2, b2 = _tables(V, R)
    W2[1, :, 3] = 1.0                         # "a token one step back exists" votes role 3
    lab = O.probe_roles(ids, W2, b2)
    assert np.all(lab[:, 0] == 0) and np.all(lab[:, 1:] == 3)


def test_out_of_vocabulary_ids_and_ties():
    W, b = _tables(5, 4, fill=0.0)
    W[2, 0] = [1, 0, 0, 0]
    ids = np.array([0, -1, 7, 0])
    # ids -1 and 7 contribute nothing: all-zero logits, a tie won by role 0
    assert O.probe_logits(ids, W, b)[1].tolist() == [0, 0, 0, 0]
    assert O.probe_roles(ids, W, b).tolist() == [0, 0, 0, 0]
    b2 = np.array([0, 1, 1, 0], dtype=np.float32)   # tie between roles 1 and 2
    assert O.probe_roles(np.array([3]), W, b2).tolist() == [1]


def test_float32_order_close_to_float64():
    r = np.random.default_rng(610)
    V, R = 1000, 6
    W = (0.1 * r.standard_normal((5, V, R))).astype(np.float32)
    b = (0.1 * r.standard_normal(R)).astype(np.float32)
    ids = r.integers(0, V, 300)
    lg = O.probe_logits(ids, W, b).astype(np.float64)
    ref = np.tile(b.astype(np.float64), (300, 1))
    for j, o in enumerate(O.PROBE_OFFSETS):
        for t in range(300):
            if 0 <= t + o < 300:
                ref[t] += W[j, ids[t + o]].astype(np.float64)
    assert np.allclose(lg, ref, rtol=0, atol=1e-6)
    # invariance: a constant added to every role of a table row changes no label
    W2 = W.copy()
    W2[2] += 0.5
    lab = O.probe_roles(ids, W, b)
    lab2 = O.probe_roles(ids, W2, b)
    same = np.sort(O.probe_logits(ids, W, b), axis=1)
    clear = (same[:, -1] - same[:, -2]) > 1e-5           # away from float32 near-ties
    assert np.array_equal(lab[clear], lab2[clear])
