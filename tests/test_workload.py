"""The synthetic input recipe: role mix, determinism and the sink strength
(checked with the oracle's per-role mass)."""

import numpy as np
import pytest

import oracle as O
import workload as WL


@pytest.mark.parametrize("name", list(WL.WORKLOADS))
def test_role_mix_within_two_points(name):
    """Within 2 points of the target mix (3 points at N < 4096, where a few
    hundred runs leave that much sampling noise)."""
    wl = WL.get_workload(name).with_(B=1)
    roles = WL.make_roles(wl)
    mix = np.bincount(roles[0], minlength=4) / wl.N
    tol = 0.02 if wl.N >= 4096 else 0.03
    assert np.all(np.abs(mix - np.array(wl.mix)) <= tol), mix
    assert roles[0, 0] == WL.SINK                      # BOS sits in the sink
    q_len = max(wl.W, 16)
    assert np.all(roles[0, wl.N - q_len:] == WL.OTHER)  # trailing question


def test_roles_are_deterministic_and_per_sample():
    wl = WL.get_workload("stack32k").with_(N=4096)
    a, b = WL.make_roles(wl), WL.make_roles(wl)
    assert np.array_equal(a, b)
    assert not np.array_equal(a[0], a[1])


def test_layer_subset_reproduces_bits():
    torch = pytest.importorskip("torch")
    wl = WL.get_workload("layer8k").with_(L=3, N=512, Hq=8, Hkv=2)
    full = WL.make_inputs(wl)
    part = WL.make_inputs(wl, layers=[2])
    assert torch.equal(full["k"][2], part["k"][0])
    assert torch.equal(full["q"][2], part["q"][0])
    assert torch.equal(full["v"][2], part["v"][0])


def _sink_ratio(wl):
    inp = WL.make_inputs(wl, with_v=False)
    roles = inp["roles"][0]
    P = wl.N - wl.W
    q = inp["q"][0, 0, 0:wl.G].double().numpy()
    k = inp["k"][0, 0, 0].double().numpy()
    s = O.h2o_mass(q, k) if wl.scorer == "h2o" else O.snapkv_mass(q, k)
    sink = s[:P][roles[:P] == WL.SINK].mean()
    content = s[:P][roles[:P] != WL.SINK].mean()
    return sink / content


@pytest.mark.parametrize("name,overrides", [
    ("tiny", {}),
    ("layer8k", {"Hq": 4, "Hkv": 1}),
    ("h2o16k", {"N": 2048, "Hq": 4, "Hkv": 1}),
])
def test_sinks_draw_10_to_30x_content_mass(name, overrides):
    wl = WL.get_workload(name).with_(**overrides)
    rho = _sink_ratio(wl)
    assert 10.0 <= rho <= 30.0, rho
