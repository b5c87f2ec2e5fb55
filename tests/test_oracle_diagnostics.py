"""Pins of the per-role diagnostics against the figures the paper prints (§1, §3)."""

import os

import numpy as np

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load():
    mass, checks = {}, {}
    with open(os.path.join(GOLDEN, "paper_role_mass.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if not line:
                continue
            t = line.split()
            if len(t) == 2:
                mass[t[0]] = float(t[1])
            else:
                checks[t[0]] = (float(t[1]), float(t[2]))
    return mass, checks


def test_paper_snr_and_ratios():
    mass, checks = _load()
    snr = O.retained_snr_db(mass["VALUE"], mass["DELIM"])
    want, tol = checks["snr_value_over_delim_db"]
    assert abs(snr - want) <= tol
    assert abs(snr - (-16.08)) < 0.01
    want, tol = checks["ratio_delim_over_value"]
    assert abs(mass["DELIM"] / mass["VALUE"] - want) <= tol
    want, tol = checks["ratio_delim_over_key"]
    assert abs(mass["DELIM"] / mass["KEY"] - want) <= tol
    assert abs(mass["VALUE"] / mass["DELIM"] - 0.025) < 0.001


def test_per_role_mean_mass_and_retention_by_hand():
    s = np.array([4.0, 1.0, 2.0, 0.5, 8.0, 3.0])
    roles = np.array([0, 1, 1, 2, 0, 3], dtype=np.int8)
    m = O.per_role_mean_mass(s, roles, 5)
    np.testing.assert_allclose(m[:4], [6.0, 1.5, 0.5, 3.0])
    assert np.isnan(m[4])
    m = O.per_role_mean_mass(s, roles, 4, upto=4)
    np.testing.assert_allclose(m[:3], [4.0, 1.5, 0.5])
    rr = O.retention_rate(np.array([0, 2, 5]), roles, 4)
    np.testing.assert_allclose(rr, [0.5, 0.5, 0.0, 1.0])
