"""Parity of the library's compatibility gate (host code behind the C ABI)
with the oracle: CIEDE2000 within 1e-9, descriptors and gate decisions
exact, the Clopper-Pearson bound within 1e-12 and the paper's 4.50 %.
No GPU is used: these entry points run on host memory."""
import json
import os

import numpy as np
import pytest

import oracle
import paper_2609_32420_amd as P
from paper_2609_32420_amd import build as B


@pytest.fixture(scope="module", autouse=True)
def _lib():
    if not os.path.exists(P.LIB_PATH):
        B.build()
    P.lib()


def test_ciede2000_matches_oracle_random_and_edges():
    rng = np.random.default_rng(1)
    n = 4000
    lab1 = np.stack([rng.uniform(0, 100, n), rng.uniform(-110, 110, n), rng.uniform(-110, 110, n)], -1)
    lab2 = lab1 + rng.normal(0, 8, (n, 3)) * (rng.random((n, 1)) < 0.7) + rng.normal(0, 40, (n, 3)) * (
        rng.random((n, 1)) < 0.3)
    # achromatic, opposite hues, hue wrap, identical
    lab1[:4] = [[50, 0, 0], [60, 20, 0], [60, 30 * np.cos(np.radians(359)), 30 * np.sin(np.radians(359))],
                [40, 10, 10]]
    lab2[:4] = [[70, 0, 0], [60, -20, 0], [60, 30 * np.cos(np.radians(1)), 30 * np.sin(np.radians(1))],
                [40, 10, 10]]
    got = P.ciede2000(lab1, lab2)
    want = oracle.ciede2000(lab1, lab2)
    assert np.abs(got - want).max() <= 1e-9
    assert got[3] == 0.0


@pytest.mark.parametrize("hw,res,seed", [((20, 30), 32, 0), ((45, 80), 32, 1), ((7, 3), 16, 2), ((64, 64), 8, 3)])
def test_shape_descriptor_matches_oracle(hw, res, seed):
    rng = np.random.default_rng(seed)
    m = np.zeros(hw, np.uint8)
    y0, x0 = rng.integers(0, hw[0] // 2), rng.integers(0, hw[1] // 2)
    m[y0:y0 + max(1, hw[0] // 3), x0:x0 + max(1, hw[1] // 2)] = 1
    m[rng.random(hw) < 0.05] = 1
    area, shape = P.shape_descriptor(m, res)
    assert area == oracle.support_area(m)
    np.testing.assert_array_equal(shape, oracle.normalized_shape(m, res))
    a0, s0 = P.shape_descriptor(np.zeros(hw, np.uint8), res)
    assert a0 == 0.0 and not s0.any()


def test_object_discrepancy_and_gate_match_oracle():
    rng = np.random.default_rng(4)
    ev = rng.random((2, 30, 40)) < 0.1
    (aq, sq), (aj, sj) = P.shape_descriptor(ev[0]), P.shape_descriptor(ev[1])
    lq, lj = np.array([55.0, 12.0, -30.0]), np.array([52.0, 20.0, -24.0])
    d = P.object_discrepancy(aq, aj, sq, sj, lq, lj)
    want = [oracle.d_size(aq, aj), oracle.d_shape(oracle.normalized_shape(ev[0]), oracle.normalized_shape(ev[1])),
            float(oracle.ciede2000(lq, lj))]
    assert d[0] == pytest.approx(want[0], abs=1e-15) and d[1] == want[1] and abs(d[2] - want[2]) < 1e-9
    assert P.object_discrepancy(0.0, 0.0, sq, sq, lq, lq)[0] == 0.0
    assert np.isinf(P.object_discrepancy(0.0, 0.1, sq, sq, lq, lq)[0])
    tau = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "gate_worked.json")))["tau_star"]
    for trial in range(200):
        dc = rng.uniform(0, 1, (rng.integers(0, 6), 4)) * np.array([3.0, 4.0, 1.2, 12.0])
        assert P.compat_gate(dc.reshape(-1, 4), tau) == oracle.first_compatible(dc.reshape(-1, 4), tau)
    assert P.compat_gate(np.array([tau]), tau) == 0  # on the thresholds: accepted


@pytest.mark.parametrize("u,n,alpha", [(0, 50, 0.10), (0, 1, 0.5), (1, 50, 0.1), (3, 70, 0.05), (10, 20, 0.2),
                                       (0, 1000, 0.01), (40, 1000, 0.1), (5, 5, 0.1)])
def test_clopper_pearson_matches_oracle(u, n, alpha):
    assert abs(P.clopper_pearson_upper(u, n, alpha) - oracle.clopper_pearson_upper(u, n, alpha)) < 1e-12


def test_paper_certification_bound():
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "gate_worked.json")))
    u = P.clopper_pearson_upper(g["unsafe"], g["accepted"], g["alpha"])
    assert round(100 * u, 2) == g["upper_bound_percent"] and u <= g["delta"]


def test_gate_entry_points_reject():
    L = P.lib()
    import ctypes
    p = ctypes.c_void_p(0x1000)
    assert L.carnator_ciede2000(None, p, 1, p) == -1
    assert L.carnator_ciede2000(p, p, -1, p) == -2
    assert L.carnator_shape_descriptor(p, 0, 5, 8, p, p) == -2
    assert L.carnator_compat_gate(p, 1, 0, p, p) == -2
    out = ctypes.c_double()
    assert L.carnator_clopper_pearson_upper(3, 2, 0.1, ctypes.byref(out)) == -2
    assert L.carnator_clopper_pearson_upper(0, 10, 1.0, ctypes.byref(out)) == -2
    assert L.carnator_clopper_pearson_upper(0, 10, 0.1, None) == -1
