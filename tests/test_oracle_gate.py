"""Pins of the compatibility-gate oracle (CPU): the paper's certification
numbers, closed forms of CIEDE2000 and of the Clopper-Pearson bound, and
brute-force descriptor loops."""
import json
import math
import os

import numpy as np
import pytest
from scipy import stats

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "gate_worked.json")


def test_paper_certification_numbers():
    g = json.load(open(GOLDEN))
    u = oracle.clopper_pearson_upper(g["unsafe"], g["accepted"], g["alpha"])
    assert round(100 * u, 2) == g["upper_bound_percent"]
    assert u <= g["delta"]
    # u = 0: the bound solves (1 - p)^n = alpha
    assert abs(u - (1 - g["alpha"] ** (1 / g["accepted"]))) < 1e-12
    assert round(100 * g["accepted"] / g["pairs"], 2) == g["coverage_percent"]


@pytest.mark.parametrize("u,n,alpha", [(0, 10, 0.1), (1, 50, 0.1), (3, 70, 0.05), (10, 20, 0.2), (5, 5, 0.1)])
def test_clopper_pearson_definition(u, n, alpha):
    # the bound p solves P(X <= u | n, p) = alpha (binomial tail), and u = n gives 1
    p = oracle.clopper_pearson_upper(u, n, alpha)
    if u == n:
        assert p == 1.0
    else:
        assert abs(stats.binom.cdf(u, n, p) - alpha) < 1e-9
        assert abs(sum(math.comb(n, i) * p ** i * (1 - p) ** (n - i) for i in range(u + 1)) - alpha) < 1e-9


def test_ciede2000_identities_and_symmetry():
    rng = np.random.default_rng(0)
    lab = np.stack([rng.uniform(0, 100, 500), rng.uniform(-100, 100, 500), rng.uniform(-100, 100, 500)], -1)
    lab2 = np.stack([rng.uniform(0, 100, 500), rng.uniform(-100, 100, 500), rng.uniform(-100, 100, 500)], -1)
    np.testing.assert_array_equal(oracle.ciede2000(lab, lab), 0.0)
    np.testing.assert_allclose(oracle.ciede2000(lab, lab2), oracle.ciede2000(lab2, lab), rtol=1e-12)
    assert (oracle.ciede2000(lab, lab2) >= 0).all()


@pytest.mark.parametrize("L1,L2", [(50, 60), (20, 80), (0, 100), (73.2, 71.9)])
def test_ciede2000_pure_lightness_closed_form(L1, L2):
    # a = b = 0: only the lightness term, |dL| / S_L with S_L at the mean L
    Lb = 0.5 * (L1 + L2)
    SL = 1 + 0.015 * (Lb - 50) ** 2 / math.sqrt(20 + (Lb - 50) ** 2)
    got = oracle.ciede2000([L1, 0, 0], [L2, 0, 0])
    assert abs(got - abs(L2 - L1) / SL) < 1e-12


@pytest.mark.parametrize("a1,a2", [(10.0, 20.0), (3.0, 40.0), (25.0, 26.0)])
def test_ciede2000_pure_chroma_on_the_a_axis(a1, a2):
    # same L, b = 0, a > 0: hue 0 for both, so only the chroma term remains:
    # a' = (1 + G) a, dC' = a2' - a1', divided by S_C = 1 + 0.045 mean C'
    Cb = 0.5 * (a1 + a2)
    G = 0.5 * (1 - math.sqrt(Cb ** 7 / (Cb ** 7 + 25 ** 7)))
    c1, c2 = (1 + G) * a1, (1 + G) * a2
    SC = 1 + 0.045 * 0.5 * (c1 + c2)
    got = oracle.ciede2000([50, a1, 0], [50, a2, 0])
    assert abs(got - abs(c2 - c1) / SC) < 1e-12


def test_ciede2000_hue_wrap_is_continuous():
    # two colours either side of the +a axis (hue 359 and 1 degree) are close,
    # as close as two colours at hue 1 and 3 degrees of the same chroma
    def lab(h):
        return [60, 30 * math.cos(math.radians(h)), 30 * math.sin(math.radians(h))]
    across = oracle.ciede2000(lab(359), lab(1))
    assert across < 1.5
    assert abs(across - oracle.ciede2000(lab(1), lab(3))) < 0.3


def test_area_and_normalized_shape_brute_force():
    m = np.zeros((20, 30), np.uint8)
    m[5:9, 10:22] = 1
    m[6, 3] = 1
    assert oracle.support_area(m) == m.sum() / 600
    s = oracle.normalized_shape(m, 8)
    ys, xs = np.nonzero(m)
    crop = m[ys.min():ys.max() + 1, xs.min():xs.max() + 1]
    h, w = crop.shape
    for y in range(8):
        for x in range(8):
            assert s[y, x] == crop[int((y + 0.5) * h / 8), int((x + 0.5) * w / 8)]
    # translation and integer scaling of a box leave the normalised shape unchanged
    a = np.zeros((40, 40), np.uint8)
    a[2:10, 5:13] = 1
    b = np.zeros((40, 40), np.uint8)
    b[20:36, 3:19] = 1
    np.testing.assert_array_equal(oracle.normalized_shape(a), oracle.normalized_shape(b))
    assert oracle.d_shape(oracle.normalized_shape(a), oracle.normalized_shape(b)) == 0.0
    assert not oracle.normalized_shape(np.zeros((5, 5))).any()


def test_discrepancies_and_gate():
    assert oracle.d_size(0.2, 0.1) == pytest.approx(math.log(2))
    assert oracle.d_size(0.1, 0.2) == pytest.approx(math.log(2))
    assert oracle.d_size(0, 0) == 0 and math.isinf(oracle.d_size(0, 0.3))
    a = np.zeros((4, 4), np.uint8)
    a[:2] = 1
    b = np.zeros((4, 4), np.uint8)
    b[:, :2] = 1
    assert oracle.d_shape(a, b) == pytest.approx(1 - 2 * 4 / 16)
    assert oracle.d_shape(a, a) == 0 and oracle.d_shape(a, 1 - a) == 1
    tau = json.load(open(GOLDEN))["tau_star"]
    assert oracle.gate([1.62, 2.17, 1.0, 7.58], tau)  # on the thresholds: accepted
    assert not oracle.gate([1.63, 0, 0, 0], tau)
    d = [[0, 0, 0, 8.0], [2.0, 0, 0, 0], [0.5, 1.0, 0.4, 3.0], [0, 0, 0, 0]]
    assert oracle.first_compatible(d, tau) == 2
    assert oracle.first_compatible(d[:2], tau) == -1


# An independent implementation of CIEDE2000: LittleCMS's cmsCIE2000DeltaE
# (its documented C API, weights kL, kC, kH), called through ctypes on the
# system's liblcms2.  It pins the hue weighting (T, delta-theta, R_T, S_H)
# that no closed form above reaches: random pairs over the whole gamut, close
# pairs, near-achromatic pairs, and a grid of hue pairs around the wrap at 0
# and 360 degrees, R_T's peak at 275 degrees and opposite hues, with zero and
# unequal chromas.
def _lcms_de2000():
    import ctypes
    import ctypes.util
    name = ctypes.util.find_library("lcms2") or "liblcms2.so.2"
    try:
        lib = ctypes.CDLL(name)
    except OSError:
        return None

    class Lab(ctypes.Structure):
        _fields_ = [("L", ctypes.c_double), ("a", ctypes.c_double), ("b", ctypes.c_double)]

    f = lib.cmsCIE2000DeltaE
    f.restype = ctypes.c_double
    f.argtypes = [ctypes.POINTER(Lab), ctypes.POINTER(Lab), ctypes.c_double, ctypes.c_double, ctypes.c_double]
    return lambda p, q: f(ctypes.byref(Lab(*map(float, p))), ctypes.byref(Lab(*map(float, q))), 1.0, 1.0, 1.0)


def test_ciede2000_against_littlecms():
    de = _lcms_de2000()
    if de is None:
        pytest.skip("liblcms2 is not installed")
    rng = np.random.default_rng(3)
    pairs = []
    for it in range(3000):
        p = rng.uniform([0, -128, -128], [100, 128, 128], size=(2, 3))
        if it % 3 == 1:
            p[1] = p[0] + rng.normal(0, 3, 3)  # close pairs
        if it % 3 == 2:
            p[:, 1:] *= rng.uniform(0, 0.05)  # near-achromatic
        pairs.append((p[0], p[1]))
    for L1, L2 in [(50, 50), (50, 60), (20, 90)]:
        for h1 in [0, 10, 90, 170, 180, 190, 270, 275, 300, 350, 359.9]:
            for h2 in [0, 5, 95, 185, 200, 275, 355, 359]:
                for C1, C2 in [(30, 30), (0, 40), (40, 0), (0, 0), (5, 80)]:
                    r1, r2 = math.radians(h1), math.radians(h2)
                    pairs.append((np.array([L1, C1 * math.cos(r1), C1 * math.sin(r1)]),
                                  np.array([L2, C2 * math.cos(r2), C2 * math.sin(r2)])))
    got = oracle.ciede2000(np.stack([p for p, _ in pairs]), np.stack([q for _, q in pairs]))
    want = np.array([de(p, q) for p, q in pairs])
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-9)
