"""Pins of the region-restricted oracle (CPU): library routines, closed forms,
hand-worked cases and brute-force loops that its functions must reproduce."""
import numpy as np
import pytest
from scipy import ndimage

import oracle


def _blobs(shape, p, seed):
    rng = np.random.default_rng(seed)
    return (rng.random(shape) < p).astype(np.uint8)


@pytest.mark.parametrize("r", [0, 1, 2, 3, 5])
def test_dilation_matches_scipy_square_structure(r):
    e = _blobs((2, 3, 13, 17), 0.03, r)
    got = oracle.dilate_frames(e, r)
    for idx in np.ndindex(e.shape[:2]):
        want = ndimage.binary_dilation(e[idx] != 0, structure=np.ones((2 * r + 1, 2 * r + 1), bool))
        np.testing.assert_array_equal(got[idx], want)


def test_chebyshev_distance_matches_scipy_chessboard_transform():
    e = _blobs((2, 4, 19, 23), 0.02, 7)
    e[0, 1] = 0  # a frame without evidence: +inf
    d = oracle.chebyshev_distance(e)
    assert np.isinf(d[0, 1]).all()
    for idx in np.ndindex(e.shape[:2]):
        if not e[idx].any():
            continue
        want = ndimage.distance_transform_cdt(e[idx] == 0, metric="chessboard")
        np.testing.assert_array_equal(d[idx], want)


def test_dilations_compose_to_the_distance_ball():
    # square(2) then square(3) is square(5), also at the frame border
    e = _blobs((1, 3, 20, 20), 0.01, 3)
    e[0, 0, 0, 0] = 1
    two_step = oracle.dilate_frames(oracle.dilate_frames(e, 2), 3)
    np.testing.assert_array_equal(two_step, oracle.dilate_frames(e, 5))
    np.testing.assert_array_equal(two_step, oracle.chebyshev_distance(e) <= 5)


def test_smoothstep_closed_forms():
    assert oracle.smoothstep(0.0) == 0.0 and oracle.smoothstep(1.0) == 1.0
    assert oracle.smoothstep(0.5) == 0.5
    assert oracle.smoothstep(0.25) == 0.15625
    t = np.linspace(0, 1, 101)
    np.testing.assert_allclose(oracle.smoothstep(t) + oracle.smoothstep(1 - t), 1.0, atol=1e-15)
    assert (np.diff(oracle.smoothstep(t)) >= 0).all()


def test_single_evidence_token_by_hand():
    # band rings at Chebyshev distance 1 and 2; the band maximum is 2, so ring 1
    # has W = 1 - s(1/2) = 1/2 and ring 2 has W = 1 - s(1) = 0
    e = np.zeros((1, 1, 15, 15), np.uint8)
    e[0, 0, 7, 7] = 1
    code, w = oracle.regions(e)
    yy, xx = np.meshgrid(np.arange(15), np.arange(15), indexing="ij")
    cheb = np.maximum(abs(yy - 7), abs(xx - 7))
    want_code = np.select([cheb == 0, cheb <= 2, cheb <= 5], [3, 2, 1], 0)
    np.testing.assert_array_equal(code[0, 0], want_code)
    want_w = np.select([cheb == 0, cheb == 1], [1.0, 0.5], 0.0)
    np.testing.assert_array_equal(w[0, 0], want_w)


def test_band_maximum_is_taken_over_all_frames():
    # frame 0: evidence everywhere but a one-token border -> its band is at
    # distance 1 only; frame 1: one token -> distances 1 and 2.  Together the
    # maximum is 2 and frame 0's border gets W = 1/2; alone it would be 0.
    e = np.zeros((1, 2, 9, 9), np.uint8)
    e[0, 0, 1:8, 1:8] = 1
    e[0, 1, 4, 4] = 1
    code, w = oracle.regions(e)
    border = np.ones((9, 9), bool)
    border[1:8, 1:8] = False
    assert (code[0, 0][border] == 2).all()
    np.testing.assert_array_equal(w[0, 0][border], 0.5)
    _, w0 = oracle.regions(e[:, :1])
    np.testing.assert_array_equal(w0[0, 0][border], 0.0)


def test_regions_nest_and_weight_bounds():
    e = _blobs((2, 5, 16, 20), 0.02, 11)
    code, w = oracle.regions(e, 2, 3)
    act = oracle.dilate_frames(e, 2)
    ctx = oracle.dilate_frames(act, 3)
    np.testing.assert_array_equal(code == 3, e != 0)
    np.testing.assert_array_equal(code >= 2, act)
    np.testing.assert_array_equal(code >= 1, ctx)
    assert ((w >= 0) & (w <= 1)).all()
    np.testing.assert_array_equal(w == 1.0, e != 0)
    assert (w[code <= 1] == 0).all()


def test_latent_fusion_end_points_and_patch_loop():
    rng = np.random.default_rng(5)
    B, C, T, H, W = 1, 3, 2, 4, 6
    zt = rng.normal(size=(B, C, T, H, W))
    zh = rng.normal(size=(B, C, T, H, W))
    np.testing.assert_array_equal(oracle.latent_fusion(zt, zh, np.ones((B, T, H, W))), zt)
    np.testing.assert_array_equal(oracle.latent_fusion(zt, zh, np.zeros((B, T, H, W))), zh)
    wt = rng.random((B, T, H // 2, W // 3))
    got = oracle.latent_fusion(zt, zh, wt, patch=(1, 2, 3))
    for c in range(C):
        for t in range(T):
            for y in range(H):
                for x in range(W):
                    a = wt[0, t, y // 2, x // 3]
                    assert got[0, c, t, y, x] == a * zt[0, c, t, y, x] + (1 - a) * zh[0, c, t, y, x]


def test_block_flags_token_loop():
    rng = np.random.default_rng(9)
    code = rng.integers(0, 4, size=(2, 3, 4, 5)).astype(np.uint8)
    code[1] = np.where(code[1] >= 2, 1, code[1])  # batch 1: no active video token
    n_text, bs = 7, 8
    act, ctx = oracle.region_block_flags(code, n_text, bs)
    n = n_text + 60
    assert act.shape == (2, -(-n // bs))
    for b in range(2):
        for i in range(act.shape[1]):
            toks = range(i * bs, min((i + 1) * bs, n))
            a = any(t < n_text or code[b].reshape(-1)[t - n_text] >= 2 for t in toks)
            c = any(t < n_text or code[b].reshape(-1)[t - n_text] >= 1 for t in toks)
            assert act[b, i] == a and ctx[b, i] == c


def test_restriction_identities():
    m = _blobs((2, 3, 9, 9), 0.4, 1)
    ones = np.ones((2, 9), np.uint8)
    zeros = np.zeros((2, 9), np.uint8)
    np.testing.assert_array_equal(oracle.restrict_mask(m, ones, ones), m)
    assert not oracle.restrict_mask(m, zeros, ones).any()
    assert not oracle.restrict_mask(m, ones, zeros).any()
    # everything active: the plain compaction, every row counted
    rp, ci, od, n = oracle.compact_restricted(m, ones, ones)
    for a, b in zip((rp, ci, od), oracle.compact_mask(m)):
        np.testing.assert_array_equal(a, b)
    assert n == 2 * 3 * 9
    # nothing active: empty lists, rows in order, none counted
    rp, ci, od, n = oracle.compact_restricted(m, zeros, ones)
    assert n == 0 and ci.size == 0 and (rp == 0).all()
    np.testing.assert_array_equal(od, np.arange(2 * 3 * 9))


def test_restricted_order_puts_active_rows_first():
    m = _blobs((1, 2, 6, 6), 0.5, 4)
    act = np.array([[1, 0, 1, 0, 0, 1]], np.uint8)
    ctx = np.array([[1, 1, 0, 1, 1, 1]], np.uint8)
    rp, ci, od, n = oracle.compact_restricted(m, act, ctx)
    lens = np.diff(rp)
    rows_active = [h * 6 + i for h in range(2) for i in range(6) if act[0, i]]
    assert n == len(rows_active) == 6
    assert sorted(od[:n]) == rows_active
    assert all(lens[od[k]] >= lens[od[k + 1]] for k in range(n - 1))
    assert list(od[n:]) == [r for r in range(12) if r not in rows_active]
    assert (lens[od[n:]] == 0).all()
    # no list holds a non-context key block
    assert not np.isin(ci, [2]).any()


def test_restricted_order_brute_force_with_empty_active_rows():
    # active rows of every length, including empty ones, sorted by
    # (-length, row) with plain Python; the inactive rows follow in row order
    rng = np.random.default_rng(12)
    m = (rng.random((2, 3, 7, 7)) < 0.4).astype(np.uint8)
    m[0, 1, 2] = 0  # an active row with nothing kept
    act = np.array([[1, 0, 1, 1, 0, 1, 0], [0, 1, 1, 0, 1, 0, 1]], np.uint8)
    ctx = np.array([[1, 1, 0, 1, 1, 1, 1], [1, 1, 1, 0, 1, 1, 0]], np.uint8)
    rp, ci, od, n = oracle.compact_restricted(m, act, ctx)
    lens = {}
    for b in range(2):
        for h in range(3):
            for i in range(7):
                r = (b * 3 + h) * 7 + i
                lens[r] = sum(1 for j in range(7) if m[b, h, i, j] and act[b, i] and ctx[b, j])
    active = [r for r in range(42) if act[r // 21, r % 7]]
    want = sorted(active, key=lambda r: (-lens[r], r)) + [r for r in range(42) if r not in active]
    assert list(od) == want and n == len(active)
    assert lens[(0 * 3 + 1) * 7 + 2] == 0 and any(lens[r] > 0 for r in active)
    np.testing.assert_array_equal(np.diff(rp), [lens[r] for r in range(42)])
