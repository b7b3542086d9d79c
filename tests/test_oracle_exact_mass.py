"""Pins of the exact-mass oracle (CPU): closed forms, invariants, the
attention oracle with one-hot block values, and a pure-Python loop."""
import math

import numpy as np
import pytest

import oracle


def _qk(B, H, N, d, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    return rng.normal(0, scale, (B, H, N, d)), rng.normal(0, scale, (B, H, N, d))


@pytest.mark.parametrize("N,bs", [(64, 16), (70, 16), (5, 8), (130, 32)])
def test_rows_sum_to_one(N, bs):
    q, k = _qk(2, 2, N, 8, N)
    M = oracle.exact_block_mass(q, k, bs)
    np.testing.assert_allclose(M.sum(axis=-1), 1.0, rtol=0, atol=1e-12)
    assert (M >= 0).all()


def test_uniform_attention_gives_block_sizes():
    # q = 0 (or all keys equal): every key weighs 1/N, so M_ij = n_j / N
    N, bs = 70, 16
    q = np.zeros((1, 1, N, 4))
    k = np.random.default_rng(0).normal(size=(1, 1, N, 4))
    M = oracle.exact_block_mass(q, k, bs)
    n = np.array([16, 16, 16, 16, 6], float)
    np.testing.assert_allclose(M[0, 0], np.broadcast_to(n / N, (5, 5)), atol=1e-15)
    q2 = np.random.default_rng(1).normal(size=(1, 1, N, 4))
    k2 = np.ones((1, 1, N, 4))
    np.testing.assert_allclose(oracle.exact_block_mass(q2, k2, bs)[0, 0], np.broadcast_to(n / N, (5, 5)),
                               atol=1e-15)


def test_two_keys_closed_form():
    # N = 2, block 1: M_00 = softmax weight of key 0 for query 0
    q = np.array([[[[1.0, 2.0]], ]]).reshape(1, 1, 1, 2)
    q = np.concatenate([q, np.array([0.5, -1.0]).reshape(1, 1, 1, 2)], axis=2)
    k = np.array([[0.3, 0.1], [-0.2, 0.4]]).reshape(1, 1, 2, 2)
    M = oracle.exact_block_mass(q, k, 1, scale=0.7)
    for a in range(2):
        s = [0.7 * (q[0, 0, a] @ k[0, 0, t]) for t in range(2)]
        w0 = 1.0 / (1.0 + math.exp(s[1] - s[0]))
        assert abs(M[0, 0, a, 0] - w0) < 1e-15 and abs(M[0, 0, a, 1] - (1 - w0)) < 1e-15


def test_matches_attention_of_one_hot_block_values():
    # O = softmax(sigma q k^T) V with V[t, j] = [t in block j] is the per-query
    # mass of each key block; averaging O over a query block gives M
    B, H, N, d, bs = 1, 2, 90, 16, 32
    q, k = _qk(B, H, N, d, 7, 0.8)
    nb = -(-N // bs)
    v = np.zeros((B, H, N, nb))
    for t in range(N):
        v[:, :, t, t // bs] = 1.0
    o, _ = oracle.block_sparse_attention(q, k, v, np.ones((B, H, nb, nb), np.uint8), bs)
    want = np.zeros((B, H, nb, nb))
    for i in range(nb):
        want[:, :, i] = o[:, :, i * bs:min((i + 1) * bs, N)].mean(axis=2)
    np.testing.assert_allclose(oracle.exact_block_mass(q, k, bs), want, rtol=1e-12, atol=1e-15)


def test_pure_python_loop_tiny():
    B, H, N, d, bs = 1, 1, 7, 3, 3
    q, k = _qk(B, H, N, d, 3)
    M = oracle.exact_block_mass(q, k, bs, scale=0.5)
    for i in range(3):
        rows = range(i * 3, min(i * 3 + 3, N))
        for j in range(3):
            tot = 0.0
            for a in rows:
                z = sum(math.exp(0.5 * sum(q[0, 0, a, c] * k[0, 0, t, c] for c in range(d))) for t in range(N))
                tot += sum(math.exp(0.5 * sum(q[0, 0, a, c] * k[0, 0, t, c] for c in range(d)))
                           for t in range(j * 3, min(j * 3 + 3, N))) / z
            assert abs(M[0, 0, i, j] - tot / len(rows)) < 1e-14


def test_rows_subset_and_nan_elsewhere():
    q, k = _qk(1, 2, 40, 4, 5)
    full = oracle.exact_block_mass(q, k, 16)
    part = oracle.exact_block_mass(q, k, 16, rows=[(0, 1, 2)])
    np.testing.assert_array_equal(part[0, 1, 2], full[0, 1, 2])
    assert np.isnan(part[0, 0]).all() and np.isnan(part[0, 1, :2]).all()


def test_selection_on_masses():
    # masses (0.5, 0.3, 0.2): tau 0.7 keeps the two largest; 0.8 exactly reaches
    # 0.5 + 0.3; ties within 1e-6 go to the lower index; tau 1 keeps all
    m = np.array([0.2, 0.5, 0.3])
    assert list(oracle.select_row_mass(m, 0.7)["keep"]) == [False, True, True]
    assert list(oracle.select_row_mass(m, 0.75)["keep"]) == [False, True, True]
    assert list(oracle.select_row_mass(m, 0.9)["keep"]) == [True, True, True]
    assert list(oracle.select_row_mass(m, 1.0)["keep"]) == [True, True, True]
    t = np.array([0.25, 0.25 + 5e-7, 0.25, 0.25 - 5e-7])
    r = oracle.select_row_mass(t, 0.4)
    assert r["k"] == 2 and list(r["keep"]) == [True, True, False, False]
    # selection depends on the masses only through their ratios
    mk, _ = oracle.mask_from_mass(np.array([[[[0.2, 0.5, 0.3], [0.1, 0.1, 0.8], [1 / 3, 1 / 3, 1 / 3]]]]), 0.6)
    assert mk[0, 0].tolist() == [[0, 1, 1], [0, 0, 1], [1, 1, 0]]


def test_admissible_masks_on_masses():
    # the list holds the selection's mask and the prefixes one shorter and
    # one longer (masses far from the tie band: no other variant)
    m = np.array([0.2, 0.5, 0.3])
    alts = [a.tolist() for a in oracle.row_admissible_masks_mass(m, 0.7)]
    assert alts == [[False, True, False], [False, True, True], [True, True, True]]
    # 0.5 + 0.25 reaches tau = 0.75 exactly (a fragile row): the prefixes of
    # length 2 and 3 are both admissible, the selection's among them
    m = np.array([0.25, 0.5, 0.25])
    r = oracle.select_row_mass(m, 0.75)
    assert r["fragile"]
    alts = [a.tolist() for a in oracle.row_admissible_masks_mass(m, 0.75)]
    assert r["keep"].tolist() in alts
    assert [True, True, False] in alts and [True, True, True] in alts and [False, True, False] in alts
    # a mass exactly 1e-6 below the cut mass: in the band or just outside it
    t = np.array([0.3 - 1e-6, 0.3, 0.4 + 1e-6])
    r = oracle.select_row_mass(t, 0.5)
    assert r["fragile"] and r["k"] == 2
    alts = [a.tolist() for a in oracle.row_admissible_masks_mass(t, 0.5)]
    assert [True, False, True] in alts and [False, True, True] in alts
    # tau >= 1 keeps everything, whatever the masses
    assert [a.tolist() for a in oracle.row_admissible_masks_mass(m, 1.0)] == [[True, True, True]]
