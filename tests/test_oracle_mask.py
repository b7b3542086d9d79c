"""Pins of the oracle's pooling, top-mass selection, merge and compaction.

Each test checks the oracle against something other than itself: hand-derived
worked examples (tests/golden), brute-force enumeration of every subset,
closed forms and set identities.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _parse_scores(text):
    vals = []
    for tok in text.split():
        v = 0.0
        for part in tok.replace("+", " +").split():
            if part.startswith("+"):
                v += float(part[1:])
            elif part.startswith("ln"):
                v += math.log(float(part[2:]))
            else:
                v += float(part)
        vals.append(v)
    return np.array(vals)


# ---------------------------------------------------------------- pooling

def test_pool_constant_blocks_and_tail_divisor():
    # Block j is filled with the constant j+1; the tail block has 3 tokens.
    bs, d = 4, 5
    n = 3 * bs + 3
    x = np.zeros((n, d))
    for j in range(4):
        x[j * bs:(j + 1) * bs] = j + 1
    p = oracle.pool_blocks(x, bs)
    assert p.shape == (4, d)
    np.testing.assert_array_equal(p, np.repeat(np.arange(1, 5, dtype=float)[:, None], d, axis=1))


def test_pool_linear_and_equals_reshape_mean():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((6 * 8, 7))
    y = rng.standard_normal((6 * 8, 7))
    px, py = oracle.pool_blocks(x, 8), oracle.pool_blocks(y, 8)
    np.testing.assert_allclose(oracle.pool_blocks(2.0 * x - 3.0 * y, 8), 2.0 * px - 3.0 * py, atol=1e-13)
    np.testing.assert_allclose(px, x.reshape(6, 8, 7).mean(axis=1), atol=1e-14)


# ---------------------------------------------------------------- selection

@pytest.mark.parametrize("case", _load("select_worked.json")["cases"], ids=lambda c: c["name"])
def test_select_worked_examples(case):
    r = oracle.select_row(_parse_scores(case["scores"]), case["tau"])
    assert r["k"] == case["k"]
    assert r["keep"].astype(int).tolist() == case["keep"]
    assert not r["fragile"]


def test_mask_worked_example():
    g = _load("mask_worked.json")
    qh = np.array(g["q_hist"], dtype=float)[None, None]
    kh = np.array(g["k_hist"], dtype=float)[None, None]
    np.testing.assert_array_equal(oracle.pool_blocks(qh[0, 0], g["block"]), np.array(g["qbar"], dtype=float))
    np.testing.assert_array_equal(oracle.pool_blocks(kh[0, 0], g["block"]), np.array(g["kbar"], dtype=float))
    for case in g["cases"]:
        m, rep = oracle.build_block_mask(qh, kh, g["block"], case["tau"], scale=g["scale"])
        assert m[0, 0].tolist() == case["mask"]
        assert rep["fragile"] == []


def _brute_force_keep(s, tau):
    """Smallest cardinality whose best subset reaches tau; among those subsets
    the one of largest mass (scores are continuous, so it is unique)."""
    n = len(s)
    p = np.exp(s - s.max())
    p /= p.sum()
    for r in range(1, n + 1):
        best, best_mass = None, -1.0
        for sub in itertools.combinations(range(n), r):
            mass = sum(p[list(sub)])
            if mass > best_mass:
                best, best_mass = sub, mass
        if best_mass >= tau:
            keep = np.zeros(n, dtype=bool)
            keep[list(best)] = True
            return keep
    return np.ones(n, dtype=bool)


@pytest.mark.parametrize("seed", range(12))
def test_select_matches_subset_enumeration(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(2, 11))
    s = rng.normal(0.0, 1.5, size=n)
    for tau in (0.3, 0.5, 0.8, 0.9, 0.97):
        r = oracle.select_row(s, tau)
        if r["fragile"]:
            continue
        np.testing.assert_array_equal(r["keep"], _brute_force_keep(s, tau))


def test_select_closed_forms():
    # tau >= 1 keeps everything.
    assert oracle.select_row(np.array([5.0, -2.0, 0.0]), 1.0)["keep"].all()
    # A dominant block alone covers any tau below its mass.
    r = oracle.select_row(np.array([0.0, 40.0, 1.0, -3.0]), 0.99)
    assert r["k"] == 1 and r["keep"].tolist() == [False, True, False, False]
    # n equal scores: k = ceil(tau * n), the lowest indices.
    for n, tau in ((7, 0.5), (10, 0.33), (5, 0.9)):
        r = oracle.select_row(np.zeros(n), tau)
        k = math.ceil(tau * n)
        assert r["k"] == k
        assert r["keep"].tolist() == [True] * k + [False] * (n - k)


def test_select_planted_tie_goes_to_lower_index():
    # Block 3 beats block 1 by 1e-7 < 1e-6: exact order keeps 3, the tie rule 1.
    s = np.array([2.0, 0.5, -1.0, 0.5 + 1e-7, -1.0])
    r = oracle.select_row(s, 0.7)
    assert r["k"] == 2
    assert r["keep"].tolist() == [True, True, False, False, False]
    # Beyond the tie band the exact order decides.
    s2 = s.copy()
    s2[3] = 0.5 + 1e-4
    assert oracle.select_row(s2, 0.7)["keep"].tolist() == [True, False, False, True, False]


def test_select_fragile_rows_list_alternatives():
    # Cumulative mass equal to tau (to rounding): reported fragile, and both
    # k and k+1 prefixes are admissible.
    s = np.log(np.array([4.0, 2.0, 1.0, 1.0]))
    r = oracle.select_row(s, 0.75)
    assert r["fragile"]
    alts = oracle.row_admissible_masks(s, 0.75)
    assert any(a.tolist() == [True, True, False, False] for a in alts)
    assert any(a.tolist() == [True, True, True, False] for a in alts)


def test_build_mask_full_threshold_and_shapes():
    rng = np.random.default_rng(3)
    qh = rng.standard_normal((2, 3, 130, 8))
    kh = rng.standard_normal((2, 3, 130, 8))
    m, rep = oracle.build_block_mask(qh, kh, 32, 1.0)
    assert m.shape == (2, 3, 5, 5) and m.dtype == np.uint8 and m.all()
    m2, rep2 = oracle.build_block_mask(qh, kh, 32, 0.6)
    assert set(np.unique(m2)) <= {0, 1}
    assert (m2.sum(axis=-1) >= 1).all()
    # The count kept equals the prefix length k of every row.
    np.testing.assert_array_equal(m2.sum(axis=-1), rep2["k"])


# ---------------------------------------------------------------- merge

def test_merge_identities():
    rng = np.random.default_rng(4)
    m = (rng.random((2, 3, 6, 6)) < 0.3).astype(np.uint8)
    none = np.zeros((2, 6), dtype=np.uint8)
    np.testing.assert_array_equal(oracle.merge_target_rows(m, none), m)
    assert oracle.merge_target_rows(m, np.ones((2, 6), dtype=np.uint8)).all()
    rows = (rng.random((2, 6)) < 0.5).astype(np.uint8)
    cols = (rng.random((2, 6)) < 0.3).astype(np.uint8)
    once = oracle.merge_target_rows(m, rows, cols)
    np.testing.assert_array_equal(oracle.merge_target_rows(once, rows, cols), once)
    for b in range(2):
        for i in np.nonzero(rows[b])[0]:
            assert once[b, :, i].all()
        for j in np.nonzero(cols[b])[0]:
            assert once[b, :, :, j].all()
    # Bytes other than 0/1 count as kept.
    m7 = m * 7
    np.testing.assert_array_equal(oracle.merge_target_rows(m7, none), m)


# ---------------------------------------------------------------- compaction

def test_compact_grouped_order_by_brute_force():
    # heads in groups of G: the order is (group, descending length, row), the
    # definition written out as a sort of tuples; one group (G >= heads) is
    # the plain longest-first order
    rng = np.random.default_rng(11)
    m = (rng.random((2, 5, 7, 7)) < 0.4).astype(np.uint8)
    m[1, 2, 4] = 0
    nb = 7
    flat = m.reshape(-1, nb)
    lens = flat.sum(axis=1)
    R = flat.shape[0]
    for G in (1, 2, 3, 4, 10, 11):
        _, _, order = oracle.compact_mask(m, group_heads=G)
        want = sorted(range(R), key=lambda r: (r // (G * nb), -int(lens[r]), r))
        assert order.tolist() == want, G
    np.testing.assert_array_equal(oracle.compact_mask(m, group_heads=10)[2], oracle.compact_mask(m)[2])
    # restricted lists: the active rows grouped the same way, the inactive
    # rows after them in row order
    act = (rng.random((2, nb)) < 0.6).astype(np.uint8)
    ctx = np.ones((2, nb), np.uint8)
    for G in (2, 3):
        rp, _, order, n_act = oracle.compact_restricted(m, act, ctx, group_heads=G)
        rl = np.diff(rp)
        active = np.broadcast_to(act[:, None, :] != 0, (2, 5, nb)).reshape(-1)
        want = sorted([r for r in range(R) if active[r]], key=lambda r: (r // (G * nb), -int(rl[r]), r))
        want += [r for r in range(R) if not active[r]]
        assert order.tolist() == want and n_act == int(active.sum())


def test_compact_roundtrip_and_order():
    rng = np.random.default_rng(5)
    m = (rng.random((1, 4, 9, 9)) < 0.35).astype(np.uint8)
    m[0, 1, 3] = 0  # an empty row
    row_ptr, col_idx, order = oracle.compact_mask(m)
    flat = m.reshape(-1, 9)
    R = flat.shape[0]
    assert row_ptr[0] == 0 and row_ptr[-1] == flat.sum()
    dense = np.zeros_like(flat)
    for r in range(R):
        cols = col_idx[row_ptr[r]:row_ptr[r + 1]]
        assert (np.diff(cols) > 0).all()
        dense[r, cols] = 1
    np.testing.assert_array_equal(dense, flat)
    lens = np.diff(row_ptr)
    assert sorted(order.tolist()) == list(range(R))
    for a, b in zip(order[:-1], order[1:]):
        assert lens[a] > lens[b] or (lens[a] == lens[b] and a < b)


# ---------------------------------------------------------------- bit-packed masks

def test_pack_single_bits_by_hand():
    # every column of a 130-wide row alone: exactly bit j mod 64 of word j // 64
    nb = 130
    for j in range(nb):
        m = np.zeros((1, nb), dtype=np.uint8)
        m[0, j] = 7
        w = oracle.pack_mask(m)
        assert w.shape == (1, 3) and w.dtype == np.uint64
        want = [0, 0, 0]
        want[j // 64] = 1 << (j % 64)
        assert [int(x) for x in w[0]] == want, j


@pytest.mark.parametrize("nb", [1, 3, 63, 64, 65, 139, 256, 931])
def test_pack_matches_numpy_packbits(nb):
    # little-endian bit order within bytes and words: packbits(bitorder="little")
    # laid out as little-endian uint64 is the same encoding
    rng = np.random.default_rng(nb)
    m = (rng.random((2, 3, nb, nb)) < 0.3).astype(np.uint8) * rng.integers(1, 255, (2, 3, nb, nb)).astype(np.uint8)
    w = (nb + 63) // 64
    pb = np.packbits(m != 0, axis=-1, bitorder="little")
    padded = np.zeros(m.shape[:-1] + (w * 8,), dtype=np.uint8)
    padded[..., :pb.shape[-1]] = pb
    np.testing.assert_array_equal(oracle.pack_mask(m), padded.view("<u8"))


@pytest.mark.parametrize("nb", [1, 64, 100, 200])
def test_unpack_inverts_pack_and_ignores_padding(nb):
    rng = np.random.default_rng(nb + 1)
    m = (rng.random((4, nb, nb)) < 0.5).astype(np.uint8)
    bits = oracle.pack_mask(m)
    np.testing.assert_array_equal(oracle.unpack_mask(bits, nb), m)
    if nb % 64:
        # the high bits of the last word are 0 when packed and ignored when read
        assert not (bits[..., -1] >> np.uint64(nb % 64)).any()
        dirty = bits.copy()
        dirty[..., -1] |= ~((np.uint64(1) << np.uint64(nb % 64)) - np.uint64(1))
        np.testing.assert_array_equal(oracle.unpack_mask(dirty, nb), m)
    # popcount of a row's words = its number of kept blocks
    pc = np.array([[bin(int(x)).count("1") for x in row] for row in bits.reshape(-1, bits.shape[-1])])
    np.testing.assert_array_equal(pc.sum(axis=1), m.reshape(-1, nb).sum(axis=1))


def test_pack_full_and_empty_rows():
    for nb, last in ((64, 2**64 - 1), (70, 2**6 - 1), (128, 2**64 - 1), (1, 1)):
        full = oracle.pack_mask(np.ones((nb, nb), dtype=np.uint8))
        assert all(int(x) == 2**64 - 1 for x in full[:, :-1].ravel())
        assert all(int(x) == last for x in full[:, -1])
        assert not oracle.pack_mask(np.zeros((nb, nb), dtype=np.uint8)).any()


def test_bank_slot_size():
    # one stored mask per (step, branch, layer): a 256-block Wan-shaped mask of
    # 12 heads takes 12 * 256 * 4 words; 50 steps x 2 branches x 30 layers of
    # them are 294,912,000 bytes, an eighth of the uint8 masks
    bits = oracle.pack_mask(np.zeros((1, 12, 256, 256), dtype=np.uint8))
    assert bits.shape == (1, 12, 256, 4)
    assert bits.nbytes * 50 * 2 * 30 == 294_912_000
    assert bits.nbytes * 8 == 12 * 256 * 256
