"""Pins of the oracle's cosine scoring and top-k.

Checked against a hand-derived worked example (tests/golden), scipy's cosine
distance, the identities cos(x, x) = 1, cos(x, -x) = -1, cos(x, a x) = 1 for
a > 0, orthogonal vectors -> 0, a NumPy argsort top-k, and a planted
near-duplicate that must rank first.
"""
import json
import os

import numpy as np
import pytest
from scipy.spatial.distance import cdist

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_cosine_worked_example():
    with open(os.path.join(GOLDEN, "cosine_worked.json")) as f:
        g = json.load(f)
    bank = np.array(g["bank"], dtype=float)
    q = np.array(g["query"], dtype=float)
    np.testing.assert_allclose(oracle.cosine_similarity(q, bank), np.array(g["sims"]), atol=1e-15)
    idx, _, _ = oracle.topk_cosine(q[:1], bank, 4)
    assert idx[0].tolist() == g["top4_q0"]
    idx, _, _ = oracle.topk_cosine(q[1:], bank, 3)
    assert idx[0].tolist() == g["top3_q1"]


def test_cosine_matches_scipy():
    rng = np.random.default_rng(0)
    q = rng.standard_normal((3, 50)).astype(np.float32)
    b = rng.standard_normal((40, 50)).astype(np.float32)
    np.testing.assert_allclose(oracle.cosine_similarity(q, b), 1.0 - cdist(q.astype(float), b.astype(float), "cosine"),
                               atol=1e-14)


def test_cosine_identities():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(64)
    y = rng.standard_normal(64)
    y -= (y @ x) / (x @ x) * x  # orthogonal to x
    bank = np.stack([x, -x, 3.5 * x, y, np.zeros(64)])
    s = oracle.cosine_similarity(x[None], bank)[0]
    np.testing.assert_allclose(s, [1.0, -1.0, 1.0, 0.0, 0.0], atol=1e-14)


@pytest.mark.parametrize("k", [1, 5, 8, 64])
def test_topk_matches_argsort(k):
    sig = synth.signature_inputs(m=500, dim=96, nq=3, seed=2)
    q, b = sig["query"].numpy(), sig["bank"].numpy()
    idx, val, frag = oracle.topk_cosine(q, b, k)
    sims = 1.0 - cdist(q.astype(float), b.astype(float), "cosine")
    for r in range(3):
        assert not frag[r]
        want = np.argsort(-sims[r], kind="stable")[:k]
        assert idx[r].tolist() == want.tolist()
        np.testing.assert_allclose(val[r], sims[r][want], atol=1e-14)


def test_planted_near_duplicate_ranks_first():
    sig = synth.signature_inputs(m=4096, dim=256, nq=2, seed=5)
    idx, val, _ = oracle.topk_cosine(sig["query"].numpy(), sig["bank"].numpy(), 8)
    assert idx[1, 0] == sig["planted"]
    assert val[1, 0] > 0.8


def test_topk_tie_rule_lower_row():
    # Rows 1 and 3 within 1e-7 of each other at the cut: the lower row wins
    # the one remaining slot even though row 3 is (barely) larger.
    base = np.array([1.0, 0.0])
    ang = np.array([0.0, 0.5, 1.2, 0.5 - 1e-7, 1.5])
    bank = np.stack([np.cos(ang), np.sin(ang)], axis=1)
    idx, _, _ = oracle.topk_cosine(base[None], bank, 2)
    assert idx[0].tolist() == [0, 1]
