"""Pins of the oracle's block-sparse attention.

Checked against: a hand-derived worked example (tests/golden), PyTorch's
scaled_dot_product_attention in fp64 on the CPU (full mask, and the block mask
expanded to a boolean token mask), scipy's logsumexp, a pure-Python triple
loop on the tiny workload, and invariants (all-target rows = dense, V = 1
gives 1, key permutations inside the allowed set change nothing).
"""
import json
import math
import os

import numpy as np
import pytest
import torch
from scipy.special import logsumexp

import oracle
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(B, H, N, d, seed):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal((B, H, N, d)) for _ in range(3)]


def _sdpa(q, k, v, bool_mask=None, scale=None):
    tq, tk, tv = (torch.from_numpy(np.ascontiguousarray(x)) for x in (q, k, v))
    am = None if bool_mask is None else torch.from_numpy(bool_mask)
    return torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=am, scale=scale).numpy()


def _token_mask(mask, N, bs):
    B, H, nb, _ = mask.shape
    rows = np.repeat(mask != 0, bs, axis=2)[:, :, :N]
    return np.repeat(rows, bs, axis=3)[:, :, :, :N]


def test_attention_worked_example():
    with open(os.path.join(GOLDEN, "attention_worked.json")) as f:
        g = json.load(f)
    q = np.array(g["q"], dtype=float)[None, None]
    k = np.array(g["k"], dtype=float)[None, None]
    v = np.array(g["v"], dtype=float)[None, None]
    conv = {"0": 0.0, "-inf": -np.inf}
    for case in g["cases"]:
        m = np.array(case["mask"], dtype=np.uint8)[None, None]
        o, lse = oracle.block_sparse_attention(q, k, v, m, g["block"], scale=g["scale"])
        np.testing.assert_allclose(o[0, 0], np.array(case["o"], dtype=float), atol=1e-12)
        want = [conv[x] if x in conv else math.log(float(x[2:])) for x in case["lse"]]
        np.testing.assert_allclose(lse[0, 0], want, atol=1e-12)


@pytest.mark.parametrize("N,bs", [(200, 64), (256, 128), (130, 64)])
def test_full_mask_equals_sdpa(N, bs):
    q, k, v = _rand(1, 2, N, 16, N)
    nb = -(-N // bs)
    o, _ = oracle.block_sparse_attention(q, k, v, np.ones((1, 2, nb, nb), np.uint8), bs)
    np.testing.assert_allclose(o, _sdpa(q, k, v), atol=1e-12, rtol=0)


@pytest.mark.parametrize("seed", range(3))
def test_block_mask_equals_sdpa_with_token_mask(seed):
    N, bs, d = 300, 64, 32
    q, k, v = _rand(2, 2, N, d, seed)
    nb = -(-N // bs)
    m = synth.random_mask(2, 2, nb, 0.4, seed)
    m[..., 0] = 1  # every row keeps at least one block (SDPA has no empty-row rule)
    o, lse = oracle.block_sparse_attention(q, k, v, m, bs, scale=0.3)
    tm = _token_mask(m, N, bs)
    np.testing.assert_allclose(o, _sdpa(q, k, v, tm, scale=0.3), atol=1e-12, rtol=0)
    s = 0.3 * np.einsum("bhnd,bhmd->bhnm", q, k)
    s[~tm] = -np.inf
    np.testing.assert_allclose(lse, logsumexp(s, axis=-1), atol=1e-12)


def test_all_target_rows_equal_dense():
    N, bs = 256, 64
    q, k, v = _rand(1, 2, N, 16, 7)
    nb = N // bs
    m = synth.random_mask(1, 2, nb, 0.2, 7)
    merged = oracle.merge_target_rows(m, np.ones((1, nb), np.uint8))
    o, _ = oracle.block_sparse_attention(q, k, v, merged, bs)
    np.testing.assert_allclose(o, _sdpa(q, k, v), atol=1e-12, rtol=0)


def test_rows_sum_to_one_with_unit_values():
    N, bs = 190, 64
    q, k, _ = _rand(1, 3, N, 8, 9)
    v = np.ones((1, 3, N, 4))
    nb = -(-N // bs)
    m = synth.random_mask(1, 3, nb, 0.5, 9)
    m[:, :, :, 1] = 1
    o, _ = oracle.block_sparse_attention(q, k, v, m, bs)
    np.testing.assert_allclose(o, 1.0, atol=1e-13, rtol=0)


def test_empty_row_gives_zero_and_minus_inf():
    N, bs = 128, 64
    q, k, v = _rand(1, 1, N, 8, 11)
    m = np.array([[[[1, 1], [0, 0]]]], dtype=np.uint8)
    o, lse = oracle.block_sparse_attention(q, k, v, m, bs)
    assert (o[0, 0, 64:] == 0).all() and np.isneginf(lse[0, 0, 64:]).all()
    assert np.isfinite(lse[0, 0, :64]).all()


def test_key_block_permutation_invariance():
    N, bs = 256, 64
    q, k, v = _rand(1, 2, N, 16, 13)
    nb = N // bs
    m = synth.random_mask(1, 2, nb, 0.5, 13)
    m[..., 2] = 1
    perm = np.array([2, 0, 3, 1])
    tok = np.concatenate([np.arange(p * bs, (p + 1) * bs) for p in perm])
    o, _ = oracle.block_sparse_attention(q, k, v, m, bs)
    o2, _ = oracle.block_sparse_attention(q, k[:, :, tok], v[:, :, tok], m[..., perm], bs)
    np.testing.assert_allclose(o2, o, atol=1e-13, rtol=0)


def _triple_loop(q, k, v, mask, bs, sigma):
    """Pure-Python definition for one head, used on the tiny workload."""
    N, d = len(q), len(q[0])
    out = []
    for a in range(N):
        i = a // bs
        keys = [t for t in range(N) if mask[i][t // bs]]
        if not keys:
            out.append([0.0] * len(v[0]))
            continue
        s = [sigma * sum(q[a][c] * k[t][c] for c in range(d)) for t in keys]
        m = max(s)
        w = [math.exp(x - m) for x in s]
        z = sum(w)
        out.append([sum(w[n] * v[t][c] for n, t in enumerate(keys)) / z for c in range(len(v[0]))])
    return out


def test_triple_loop_tiny_workload():
    wl = synth.WORKLOADS[0]
    x = synth.attention_inputs(wl, seed=0)
    q, k, v = (oracle.to_f64(x[n]) for n in ("q", "k", "v"))
    mh, _ = oracle.build_block_mask(oracle.to_f64(x["q_hist"]), oracle.to_f64(x["k_hist"]), wl.block, wl.tau)
    m = oracle.merge_target_rows(mh, x["row_flags"].numpy())
    o, _ = oracle.block_sparse_attention(q, k, v, m, wl.block)
    h = 1
    ref = _triple_loop(q[0, h].tolist(), k[0, h].tolist(), v[0, h].tolist(), m[0, h].tolist(),
                       wl.block, 1.0 / math.sqrt(wl.head_dim))
    np.testing.assert_allclose(o[0, h], np.array(ref), atol=1e-12, rtol=0)


def test_row_subset_matches_full():
    N, bs = 256, 64
    q, k, v = _rand(1, 2, N, 16, 17)
    m = synth.random_mask(1, 2, 4, 0.5, 17)
    o, lse = oracle.block_sparse_attention(q, k, v, m, bs)
    rows = [(0, 1, 2), (0, 0, 3)]
    o2, lse2 = oracle.block_sparse_attention(q, k, v, m, bs, rows=rows)
    for (b, h, i) in rows:
        np.testing.assert_array_equal(o2[b, h, i * bs:(i + 1) * bs], o[b, h, i * bs:(i + 1) * bs])
        np.testing.assert_array_equal(lse2[b, h, i * bs:(i + 1) * bs], lse[b, h, i * bs:(i + 1) * bs])
    assert np.isnan(o2[0, 0, :bs]).all()
