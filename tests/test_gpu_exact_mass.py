"""Parity of the exact-mass builder (through the C ABI) with the oracle.

Block masses: |dM| <= 1e-4 M + 1e-7 against the fp64 oracle (bf16 inputs,
fp32 scores and softmax statistics: about 1e-6 relative per score, 1e-5
after the exponent), rows summing to 1 within 1e-5.  Selection on given
masses: bit-exact against the oracle's selection on the same fp64 masses,
except rows whose decision lies within 1e-9 of a threshold (reported).
"""
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_32420_amd as P
import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _rand(B, H, N, d, seed, scale):
    g = torch.Generator().manual_seed(seed)
    q = (torch.randn(B, H, N, d, generator=g) * scale).to(torch.bfloat16)
    k = (torch.randn(B, H, N, d, generator=g) * scale).to(torch.bfloat16)
    return q.to(DEV), k.to(DEV)


def _check_fragile_rows(got, want, m, rep, tau):
    """Rows where the GPU's mask differs must be fragile, and the GPU's mask
    one of the oracle's admissible masks for that row."""
    bad = [tuple(int(v) for v in r) for r in np.argwhere((got != want).any(axis=-1))]
    assert set(bad) <= set(rep["fragile"]), bad[:5]
    for (b, h, i) in bad:
        alts = oracle.row_admissible_masks_mass(m[b, h, i], tau)
        assert any(np.array_equal(got[b, h, i] != 0, a) for a in alts), (b, h, i)
    _say("selection rows differing: %d (all fragile and admissible), fragile %d" % (len(bad), len(rep["fragile"])))


def _check_mass(got, want):
    g = got.cpu().numpy()
    ok = ~np.isnan(want)
    err = np.abs(g[ok] - want[ok])
    assert (err <= 1e-4 * want[ok] + 1e-7).all(), float((err / (want[ok] + 1e-7)).max())
    return g


@pytest.mark.parametrize("N,bs,d,scale", [(50, 64, 64, 1.0), (64, 64, 128, 0.6), (200, 64, 128, 1.0),
                                          (333, 128, 64, 1.5), (1000, 128, 128, 1.0), (257, 128, 128, 3.0)])
def test_block_mass_random_shapes(N, bs, d, scale):
    q, k = _rand(2, 2, N, d, N + d, scale)
    _say("mass", N, bs, d, scale)
    got = P.block_mass_exact(q, k, bs)
    want = oracle.exact_block_mass(oracle.to_f64(q), oracle.to_f64(k), bs)
    g = _check_mass(got, want)
    np.testing.assert_allclose(g.sum(axis=-1), 1.0, atol=1e-5)


def test_block_mass_explicit_scale_and_strided_views():
    # [B, N, H, d] storage viewed as [B, H, N, d]
    g = torch.Generator().manual_seed(3)
    base = (torch.randn(1, 300, 3, 64, generator=g)).to(torch.bfloat16).to(DEV)
    kb = (torch.randn(1, 300, 3, 64, generator=g)).to(torch.bfloat16).to(DEV)
    q, k = base.permute(0, 2, 1, 3), kb.permute(0, 2, 1, 3)
    got = P.block_mass_exact(q, k, 64, scale=0.3)
    want = oracle.exact_block_mass(oracle.to_f64(q), oracle.to_f64(k), 64, scale=0.3)
    _check_mass(got, want)


@pytest.mark.parametrize("wid", [0, 1, 2])
def test_block_mass_workloads(wid):
    wl = synth.WORKLOADS[wid]
    heads = None if wid == 0 else 2
    x = synth.attention_inputs(wl, seed=0, device=DEV, heads=heads)
    _say("mass workload", wl.name, "heads", heads)
    got = P.block_mass_exact(x["q_hist"], x["k_hist"], wl.block)
    nb = wl.n_blocks
    rng = np.random.default_rng(wid)
    H = x["q_hist"].shape[1]
    rows = sorted({(0, int(rng.integers(0, H)), int(rng.integers(0, nb))) for _ in range(6)} |
                  {(0, H - 1, nb - 1), (0, 0, 0)})
    want = oracle.exact_block_mass(oracle.to_f64(x["q_hist"]), oracle.to_f64(x["k_hist"]), wl.block, rows=rows)
    g = _check_mass(got, want)
    np.testing.assert_allclose(g.sum(axis=-1), 1.0, atol=1e-5)


@pytest.mark.parametrize("wid", [1, 3])
def test_selection_on_masses_bit_exact(wid):
    wl = synth.WORKLOADS[wid]
    x = synth.attention_inputs(wl, seed=1, device=DEV, heads=2)
    mass = P.block_mass_exact(x["q_hist"], x["k_hist"], wl.block)
    m = mass.cpu().numpy()
    want, rep = oracle.mask_from_mass(m, wl.tau)
    got = P.select_block_mask(mass, wl.tau).cpu().numpy()
    _check_fragile_rows(got, want, m, rep, wl.tau)
    # sampled rows of the masses themselves against the fp64 oracle
    rng = np.random.default_rng(10 + wid)
    nb = wl.n_blocks
    rows = sorted({(0, int(rng.integers(0, 2)), int(rng.integers(0, nb))) for _ in range(4)} | {(0, 1, nb - 1)})
    ref = oracle.exact_block_mass(oracle.to_f64(x["q_hist"]), oracle.to_f64(x["k_hist"]), wl.block, rows=rows)
    _check_mass(mass, ref)
    bits = P.select_block_mask(mass, wl.tau, bits=True)
    np.testing.assert_array_equal(bits.cpu().numpy().view(np.uint64), oracle.pack_mask(got))
    pooled = P.build_block_mask(x["q_hist"], x["k_hist"], wl.block, wl.tau).cpu().numpy()
    inter = (pooled & got).sum()
    _say("exact vs pooled: density %.4f vs %.4f, jaccard %.3f, fragile %d" % (
        got.mean(), pooled.mean(), inter / max((pooled | got).sum(), 1), len(rep["fragile"])))


@pytest.mark.parametrize("nb,tau", [(10, 0.45), (300, 0.123), (129, 1.0)])
def test_selection_on_equal_masses(nb, tau):
    # every mass equal: k = ceil(tau nB), the lowest blocks (tau = 1: all)
    mass = torch.full((1, 2, nb, nb), 1.0 / nb, dtype=torch.float64, device=DEV)
    got = P.select_block_mask(mass, tau).cpu().numpy()
    k = nb if tau >= 1 else int(np.ceil(tau * nb))
    want = np.zeros(nb, np.uint8)
    want[:k] = 1
    assert (got == want).all()


# every launch shape of the selection's mass mode: nB <= 512 (16 rows, 16
# waves), <= 1024 (16 rows, 8 waves), up to 2048 (8 rows, 8 waves), with
# masses that repeat exactly (ties at the cut)
@pytest.mark.parametrize("nb,tau", [(1, 0.9), (63, 0.5), (700, 0.9), (1025, 0.8), (2048, 0.95)])
def test_selection_on_synthetic_masses_all_launch_shapes(nb, tau):
    rng = np.random.default_rng(nb)
    m = rng.random((1, 2, nb, nb)) ** 6
    m[..., ::7] = m[..., :1]  # exact repeats of the first mass in every row
    m /= m.sum(axis=-1, keepdims=True)
    want, rep = oracle.mask_from_mass(m, tau)
    got = P.select_block_mask(torch.as_tensor(m, device=DEV), tau).cpu().numpy()
    _check_fragile_rows(got, want, m, rep, tau)
    bits = P.select_block_mask(torch.as_tensor(m, device=DEV), tau, bits=True).cpu().numpy().view(np.uint64)
    np.testing.assert_array_equal(bits, oracle.pack_mask(got))


def test_block_mass_heads_in_chunks():
    # The 75.6K-token shape with all 40 heads: 358 MB of records per head, so
    # the pass runs in chunks of 12 heads (the 4 GiB cap).  Sampled rows of
    # heads in every chunk against the fp64 oracle; every row sums to 1.
    wl = synth.WORKLOADS[3]
    x = synth.attention_inputs(wl, seed=2, device=DEV)
    _say("mass in chunks", wl.name)
    mass = P.block_mass_exact(x["q_hist"], x["k_hist"], wl.block)
    g = mass.cpu().numpy()
    np.testing.assert_allclose(g.sum(axis=-1), 1.0, atol=1e-5)
    nb = wl.n_blocks
    rows = [(0, 0, 0), (0, 11, 300), (0, 12, 5), (0, 25, nb - 1), (0, 36, 200), (0, 39, 17)]
    for (b, h, i) in rows:
        ref = oracle.exact_block_mass(oracle.to_f64(x["q_hist"][:, h:h + 1]), oracle.to_f64(x["k_hist"][:, h:h + 1]),
                                      wl.block, rows=[(b, 0, i)])
        _check_mass(mass[:, h:h + 1], ref)
