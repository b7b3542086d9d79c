"""Parity of the region-restricted path (through the C ABI) with the oracle.

Region codes, block flags and restricted lists must match bit for bit; W
within 1e-6 (fp32 of d / d_max and the smoothstep polynomial); the latent
blend within 2^-22 (|z_target| + |z_hist|) and exactly where W is 0 or 1;
attention of the active rows within the tolerances of the main parity tests,
the rows left out untouched.
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


def _check_regions(ev, ra=2, rc=3):
    code, w = P.region_weights(torch.as_tensor(ev, device=DEV), ra, rc)
    want_code, want_w = oracle.regions(ev, ra, rc)
    np.testing.assert_array_equal(code.cpu().numpy(), want_code)
    got_w = w.cpu().numpy().astype(np.float64)
    assert np.abs(got_w - want_w).max() <= 1e-6
    assert (got_w[want_w == 1.0] == 1.0).all() and (got_w[want_w == 0.0] == 0.0).all()
    return code, w


@pytest.mark.parametrize("wid", [0, 1, 2, 3, 4])
def test_region_weights_workloads(wid):
    wl = synth.WORKLOADS[wid]
    ev = synth.evidence_region(wl, seed=wid)
    _say("regions", wl.name, ev.shape, "evidence %.3f" % ev.mean())
    _check_regions(ev)


@pytest.mark.parametrize("shape,ra,rc", [((1, 1, 1, 1), 2, 3), ((2, 3, 5, 7), 2, 3), ((1, 2, 9, 70), 0, 0),
                                         ((1, 4, 33, 17), 1, 4), ((3, 2, 64, 64), 2, 3), ((1, 1, 256, 256), 6, 9)])
def test_region_weights_shapes_and_radii(shape, ra, rc):
    rng = np.random.default_rng(sum(shape) + ra)
    ev = (rng.random(shape) < 0.02).astype(np.uint8) * np.uint8(5)
    ev[0, 0].flat[0] = 1
    if shape[1] > 1:
        ev[-1, -1] = 0  # a frame without evidence
    _check_regions(ev, ra, rc)


def test_region_weights_degenerate_evidence():
    # no evidence anywhere: W = 0 and every code 0; evidence everywhere: W = 1;
    # evidence all but a border of one token: the band maximum is 1
    for ev in (np.zeros((1, 3, 12, 12), np.uint8), np.ones((1, 2, 12, 12), np.uint8)):
        _check_regions(ev)
    ev = np.zeros((1, 2, 9, 9), np.uint8)
    ev[0, :, 1:8, 1:8] = 1
    _check_regions(ev)


def test_region_weights_batch_entries_share_a_workgroup():
    # 6 batch entries of 2 x 3 x 7 tokens (252 tokens, one workgroup of the
    # weight pass) whose band maxima differ: 1 (evidence all but a border),
    # 2 (one evidence token), none (no evidence) and three random entries
    ev = np.zeros((6, 2, 3, 7), np.uint8)
    ev[0, :, 1:2, 1:6] = 1
    ev[0, 1] = 0
    ev[1, 0, 1, 3] = 1
    rng = np.random.default_rng(7)
    ev[3:] = (rng.random((3, 2, 3, 7)) < 0.1).astype(np.uint8)
    ev[3, 0, 0, 0] = 1
    _check_regions(ev)
    want_code, _ = oracle.regions(ev, 2, 3)
    assert len({int(x) for x in (want_code == 2).reshape(6, -1).sum(1)}) > 2


@pytest.mark.parametrize("wid,channels,patch", [(1, 16, (1, 2, 2)), (0, 4, (1, 1, 1)), (2, 3, (1, 2, 3)),
                                                (3, 16, (1, 2, 2))])
def test_latent_fusion(wid, channels, patch):
    wl = synth.WORKLOADS[wid]
    ev = synth.evidence_region(wl, seed=1)
    _, w = P.region_weights(torch.as_tensor(ev, device=DEV))
    zt, zh = synth.latents(wl, channels, patch, seed=1, device=DEV)
    _say("fusion", wl.name, tuple(zt.shape), "patch", patch)
    got = P.latent_fusion(zt, zh, w).cpu().numpy().astype(np.float64)
    want = oracle.latent_fusion(zt.cpu().numpy(), zh.cpu().numpy(), w.cpu().numpy(), patch)
    bound = 2.0 ** -22 * (np.abs(zt.cpu().numpy()) + np.abs(zh.cpu().numpy())) + 1e-30
    assert (np.abs(got - want) <= bound).all()
    wr = np.repeat(np.repeat(np.repeat(w.cpu().numpy(), patch[0], 1), patch[1], 2), patch[2], 3)[:, None]
    wr = np.broadcast_to(wr, got.shape)
    np.testing.assert_array_equal(got[wr == 1.0], zt.cpu().numpy()[wr == 1.0])
    np.testing.assert_array_equal(got[wr == 0.0], zh.cpu().numpy()[wr == 0.0])
    # in place over the historical latent
    zh2 = zh.clone()
    P.latent_fusion(zt, zh2, w, out=zh2)
    np.testing.assert_array_equal(zh2.cpu().numpy(), got.astype(np.float32))


@pytest.mark.parametrize("wid", [0, 1, 2, 3, 4])
def test_region_block_flags(wid):
    wl = synth.WORKLOADS[wid]
    ev = synth.evidence_region(wl, seed=2)
    code, _ = P.region_weights(torch.as_tensor(ev, device=DEV))
    act, ctx = P.region_block_flags(code, wl.n_text, wl.block)
    want_act, want_ctx = oracle.region_block_flags(code.cpu().numpy(), wl.n_text, wl.block)
    np.testing.assert_array_equal(act.cpu().numpy(), want_act)
    np.testing.assert_array_equal(ctx.cpu().numpy(), want_ctx)
    _say("flags", wl.name, "active %d context %d of %d" % (want_act.sum(), want_ctx.sum(), want_act.size))


# nB = 2^k - 1 exercises the key of the left-out rows next to the longest
# list; (2048, 7) keeps the sort's lengths in memory
@pytest.mark.parametrize("nb,density,heads,p_act", [(3, 0.5, 5, 0.5), (7, 0.6, 3, 0.4), (63, 0.3, 3, 0.3),
                                                    (139, 0.3, 5, 0.2), (256, 0.2, 4, 0.15), (591, 0.1, 2, 0.2),
                                                    (2048, 0.05, 7, 0.1), (931, 0.1, 12, 0.2), (100, 1.0, 2, 0.5),
                                                    (50, 0.4, 2, 0.0),
                                                    (50, 0.4, 2, 1.0)])
def test_compaction_region_bit_exact(nb, density, heads, p_act):
    B = 2
    m = synth.random_mask(B, heads, nb, density, nb + 3)
    rng = np.random.default_rng(nb)
    act = (rng.random((B, nb)) < p_act).astype(np.uint8)
    ctx = np.maximum(act, (rng.random((B, nb)) < 0.5).astype(np.uint8))
    bits = torch.as_tensor(oracle.pack_mask(m).view(np.int64), device=DEV)
    rp, ci, order, n = P.compact_block_mask_bits_region(bits, act, ctx)
    wrp, wci, word, wn = oracle.compact_restricted(m, act, ctx, group_heads=P.order_group_heads(B, heads, nb))
    assert int(n.item()) == wn
    np.testing.assert_array_equal(rp.cpu().numpy(), wrp)
    np.testing.assert_array_equal(ci[:int(wrp[-1])].cpu().numpy(), wci)
    np.testing.assert_array_equal(order.cpu().numpy(), word)


@pytest.mark.parametrize("wid", [0, 1, 2])
def test_region_restricted_attention(wid):
    """Historical mask -> bank slot -> regions from the evidence -> block flags
    -> restricted lists -> attention of the active rows only."""
    wl = synth.WORKLOADS[wid]
    x = synth.attention_inputs(wl, seed=0, device=DEV)
    ev = synth.evidence_region(wl, seed=0)
    bits = P.build_block_mask_bits(x["q_hist"], x["k_hist"], wl.block, wl.tau)
    code, _ = P.region_weights(torch.as_tensor(ev, device=DEV))
    act, ctx = P.region_block_flags(code, wl.n_text, wl.block)
    rp, ci, order, n = P.compact_block_mask_bits_region(bits, act, ctx)
    sentinel = torch.full_like(x["q"], 3.0)
    lse = torch.full((wl.batch, wl.heads, wl.seq_len), 7.0, dtype=torch.float32, device=DEV)
    o, lse = P.block_sparse_attn_lists(x["q"], x["k"], x["v"], (rp, ci, order), wl.block, out=sentinel,
                                       n_rows=n, return_lse=True, lse=lse)
    # the kernel without the LSE writes the same rows, bit for bit
    o_plain = P.block_sparse_attn_lists(x["q"], x["k"], x["v"], (rp, ci, order), wl.block,
                                        out=torch.full_like(x["q"], 3.0), n_rows=n)
    torch.cuda.synchronize()
    assert torch.equal(o.view(torch.int16), o_plain.view(torch.int16))
    nb = wl.n_blocks
    mask = oracle.unpack_mask(bits.cpu().numpy().view(np.uint64), nb)
    act_np, ctx_np = act.cpu().numpy(), ctx.cpu().numpy()
    restricted = oracle.restrict_mask(mask, act_np, ctx_np)
    n_act = int(n.item())
    assert n_act == int(act_np.sum()) * wl.heads
    active_rows = [(0, h, i) for h in range(wl.heads) for i in range(nb) if act_np[0, i]]
    rng = np.random.default_rng(wid)
    if len(active_rows) > 24:
        active_rows = [active_rows[k] for k in sorted(rng.choice(len(active_rows), 24, replace=False))]
    ro, rl = oracle.block_sparse_attention(oracle.to_f64(x["q"]), oracle.to_f64(x["k"]), oracle.to_f64(x["v"]),
                                           restricted, wl.block, rows=active_rows)
    og = o.float().cpu().numpy()
    lg = lse.cpu().numpy()
    d, r = [], []
    for (b, h, i) in active_rows:
        a0, a1 = i * wl.block, min((i + 1) * wl.block, wl.seq_len)
        d.append((og[b, h, a0:a1] - ro[b, h, a0:a1]).ravel())
        r.append(ro[b, h, a0:a1].ravel())
        fin = np.isfinite(rl[b, h, a0:a1])
        assert (np.isneginf(lg[b, h, a0:a1]) == ~fin).all()
        if fin.any():
            assert np.abs(lg[b, h, a0:a1][fin] - rl[b, h, a0:a1][fin]).max() <= 1e-3
    d, r = np.concatenate(d), np.concatenate(r)
    _say("restricted rows %d of %d active, max|d| %.3e" % (len(active_rows), n_act, np.abs(d).max()))
    assert np.abs(d).max() <= 2e-2
    assert np.linalg.norm(d) / max(np.linalg.norm(r), 1e-30) <= 5e-3
    # inactive query blocks: output and LSE untouched
    for i in range(nb):
        if act_np[0, i]:
            continue
        a0, a1 = i * wl.block, min((i + 1) * wl.block, wl.seq_len)
        assert (og[:, :, a0:a1] == 3.0).all() and (lg[:, :, a0:a1] == 7.0).all()
