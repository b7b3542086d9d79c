"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Masks, merged masks and compacted lists must match bit for bit (rows the
oracle reports as fragile -- a decision within 1e-9 of a threshold -- may take
any admissible value).  Attention must match within max-abs 2e-2 and relative
L2 5e-3 on the valid tokens compared; top-k indices exactly and cosines within
1e-6.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2609_32420_amd as P
import synth

pytestmark = pytest.mark.gpu

DEV = "cuda"
ATOL = 2e-2
REL_L2 = 5e-3


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _inputs(wid, seed=0, heads=None):
    wl = synth.WORKLOADS[wid]
    _say("inputs", wl.name, "seed", seed, "heads", heads)
    return wl, synth.attention_inputs(wl, seed=seed, device=DEV, heads=heads)


def _oracle_mask(x, wl):
    """Oracle mask, built one head at a time to bound host memory."""
    B, H = x["q_hist"].shape[:2]
    nb = wl.n_blocks
    m = np.zeros((B, H, nb, nb), dtype=np.uint8)
    fragile = {}
    for h in range(H):
        mh, rep = oracle.build_block_mask(oracle.to_f64(x["q_hist"][:, h:h + 1]),
                                          oracle.to_f64(x["k_hist"][:, h:h + 1]), wl.block, wl.tau)
        m[:, h] = mh[:, 0]
        for (b, _, i) in rep["fragile"]:
            fragile[(b, h, i)] = rep["scores"][(b, 0, i)]
    return m, fragile


def _assert_masks_equal(got, want, fragile, tau):
    got = got.cpu().numpy()
    bad = np.argwhere((got != want).any(axis=-1))
    for (b, h, i) in bad:
        key = (int(b), int(h), int(i))
        assert key in fragile, "mask row %s differs (k gpu %d, oracle %d)" % (
            key, got[b, h, i].sum(), want[b, h, i].sum())
        alts = oracle.row_admissible_masks(fragile[key], tau)
        assert any(np.array_equal(got[b, h, i] != 0, a) for a in alts), key
    _say("mask rows compared:", got.shape[0] * got.shape[1] * got.shape[2], "fragile:", len(fragile),
         "density: %.4f" % got.mean())


def _compare_rows(o_gpu, o_ref, lse_gpu, lse_ref, rows, N, bs):
    og = o_gpu.float().cpu().numpy()
    diffs, refs = [], []
    for (b, h, i) in rows:
        a0, a1 = i * bs, min((i + 1) * bs, N)
        diffs.append((og[b, h, a0:a1] - o_ref[b, h, a0:a1]).ravel())
        refs.append(o_ref[b, h, a0:a1].ravel())
        if lse_gpu is not None:
            lg = lse_gpu[b, h, a0:a1].cpu().numpy().astype(np.float64)
            lr = lse_ref[b, h, a0:a1]
            fin = np.isfinite(lr)
            assert (np.isneginf(lg) == np.isneginf(lr)).all()
            if fin.any():
                assert np.abs(lg[fin] - lr[fin]).max() <= 1e-3
    d = np.concatenate(diffs)
    r = np.concatenate(refs)
    mx = float(np.abs(d).max()) if d.size else 0.0
    rel = float(np.linalg.norm(d) / max(np.linalg.norm(r), 1e-30))
    _say("attention rows %d  max|d| %.3e  relL2 %.3e" % (len(rows), mx, rel))
    assert mx <= ATOL
    assert rel <= REL_L2


def _group_heads(m, attn=None):
    """Heads per group of the row order the library writes for masks shaped
    like m (and the attention shape attn)."""
    B, H, nb = m.shape[:3]
    return P.order_group_heads(B, H, nb, attn)


def _sample_rows(wl, merged, rows_flags, heads, n_random=32, seed=0):
    """Every target row of head 0, seeded random rows, and the last block of
    every head."""
    nb = wl.n_blocks
    rows = set()
    for i in np.nonzero(rows_flags[0])[0]:
        rows.add((0, 0, int(i)))
    rng = np.random.default_rng(seed)
    for _ in range(n_random):
        rows.add((0, int(rng.integers(0, heads)), int(rng.integers(0, nb))))
    for h in range(heads):
        rows.add((0, h, nb - 1))
    return sorted(rows)


# ---------------------------------------------------------------- mask builder

@pytest.mark.parametrize("wid", [0, 1, 2, 3, 4])
def test_mask_builder_bit_exact(wid):
    wl, x = _inputs(wid)
    got = P.build_block_mask(x["q_hist"], x["k_hist"], wl.block, wl.tau)
    torch.cuda.synchronize()
    want, fragile = _oracle_mask(x, wl)
    _assert_masks_equal(got, want, fragile, wl.tau)


@pytest.mark.parametrize("tau", [0.3, 0.97, 1.0])
def test_mask_builder_thresholds_and_explicit_scale(tau):
    wl, x = _inputs(0, seed=3)
    got = P.build_block_mask(x["q_hist"], x["k_hist"], wl.block, tau, scale=0.05)
    torch.cuda.synchronize()
    want, rep = oracle.build_block_mask(oracle.to_f64(x["q_hist"]), oracle.to_f64(x["k_hist"]), wl.block, tau,
                                        scale=0.05)
    fragile = {k: rep["scores"][k] for k in rep["fragile"]}
    _assert_masks_equal(got, want, fragile, tau)


@pytest.mark.parametrize("N,bs,d", [(50, 64, 64), (1000, 64, 128), (4100, 128, 64), (9000, 64, 64),
                                   (22350, 64, 64), (47300, 64, 128), (70000, 64, 64), (102380, 64, 64),
                                   (131032, 64, 64)])
def test_mask_builder_ragged_random(N, bs, d):
    # up to nB = 2048 key blocks (131032 tokens of block 64), the largest
    g = torch.Generator(device=DEV).manual_seed(N)
    qh = torch.randn(2, 3, N, d, generator=g, device=DEV).to(torch.bfloat16)
    kh = (qh.float() + 0.3 * torch.randn(2, 3, N, d, generator=g, device=DEV)).to(torch.bfloat16)
    got = P.build_block_mask(qh, kh, bs, 0.8)
    torch.cuda.synchronize()
    want, rep = oracle.build_block_mask(oracle.to_f64(qh), oracle.to_f64(kh), bs, 0.8)
    fragile = {k: rep["scores"][k] for k in rep["fragile"]}
    _assert_masks_equal(got, want, fragile, 0.8)


@pytest.mark.parametrize("nb,tau,k", [(10, 0.45, 5), (300, 0.123, 37), (1100, 0.4537, 500)])
def test_mask_builder_constant_input_ties(nb, tau, k):
    # All pooled logits equal: k = ceil(tau * nB) (tau nB not an integer), the
    # lowest blocks of every row.
    x = torch.ones(1, 1, nb * 64, 64, dtype=torch.bfloat16, device=DEV)
    got = P.build_block_mask(x, x, 64, tau).cpu().numpy()
    assert (got[0, 0] == np.array([1] * k + [0] * (nb - k), dtype=np.uint8)[None, :]).all()


# ---------------------------------------------------------------- merge, compaction

@pytest.mark.parametrize("wid", [1, 2, 4])
def test_merge_bit_exact(wid):
    wl = synth.WORKLOADS[wid]
    rows, cols, _ = synth.region_flags(wl, 0)
    m = synth.random_mask(1, 3, wl.n_blocks, 0.2, wid) * np.uint8(5)  # nonzero bytes other than 1
    got = P.merge_target_rows(torch.as_tensor(m, device=DEV), rows, cols).cpu().numpy()
    np.testing.assert_array_equal(got, oracle.merge_target_rows(m, rows, cols))


# Rows shorter than, equal to and just over the 16 bytes a thread widens (a
# thread's bytes then span several rows, heads and batch entries), with and
# without dense columns, from 16-byte aligned and unaligned mask addresses.
@pytest.mark.parametrize("nb", [1, 3, 15, 16, 17, 33, 130])
@pytest.mark.parametrize("offset", [0, 1, 7])
def test_merge_short_rows_and_unaligned(nb, offset):
    rng = np.random.default_rng(nb * 10 + offset)
    B, H = 2, 3
    m = (rng.random((B, H, nb, nb)) < 0.3).astype(np.uint8) * rng.integers(1, 255, (B, H, nb, nb), dtype=np.uint8)
    rows = (rng.random((B, nb)) < 0.2).astype(np.uint8)
    cols = (rng.random((B, nb)) < 0.2).astype(np.uint8)
    for c in (cols, None):
        buf = torch.zeros(m.size + offset + 16, dtype=torch.uint8, device=DEV)
        dm = buf[offset:offset + m.size].view(m.shape)
        dm.copy_(torch.as_tensor(m))
        P.merge_target_rows(dm, rows, c)
        np.testing.assert_array_equal(dm.cpu().numpy(), oracle.merge_target_rows(m, rows, c))
        # the bytes around the mask are untouched
        assert int(buf[:offset].sum()) == 0 and int(buf[offset + m.size:].sum()) == 0


# R = heads * nb rows in chunks of 1024: one chunk up to (931, 1); 3, 5, 10,
# 14 and 22 chunks (the last partial) keep a key's chunk counts in registers
# in the scan; (2048, 17) has 34 chunks and takes the two-pass scan.  Rows of
# 1100 key blocks span two rounds of 16-byte chunks per lane, rows of 2048
# three.
@pytest.mark.parametrize("nb,density,heads", [(3, 0.5, 5), (139, 0.3, 5), (256, 0.2, 5), (931, 0.1, 5),
                                              (1100, 0.1, 3), (2048, 0.05, 5), (2048, 0.05, 7),
                                              (931, 0.1, 24), (2048, 0.02, 17),
                                              # every row full but one: one length group in row order
                                              (64, 1.0, 3)])
def test_compaction_bit_exact(nb, density, heads):
    m = synth.random_mask(1, heads, nb, density, nb)
    m[0, 1, 0] = 0
    m[0, 2, 1] = 1
    dm = torch.as_tensor(m, device=DEV)
    rp, ci, order = P.compact_block_mask(dm)
    wrp, wci, word = oracle.compact_mask(m, group_heads=_group_heads(m))
    np.testing.assert_array_equal(rp.cpu().numpy(), wrp)
    np.testing.assert_array_equal(ci.cpu().numpy(), wci)
    np.testing.assert_array_equal(order.cpu().numpy(), word)


# The row order for the attention shapes whose K and V exceed the 256 MiB
# Infinity Cache: heads in groups (6 of 40 at 75.6K tokens, 4 of 24 at 119K),
# each group's rows longest first; from the uint8 mask, from bits and
# restricted, each equal to the oracle's; the attention's output does not
# depend on the order.
# nB = 591 and 931 take the single-pass scan (a thread per key, group totals
# in LDS), nB = 1024 and 2048 the scan through memory (more keys than
# threads; 40 chunks at (40, 1024)); (2, 20, 591) has groups of 6 heads
# across the two batch entries; (1, 5, 300) is one group; (1, 63, 2048) has
# (1, 126, 2048) the most groups an order can have, 63 of two heads (252
# chunks).
@pytest.mark.parametrize("batch,heads,nb,attn,G", [(1, 40, 591, (75600, 128, 128), 6),
                                                   (1, 24, 931, (119056, 128, 128), 4),
                                                   (2, 20, 591, (75600, 128, 128), 6),
                                                   (1, 5, 300, (38400, 128, 128), 5),
                                                   (1, 3, 2048, (262144, 128, 128), 2),
                                                   (1, 6, 2048, (262144, 128, 128), 2),
                                                   (1, 40, 1024, (131072, 128, 128), 4),
                                                   (1, 126, 2048, (262144, 128, 128), 2)])
def test_compaction_grouped_order(batch, heads, nb, attn, G):
    big = batch * heads * nb * nb > 10 ** 8
    if big:  # one head's random mask with its rows rotated per head (quick to draw)
        one = synth.random_mask(1, 1, nb, 0.15, heads)[0, 0]
        m = np.stack([np.roll(one, 37 * h, axis=0) for h in range(heads)])[None]
    else:
        m = synth.random_mask(batch, heads, nb, 0.15, heads)
    assert P.order_group_heads(batch, heads, nb, attn) == G
    rp, ci, order = P.compact_block_mask(torch.as_tensor(m, device=DEV), attn=attn)
    wrp, _, word = oracle.compact_mask(m, group_heads=G)
    np.testing.assert_array_equal(rp.cpu().numpy(), wrp)
    np.testing.assert_array_equal(order.cpu().numpy(), word)
    if big:
        return  # the bit-packed and restricted calls share the sort checked above
    bits = torch.as_tensor(oracle.pack_mask(m).view(np.int64), device=DEV)
    _, _, order_b = P.compact_block_mask_bits(bits, attn=attn)
    np.testing.assert_array_equal(order_b.cpu().numpy(), word)
    rng = np.random.default_rng(heads)
    act = (rng.random((batch, nb)) < 0.3).astype(np.uint8)
    ctx = np.maximum(act, (rng.random((batch, nb)) < 0.5).astype(np.uint8))
    _, _, order_r, n = P.compact_block_mask_bits_region(bits, act, ctx, attn=attn)
    _, _, word_r, wn = oracle.compact_restricted(m, act, ctx, group_heads=G)
    assert int(n.item()) == wn
    np.testing.assert_array_equal(order_r.cpu().numpy(), word_r)


def test_attention_independent_of_row_order():
    wl, x = _inputs(1, heads=4)
    mask = P.build_block_mask(x["q_hist"], x["k_hist"], wl.block, wl.tau)
    rp, ci, order = P.compact_block_mask(mask)
    o1 = P.block_sparse_attn_lists(x["q"], x["k"], x["v"], (rp, ci, order), wl.block)
    rev = torch.flip(order, [0]).contiguous()
    o2 = P.block_sparse_attn_lists(x["q"], x["k"], x["v"], (rp, ci, rev), wl.block)
    torch.cuda.synchronize()
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))


# ---------------------------------------------------------------- bit-packed masks

def _u64(bits: torch.Tensor) -> np.ndarray:
    return bits.cpu().numpy().view(np.uint64)


@pytest.mark.parametrize("nb,heads", [(1, 3), (3, 5), (64, 2), (139, 5), (256, 4), (931, 2), (2048, 1)])
def test_pack_unpack_bit_exact(nb, heads):
    m = synth.random_mask(2, heads, nb, 0.3, nb) * np.uint8(3)  # nonzero bytes other than 1
    bits = P.pack_block_mask(torch.as_tensor(m, device=DEV))
    np.testing.assert_array_equal(_u64(bits), oracle.pack_mask(m))
    # unpack from words whose unused high bits are set: they are ignored
    dirty = oracle.pack_mask(m)
    if nb % 64:
        dirty[..., -1] |= ~((np.uint64(1) << np.uint64(nb % 64)) - np.uint64(1))
    got = P.unpack_block_mask(torch.as_tensor(dirty.view(np.int64), device=DEV))
    np.testing.assert_array_equal(got.cpu().numpy(), oracle.unpack_mask(dirty, nb))


@pytest.mark.parametrize("wid", [0, 1, 2, 4])
def test_mask_builder_bits_bit_exact(wid):
    wl, x = _inputs(wid, heads=2 if wid else None)
    want, fragile = _oracle_mask(x, wl)
    bits = P.build_block_mask_bits(x["q_hist"], x["k_hist"], wl.block, wl.tau)
    got = oracle.unpack_mask(_u64(bits), wl.n_blocks)
    _assert_masks_equal(torch.as_tensor(got), want, fragile, wl.tau)
    # unused high bits of each row's last word are written as 0
    if wl.n_blocks % 64:
        assert not (_u64(bits)[..., -1] >> np.uint64(wl.n_blocks % 64)).any()


@pytest.mark.parametrize("nb", [3, 100, 256])
def test_mask_builder_bits_full_threshold(nb):
    x = torch.randn(1, 2, nb * 64 - 5, 64, device=DEV).to(torch.bfloat16)
    bits = P.build_block_mask_bits(x, x, 64, 1.0)
    np.testing.assert_array_equal(_u64(bits), oracle.pack_mask(np.ones((1, 2, nb, nb), dtype=np.uint8)))


# widened or not; R = B * heads * nb rows (2048 x 7 x 2: 28 chunks of the
# sort)
@pytest.mark.parametrize("nb,density,heads,widen", [(3, 0.5, 5, False), (139, 0.3, 5, True), (256, 0.2, 5, True),
                                                    (256, 0.2, 5, False), (931, 0.1, 3, True),
                                                    (2048, 0.05, 7, True), (64, 1.0, 3, False)])
def test_compaction_from_bits_bit_exact(nb, density, heads, widen):
    B = 2
    m = synth.random_mask(B, heads, nb, density, nb + 7)
    m[0, 1, 0] = 0
    rows = cols = None
    if widen:
        rng = np.random.default_rng(nb)
        rows = (rng.random((B, nb)) < 0.1).astype(np.uint8)
        cols = (rng.random((B, nb)) < 0.05).astype(np.uint8) * np.uint8(9)
    bits = oracle.pack_mask(m)
    if nb % 64:
        bits[..., -1] |= np.uint64(1) << np.uint64(63)  # an unused bit set: ignored
    dbits = torch.as_tensor(bits.view(np.int64), device=DEV)
    before = dbits.clone()
    rp, ci, order = P.compact_block_mask_bits(dbits, rows, cols)
    merged = oracle.merge_target_rows(m, rows, cols) if widen else m
    wrp, wci, word = oracle.compact_mask(merged, group_heads=_group_heads(merged))
    np.testing.assert_array_equal(rp.cpu().numpy(), wrp)
    np.testing.assert_array_equal(ci.cpu().numpy(), wci)
    np.testing.assert_array_equal(order.cpu().numpy(), word)
    assert torch.equal(dbits, before)  # the stored mask is only read


def test_mask_bank_record_and_reuse():
    # a bank of 2 steps x 2 branches x 2 layers for the tiny workload: each
    # slot recorded from its own historical Q/K, then compacted for the target
    # and walked by the attention kernel
    wl = synth.WORKLOADS[0]
    bank = P.MaskBank(2, 2, 2, 1, 2, wl.n_blocks, device=DEV)
    assert bank.nbytes == 8 * 2 * 2 * 2 * 2 * wl.n_blocks * 1
    want = {}
    for t in range(2):
        for c in range(2):
            for layer in range(2):
                seed = 100 * t + 10 * c + layer
                x = synth.attention_inputs(wl, seed=seed, device=DEV)
                bank.record(t, c, layer, x["q_hist"], x["k_hist"], wl.block, wl.tau)
                want[(t, c, layer)] = (x, _oracle_mask(x, wl))
    for (t, c, layer), (x, (m, fragile)) in want.items():
        _say("slot", t, c, layer)
        got = oracle.unpack_mask(_u64(bank.slot(t, c, layer)), wl.n_blocks)
        _assert_masks_equal(torch.as_tensor(got), m, fragile, wl.tau)
        lists = bank.lists(t, c, layer, x["row_flags"])
        merged = oracle.merge_target_rows(got, x["row_flags"].cpu().numpy())
        for g, w in zip(lists, oracle.compact_mask(merged, group_heads=_group_heads(merged))):
            np.testing.assert_array_equal(g.cpu().numpy(), w)
        o = P.block_sparse_attn_lists(x["q"], x["k"], x["v"], lists, wl.block)
        o_ref, _ = oracle.block_sparse_attention(oracle.to_f64(x["q"]), oracle.to_f64(x["k"]),
                                                 oracle.to_f64(x["v"]), merged, wl.block)
        rows = [(0, h, i) for h in range(2) for i in range(wl.n_blocks)]
        _compare_rows(o, o_ref, None, None, rows, wl.seq_len, wl.block)


# ---------------------------------------------------------------- attention

def test_attention_tiny_workload_full():
    wl, x = _inputs(0)
    want_mask, _ = _oracle_mask(x, wl)
    merged = oracle.merge_target_rows(want_mask, x["row_flags"].cpu().numpy())
    o, lse = P.block_sparse_attn(x["q"], x["k"], x["v"], torch.as_tensor(merged, device=DEV), wl.block,
                                 return_lse=True)
    torch.cuda.synchronize()
    ro, rl = oracle.block_sparse_attention(oracle.to_f64(x["q"]), oracle.to_f64(x["k"]), oracle.to_f64(x["v"]),
                                           merged, wl.block)
    rows = [(0, h, i) for h in range(wl.heads) for i in range(wl.n_blocks)]
    _compare_rows(o, ro, lse, rl, rows, wl.seq_len, wl.block)


# The 32K and CogVideoX-shaped workloads in full: every query block of every
# head, through the call and kernel the bench times (compacted lists, no LSE:
# bsattn_kernel<128, 128, false> and <64, 128, false>), with the oracle run
# one head at a time.  The heads are split over several tests so that each
# stays well inside the per-test time limit; the GPU outputs are computed
# once per workload.
_FULL = {}


def _full_workload(wid):
    if wid not in _FULL:
        _FULL.clear()
        wl, x = _inputs(wid)
        want_mask, _ = _oracle_mask(x, wl)
        cols = None if x["col_flags"] is None else x["col_flags"].cpu().numpy()
        merged = oracle.merge_target_rows(want_mask, x["row_flags"].cpu().numpy(), cols)
        dm = torch.as_tensor(merged, device=DEV)
        lists = P.compact_block_mask(dm)
        o = P.block_sparse_attn_lists(x["q"], x["k"], x["v"], lists, wl.block)
        o_lse, lse = P.block_sparse_attn(x["q"], x["k"], x["v"], dm, wl.block, return_lse=True)
        torch.cuda.synchronize()
        _say("merged density %.4f" % merged.mean())
        _FULL[wid] = (wl, x, merged, o, o_lse, lse)
    return _FULL[wid]


@pytest.mark.parametrize("wid,part,parts", [(1, 0, 2), (1, 1, 2), (2, 0, 4), (2, 1, 4), (2, 2, 4), (2, 3, 4)])
def test_attention_full_workload(wid, part, parts):
    wl, x, merged, o, o_lse, lse = _full_workload(wid)
    H, N, bs = wl.heads, wl.seq_len, wl.block
    # the LSE kernel computes the same O bit for bit
    assert torch.equal(o.view(torch.int16), o_lse.view(torch.int16))
    og = o.float().cpu().numpy()
    lg = lse.cpu().numpy().astype(np.float64)
    worst = (0.0, -1)
    dd = rr = 0.0
    for h in range(part * H // parts, (part + 1) * H // parts):
        ro, rl = oracle.block_sparse_attention(oracle.to_f64(x["q"][:, h:h + 1]), oracle.to_f64(x["k"][:, h:h + 1]),
                                               oracle.to_f64(x["v"][:, h:h + 1]), merged[:, h:h + 1], bs)
        d = og[:, h] - ro[:, 0]
        mx = float(np.abs(d).max())
        worst = max(worst, (mx, h))
        dd += float((d * d).sum())
        rr += float((ro * ro).sum())
        assert mx <= ATOL, (h, mx)
        hd = float(np.linalg.norm(d) / np.linalg.norm(ro))
        assert hd <= REL_L2, (h, hd)
        assert np.abs(lg[:, h] - rl[:, 0]).max() <= 1e-3
    rel = math.sqrt(dd / rr)
    _say("%s heads %d..%d of %d, all %d rows: worst head %d max|d| %.3e, relL2 %.3e" % (
        wl.name, part * H // parts, (part + 1) * H // parts - 1, H, wl.n_blocks, worst[1], worst[0], rel))
    assert rel <= REL_L2
    if part == parts - 1:
        _FULL.clear()


@pytest.mark.parametrize("wid", [3, 4])
def test_attention_sampled_rows(wid):
    wl, x = _inputs(wid)
    H = wl.heads
    # the oracle mask of the historical copy, widened on the host
    want_mask, _ = _oracle_mask(x, wl)
    rows_flags = x["row_flags"].cpu().numpy()
    cols = None if x["col_flags"] is None else x["col_flags"].cpu().numpy()
    merged = oracle.merge_target_rows(want_mask, rows_flags, cols)
    _say("merged density %.4f" % merged.mean())
    o, lse = P.block_sparse_attn(x["q"], x["k"], x["v"], torch.as_tensor(merged, device=DEV), wl.block,
                                 return_lse=True)
    torch.cuda.synchronize()
    rows = _sample_rows(wl, merged, rows_flags, H)
    heads = sorted({h for (_, h, _) in rows})
    o_ref = np.full(o.shape, np.nan)
    l_ref = np.full(lse.shape, np.nan)
    for h in heads:
        hr = [(b, 0, i) for (b, hh, i) in rows if hh == h]
        ro, rl = oracle.block_sparse_attention(oracle.to_f64(x["q"][:, h:h + 1]), oracle.to_f64(x["k"][:, h:h + 1]),
                                               oracle.to_f64(x["v"][:, h:h + 1]), merged[:, h:h + 1], wl.block,
                                               rows=hr)
        o_ref[:, h] = ro[:, 0]
        l_ref[:, h] = rl[:, 0]
    _compare_rows(o, o_ref, lse, l_ref, rows, wl.seq_len, wl.block)


@pytest.mark.parametrize("wid", [0, 1, 2])
def test_end_to_end_path(wid):
    """GPU builder -> GPU merge -> GPU attention against the oracle chain."""
    wl, x = _inputs(wid)
    mask = P.build_block_mask(x["q_hist"], x["k_hist"], wl.block, wl.tau)
    P.merge_target_rows(mask, x["row_flags"], x["col_flags"])
    o = P.block_sparse_attn(x["q"], x["k"], x["v"], mask, wl.block)
    torch.cuda.synchronize()
    want_mask, fragile = _oracle_mask(x, wl)
    assert not fragile
    cols = None if x["col_flags"] is None else x["col_flags"].cpu().numpy()
    merged = oracle.merge_target_rows(want_mask, x["row_flags"].cpu().numpy(), cols)
    np.testing.assert_array_equal(mask.cpu().numpy(), merged)
    rows = _sample_rows(wl, merged, x["row_flags"].cpu().numpy(), min(wl.heads, 2), n_random=8)
    ro, rl = oracle.block_sparse_attention(oracle.to_f64(x["q"][:, :2]), oracle.to_f64(x["k"][:, :2]),
                                           oracle.to_f64(x["v"][:, :2]), merged[:, :2], wl.block,
                                           rows=[r for r in rows if r[1] < 2])
    _compare_rows(o, ro, None, None, [r for r in rows if r[1] < 2], wl.seq_len, wl.block)


@pytest.mark.parametrize("wid", [0, 1, 2])
def test_attention_from_lists_matches_mask_call(wid):
    """carnator_block_sparse_attn_lists on the lists of carnator_compact_block_mask
    runs the same kernel as carnator_block_sparse_attn: bit-identical O and LSE."""
    wl, x = _inputs(wid)
    mask = P.build_block_mask(x["q_hist"], x["k_hist"], wl.block, wl.tau)
    P.merge_target_rows(mask, x["row_flags"], x["col_flags"])
    o1, l1 = P.block_sparse_attn(x["q"], x["k"], x["v"], mask, wl.block, return_lse=True)
    lists = P.compact_block_mask(mask, trim=False)
    o2, l2 = P.block_sparse_attn_lists(x["q"], x["k"], x["v"], lists, wl.block, return_lse=True)
    o3 = P.block_sparse_attn_lists(x["q"], x["k"], x["v"], lists, wl.block)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(o1, o3)
    assert torch.equal(l1, l2)


@pytest.mark.parametrize("N,bs,d", [(50, 64, 64), (64, 64, 128), (200, 128, 64), (333, 64, 128),
                                    (1000, 128, 128), (2048, 64, 64)])
def test_attention_ragged_shapes_and_dims(N, bs, d):
    g = torch.Generator(device=DEV).manual_seed(7 + N)
    q, k, v = (torch.randn(2, 2, N, d, generator=g, device=DEV).to(torch.bfloat16) for _ in range(3))
    nb = -(-N // bs)
    m = synth.random_mask(2, 2, nb, 0.5, N)
    m[..., -1] = 1  # the partial tail block is visited by every row
    o, lse = P.block_sparse_attn(q, k, v, torch.as_tensor(m, device=DEV), bs, return_lse=True)
    o_plain = P.block_sparse_attn(q, k, v, torch.as_tensor(m, device=DEV), bs)
    torch.cuda.synchronize()
    ro, rl = oracle.block_sparse_attention(oracle.to_f64(q), oracle.to_f64(k), oracle.to_f64(v), m, bs)
    rows = [(b, h, i) for b in range(2) for h in range(2) for i in range(nb)]
    _compare_rows(o, ro, lse, rl, rows, N, bs)
    # the kernel without the LSE (its own code object for every (d, block))
    _compare_rows(o_plain, ro, None, None, rows, N, bs)
    assert torch.equal(o.view(torch.int16), o_plain.view(torch.int16))


@pytest.mark.parametrize("N,bs,d", [(131035, 64, 64), (262100, 128, 128)])
def test_attention_longest_lists(N, bs, d):
    # nB = 2048, the largest number of key blocks: rows 0, 5 and the last keep
    # every key block (the longest list a row can have, the ragged tail
    # included); the others about 5 % of them
    g = torch.Generator(device=DEV).manual_seed(N)
    q, k, v = (torch.randn(1, 1, N, d, generator=g, device=DEV).to(torch.bfloat16) for _ in range(3))
    nb = -(-N // bs)
    assert nb == 2048
    m = synth.random_mask(1, 1, nb, 0.05, 5)
    m[0, 0, [0, 5, nb - 1]] = 1
    o, lse = P.block_sparse_attn(q, k, v, torch.as_tensor(m, device=DEV), bs, return_lse=True)
    o_plain = P.block_sparse_attn(q, k, v, torch.as_tensor(m, device=DEV), bs)
    torch.cuda.synchronize()
    rows = [(0, 0, i) for i in (0, 5, 700, 1500, nb - 1)]
    ro, rl = oracle.block_sparse_attention(oracle.to_f64(q), oracle.to_f64(k), oracle.to_f64(v), m, bs,
                                           rows=rows)
    _compare_rows(o, ro, lse, rl, rows, N, bs)
    _compare_rows(o_plain, ro, None, None, rows, N, bs)


def test_attention_empty_rows_and_explicit_scale():
    N, bs, d = 512, 128, 128
    g = torch.Generator(device=DEV).manual_seed(11)
    q, k, v = (torch.randn(1, 2, N, d, generator=g, device=DEV).to(torch.bfloat16) for _ in range(3))
    m = synth.random_mask(1, 2, 4, 0.5, 11)
    m[0, 0, 2] = 0  # no kept block: zeros and -inf
    m[0, 1, 0] = 0
    m[0, 1, 3, :] = 1
    o, lse = P.block_sparse_attn(q, k, v, torch.as_tensor(m, device=DEV), bs, scale=0.2, return_lse=True)
    torch.cuda.synchronize()
    assert (o[0, 0, 256:384] == 0).all() and torch.isneginf(lse[0, 0, 256:384]).all()
    ro, rl = oracle.block_sparse_attention(oracle.to_f64(q), oracle.to_f64(k), oracle.to_f64(v), m, bs, scale=0.2)
    _compare_rows(o, ro, lse, rl, [(0, h, i) for h in range(2) for i in range(4)], N, bs)


def test_attention_strided_views():
    # Q, K, V as [B, N, H, d] storage viewed as [B, H, N, d]; O into a strided view.
    N, bs, d, H = 300, 64, 64, 3
    g = torch.Generator(device=DEV).manual_seed(5)
    base = [torch.randn(1, N, H, d, generator=g, device=DEV).to(torch.bfloat16) for _ in range(3)]
    q, k, v = (t.permute(0, 2, 1, 3) for t in base)
    nb = -(-N // bs)
    m = synth.random_mask(1, H, nb, 0.6, 5)
    m[..., 0] = 1
    out_store = torch.zeros(1, N, H, d, dtype=torch.bfloat16, device=DEV)
    out = out_store.permute(0, 2, 1, 3)
    P.block_sparse_attn(q, k, v, torch.as_tensor(m, device=DEV), bs, out=out)
    torch.cuda.synchronize()
    ro, _ = oracle.block_sparse_attention(oracle.to_f64(q), oracle.to_f64(k), oracle.to_f64(v), m, bs)
    _compare_rows(out, ro, None, None, [(0, h, i) for h in range(H) for i in range(nb)], N, bs)


def test_attention_full_mask_matches_dense_reference():
    # All rows target-specific: the sparse path reduces to dense attention.
    N, bs, d = 640, 128, 128
    g = torch.Generator(device=DEV).manual_seed(3)
    q, k, v = (torch.randn(1, 2, N, d, generator=g, device=DEV).to(torch.bfloat16) for _ in range(3))
    m = np.zeros((1, 2, 5, 5), np.uint8)
    merged = P.merge_target_rows(torch.as_tensor(m, device=DEV), np.ones((1, 5), np.uint8))
    o = P.block_sparse_attn(q, k, v, merged, bs)
    ref = torch.nn.functional.scaled_dot_product_attention(q.double().cpu(), k.double().cpu(), v.double().cpu())
    d_ = (o.double().cpu() - ref)
    assert d_.abs().max().item() <= ATOL
    assert (d_.norm() / ref.norm()).item() <= REL_L2


def test_deterministic_repeat():
    wl, x = _inputs(1, heads=2)
    m1 = P.build_block_mask(x["q_hist"], x["k_hist"], wl.block, wl.tau)
    m2 = P.build_block_mask(x["q_hist"], x["k_hist"], wl.block, wl.tau)
    assert torch.equal(m1, m2)
    P.merge_target_rows(m1, x["row_flags"])
    o1 = P.block_sparse_attn(x["q"], x["k"], x["v"], m1, wl.block)
    o2 = P.block_sparse_attn(x["q"], x["k"], x["v"], m1, wl.block)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))


# ---------------------------------------------------------------- signature scan

def _check_topk(idx, sim, q, bank, k):
    wi, wv, frag = oracle.topk_cosine(q, bank, k)
    gi = idx.cpu().numpy()
    gv = sim.cpu().numpy().astype(np.float64)
    for r in range(q.shape[0]):
        if frag[r]:
            assert set(gi[r]) == set(wi[r])
        else:
            assert gi[r].tolist() == wi[r].tolist()
        assert np.abs(gv[r] - wv[r]).max() <= 1e-6


def test_signature_bank_workload():
    sig = synth.signature_inputs(device=DEV)
    q, b = sig["query"], sig["bank"]
    idx, sim, allsim = P.signature_sim(q, b, synth.SIG_TOPK, return_all=True)
    torch.cuda.synchronize()
    qn, bn = q.cpu().numpy(), b.cpu().numpy()
    _check_topk(idx, sim, qn, bn, synth.SIG_TOPK)
    assert int(idx[1, 0]) == sig["planted"]
    ref = oracle.cosine_similarity(qn, bn)
    assert np.abs(allsim.cpu().numpy() - ref).max() <= 1e-6


@pytest.mark.parametrize("m,dim,ld,nq,k", [
    (1, 4, 4, 1, 1), (100, 64, 72, 6, 64), (5000, 256, 256, 3, 17),
    # every row in registers, candidate filter with k = 16, queries in passes of 4 + 1
    (8192, 64, 64, 5, 16),
    # more rows than the top-k keeps in registers
    (9000, 128, 132, 2, 8),
    # query rows too long to stage in LDS
    (300, 40000, 40000, 2, 5)])
def test_signature_shapes(m, dim, ld, nq, k):
    g = torch.Generator(device=DEV).manual_seed(m)
    bank_store = torch.randn(m, ld, generator=g, device=DEV)
    bank = bank_store[:, :dim]
    q = torch.randn(nq, dim, generator=g, device=DEV)
    if m > 1:
        bank_store[min(3, m - 1)] = 0.0  # zero-norm row scores 0
    idx, sim = P.signature_sim(q, bank, k)
    torch.cuda.synchronize()
    _check_topk(idx, sim, q.cpu().numpy(), bank.cpu().numpy(), k)


@pytest.mark.parametrize("n_top,n_tied,k", [(3, 10, 8), (0, 30, 20), (3, 61, 50), (5, 2, 6), (1, 1, 2)])
def test_signature_tie_band_among_few_candidates(n_top, n_tied, k):
    # Unit vectors in a plane: n_top rows at cosine 1, n_tied rows a few 1e-9
    # apart around cosine 0.999 (one tie band), every other row at cosine
    # <= 0.71.  The cut falls inside the band, so the rule keeps its lowest
    # rows; the candidates stay few, which is the single-wave selection.
    m = 5000
    rng = np.random.default_rng(1000 * n_top + n_tied)
    theta = rng.uniform(np.pi / 4, 2 * np.pi - np.pi / 4, m)
    rows = rng.choice(m, n_top + n_tied, replace=False)
    theta[rows[:n_top]] = 0.0
    theta[rows[n_top:]] = 0.0447 + 1e-7 * rng.random(n_tied)
    bank = np.zeros((m, 4), np.float32)
    bank[:, 0] = np.cos(theta)
    bank[:, 1] = np.sin(theta)
    q = np.array([[1.0, 0.0, 0.0, 0.0]], np.float32)
    idx, sim = P.signature_sim(torch.as_tensor(q, device=DEV), torch.as_tensor(bank, device=DEV), k)
    torch.cuda.synchronize()
    _check_topk(idx, sim, q, bank, k)
    wi, _, _ = oracle.topk_cosine(q, bank, k)
    assert idx[0].tolist() == wi[0].tolist()


@pytest.mark.parametrize("m", [10, 3000, 9000])
def test_signature_ties_lower_row(m):
    # Row 7 is parallel to the query (cosine 1); the others sit 5e-11 below.
    # Within 1e-6 of the cut every row is tied, so the three lowest rows win.
    bank = torch.zeros(m, 8, device=DEV)
    bank[:, 0] = 1.0
    bank[7, 1] = 1e-5
    q = torch.zeros(1, 8, device=DEV)
    q[0, 0] = 1.0
    q[0, 1] = 1e-5
    idx, sim = P.signature_sim(q, bank, 3)
    assert idx[0].tolist() == [0, 1, 2]
    wi, _, _ = oracle.topk_cosine(q.cpu().numpy(), bank.cpu().numpy(), 3)
    assert wi[0].tolist() == [0, 1, 2]
