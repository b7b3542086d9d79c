"""Benchmark of the whole cache-hit block-sparse attention path on one MI355X.

One step = the four rows of the path on one batch of synthetic input that is
already resident in HBM:
  1. historical block mask from pooled Q_hist.K_hist (carnator_build_block_mask)
  2. target-row widening (carnator_merge_target_rows)
  3. block-sparse attention of the target Q, K, V: the mask compacted into
     per-row block lists (carnator_compact_block_mask), then the attention
     kernel from those lists (carnator_block_sparse_attn_lists; the same two
     steps carnator_block_sparse_attn runs in one call)
  4. Early-Signature cosine top-k against the 4096 x 3072 bank
     (carnator_signature_sim)
Three input sets are rotated so the 256 MB Infinity Cache does not serve
repeated reads of the HBM-bound steps.

Prints one JSON line.  ``value`` is executed attention TFLOP per step divided
by the step time (whole-job throughput); ``roofline`` describes the attention
kernel (one launch, timed with events on its stream) against the bf16 MFMA
peak.  ``roofline.traffic`` is the kernel's HBM traffic per launch from
rocprofv3 FETCH_SIZE / WRITE_SIZE passes, scaled by the same counters on a
copy of known size (paper_2609_32420_amd/measured_traffic.json); it is null
when the kernel source no longer matches the one those counters were taken
on.

``region_restricted`` (after the timed region, skipped with --no-region):
the middle-layer variant -- regions and blend weight from an evidence
region, the latent blend (HBM-bound; its GB/s against the 8 TB/s peak),
block flags, compaction restricted to active rows and context keys, and
the attention of the active rows only -- each timed alone.

After the timed steps the attention is also timed with its compaction, as
one mask-in call (``attn_with_compaction_ms_per_call``); the timed steps'
attention launches give ``attn_ms_p10_p50_p90``.

``exact_mass`` (after the timed region, skipped with --no-exact): the
builder on the token-level attention mass -- the dense mass pass against
the bf16 MFMA peak and the selection on its masses -- with the exact masks
compared to the pooled ones.

``mask_bank`` (after the timed region, skipped with --no-bank): the same
masks in their stored, bit-packed form -- the builder writing a bank slot
directly, compaction of a slot with the widening applied while reading, and
packing a uint8 mask -- each timed alone, with a check that the lists equal
those of the uint8 path.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "block-sparse attn ms/call + executed TFLOP/s (% bf16 MFMA peak) at 32K tokens"
PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 4096 FLOP/clk x 2.4 GHz (dense)
PEAK_HBM_GBPS = 8000.0


def executed_flops(mask: np.ndarray, N: int, bs: int, d: int) -> float:
    """sum over kept (b,h,i,j) of 4 d n_i n_j (QK^T and PV, valid tokens only)."""
    nb = mask.shape[-1]
    n = np.full(nb, bs, dtype=np.float64)
    n[-1] = N - (nb - 1) * bs
    kept = (mask != 0).astype(np.float64)
    return float(4.0 * d * np.einsum("bhij,i,j->", kept, n, n))


def dense_flops(B, H, N, d) -> float:
    return 4.0 * d * B * H * float(N) * float(N)


TRAFFIC_FILE = os.path.join(ROOT, "paper_2609_32420_amd", "measured_traffic.json")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2609_32420_amd", "csrc", "attn_kernels.hip")


def measured_traffic(d: int, bs: int):
    """HBM bytes per launch of the attention kernel from the recorded
    FETCH_SIZE / WRITE_SIZE passes, or None when there is no record for this
    configuration or the kernel source changed since it was taken."""
    import hashlib
    try:
        rec = json.load(open(TRAFFIC_FILE))
        src = hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256") != src or rec.get("head_dim") != d or rec.get("block") != bs:
        return None
    return rec.get("bytes_per_launch")


def cpu_baseline(wl, heads: int = 8):
    """The oracle, as it stands, on a bounded sample: every step of the path
    for ``heads`` heads of the workload (mask, widening, attention of all
    query blocks of those heads) plus the full signature scan."""
    import oracle
    import synth
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas = 1
    x = synth.attention_inputs(wl, seed=0, device="cpu", heads=heads)
    sig = synth.signature_inputs()
    t0 = time.perf_counter()
    m, _ = oracle.build_block_mask(oracle.to_f64(x["q_hist"]), oracle.to_f64(x["k_hist"]), wl.block, wl.tau)
    cols = None if x["col_flags"] is None else x["col_flags"].numpy()
    merged = oracle.merge_target_rows(m, x["row_flags"].numpy(), cols)
    oracle.block_sparse_attention(oracle.to_f64(x["q"]), oracle.to_f64(x["k"]), oracle.to_f64(x["v"]), merged,
                                  wl.block)
    oracle.topk_cosine(sig["query"].numpy(), sig["bank"].numpy(), 8)
    dt = time.perf_counter() - t0
    fl = executed_flops(merged, wl.seq_len, wl.block, wl.head_dim)
    return {"value": fl / dt / 1e12, "unit": "TFLOP/s", "cores": blas, "kind": "oracle",
            "host_cpus": len(os.sched_getaffinity(0)), "seconds": dt,
            "sample": "%d of %d heads of %s, full path (mask, widening, attention of all %d query blocks) "
                      "+ 1 signature scan" % (heads, wl.heads, wl.name, wl.n_blocks)}


# a request's stored connectivity: denoising steps x guidance branches x layers
BANK_SLOTS = (50, 2, 30)


def bank_pass(P, torch, stream, sets, flags, masks, lists, ws_mask, wl, steps):
    """The bit-packed mask bank on the same inputs, outside the timed region:
    the builder writing a bank slot directly, compaction of that slot for the
    target (widening applied while reading the bits), and packing a uint8
    mask.  Each call is timed alone between two events; the lists must equal
    those of the uint8 path on the same masks."""
    B, H, nb = wl.batch, wl.heads, wl.n_blocks
    dev = masks[0].device
    slots = [torch.empty(B, H, nb, P.mask_words(nb), dtype=torch.int64, device=dev) for _ in sets]
    packed = torch.empty_like(slots[0])
    ws_cb = P.compact_block_mask_bits_workspace(slots[0])
    R = B * H * nb
    lb = (torch.empty(R + 1, dtype=torch.int32, device=dev), torch.empty(R * nb, dtype=torch.int32, device=dev),
          torch.empty(R, dtype=torch.int32, device=dev))
    t = {k: [] for k in ("build_bits", "compact_bits", "pack")}
    same = True
    for i in range(steps + 1):
        si = i % len(sets)
        x = sets[si][0]
        e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
        e[0].record(stream)
        P.build_block_mask_bits(x["q_hist"], x["k_hist"], wl.block, wl.tau, out=slots[si], workspace=ws_mask)
        e[1].record(stream)
        P.compact_block_mask_bits(slots[si], flags[si][0], flags[si][1], trim=False, out=lb, workspace=ws_cb,
                                  attn=(wl.seq_len, wl.head_dim, wl.block))
        e[2].record(stream)
        P.pack_block_mask(masks[si], out=packed)
        e[3].record(stream)
        if i == 0:
            continue  # warm-up
        for k, (a, b) in zip(t, ((0, 1), (1, 2), (2, 3))):
            t[k].append((e[a], e[b]))
        if i <= len(sets):
            # masks[si] holds the widened uint8 mask of this set and `lists`
            # its compaction from the last step of the per-call pass
            P.compact_block_mask(masks[si], trim=False, out=lists, attn=(wl.seq_len, wl.head_dim, wl.block))
            nnz = int(lists[0][-1].item())
            same &= bool(torch.equal(lists[0], lb[0]) and torch.equal(lists[2], lb[2])
                         and torch.equal(lists[1][:nnz], lb[1][:nnz]))
    torch.cuda.synchronize()
    ms = {k: float(np.mean([a.elapsed_time(b) for a, b in v])) for k, v in t.items()}
    slot_bytes = slots[0].numel() * 8
    return {
        "layout": "uint64 [B, H, nB, ceil(nB/64)] per (step, branch, layer)",
        "slot_bytes": slot_bytes,
        "slot_bytes_uint8": B * H * nb * nb,
        "request_bank_MB": round(slot_bytes * int(np.prod(BANK_SLOTS)) / 1e6, 1),
        "request_bank_slots": list(BANK_SLOTS),
        "build_bits_ms_per_call": round(ms["build_bits"], 4),
        "compact_bits_ms_per_call": round(ms["compact_bits"], 4),
        "pack_ms_per_call": round(ms["pack"], 4),
        "lists_equal_uint8_path": same,
    }


LATENT_CHANNELS, LATENT_PATCH = 16, (1, 2, 2)


def exact_mass_pass(P, torch, stream, sets, wl, steps):
    """The exact-mass builder on the same historical Q/K, after the timed
    region: token-level block masses (one dense bf16 QK^T pass and the
    reduction) and the selection on them, each call timed alone; the mass
    pass against the bf16 MFMA peak (dense QK^T FLOPs 2 d N^2 per head); the
    exact masks compared with the pooled ones of the same sets (before
    widening)."""
    B, H, N, d, bs, nb = wl.batch, wl.heads, wl.seq_len, wl.head_dim, wl.block, wl.n_blocks
    dev = sets[0][0]["q"].device
    mass = torch.empty(B, H, nb, nb, dtype=torch.float64, device=dev)
    ws = torch.empty(P.lib().carnator_block_mass_exact_workspace_size(ctypes_shape(P, wl)), dtype=torch.uint8,
                     device=dev)
    mask = torch.empty(B, H, nb, nb, dtype=torch.uint8, device=dev)
    t_mass, t_sel = [], []
    agree = []
    for i in range(steps + 1):
        si = i % len(sets)
        x = sets[si][0]
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record(stream)
        P.block_mass_exact(x["q_hist"], x["k_hist"], bs, out=mass, workspace=ws)
        e[1].record(stream)
        P.select_block_mask(mass, wl.tau, out=mask)
        e[2].record(stream)
        if i == 0:
            continue
        t_mass.append((e[0], e[1]))
        t_sel.append((e[1], e[2]))
        if i <= len(sets):
            pooled = P.build_block_mask(x["q_hist"], x["k_hist"], bs, wl.tau)
            inter = int((pooled & mask).sum().item())
            union = int((pooled | mask).sum().item())
            agree.append((float(mask.float().mean().item()), float(pooled.float().mean().item()),
                          inter / max(union, 1)))
    torch.cuda.synchronize()
    ms_mass = float(np.mean([a.elapsed_time(b) for a, b in t_mass]))
    ms_sel = float(np.mean([a.elapsed_time(b) for a, b in t_sel]))
    flops = 2.0 * d * float(N) * float(N) * B * H
    return {
        "mass_ms_per_call": round(ms_mass, 4),
        "mass_qk_tflop": round(flops / 1e12, 4),
        "mass_tflops": round(flops / (ms_mass * 1e-3) / 1e12, 2),
        "mass_pct_bf16_peak": round(100.0 * flops / (ms_mass * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2),
        "select_ms_per_call": round(ms_sel, 4),
        "workspace_GB": round(ws.numel() / 1e9, 3),
        "density_exact": [round(a[0], 4) for a in agree],
        "density_pooled": [round(a[1], 4) for a in agree],
        "jaccard_exact_pooled": [round(a[2], 4) for a in agree],
    }


def workload_pass(P, torch, stream, wids, steps):
    """The other workload shapes of the paper's backbones (CogVideoX-5B 17.8K
    tokens at d = 64, Wan2.1-14B 75.6K, HunyuanVideo 119K), measured in the
    same run after the timed region: one input set each (its historical Q/K
    alone exceed the 256 MB Infinity Cache, so the builder reads HBM), every
    call timed alone between two events, the attention from the lists (the
    kernel the headline times) against the bf16 peak on executed FLOPs."""
    import synth
    out = {}
    dev = torch.device("cuda:0")
    for wid in wids:
        wl = synth.WORKLOADS[wid]
        B, H, N, d, bs, nb = wl.batch, wl.heads, wl.seq_len, wl.head_dim, wl.block, wl.n_blocks
        print("bench: workload %s" % wl.name, file=sys.stderr, flush=True)
        x = synth.attention_inputs(wl, seed=0, device=dev)
        mask = torch.empty(B, H, nb, nb, dtype=torch.uint8, device=dev)
        ws_mask = P.build_block_mask_workspace(x["q_hist"], bs)
        ws_cmp = P.compact_block_mask_workspace(mask)
        R = B * H * nb
        lists = (torch.empty(R + 1, dtype=torch.int32, device=dev), torch.empty(R * nb, dtype=torch.int32, device=dev),
                 torch.empty(R, dtype=torch.int32, device=dev))
        o = torch.empty_like(x["q"])
        rows = x["row_flags"].contiguous()
        cols = None if x["col_flags"] is None else x["col_flags"].contiguous()
        t = {k: [] for k in ("build", "merge", "compact", "attn")}
        for i in range(steps + 1):
            e = [torch.cuda.Event(enable_timing=True) for _ in range(8)]
            e[0].record(stream)
            P.build_block_mask(x["q_hist"], x["k_hist"], bs, wl.tau, out=mask, workspace=ws_mask)
            e[1].record(stream)
            e[2].record(stream)
            P.merge_target_rows(mask, rows, cols)
            e[3].record(stream)
            e[4].record(stream)
            P.compact_block_mask(mask, trim=False, out=lists, workspace=ws_cmp, attn=(N, d, bs))
            e[5].record(stream)
            e[6].record(stream)
            P.block_sparse_attn_lists(x["q"], x["k"], x["v"], lists, bs, out=o)
            e[7].record(stream)
            if i > 0:
                for k_, (a_, b_) in zip(("build", "merge", "compact", "attn"), ((0, 1), (2, 3), (4, 5), (6, 7))):
                    t[k_].append((e[a_], e[b_]))
        torch.cuda.synchronize()
        ms = {k: float(np.median([a.elapsed_time(b) for a, b in v])) for k, v in t.items()}
        fl = executed_flops(mask.cpu().numpy(), N, bs, d)
        tf = fl / (ms["attn"] * 1e-3) / 1e12
        bbytes = 2.0 * B * H * N * d * 2 + B * H * nb * nb
        out[wl.name] = {
            "heads": H, "seq_len": N, "head_dim": d, "block": bs, "mask_density": round(float(mask.float().mean().item()), 4),
            "attn_ms_per_call": round(ms["attn"], 4), "attn_executed_tflop": round(fl / 1e12, 4),
            "attn_executed_tflops": round(tf, 2), "attn_frac_bf16_peak": round(tf / PEAK_BF16_TFLOPS, 4),
            "attn_dense_equiv_tflops": round(dense_flops(B, H, N, d) / (ms["attn"] * 1e-3) / 1e12, 2),
            "builder_ms_per_call": round(ms["build"], 4), "builder_GBps": round(bbytes / (ms["build"] * 1e-3) / 1e9, 1),
            "builder_pct_hbm_peak": round(100.0 * bbytes / (ms["build"] * 1e-3) / 1e9 / PEAK_HBM_GBPS, 2),
            "merge_ms_per_call": round(ms["merge"], 4), "compact_ms_per_call": round(ms["compact"], 4),
            "timing": "median of %d calls, each alone between two events" % steps,
        }
        del x, mask, ws_mask, ws_cmp, lists, o
        torch.cuda.empty_cache()
    return out


def ctypes_shape(P, wl):
    import ctypes
    return ctypes.byref(P.Shape(wl.batch, wl.heads, wl.seq_len, wl.head_dim, wl.block))


def region_pass(P, torch, stream, sets, wl, steps):
    """The region-restricted middle-layer path on the same inputs, after the
    timed region: regions and W from a seeded evidence region, the latent
    blend over a 16-channel latent twice as fine as the token grid in H and
    W, block flags, compaction of the stored mask restricted to active rows
    and context keys, and the attention of the active rows only.  Each call
    timed alone between two events."""
    import synth
    B, H, nb, N, d, bs = wl.batch, wl.heads, wl.n_blocks, wl.seq_len, wl.head_dim, wl.block
    dev = sets[0][0]["q"].device
    ev = [torch.as_tensor(synth.evidence_region(wl, seed=i), device=dev) for i in range(len(sets))]
    zs = [synth.latents(wl, LATENT_CHANNELS, LATENT_PATCH, seed=i, device=dev) for i in range(len(sets))]
    zout = torch.empty_like(zs[0][0])
    T, Hg, Wg = wl.grid
    region = (torch.empty(B, T, Hg, Wg, dtype=torch.uint8, device=dev),
              torch.empty(B, T, Hg, Wg, dtype=torch.float32, device=dev))
    ws_reg = torch.empty(max(P.lib().carnator_region_weights_workspace_size(B, T, Hg, Wg), 1), dtype=torch.uint8,
                         device=dev)
    flags = (torch.empty(B, nb, dtype=torch.uint8, device=dev), torch.empty(B, nb, dtype=torch.uint8, device=dev))
    slots = [P.build_block_mask_bits(x["q_hist"], x["k_hist"], bs, wl.tau) for x, _ in sets]
    ws_cb = P.compact_block_mask_bits_workspace(slots[0])
    R = B * H * nb
    lists = (torch.empty(R + 1, dtype=torch.int32, device=dev), torch.empty(R * nb, dtype=torch.int32, device=dev),
             torch.empty(R, dtype=torch.int32, device=dev), torch.empty(1, dtype=torch.int32, device=dev))
    outs = [torch.empty(B, H, N, d, dtype=torch.bfloat16, device=dev) for _ in sets]
    names = ("regions", "fusion", "flags", "compact", "attn")
    t = {k: [] for k in names}
    used = []
    for i in range(steps + 1):
        si = i % len(sets)
        x = sets[si][0]
        e = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
        e[0].record(stream)
        P.region_weights(ev[si], 2, 3, out=region, workspace=ws_reg)
        e[1].record(stream)
        P.latent_fusion(zs[si][0], zs[si][1], region[1], out=zout)
        e[2].record(stream)
        P.region_block_flags(region[0], wl.n_text, bs, out=flags)
        e[3].record(stream)
        P.compact_block_mask_bits_region(slots[si], flags[0], flags[1], out=lists, workspace=ws_cb,
                                         attn=(wl.seq_len, wl.head_dim, bs))
        e[4].record(stream)
        P.block_sparse_attn_lists(x["q"], x["k"], x["v"], lists[:3], bs, out=outs[si], n_rows=lists[3])
        e[5].record(stream)
        if i == 0:
            continue
        used.append(si)
        for k, a in zip(names, range(5)):
            t[k].append((e[a], e[a + 1]))
    torch.cuda.synchronize()
    ms = {k: [a.elapsed_time(b) for a, b in v] for k, v in t.items()}
    # executed attention work of each set's restricted mask (untimed)
    shifts = torch.arange(64, device=dev, dtype=torch.int64)
    per_set = []
    for si in range(len(sets)):
        P.region_weights(ev[si], 2, 3, out=region, workspace=ws_reg)
        P.region_block_flags(region[0], wl.n_text, bs, out=flags)
        m = ((slots[si][..., :, None] >> shifts) & 1).reshape(B, H, nb, -1)[..., :nb].bool()
        m &= flags[0].bool()[:, None, :, None] & flags[1].bool()[:, None, None, :]
        per_set.append({"flops": executed_flops(m.to(torch.uint8).cpu().numpy(), N, bs, d),
                        "active_q": int(flags[0].sum().item()), "context_k": int(flags[1].sum().item()),
                        "evidence": float(ev[si].float().mean().item())})
    fl_total = sum(per_set[si]["flops"] for si in used)
    attn_s = sum(ms["attn"]) * 1e-3
    ms = {k: float(np.mean(v)) for k, v in ms.items()}
    zbytes = 3.0 * zs[0][0].numel() * 4 + region[1].numel() * 4
    return {
        "evidence_fraction": [round(p_["evidence"], 4) for p_ in per_set],
        "active_query_blocks": [p_["active_q"] for p_ in per_set],
        "context_key_blocks": [p_["context_k"] for p_ in per_set],
        "n_blocks": nb, "heads": H,
        "latent": [B, LATENT_CHANNELS, T * LATENT_PATCH[0], Hg * LATENT_PATCH[1], Wg * LATENT_PATCH[2]],
        "regions_ms_per_call": round(ms["regions"], 4),
        "fusion_ms_per_call": round(ms["fusion"], 4),
        "fusion_GBps": round(zbytes / (ms["fusion"] * 1e-3) / 1e9, 1),
        "fusion_pct_hbm_peak": round(100.0 * zbytes / (ms["fusion"] * 1e-3) / 1e9 / PEAK_HBM_GBPS, 2),
        "flags_ms_per_call": round(ms["flags"], 4),
        "compact_ms_per_call": round(ms["compact"], 4),
        "attn_rows_ms_per_call": round(ms["attn"], 4),
        "attn_rows_executed_tflop_per_call": round(fl_total / len(used) / 1e12, 4),
        "attn_rows_executed_tflops": round(fl_total / attn_s / 1e12, 2),
    }


def dense_reference(P, torch, wl, steps):
    """The attention kernel under an all-ones block mask beside torch's own
    scaled_dot_product_attention (flash and memory-efficient backends) on the
    same random bf16 Q, K, V of the workload's shape: dense attention, the
    same FLOPs for both, events around each call.  One JSON line."""
    from torch.nn.attention import SDPBackend, sdpa_kernel
    dev = torch.device("cuda:0")
    B, H, N, d, bs, nb = wl.batch, wl.heads, wl.seq_len, wl.head_dim, wl.block, wl.n_blocks
    gen = torch.Generator(device=dev).manual_seed(0)
    q, k, v = (torch.randn(B, H, N, d, device=dev, dtype=torch.bfloat16, generator=gen) for _ in range(3))
    mask = torch.ones(B, H, nb, nb, dtype=torch.uint8, device=dev)
    lists = P.compact_block_mask(mask, attn=(N, d, bs))
    out = torch.empty_like(q)
    flops = dense_flops(B, H, N, d)

    def timed(f):
        for _ in range(3):
            f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ts = []
        for _ in range(steps):
            e0.record()
            f()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return sorted(ts)[len(ts) // 2]

    res = {"metric": "dense attention ms/call and TFLOP/s, all-ones block mask against torch SDPA",
           "config": {"workload": wl.name, "batch": B, "heads": H, "seq_len": N, "head_dim": d, "block": bs},
           "dense_tflop": round(flops / 1e12, 4), "peak_bf16_tflops": PEAK_BF16_TFLOPS}
    ms = timed(lambda: P.block_sparse_attn_lists(q, k, v, lists, bs, out=out))
    res["carnator_ms"] = round(ms, 4)
    res["carnator_tflops"] = round(flops / ms / 1e9, 1)
    for name, be in (("flash", SDPBackend.FLASH_ATTENTION), ("efficient", SDPBackend.EFFICIENT_ATTENTION)):
        try:
            with sdpa_kernel(be):
                ms = timed(lambda: torch.nn.functional.scaled_dot_product_attention(q, k, v))
                ref = torch.nn.functional.scaled_dot_product_attention(q, k, v)
            torch.cuda.synchronize()
            res["sdpa_%s_ms" % name] = round(ms, 4)
            res["sdpa_%s_tflops" % name] = round(flops / ms / 1e9, 1)
            res["sdpa_%s_max_abs_diff" % name] = float((ref.float() - out.float()).abs().max().item())
        except RuntimeError as e:  # the backend is not built for this device or shape
            res["sdpa_%s" % name] = "unavailable: %s" % str(e)[:120]
    print(json.dumps(res), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=1)
    ap.add_argument("--sets", type=int, default=3, help="input sets rotated across steps")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-bank", action="store_true", help="skip the bit-packed mask bank pass")
    ap.add_argument("--no-region", action="store_true", help="skip the region-restricted pass")
    ap.add_argument("--no-exact", action="store_true", help="skip the exact-mass builder pass")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the pass over the 17.8K, 75.6K and 119K-token workload shapes")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="before timing, copy a buffer of this size once (a reference kernel of known "
                         "traffic for hardware byte counters)")
    ap.add_argument("--dense-reference", action="store_true",
                    help="only time the kernel under an all-ones mask beside torch SDPA (one JSON line)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(the attention, mask and scan shard by head / bank rows with no exchange inside "
              "an operator; see the design notes).", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2609_32420_amd as P
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    wl = synth.WORKLOADS[args.workload]
    if args.dense_reference:
        dense_reference(P, torch, wl, max(args.steps, 5))
        return
    B, H, N, d, bs, nb = wl.batch, wl.heads, wl.seq_len, wl.head_dim, wl.block, wl.n_blocks
    print("bench: generating %d input sets of %s" % (args.sets, wl.name), file=sys.stderr, flush=True)
    sets = []
    for sidx in range(args.sets):
        x = synth.attention_inputs(wl, seed=sidx, device=dev)
        sg = synth.signature_inputs(seed=sidx, device=dev)
        sets.append((x, sg))
    stream = torch.cuda.current_stream(dev)
    # persistent outputs and workspaces: nothing is allocated inside the timed region
    masks = [torch.empty(B, H, nb, nb, dtype=torch.uint8, device=dev) for _ in sets]
    outs = [torch.empty(B, H, N, d, dtype=torch.bfloat16, device=dev) for _ in sets]
    ws_cmp = P.compact_block_mask_workspace(masks[0])
    R = B * H * nb
    lists = (torch.empty(R + 1, dtype=torch.int32, device=dev),
             torch.empty(R * nb, dtype=torch.int32, device=dev),
             torch.empty(R, dtype=torch.int32, device=dev))
    ws_mask = P.build_block_mask_workspace(sets[0][0]["q_hist"], bs)
    ws_sig = P.signature_sim_workspace(synth.SIG_NQ, synth.SIG_M, synth.SIG_TOPK, dev)
    sig_out = (torch.empty(synth.SIG_NQ, synth.SIG_TOPK, dtype=torch.int32, device=dev),
               torch.empty(synth.SIG_NQ, synth.SIG_TOPK, dtype=torch.float32, device=dev))
    flags = [(x["row_flags"].contiguous(), None if x["col_flags"] is None else x["col_flags"].contiguous())
             for x, _ in sets]

    ev = {k: [] for k in ("build", "merge", "compact", "attn", "sig")}

    # record: None (no events), "attn" (events around the attention launch
    # only) or "all" (around every call).  Each recorded event leaves the
    # stream idle for a few microseconds, so the timed steps carry only the
    # attention pair and the per-call breakdown comes from a separate pass.
    def step(i, record):
        si = i % len(sets)
        x, sg = sets[si]
        e = [torch.cuda.Event(enable_timing=True) for _ in range(6)] if record else None
        if record == "all":
            e[0].record(stream)
        P.build_block_mask(x["q_hist"], x["k_hist"], bs, wl.tau, out=masks[si], workspace=ws_mask)
        if record == "all":
            e[1].record(stream)
        P.merge_target_rows(masks[si], flags[si][0], flags[si][1])
        if record == "all":
            e[2].record(stream)
        P.compact_block_mask(masks[si], trim=False, out=lists, workspace=ws_cmp, attn=(N, d, bs))
        if record:
            e[3].record(stream)
        P.block_sparse_attn_lists(x["q"], x["k"], x["v"], lists, bs, out=outs[si])
        if record:
            e[4].record(stream)
        P.signature_sim(sg["query"], sg["bank"], synth.SIG_TOPK, workspace=ws_sig, out=sig_out)
        if record == "all":
            e[5].record(stream)
            for k_, (a_, b_) in zip(("build", "merge", "compact", "sig"), ((0, 1), (1, 2), (2, 3), (4, 5))):
                ev[k_].append((e[a_], e[b_]))
        elif record:
            ev["attn"].append((e[3], e[4]))

    if args.copy_calibration_mib > 0:
        nbytes = args.copy_calibration_mib << 20
        src = torch.ones(nbytes, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    for i in range(args.warmup):
        step(i, None)
    torch.cuda.synchronize()
    print("bench: warmup done, timing %d steps" % args.steps, file=sys.stderr, flush=True)
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i, "attn")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = wall * 1e3 / args.steps
    # per-call breakdown of the other calls: a second pass of the same steps
    # with events around each call (outside the timed region)
    for i in range(args.steps):
        step(i, "all")
    torch.cuda.synchronize()

    def avg_ms(name):
        return float(np.mean([a.elapsed_time(b) for a, b in ev[name]]))

    # the attention timed with its compaction: one mask-in call
    # (carnator_block_sparse_attn: compaction + attention), events around it
    ws_attn = P.block_sparse_attn_workspace(sets[0][0]["q"], bs)
    with_cmp = []
    for i in range(args.steps + 1):
        si = i % len(sets)
        x = sets[si][0]
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        P.block_sparse_attn(x["q"], x["k"], x["v"], masks[si], bs, out=outs[si], workspace=ws_attn)
        e1.record(stream)
        if i > 0:
            with_cmp.append((e0, e1))
    torch.cuda.synchronize()
    attn_times = np.array([a.elapsed_time(b) for a, b in ev["attn"]])
    with_cmp_ms = float(np.mean([a.elapsed_time(b) for a, b in with_cmp]))

    bank = None if args.no_bank else bank_pass(P, torch, stream, sets, flags, masks, lists, ws_mask, wl,
                                                args.steps)
    region = None if args.no_region else region_pass(P, torch, stream, sets, wl, args.steps)
    exact = None if args.no_exact else exact_mass_pass(P, torch, stream, sets, wl, min(args.steps, 6))

    # algorithmic work of one step (averaged over the rotated sets)
    fl_exec = float(np.mean([executed_flops(m.cpu().numpy(), N, bs, d) for m in masks]))
    density = float(np.mean([m.float().mean().item() for m in masks]))
    fl_dense = dense_flops(B, H, N, d)
    attn_ms = avg_ms("attn")
    build_ms = avg_ms("build")
    sig_ms = avg_ms("sig")
    builder_bytes = 2.0 * B * H * N * d * 2 + B * H * nb * nb
    sig_bytes = 4.0 * synth.SIG_M * synth.SIG_D + 4.0 * synth.SIG_NQ * synth.SIG_D + 8.0 * synth.SIG_NQ * synth.SIG_TOPK
    attn_tflops = fl_exec / (attn_ms * 1e-3) / 1e12
    res = {
        "metric": METRIC,
        "value": round(fl_exec / (ms_step * 1e-3) / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": B, "heads": H, "seq_len": N, "head_dim": d, "block": bs,
                   "mass_threshold": wl.tau, "mask_density": round(density, 4),
                   "signature_bank": [synth.SIG_M, synth.SIG_D], "topk": synth.SIG_TOPK,
                   "input_sets": len(sets), "parallelism": "none (1 GPU)"},
        "attn_ms_per_call": round(attn_ms, 4),
        "attn_ms_p10_p50_p90": [round(float(np.percentile(attn_times, p_)), 4) for p_ in (10, 50, 90)],
        "attn_with_compaction_ms_per_call": round(with_cmp_ms, 4),
        "attn_executed_tflop": round(fl_exec / 1e12, 4),
        "attn_dense_equiv_tflop": round(fl_dense / 1e12, 4),
        "attn_executed_tflops": round(attn_tflops, 2),
        "attn_dense_equiv_tflops": round(fl_dense / (attn_ms * 1e-3) / 1e12, 2),
        "attn_pct_bf16_peak": round(100.0 * attn_tflops / PEAK_BF16_TFLOPS, 2),
        "per_call_pass": "builder, merge, compaction and signature times come from a second pass of "
                         "the same steps with events around every call",
        "builder_ms_per_call": round(build_ms, 4),
        "builder_GBps": round(builder_bytes / (build_ms * 1e-3) / 1e9, 1),
        "builder_pct_hbm_peak": round(100.0 * builder_bytes / (build_ms * 1e-3) / 1e9 / PEAK_HBM_GBPS, 2),
        "merge_ms_per_call": round(avg_ms("merge"), 4),
        "compact_ms_per_call": round(avg_ms("compact"), 4),
        "sig_ms_per_call": round(sig_ms, 4),
        "sig_GBps": round(sig_bytes / (sig_ms * 1e-3) / 1e9, 1),
        "roofline": {"bound": "mfma", "achieved": round(attn_tflops, 2), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic(d, bs),
                     "kernel": "bsattn_kernel<%d, %d> (one launch of carnator_block_sparse_attn_lists)" % (d, bs)},
    }
    if bank is not None:
        res["mask_bank"] = bank
    if region is not None:
        res["region_restricted"] = region
    if exact is not None:
        res["exact_mass"] = exact
    if not args.no_workloads:
        del sets, masks, outs, lists
        torch.cuda.empty_cache()
        res["workloads"] = workload_pass(P, torch, stream, [w for w in (2, 3, 4) if w != args.workload], 5)
    if not args.no_cpu_baseline:
        print("bench: timing the oracle on the host", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
