"""Seeded synthetic inputs shaped like the video-DiT workloads of the paper.

This module only *makes inputs*.  It holds none of the method's arithmetic
(no pooling, no scoring, no selection, no attention, no cosine): both the HIP
path and the CPU oracle consume what it produces, and neither imports the
other.

The paper evaluates on real prompts (VidProM) with Wan2.2-TI2V-5B,
Wan2.1-T2V-1.3B and LTX-Video-13B (Sec. 4.1, "Models and Hardware" and
"Workload and Cache Settings"); none of those prompts, weights or cached
requests are used or reproduced here.  The tensors below stand in for the
Q/K/V of one self-attention layer of such a backbone:

* every (tensor, head, channel) carries a smooth spatiotemporal field over the
  latent grid (T, H, W): a sum of four sinusoids with integer frequencies in
  {0,1,2}^3 \\ {0}, uniform phases and N(0, 1/4) amplitudes, scaled by ``alpha``;
  Q and K share their field parameters (so attention is local in space-time,
  as it is in video DiTs), V has its own;
* each of Q, K, V then receives independent N(0, 0.5^2) noise;
* text tokens (where a workload has them) are packed first and are N(0, 1);
* the historical copy used to build the reused mask is
  Q_hist = bf16(Q + sigma_hist * N(0, 1)) and the same for K;
* target-specific query blocks come from an axis-aligned box in (t, y, x) grown
  from a seeded centre until it touches the requested number of blocks
  (a block is flagged when any of its tokens lies in the box); blocks holding
  text tokens are flagged as dense rows and dense columns.

Randomness: ``numpy.random.SeedSequence([seed, workload_id])`` spawns
independent child streams for the field parameters, the noise of each tensor,
the historical perturbations, the text tokens, the region and the signature
bank.  Large tensors are drawn with ``torch.Generator`` on the device that will
hold them, so the same seed yields the same bits on a given device type.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Optional

import numpy as np
import torch

# Field amplitude.  Calibrated once on the Wan-2.1-1.3B-shaped workload so that
# the historical mask density at mass threshold 0.9 lies in the 15-25 % band.
ALPHA = 1.85

QKV_NOISE_STD = 0.5


@dataclass(frozen=True)
class Workload:
    wid: int
    name: str
    batch: int
    heads: int
    head_dim: int
    grid: tuple  # (T, H, W) latent grid of video tokens
    n_text: int
    block: int
    tau: float
    sigma_hist: float
    target_blocks: int  # requested number of target-specific video query blocks
    region: str  # "block1" | "spatial" | "box3d"
    # signature scan (Early-Signature cosine scoring): (M, D, topk, nq) or None
    sig: Optional[tuple] = None

    @property
    def n_video(self) -> int:
        t, h, w = self.grid
        return t * h * w

    @property
    def seq_len(self) -> int:
        return self.n_text + self.n_video

    @property
    def n_blocks(self) -> int:
        return -(-self.seq_len // self.block)

    @property
    def tail_valid(self) -> int:
        r = self.seq_len - (self.n_blocks - 1) * self.block
        return r


WORKLOADS = {
    0: Workload(0, "tiny-3x8x8", 1, 2, 64, (3, 8, 8), 0, 64, 0.9, 0.3, 1, "block1"),
    1: Workload(1, "wan2.1-1.3b-21x30x52", 1, 12, 128, (21, 30, 52), 0, 128, 0.9, 0.2, 26, "spatial"),
    2: Workload(2, "cogvideox-5b-226+13x30x45", 1, 48, 64, (13, 30, 45), 226, 128, 0.85, 0.2, 21, "box3d",
                sig=(4096, 3072, 8, 2)),
    3: Workload(3, "wan2.1-14b-21x45x80", 1, 40, 128, (21, 45, 80), 0, 128, 0.9, 0.25, 119, "box3d"),
    4: Workload(4, "hunyuanvideo-256+33x45x80", 1, 24, 128, (33, 45, 80), 256, 128, 0.8, 0.2, 47, "box3d"),
}

# Signature bank of the CogVideoX-shaped workload (the only bank shape given).
SIG_M, SIG_D, SIG_TOPK, SIG_NQ = WORKLOADS[2].sig

_STREAMS = ("qk_field", "v_field", "q_noise", "k_noise", "v_noise",
            "qh_noise", "kh_noise", "text", "region", "signature", "evidence", "latent")


def _children(seed: int, wid: int) -> dict:
    ss = np.random.SeedSequence([int(seed), int(wid)])
    kids = ss.spawn(len(_STREAMS))
    return dict(zip(_STREAMS, kids))


def _torch_gen(child: np.random.SeedSequence, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(child.generate_state(1, dtype=np.uint64)[0] & ((1 << 63) - 1)))
    return g


def _field_params(child: np.random.SeedSequence, heads: int, dim: int):
    """Per (head, channel, term): frequency in {0,1,2}^3 minus the origin,
    phase ~ U[0, 2pi), amplitude ~ N(0, 1/4)."""
    rng = np.random.default_rng(child)
    freqs = np.array([(a, b, c) for a in range(3) for b in range(3) for c in range(3)
                      if (a, b, c) != (0, 0, 0)], dtype=np.float64)
    pick = rng.integers(0, len(freqs), size=(heads, dim, 4))
    f = freqs[pick]  # [H, C, 4, 3]
    phi = rng.uniform(0.0, 2.0 * math.pi, size=(heads, dim, 4))
    amp = rng.normal(0.0, 0.5, size=(heads, dim, 4))
    return f, phi, amp


def _video_coords(grid, device):
    T, H, W = grid
    t = torch.arange(T, device=device, dtype=torch.float32) / T
    y = torch.arange(H, device=device, dtype=torch.float32) / H
    x = torch.arange(W, device=device, dtype=torch.float32) / W
    tt = t[:, None, None].expand(T, H, W).reshape(-1)
    yy = y[None, :, None].expand(T, H, W).reshape(-1)
    xx = x[None, None, :].expand(T, H, W).reshape(-1)
    return tt, yy, xx


def _field_head(params, h: int, coords, alpha: float, device) -> torch.Tensor:
    """Smooth field of one head: [n_video, C] float32."""
    f, phi, amp = params
    tt, yy, xx = coords
    fh = torch.as_tensor(f[h], dtype=torch.float32, device=device)  # [C,4,3]
    ph = torch.as_tensor(phi[h], dtype=torch.float32, device=device)  # [C,4]
    ah = torch.as_tensor(amp[h], dtype=torch.float32, device=device)  # [C,4]
    out = torch.zeros(fh.shape[0], tt.shape[0], dtype=torch.float32, device=device)
    two_pi = 2.0 * math.pi
    for m in range(4):
        theta = (fh[:, m, 0:1] * tt[None, :] + fh[:, m, 1:2] * yy[None, :]
                 + fh[:, m, 2:3] * xx[None, :]) * two_pi + ph[:, m:m + 1]
        out.add_(ah[:, m:m + 1] * torch.sin(theta))
    out.mul_(alpha)
    return out.t().contiguous()


def region_flags(wl: Workload, seed: int = 0):
    """Target-specific query blocks and dense text columns.

    Returns (row_flags uint8 [B, nB], col_flags uint8 [B, nB] or None, info).
    """
    kids = _children(seed, wl.wid)
    nB = wl.n_blocks
    bs = wl.block
    rows = np.zeros((wl.batch, nB), dtype=np.uint8)
    cols = None
    info = {}
    if wl.region == "block1":
        rows[:, 1] = 1
        info["region"] = "query block 1"
        info["target_blocks"] = 1
    else:
        rng = np.random.default_rng(kids["region"])
        T, H, W = wl.grid
        centre = np.array([rng.integers(0, T), rng.integers(0, H), rng.integers(0, W)])
        lo = centre.copy()
        hi = centre.copy()
        if wl.region == "spatial":
            lo[0], hi[0] = 0, T - 1
            moves = [(1, +1), (2, +1), (1, -1), (2, -1)]
        else:
            moves = [(0, +1), (1, +1), (2, +1), (0, -1), (1, -1), (2, -1)]
        dims = np.array([T, H, W])

        def touched(lo_, hi_):
            t = np.arange(lo_[0], hi_[0] + 1)
            y = np.arange(lo_[1], hi_[1] + 1)
            x = np.arange(lo_[2], hi_[2] + 1)
            tok = wl.n_text + (t[:, None, None] * (H * W) + y[None, :, None] * W + x[None, None, :])
            return np.unique(tok.reshape(-1) // bs)

        blocks = touched(lo, hi)
        step = 0
        while len(blocks) < wl.target_blocks:
            d, s = moves[step % len(moves)]
            step += 1
            if s > 0 and hi[d] < dims[d] - 1:
                hi[d] += 1
            elif s < 0 and lo[d] > 0:
                lo[d] -= 1
            else:
                if all((hi[dd] == dims[dd] - 1 and lo[dd] == 0) for dd, _ in moves):
                    break
                continue
            blocks = touched(lo, hi)
        rows[:, blocks] = 1
        info["region"] = {"t": [int(lo[0]), int(hi[0])], "y": [int(lo[1]), int(hi[1])],
                          "x": [int(lo[2]), int(hi[2])]}
        info["target_blocks"] = int(len(blocks))
    if wl.n_text > 0:
        text_blocks = np.unique(np.arange(wl.n_text) // bs)
        rows[:, text_blocks] = 1
        cols = np.zeros((wl.batch, nB), dtype=np.uint8)
        cols[:, text_blocks] = 1
        info["text_blocks"] = [int(b) for b in text_blocks]
    return rows, cols, info


def attention_inputs(wl: Workload, seed: int = 0, device="cpu", alpha: float = ALPHA,
                     heads: Optional[int] = None):
    """Q, K, V and the historical Q_hist, K_hist as bf16 [B, H, N, d].

    ``heads`` (optional) generates only the first ``heads`` heads with the same
    bits those heads have in the full workload.
    """
    kids = _children(seed, wl.wid)
    Hn = wl.heads if heads is None else heads
    B, d, N, nt = wl.batch, wl.head_dim, wl.seq_len, wl.n_text
    dev = torch.device(device)
    qk_params = _field_params(kids["qk_field"], wl.heads, d)
    v_params = _field_params(kids["v_field"], wl.heads, d)
    coords = _video_coords(wl.grid, dev)
    gens = {k: _torch_gen(kids[k], dev) for k in
            ("q_noise", "k_noise", "v_noise", "qh_noise", "kh_noise", "text")}
    out = {k: torch.empty(B, Hn, N, d, dtype=torch.bfloat16, device=dev)
           for k in ("q", "k", "v", "q_hist", "k_hist")}
    for b in range(B):
        for h in range(Hn):
            fqk = _field_head(qk_params, h, coords, alpha, dev)
            fv = _field_head(v_params, h, coords, alpha, dev)
            vals = {}
            for name, fld, gname in (("q", fqk, "q_noise"), ("k", fqk, "k_noise"), ("v", fv, "v_noise")):
                x = torch.empty(N, d, dtype=torch.float32, device=dev)
                if nt:
                    x[:nt] = torch.randn(nt, d, generator=gens["text"], device=dev)
                noise = torch.randn(N - nt, d, generator=gens[gname], device=dev)
                x[nt:] = fld + QKV_NOISE_STD * noise
                vals[name] = x.to(torch.bfloat16)
            qh = (vals["q"].float() + wl.sigma_hist * torch.randn(N, d, generator=gens["qh_noise"], device=dev))
            kh = (vals["k"].float() + wl.sigma_hist * torch.randn(N, d, generator=gens["kh_noise"], device=dev))
            out["q"][b, h] = vals["q"]
            out["k"][b, h] = vals["k"]
            out["v"][b, h] = vals["v"]
            out["q_hist"][b, h] = qh.to(torch.bfloat16)
            out["k_hist"][b, h] = kh.to(torch.bfloat16)
    rows, cols, info = region_flags(wl, seed)
    out["row_flags"] = torch.as_tensor(rows, device=dev)
    out["col_flags"] = None if cols is None else torch.as_tensor(cols, device=dev)
    out["info"] = info
    return out


def signature_inputs(m: int = SIG_M, dim: int = SIG_D, nq: int = SIG_NQ, seed: int = 0,
                     device="cpu", wid: int = 2):
    """Bank [m, dim] of N(0,1) fp32 signatures and nq queries.

    Query 0 is pure N(0,1); query 1 (if nq > 1) is a planted near-duplicate
    ``bank[r] + 0.5 * N(0,1)`` of a seeded bank row r; further queries are
    N(0,1).
    """
    kids = _children(seed, wid)
    rng = np.random.default_rng(kids["signature"])
    bank = rng.standard_normal((m, dim), dtype=np.float32)
    q = rng.standard_normal((nq, dim), dtype=np.float32)
    planted = int(rng.integers(0, m))
    if nq > 1:
        q[1] = bank[planted] + np.float32(0.5) * rng.standard_normal(dim, dtype=np.float32)
    dev = torch.device(device)
    return {"query": torch.as_tensor(q, device=dev), "bank": torch.as_tensor(bank, device=dev),
            "planted": planted}


def random_mask(batch: int, heads: int, nb: int, density: float, seed: int = 0) -> np.ndarray:
    """Uniform random 0/1 block mask (for boundary and edge-case tests)."""
    rng = np.random.default_rng(np.random.SeedSequence([seed, 99]))
    return (rng.random((batch, heads, nb, nb)) < density).astype(np.uint8)


def evidence_region(wl: Workload, seed: int = 0) -> np.ndarray:
    """An object-like evidence region on the token grid, uint8 [B, T, H, W].

    Per frame, the tokens inside an ellipse whose centre drifts linearly over
    the frames, with radii of 1/6 to 1/4 of the frame, and a ragged boundary
    (tokens within one token of the ellipse edge flipped with probability
    0.3).  A random quarter of the frames (never all) hold no evidence.
    """
    kids = _children(seed, wl.wid)
    rng = np.random.default_rng(kids["evidence"])
    T, H, W = wl.grid
    out = np.zeros((wl.batch, T, H, W), dtype=np.uint8)
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    for b in range(wl.batch):
        c0 = np.array([rng.uniform(0.25, 0.75) * H, rng.uniform(0.25, 0.75) * W])
        drift = rng.uniform(-0.15, 0.15, size=2) * np.array([H, W]) / max(T, 1)
        radii = np.array([rng.uniform(1 / 6, 1 / 4) * H, rng.uniform(1 / 6, 1 / 4) * W])
        empty = rng.random(T) < 0.25
        if empty.all():
            empty[rng.integers(0, T)] = False
        for t in range(T):
            if empty[t]:
                continue
            cy, cx = c0 + drift * t
            r = np.sqrt(((yy - cy) / radii[0]) ** 2 + ((xx - cx) / radii[1]) ** 2)
            inside = r <= 1.0
            edge = np.abs(r - 1.0) * min(radii) <= 1.0
            flip = edge & (rng.random((H, W)) < 0.3)
            out[b, t] = (inside ^ flip).astype(np.uint8)
    return out


def latents(wl: Workload, channels: int = 16, patch=(1, 2, 2), seed: int = 0, device="cpu"):
    """Target-updated and historical latents, fp32 [B, C, T*pt, H*ph, W*pw]
    of N(0, 1) (the scale of a diffusion latent)."""
    kids = _children(seed, wl.wid)
    T, H, W = wl.grid
    shape = (wl.batch, channels, T * patch[0], H * patch[1], W * patch[2])
    g = _torch_gen(kids["latent"], "cpu")
    zt = torch.randn(shape, generator=g, dtype=torch.float32)
    zh = torch.randn(shape, generator=g, dtype=torch.float32)
    return zt.to(device), zh.to(device)
