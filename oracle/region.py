"""Region-restricted reuse in the middle layers (oracle test infrastructure;
fp64 NumPy, brute force).

Paper: Sec. 3.3 ("Region-Guided Latent Reuse") grows the Evidence Region into
an Active Region and a larger Context Region, nested in that order over the
T x H x W token domain; the latent of every later step blends the
target-updated latent and the historical one with a weight W that is 1 on the
evidence, falls through the transition band (active minus evidence) as one
minus the smoothstep of the normalised Chebyshev distance to the evidence, and
is 0 outside the active region.  Sec. 3.3 ("Joint Reuse in Intermediate
Layers") keeps, in the middle layers, only the historical connectivity of
active queries and their context keys; tokens outside the active region keep
their cached computation.  Appendix C.3 fixes the radii: active = evidence
dilated by 2 tokens, context = active dilated by 3 more, per latent frame on
the H x W grid, the band distance normalised by its maximum over the band.

Readings (the paper is silent on these points):

1. Dilation by radius r uses the square (2r + 1) x (2r + 1) window, i.e. the
   Chebyshev ball, clipped at the frame border, the same metric as the band
   distance.
2. The Chebyshev distance of a token is taken within its own frame; the
   normalising maximum is taken over the whole band of a batch entry (all
   frames).  An empty band needs no normalisation.
3. smoothstep s(t) = 3 t^2 - 2 t^3 on [0, 1].
4. Latents are finer than the token grid by a patch (pt, ph, pw); a latent
   element takes the weight of the token whose patch holds it.
5. Restriction works on blocks of the attention's token order: a query block
   is active if one of its tokens is active, a key block is context if one of
   its tokens is in the context region.  Text tokens (placed before the video
   tokens) carry the target prompt and are recomputed: they count as active
   and as context.
6. Rows of inactive query blocks are not computed at all: the restricted
   lists order the active rows first (longest first, lower row on equal
   length; per group of heads when a group size is given, as in
   ``compact_mask``), then the inactive rows in row order, and report how many
   rows are active; the attention walks only those.
"""
import numpy as np

from .mask import group_rows_order

EVIDENCE, BAND, CONTEXT, OUTSIDE = 3, 2, 1, 0


def dilate_frames(mask: np.ndarray, r: int) -> np.ndarray:
    """Dilation of a binary [..., H, W] mask by the (2r+1)^2 square, per frame."""
    m = np.asarray(mask) != 0
    H, W = m.shape[-2:]
    out = np.zeros_like(m)
    for dy in range(-r, r + 1):
        for dx in range(-r, r + 1):
            ys, yd = (slice(0, H - dy), slice(dy, H)) if dy >= 0 else (slice(-dy, H), slice(0, H + dy))
            xs, xd = (slice(0, W - dx), slice(dx, W)) if dx >= 0 else (slice(-dx, W), slice(0, W + dx))
            out[..., yd, xd] |= m[..., ys, xs]
    return out


def chebyshev_distance(evidence: np.ndarray) -> np.ndarray:
    """Per frame, min over evidence tokens (y', x') of max(|y - y'|, |x - x'|);
    +inf in a frame without evidence.  Brute force over all pairs."""
    e = np.asarray(evidence) != 0
    H, W = e.shape[-2:]
    yy, xx = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    out = np.full(e.shape, np.inf)
    for idx in np.ndindex(e.shape[:-2]):
        ey, ex = np.nonzero(e[idx])
        if ey.size == 0:
            continue
        d = np.maximum(np.abs(yy[..., None] - ey), np.abs(xx[..., None] - ex))
        out[idx] = d.min(axis=-1)
    return out


def smoothstep(t):
    t = np.clip(np.asarray(t, dtype=np.float64), 0.0, 1.0)
    return t * t * (3.0 - 2.0 * t)


def regions(evidence: np.ndarray, r_active: int = 2, r_context: int = 3):
    """Evidence [B, T, H, W] -> (region code, W), both [B, T, H, W].

    Codes: 3 evidence, 2 transition band (active minus evidence), 1 context
    minus active, 0 outside the context region."""
    e = np.asarray(evidence) != 0
    active = dilate_frames(e, r_active)
    context = dilate_frames(active, r_context)
    code = np.where(e, EVIDENCE, np.where(active, BAND, np.where(context, CONTEXT, OUTSIDE))).astype(np.uint8)
    d = chebyshev_distance(e)
    w = np.zeros(e.shape, dtype=np.float64)
    w[e] = 1.0
    for b in range(e.shape[0]):
        band = code[b] == BAND
        if band.any():
            dmax = d[b][band].max()
            w[b][band] = 1.0 - smoothstep(d[b][band] / dmax)
    return code, w


def latent_fusion(z_target: np.ndarray, z_hist: np.ndarray, weight: np.ndarray, patch=(1, 1, 1)) -> np.ndarray:
    """z = W * z_target + (1 - W) * z_hist for latents [B, C, T, H, W]; the
    weight [B, T/pt, H/ph, W/pw] is repeated over each token's patch and over
    the channels."""
    pt, ph, pw = patch
    w = np.asarray(weight, dtype=np.float64)
    w = np.repeat(np.repeat(np.repeat(w, pt, axis=1), ph, axis=2), pw, axis=3)[:, None]
    zt = np.asarray(z_target, dtype=np.float64)
    zh = np.asarray(z_hist, dtype=np.float64)
    return w * zt + (1.0 - w) * zh


def region_block_flags(code: np.ndarray, n_text: int, block: int):
    """(active query blocks, context key blocks), uint8 [B, nB] each, for
    token order [text tokens, video tokens in (t, y, x) raster order]."""
    c = np.asarray(code).reshape(code.shape[0], -1)
    B, nv = c.shape
    n = n_text + nv
    nb = -(-n // block)
    tok_active = np.concatenate([np.ones((B, n_text), bool), c >= BAND], axis=1)
    tok_context = np.concatenate([np.ones((B, n_text), bool), c >= CONTEXT], axis=1)
    act = np.zeros((B, nb), np.uint8)
    ctx = np.zeros((B, nb), np.uint8)
    for i in range(nb):
        sl = slice(i * block, min((i + 1) * block, n))
        act[:, i] = tok_active[:, sl].any(axis=1)
        ctx[:, i] = tok_context[:, sl].any(axis=1)
    return act, ctx


def restrict_mask(mask: np.ndarray, active_q: np.ndarray, context_k: np.ndarray) -> np.ndarray:
    """M'[b,h,i,j] = M[b,h,i,j] and active_q[b,i] and context_k[b,j] (0/1)."""
    m = np.asarray(mask) != 0
    a = (np.asarray(active_q) != 0)[:, None, :, None]
    c = (np.asarray(context_k) != 0)[:, None, None, :]
    return (m & a & c).astype(np.uint8)


def compact_restricted(mask: np.ndarray, active_q: np.ndarray, context_k: np.ndarray,
                       group_heads: int = None):
    """Lists of the restricted mask: (row_ptr, col_idx, order, n_active).

    Rows are (b, h, i) in row-major order; order lists the active rows by
    descending length (lower row first on equal length; with ``group_heads``
    G, that order per group of G consecutive heads, group after group), then
    the inactive rows in ascending order; n_active is the number of active
    rows."""
    m = restrict_mask(mask, active_q, context_k)
    B, H, nb, _ = m.shape
    flat = m.reshape(-1, nb)
    counts = flat.sum(axis=1, dtype=np.int64)  # signed: the order negates it
    row_ptr = np.zeros(flat.shape[0] + 1, dtype=np.int64)
    row_ptr[1:] = np.cumsum(counts)
    col_idx = np.nonzero(flat)[1]
    row_active = np.broadcast_to((np.asarray(active_q) != 0)[:, None, :], (B, H, nb)).reshape(-1)
    rows = np.arange(flat.shape[0])
    act = rows[row_active]
    act = act[np.argsort(-counts[act], kind="stable")]
    if group_heads is not None:
        act = group_rows_order(act, int(group_heads) * nb)
    order = np.concatenate([act, rows[~row_active]])
    return (row_ptr.astype(np.int32), col_idx.astype(np.int32), order.astype(np.int32), int(act.size))
