"""Historical block-connectivity mask, target widening and compaction
(oracle test infrastructure; fp64 NumPy).

Paper: Appendix C.3 ("Reuse-Scope Implementation Details") partitions the
historical self-attention into query-key blocks and, for each head and query
block, keeps the smallest set of key blocks that covers a fixed fraction of
the attention mass; the binary masks are stored per step, guidance branch and
layer.  Sec. 3.3 ("Historical Sparse-Connectivity Reuse") reuses that structure
for the target; Sec. 3.3 ("Joint Reuse in Intermediate Layers") keeps
target-specific computation where the evidence region lies.

Readings (the paper is silent on these points):

1. The mass of key block j for query block i is the softmax over j of the
   block-pooled logit s_ij = sigma * <mean_i(Q_hist), mean_j(K_hist)>, with
   sigma = 1/sqrt(d) unless given, and no block-size weighting.
2. Pooling is the mean over the valid tokens of a block (the last block may
   be partial; padding never enters a mean).
3. "Covering a fraction tau" means the cumulative mass of the kept set is
   >= tau; the smallest such set is the prefix of the key blocks sorted by
   descending score (lower index first on exact equality).  k >= 1 always;
   tau >= 1 keeps every block.
4. Ties: scores within TIE_EPS = 1e-6 of the cut score count as tied, and
   among tied blocks the lower block indices are kept (the count kept is the
   one the sorted prefix gives).
5. Target widening: a flagged query block becomes a full row; a flagged key
   block (dense text columns) becomes a full column.
6. Stored form: the paper keeps the binary masks but names no encoding.  One
   bit per block pair, key block j of a row at bit j mod 64 (least
   significant first) of the row's 64-bit word j // 64, unused high bits of
   the last word zero.
"""
import numpy as np

TIE_EPS = 1e-6
# Decisions closer than this to a threshold are reported as fragile: an
# implementation that rounds differently (order of a dot product, of a prefix
# sum, an exp that is 1 ulp off) may legitimately land on the other side.
FRAGILE_EPS = 1e-9


def _block_bounds(n: int, bs: int):
    nb = -(-n // bs)
    return [(j * bs, min((j + 1) * bs, n)) for j in range(nb)]


def pool_blocks(x: np.ndarray, bs: int) -> np.ndarray:
    """Mean over the valid tokens of each block.  x: fp64 [N, d] -> [nB, d]."""
    x = np.asarray(x, dtype=np.float64)
    out = np.empty((-(-x.shape[0] // bs), x.shape[1]), dtype=np.float64)
    for j, (a, b) in enumerate(_block_bounds(x.shape[0], bs)):
        out[j] = x[a:b].sum(axis=0) / (b - a)
    return out


def block_scores(qbar: np.ndarray, kbar: np.ndarray, sigma: float) -> np.ndarray:
    """s_ij = sigma * <qbar_i, kbar_j>  (fp64)."""
    return sigma * (qbar @ kbar.T)


def _keep_from_cut(s: np.ndarray, order: np.ndarray, k: int, tie_eps: float) -> np.ndarray:
    """Keep set for prefix length k under the tie rule (reading 4)."""
    c = s[order[k - 1]]
    splus = np.nonzero(s > c + tie_eps)[0]
    tie = np.nonzero(np.abs(s - c) <= tie_eps)[0]  # ascending block index
    need = k - len(splus)
    keep = np.zeros(len(s), dtype=bool)
    keep[splus] = True
    keep[tie[:need]] = True
    return keep


def select_row(s: np.ndarray, tau: float, tie_eps: float = TIE_EPS) -> dict:
    """Top-mass selection of one query-block row.

    Returns ``keep`` (bool [nB]), ``k``, the cut score and a fragility flag.
    """
    s = np.asarray(s, dtype=np.float64)
    n = len(s)
    if tau >= 1.0:
        return {"keep": np.ones(n, dtype=bool), "k": n, "cut": None, "fragile": False}
    e = np.exp(s - s.max())
    p = e / e.sum()
    order = np.lexsort((np.arange(n), -s))  # descending score, lower index first
    cum = np.cumsum(p[order])
    hit = np.nonzero(cum >= tau)[0]
    k = int(hit[0]) + 1 if len(hit) else n
    keep = _keep_from_cut(s, order, k, tie_eps)
    c = s[order[k - 1]]
    fragile = bool(abs(cum[k - 1] - tau) < FRAGILE_EPS
                   or (k >= 2 and abs(cum[k - 2] - tau) < FRAGILE_EPS)
                   or np.any(np.abs(np.abs(s - c) - tie_eps) < FRAGILE_EPS))
    return {"keep": keep, "k": k, "cut": float(c), "fragile": fragile}


def row_admissible_masks(s: np.ndarray, tau: float, tie_eps: float = TIE_EPS) -> list:
    """Every keep set a correct implementation may produce for a fragile row:
    prefix length k-1, k or k+1, and the tie band taken just inside or just
    outside 1e-6."""
    s = np.asarray(s, dtype=np.float64)
    n = len(s)
    base = select_row(s, tau, tie_eps)
    if tau >= 1.0:
        return [base["keep"]]
    order = np.lexsort((np.arange(n), -s))
    out = []
    for k in (base["k"] - 1, base["k"], base["k"] + 1):
        if not 1 <= k <= n:
            continue
        for eps in (tie_eps - 2 * FRAGILE_EPS, tie_eps, tie_eps + 2 * FRAGILE_EPS):
            m = _keep_from_cut(s, order, k, eps)
            if not any(np.array_equal(m, o) for o in out):
                out.append(m)
    return out


def build_block_mask(q_hist: np.ndarray, k_hist: np.ndarray, bs: int, tau: float,
                     scale: float = None):
    """Historical block mask.  q_hist, k_hist: fp64 [B, H, N, d].

    Returns ``(mask uint8 [B, H, nB, nB], report)``; ``report['fragile']`` lists
    the (b, h, i) rows whose decision lies within FRAGILE_EPS of a threshold and
    ``report['scores']`` holds the pooled scores of those rows.
    """
    B, H, N, d = q_hist.shape
    sigma = (1.0 / np.sqrt(float(d))) if (scale is None or scale <= 0) else float(scale)
    nb = -(-N // bs)
    mask = np.zeros((B, H, nb, nb), dtype=np.uint8)
    report = {"fragile": [], "scores": {}, "k": np.zeros((B, H, nb), dtype=np.int64)}
    for b in range(B):
        for h in range(H):
            qbar = pool_blocks(q_hist[b, h], bs)
            kbar = pool_blocks(k_hist[b, h], bs)
            s = block_scores(qbar, kbar, sigma)
            for i in range(nb):
                r = select_row(s[i], tau)
                mask[b, h, i] = r["keep"]
                report["k"][b, h, i] = r["k"]
                if r["fragile"]:
                    report["fragile"].append((b, h, i))
                    report["scores"][(b, h, i)] = s[i].copy()
    report["tau"] = tau
    return mask, report


def merge_target_rows(mask: np.ndarray, row_flags: np.ndarray, col_flags: np.ndarray = None) -> np.ndarray:
    """M'[b,h,i,j] = M[b,h,i,j] or row_flags[b,i] or col_flags[b,j] (0/1 bytes)."""
    out = (np.asarray(mask) != 0)
    out = out | (np.asarray(row_flags) != 0)[:, None, :, None]
    if col_flags is not None:
        out = out | (np.asarray(col_flags) != 0)[:, None, None, :]
    return out.astype(np.uint8)


def group_rows_order(order: np.ndarray, group_rows: int) -> np.ndarray:
    """The row order taken apart by head group, each group keeping its order.

    Rows are (b, h, i) in row-major order, so heads [g G, (g + 1) G) are the
    rows [g group_rows, (g + 1) group_rows), group_rows = G nB.  The result
    lists group 0's rows in the order they have in ``order``, then group 1's,
    and so on (an execution schedule; the paper does not fix one).
    """
    order = np.asarray(order)
    if group_rows is None or order.size == 0:
        return order
    return order[np.argsort(order // int(group_rows), kind="stable")]


def compact_mask(mask: np.ndarray, group_heads: int = None):
    """Per-row list of kept key blocks.

    Rows are (b, h, i) in row-major order.  Returns ``row_ptr`` (int32
    [R+1]), ``col_idx`` (int32 [nnz], ascending within a row) and ``order``
    (int32 [R]: rows by descending list length, lower row first on equal
    length; with ``group_heads`` G, that order per group of G consecutive
    heads, group after group).
    """
    m = (np.asarray(mask) != 0)
    nb = m.shape[-1]
    flat = m.reshape(-1, nb)
    counts = flat.sum(axis=1)
    row_ptr = np.zeros(flat.shape[0] + 1, dtype=np.int64)
    row_ptr[1:] = np.cumsum(counts)
    col_idx = np.nonzero(flat)[1]
    order = np.argsort(-counts, kind="stable")
    if group_heads is not None:
        order = group_rows_order(order, int(group_heads) * nb)
    return row_ptr.astype(np.int32), col_idx.astype(np.int32), order.astype(np.int32)


def pack_mask(mask: np.ndarray) -> np.ndarray:
    """Bit-packed form of a block mask [..., nB, nB]: uint64 [..., nB, W],
    W = ceil(nB / 64); word w of a row holds key blocks 64 w .. 64 w + 63,
    block j at bit j - 64 w.  Bits past nB are 0."""
    m = (np.asarray(mask) != 0)
    nb = m.shape[-1]
    w = (nb + 63) // 64
    padded = np.zeros(m.shape[:-1] + (w * 64,), dtype=np.uint64)
    padded[..., :nb] = m
    chunks = padded.reshape(m.shape[:-1] + (w, 64))
    weights = np.left_shift(np.uint64(1), np.arange(64, dtype=np.uint64))
    # distinct powers of two: the sum is the bitwise OR
    return (chunks * weights).sum(axis=-1, dtype=np.uint64)


def unpack_mask(bits: np.ndarray, nb: int) -> np.ndarray:
    """Inverse of pack_mask: 0/1 bytes [..., nB, nB]; bits past nB are
    ignored."""
    b = np.asarray(bits, dtype=np.uint64)
    shifts = np.arange(64, dtype=np.uint64)
    cols = (b[..., :, None] >> shifts) & np.uint64(1)
    flat = cols.reshape(b.shape[:-1] + (b.shape[-1] * 64,))
    return flat[..., :nb].astype(np.uint8)
