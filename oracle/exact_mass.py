"""Exact (token-level) attention mass per block pair and the selection on it
(oracle test infrastructure; fp64 NumPy).

Paper: Appendix C.3 partitions the historical self-attention into query-key
blocks and keeps, for each head and query block, the smallest set of key
blocks covering a fixed fraction of the source attention mass.  Here the mass
is the historical run's own softmax attention summed over the tokens of each
block pair -- the literal reading of "source attention mass" -- rather than
the block-pooled estimate of ``oracle.mask``.

Readings:

1. M[b,h,i,j] = (1 / n_i) sum over the valid queries a of block i and the
   keys t of block j of softmax_t(sigma q_a . k_t), the softmax taken over
   all N keys; sigma = 1/sqrt(d) unless given.  Each row sums to 1.
2. Selection on a row of masses: the smallest prefix of the key blocks by
   descending mass (lower index first on equal mass) whose mass reaches
   tau (of the row total); masses within 1e-6 of the cut mass are tied and
   the lower block indices among them are kept -- the pooled builder's rule
   with the mass in place of the pooled logit.
"""
import numpy as np

from .mask import TIE_EPS, FRAGILE_EPS, _keep_from_cut


def exact_block_mass(q: np.ndarray, k: np.ndarray, bs: int, scale: float = None, rows=None) -> np.ndarray:
    """q, k: fp64 [B, H, N, d].  Returns fp64 [B, H, nB, nB]; with ``rows``
    (an iterable of (b, h, i)) only those rows are computed and the others
    are NaN."""
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    B, H, N, d = q.shape
    sigma = (1.0 / np.sqrt(float(d))) if (scale is None or scale <= 0) else float(scale)
    nb = -(-N // bs)
    out = np.full((B, H, nb, nb), np.nan)
    todo = [(b, h, i) for b in range(B) for h in range(H) for i in range(nb)] if rows is None else list(rows)
    for (b, h, i) in todo:
        a0, a1 = i * bs, min((i + 1) * bs, N)
        s = sigma * (q[b, h, a0:a1] @ k[b, h].T)  # [n_i, N]
        p = np.exp(s - s.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        for j in range(nb):
            t0, t1 = j * bs, min((j + 1) * bs, N)
            out[b, h, i, j] = p[:, t0:t1].sum() / (a1 - a0)
    return out


def select_row_mass(m: np.ndarray, tau: float, tie_eps: float = TIE_EPS) -> dict:
    """Top-mass selection of one row of block masses (reading 2)."""
    m = np.asarray(m, dtype=np.float64)
    n = len(m)
    if tau >= 1.0:
        return {"keep": np.ones(n, dtype=bool), "k": n, "fragile": False}
    p = m / m.sum()
    order = np.lexsort((np.arange(n), -m))
    cum = np.cumsum(p[order])
    hit = np.nonzero(cum >= tau)[0]
    k = int(hit[0]) + 1 if len(hit) else n
    keep = _keep_from_cut(m, order, k, tie_eps)
    c = m[order[k - 1]]
    fragile = bool(abs(cum[k - 1] - tau) < FRAGILE_EPS
                   or (k >= 2 and abs(cum[k - 2] - tau) < FRAGILE_EPS)
                   or np.any(np.abs(np.abs(m - c) - tie_eps) < FRAGILE_EPS))
    return {"keep": keep, "k": k, "fragile": fragile}


def row_admissible_masks_mass(m: np.ndarray, tau: float, tie_eps: float = TIE_EPS) -> list:
    """Every keep set a correct implementation may produce for a fragile row
    of masses: prefix length k-1, k or k+1 of the descending-mass order, and
    the tie band taken just inside or just outside tie_eps (the selection of
    reading 2 with a decision moved across a threshold it lies within
    FRAGILE_EPS of)."""
    m = np.asarray(m, dtype=np.float64)
    n = len(m)
    base = select_row_mass(m, tau, tie_eps)
    if tau >= 1.0:
        return [base["keep"]]
    order = np.lexsort((np.arange(n), -m))
    out = []
    for k in (base["k"] - 1, base["k"], base["k"] + 1):
        if not 1 <= k <= n:
            continue
        for eps in (tie_eps - 2 * FRAGILE_EPS, tie_eps, tie_eps + 2 * FRAGILE_EPS):
            keep = _keep_from_cut(m, order, k, eps)
            if not any(np.array_equal(keep, o) for o in out):
                out.append(keep)
    return out


def mask_from_mass(mass: np.ndarray, tau: float):
    """Block mask uint8 [B, H, nB, nB] from masses [B, H, nB, nB]; the report
    lists the fragile rows (a decision within FRAGILE_EPS of a threshold)."""
    M = np.asarray(mass, dtype=np.float64)
    B, H, nb, _ = M.shape
    mask = np.zeros(M.shape, dtype=np.uint8)
    fragile = []
    for b in range(B):
        for h in range(H):
            for i in range(nb):
                r = select_row_mass(M[b, h, i], tau)
                mask[b, h, i] = r["keep"]
                if r["fragile"]:
                    fragile.append((b, h, i))
    return mask, {"fragile": fragile}
