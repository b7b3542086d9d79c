"""Cosine scoring of an early-step signature against a cached bank
(oracle test infrastructure; fp64 NumPy).

Paper: Sec. 3.1 (a target request is compared against a cache bank built
from completed requests), Sec. 3.2 ("Early Signature Construction": the
signature summarises the partially formed generation state of an early probe)
and Sec. 4.1 ("Candidate Recall": histories are ranked by similarity and the
top K are retained).  The signature here is an early-step hidden state
(a D-dimensional vector) and the similarity is the cosine.

Readings: cos = <q, b> / (|q| |b|) in fp64; a zero-norm vector scores 0.
Top-k keeps the k best by the same rule as the block selection: sort by
descending similarity (lower bank row first on equality), cut at position k,
and among scores within 1e-6 of the cut keep the lower rows.  The returned
indices are ordered by descending similarity, lower row first on equality.
"""
import numpy as np

TIE_EPS = 1e-6
FRAGILE_EPS = 1e-9


def cosine_similarity(query: np.ndarray, bank: np.ndarray) -> np.ndarray:
    """query [nq, D], bank [M, D] -> fp64 [nq, M]."""
    qd = np.asarray(query, dtype=np.float64)
    bd = np.asarray(bank, dtype=np.float64)
    dots = qd @ bd.T
    qn = np.sqrt((qd * qd).sum(axis=1))
    bn = np.sqrt((bd * bd).sum(axis=1))
    den = qn[:, None] * bn[None, :]
    out = np.zeros_like(dots)
    nz = den > 0
    out[nz] = dots[nz] / den[nz]
    return out


def topk_cosine(query: np.ndarray, bank: np.ndarray, k: int):
    """Returns ``(idx int64 [nq, k], sim fp64 [nq, k], fragile bool [nq])``."""
    sims = cosine_similarity(query, bank)
    nq, m = sims.shape
    if not 1 <= k <= m:
        raise ValueError("k must be in [1, M]")
    idx = np.zeros((nq, k), dtype=np.int64)
    val = np.zeros((nq, k), dtype=np.float64)
    fragile = np.zeros(nq, dtype=bool)
    for r in range(nq):
        s = sims[r]
        order = np.lexsort((np.arange(m), -s))
        c = s[order[k - 1]]
        splus = np.nonzero(s > c + TIE_EPS)[0]
        tie = np.nonzero(np.abs(s - c) <= TIE_EPS)[0]
        chosen = np.concatenate([splus, tie[:k - len(splus)]])
        chosen = chosen[np.lexsort((chosen, -s[chosen]))]
        idx[r] = chosen
        val[r] = s[chosen]
        ch = s[chosen]
        fragile[r] = bool(np.any(np.abs(np.abs(s - c) - TIE_EPS) < FRAGILE_EPS)
                          or np.any(np.abs(np.diff(ch)) < FRAGILE_EPS))
    return idx, val, fragile
