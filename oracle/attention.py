"""Block-sparse softmax attention under a reused block mask
(oracle test infrastructure; fp64 NumPy).

Paper: Sec. 3.3, "Historical Sparse-Connectivity Reuse", and Appendix C.3:
the target's Q, K and V are recomputed and only the query-key block pairs the
historical structure keeps are evaluated; the historical attention values are
not reused.

Definition (two-pass, no tiling, no online rescaling): for a valid query token
a in block i, the allowed keys are A(a) = { t < N : mask[b,h,i,t // bs] != 0 };

    s_t = sigma * <q_a, k_t>,  m = max s,  w_t = exp(s_t - m),  Z = sum w,
    o_a = sum_t (w_t / Z) v_t,  lse_a = m + log Z,

and a query whose A(a) is empty gets o_a = 0 and lse_a = -inf (a reading: the
paper never produces such rows; they arise only from a caller's mask).
sigma = 1/sqrt(d) unless given.  Padding tokens beyond N are never read.
"""
import numpy as np


def token_mask_from_blocks(block_mask_row: np.ndarray, n: int, bs: int) -> np.ndarray:
    """Boolean token mask [nB*bs clipped to n] of one (b, h, i) row."""
    return np.repeat(np.asarray(block_mask_row) != 0, bs)[:n]


def block_sparse_attention(q, k, v, mask, bs: int, scale: float = None, rows=None):
    """q, k, v: fp64 [B, H, N, d]; mask: 0/1 [B, H, nB, nB].

    Returns ``(o, lse)`` as fp64 [B, H, N, d] and [B, H, N].  With ``rows``
    (an iterable of (b, h, i)), only those query blocks are computed and every
    other entry is NaN.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, H, N, d = q.shape
    sigma = (1.0 / np.sqrt(float(d))) if (scale is None or scale <= 0) else float(scale)
    nb = -(-N // bs)
    if rows is None:
        rows = [(b, h, i) for b in range(B) for h in range(H) for i in range(nb)]
        o = np.zeros((B, H, N, v.shape[-1]), dtype=np.float64)
        lse = np.zeros((B, H, N), dtype=np.float64)
    else:
        o = np.full((B, H, N, v.shape[-1]), np.nan, dtype=np.float64)
        lse = np.full((B, H, N), np.nan, dtype=np.float64)
    for (b, h, i) in rows:
        a0, a1 = i * bs, min((i + 1) * bs, N)
        allowed = token_mask_from_blocks(mask[b, h, i], N, bs)
        if not allowed.any():
            o[b, h, a0:a1] = 0.0
            lse[b, h, a0:a1] = -np.inf
            continue
        kk = k[b, h, allowed]
        vv = v[b, h, allowed]
        s = sigma * (q[b, h, a0:a1] @ kk.T)
        m = s.max(axis=1, keepdims=True)
        w = np.exp(s - m)
        z = w.sum(axis=1, keepdims=True)
        o[b, h, a0:a1] = (w / z) @ vv
        lse[b, h, a0:a1] = (m + np.log(z))[:, 0]
    return o, lse
