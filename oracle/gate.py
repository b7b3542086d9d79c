"""Compatibility gate of a recalled cache (oracle test infrastructure; fp64
NumPy / SciPy).

Paper: Sec. 3.2 ("Reuse Validity with Generation-Native Evidence") builds, per
object (noun) of a request, an Early Signature
from its support mask in the tail latent frame: the normalised support size
A (the mean of the binary mask over the H x W grid), the mask itself and a
CIELAB colour.  Against a candidate the discrepancies are the colour
difference d_color (CIEDE2000), d_size = |ln(A_q / A_j)|, and d_shape, one
minus the Dice overlap of the two masks each cropped to its bounding box and
resized to a common grid; d_context is the largest CIEDE2000 over the objects
both requests share (0 when none).  A candidate is compatible when every
discrepancy is within its threshold (the gate is the product of the
indicators); candidates are tried in recall order and the first compatible
one is reused, otherwise the request runs dense ("Compatibility
Filtering").  Sec. 3.2 ("Risk-Aware Compatibility Decisions") and Appendix F
certify a threshold setting with the one-sided Clopper-Pearson upper bound on
the unsafe-reuse rate (u unsafe among n accepted pairs) at level alpha.

Readings (the paper is silent on these points):

1. CIEDE2000 with kL = kC = kH = 1 (Sharma, Wu and Dalal, 2005), hue angles in
   degrees in [0, 360), the hue of a zero-chroma colour taken as 0.
2. The shape grid is res x res (res = 32 here), nearest-neighbour sampling:
   target cell (y, x) reads source (floor((y + 0.5) h / res), floor((x + 0.5)
   w / res)) of the h x w bounding-box crop.  An empty mask has area 0 and an
   all-zero shape; d_size is +inf when exactly one area is 0, 0 when both are.
   d_shape is 0 for two empty shapes.
3. The Clopper-Pearson upper bound at u = n is 1.

Pins: ``ciede2000`` is pinned in its lightness and chroma terms by closed
forms, and as a whole (the hue weighting T, delta-theta, R_T, S_H included)
by LittleCMS's independent cmsCIE2000DeltaE on random, close,
near-achromatic and hue-wrap pairs (within 1e-9).
"""
import math

import numpy as np
from scipy import stats

SHAPE_RES = 32


def ciede2000(lab1, lab2) -> np.ndarray:
    """CIEDE2000 colour difference of [..., 3] CIELAB arrays (reading 1)."""
    lab1 = np.asarray(lab1, dtype=np.float64)
    lab2 = np.asarray(lab2, dtype=np.float64)
    L1, a1, b1 = lab1[..., 0], lab1[..., 1], lab1[..., 2]
    L2, a2, b2 = lab2[..., 0], lab2[..., 1], lab2[..., 2]
    C1 = np.hypot(a1, b1)
    C2 = np.hypot(a2, b2)
    Cbar = 0.5 * (C1 + C2)
    G = 0.5 * (1.0 - np.sqrt(Cbar ** 7 / (Cbar ** 7 + 25.0 ** 7)))
    a1p, a2p = (1.0 + G) * a1, (1.0 + G) * a2
    C1p, C2p = np.hypot(a1p, b1), np.hypot(a2p, b2)
    h1p = np.where(C1p == 0, 0.0, np.degrees(np.arctan2(b1, a1p)) % 360.0)
    h2p = np.where(C2p == 0, 0.0, np.degrees(np.arctan2(b2, a2p)) % 360.0)
    dLp = L2 - L1
    dCp = C2p - C1p
    dh = h2p - h1p
    dh = np.where(dh > 180.0, dh - 360.0, np.where(dh < -180.0, dh + 360.0, dh))
    dh = np.where(C1p * C2p == 0, 0.0, dh)
    dHp = 2.0 * np.sqrt(C1p * C2p) * np.sin(np.radians(dh) / 2.0)
    Lbarp = 0.5 * (L1 + L2)
    Cbarp = 0.5 * (C1p + C2p)
    hsum = h1p + h2p
    habs = np.abs(h1p - h2p)
    hbarp = np.where(C1p * C2p == 0, hsum,
                     np.where(habs <= 180.0, 0.5 * hsum,
                              np.where(hsum < 360.0, 0.5 * (hsum + 360.0), 0.5 * (hsum - 360.0))))
    T = (1.0 - 0.17 * np.cos(np.radians(hbarp - 30.0)) + 0.24 * np.cos(np.radians(2.0 * hbarp))
         + 0.32 * np.cos(np.radians(3.0 * hbarp + 6.0)) - 0.20 * np.cos(np.radians(4.0 * hbarp - 63.0)))
    dtheta = 30.0 * np.exp(-((hbarp - 275.0) / 25.0) ** 2)
    RC = 2.0 * np.sqrt(Cbarp ** 7 / (Cbarp ** 7 + 25.0 ** 7))
    SL = 1.0 + 0.015 * (Lbarp - 50.0) ** 2 / np.sqrt(20.0 + (Lbarp - 50.0) ** 2)
    SC = 1.0 + 0.045 * Cbarp
    SH = 1.0 + 0.015 * Cbarp * T
    RT = -np.sin(np.radians(2.0 * dtheta)) * RC
    tl, tc, th = dLp / SL, dCp / SC, dHp / SH
    return np.sqrt(tl * tl + tc * tc + th * th + RT * tc * th)


def support_area(mask_tail: np.ndarray) -> float:
    """A = (1 / HW) sum of the binary tail-frame mask."""
    return float((np.asarray(mask_tail) != 0).mean())


def normalized_shape(mask_tail: np.ndarray, res: int = SHAPE_RES) -> np.ndarray:
    """The mask cropped to its bounding box and resampled to res x res
    (reading 2); uint8 0/1."""
    m = np.asarray(mask_tail) != 0
    out = np.zeros((res, res), dtype=np.uint8)
    ys, xs = np.nonzero(m)
    if ys.size == 0:
        return out
    crop = m[ys.min():ys.max() + 1, xs.min():xs.max() + 1]
    h, w = crop.shape
    for y in range(res):
        sy = int(math.floor((y + 0.5) * h / res))
        for x in range(res):
            sx = int(math.floor((x + 0.5) * w / res))
            out[y, x] = crop[sy, sx]
    return out


def d_size(area_q: float, area_j: float) -> float:
    if area_q == 0 and area_j == 0:
        return 0.0
    if area_q == 0 or area_j == 0:
        return math.inf
    return abs(math.log(area_q / area_j))


def d_shape(shape_q: np.ndarray, shape_j: np.ndarray) -> float:
    a = np.asarray(shape_q) != 0
    b = np.asarray(shape_j) != 0
    tot = int(a.sum()) + int(b.sum())
    if tot == 0:
        return 0.0
    return 1.0 - 2.0 * int((a & b).sum()) / tot


def gate(d: np.ndarray, tau: np.ndarray) -> bool:
    """Product of the indicators d_k <= tau_k."""
    return bool(np.all(np.asarray(d, dtype=np.float64) <= np.asarray(tau, dtype=np.float64)))


def first_compatible(d_candidates: np.ndarray, tau: np.ndarray) -> int:
    """Index of the first candidate (recall order) passing the gate, or -1
    (dense generation)."""
    for i, d in enumerate(np.asarray(d_candidates, dtype=np.float64)):
        if gate(d, tau):
            return i
    return -1


def clopper_pearson_upper(u: int, n: int, alpha: float) -> float:
    """One-sided upper confidence bound on a rate from u failures in n trials
    at level alpha: the (1 - alpha) quantile of Beta(u + 1, n - u)."""
    if u >= n:
        return 1.0
    return float(stats.beta.ppf(1.0 - alpha, u + 1, n - u))
