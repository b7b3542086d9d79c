"""Exact widening of inputs to fp64 (oracle test infrastructure).

bf16 -> fp32 -> fp64 is exact, so the oracle sees the very bits the GPU reads.
"""
import numpy as np


def to_f64(x) -> np.ndarray:
    """Torch tensor (any device; bf16, fp16, fp32 or fp64) or array -> fp64 ndarray."""
    if hasattr(x, "detach"):
        x = x.detach().cpu()
        if x.is_floating_point():
            x = x.double()  # exact for every narrower float format
        return x.numpy().astype(np.float64)
    return np.asarray(x, dtype=np.float64)
