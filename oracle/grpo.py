"""Group-relative advantages (oracle), Eq. grpo of section 2.

A_i = (r_i - mean(r)) / (std(r) + eps) within each group, with the unbiased
(divide by m - 1) standard deviation and eps = 1e-6 (the paper does not fix
either).  A saturated group has zero spread and every A_i is exactly 0, the
fact behind Definition 1.  Groups are given in CSR form (offsets, rewards).
"""
import numpy as np


def advantages(rewards, offsets, eps: float = 1e-6, unbiased: bool = True) -> np.ndarray:
    r = np.asarray(rewards, dtype=np.float64)
    out = np.zeros_like(r)
    for g in range(len(offsets) - 1):
        lo, hi = int(offsets[g]), int(offsets[g + 1])
        m = hi - lo
        if m == 0:
            continue
        x = r[lo:hi]
        mean = x.sum() / m
        if m < 2:
            continue
        var = ((x - mean) ** 2).sum() / ((m - 1) if unbiased else m)
        out[lo:hi] = (x - mean) / (np.sqrt(var) + eps)
    return out
