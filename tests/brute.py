"""Independent NumPy references used to pin the oracle.

Nothing here calls the oracle.  The PBB mask is built from the direct-coverage form
``C(d, r) = 1{0 <= d <= r} + 1{r < h, r < d <= r + h}`` (Sec. 3, "Coverage and arithmetic";
Appendix A.4) for non-initial blocks, with plain causal attention inside the first block,
and the attention is a textbook dense masked softmax in "prefill form" (all targets at once).
"""
from __future__ import annotations

import numpy as np


def coverage_mask(n: int, block: int, bridge: int | None = None) -> np.ndarray:
    """Bool [n][n]: M[t, s] = True iff source s feeds target t under PBB."""
    h = block // 2 if bridge is None else bridge
    t = np.arange(n).reshape(-1, 1)
    s = np.arange(n).reshape(1, -1)
    dist = t - s
    r = t % block
    initial = (t // block) == 0
    cov = ((dist >= 0) & (dist <= r)) | ((r < h) & (dist > r) & (dist <= r + h))
    causal = dist >= 0
    return np.where(initial, causal, cov)


def coverage_mask_window(t_lo: int, nt: int, s_lo: int, ns: int, block: int,
                         bridge: int | None = None) -> np.ndarray:
    """Bool [nt][ns]: the coverage mask of targets t_lo .. t_lo+nt-1 over sources
    s_lo .. s_lo+ns-1 (same rule as :func:`coverage_mask`, on absolute positions)."""
    h = block // 2 if bridge is None else bridge
    t = t_lo + np.arange(nt).reshape(-1, 1)
    s = s_lo + np.arange(ns).reshape(1, -1)
    dist = t - s
    r = t % block
    initial = (t // block) == 0
    cov = ((dist >= 0) & (dist <= r)) | ((r < h) & (dist > r) & (dist <= r + h))
    causal = dist >= 0
    return np.where(initial, causal, cov)


def interval_start(t: int, block: int) -> int:
    """Left end a(t) = max(0, h*(floor(t/h) - 1)) of the interval form (Sec. 3 "Flash-PBB";
    Appendix A.3, Eq.(pbb_relay)), h = block/2."""
    h = block // 2
    return max(0, h * (t // h - 1))


def window_mask(n: int, window: int) -> np.ndarray:
    t = np.arange(n).reshape(-1, 1)
    s = np.arange(n).reshape(1, -1)
    return (s <= t) & (s > t - window)


def block_causal_mask(n: int, block: int) -> np.ndarray:
    t = np.arange(n).reshape(-1, 1)
    s = np.arange(n).reshape(1, -1)
    return (s <= t) & (s // block == t // block)


def masked_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, mask: np.ndarray,
                     scale: float) -> np.ndarray:
    """Dense masked softmax attention, fp64: q [n][d], k [n][d], v [n][d], mask [n][n]."""
    z = (q.astype(np.float64) @ k.astype(np.float64).T) * scale
    z = np.where(mask, z, -np.inf)
    z = z - z.max(axis=1, keepdims=True)
    w = np.exp(z)
    w = w / w.sum(axis=1, keepdims=True)
    return w @ v.astype(np.float64)
