"""Exact and compressed decode attention, and total variation (Sec. 3, setup).

For one (layer, head, decode step): logits l_t = (q . k_t) / sqrt(d) over the S
cached tokens, p = softmax(l), output y = sum_t p_t v_t.  The compressed
attention uses the reconstructed keys/values (khat, vhat) and gives ptilde and
yhat.  TV(p, ptilde) = 1/2 sum_t |p_t - ptilde_t|.  All float64, max-subtracted
softmax.  Pinned against torch's float64 scaled_dot_product_attention.
"""
from __future__ import annotations

import numpy as np


def softmax(logits: np.ndarray) -> np.ndarray:
    z = np.asarray(logits, dtype=np.float64)
    z = z - np.max(z, axis=-1, keepdims=True)
    e = np.exp(z)
    return e / np.sum(e, axis=-1, keepdims=True)


def logits(q: np.ndarray, k: np.ndarray, sm_scale: float) -> np.ndarray:
    """q [..., d], k [S, d] -> [..., S]."""
    return (np.asarray(q, dtype=np.float64) @ np.asarray(k, dtype=np.float64).T) * sm_scale


def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, sm_scale: float):
    """Returns (p [..., S], y [..., d])."""
    p = softmax(logits(q, k, sm_scale))
    return p, p @ np.asarray(v, dtype=np.float64)


def tv(p: np.ndarray, ptilde: np.ndarray) -> np.ndarray:
    return 0.5 * np.sum(np.abs(np.asarray(p) - np.asarray(ptilde)), axis=-1)
