"""Threshold gate and exact fallback (the meter loop's gate, Sec. 6; Sec. 4.3).

A query head is gated when its meter exceeds tau.  For tau < 1 the comparison is
on the certified meter min(1, raw) ("certified" gating); for tau >= 1 the meter
is saturated by definition, so the raw risk score is compared instead
("risk-ranked" gating).  Strict ">" ("exceeds").  Routing is per KV head: a KV
head is sent back to the uncompressed path if any of its G query heads is gated
(the any-of-G statistic of Sec. 5).  The fallback replaces the outputs of every
query head of a routed KV head with exact attention from the uncompressed cache.
"""
from __future__ import annotations

import numpy as np


def gate_q(meter: np.ndarray, raw: np.ndarray, tau: float) -> np.ndarray:
    """bool [..., n_q]: query heads whose meter (raw if tau >= 1) exceeds tau."""
    val = np.asarray(raw if tau >= 1.0 else meter, dtype=np.float64)
    return val > tau


def gate_kv(mask_q: np.ndarray, group: int) -> np.ndarray:
    """bool [..., n_kv]: any-of-G routing of query-head decisions."""
    m = np.asarray(mask_q, dtype=bool)
    return m.reshape(m.shape[:-1] + (m.shape[-1] // group, group)).any(axis=-1)


def apply_fallback(out_compressed: np.ndarray, out_exact: np.ndarray, mask_kv: np.ndarray,
                   group: int) -> np.ndarray:
    """out [..., n_q, d]: exact output for every query head of a routed KV head."""
    sel = np.repeat(np.asarray(mask_kv, dtype=bool), group, axis=-1)[..., None]
    return np.where(sel, out_exact, out_compressed)
