"""One metered decode step, composed from the oracle's definitions (the meter loop, Sec. 6).

Write path (once per token): quantize k -> khat with a scheme, store the witness
w_{t,b} of the key residual (Tier A).  Read path, per query head h of KV head
kv = h // G: compressed attention over the reconstructed cache, the per-token
bounds c_t from the stored witness, A - 1 = E_ptilde[e^c - 1], raw = (A^2-1)/2,
meter = min(1, raw).  Gate: see ``gate``.  All float64, one sequence at a time,
no blocking or splitting of the token axis.
"""
from __future__ import annotations

import numpy as np

from . import attention, bypass, groupscale, meter as mt, quantizer, value
from .philox import dither_values

KINDS = ("int8_dither", "fp8_raw", "bf16")


def write_cache(kind: str, k: np.ndarray, v: np.ndarray, slots: np.ndarray, layer: int,
                seed: int, n_bands: int, layout: str = "half", pairs=None,
                group_scales: bool = False) -> dict:
    """Quantize one sequence's tokens for every KV head.

    k, v: stored inputs [S, n_kv, d] (float); slots: int [S] physical slots.
    pairs: int [n_kv, m] bypassed RoPE pairs of the keys (int8 only; ``bypass``).
    group_scales: int8 with one fp16 scale per token and 32-channel group
    (``groupscale``).
    Returns reconstructions khat/vhat [S, n_kv, d], key witness kw [S, n_kv, B],
    for the quantized kinds the value residual and value norms vr, vn [S, n_kv]
    (``value``) and, for int8, codes and scales ks, vs ([S, n_kv], or with group
    scales [S, n_kv, d/32]); with pairs also the stored fp16 values ko [S, n_kv, 2m]
    and their channels chans [n_kv, 2m].
    """
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    S, n_kv, d = k.shape
    out = {"khat": np.empty_like(k), "vhat": np.empty_like(v),
           "kw": np.zeros((S, n_kv, n_bands))}
    if group_scales and kind != "int8_dither":
        raise ValueError("group scales are defined for the int8 cache")
    if kind == "int8_dither":
        for key in ("kcode", "vcode"):
            out[key] = np.empty((S, n_kv, d), dtype=np.int64)
        for key in ("ks", "vs"):
            out[key] = np.empty((S, n_kv, d // groupscale.GROUP) if group_scales else (S, n_kv))
    if pairs is not None:
        if kind != "int8_dither":
            raise ValueError("the outlier bypass is defined for the int8 cache")
        pairs = np.asarray(pairs, dtype=np.int64)
        out["chans"] = np.stack([bypass.bypass_channels(pairs[h], d, layout) for h in range(n_kv)])
        out["ko"] = np.empty((S, n_kv, out["chans"].shape[1]))
    for h in range(n_kv):
        if kind == "int8_dither" and group_scales:
            xi = dither_values(slots, d, layer, h, seed)
            ch = None if pairs is None else out["chans"][h]
            kc, ks, ko, kh = groupscale.quantize(k[:, h], xi, ch)
            vc, vs, _, vh = groupscale.quantize(v[:, h], xi)
            out["kcode"][:, h], out["ks"][:, h] = kc, ks
            out["vcode"][:, h], out["vs"][:, h] = vc, vs
            if ko is not None:
                out["ko"][:, h] = ko
        elif kind == "int8_dither" and pairs is not None:
            xi = dither_values(slots, d, layer, h, seed)
            kc, ks, ko, kh = bypass.quantize_bypass(k[:, h], xi, out["chans"][h])
            vc, vs, _, vh = quantizer.int8_quantize_slots(v[:, h], slots, layer, h, seed)
            out["kcode"][:, h], out["ks"][:, h], out["ko"][:, h] = kc, ks, ko
            out["vcode"][:, h], out["vs"][:, h] = vc, vs
        elif kind == "int8_dither":
            kc, ks, _, kh = quantizer.int8_quantize_slots(k[:, h], slots, layer, h, seed)
            vc, vs, _, vh = quantizer.int8_quantize_slots(v[:, h], slots, layer, h, seed)
            out["kcode"][:, h], out["ks"][:, h] = kc, ks
            out["vcode"][:, h], out["vs"][:, h] = vc, vs
        elif kind == "fp8_raw":
            kh, vh = quantizer.fp8_raw(k[:, h]), quantizer.fp8_raw(v[:, h])
        elif kind == "bf16":
            kh, vh = k[:, h], v[:, h]
        else:
            raise ValueError(kind)
        out["khat"][:, h], out["vhat"][:, h] = kh, vh
        if kind != "bf16":
            out["kw"][:, h] = quantizer.witness(k[:, h], kh, n_bands, layout)
    if kind != "bf16":   # value side: stored residual norm (up) and value norm (down)
        out["vr"] = value.value_residual(v, out["vhat"])
        out["vn"] = value.value_norm(v)
    return out


def metered_decode(q: np.ndarray, khat: np.ndarray, vhat: np.ndarray, kw: np.ndarray,
                   sm_scale: float, n_bands: int, layout: str = "half") -> dict:
    """q [n_q, d]; khat, vhat [S, n_kv, d]; kw [S, n_kv, B] stored witness.

    Returns out [n_q, d], raw [n_q], meter [n_q], ptilde [n_q, S], c [n_q, S].
    """
    q = np.asarray(q, dtype=np.float64)
    n_q, d = q.shape
    n_kv = khat.shape[1]
    g = n_q // n_kv
    S = khat.shape[0]
    out = np.empty((n_q, d))
    raw = np.empty(n_q)
    pt = np.empty((n_q, S))
    cc = np.empty((n_q, S))
    for h in range(n_q):
        kv = h // g
        z = attention.logits(q[h], khat[:, kv], sm_scale)
        p = attention.softmax(z)
        c = mt.logit_bound(q[h], kw[:, kv], sm_scale, n_bands, layout)
        out[h] = p @ vhat[:, kv]
        raw[h] = mt.raw_from_am1(mt.a_minus_one_logits(z, c))
        pt[h], cc[h] = p, c
    return {"out": out, "raw": raw, "meter": mt.meter(raw), "ptilde": pt, "c": cc}


def exact_decode(q: np.ndarray, k: np.ndarray, v: np.ndarray, sm_scale: float) -> dict:
    """Uncompressed attention: q [n_q, d], k, v [S, n_kv, d] -> out [n_q, d], p [n_q, S]."""
    q = np.asarray(q, dtype=np.float64)
    n_q, d = q.shape
    g = n_q // k.shape[1]
    out = np.empty((n_q, d))
    p_all = np.empty((n_q, k.shape[0]))
    for h in range(n_q):
        p, y = attention.attend(q[h], k[:, h // g], v[:, h // g], sm_scale)
        out[h], p_all[h] = y, p
    return {"out": out, "p": p_all}


def true_tv(q: np.ndarray, k: np.ndarray, khat: np.ndarray, sm_scale: float) -> np.ndarray:
    """TV(p, ptilde) per query head (Sec. 3): p from exact keys, ptilde from khat."""
    p = exact_decode(q, k, k, sm_scale)["p"]
    q = np.asarray(q, dtype=np.float64)
    g = q.shape[0] // k.shape[1]
    ptl = np.stack([attention.softmax(attention.logits(q[h], khat[:, h // g], sm_scale))
                    for h in range(q.shape[0])])
    return attention.tv(p, ptl)
