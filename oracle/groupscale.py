"""Per-token scales over 32-channel groups for the dithered INT8 cache.

TEST INFRASTRUCTURE ONLY (see the package header).

Definitions followed (Sec. 6.2, storage side: "scale per token, per group of G_c
channels", G_c = 32 as the default, Table 4 (granularity); Sec. 4.2 subtractive
dither and Tier B, whose proxy sums q_c^2 s_c^2 over the channels):

* Groups: channels 32g .. 32g+31 of the stored vector (d/32 groups).
* Storage reading.  The paper does not state how the group scales are stored.
  Here one fp16 scale per token and tensor (the token scale of the plain
  quantizer, s = fp16_round_up(fl32(amax / 126.5)) over the kept channels) and
  one exponent e_g in [0, 14] per group: the group's scale is s_g = s * 2^-e_g,
  with e_g the largest exponent such that amax_g * 2^e_g <= amax (amax_g the
  group's largest magnitude over its kept channels; 14 for an all-zero group).
  The group scale is then within a factor 2 of amax_g / 126.5 (or at the 2^-14
  floor), and power-of-two ratios keep the decode's operands exact: a code times
  2^-e, e <= 14, is still an exact normal fp16 number.
* Quantization with the stored scales, operation by operation in fp32:
      inv_g = fl32(1/s) * 2^e_g   (exact: a power-of-two scaling)
      y     = fl32(x * inv_g)
      z     = fl32(y + xi)
      code  = round-half-to-even(z)
  Since amax_g 2^e_g <= amax, |y| is bounded exactly as in the plain quantizer,
  so no code is ever clipped.  Decoding is exact: xhat = s 2^-e_g (code - xi).
* Bypassed pairs (``bypass``) leave both the token amax and the group amaxes;
  their codes are 0 and their values are the stored fp16 values.
* Tier B: the residual of channel c is the lattice-dither residual of step s_g(c),
  so varsigma_t^2 = (sm^2 / 12) sum_g s_{t,g}^2 ||q_g||^2 and the lattice bias is
  sm sum_g s_{t,g} ||q_g||_1 / 256 (both over the kept channels); the bypassed
  channels add their fp16 rounding term as in ``bypass.radius``.
"""
from __future__ import annotations

import numpy as np

from . import attention, bypass, meter as mt
from .fpformats import f16_round_up, f32
from .quantizer import S_DIV

GROUP = 32
E_MAX = 14


def keep_mask(d: int, chans=None) -> np.ndarray:
    """bool [d]: channels quantized as INT8 (not bypassed)."""
    keep = np.ones(d, dtype=bool)
    if chans is not None:
        keep[np.asarray(chans, dtype=np.int64)] = False
    return keep


def scales(x: np.ndarray, chans=None):
    """Token scale s [n] (fp16 round-up, as float64) and group exponents e [n, d/32]."""
    x = np.asarray(x, dtype=np.float64)
    n, d = x.shape
    ax = np.where(keep_mask(d, chans), np.abs(x), 0.0)
    amax = ax.max(axis=1)
    s = f16_round_up(f32(amax / S_DIV))
    ag = ax.reshape(n, d // GROUP, GROUP).max(axis=2)               # group amaxes [n, d/32]
    # the largest k <= E_MAX with ag 2^k <= amax: the condition holds for every
    # smaller k once it holds for k, so e counts the k = 1 .. E_MAX for which it holds
    e = np.zeros((n, d // GROUP), dtype=np.int64)
    for k in range(1, E_MAX + 1):
        e += (ag * 2.0 ** k <= amax[:, None]).astype(np.int64)
    return s, e


def group_steps(s: np.ndarray, e: np.ndarray) -> np.ndarray:
    """Per-channel scale s_c = s 2^-e_{g(c)}, [n, d]."""
    return np.repeat(np.asarray(s, dtype=np.float64)[:, None] * 2.0 ** -np.asarray(e, dtype=np.float64),
                     GROUP, axis=1)


def encode(x: np.ndarray, xi: np.ndarray, chans=None):
    """Codes (int64 [n, d]), token scales s [n] and group exponents e [n, d/32]."""
    x = np.asarray(x, dtype=np.float64)
    keep = keep_mask(x.shape[-1], chans)
    s, e = scales(x, chans)
    with np.errstate(divide="ignore"):
        inv_s = np.where(s > 0, f32(1.0 / np.where(s > 0, s, 1.0)), 0.0)
    inv_c = np.repeat(inv_s[:, None] * 2.0 ** e, GROUP, axis=1)
    y = f32(np.where(keep, x, 0.0) * inv_c)
    z = f32(y + xi)
    code = np.rint(z).astype(np.int64)
    code[:, ~keep] = 0
    return code, s, e


def decode(code: np.ndarray, s: np.ndarray, e: np.ndarray, xi: np.ndarray) -> np.ndarray:
    """xhat = s 2^-e_g (code - xi), exact in float64."""
    return group_steps(s, e) * (np.asarray(code, dtype=np.float64) - xi)


def quantize(x: np.ndarray, xi: np.ndarray, chans=None):
    """(code, s, e, ovals or None, xhat) of rows x [n, d] with dither xi [n, d]."""
    x = np.asarray(x, dtype=np.float64)
    code, s, e = encode(x, xi, chans)
    xh = decode(code, s, e, xi)
    ovals = None
    if chans is not None and len(chans):
        ch = np.asarray(chans, dtype=np.int64)
        ovals = bypass.f16_nearest(x[:, ch])
        xh[:, ch] = ovals
    return code, s, e, ovals, xh


def radius(q: np.ndarray, s_tok: np.ndarray, e: np.ndarray, sm_scale: float, n_tokens: int,
           dloc: float, ovals=None, chans=None) -> np.ndarray:
    """Tier-B radius u_t [S] of one query head over group-scaled keys."""
    q = np.asarray(q, dtype=np.float64)
    keep = keep_mask(q.shape[-1], chans)
    qk = np.where(keep, q, 0.0)
    sc = group_steps(s_tok, e)                              # [S, d]
    var = sm_scale ** 2 / 12.0 * (sc ** 2 @ qk ** 2)
    bias = sm_scale * (sc @ np.abs(qk)) / 256.0
    u = bias + np.sqrt(2.0 * var * np.log(2.0 * n_tokens / dloc))
    if chans is not None and len(chans):
        u = u + sm_scale * bypass.rounding_bound(ovals) @ np.abs(q[np.asarray(chans, dtype=np.int64)])
    return u


def tierb_decode(q: np.ndarray, khat: np.ndarray, vhat: np.ndarray, ks: np.ndarray, ke: np.ndarray,
                 sm_scale: float, dloc: float, ko=None, chans=None) -> dict:
    """Tier-B decode step over a group-scaled cache.

    q [n_q, d]; khat, vhat [S, n_kv, d]; ks [S, n_kv] token scales; ke [S, n_kv, d/32]
    group exponents; with bypassed pairs ko [S, n_kv, 2m] and chans [n_kv, 2m].
    Returns out, raw, meter [n_q] and u [n_q, S].
    """
    q = np.asarray(q, dtype=np.float64)
    n_q, d = q.shape
    S, n_kv = khat.shape[:2]
    g = n_q // n_kv
    out = np.empty((n_q, d))
    raw = np.empty(n_q)
    uu = np.empty((n_q, S))
    for h in range(n_q):
        kv = h // g
        z = attention.logits(q[h], khat[:, kv], sm_scale)
        p = attention.softmax(z)
        u = radius(q[h], ks[:, kv], ke[:, kv], sm_scale, S, dloc,
                   None if ko is None else ko[:, kv], None if chans is None else chans[kv])
        out[h] = p @ vhat[:, kv]
        raw[h] = mt.raw_from_am1(mt.a_minus_one_logits(z, u))
        uu[h] = u
    return {"out": out, "raw": raw, "meter": mt.meter(raw), "u": uu}
