"""Per-token, per-32-channel-group scales for the dithered INT8 cache.

TEST INFRASTRUCTURE ONLY (see the package header).

Definitions followed (Sec. 6.2, storage side: the serving store keeps, for each
token, one scale per run of G_c consecutive channels, G_c = 32 by default; Table 4 (granularity):
272 bytes per token and KV head for K + V at G_c = 32, i.e. per side 128 codes
and four 2-byte scales; Sec. 4.2 subtractive dither and Tier B, whose proxy sums
q_c^2 s_c^2 over the channels):

* Groups: channels 32g .. 32g+31 of the stored vector (d/32 groups).
* Each group g of each token has its own fp16 scale, formed like the token
  scale of the plain quantizer (Sec. 4.2, s = amax / (Q - 1/2); reading: fp32
  quotient rounded up to fp16):
      s_g = fp16_round_up(fl32(amax_g / 126.5)),
  amax_g the group's largest magnitude over its quantized channels (0 for an
  all-zero group, whose codes are then 0).
* Quantization with the stored scale, operation by operation in fp32:
      inv_g = fl32(1 / s_g),  y = fl32(x * inv_g),  z = fl32(y + xi),
      code  = round-half-to-even(z)
  (|y| <= 126.5 (1 + 2^-24) since s_g >= amax_g / 126.5, so no code is clipped);
  decoding is exact: xhat = s_g (code - xi).
* Bypassed pairs (``bypass``) leave the group amaxes; their codes are 0 and their
  values are the stored fp16 values.
* Tier B: the residual of channel c is the lattice-dither residual of step s_{g(c)},
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


def bytes_per_token_head(d: int, group: int | None, code_bytes: int = 1, scale_bytes: int = 2) -> int:
    """K + V storage of one token and KV head: codes plus one scale per group and
    side (group None: one scale per token and side), the byte account of Table 4."""
    per_side = d * code_bytes + scale_bytes * (1 if group is None else d // group)
    return 2 * per_side


def keep_mask(d: int, chans=None) -> np.ndarray:
    """bool [d]: channels quantized as INT8 (not bypassed)."""
    keep = np.ones(d, dtype=bool)
    if chans is not None:
        keep[np.asarray(chans, dtype=np.int64)] = False
    return keep


def scales(x: np.ndarray, chans=None) -> np.ndarray:
    """Group scales s [n, d/32] (fp16 round-up of fl32(amax_g / 126.5), as float64)."""
    x = np.asarray(x, dtype=np.float64)
    n, d = x.shape
    ax = np.where(keep_mask(d, chans), np.abs(x), 0.0)
    ag = ax.reshape(n, d // GROUP, GROUP).max(axis=2)
    return f16_round_up(f32(ag / S_DIV))


def channel_steps(s: np.ndarray) -> np.ndarray:
    """Per-channel step s_{g(c)}, [n, d]."""
    return np.repeat(np.asarray(s, dtype=np.float64), GROUP, axis=-1)


def encode(x: np.ndarray, xi: np.ndarray, chans=None):
    """Codes (int64 [n, d]) and group scales s [n, d/32]."""
    x = np.asarray(x, dtype=np.float64)
    keep = keep_mask(x.shape[-1], chans)
    s = scales(x, chans)
    with np.errstate(divide="ignore"):
        inv = np.where(s > 0, f32(1.0 / np.where(s > 0, s, 1.0)), 0.0)
    y = f32(np.where(keep, x, 0.0) * channel_steps(inv))
    z = f32(y + xi)
    code = np.rint(z).astype(np.int64)
    code[:, ~keep] = 0
    return code, s


def decode(code: np.ndarray, s: np.ndarray, xi: np.ndarray) -> np.ndarray:
    """xhat = s_g (code - xi), exact in float64."""
    return channel_steps(s) * (np.asarray(code, dtype=np.float64) - xi)


def quantize(x: np.ndarray, xi: np.ndarray, chans=None):
    """(code, s, ovals or None, xhat) of rows x [n, d] with dither xi [n, d]."""
    x = np.asarray(x, dtype=np.float64)
    code, s = encode(x, xi, chans)
    xh = decode(code, s, xi)
    ovals = None
    if chans is not None and len(chans):
        ch = np.asarray(chans, dtype=np.int64)
        ovals = bypass.f16_nearest(x[:, ch])
        xh[:, ch] = ovals
    return code, s, ovals, xh


def radius(q: np.ndarray, s: np.ndarray, sm_scale: float, n_tokens: int, dloc: float, ovals=None,
           chans=None) -> np.ndarray:
    """Tier-B radius u_t [S] of one query head over group-scaled keys (s [S, d/32])."""
    q = np.asarray(q, dtype=np.float64)
    keep = keep_mask(q.shape[-1], chans)
    qk = np.where(keep, q, 0.0)
    sc = channel_steps(s)                                   # [S, d]
    var = sm_scale ** 2 / 12.0 * (sc ** 2 @ qk ** 2)
    bias = sm_scale * (sc @ np.abs(qk)) / 256.0
    u = bias + np.sqrt(2.0 * var * np.log(2.0 * n_tokens / dloc))
    if chans is not None and len(chans):
        u = u + sm_scale * bypass.rounding_bound(ovals) @ np.abs(q[np.asarray(chans, dtype=np.int64)])
    return u


def tierb_decode(q: np.ndarray, khat: np.ndarray, vhat: np.ndarray, ks: np.ndarray, sm_scale: float,
                 dloc: float, ko=None, chans=None) -> dict:
    """Tier-B decode step over a group-scaled cache.

    q [n_q, d]; khat, vhat [S, n_kv, d]; ks [S, n_kv, d/32] key group scales; with
    bypassed pairs ko [S, n_kv, 2m] and chans [n_kv, 2m].
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
        u = radius(q[h], ks[:, kv], sm_scale, S, dloc,
                   None if ko is None else ko[:, kv], None if chans is None else chans[kv])
        out[h] = p @ vhat[:, kv]
        raw[h] = mt.raw_from_am1(mt.a_minus_one_logits(z, u))
        uu[h] = u
    return {"out": out, "raw": raw, "meter": mt.meter(raw), "u": uu}
