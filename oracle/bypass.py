"""Fixed-channel outlier-pair bypass of the dithered INT8 key cache.

TEST INFRASTRUCTURE ONLY (see the package header).

Definitions followed (Sec. 4.2, outlier RoPE pairs; Sec. 6.2, fixed-channel
bypass, where keeping the pairs in fp16 and taking them out of the amax are both
needed; Tables 5 and 6):

* A small set P of m RoPE frequency pairs per (layer, KV head) is kept in fp16
  instead of INT8.  A pair is bypassed whole (both of its channels), because
  RoPE mixes exactly the two channels of a pair (Lemma RoPE band unitarity).
* The set is fixed per (layer, KV head): chosen once from the keys of a prefill
  by pair energy and reused for every token (Sec. 6.2 finds the massive pairs
  stable across tokens).  Reading: the energy of pair j is
  E_j = sum_t ||(k_t)_pair j||^2, which RoPE leaves unchanged; the m pairs of
  largest energy are taken, ties to the lower pair index; P is kept in
  ascending order.
* Step two of the section: the bypassed channels leave the amax, so
  s = fp16_round_up(fl32(max_{c not in P} |x_c| / 126.5)); the other channels are
  quantized with this smaller scale exactly as without bypass (no clipping).
  ``exclude_from_amax=False`` gives Table 5's middle row (bypass alone), which
  the product never uses; it exists to pin the table's finding.
* Storage: the bypassed channels' codes are 0, and their values are stored as
  fp16, rounded to nearest even (the paper's "FP16 outliers"), in the order
  (pair P_0 first channel, P_0 second channel, P_1 first, ...): 2m values, 4m
  bytes per token and KV head (16 B at m = 4).  Values stay within the fp16
  range (|x| <= 65504).
* Reconstruction: xhat_c = s (code_c - xi_c) for c not in P, xhat_c = fp16(x_c)
  for c in P.  The Tier-A witness is the band norm of xhat - x over all channels
  (Eq. witness; the scheme is a black box to it).
* Tier B: the bypassed channels are excluded from the variance term (Sec. 4.2).
  Their residual is the deterministic fp16 rounding error, bounded by
  |fp16(x) - x| <= 2^-11 |fp16(x)| + 2^-25 (half a unit in the last place of a
  normal fp16 value, or of the subnormal spacing 2^-24), so the radius becomes
      u_t = (alpha' + beta') s_t + sm * sum_{c in P} |q_c| (2^-11 |xhat_c| + 2^-25)
  with alpha', beta' computed from q restricted to the channels not in P
  (the union bound applies to the dithered part only; the rest is a worst case).
"""
from __future__ import annotations

import numpy as np

from . import attention, meter as mt
from .fpformats import f16_round_up, f32
from .quantizer import S_DIV, int8_decode

F16_REL = 2.0 ** -11     # half an fp16 ulp, relative to the rounded value
F16_ABS = 2.0 ** -25     # half the fp16 subnormal spacing


def pair_channels(j: int, d: int, layout: str = "half") -> tuple[int, int]:
    """The two channels of RoPE pair j."""
    if layout == "half":
        return j, j + d // 2
    if layout == "interleaved":
        return 2 * j, 2 * j + 1
    raise ValueError(layout)


def bypass_channels(pairs, d: int, layout: str = "half") -> np.ndarray:
    """int [2m]: channels of the pairs in storage order."""
    out = []
    for j in pairs:
        out.extend(pair_channels(int(j), d, layout))
    return np.asarray(out, dtype=np.int64)


def pair_energy(k: np.ndarray, layout: str = "half") -> np.ndarray:
    """E_j = sum over tokens of the squared norm of pair j, float64 [d/2]."""
    k = np.asarray(k, dtype=np.float64)
    d = k.shape[-1]
    e = np.empty(d // 2)
    for j in range(d // 2):
        c0, c1 = pair_channels(j, d, layout)
        e[j] = np.sum(k[:, c0] ** 2) + np.sum(k[:, c1] ** 2)
    return e


def select_pairs(k: np.ndarray, m: int, layout: str = "half") -> np.ndarray:
    """The m pairs of largest energy over the rows of k [S, d] (ties: lower
    index first), returned in ascending order."""
    e = pair_energy(k, layout)
    order = sorted(range(e.size), key=lambda j: (-e[j], j))
    return np.sort(np.asarray(order[:m], dtype=np.int64))


def f16_nearest(x) -> np.ndarray:
    """fp16 round-to-nearest-even of x, as float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float16).astype(np.float64)


def int8_encode_bypass(x: np.ndarray, xi: np.ndarray, chans: np.ndarray,
                       exclude_from_amax: bool = True):
    """Codes (int64 [n, d], 0 on the bypassed channels) and scales (float64 [n])."""
    x = np.asarray(x, dtype=np.float64)
    keep = np.ones(x.shape[-1], dtype=bool)
    keep[np.asarray(chans, dtype=np.int64)] = False
    src = x[:, keep] if exclude_from_amax else x
    s = f16_round_up(f32(np.max(np.abs(src), axis=-1, initial=0.0) / S_DIV))
    with np.errstate(divide="ignore"):
        inv_s = np.where(s > 0, f32(1.0 / np.where(s > 0, s, 1.0)), 0.0)
    y = f32(np.where(keep, x, 0.0) * inv_s[:, None])
    z = f32(y + xi)
    code = np.rint(z).astype(np.int64)
    code[:, ~keep] = 0
    return code, s


def reconstruct(code: np.ndarray, s: np.ndarray, xi: np.ndarray, ovals: np.ndarray,
                chans: np.ndarray) -> np.ndarray:
    """xhat [n, d]: dequantized codes, the stored fp16 values on the bypassed channels."""
    xh = int8_decode(code, s, xi)
    xh[:, np.asarray(chans, dtype=np.int64)] = ovals
    return xh


def quantize_bypass(x: np.ndarray, xi: np.ndarray, chans: np.ndarray,
                    exclude_from_amax: bool = True):
    """(code, s, ovals [n, 2m], xhat) of rows x [n, d] with dither xi [n, d]."""
    x = np.asarray(x, dtype=np.float64)
    code, s = int8_encode_bypass(x, xi, chans, exclude_from_amax)
    ovals = f16_nearest(x[:, np.asarray(chans, dtype=np.int64)])
    return code, s, ovals, reconstruct(code, s, xi, ovals, chans)


def rounding_bound(ovals) -> np.ndarray:
    """Bound on |fp16(x) - x| from the stored value fp16(x)."""
    return F16_REL * np.abs(np.asarray(ovals, dtype=np.float64)) + F16_ABS


def radius(q: np.ndarray, s_tok: np.ndarray, ovals: np.ndarray, chans: np.ndarray,
           sm_scale: float, n_tokens: int, dloc: float) -> np.ndarray:
    """Tier-B radius u_t [S] with the bypassed channels out of the variance term."""
    q = np.asarray(q, dtype=np.float64)
    s_tok = np.asarray(s_tok, dtype=np.float64)
    keep = np.ones(q.shape[-1], dtype=bool)
    keep[np.asarray(chans, dtype=np.int64)] = False
    qk = q[keep]
    var = sm_scale ** 2 / 12.0 * np.sum(qk ** 2) * s_tok ** 2
    bias = sm_scale * s_tok * np.sum(np.abs(qk)) / 256.0
    det = sm_scale * rounding_bound(ovals) @ np.abs(q[np.asarray(chans, dtype=np.int64)])
    return bias + np.sqrt(2.0 * var * np.log(2.0 * n_tokens / dloc)) + det


def tierb_decode(q: np.ndarray, khat: np.ndarray, vhat: np.ndarray, ks: np.ndarray,
                 ko: np.ndarray, chans: np.ndarray, sm_scale: float, dloc: float) -> dict:
    """Tier-B decode step over a bypassed cache.

    q [n_q, d]; khat, vhat [S, n_kv, d]; ks [S, n_kv] key scales; ko [S, n_kv, 2m]
    stored fp16 values; chans [n_kv, 2m] their channels.
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
        u = radius(q[h], ks[:, kv], ko[:, kv], chans[kv], sm_scale, S, dloc)
        out[h] = p @ vhat[:, kv]
        raw[h] = mt.raw_from_am1(mt.a_minus_one_logits(z, u))
        uu[h] = u
    return {"out": out, "raw": raw, "meter": mt.meter(raw), "u": uu}
