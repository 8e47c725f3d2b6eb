"""Tier-A meter: per-token logit bounds, the e-form TV bound, saturation reporting.

* ``logit_bound`` -- Theorem (sound black-box logit bound), Sec. 4.1:
      c_t = (1/sqrt d) * sum_b ||q_b|| * w_{t,b}
  with q the post-RoPE query, w the stored (fp16) witness and the same band map
  as the witness.  Cauchy-Schwarz within each band gives |q . r_t|/sqrt d <= c_t.
* ``a_minus_one`` / ``raw_bound`` -- Theorem (sound replacement), Sec. 3:
      A = E_ptilde[e^c],  TV(p, ptilde) <= (A^2 - 1)/2.
  Evaluated as A - 1 = sum_t ptilde_t * expm1(c_t) and (A^2-1)/2 = (A-1)(2+(A-1))/2,
  which keeps relative precision when A is close to 1.  Overflow gives +inf,
  which is still a valid (vacuous) bound (Sec. 3, last paragraph; Sec. 6.2,
  telemetry: an overflowed certificate is +inf, counted over threshold).
* ``meter`` -- Sec. 4.3: the reported meter is min(1, raw); raw above 1 is a risk
  score, not a guarantee.
* ``flawed_bound`` -- Eq. (flawed), kept only as the regression value of the
  Sec. 3 counterexample.
* ``two_sided_bound`` -- Proposition (two-sided form), Sec. 4.3, for soundness tests.

The expectation is under ptilde, the *compressed* attention distribution, which
is what a decode kernel has (Theorem sound replacement; the meter-loop read path).
"""
from __future__ import annotations

import numpy as np

from .quantizer import band_norms


def logit_bound(q: np.ndarray, w: np.ndarray, sm_scale: float, n_bands: int,
                layout: str = "half") -> np.ndarray:
    """q [..., d], w [S, B] -> c [..., S]."""
    qn = band_norms(q, n_bands, layout)                  # [..., B]
    return sm_scale * (qn @ np.asarray(w, dtype=np.float64).T)


def a_minus_one(ptilde: np.ndarray, c: np.ndarray) -> np.ndarray:
    with np.errstate(over="ignore", invalid="ignore"):
        terms = np.asarray(ptilde, dtype=np.float64) * np.expm1(np.asarray(c, dtype=np.float64))
        # ptilde_t == 0 with an overflowing expm1 would be 0*inf; such a token has
        # no attention mass in float64 and contributes nothing.
        terms = np.where(np.asarray(ptilde) == 0, 0.0, terms)
        return np.sum(terms, axis=-1)


def a_minus_one_logits(logits: np.ndarray, c: np.ndarray) -> np.ndarray:
    """A - 1 from the compressed logits (ptilde = softmax(logits)) in the log
    domain: ptilde_t e^{c_t} - ptilde_t = exp(log ptilde_t + c_t) - ptilde_t, so a
    token whose mass underflows but whose bound is huge still counts (Sec. 3:
    evaluate A in the log domain, never truncate c)."""
    z = np.asarray(logits, dtype=np.float64)
    c = np.asarray(c, dtype=np.float64)
    m = np.max(z, axis=-1, keepdims=True)
    lse = m + np.log(np.sum(np.exp(z - m), axis=-1, keepdims=True))
    lp = z - lse
    with np.errstate(over="ignore", invalid="ignore"):
        big = np.exp(lp + c) - np.exp(lp)
        small = np.exp(lp) * np.expm1(c)
        terms = np.where(c > 1.0, big, small)
        return np.sum(terms, axis=-1)


def raw_from_am1(am1: np.ndarray) -> np.ndarray:
    am1 = np.asarray(am1, dtype=np.float64)
    with np.errstate(over="ignore", invalid="ignore"):
        raw = 0.5 * am1 * (2.0 + am1)
    return np.where(np.isfinite(raw), raw, np.inf)


def raw_bound(ptilde: np.ndarray, c: np.ndarray) -> np.ndarray:
    """(A^2 - 1)/2 with A = E_ptilde[e^c] (Theorem sound replacement)."""
    return raw_from_am1(a_minus_one(ptilde, c))


def meter(raw: np.ndarray) -> np.ndarray:
    """Reported meter min(1, raw) (Sec. 4.3)."""
    return np.minimum(1.0, np.asarray(raw, dtype=np.float64))


def flawed_bound(ptilde: np.ndarray, c: np.ndarray) -> np.ndarray:
    """Eq. (flawed): 1/2 e^{2 c_max} (E|c - cbar| + cbar (e^{c_max} - 1)); unsound."""
    p = np.asarray(ptilde, dtype=np.float64)
    c = np.asarray(c, dtype=np.float64)
    cbar = np.sum(p * c, axis=-1, keepdims=True)
    cmax = np.max(c, axis=-1, keepdims=True)
    disp = np.sum(p * np.abs(c - cbar), axis=-1, keepdims=True)
    return (0.5 * np.exp(2 * cmax) * (disp + cbar * np.expm1(cmax)))[..., 0]


def two_sided_bound(ptilde: np.ndarray, c: np.ndarray) -> np.ndarray:
    """Proposition (two-sided form): 1/2 (A/A^- - A^-/A), A^- = E_ptilde[e^{-c}]."""
    p = np.asarray(ptilde, dtype=np.float64)
    c = np.asarray(c, dtype=np.float64)
    a = np.sum(p * np.exp(c), axis=-1)
    am = np.sum(p * np.exp(-c), axis=-1)
    return 0.5 * (a / am - am / a)
