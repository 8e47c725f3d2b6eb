"""Tier-B sub-Gaussian certificate of the dithered INT8 cache (Sec. 4.2, Tier B).

TEST INFRASTRUCTURE ONLY (see the package header).

* Lemma (uniform sub-Gaussian proxy), Sec. 4.2: for X ~ U[-a, a],
      E[e^{lambda X}] = sinh(lambda a) / (lambda a) <= e^{lambda^2 a^2 / 6};
  the subtractive-dither residual of step s (a = s/2) is sub-Gaussian with
  proxy s^2 / 12, its variance.  ``mgf_uniform`` is the left side.
* Logit-error proxy (same paragraph; Sec. 6.2 storage side computes it in the
  kernel): with eps_t = sm * q . r_t,
      varsigma_t^2 = (sm^2 / 12) * sum_c q_c^2 s_{c,t}^2,
  which for one scale per token is (sm * ||q|| * s_t)^2 / 12.
* Radius: with probability at least 1 - delta_loc jointly over the S tokens,
  |eps_t| <= u_t = sqrt(2 varsigma_t^2 log(2S / delta_loc))  (a union bound of
  the two-sided sub-Gaussian tail 2 exp(-u^2 / (2 varsigma^2)) over S tokens).
  With one scale per token u_t = alpha * s_t, alpha = sm ||q|| sqrt(2 log(2S /
  delta_loc) / 12): the square root leaves the token loop (Sec. 6.2, serving
  integration with one scalar scale per token).
* Lattice bias.  The Lemma is stated for a continuous dither; the cache's dither
  is the 8-bit midpoint lattice (xi = (u - 127.5)/256).  For a fixed input its
  residual over the 256 dither values is a lattice of spacing s/256 whose mean is
  at most s/512 in magnitude (a little more where fp32 rounding moves one code
  across a rounding boundary), so per channel
      E[e^{lambda r}] <= e^{|lambda| s / 256 + lambda^2 s^2 / 24}
  (checked by enumerating the dither for each input in the tests), and the
  radius gains the term b_t = sm * s_t * ||q||_1 / 256:
      u_t = b_t + sqrt(2 varsigma_t^2 log(2S / delta_loc)) = (alpha + beta) s_t,
      beta = sm ||q||_1 / 256.
* Request-level budget (Sec. 4.2): delta_loc = delta_req / (L * H * T) over
  layers, query heads and decode steps.
* Certificate: the radius takes the place of the witness bound c_t in the
  e-form propagation, A = sum_t ptilde_t e^{u_t}, raw = (A^2 - 1)/2,
  meter = min(1, raw) (Theorem sound replacement; Sec. 4.3).  The guarantee is
  probabilistic and stated for non-adaptive queries (Sec. 4.2, scope).

No witness is read: u_t depends only on the stored key scales and the query.
"""
from __future__ import annotations

import numpy as np

from . import attention, meter as mt


def mgf_uniform(lam, a) -> np.ndarray:
    """E[e^{lambda X}] for X ~ U[-a, a]: sinh(lambda a) / (lambda a), 1 at 0."""
    x = np.asarray(lam, dtype=np.float64) * np.asarray(a, dtype=np.float64)
    with np.errstate(invalid="ignore", divide="ignore", over="ignore"):
        r = np.sinh(x) / x
    return np.where(x == 0, 1.0, r)


def delta_loc(delta_req: float, n_layers: int, n_heads: int, n_steps: int) -> float:
    """Per-(layer, head, step) failure budget of a request-level budget."""
    return float(delta_req) / (n_layers * n_heads * n_steps)


def variance_proxy(q: np.ndarray, s: np.ndarray, sm_scale: float) -> np.ndarray:
    """varsigma^2 = (sm^2/12) sum_c q_c^2 s_c^2.

    q [d]; s [..., d] per-channel scales (a per-token scale broadcast over d).
    """
    q = np.asarray(q, dtype=np.float64)
    s = np.asarray(s, dtype=np.float64)
    return sm_scale ** 2 / 12.0 * np.sum(q ** 2 * s ** 2, axis=-1)


def lattice_bias(q: np.ndarray, s_tok: np.ndarray, sm_scale: float) -> np.ndarray:
    """b_t = sm * s_t * ||q||_1 / 256: bound on |E eps_t| from the lattice dither."""
    return sm_scale * np.asarray(s_tok, dtype=np.float64) * np.sum(np.abs(np.asarray(q, dtype=np.float64))) / 256.0


def radius(q: np.ndarray, s_tok: np.ndarray, sm_scale: float, n_tokens: int, dloc: float) -> np.ndarray:
    """u_t = b_t + sqrt(2 varsigma_t^2 log(2S/delta_loc)) for per-token scales s_tok [S]."""
    s_tok = np.asarray(s_tok, dtype=np.float64)
    d = np.asarray(q).shape[-1]
    var = variance_proxy(q, np.repeat(s_tok[:, None], d, axis=1), sm_scale)
    return lattice_bias(q, s_tok, sm_scale) + np.sqrt(2.0 * var * np.log(2.0 * n_tokens / dloc))


def alpha(q: np.ndarray, sm_scale: float, n_tokens: int, dloc: float) -> float:
    """The per-head factor with u_t = alpha * s_t (one scale per token), bias included."""
    q = np.asarray(q, dtype=np.float64)
    return sm_scale * (np.sum(np.abs(q)) / 256.0 +
                       np.linalg.norm(q) * np.sqrt(2.0 * np.log(2.0 * n_tokens / dloc) / 12.0))


def tierb_decode(q: np.ndarray, khat: np.ndarray, vhat: np.ndarray, ks: np.ndarray,
                 sm_scale: float, dloc: float) -> dict:
    """One metered decode step under the Tier-B certificate.

    q [n_q, d]; khat, vhat [S, n_kv, d] reconstructions; ks [S, n_kv] stored key
    scales.  S is the number of attended tokens (the union bound's S).
    Returns out [n_q, d], raw [n_q], meter [n_q], ptilde [n_q, S], u [n_q, S].
    """
    q = np.asarray(q, dtype=np.float64)
    n_q, d = q.shape
    n_kv = khat.shape[1]
    g = n_q // n_kv
    S = khat.shape[0]
    out = np.empty((n_q, d))
    raw = np.empty(n_q)
    pt = np.empty((n_q, S))
    uu = np.empty((n_q, S))
    for h in range(n_q):
        kv = h // g
        z = attention.logits(q[h], khat[:, kv], sm_scale)
        p = attention.softmax(z)
        u = radius(q[h], ks[:, kv], sm_scale, S, dloc)
        out[h] = p @ vhat[:, kv]
        raw[h] = mt.raw_from_am1(mt.a_minus_one_logits(z, u))
        pt[h], uu[h] = p, u
    return {"out": out, "raw": raw, "meter": mt.meter(raw), "ptilde": pt, "u": uu}
