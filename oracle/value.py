"""Value side of the certificate and the joint K+V event.

TEST INFRASTRUCTURE ONLY (see the package header).

Definitions followed:

* Output bound (Sec. 3, setup): with p, ptilde the exact and compressed
  attention distributions and rho_t = ||vhat_t - v_t|| the value reconstruction
  error of token t,
      ||y - yhat|| <= 2 TV(p, ptilde) max_t ||v_t|| + sum_t ptilde_t rho_t
  (y - yhat = sum_t (p_t - ptilde_t) v_t + sum_t ptilde_t (v_t - vhat_t), then the
  triangle inequality).  The value term is deterministic given ptilde and
  consumes no probability budget (Sec. 4.2, value side; Sec. 5, limitations).
* Joint event (Sec. 4.2): pass_K and pass_V per (layer, KV head, position), with
  tau_K = 0.2 and tau_V = 0.05 (Sec. 5 defaults, derived by walking an output
  tolerance back through the output bound, Sec. 7).
* Reading (the paper names pass_V's quantity only through that derivation): the
  value meter is the value term in units of the largest value norm,
      meter_V = sum_t ptilde_t rho_t / max_t ||v_t||,
  so that ||y - yhat|| / max_t ||v_t|| <= 2 meter_K + meter_V, the same units as
  the key side's 2 TV; pass_V is meter_V <= tau_V, and a query head is routed
  when pass_K and pass_V do not both hold.
* Storage: rho_t rounded up to fp16 and ||v_t|| rounded down to fp16, both from
  float64 norms, one of each per (token, KV head): the stored rho is never below
  the true error and the stored norm never above the true norm, so the value
  meter computed from them is never below the true ratio.  With every stored
  norm 0 the meter is 0 when the numerator is 0 and +inf otherwise.
"""
from __future__ import annotations

import numpy as np

from . import attention, gate as ogate, meter as mt
from .fpformats import f16_round_down, f16_round_up


def value_residual(v: np.ndarray, vhat: np.ndarray) -> np.ndarray:
    """Stored rho [...]: fp16 round-up of ||vhat - v|| over the last axis."""
    r = np.asarray(vhat, dtype=np.float64) - np.asarray(v, dtype=np.float64)
    return f16_round_up(np.sqrt(np.sum(r * r, axis=-1)))


def value_norm(v: np.ndarray) -> np.ndarray:
    """Stored ||v|| [...]: fp16 round-down of the float64 norm over the last axis."""
    v = np.asarray(v, dtype=np.float64)
    return f16_round_down(np.sqrt(np.sum(v * v, axis=-1)))


def value_meter(ptilde: np.ndarray, rho: np.ndarray, vnorm: np.ndarray) -> float:
    """sum_t ptilde_t rho_t / max_t vnorm_t (0/0 = 0, x/0 = +inf)."""
    e = float(np.dot(np.asarray(ptilde, dtype=np.float64), np.asarray(rho, dtype=np.float64)))
    m = float(np.max(vnorm)) if np.size(vnorm) else 0.0
    if m > 0:
        return e / m
    return 0.0 if e == 0 else float("inf")


def output_bound_units(meter_k: float, meter_v: float) -> float:
    """Bound on ||y - yhat|| / max_t ||v_t||: 2 meter_K + meter_V."""
    return 2.0 * meter_k + meter_v


def joint_gate_q(meter_k, raw_k, meter_v, tau_k: float, tau_v: float) -> np.ndarray:
    """Query heads routed because pass_K and pass_V do not both hold."""
    return ogate.gate_q(meter_k, raw_k, tau_k) | (np.asarray(meter_v, dtype=np.float64) > tau_v)


def joint_decode(q: np.ndarray, khat: np.ndarray, vhat: np.ndarray, c: np.ndarray,
                 rho: np.ndarray, vnorm: np.ndarray, sm_scale: float) -> dict:
    """One decode step with both meters.

    q [n_q, d]; khat, vhat [S, n_kv, d]; c [n_q, S] the key-side per-token bounds
    (Tier A: the witness bound; Tier B: the radius); rho, vnorm [S, n_kv] stored.
    Returns out, raw_k, meter_k, meter_v [n_q].
    """
    q = np.asarray(q, dtype=np.float64)
    n_q, d = q.shape
    n_kv = khat.shape[1]
    g = n_q // n_kv
    out = np.empty((n_q, d))
    raw = np.empty(n_q)
    mv = np.empty(n_q)
    for h in range(n_q):
        kv = h // g
        z = attention.logits(q[h], khat[:, kv], sm_scale)
        p = attention.softmax(z)
        out[h] = p @ vhat[:, kv]
        raw[h] = mt.raw_from_am1(mt.a_minus_one_logits(z, c[h]))
        mv[h] = value_meter(p, rho[:, kv], vnorm[:, kv])
    return {"out": out, "raw": raw, "meter": mt.meter(raw), "meter_v": mv}
