"""Pins of the oracle's meter (CPU).

* the Sec. 3 counterexample: TV and Eq. (flawed) values printed in the paper;
* Theorem (sound replacement) checked adversarially on >= 500,000 random cells
  (Sec. 3 adversarial suite: residual signs all one way or alternating, softmax
  mass on one token or spread evenly, bounds up to several units), with the
  sign convention p_t = ptilde_t e^{-eps_t} / Z of the machine-checked statement;
* closed forms: constant c gives (e^{2c} - 1)/2; A >= 1;
* 50-digit mpmath evaluation of the same definition on tiny cells;
* overflow gives +inf raw and meter 1 (Sec. 3; Sec. 6.2 telemetry);
* Proposition (two-sided form) is sound on the same suite and is looser than the
  e-form at A = 2, A^- = 0.6 as the paper states.
"""
import json
import os

import mpmath
import numpy as np
import pytest

from oracle import attention, meter as mt

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def test_counterexample_values():
    g = json.load(open(os.path.join(GOLD, "counterexample.json")))
    pt, c, eps = (np.array(g[k]) for k in ("ptilde", "c", "eps"))
    p = pt * np.exp(-eps)
    p /= p.sum()
    assert round(float(attention.tv(p, pt)), 6) == g["tv"]
    assert round(float(mt.flawed_bound(pt, c)), 6) == g["flawed"]
    eform = float(mt.raw_bound(pt, c))
    assert eform == pytest.approx(0.5 * np.expm1(0.2), rel=1e-14)
    assert round(eform, 6) == 0.110701
    assert eform >= g["tv"] > g["flawed"]               # flawed is unsound, e-form is not
    # two-token closed form: TV = tanh(eps)/2 for ptilde = (1/2, 1/2), eps = (e, -e)
    assert float(attention.tv(p, pt)) == pytest.approx(0.5 * np.tanh(0.1), rel=1e-13)


def _adversarial_batch(rng, n, S):
    alpha = rng.choice([0.02, 0.2, 1.0, 10.0])
    pt = rng.dirichlet(np.full(S, alpha), size=n)
    pt = np.maximum(pt, 1e-300)
    pt /= pt.sum(axis=1, keepdims=True)
    scale = np.exp(rng.uniform(np.log(1e-4), np.log(8.0), size=(n, 1)))
    c = rng.uniform(0, 1, size=(n, S)) * scale
    c[rng.uniform(size=(n, S)) < 0.2] = 0.0
    mode = rng.integers(0, 4)
    if mode == 0:                                        # random signs
        sgn = rng.choice([-1.0, 1.0], size=(n, S))
    elif mode == 1:                                      # + on the heaviest tokens
        sgn = np.where(pt >= np.median(pt, axis=1, keepdims=True), 1.0, -1.0)
    elif mode == 2:                                      # - on the heaviest tokens
        sgn = np.where(pt >= np.median(pt, axis=1, keepdims=True), -1.0, 1.0)
    else:                                                # one token against the rest
        sgn = -np.ones((n, S))
        sgn[np.arange(n), rng.integers(0, S, n)] = 1.0
    frac = np.where(rng.uniform(size=(n, 1)) < 0.5, 1.0, rng.uniform(0, 1, size=(n, S)))
    eps = sgn * c * frac
    return pt, c, eps


def test_theorem_sound_replacement_adversarial_500k():
    rng = np.random.default_rng(2026)
    total = 0
    worst = 0.0
    for S in (2, 3, 5, 16, 64, 257):
        n = 500_000 // 6 + 1
        for chunk in range(0, n, 20000):
            m = min(20000, n - chunk)
            pt, c, eps = _adversarial_batch(rng, m, S)
            for sign in (1.0, -1.0):                     # p = ptilde e^{-eps}/Z and the mirror
                p = pt * np.exp(-sign * eps)
                p /= p.sum(axis=1, keepdims=True)
                t = attention.tv(p, pt)
                b = mt.raw_bound(pt, c)
                assert np.all(t <= b * (1 + 1e-12) + 1e-15)
                assert np.all(t <= mt.two_sided_bound(pt, c) * (1 + 1e-12) + 1e-15)
                worst = max(worst, float(np.max(t / np.maximum(b, 1e-300))))
            total += m
    assert total >= 500_000
    assert worst > 0.3          # the suite gets close to the bound somewhere


def test_closed_forms_and_invariants():
    rng = np.random.default_rng(3)
    for cval in (0.0, 1e-9, 1e-3, 0.1, 1.0, 5.0):
        pt = rng.dirichlet(np.ones(10))
        assert float(mt.raw_bound(pt, np.full(10, cval))) == pytest.approx(
            0.5 * np.expm1(2 * cval), rel=1e-12, abs=1e-300)
    pt = rng.dirichlet(np.ones(50), size=100)
    c = rng.uniform(0, 2, size=(100, 50))
    assert np.all(mt.a_minus_one(pt, c) >= 0)                       # A >= 1
    z = rng.standard_normal((100, 50)) * 5
    assert np.allclose(mt.a_minus_one_logits(z, c), mt.a_minus_one(attention.softmax(z), c),
                       rtol=1e-12)
    m = mt.meter(mt.raw_bound(pt, c))
    assert np.all((m >= 0) & (m <= 1))


def test_overflow_is_infinite_raw_and_saturated_meter():
    z = np.array([0.0, -800.0])                 # second token's mass underflows in float64
    c = np.array([0.0, 2000.0])                 # but its bound is astronomically large
    raw = mt.raw_from_am1(mt.a_minus_one_logits(z, c))
    assert np.isinf(raw) and mt.meter(raw) == 1.0
    # moderate: the log-domain term is finite and counted although ptilde_t underflows
    z = np.array([0.0, -760.0])
    c = np.array([0.0, 770.0])
    am1 = mt.a_minus_one_logits(z, c)
    assert np.isfinite(am1) and am1 == pytest.approx(np.exp(10.0), rel=1e-9)


def test_mpmath_50_digit_agreement():
    mpmath.mp.dps = 50
    rng = np.random.default_rng(4)
    for _ in range(200):
        S = int(rng.integers(1, 9))
        z = rng.standard_normal(S) * 3
        c = np.exp(rng.uniform(np.log(1e-8), np.log(3.0), S))
        ez = [mpmath.e ** mpmath.mpf(float(v)) for v in z]
        zs = mpmath.fsum(ez)
        a = mpmath.fsum(e / zs * mpmath.e ** mpmath.mpf(float(cv)) for e, cv in zip(ez, c))
        raw_mp = (a * a - 1) / 2
        raw = float(mt.raw_from_am1(mt.a_minus_one_logits(z, c)))
        assert raw == pytest.approx(float(raw_mp), rel=1e-12)


def test_two_sided_is_looser_at_the_papers_example():
    # A = 2, A^- = 0.6: (A/A^- - A^-/A)/2 = 1.5167 > (A^2-1)/2 = 1.5
    a, am = 2.0, 0.6
    assert 0.5 * (a / am - am / a) > 0.5 * (a * a - 1)
