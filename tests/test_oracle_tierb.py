"""Pins of the Tier-B oracle (Sec. 4.2, Tier B) against the mathematics and the quantizer.

* Lemma uniform sub-Gaussian proxy: the closed form against numerical
  integration, and the inequality sinh(x)/x <= e^{x^2/6} on a wide grid.
* The actual quantizer's residual, enumerated over all 256 dither values for
  random and rounding-boundary inputs, satisfies the per-channel MGF bound with
  the lattice bias: E[e^{lambda r}] <= e^{|lambda| s/256 + lambda^2 s^2/24}.
* The radius: union-bound identity S * 2 e^{-(u-b)^2 / (2 varsigma^2)} = delta,
  the hoisted form u_t = alpha * s_t, and the per-channel variance formula.
* Monte Carlo through the real dithered quantizer (many Philox keys): the logit
  error's variance matches varsigma^2 and the joint event max_t |eps_t| > u_t
  is no more frequent than delta_loc.
* The certificate: constant radius closed form A = e^u, and raw >= true TV on
  every cell at the budgets used in the tests.
"""
import numpy as np
import pytest

from oracle import attention, decode as odec, meter as mt, quantizer as qz, tierb

LATTICE = (np.arange(256) - 127.5) / 256.0


def test_uniform_mgf_closed_form_and_lemma():
    a = 0.37
    xs = np.linspace(-a, a, 400001)
    for lam in (-30.0, -3.0, -0.2, 0.0, 0.5, 4.0, 25.0):
        num = np.trapezoid(np.exp(lam * xs), xs) / (2 * a)
        assert tierb.mgf_uniform(lam, a) == pytest.approx(num, rel=1e-9)
    x = np.concatenate([np.linspace(-80, 80, 160001), [1e-8, -1e-8]])
    lhs = np.log(tierb.mgf_uniform(x, 1.0))
    assert np.all(lhs <= x ** 2 / 6 + 1e-15)
    # the proxy is the variance: the bound is tight to second order at 0
    small = np.array([1e-3, 2e-3])
    assert np.allclose(lhs[-2:], 0.0, atol=1e-15)
    assert np.allclose(np.log(tierb.mgf_uniform(small, 1.0)) / small ** 2, 1 / 6, rtol=1e-5)


def _enumerated_residual(xv, amax):
    x = np.zeros((256, 8))
    x[:, 0] = amax
    x[:, 1] = xv
    xi = np.repeat(LATTICE[:, None], 8, axis=1)
    c, s = qz.int8_encode(x, xi)
    return (qz.int8_decode(c, s, xi) - x)[:, 1], s[0]


def test_dither_residual_mgf_with_lattice_bias():
    rng = np.random.default_rng(11)
    lams = np.linspace(-80, 80, 321)
    inputs = [(rng.uniform(-a, a), a) for a in rng.uniform(0.01, 100, 150)]
    # inputs placed within 3e-5 steps of a rounding boundary of one dither value
    for _ in range(150):
        amax = rng.uniform(0.5, 50)
        s = qz.int8_scale(np.array([[amax]]))[0]
        y = rng.integers(-100, 100) + 0.5 - LATTICE[rng.integers(0, 256)] + rng.uniform(-3e-5, 3e-5)
        inputs.append((y * s, amax))
    for xv, amax in inputs:
        r, s = _enumerated_residual(xv, amax)
        assert abs(r.mean()) <= s / 256
        lam = lams / s
        mgf = np.mean(np.exp(lam[:, None] * r[None, :]), axis=1)
        assert np.all(np.log(mgf) <= np.abs(lam) * s / 256 + lam ** 2 * s ** 2 / 24 + 1e-12)


def test_radius_union_bound_and_hoisting():
    rng = np.random.default_rng(12)
    for _ in range(20):
        d = int(rng.choice([64, 128]))
        q = rng.normal(size=d) * rng.uniform(0.1, 5)
        s = rng.uniform(1e-3, 2.0, size=37)
        S, dloc, sm = int(rng.integers(1, 100000)), 10 ** rng.uniform(-12, -1), 1 / np.sqrt(d)
        u = tierb.radius(q, s, sm, S, dloc)
        var = sm ** 2 / 12 * np.sum(q ** 2) * s ** 2
        b = sm * s * np.sum(np.abs(q)) / 256
        # the two-sided sub-Gaussian tail at u - b, union-bounded over S tokens, is delta_loc
        assert np.allclose(S * 2 * np.exp(-(u - b) ** 2 / (2 * var)), dloc, rtol=1e-9)
        assert np.allclose(u, tierb.alpha(q, sm, S, dloc) * s, rtol=1e-12)
        # per-channel form with a constant scale equals the per-token form
        assert np.allclose(tierb.variance_proxy(q, np.full(d, s[0]), sm), var[0], rtol=1e-12)
    assert tierb.delta_loc(1e-2, 28, 28, 256) == pytest.approx(1e-2 / (28 * 28 * 256))


def test_monte_carlo_variance_and_joint_tail():
    """Many Philox keys over one set of keys: the empirical logit error."""
    rng = np.random.default_rng(13)
    d, S, n_seeds = 64, 24, 1500
    sm = 1 / np.sqrt(d)
    k = rng.normal(size=(S, d)) * np.exp(rng.uniform(np.log(0.5), np.log(4), d))
    q = rng.normal(size=d) * 2.0
    slots = np.arange(S) + 1000
    eps = np.empty((n_seeds, S))
    s_tok = None
    for i in range(n_seeds):
        _, s, _, kh = qz.int8_quantize_slots(k, slots, 3, 1, 0x1234_0000 + i)
        eps[i] = sm * (kh - k) @ q
        s_tok = s
    var = tierb.variance_proxy(q, np.repeat(s_tok[:, None], d, axis=1), sm)
    # lattice variance (1 - 4^-8)/12 per channel, up to sampling error (1500 draws)
    emp = eps.var(axis=0)
    assert np.all(np.abs(emp / var - 1) < 0.15)
    assert abs(np.mean(emp / var) - 1) < 0.03
    for dloc in (0.5, 0.2, 0.05):
        u = tierb.radius(q, s_tok, sm, S, dloc)
        viol = np.mean(np.any(np.abs(eps) > u[None, :], axis=1))
        assert viol <= dloc


def test_constant_radius_closed_form_and_tv_bound():
    # c_t == u for every token: A = e^u, raw = (e^{2u} - 1)/2
    z = np.random.default_rng(14).normal(size=50)
    for u in (1e-6, 0.01, 0.3, 2.0):
        raw = mt.raw_from_am1(mt.a_minus_one_logits(z, np.full(50, u)))
        assert raw == pytest.approx(0.5 * np.expm1(2 * u), rel=1e-12)
    # Tier-B raw bounds the true TV on every cell of a small decode
    rng = np.random.default_rng(15)
    d, S, n_kv, n_q = 64, 200, 2, 6
    k = rng.normal(size=(S, n_kv, d)) * np.exp(rng.uniform(np.log(0.5), np.log(4), (n_kv, d)))
    v = rng.normal(size=(S, n_kv, d))
    for scale in (1.0, 1 / 16):
        q = rng.normal(size=(n_q, d)) * scale
        for seed in range(5):
            c = odec.write_cache("int8_dither", k, v, np.arange(S), 0, 777 + seed, 4)
            res = tierb.tierb_decode(q, c["khat"], c["vhat"], c["ks"], 1 / np.sqrt(d), 1e-6)
            tv = odec.true_tv(q, k, c["khat"], 1 / np.sqrt(d))
            assert np.all(res["raw"] >= tv)
            # same attention output as the Tier-A decode of the same cache
            ra = odec.metered_decode(q, c["khat"], c["vhat"], c["kw"], 1 / np.sqrt(d), 4)
            assert np.allclose(res["out"], ra["out"], rtol=0, atol=0)
            p = attention.softmax(attention.logits(q[0], c["khat"][:, 0], 1 / np.sqrt(d)))
            assert np.allclose(res["ptilde"][0], p)
