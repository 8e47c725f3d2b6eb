"""Pins of the group-scale oracle (Sec. 6.2 storage side, Table 4 granularity).

What the paper and the mathematics fix, and these tests check:
* no code is ever clipped, and every channel's error stays within half of its
  group's step (Sec. 4.2 quantizer law; Sec. 6.2 storage validation, max ratio
  1.0000), the bound attained;
* the group exponent is the largest one that keeps the group inside the token
  scale's range (brute force over all 15 exponents), so the group step is within
  a factor 2 of the group's own amax / 126.5;
* with every exponent 0 the quantizer is the plain token-scalar one bit for bit
  (codes and reconstructions), and an all-zero group gets the largest exponent;
* the dither stays subtractive per group: over the 256 dither values a kept
  channel's residual is the lattice of spacing s_g / 256 whatever the input;
* bypassed pairs leave the group amaxes as they leave the token amax;
* Tier B: over many Philox keys the logit error's variance is the proxy
  (sm^2/12) sum_g s_g^2 ||q_g||^2 and the joint tail stays within delta_loc; with
  all exponents 0 the radius is the token-scalar radius;
* Table 4's finding, on channel-scaled data: group scales give a smaller
  residual than the token scalar, and both tiers stay sound (raw >= true TV).
"""
import numpy as np
import pytest

import synth
from oracle import bypass as bp
from oracle import decode as odec
from oracle import groupscale as gs
from oracle import meter as mt
from oracle import philox, quantizer as qz, tierb


def _rows(n, d, seed, outliers=2):
    rng = np.random.default_rng(seed)
    sig = synth.channel_scales(rng, d, outliers, 10.0)
    return synth.bf16_round(rng.standard_normal((n, d)) * sig).astype(np.float64)


@pytest.mark.parametrize("d", [64, 128])
def test_no_clipping_and_half_group_step(d):
    x = _rows(3000, d, 50)
    # groups of very different magnitude, an all-zero group, a group at the amax
    x[:100, :32] *= 1e-3
    x[100:200, 32:64] = 0.0
    xi = philox.dither_values(np.arange(3000), d, 1, 0, 71)
    code, s, e, _, xh = gs.quantize(x, xi)
    assert code.min() >= -127 and code.max() <= 127
    step = gs.group_steps(s, e)
    err = np.abs(xh - x)
    assert np.all(err <= step * (0.5 + 2.0 ** -14))
    ratio = (err / (step / 2)).max()
    assert 0.99 < ratio <= 1.0 + 2.0 ** -13
    assert np.all(e[100:200, 1] == gs.E_MAX)
    assert np.all(code[100:200, 32:64] == 0)


def test_exponent_is_the_largest_that_fits():
    x = _rows(500, 128, 51)
    x[:50, 64:96] *= 2.0 ** -9
    s, e = gs.scales(x)
    amax = np.abs(x).max(axis=1)
    for i in range(x.shape[0]):
        for g in range(4):
            ag = np.abs(x[i, 32 * g:32 * g + 32]).max()
            fits = [k for k in range(gs.E_MAX + 1) if ag * 2.0 ** k <= amax[i]]
            assert e[i, g] == max(fits)
            # the group step is within a factor 2 of the group's own amax / 126.5
            sg = s[i] * 2.0 ** -e[i, g]
            if e[i, g] < gs.E_MAX:
                assert ag / 126.5 <= sg * (1 + 2.0 ** -10) and sg < 2 * ag / 126.5 * (1 + 2.0 ** -9)
    assert np.array_equal(s, qz.int8_scale(x))


def test_reduces_to_the_token_scalar_quantizer():
    # every group holds a value above half the row's amax: every exponent is 0
    rng = np.random.default_rng(52)
    x = rng.normal(size=(400, 128))
    for g in range(4):
        x[:, 32 * g] = 3.0 * np.sign(rng.normal(size=400)) + 1e-3 * g
    xi = philox.dither_values(np.arange(400), 128, 0, 2, 9)
    code, s, e, _, xh = gs.quantize(x, xi)
    assert np.all(e == 0)
    c0, s0 = qz.int8_encode(x, xi)
    assert np.array_equal(code, c0) and np.array_equal(s, s0)
    assert np.array_equal(xh, qz.int8_decode(c0, s0, xi))


def test_subtractive_law_per_group():
    rng = np.random.default_rng(53)
    d = 64
    lattice = (np.arange(256) - 127.5) / 256.0
    for _ in range(20):
        x = np.tile(rng.normal(size=d) * np.repeat([4.0, 0.1], 32), (256, 1))
        xi = np.repeat(lattice[:, None], d, axis=1)
        code, s, e, _, xh = gs.quantize(x, xi)
        assert e[0, 0] == 0 and e[0, 1] >= 4
        for c in (3, 40):
            step = s[0] * 2.0 ** -e[0, c // 32]
            r = (xh - x)[:, c] / step
            assert np.allclose(np.diff(np.sort(r)), 1 / 256, atol=1e-9)
            assert abs(np.var(r) - (1 - 4.0 ** -8) / 12) < 1e-9


def test_bypassed_pairs_leave_the_group_amax():
    rng = np.random.default_rng(54)
    d = 128
    x = rng.normal(size=(200, d))
    ch = bp.bypass_channels([5, 40], d, "half")       # channels 5, 69, 40, 104
    x[:, ch] *= 500.0
    xi = philox.dither_values(np.arange(200), d, 0, 0, 3)
    code, s, e, ov, xh = gs.quantize(x, xi, ch)
    keep = gs.keep_mask(d, ch)
    s_ref, e_ref = gs.scales(np.where(keep, x, 0.0))
    assert np.array_equal(s, s_ref) and np.array_equal(e, e_ref)
    assert np.all(code[:, ch] == 0)
    assert np.array_equal(xh[:, ch], bp.f16_nearest(x[:, ch]))
    assert np.all(np.abs(xh - x)[:, keep] <= gs.group_steps(s, e)[:, keep] * (0.5 + 2.0 ** -14))


def test_tierb_monte_carlo_and_reduction():
    rng = np.random.default_rng(55)
    d, S, n_seeds = 64, 24, 1500
    sm = 1 / np.sqrt(d)
    k = rng.normal(size=(S, d)) * np.exp(rng.uniform(np.log(0.5), np.log(4), d))
    k[:, 32:] *= 0.05                                  # a small group: exponent >= 3
    q = rng.normal(size=d) * 2.0
    slots = np.arange(S) + 2000
    eps = np.empty((n_seeds, S))
    for i in range(n_seeds):
        xi = philox.dither_values(slots, d, 3, 1, 0x6600_0000 + i)
        _, s, e, _, kh = gs.quantize(k, xi)
        eps[i] = sm * (kh - k) @ q
    assert np.all(e[:, 1] >= 3)
    var = tierb.variance_proxy(q, gs.group_steps(s, e), sm)
    emp = eps.var(axis=0)
    assert np.all(np.abs(emp / var - 1) < 0.15)
    assert abs(np.mean(emp / var) - 1) < 0.03
    for dloc in (0.5, 0.2, 0.05):
        u = gs.radius(q, s, e, sm, S, dloc)
        assert np.mean(np.any(np.abs(eps) > u[None, :], axis=1)) <= dloc
    # all exponents 0: the token-scalar radius
    s0 = rng.uniform(0.01, 1, 20)
    assert np.allclose(gs.radius(q, s0, np.zeros((20, 2), np.int64), sm, 100, 1e-3),
                       tierb.radius(q, s0, sm, 100, 1e-3), rtol=1e-13)


def test_table4_group_scales_are_more_accurate_and_sound():
    rng = np.random.default_rng(56)
    d, S, n_kv, n_q, B = 128, 256, 2, 8, 8
    sm = 1 / np.sqrt(d)
    k = np.stack([_rows(S, d, 60 + h) for h in range(n_kv)], axis=1)
    v = np.stack([_rows(S, d, 70 + h) for h in range(n_kv)], axis=1)
    plain = odec.write_cache("int8_dither", k, v, np.arange(S), 0, 11, B)
    grp = odec.write_cache("int8_dither", k, v, np.arange(S), 0, 11, B, group_scales=True)
    assert np.any(grp["ke"] > 0)
    for kh in ("khat", "vhat"):
        x = k if kh == "khat" else v
        assert np.mean((grp[kh] - x) ** 2) < 0.8 * np.mean((plain[kh] - x) ** 2)
    for scale in (1.0, 1 / 16):
        q = rng.normal(size=(n_q, d)) * scale
        tv = odec.true_tv(q, k, grp["khat"], sm)
        ra = odec.metered_decode(q, grp["khat"], grp["vhat"], grp["kw"], sm, B)
        assert np.all(ra["raw"] >= tv)
        rb = gs.tierb_decode(q, grp["khat"], grp["vhat"], grp["ks"], grp["ke"], sm, 1e-6)
        assert np.all(rb["raw"] >= tv)
        assert np.array_equal(rb["out"], ra["out"])
        rp = odec.metered_decode(q, plain["khat"], plain["vhat"], plain["kw"], sm, B)
        assert np.median(ra["raw"]) < np.median(rp["raw"])
        for h in range(n_q):
            kv = h // (n_q // n_kv)
            err = np.abs(sm * (grp["khat"][:, kv] - k[:, kv]) @ q[h])
            assert np.all(err <= mt.logit_bound(q[h], grp["kw"][:, kv], sm, B) * (1 + 1e-12))
