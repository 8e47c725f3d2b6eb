"""Pins of the group-scale oracle (Sec. 6.2 storage side, Table 4 granularity).

What the paper and the mathematics fix, and these tests check:
* Table 4's byte account: K + V of one token and KV head take 272 bytes at
  32-channel groups (128 codes and four 2-byte scales per side), 288 at 16-channel
  groups and 260 for one token scale;
* each group's stored scale is the smallest fp16 value at or above fl32(amax_g /
  126.5) (brute force over the fp16 values), so no code is ever clipped and every
  channel's error stays within half its group's step (Sec. 4.2 quantizer law;
  Sec. 6.2 storage validation, max ratio 1.0000), the bound attained; an all-zero
  group stores scale 0 and codes 0;
* groups sharing the token's amax give the plain token-scalar quantizer bit for
  bit (codes, scales and reconstructions);
* the dither stays subtractive per group: over the 256 dither values a kept
  channel's residual is the lattice of spacing s_g / 256 whatever the input;
* bypassed pairs leave the group amaxes;
* Tier B: over many Philox keys the logit error's variance is the proxy
  (sm^2/12) sum_g s_g^2 ||q_g||^2 and the joint tail stays within delta_loc; with
  equal group scales the radius is the token-scalar radius;
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


def test_table4_byte_account():
    assert gs.bytes_per_token_head(128, 32) == 272
    assert gs.bytes_per_token_head(128, 16) == 288
    assert gs.bytes_per_token_head(128, None) == 260


def test_stored_scale_is_the_fp16_round_up():
    # every positive finite fp16 value, as float64, in increasing order
    f16 = np.arange(1, 0x7C00, dtype=np.uint16).view(np.float16).astype(np.float64)
    x = _rows(400, 128, 49)
    x[:40, 32:64] *= 2.0 ** -12           # subnormal-range group scales
    s = gs.scales(x)
    ag = np.abs(x).reshape(400, 4, 32).max(axis=2)
    want = np.float32(ag / 126.5).astype(np.float64)
    idx = np.searchsorted(f16, want, side="left")  # first fp16 >= want
    assert np.array_equal(s, np.where(want > 0, f16[np.minimum(idx, f16.size - 1)], 0.0))


@pytest.mark.parametrize("d", [64, 128])
def test_no_clipping_and_half_group_step(d):
    x = _rows(3000, d, 50)
    # groups of very different magnitude, an all-zero group
    x[:100, :32] *= 1e-3
    x[100:200, 32:64] = 0.0
    xi = philox.dither_values(np.arange(3000), d, 1, 0, 71)
    code, s, _, xh = gs.quantize(x, xi)
    assert code.min() >= -127 and code.max() <= 127
    step = gs.channel_steps(s)
    err = np.abs(xh - x)
    assert np.all(err <= step * (0.5 + 2.0 ** -14))
    nz = step > 0
    ratio = (err[nz] / (step[nz] / 2)).max()
    assert 0.99 < ratio <= 1.0 + 2.0 ** -13
    assert np.all(s[100:200, 1] == 0) and np.all(code[100:200, 32:64] == 0) and np.all(xh[100:200, 32:64] == 0)
    # a group's step follows its own amax: the group scaled by 1e-3 errs ~1e-3 as much
    assert np.max(err[:100, :32]) < 1e-2 * np.max(err[:100, 32:])


def test_reduces_to_the_token_scalar_quantizer():
    # every group holds the row's amax (up to sign): all group scales equal the token scale
    rng = np.random.default_rng(52)
    x = rng.normal(size=(400, 128))
    amax = 10.0 + np.abs(rng.normal(size=400))
    for g in range(4):
        x[:, 32 * g + g] = amax * np.sign(rng.normal(size=400))
    xi = philox.dither_values(np.arange(400), 128, 0, 2, 9)
    code, s, _, xh = gs.quantize(x, xi)
    c0, s0 = qz.int8_encode(x, xi)
    assert np.array_equal(s, np.repeat(s0[:, None], 4, axis=1))
    assert np.array_equal(code, c0)
    assert np.array_equal(xh, qz.int8_decode(c0, s0, xi))


def test_subtractive_law_per_group():
    rng = np.random.default_rng(53)
    d = 64
    lattice = (np.arange(256) - 127.5) / 256.0
    for _ in range(20):
        x = np.tile(rng.normal(size=d) * np.repeat([4.0, 0.1], 32), (256, 1))
        xi = np.repeat(lattice[:, None], d, axis=1)
        code, s, _, xh = gs.quantize(x, xi)
        assert s[0, 1] < 0.1 * s[0, 0]
        for c in (3, 40):
            step = s[0, c // 32]
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
    code, s, ov, xh = gs.quantize(x, xi, ch)
    keep = gs.keep_mask(d, ch)
    assert np.array_equal(s, gs.scales(np.where(keep, x, 0.0)))
    assert np.all(code[:, ch] == 0)
    assert np.array_equal(xh[:, ch], bp.f16_nearest(x[:, ch]))
    assert np.all(np.abs(xh - x)[:, keep] <= gs.channel_steps(s)[:, keep] * (0.5 + 2.0 ** -14))


def test_tierb_monte_carlo_and_reduction():
    rng = np.random.default_rng(55)
    d, S, n_seeds = 64, 24, 1500
    sm = 1 / np.sqrt(d)
    k = rng.normal(size=(S, d)) * np.exp(rng.uniform(np.log(0.5), np.log(4), d))
    k[:, 32:] *= 0.05                                  # a small group
    q = rng.normal(size=d) * 2.0
    slots = np.arange(S) + 2000
    eps = np.empty((n_seeds, S))
    for i in range(n_seeds):
        xi = philox.dither_values(slots, d, 3, 1, 0x6600_0000 + i)
        _, s, _, kh = gs.quantize(k, xi)
        eps[i] = sm * (kh - k) @ q
    assert np.all(s[:, 1] < 0.2 * s[:, 0])
    var = tierb.variance_proxy(q, gs.channel_steps(s), sm)
    emp = eps.var(axis=0)
    assert np.all(np.abs(emp / var - 1) < 0.15)
    assert abs(np.mean(emp / var) - 1) < 0.03
    for dloc in (0.5, 0.2, 0.05):
        u = gs.radius(q, s, sm, S, dloc)
        assert np.mean(np.any(np.abs(eps) > u[None, :], axis=1)) <= dloc
    # equal group scales: the token-scalar radius
    s0 = rng.uniform(0.01, 1, 20)
    assert np.allclose(gs.radius(q, np.repeat(s0[:, None], 2, axis=1), sm, 100, 1e-3),
                       tierb.radius(q, s0, sm, 100, 1e-3), rtol=1e-13)


def test_table4_group_scales_are_more_accurate_and_sound():
    rng = np.random.default_rng(56)
    d, S, n_kv, n_q, B = 128, 256, 2, 8, 8
    sm = 1 / np.sqrt(d)
    k = np.stack([_rows(S, d, 60 + h) for h in range(n_kv)], axis=1)
    v = np.stack([_rows(S, d, 70 + h) for h in range(n_kv)], axis=1)
    plain = odec.write_cache("int8_dither", k, v, np.arange(S), 0, 11, B)
    grp = odec.write_cache("int8_dither", k, v, np.arange(S), 0, 11, B, group_scales=True)
    assert grp["ks"].shape == (S, n_kv, d // 32)
    for kh in ("khat", "vhat"):
        x = k if kh == "khat" else v
        assert np.mean((grp[kh] - x) ** 2) < 0.8 * np.mean((plain[kh] - x) ** 2)
    for scale in (1.0, 1 / 16):
        q = rng.normal(size=(n_q, d)) * scale
        tv = odec.true_tv(q, k, grp["khat"], sm)
        ra = odec.metered_decode(q, grp["khat"], grp["vhat"], grp["kw"], sm, B)
        assert np.all(ra["raw"] >= tv)
        rb = gs.tierb_decode(q, grp["khat"], grp["vhat"], grp["ks"], sm, 1e-6)
        assert np.all(rb["raw"] >= tv)
        assert np.array_equal(rb["out"], ra["out"])
        rp = odec.metered_decode(q, plain["khat"], plain["vhat"], plain["kw"], sm, B)
        assert np.median(ra["raw"]) < np.median(rp["raw"])
        for h in range(n_q):
            kv = h // (n_q // n_kv)
            err = np.abs(sm * (grp["khat"][:, kv] - k[:, kv]) @ q[h])
            assert np.all(err <= mt.logit_bound(q[h], grp["kw"][:, kv], sm, B) * (1 + 1e-12))
