"""Pins of the outlier-pair bypass oracle (Sec. 4.2 outlier RoPE pairs; Sec. 6.2
fixed-channel bypass, Tables 5 and 6) against the mathematics and the paper.

* Pair selection: brute force over every m-subset on small heads (the chosen set
  has the largest total energy, ties to lower indices); RoPE leaves the pair
  energies and hence the set unchanged at any positions (a mispaired channel
  map fails this); on the workloads' keys the set is exactly the pairs of the
  injected massive channels.
* Amax exclusion: the scale is the plain INT8 scale of the row without the
  bypassed channels; no code is clipped even with bypassed values 10^3 times
  larger; the half-step error bound holds on the other channels; bypassed
  channels reconstruct to their fp16 value (exactly the input for bf16 data);
  with no pairs everything reduces to the plain quantizer.
* Table 5: bypass alone barely moves the meter, bypass with the channels out of
  the amax lowers it by an order of magnitude (controlled experiment with four
  injected massive RoPE pairs).
* The fp16 rounding bound used for the bypassed channels in Tier B holds on
  every binade and subnormal, and is attained at the bottom of every binade.
* Tier B with bypass: reduces to the plain radius with no pairs; Monte Carlo over
  Philox keys through the real quantizer (fp32 data, so the bypassed channels
  carry a rounding residual) stays within delta_loc; raw bounds the true TV for
  both tiers on small decodes.
"""
import itertools

import numpy as np
import pytest

import synth
from oracle import attention, bypass as bp, decode as odec, meter as mt, philox
from oracle import quantizer as qz, tierb


def test_pair_selection_brute_force():
    rng = np.random.default_rng(21)
    d = 12
    for trial in range(40):
        k = rng.normal(size=(7, d)) * rng.uniform(0.1, 3, size=d)
        if trial % 4 == 0:            # exact ties between two pairs
            k[:, 4] = k[:, 1]
            k[:, 10] = k[:, 7]
        for layout in ("half", "interleaved"):
            e = bp.pair_energy(k, layout)
            for m in range(0, d // 2 + 1):
                got = bp.select_pairs(k, m, layout)
                assert list(got) == sorted(got) and len(set(got)) == m
                best = max(itertools.combinations(range(d // 2), m),
                           key=lambda c: (round(sum(e[list(c)]), 9), [-j for j in sorted(c)]))
                assert np.isclose(e[list(got)].sum(), e[list(best)].sum(), rtol=1e-12)
                assert tuple(got) == tuple(sorted(best))


def test_pair_energy_is_rope_invariant():
    rng = np.random.default_rng(22)
    d, S = 64, 50
    pre = rng.normal(size=(S, d)) * rng.uniform(0.1, 5, size=d)
    pos = rng.integers(0, 10 ** 6, size=S)
    for layout in ("half", "interleaved"):
        post = synth.rope_rotate(pre, pos, 1e6, layout)
        assert np.allclose(bp.pair_energy(pre, layout), bp.pair_energy(post, layout), rtol=1e-10)
        for m in (1, 4, 8):
            assert np.array_equal(bp.select_pairs(pre, m, layout), bp.select_pairs(post, m, layout))
    # the other layout's pairing is not rotation invariant: the test has power
    post = synth.rope_rotate(pre, pos, 1e6, "half")
    assert not np.allclose(bp.pair_energy(pre, "interleaved"), bp.pair_energy(post, "interleaved"), rtol=1e-3)


def test_selection_finds_the_injected_massive_pairs():
    wl = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]
    for layer, kv in ((0, 0), (3, 2)):
        k = synth.gen_kv(wl, layer, kv, 0, "k", np.arange(512)).astype(np.float64)
        srng = synth.cell_rng(wl.wid, layer, kv, 0, 1 << 20)
        sig = synth.channel_scales(srng, wl.d, wl.n_outliers, wl.outlier_mult)
        massive = np.argsort(-sig)[:wl.n_outliers]
        want = np.unique(massive % (wl.d // 2))     # rotate-half pair of each channel
        got = bp.select_pairs(k, want.size, wl.rope_layout)
        assert np.array_equal(got, want)


def _bf16_rows(n, d, seed):
    rng = np.random.default_rng(seed)
    return synth.bf16_round(rng.standard_normal((n, d)) * rng.uniform(0.5, 4, size=d)).astype(np.float64)


@pytest.mark.parametrize("layout", ["half", "interleaved"])
def test_amax_exclusion_and_storage(layout):
    d, n = 128, 3000
    x = _bf16_rows(n, d, 23)
    pairs = np.array([3, 17, 40, 63])
    ch = bp.bypass_channels(pairs, d, layout)
    x[:, ch] = synth.bf16_round(np.clip(x[:, ch] * 1e3, -6e4, 6e4))   # massive, inside the fp16 range
    xi = philox.dither_values(np.arange(n), d, 1, 0, 77)
    code, s, ov, xh = bp.quantize_bypass(x, xi, ch)
    keep = np.ones(d, bool)
    keep[ch] = False
    assert np.array_equal(s, qz.int8_scale(x[:, keep]))
    assert code.min() >= -127 and code.max() <= 127
    assert np.all(code[:, ch] == 0)
    err = np.abs(xh - x)[:, keep]
    assert np.all(err <= s[:, None] * (0.5 + 2.0 ** -14))
    # the bypassed channels hold their fp16 value; bf16 data in the fp16 range is exact
    assert np.array_equal(xh[:, ch], ov)
    assert np.array_equal(ov, x[:, ch])
    # the codes of the other channels are the plain quantizer's on the kept channels
    c2, s2 = qz.int8_encode(x[:, keep], xi[:, keep])
    assert np.array_equal(code[:, keep], c2) and np.array_equal(s, s2)
    # without exclusion (Table 5 middle row) the scale is the full row's
    _, s3 = bp.int8_encode_bypass(x, xi, ch, exclude_from_amax=False)
    assert np.array_equal(s3, qz.int8_scale(x))
    # no pairs: the plain quantizer
    c0, s0, ov0, xh0 = bp.quantize_bypass(x, xi, np.zeros(0, np.int64))
    c1, s1 = qz.int8_encode(x, xi)
    assert np.array_equal(c0, c1) and np.array_equal(s0, s1) and ov0.shape == (n, 0)
    assert np.array_equal(xh0, qz.int8_decode(c1, s1, xi))


def test_subtractive_law_on_the_kept_channels():
    """Over the 256 dither values the residual of a kept channel is the 1/256
    lattice for any input, as without bypass."""
    rng = np.random.default_rng(24)
    d = 16
    ch = bp.bypass_channels([2], d, "half")
    lattice = (np.arange(256) - 127.5) / 256.0
    for _ in range(30):
        x = np.tile(rng.normal(size=d) * 3, (256, 1))
        x[:, ch] *= 1000
        xi = np.repeat(lattice[:, None], d, axis=1)
        code, s, ov, xh = bp.quantize_bypass(x, xi, ch)
        r = (xh - x)[:, 0] / s[0]
        steps = np.sort(r)
        assert np.allclose(np.diff(steps), 1 / 256, atol=1e-9)
        assert abs(np.var(r) - (1 - 4.0 ** -8) / 12) < 1e-9


def _massive_case(rng, S, d, n_pairs, mult):
    pre = rng.normal(size=(S, d))
    pairs = rng.choice(d // 2, size=n_pairs, replace=False)
    pre[:, pairs] *= mult
    return synth.rope_rotate(pre, np.arange(S), 1e4, "half"), np.sort(pairs)


def test_table5_both_steps_are_needed():
    """Controlled experiment of Table 5: four injected massive RoPE pairs.  The
    paper measures median meters 1.0311 (no bypass), 0.9608 (bypass alone) and
    0.0620 (bypass with amax exclusion)."""
    rng = np.random.default_rng(25)
    S, d, B = 512, 64, 4
    sm = 1 / np.sqrt(d)
    med = {}
    for mode in ("none", "alone", "excluded"):
        raws = []
        for cell in range(6):
            crng = np.random.default_rng(1000 + cell)
            k, pairs = _massive_case(crng, S, d, 4, 30.0)
            q = crng.normal(size=(4, d)) * 0.35
            xi = philox.dither_values(np.arange(S), d, 0, 0, 500 + cell)
            if mode == "none":
                code, s = qz.int8_encode(k, xi)
                kh = qz.int8_decode(code, s, xi)
            else:
                ch = bp.bypass_channels(pairs, d, "half")
                _, _, _, kh = bp.quantize_bypass(k, xi, ch, exclude_from_amax=(mode == "excluded"))
            w = qz.witness(k, kh, B)
            for h in range(q.shape[0]):
                z = attention.logits(q[h], kh, sm)
                c = mt.logit_bound(q[h], w, sm, B)
                raws.append(mt.raw_from_am1(mt.a_minus_one_logits(z, c)))
        med[mode] = np.median(raws)
    assert med["alone"] <= med["none"] and med["alone"] >= 0.5 * med["none"]
    assert med["excluded"] <= med["alone"] / 8


def test_fp16_rounding_bound():
    rng = np.random.default_rng(26)
    x = np.concatenate([
        rng.uniform(-1, 1, 20000) * 10.0 ** rng.uniform(-9, 4.8, 20000),
        rng.uniform(-2.0 ** -14, 2.0 ** -14, 5000),                      # subnormal range
        (2.0 ** np.arange(-24, 16))[:, None].repeat(3, 1).ravel() * (1 + np.tile([-1e-4, 0, 1e-4], 40)),
    ])
    x = x[np.abs(x) <= 65504]
    h = bp.f16_nearest(x)
    assert np.all(np.abs(h - x) <= bp.rounding_bound(h))
    # attained: the midpoint above 2^e rounds (to even) down to 2^e, half an ulp away
    p2 = 2.0 ** np.arange(-14, 16)
    mid = p2 * (1 + 2.0 ** -11)
    hm = bp.f16_nearest(mid)
    assert np.array_equal(hm, p2)
    assert np.array_equal(np.abs(hm - mid), bp.rounding_bound(hm) - bp.F16_ABS)


def test_tierb_radius_with_bypass_reduces_and_covers():
    rng = np.random.default_rng(27)
    d = 64
    q = rng.normal(size=d)
    s = rng.uniform(0.01, 1, 20)
    none = np.zeros(0, np.int64)
    assert np.allclose(bp.radius(q, s, np.zeros((20, 0)), none, 0.125, 100, 1e-3),
                       tierb.radius(q, s, 0.125, 100, 1e-3), rtol=1e-13)
    # Monte Carlo through the real quantizer on fp32 data (nonzero fp16 residual)
    S, n_seeds, sm = 24, 1500, 1 / np.sqrt(d)
    crng = np.random.default_rng(28)
    k, pairs = _massive_case(crng, S, d, 2, 40.0)
    k = k.astype(np.float32).astype(np.float64)
    ch = bp.bypass_channels(pairs, d, "half")
    q = crng.normal(size=d) * 2
    eps = np.empty((n_seeds, S))
    for i in range(n_seeds):
        xi = philox.dither_values(np.arange(S) + 4000, d, 2, 0, 0x5150_0000 + i)
        _, s_tok, ov, kh = bp.quantize_bypass(k, xi, ch)
        eps[i] = sm * (kh - k) @ q
    assert np.any(ov != k[:, ch])                 # the deterministic term is exercised
    for dloc in (0.5, 0.2, 0.05):
        u = bp.radius(q, s_tok, ov, ch, sm, S, dloc)
        assert np.mean(np.any(np.abs(eps) > u[None, :], axis=1)) <= dloc


def test_both_tiers_sound_with_bypass():
    rng = np.random.default_rng(29)
    d, S, n_kv, n_q, B = 64, 200, 2, 6, 4
    sm = 1 / np.sqrt(d)
    k = np.empty((S, n_kv, d))
    pairs = np.empty((n_kv, 3), np.int64)
    for h in range(n_kv):
        k[:, h], pairs[h] = _massive_case(rng, S, d, 3, 25.0)
    k = k.astype(np.float32).astype(np.float64)
    v = rng.normal(size=(S, n_kv, d))
    for scale in (1.0, 1 / 8):
        q = rng.normal(size=(n_q, d)) * scale
        for seed in range(4):
            c = odec.write_cache("int8_dither", k, v, np.arange(S), 0, 900 + seed, B, "half", pairs=pairs)
            tv = odec.true_tv(q, k, c["khat"], sm)
            ra = odec.metered_decode(q, c["khat"], c["vhat"], c["kw"], sm, B)
            assert np.all(ra["raw"] >= tv)
            rb = bp.tierb_decode(q, c["khat"], c["vhat"], c["ks"], c["ko"], c["chans"], sm, 1e-6)
            assert np.all(rb["raw"] >= tv)
            assert np.array_equal(rb["out"], ra["out"])
            # the witness still bounds every logit error (Cauchy-Schwarz per band)
            for h in range(n_q):
                err = np.abs(sm * (c["khat"][:, h // 3] - k[:, h // 3]) @ q[h])
                assert np.all(err <= mt.logit_bound(q[h], c["kw"][:, h // 3], sm, B) * (1 + 1e-12))
