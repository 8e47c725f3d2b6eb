"""Pins of the oracle's write path: dithered INT8 quantizer, band map, witness (CPU).

What the paper fixes and these tests check:
* no clipping: s = amax/126.5 keeps every code inside [-127, 127] (Sec. 4.2);
* the reconstruction error stays within half a step (Sec. 6.2 storage validation:
  |err| <= s/2, max ratio 1.0000);
* subtractive dither: over the dither, the residual is uniform and does not
  depend on the input (Sec. 4.2, classical dither theory);
* every RoPE pair lies inside one band, so band norms are unchanged by RoPE at
  any position (Lemma RoPE band unitarity);
* Cauchy-Schwarz per band bounds |q . r| and is attained when q_b is parallel
  to r_b in every band (Theorem black-box logit bound).
"""
import numpy as np
import pytest

import synth
from oracle import fpformats as fp
from oracle import philox, quantizer as qz


def _rows(n, d, seed, outliers=2):
    rng = np.random.default_rng(seed)
    sig = synth.channel_scales(rng, d, outliers, 10.0)
    return synth.bf16_round(rng.standard_normal((n, d)) * sig).astype(np.float64)


@pytest.mark.parametrize("d", [64, 128])
def test_no_clipping_and_half_step_error(d):
    x = _rows(4000, d, 3)
    code, s, xi, xh = qz.int8_quantize_slots(x, np.arange(4000), 2, 1, 99)
    assert code.min() >= -127 and code.max() <= 127
    amax = np.abs(x).max(axis=1)
    # the stored scale never lets amax/s exceed 126.5 (beyond fp32 rounding of the division)
    assert np.all(amax / s <= 126.5 * (1 + 2.0 ** -23))
    err = np.abs(xh - x)
    assert np.all(err <= s[:, None] * (0.5 + 2.0 ** -14))
    ratio = (err / (s[:, None] / 2)).max()
    assert 0.99 < ratio <= 1.0 + 2.0 ** -13


def test_scale_is_stored_fp16_rounded_up():
    x = _rows(2000, 128, 4)
    s = qz.int8_scale(x)
    q = fp.f32(np.abs(x).max(axis=1) / 126.5)
    assert np.all(s >= q)
    assert np.array_equal(s, s.astype(np.float16).astype(np.float64))
    prev = np.nextafter(s.astype(np.float16), np.float16(0)).astype(np.float64)
    assert np.all(prev < q)
    # tiny amax gives a subnormal fp16 scale that still never clips
    tiny = np.full((1, 64), 1e-5)
    c, st = qz.int8_encode(tiny, np.zeros((1, 64)))
    assert st[0] > 0 and np.abs(c).max() <= 127


def test_zero_row_and_extreme_values():
    x = np.zeros((3, 64))
    xi = philox.dither_values([0, 1, 2], 64, 0, 0, 5)
    c, s = qz.int8_encode(x, xi)
    assert np.all(s == 0) and np.all(c == 0)
    assert np.all(qz.int8_decode(c, s, xi) == 0)
    # x = +-amax maps to +-126 or +-127 depending on the dither
    x = np.zeros((512, 64))
    x[:, 0] = 3.0
    x[:, 1] = -3.0
    c, s, xi, _ = qz.int8_quantize_slots(x, np.arange(512), 0, 0, 6)
    assert set(np.unique(c[:, 0])) <= {126, 127} and set(np.unique(c[:, 1])) <= {-127, -126}
    assert len(np.unique(c[:, 0])) == 2


def test_subtractive_dither_residual_is_uniform_and_input_independent():
    """Enumerate all 256 dither values: for any input the residual (in steps) is the
    256-point lattice of spacing 1/256 inside [-1/2, 1/2], shifted by less than one
    spacing, so its variance is exactly (1 - 4^-8)/12 whatever the input."""
    lattice = (np.arange(256) - 127.5) / 256.0
    rng = np.random.default_rng(5)
    amax = 2.5
    for _ in range(40):
        xv = rng.uniform(-amax, amax)
        x = np.zeros((256, 8))
        x[:, 0] = amax
        x[:, 1] = xv
        xi = np.repeat(lattice[:, None], 8, axis=1)
        c, s = qz.int8_encode(x, xi)
        r = (qz.int8_decode(c, s, xi) - x)[:, 1] / s[0]
        rs = np.sort(r)
        gaps = np.diff(rs)
        assert np.allclose(gaps, 1 / 256, atol=1e-5)
        assert rs[0] >= -0.5 - 1e-5 and rs[-1] <= 0.5 + 1e-5
        assert abs(r.mean()) <= 1 / 512 + 1e-5
        assert abs(r.var() - (1 - 4.0 ** -8) / 12) < 1e-5


@pytest.mark.parametrize("d,B", [(64, 4), (128, 8), (128, 16), (16, 2)])
@pytest.mark.parametrize("layout", ["half", "interleaved"])
def test_band_map_keeps_pairs_together(d, B, layout):
    band = qz.band_index(d, B, layout)
    half = d // 2
    for j in range(half):
        a, b = (j, j + half) if layout == "half" else (2 * j, 2 * j + 1)
        assert band[a] == band[b]
        assert band[a] == j // (half // B)          # contiguous runs of pairs
    assert np.all(np.bincount(band) == d // B)


@pytest.mark.parametrize("layout", ["half", "interleaved"])
def test_lemma_rope_band_unitarity(layout):
    rng = np.random.default_rng(8)
    r = rng.standard_normal((50, 128)) * synth.channel_scales(rng, 128, 2, 10.0)
    before = qz.band_norms(r, 8, layout)
    for n in (1, 7, 4095, 131071, 10 ** 6):
        rot = synth.rope_rotate(r, np.full(50, n), 1e6, layout)
        assert np.allclose(qz.band_norms(rot, 8, layout), before, rtol=1e-12, atol=1e-12)
    # teeth: a band map that separates the two channels of one pair is not invariant
    band = qz.band_index(128, 8, layout).copy()
    partner = 64 if layout == "half" else 1
    j = int(np.flatnonzero(band != band[0])[0])
    band[partner], band[j] = band[j], band[partner]

    def norms(x):
        return np.stack([np.linalg.norm(x[:, band == b], axis=1) for b in range(8)], axis=1)
    rot = synth.rope_rotate(r, np.full(50, 12345), 1e6, layout)
    assert not np.allclose(norms(rot), norms(r), rtol=1e-3)


def test_witness_partition_identity_and_roundup():
    x = _rows(500, 128, 9)
    _, _, _, xh = qz.int8_quantize_slots(x, np.arange(500), 0, 0, 3)
    w = qz.witness(x, xh, 8)
    exact = qz.band_norms(xh - x, 8)
    assert np.all(w >= exact)
    assert np.all(w <= exact * (1 + 2.0 ** -10) + 2.0 ** -24)
    assert np.allclose(np.sum(w ** 2, axis=1), np.sum((xh - x) ** 2, axis=1), rtol=3e-3)
    assert np.all(qz.witness(x, x, 8) == 0)


def test_cauchy_schwarz_bound_and_its_equality_case():
    rng = np.random.default_rng(10)
    d, B = 128, 8
    band = qz.band_index(d, B)
    for _ in range(200):
        r = rng.standard_normal(d) * rng.uniform(0.01, 3)
        q = rng.standard_normal(d) * rng.uniform(0.1, 30)
        w = qz.band_norms(r[None], B)[0]
        qn = qz.band_norms(q[None], B)[0]
        assert abs(q @ r) <= qn @ w * (1 + 1e-12)
        # q_b parallel to r_b (positive multiples per band): equality
        lam = rng.uniform(0.1, 5, size=B)
        qa = r * lam[band]
        assert np.isclose(qa @ r, qz.band_norms(qa[None], B)[0] @ w, rtol=1e-12)


def test_fp8_raw_witness_is_residual_of_cast():
    x = _rows(300, 128, 11)
    xh = qz.fp8_raw(x)
    w = qz.witness(x, xh, 8)
    assert np.all(w >= qz.band_norms(xh - x, 8))
    # relative cast error of e4m3 is at most 2^-4 per element (3 mantissa bits, RNE)
    normal = np.abs(x) >= 2.0 ** -6
    assert np.all(np.abs(xh - x)[normal] <= np.abs(x)[normal] * 2.0 ** -4)
