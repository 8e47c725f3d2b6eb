"""Pins of the oracle's floating-point storage formats (CPU)."""
import numpy as np
import torch

from oracle import fpformats as fp

ALL_F16 = np.arange(0, 0x7C00, dtype=np.uint16).view(np.float16).astype(np.float64)  # +0 .. max finite


def test_f16_round_up_is_smallest_fp16_not_below():
    rng = np.random.default_rng(0)
    x = np.concatenate([
        np.exp(rng.uniform(np.log(1e-9), np.log(6e4), 20000)),
        ALL_F16[1:2000],                                   # exact fp16 values stay
        ALL_F16[1:2000] * (1 + 1e-9),                      # just above -> next value
        [0.0, 65504.0],
    ])
    got = fp.f16_round_up(x)
    idx = np.searchsorted(ALL_F16, x, side="left")          # brute force: first value >= x
    assert np.array_equal(got, ALL_F16[idx])


def test_f32_emulation_is_correctly_rounded():
    rng = np.random.default_rng(1)
    a = rng.standard_normal(50000).astype(np.float32) * np.float32(100)
    b = (rng.standard_normal(50000) * 0.01).astype(np.float32)
    a64, b64 = a.astype(np.float64), b.astype(np.float64)
    assert np.array_equal(fp.f32(a64 * b64), (a * b).astype(np.float64))
    assert np.array_equal(fp.f32(a64 + b64), (a + b).astype(np.float64))
    nz = b != 0
    assert np.array_equal(fp.f32(a64[nz] / b64[nz]), (a[nz] / b[nz]).astype(np.float64))


def _all_bf16():
    bits = np.arange(65536, dtype=np.uint32) << 16
    v = bits.view(np.float32)
    return v[np.isfinite(v)].astype(np.float64)


def test_e4m3_matches_torch_cast_exhaustively_in_range():
    x = _all_bf16()
    inr = np.abs(x) < 464.0          # torch's CPU cast is finite here (RNE, no overflow)
    t = torch.from_numpy(x[inr].astype(np.float32)).to(torch.float8_e4m3fn)
    ref_val = t.to(torch.float64).numpy()
    ref_bits = t.view(torch.uint8).numpy()
    assert np.array_equal(fp.e4m3_round(x[inr]), ref_val)
    assert np.array_equal(fp.e4m3_encode(x[inr]), ref_bits)


def test_e4m3_saturates_and_roundtrips():
    x = _all_bf16()
    big = np.abs(x) >= 448.0
    assert np.all(np.abs(fp.e4m3_round(x[big])) == 448.0)
    v = fp.e4m3_round(x)
    assert np.array_equal(fp.e4m3_decode(fp.e4m3_encode(x)), v)
    # every finite code decodes to a value that rounds to itself
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)
    vals = fp.e4m3_decode(codes)
    assert np.array_equal(fp.e4m3_round(vals), vals)
    assert np.array_equal(fp.e4m3_encode(vals), codes)
