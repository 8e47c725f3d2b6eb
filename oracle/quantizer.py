"""Write-path definitions: band map, dithered INT8 quantizer, raw fp8 cast, witness.

Band map (Sec. 4.1, Tier A; Lemma RoPE band unitarity).  The d/2 RoPE frequency
pairs are grouped into B contiguous bands of P = d/(2B) pairs; band b holds the
coordinates of pairs bP .. bP+P-1, so every pair lies inside one band.  With the
rotate-half layout pair j is channels (j, j + d/2); with the interleaved layout
it is channels (2j, 2j+1).  The paper does not state its layout; rotate-half is
our default reading.

Dithered quantizer (Sec. 4.2, subtractive dither; Sec. 6.2, research kernels):
    xhat = s * (round(x/s + xi) - xi),   s = amax / (Q - 1/2) = amax / 126.5,
quantizing with the *stored* fp16 scale.  Operation by operation, in fp32:
    s      = f16_round_up(f32(amax / 126.5))
    inv_s  = f32(1 / s)               (0 when s == 0)
    y      = f32(x * inv_s)
    z      = f32(y + xi)
    code   = round-half-to-even(z)    in [-127, 127]; never clipped
Decoding is exact: xhat = s * (code - xi) in float64.

Residual witness (Eq. witness): w_{t,b} = ||(xhat_t - x_t)_b||, stored in fp16
rounded up.  Parity: codes and scales are pinned by the error bound, the
no-clipping guarantee and the subtractive residual law; the witness by the
partition identity, Lemma RoPE band unitarity and the Cauchy-Schwarz bound.
"""
from __future__ import annotations

import numpy as np

from .fpformats import e4m3_round, f16_round_up, f32
from .philox import dither_values

Q_TOP = 127
S_DIV = Q_TOP - 0.5  # 126.5


def band_index(d: int, n_bands: int, layout: str = "half") -> np.ndarray:
    """int [d]: band of each channel."""
    if d % (2 * n_bands):
        raise ValueError("d must be a multiple of 2*B")
    half = d // 2
    pairs_per_band = half // n_bands
    band = np.empty(d, dtype=np.int64)
    for j in range(half):                       # pair j
        b = j // pairs_per_band
        if layout == "half":
            band[j] = b
            band[j + half] = b
        elif layout == "interleaved":
            band[2 * j] = b
            band[2 * j + 1] = b
        else:
            raise ValueError(layout)
    return band


def int8_scale(x: np.ndarray) -> np.ndarray:
    """Per-row fp16 scale s (float64 values) of x [n, d]."""
    amax = np.max(np.abs(np.asarray(x, dtype=np.float64)), axis=-1)
    return f16_round_up(f32(amax / S_DIV))


def int8_encode(x: np.ndarray, xi: np.ndarray):
    """Codes (int64 [n, d]) and scales (float64 [n]) of rows x with dither xi."""
    x = np.asarray(x, dtype=np.float64)
    s = int8_scale(x)
    with np.errstate(divide="ignore"):
        inv_s = np.where(s > 0, f32(1.0 / np.where(s > 0, s, 1.0)), 0.0)
    y = f32(x * inv_s[:, None])
    z = f32(y + xi)
    code = np.rint(z).astype(np.int64)          # numpy rint: ties to even
    return code, s


def int8_decode(code: np.ndarray, s: np.ndarray, xi: np.ndarray) -> np.ndarray:
    return np.asarray(s, dtype=np.float64)[..., None] * (np.asarray(code, dtype=np.float64) - xi)


def int8_quantize_slots(x: np.ndarray, slots, layer: int, kv_head: int, seed: int):
    """Quantize rows x [n, d] written to ``slots``: returns (code, s, xi, xhat)."""
    x = np.asarray(x, dtype=np.float64)
    xi = dither_values(slots, x.shape[-1], layer, kv_head, seed)
    code, s = int8_encode(x, xi)
    return code, s, xi, int8_decode(code, s, xi)


def fp8_raw(x: np.ndarray) -> np.ndarray:
    """Reconstruction of the raw fp8 E4M3 cast (no scale), float64."""
    return e4m3_round(x)


def band_norms(r: np.ndarray, n_bands: int, layout: str = "half") -> np.ndarray:
    """Exact (float64) per-band Euclidean norms of rows r [n, d] -> [n, B]."""
    r = np.asarray(r, dtype=np.float64)
    band = band_index(r.shape[-1], n_bands, layout)
    out = np.zeros(r.shape[:-1] + (n_bands,), dtype=np.float64)
    for b in range(n_bands):
        out[..., b] = np.sqrt(np.sum(r[..., band == b] ** 2, axis=-1))
    return out


def witness(x: np.ndarray, xhat: np.ndarray, n_bands: int, layout: str = "half") -> np.ndarray:
    """Stored witness (fp16 rounded up, as float64) of any cache-preserving scheme:
    the band norms of the residual xhat - x (Eq. witness)."""
    r = np.asarray(xhat, dtype=np.float64) - np.asarray(x, dtype=np.float64)
    return f16_round_up(band_norms(r, n_bands, layout))
