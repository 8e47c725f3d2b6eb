"""Philox4x32-10 counter-based generator, from its published definition.

Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3",
SC'11, Sec. 3 (the Philox S-box family).  The paper draws its dither from this
generator with a tuple counter so that the read side can regenerate exactly what
the write side used (Sec. 6.2, research kernels: five-tuple counter; Sec. 6.2,
storage side: the counter holds the cache slot rather than the token's position
in its sequence).

One round on a 4x32-bit counter (x0, x1, x2, x3) with 2x32-bit key (k0, k1):
    (hi0, lo0) = M0 * x0 as a 64-bit product,  (hi1, lo1) = M1 * x2
    x' = (hi1 ^ x1 ^ k0,  lo1,  hi0 ^ x3 ^ k1,  lo0)
and between rounds the key is bumped by the Weyl constants (W0, W1) mod 2^32.
Ten rounds, the key bumped after each of the first nine.  Constants are the
published Philox4x32 multipliers and the golden-ratio / sqrt(3)-1 Weyl words.

Pinned against rocRAND's philox4x32_10 engine (tests/test_oracle_philox.py).
"""
from __future__ import annotations

import numpy as np

M0 = np.uint64(0xD2511F53)
M1 = np.uint64(0xCD9E8D57)
W0 = np.uint64(0x9E3779B9)
W1 = np.uint64(0xBB67AE85)
MASK = np.uint64(0xFFFFFFFF)
SH = np.uint64(32)


def philox4x32_10(counter: np.ndarray, key: tuple[int, int]) -> np.ndarray:
    """counter: uint32-like [..., 4]; key: (k0, k1).  Returns uint32 [..., 4]."""
    c = np.asarray(counter, dtype=np.uint64) & MASK
    x0, x1, x2, x3 = c[..., 0], c[..., 1], c[..., 2], c[..., 3]
    k0 = np.uint64(int(key[0]) & 0xFFFFFFFF)
    k1 = np.uint64(int(key[1]) & 0xFFFFFFFF)
    for rnd in range(10):
        if rnd > 0:
            k0 = (k0 + W0) & MASK
            k1 = (k1 + W1) & MASK
        p0 = M0 * x0            # < 2^64: exact in uint64
        p1 = M1 * x2
        hi0, lo0 = p0 >> SH, p0 & MASK
        hi1, lo1 = p1 >> SH, p1 & MASK
        x0, x1, x2, x3 = (hi1 ^ x1 ^ k0), lo1, (hi0 ^ x3 ^ k1), lo0
    return np.stack([x0, x1, x2, x3], axis=-1).astype(np.uint32)


def seed_key(seed: int) -> tuple[int, int]:
    """The 64-bit dither seed split into the 2x32-bit Philox key (low word first)."""
    return (seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF)


def dither_counter(slot, group, layer: int, kv_head: int) -> np.ndarray:
    """Counter words for the dither of channels 16*group .. 16*group+15 of one slot.

    Reading of the paper's serving tuple (layer, kv_head, slot, channel):
    x0 = channel group, x1/x2 = low/high word of the slot, x3 = layer<<16 | kv_head.
    Keys and values of a slot share the counter (the tuple has no K/V field).
    """
    slot = np.asarray(slot, dtype=np.int64)
    group = np.asarray(group, dtype=np.int64)
    slot, group = np.broadcast_arrays(slot, group)
    out = np.empty(slot.shape + (4,), dtype=np.uint64)
    out[..., 0] = group.astype(np.uint64)
    out[..., 1] = slot.astype(np.uint64) & 0xFFFFFFFF
    out[..., 2] = (slot.astype(np.uint64) >> np.uint64(32)) & 0xFFFFFFFF
    out[..., 3] = np.uint64(((int(layer) & 0xFFFF) << 16) | (int(kv_head) & 0xFFFF))
    return out


def dither_bytes(slots, d: int, layer: int, kv_head: int, seed: int) -> np.ndarray:
    """uint8 [n, d]: byte u of channel c = byte (c mod 4) of output word (c mod 16) div 4
    of the Philox call for group c div 16 (little-endian bytes within each word)."""
    slots = np.atleast_1d(np.asarray(slots, dtype=np.int64))
    ngroups = d // 16
    ctr = dither_counter(slots[:, None], np.arange(ngroups)[None, :], layer, kv_head)
    words = philox4x32_10(ctr, seed_key(seed))             # [n, groups, 4] uint32
    by = words.astype("<u4").view(np.uint8)                # [n, groups, 16]
    return by.reshape(slots.size, d)


def dither_values(slots, d: int, layer: int, kv_head: int, seed: int) -> np.ndarray:
    """float64 [n, d] dither xi = (u - 127.5)/256 in (-1/2, 1/2): the 8-bit midpoint
    lattice reading of xi ~ U[-1/2, 1/2) (Sec. 4.2, subtractive dither)."""
    u = dither_bytes(slots, d, layer, kv_head, seed).astype(np.float64)
    return (u - 127.5) / 256.0
