"""Workload recipes and seeded generators (shared by oracle tests, GPU tests, bench).

Recipe (the synthetic stand-in for the paper's post-RoPE activations of 7B-class
GQA models, Sec. 6.3 quad report and the real-activation studies):

* pre-RoPE keys, values and queries are N(0, 1) * sigma_c per channel, with
  sigma_c = exp(U[ln 0.5, ln 4]) drawn once per (layer, head, tensor) and two
  seeded "massive activation" channels multiplied by 10;
* keys and queries are rotated by RoPE (theta_j = base^(-2j/d)) at their token
  positions; values carry no RoPE;
* everything is rounded to the storage dtype (fp32, or bf16 with
  round-to-nearest-even) and these stored values are what every consumer sees.

Every cell (layer, head, sequence, tensor, step) has its own PCG64 stream keyed
by ``SeedSequence(ROOT_SEED, spawn_key=...)`` so any cell can be regenerated
alone.  Nothing here quantizes, measures or attends.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

ROOT_SEED = 20260728
BLOCK = 16  # tokens per paged block


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    wid: int                 # numeric id used in seed keys
    n_layers: int
    n_q: int
    n_kv: int
    d: int
    bands: int
    rope_base: float
    dtype: str               # "f32" | "bf16"
    ctx: int                 # prefill length (max length for ragged mixes)
    batch: int
    steps: int
    ragged: bool = False
    len_lo: int = 0
    chunk: int = 0           # prefill-chunk tokens per step (serving mix)
    taus: tuple = ()
    n_outliers: int = 2
    outlier_mult: float = 10.0
    q_scale: float = 1.0     # < 1 gives the informative (unsaturated) regime
    rope_layout: str = "half"  # "half" (rotate_half pairs j, j+d/2) | "interleaved"

    @property
    def group(self) -> int:
        return self.n_q // self.n_kv

    def philox_seed(self) -> int:
        return 0x5EED000000000000 + self.wid

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


WORKLOADS = {
    # 1 layer, 1q/1kv, d=64, 4 bands, fp32, 256-token context, 16 decode steps
    "tiny-d64-s256": Workload("tiny-d64-s256", 1, 1, 1, 1, 64, 4, 1e4, "f32", 256, 1, 16),
    # 28 layers, 28q/4kv, d=128, 8 bands, bf16, 4k context, batch 8, 32 steps
    "gqa-28x4-d128-s4k-b8": Workload("gqa-28x4-d128-s4k-b8", 2, 28, 28, 4, 128, 8, 1e6,
                                     "bf16", 4096, 8, 32),
    # same shape at 32k context, batch 4, gate thresholds
    "gqa-28x4-d128-s32k-b4": Workload("gqa-28x4-d128-s32k-b4", 3, 28, 28, 4, 128, 8, 1e6,
                                      "bf16", 32768, 4, 8, taus=(0.05, 0.1, 0.2)),
    # long context: one sequence of 131072 tokens
    "gqa-28x4-d128-s131k-b1": Workload("gqa-28x4-d128-s131k-b1", 4, 28, 28, 4, 128, 8, 1e6,
                                       "bf16", 131072, 1, 8),
    # serving mix: 64 ragged sequences (log-uniform 512..32768), permuted paging,
    # one 2048-token prefill chunk written per step
    "serving-64seq-paged": Workload("serving-64seq-paged", 5, 28, 28, 4, 128, 8, 1e6,
                                    "bf16", 32768, 64, 8, ragged=True, len_lo=512, chunk=2048),
}

_TENSOR_ID = {"k": 0, "v": 1, "q": 2}


def cell_rng(wid: int, *key: int) -> np.random.Generator:
    """Independent PCG64 stream for one cell of a workload."""
    ss = np.random.SeedSequence(ROOT_SEED, spawn_key=(int(wid),) + tuple(int(k) for k in key))
    return np.random.Generator(np.random.PCG64(ss))


def channel_scales(rng: np.random.Generator, d: int, n_outliers: int, mult: float) -> np.ndarray:
    sig = np.exp(rng.uniform(math.log(0.5), math.log(4.0), size=d))
    if n_outliers > 0:
        idx = rng.choice(d, size=n_outliers, replace=False)
        sig[idx] *= mult
    return sig


def rope_rotate(x: np.ndarray, positions: np.ndarray, base: float, layout: str = "half") -> np.ndarray:
    """Rotate rows of x [n, d] by RoPE at the given positions (float64)."""
    x = np.asarray(x, dtype=np.float64)
    n, d = x.shape
    half = d // 2
    j = np.arange(half, dtype=np.float64)
    theta = base ** (-2.0 * j / d)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * theta[None, :]
    cos, sin = np.cos(ang), np.sin(ang)
    out = np.empty_like(x)
    if layout == "half":
        a, b = x[:, :half], x[:, half:]
        out[:, :half] = a * cos - b * sin
        out[:, half:] = b * cos + a * sin
    elif layout == "interleaved":
        a, b = x[:, 0::2], x[:, 1::2]
        out[:, 0::2] = a * cos - b * sin
        out[:, 1::2] = b * cos + a * sin
    else:
        raise ValueError(layout)
    return out


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float values to bf16 (nearest-even) and return the uint16 bit patterns."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return u.astype(np.uint16)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Values of x rounded to bf16 (nearest-even), returned as float32."""
    bits = to_bf16_bits(x).astype(np.uint32) << 16
    return bits.view(np.float32)


def _store(x: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32)
    if dtype == "bf16":
        return bf16_round(x)
    raise ValueError(dtype)


def gen_kv(wl: Workload, layer: int, kv_head: int, seq: int, tensor: str,
           positions: np.ndarray, step: int = -1) -> np.ndarray:
    """Stored K (post-RoPE) or V rows for one (layer, kv head, sequence) cell.

    ``step=-1`` is the prefill cell; ``step>=0`` the token written at decode step
    ``step``.  Returns float32 [len(positions), d] holding dtype-rounded values.
    """
    tid = _TENSOR_ID[tensor]
    srng = cell_rng(wl.wid, layer, kv_head, tid, 1 << 20)
    sig = channel_scales(srng, wl.d, wl.n_outliers, wl.outlier_mult)
    rng = cell_rng(wl.wid, layer, kv_head, tid, seq, step + 1)
    positions = np.asarray(positions)
    x = rng.standard_normal((positions.size, wl.d)) * sig[None, :]
    if tensor == "k":
        x = rope_rotate(x, positions, wl.rope_base, wl.rope_layout)
    return _store(x, wl.dtype)


def gen_q(wl: Workload, layer: int, seq: int, step: int, position: int) -> np.ndarray:
    """Stored post-RoPE queries [n_q, d] of one sequence at one decode step."""
    out = np.empty((wl.n_q, wl.d), dtype=np.float64)
    for h in range(wl.n_q):
        srng = cell_rng(wl.wid, layer, h, _TENSOR_ID["q"], 1 << 20)
        sig = channel_scales(srng, wl.d, wl.n_outliers, wl.outlier_mult)
        rng = cell_rng(wl.wid, layer, h, _TENSOR_ID["q"], seq, step + 1)
        out[h] = rng.standard_normal(wl.d) * sig * wl.q_scale
    out = rope_rotate(out, np.full(wl.n_q, position), wl.rope_base, wl.rope_layout)
    return _store(out, wl.dtype)


def serving_lengths(n: int, lo: int, hi: int, wid: int = 5) -> np.ndarray:
    """Sequence lengths round(exp(U[ln lo, ln hi])) for a ragged serving mix."""
    rng = cell_rng(wid, 1 << 21)
    return np.rint(np.exp(rng.uniform(math.log(lo), math.log(hi), size=n))).astype(np.int64)


def block_table(seq_capacity: np.ndarray, permute: bool, seed_key: int = 0) -> tuple[np.ndarray, int]:
    """Paged block table for sequences that can hold ``seq_capacity[b]`` tokens.

    Returns (table int32 [batch, max_blocks], num_blocks).  Unused entries are 0
    and never read.  With ``permute`` the physical blocks are a seeded random
    permutation, so consecutive tokens of a sequence land in scattered slots.
    """
    nb = [(int(c) + BLOCK - 1) // BLOCK for c in seq_capacity]
    total = int(sum(nb))
    maxb = max(nb) if nb else 0
    ids = np.arange(total, dtype=np.int64)
    if permute:
        ids = cell_rng(99, seed_key, 1 << 22).permutation(total)
    table = np.zeros((len(nb), max(maxb, 1)), dtype=np.int32)
    o = 0
    for b, n in enumerate(nb):
        table[b, :n] = ids[o:o + n]
        o += n
    return table, total


def decode_positions(prefill: int, step: int) -> int:
    """Token position written (and queried) at decode step ``step``: prefill occupies
    positions 0..prefill-1, step i writes position prefill+i and attends over
    prefill+i+1 tokens."""
    return prefill + step


def slots_of(table: np.ndarray, seq: int, positions: np.ndarray) -> np.ndarray:
    """Physical slots (block*16 + offset) of token positions of one sequence."""
    positions = np.asarray(positions, dtype=np.int64)
    return table[seq, positions // BLOCK].astype(np.int64) * BLOCK + positions % BLOCK
