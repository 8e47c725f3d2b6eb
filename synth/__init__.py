"""Seeded synthetic inputs for the WitCert hot path.

This package is the only code shared by the oracle side and the HIP side.  It
draws keys, values and queries with the statistics the paper's workloads have
(per-channel scales, a few massive-activation channels, keys and queries
stored after RoPE), rounds them to the storage dtype, and lays out paged block
tables.  It contains none of the method's arithmetic: no quantizer, no
witness, no attention, no meter.
"""
from .workloads import (  # noqa: F401
    WORKLOADS,
    Workload,
    bf16_round,
    block_table,
    cell_rng,
    channel_scales,
    decode_positions,
    gen_kv,
    gen_q,
    rope_rotate,
    serving_lengths,
    slots_of,
    to_bf16_bits,
)
