"""WitCert hot path on MI355X: dithered INT8 KV write with residual witness,
metered GQA decode attention, threshold gate and exact fallback.

The compute lives in libwitcert.so (HIP, gfx950; C-ABI in include/witcert.h);
this package is its Python binding.  Importing it does not load the library;
the first call does, and fails loudly if the library is not built.
"""
from .api import (  # noqa: F401
    KINDS,
    block_repair,
    LAYOUTS,
    PagedCache,
    cache_bytes,
    decode_workspace,
    exact_decode_attention,
    gate,
    joint_decode_gate,
    metered_decode_attention,
    metered_decode_gate,
    step_metered_decode_gate,
    step_certified_decode,
    step_certified_decode_speculative,
    certified_workspace,
    step_metered_decode_gate_noalloc,
    quantize_write,
    quantize_write_pair,
    repair_workspace,
    repair_write_back,
    select_outlier_pairs,
    speculative_split_tokens,
    split_tokens_for,
    tierb_decode_attention,
    tierb_delta_loc,
    witness,
)
from ._lib import LIB_PATH, WitCertError, lib  # noqa: F401
