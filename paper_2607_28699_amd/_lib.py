"""ctypes view of libwitcert.so (the C-ABI declared in include/witcert.h).

Loading fails loudly when the library has not been built: there is no
fallback implementation of any step of the hot path.
"""
from __future__ import annotations

import ctypes
import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libwitcert.so")

WC_OK, WC_EINVAL, WC_EUNSUPPORTED, WC_EHIP, WC_EWORKSPACE, WC_ESCRATCH = 0, -1, -2, -3, -4, -5
WC_NOALLOC_SCRATCH_BYTES = 16 << 20
WC_F32, WC_BF16, WC_F16 = 0, 1, 2
WC_KIND_INT8_DITHER, WC_KIND_FP8_RAW, WC_KIND_BF16 = 0, 1, 2
WC_ROPE_HALF, WC_ROPE_INTERLEAVED = 0, 1
WC_BLOCK_TOKENS = 16

EXPORTS = (
    "wc_strerror", "wc_version", "wc_cache_bytes", "wc_quantize_write", "wc_quantize_write_pair",
    "wc_witness", "wc_select_workspace_size", "wc_select_outlier_pairs", "wc_decode_workspace_size",
    "wc_decode_split_tokens", "wc_speculative_split_tokens", "wc_metered_decode_attention",
    "wc_metered_decode_gate", "wc_step_metered_decode_gate", "wc_step_metered_decode_gate_noalloc",
    "wc_tierb_decode_attention", "wc_tierb_delta_loc", "wc_joint_decode_gate", "wc_gate",
    "wc_exact_decode_attention", "wc_block_repair", "wc_block_repair_workspace_size",
    "wc_repair_write_back", "wc_certified_workspace_size", "wc_step_certified_decode",
    "wc_step_certified_decode_speculative",
)


class WcCache(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
        ("n_bands", ctypes.c_int32), ("rope_layout", ctypes.c_int32), ("layer", ctypes.c_int32),
        ("num_blocks", ctypes.c_int64), ("seed", ctypes.c_uint64),
        ("k_data", ctypes.c_void_p), ("v_data", ctypes.c_void_p), ("k_scale", ctypes.c_void_p),
        ("v_scale", ctypes.c_void_p), ("k_witness", ctypes.c_void_p),
        ("n_outlier_pairs", ctypes.c_int32), ("group_scales", ctypes.c_int32),
        ("outlier_pairs", ctypes.c_void_p), ("k_outlier", ctypes.c_void_p),
        ("v_resid", ctypes.c_void_p), ("v_norm", ctypes.c_void_p),
        ("repaired", ctypes.c_void_p), ("exact_k", ctypes.c_void_p), ("exact_v", ctypes.c_void_p),
    ]


class WitCertError(RuntimeError):
    pass


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise WitCertError(
            f"{LIB_PATH} is missing: build the HIP library first "
            "(python -m paper_2607_28699_amd.build_lib); there is no CPU fallback")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u64, f32, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64,
                                  ctypes.c_float, ctypes.c_size_t)
    cp = ctypes.POINTER(WcCache)
    sig = {
        "wc_strerror": (ctypes.c_char_p, [ctypes.c_int]),
        "wc_version": (ctypes.c_int, []),
        "wc_cache_bytes": (sz, [ctypes.c_int, i64, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.POINTER(sz)]),
        "wc_select_workspace_size": (sz, [i64, ctypes.c_int, ctypes.c_int]),
        "wc_select_outlier_pairs": (ctypes.c_int, [vp, ctypes.c_int, i64, ctypes.c_int, ctypes.c_int,
                                                   ctypes.c_int, ctypes.c_int, vp, vp, sz, vp]),
        "wc_quantize_write": (ctypes.c_int, [cp, vp, vp, ctypes.c_int, vp, i64, vp]),
        "wc_quantize_write_pair": (ctypes.c_int, [cp, cp, vp, vp, ctypes.c_int, vp, i64, vp]),
        "wc_witness": (ctypes.c_int, [vp, ctypes.c_int, vp, ctypes.c_int, i64, ctypes.c_int,
                                      ctypes.c_int, ctypes.c_int, vp, vp]),
        "wc_decode_workspace_size": (sz, [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                          i64, ctypes.c_int]),
        "wc_decode_split_tokens": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, i64, i64, ctypes.c_int]),
        "wc_speculative_split_tokens": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, i64, i64, ctypes.c_int]),
        "wc_metered_decode_attention": (ctypes.c_int, [cp, vp, ctypes.c_int, ctypes.c_int,
                                                       ctypes.c_int, vp, ctypes.c_int, vp, i64, f32,
                                                       vp, ctypes.c_int, vp, vp, ctypes.c_int, vp,
                                                       sz, vp]),
        "wc_metered_decode_gate": (ctypes.c_int, [cp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                                  vp, ctypes.c_int, vp, i64, f32, vp, ctypes.c_int,
                                                  vp, vp, ctypes.c_int, f32, vp, vp, vp, vp, sz,
                                                  vp]),
        "wc_step_metered_decode_gate": (ctypes.c_int, [cp, cp, vp, vp, ctypes.c_int, vp, vp, ctypes.c_int,
                                                       ctypes.c_int, ctypes.c_int, vp, ctypes.c_int, vp, i64,
                                                       f32, vp, ctypes.c_int, vp, vp, ctypes.c_int, f32, vp,
                                                       vp, vp, vp, sz, vp]),
        "wc_certified_workspace_size": (sz, [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                             i64, ctypes.c_int]),
        "wc_step_certified_decode": (ctypes.c_int, [cp, cp, vp, vp, ctypes.c_int, vp, vp, ctypes.c_int,
                                                    ctypes.c_int, ctypes.c_int, vp, ctypes.c_int, vp, i64,
                                                    f32, vp, ctypes.c_int, vp, vp, ctypes.c_int, f32, vp,
                                                    vp, vp, vp, sz, vp]),
        "wc_step_certified_decode_speculative": (ctypes.c_int, [cp, cp, vp, vp, ctypes.c_int, vp, vp, ctypes.c_int,
                                                                ctypes.c_int, ctypes.c_int, vp, ctypes.c_int, vp,
                                                                i64, f32, vp, ctypes.c_int, vp, vp, ctypes.c_int,
                                                                f32, vp, vp, vp, vp, sz, vp]),
        "wc_step_metered_decode_gate_noalloc": (ctypes.c_int, [cp, cp, vp, vp, ctypes.c_int, vp, vp,
                                                               ctypes.c_int, ctypes.c_int, ctypes.c_int, vp,
                                                               ctypes.c_int, vp, i64, f32, vp, ctypes.c_int, vp,
                                                               vp, ctypes.c_int, f32, vp, vp, vp, vp]),
        "wc_tierb_delta_loc": (ctypes.c_double, [ctypes.c_double, ctypes.c_int, ctypes.c_int, ctypes.c_int]),
        "wc_tierb_decode_attention": (ctypes.c_int, [cp, vp, ctypes.c_int, ctypes.c_int,
                                                     ctypes.c_int, vp, ctypes.c_int, vp, i64, f32,
                                                     vp, ctypes.c_int, vp, vp, ctypes.c_int, f32,
                                                     vp, sz, vp]),
        "wc_joint_decode_gate": (ctypes.c_int, [cp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                                vp, ctypes.c_int, vp, i64, f32, vp, ctypes.c_int,
                                                vp, vp, vp, ctypes.c_int, f32, f32, f32, vp, vp, vp,
                                                vp, sz, vp]),
        "wc_block_repair": (ctypes.c_int, [cp, cp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, vp,
                                           ctypes.c_int, vp, i64, f32, ctypes.c_int, f32, f32,
                                           ctypes.c_int, vp, sz, vp, ctypes.c_int, vp, vp, vp, vp, vp,
                                           vp, sz, vp]),
        "wc_block_repair_workspace_size": (sz, [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                                ctypes.c_int]),
        "wc_repair_write_back": (ctypes.c_int, [cp, ctypes.c_int, vp, ctypes.c_int, vp, vp, vp, ctypes.c_int,
                                                vp, vp]),
        "wc_gate": (ctypes.c_int, [vp, vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, f32, vp, vp,
                                   vp, vp]),
        "wc_exact_decode_attention": (ctypes.c_int, [cp, vp, ctypes.c_int, ctypes.c_int,
                                                     ctypes.c_int, vp, ctypes.c_int, vp, i64, f32,
                                                     vp, vp, ctypes.c_int, ctypes.c_int, vp, sz,
                                                     vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    del u64, i32
    _lib = L
    return L


def check(status: int, what: str) -> None:
    if status != WC_OK:
        msg = lib().wc_strerror(status).decode()
        raise WitCertError(f"{what} failed: {msg} ({status})")
