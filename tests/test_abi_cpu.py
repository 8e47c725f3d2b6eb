"""The C-ABI library loads and exports every entry point of include/witcert.h;
host-side argument checks and size queries work without a GPU (no compute call)."""
import ctypes
import os
import re

import pytest

from paper_2607_28699_amd import _lib

HDR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "witcert.h")


def declared_functions():
    text = open(HDR).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wc_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(_lib.LIB_PATH):
        pytest.fail("libwitcert.so is not built (run __graft_entry__.build())")
    return _lib.lib()


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert set(names) == set(_lib.EXPORTS)
    for n in names:
        assert hasattr(L, n), n


def test_status_strings_and_version(L):
    assert L.wc_strerror(0) == b"ok"
    assert L.wc_strerror(_lib.WC_EINVAL) == b"invalid argument"
    assert L.wc_strerror(_lib.WC_EWORKSPACE) == b"workspace too small"
    assert L.wc_version() >= 100


def test_cache_byte_account(L):
    sizes = (ctypes.c_size_t * 8)()
    # one KV head, 32768 tokens, d = 128, B = 8: 128 + 128 + 2 + 2 + 16 = 276 B per token
    tot = L.wc_cache_bytes(_lib.WC_KIND_INT8_DITHER, 2048, 1, 128, 8, 0, 0, 0, sizes)
    assert tot == 32768 * 276
    assert list(sizes) == [32768 * 128, 32768 * 128, 65536, 65536, 32768 * 16, 0, 0, 0]
    assert L.wc_cache_bytes(_lib.WC_KIND_FP8_RAW, 2048, 1, 128, 8, 0, 0, 0, sizes) == 32768 * 272
    assert L.wc_cache_bytes(_lib.WC_KIND_BF16, 2048, 1, 128, 0, 0, 0, 0, sizes) == 32768 * 512
    assert L.wc_cache_bytes(7, 1, 1, 128, 8, 0, 0, 0, sizes) == 0
    # bypassed pairs: 2m fp16 values per token and KV head (Table 6: 16 B at m = 4)
    for m in (2, 4, 8, 16):
        tot = L.wc_cache_bytes(_lib.WC_KIND_INT8_DITHER, 2048, 1, 128, 8, m, 0, 0, sizes)
        assert sizes[5] == 32768 * 4 * m and tot == 32768 * (276 + 4 * m)
    for bad in (-2, 3, 18):
        assert L.wc_cache_bytes(_lib.WC_KIND_INT8_DITHER, 2048, 1, 128, 8, bad, 0, 0, sizes) == 0
    assert L.wc_cache_bytes(_lib.WC_KIND_FP8_RAW, 2048, 1, 128, 8, 4, 0, 0, sizes) == 0
    # value side: 2 + 2 bytes per token-head (residual and value norms), quantized kinds only
    tot = L.wc_cache_bytes(_lib.WC_KIND_INT8_DITHER, 2048, 1, 128, 8, 0, 1, 0, sizes)
    assert tot == 32768 * 280 and sizes[6] == sizes[7] == 65536
    assert L.wc_cache_bytes(_lib.WC_KIND_FP8_RAW, 2048, 1, 128, 8, 0, 1, 0, sizes) == 32768 * 276
    assert L.wc_cache_bytes(_lib.WC_KIND_BF16, 2048, 1, 128, 0, 0, 1, 0, sizes) == 0
    # group scales: one fp16 scale per 32-channel group and tensor, INT8 only: K + V
    # take 272 bytes per token-head (Table 4), 288 with the 16-byte key witness
    tot = L.wc_cache_bytes(_lib.WC_KIND_INT8_DITHER, 2048, 1, 128, 8, 0, 0, 1, sizes)
    assert tot == 32768 * 288 and sizes[2] == sizes[3] == 32768 * 8
    assert sizes[0] + sizes[1] + sizes[2] + sizes[3] == 32768 * 272
    assert L.wc_cache_bytes(_lib.WC_KIND_FP8_RAW, 2048, 1, 128, 8, 0, 0, 1, sizes) == 0


def test_workspace_size_and_argument_checks(L):
    n = L.wc_decode_workspace_size(4, 28, 4, 128, 32768, 0)
    assert n > 0 and n % 4 == 0
    # partial records (batch, q heads, 64 splits, head_dim + 8 floats), one int32 per
    # (sequence, KV head) for the fused gate, each part rounded up to 256 bytes, then
    # the block segments: per (query head, split) 4 waves x 2 slots of 16 bytes (a
    # wave's 8 pages touch at most 2 of the 256-token repair blocks)
    assert L.wc_decode_workspace_size(4, 28, 4, 128, 32768, 512) == \
        4 * 28 * 64 * 136 * 4 + 256 + 4 * 28 * 64 * 8 * 16
    assert L.wc_decode_workspace_size(-1, 28, 4, 128, 100, 0) == 0
    # null cache / pointers are rejected before anything is launched
    assert L.wc_quantize_write(None, None, None, 0, None, 1, None) == _lib.WC_EINVAL
    c = _lib.WcCache(0, 96, 1, 8, 0, 0, 1, 0, 16, 16, 16, 16, 16, 0, 0, None, None, None, None)
    assert L.wc_quantize_write(ctypes.byref(c), 16, 16, 0, 16, 1, None) == _lib.WC_EUNSUPPORTED
    c.head_dim = 128
    c.k_data = 8                              # misaligned
    assert L.wc_quantize_write(ctypes.byref(c), 16, 16, 0, 16, 1, None) == _lib.WC_EINVAL
    assert L.wc_gate(None, None, 1, 28, 7, 0.2, None, None, None, None) == _lib.WC_EINVAL
    assert L.wc_witness(None, 0, None, 0, 4, 128, 7, 0, None, None) == _lib.WC_EINVAL
    c.k_data = 16
    # workspace too small
    st = L.wc_metered_decode_attention(ctypes.byref(c), 16, 1, 1, 7, 16, 4, 16, 64, 0.1, 16, 0,
                                       16, 16, 0, 16, 8, None)
    assert st == _lib.WC_EWORKSPACE
    # bypassed pairs: INT8 only, m even and <= 16, pair list and value array required
    c.n_outlier_pairs = 4
    assert L.wc_quantize_write(ctypes.byref(c), 16, 16, 0, 16, 1, None) == _lib.WC_EINVAL
    c.outlier_pairs, c.k_outlier = 16, 16
    c.n_outlier_pairs = 3
    assert L.wc_quantize_write(ctypes.byref(c), 16, 16, 0, 16, 1, None) == _lib.WC_EINVAL
    c.n_outlier_pairs, c.kind = 4, _lib.WC_KIND_FP8_RAW
    assert L.wc_quantize_write(ctypes.byref(c), 16, 16, 0, 16, 1, None) == _lib.WC_EINVAL
    c.kind = _lib.WC_KIND_INT8_DITHER
    c.k_outlier = 24                          # misaligned
    assert L.wc_quantize_write(ctypes.byref(c), 16, 16, 0, 16, 1, None) == _lib.WC_EINVAL
    c.k_outlier, c.n_outlier_pairs, c.outlier_pairs = None, 0, None
    # value side: both arrays or neither; the joint decode needs it
    c.v_resid = 16
    assert L.wc_quantize_write(ctypes.byref(c), 16, 16, 0, 16, 1, None) == _lib.WC_EINVAL
    c.v_resid = None
    st = L.wc_joint_decode_gate(ctypes.byref(c), 16, 1, 1, 7, 16, 4, 16, 64, 0.1, 16, 0, 16, 16, 16,
                                0, 0.0, 0.2, 0.05, 16, 16, None, 16, 1 << 20, None)
    assert st == _lib.WC_EINVAL
    # pair selection: m within the pairs, head_dim 64 / 128, n_tok >= 1, a workspace of
    # float64 partial energies per (KV head, chunk of 2048 rows, pair), up to 64 chunks
    assert L.wc_select_workspace_size(131072, 4, 128) == 4 * 64 * 64 * 8
    assert L.wc_select_workspace_size(1000, 2, 64) == 2 * 1 * 32 * 8
    assert L.wc_select_workspace_size(10 ** 7, 1, 128) == 64 * 64 * 8
    assert L.wc_select_workspace_size(0, 4, 128) == 0
    assert L.wc_select_outlier_pairs(16, 1, 10, 4, 128, 0, 65, 16, 16, 4096, None) == _lib.WC_EINVAL
    assert L.wc_select_outlier_pairs(16, 1, 0, 4, 128, 0, 4, 16, 16, 4096, None) == _lib.WC_EINVAL
    assert L.wc_select_outlier_pairs(16, 1, 10, 4, 96, 0, 4, 16, 16, 4096, None) == _lib.WC_EUNSUPPORTED
    assert L.wc_select_outlier_pairs(None, 1, 10, 4, 128, 0, 4, 16, 16, 4096, None) == _lib.WC_EINVAL
    assert L.wc_select_outlier_pairs(16, 1, 10, 4, 128, 0, 4, 16, 16, 8, None) == _lib.WC_EWORKSPACE
    assert L.wc_select_outlier_pairs(16, 1, 10, 4, 128, 0, 0, None, None, 0, None) == _lib.WC_OK


def test_split_tokens_query(L):
    # the library's choice is a multiple of 64, at least 256, and an explicit
    # request is rounded up to a multiple of 64
    for batch, n_kv, s in ((4, 4, 32769), (1, 4, 131072), (8, 4, 4096), (1, 1, 10)):
        st = L.wc_decode_split_tokens(batch, n_kv, s, 0, 0)
        assert st >= 256 and st % 64 == 0
        # balanced over the total tokens: the same choice when every length is s
        if s >= 256:
            assert L.wc_decode_split_tokens(batch, n_kv, s, batch * s, 0) == st
    assert L.wc_decode_split_tokens(4, 4, 32769, 0, 100) == 128
    assert L.wc_decode_split_tokens(4, 0, 100, 0, 0) == 0
    assert L.wc_decode_split_tokens(-1, 4, 100, 0, 0) == 0
    # a ragged batch (64 sequences, 496k tokens, longest 32k): splits of ~3.9k tokens
    # instead of 16k from the longest alone
    assert L.wc_decode_split_tokens(64, 4, 32768, 0, 0) == 16384
    assert L.wc_decode_split_tokens(64, 4, 32768, 496384, 0) == 3904


def test_speculative_split_tokens_query(L):
    """The speculative step's split: about 256 workgroups per decode instead of 512
    (its one launch holds both decodes' workgroups), so about twice the decode
    calls' split where that split is not at its floor of 256 tokens; an explicit
    request is rounded as for the decode calls."""
    # 32k x 4 sequences, 4 KV heads: 16 splits of 2112 tokens (512 workgroups in
    # the step's launch) against 31 of 1088
    assert L.wc_decode_split_tokens(4, 4, 32770, 4 * 32770, 0) == 1088
    assert L.wc_speculative_split_tokens(4, 4, 32770, 4 * 32770, 0) == 2112
    assert L.wc_speculative_split_tokens(4, 4, 32770, 0, 0) == 2112
    for batch, n_kv, s in ((4, 4, 32769), (1, 4, 131072), (8, 4, 4096), (64, 4, 32768), (1, 1, 10)):
        st, sp = L.wc_decode_split_tokens(batch, n_kv, s, 0, 0), L.wc_speculative_split_tokens(batch, n_kv, s, 0, 0)
        assert sp >= 256 and sp % 64 == 0 and st <= sp <= 2 * st + 64, (batch, n_kv, s, st, sp)
    assert L.wc_speculative_split_tokens(4, 4, 32769, 0, 100) == 128
    assert L.wc_speculative_split_tokens(4, 0, 100, 0, 0) == 0
    assert L.wc_speculative_split_tokens(-1, 4, 100, 0, 0) == 0


def test_group_scale_and_repair_argument_checks(L):
    # group scales: a flag of 0 or 1, INT8 only
    c = _lib.WcCache(0, 128, 1, 8, 0, 0, 1, 0, 16, 16, 16, 16, 16, 0, 2, None, None, None, None)
    assert L.wc_quantize_write(ctypes.byref(c), 16, 16, 0, 16, 1, None) == _lib.WC_EINVAL
    c.group_scales, c.kind = 1, _lib.WC_KIND_FP8_RAW
    assert L.wc_quantize_write(ctypes.byref(c), 16, 16, 0, 16, 1, None) == _lib.WC_EINVAL
    c.kind = _lib.WC_KIND_INT8_DITHER
    assert L.wc_quantize_write(ctypes.byref(c), 16, 16, 0, 16, 0, None) == _lib.WC_OK   # no tokens
    # repair workspace: a 1 KB header and one record of G (d + 2) doubles per
    # (candidate block, 64-token tile) for every (sequence, KV head); blocks are
    # fixed 256-token runs, so four tiles each
    unit = 1024 + 64 * 4 * 7 * 130 * 8
    assert L.wc_block_repair_workspace_size(4, 28, 4, 128, 64) == 16 * ((unit + 255) // 256 * 256)
    assert L.wc_block_repair_workspace_size(4, 28, 4, 128, 65) == 0
    assert L.wc_block_repair_workspace_size(4, 27, 4, 128, 8) == 0
    ex = _lib.WcCache(_lib.WC_KIND_BF16, 128, 1, 0, 0, 0, 1, 0, 16, 16)
    c.group_scales = 0

    def rep(max_rep, rws, rws_bytes):
        return L.wc_block_repair(ctypes.byref(c), ctypes.byref(ex), 16, 1, 1, 7, 16, 4, 16, 64, 0.1, 0, 0.0,
                                 0.2, max_rep, 16, 1 << 30, 16, 0, 16, 16, 16, None, None, rws, rws_bytes, None)
    assert rep(65, 256, 1 << 30) == _lib.WC_EINVAL            # budget above 64 blocks
    assert rep(8, None, 1 << 30) == _lib.WC_EINVAL            # no repair workspace
    assert rep(8, 16, 1 << 30) == _lib.WC_EINVAL              # not 256-byte aligned
    assert rep(8, 256, 64) == _lib.WC_EWORKSPACE              # too small


def test_step_call_argument_checks(L):
    """wc_step_metered_decode_gate checks the write's and the decode's arguments on
    the host before anything is launched."""
    c = _lib.WcCache(_lib.WC_KIND_INT8_DITHER, 128, 1, 8, 0, 0, 1, 0, 16, 16, 16, 16, 16, 0, 0,
                     None, None, None, None)
    ex = _lib.WcCache(_lib.WC_KIND_BF16, 128, 1, 0, 0, 0, 1, 0, 16, 16)

    def step(cache, exact, in_dtype=_lib.WC_BF16, new_k=16, ws_bytes=1 << 30, ws=256, tau=0.2):
        return L.wc_step_metered_decode_gate(
            cache, exact, new_k, 16, in_dtype, 16, 16, _lib.WC_BF16, 1, 7, 16, 4, 16, 64, 0.1, 16, 0,
            16, 16, 0, tau, 16, 16, None, ws, ws_bytes, None)
    assert step(ctypes.byref(c), None) == _lib.WC_EINVAL                       # no exact cache
    assert step(ctypes.byref(c), ctypes.byref(c)) == _lib.WC_EINVAL            # exact must be bf16
    assert step(ctypes.byref(c), ctypes.byref(ex), in_dtype=_lib.WC_F16) == _lib.WC_EINVAL
    assert step(ctypes.byref(c), ctypes.byref(ex), new_k=8) == _lib.WC_EINVAL  # misaligned input
    assert step(ctypes.byref(c), ctypes.byref(ex), tau=-1.0) == _lib.WC_EINVAL
    assert step(ctypes.byref(c), ctypes.byref(ex), ws_bytes=64) == _lib.WC_EWORKSPACE
    assert step(ctypes.byref(ex), ctypes.byref(ex)) == _lib.WC_EINVAL         # the metered cache is quantized


def test_certified_step_checks_and_workspace(L):
    """wc_step_certified_decode: workspace = the metered decode's plus one more region
    of split records; host checks before anything is launched."""
    for args in [(4, 28, 4, 128, 32768, 0), (4, 28, 4, 128, 32768, 512), (64, 28, 4, 128, 32832, 1088)]:
        b, nq, nkv, d, L_, st = args
        base = L.wc_decode_workspace_size(*args)
        split = L.wc_decode_split_tokens(b, nkv, L_, 0, st)
        ns = (L_ + split - 1) // split
        rec = (b * nq * ns * (d + 8) * 4 + 255) // 256 * 256
        assert L.wc_certified_workspace_size(*args) == base + rec
    assert L.wc_certified_workspace_size(-1, 28, 4, 128, 100, 0) == 0
    c = _lib.WcCache(_lib.WC_KIND_INT8_DITHER, 128, 1, 8, 0, 0, 1, 0, 16, 16, 16, 16, 16, 0, 0,
                     None, None, None, None)
    ex = _lib.WcCache(_lib.WC_KIND_BF16, 128, 1, 0, 0, 0, 1, 0, 16, 16)
    ex64 = _lib.WcCache(_lib.WC_KIND_BF16, 64, 1, 0, 0, 0, 1, 0, 16, 16)

    need = L.wc_certified_workspace_size(1, 7, 1, 128, 64, 0)
    # (the speculative form takes the same arguments and checks)
    for fn in (L.wc_step_certified_decode, L.wc_step_certified_decode_speculative):
        def step(cache, exact, ws_bytes=1 << 30, tau=0.2, meter=16):
            return fn(cache, exact, 16, 16, _lib.WC_BF16, 16, 16, _lib.WC_BF16, 1, 7, 16, 4, 16, 64, 0.1, 16, 0,
                      meter, 16, 0, tau, 16, 16, None, 256, ws_bytes, None)
        assert step(ctypes.byref(c), None) == _lib.WC_EINVAL                   # no exact cache
        assert step(ctypes.byref(c), ctypes.byref(c)) == _lib.WC_EINVAL        # exact must be bf16
        assert step(ctypes.byref(c), ctypes.byref(ex64)) == _lib.WC_EINVAL     # same head size
        assert step(ctypes.byref(ex), ctypes.byref(ex)) == _lib.WC_EINVAL      # the metered cache is quantized
        assert step(ctypes.byref(c), ctypes.byref(ex), tau=-1.0) == _lib.WC_EINVAL
        assert step(ctypes.byref(c), ctypes.byref(ex), meter=None) == _lib.WC_EINVAL
        assert step(ctypes.byref(c), ctypes.byref(ex), ws_bytes=need - 1) == _lib.WC_EWORKSPACE


def test_noalloc_step_call_checks(L):
    """wc_step_metered_decode_gate_noalloc refuses sizes beyond its static scratch
    before touching any device, and a missing cache."""
    c = _lib.WcCache(_lib.WC_KIND_INT8_DITHER, 128, 4, 8, 0, 0, 1 << 20, 0, 16, 16, 16, 16, 16, 0, 0,
                     None, None, None, None)
    ex = _lib.WcCache(_lib.WC_KIND_BF16, 128, 4, 0, 0, 0, 1 << 20, 0, 16, 16)

    def step(cache, batch, max_len, split=0):
        return L.wc_step_metered_decode_gate_noalloc(
            cache, ctypes.byref(ex), 16, 16, _lib.WC_BF16, 16, 16, _lib.WC_BF16, batch, 28, 16,
            (max_len + 15) // 16, 16, max_len, 0.1, 16, _lib.WC_BF16, 16, 16, split, 0.2, 16, 16, None, None)
    need = L.wc_decode_workspace_size(512, 28, 4, 128, 1 << 17, 256)
    assert need > _lib.WC_NOALLOC_SCRATCH_BYTES
    assert step(ctypes.byref(c), 512, 1 << 17, 256) == _lib.WC_ESCRATCH
    assert step(None, 4, 32768) == _lib.WC_EINVAL
    assert L.wc_strerror(_lib.WC_ESCRATCH).startswith(b"sizes exceed the static scratch")
    # the workloads' sizes fit: 4 x 32k and the 64-sequence serving mix's balanced split
    assert L.wc_decode_workspace_size(4, 28, 4, 128, 32768 + 64, 0) <= _lib.WC_NOALLOC_SCRATCH_BYTES
    st = L.wc_decode_split_tokens(64, 4, 32768 + 64, 64 * 7756, 0)
    assert L.wc_decode_workspace_size(64, 28, 4, 128, 32768 + 64, st) <= _lib.WC_NOALLOC_SCRATCH_BYTES


def test_tierb_delta_loc(L):
    """The request-level budget split over layers x query heads x steps (Sec. 4.2)."""
    assert L.wc_tierb_delta_loc(1e-2, 28, 28, 256) == pytest.approx(1e-2 / (28 * 28 * 256), rel=1e-15)
    assert L.wc_tierb_delta_loc(0.5, 1, 1, 1) == 0.5
    for bad in ((0.0, 1, 1, 1), (1.0, 1, 1, 1), (1e-2, 0, 1, 1), (1e-2, 1, 0, 1), (1e-2, 1, 1, 0)):
        assert L.wc_tierb_delta_loc(*bad) == -1.0
