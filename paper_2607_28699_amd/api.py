"""Thin Python binding of libwitcert: argument marshalling only.

PyTorch is used for device memory and the current HIP stream; every step of the
hot path runs in the library's kernels.  Function names follow the C-ABI
(``wc_quantize_write`` -> ``quantize_write`` and so on).
"""
from __future__ import annotations

import ctypes
from dataclasses import dataclass, field

import torch

from . import _lib
from ._lib import (WC_BF16, WC_BLOCK_TOKENS, WC_F16, WC_F32, WC_KIND_BF16, WC_KIND_FP8_RAW,
                   WC_KIND_INT8_DITHER, WC_ROPE_HALF, WC_ROPE_INTERLEAVED, WcCache, check, lib)

KINDS = {"int8_dither": WC_KIND_INT8_DITHER, "fp8_raw": WC_KIND_FP8_RAW, "bf16": WC_KIND_BF16}
LAYOUTS = {"half": WC_ROPE_HALF, "interleaved": WC_ROPE_INTERLEAVED}
_DT = {torch.float32: WC_F32, torch.bfloat16: WC_BF16, torch.float16: WC_F16}


def _ptr(t: torch.Tensor | None) -> int | None:
    return None if t is None else t.data_ptr()


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _dt(t: torch.Tensor) -> int:
    try:
        return _DT[t.dtype]
    except KeyError:
        raise _lib.WitCertError(f"unsupported dtype {t.dtype}") from None


def _dev_check(*ts):
    for t in ts:
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise _lib.WitCertError("tensors must be contiguous device tensors")


def cache_bytes(kind: str, num_blocks: int, n_kv: int, head_dim: int, n_bands: int,
                n_outlier_pairs: int = 0, value_side: bool = False, group_scales: bool = False):
    sizes = (ctypes.c_size_t * 8)()
    total = lib().wc_cache_bytes(KINDS[kind], num_blocks, n_kv, head_dim, n_bands, n_outlier_pairs,
                                 int(value_side), int(group_scales), sizes)
    if total == 0:
        raise _lib.WitCertError("bad cache geometry")
    return total, list(sizes)


@dataclass
class PagedCache:
    """One layer's paged cache in device memory (layout: include/witcert.h); with
    host=True in pinned host memory, which the kernels read over the host link
    (an exact store kept off the GPU, as the paper's CPU copy)."""
    kind: str
    num_blocks: int
    n_kv: int
    head_dim: int
    n_bands: int
    layer: int = 0
    seed: int = 0
    rope_layout: str = "half"
    device: str = "cuda"
    n_outlier_pairs: int = 0
    value_side: bool = False
    group_scales: bool = False
    tensors: dict = field(default_factory=dict)
    exact_store: object = None   # persistent repair: the bf16 PagedCache of marked pages
    host: bool = False            # pinned host memory instead of device memory

    def __post_init__(self):
        m = self.n_outlier_pairs
        total, sizes = cache_bytes(self.kind, self.num_blocks, self.n_kv, self.head_dim, self.n_bands, m,
                                   self.value_side, self.group_scales)
        names = ("k_data", "v_data", "k_scale", "v_scale", "k_witness", "k_outlier", "v_resid", "v_norm")
        slots = self.num_blocks * WC_BLOCK_TOKENS * self.n_kv
        # pages of 16-byte pieces [CL][4][16][16 bytes], CL = head_dim * E / 64 (E bytes per element)
        esz = 2 if self.kind == "bf16" else 1
        piece_shape = (self.num_blocks, self.n_kv, self.head_dim * esz // 64, 4, WC_BLOCK_TOKENS, 16 // esz)
        shapes = {
            "k_data": piece_shape,
            "v_data": piece_shape,
            # one fp16 scale per token, or per 32-channel group (Table 4)
            "k_scale": (self.num_blocks, self.n_kv, WC_BLOCK_TOKENS) + ((self.head_dim // 32,)
                                                                        if self.group_scales else ()),
            "v_scale": (self.num_blocks, self.n_kv, WC_BLOCK_TOKENS) + ((self.head_dim // 32,)
                                                                        if self.group_scales else ()),
            "k_witness": (self.num_blocks, self.n_kv, WC_BLOCK_TOKENS, self.n_bands),
            "k_outlier": (self.num_blocks, self.n_kv, WC_BLOCK_TOKENS, 2 * m),
            "v_resid": (self.num_blocks, self.n_kv, WC_BLOCK_TOKENS),
            "v_norm": (self.num_blocks, self.n_kv, WC_BLOCK_TOKENS),
        }
        # int8 codes are stored excess-128 (byte = code + 128)
        el = {"int8_dither": torch.uint8, "fp8_raw": torch.uint8, "bf16": torch.bfloat16}[self.kind]
        for n, s in zip(names, sizes):
            if s == 0:
                self.tensors[n] = None
                continue
            dt = el if n in ("k_data", "v_data") else torch.uint16
            if self.host:
                t = torch.empty(shapes[n], dtype=dt, pin_memory=True)
                t.zero_()
            else:
                t = torch.zeros(shapes[n], dtype=dt, device=self.device)
            assert t.numel() * t.element_size() == s, (n, s, slots)
            self.tensors[n] = t
        self.total_bytes = total
        # bypassed RoPE pairs per KV head (set with set_outlier_pairs before writing)
        self.tensors["outlier_pairs"] = (
            torch.arange(m, dtype=torch.int32, device=self.device).repeat(self.n_kv, 1) if m else None)

    def host_copy(self) -> "PagedCache":
        """The same cache, contents included, in pinned host memory."""
        c = PagedCache(self.kind, self.num_blocks, self.n_kv, self.head_dim, self.n_bands, self.layer, self.seed,
                       self.rope_layout, self.device, self.n_outlier_pairs, self.value_side, self.group_scales,
                       host=True)
        for n, t in self.tensors.items():
            if t is not None and n != "outlier_pairs":
                c.tensors[n].copy_(t)
        if self.tensors.get("outlier_pairs") is not None:
            c.tensors["outlier_pairs"].copy_(self.tensors["outlier_pairs"])
        return c

    def set_outlier_pairs(self, pairs: torch.Tensor) -> None:
        """pairs [n_kv, m] int32, ascending per row (e.g. from select_outlier_pairs)."""
        t = self.tensors["outlier_pairs"]
        if t is None or tuple(pairs.shape) != tuple(t.shape):
            raise _lib.WitCertError("outlier pairs do not match the cache")
        t.copy_(pairs.to(device=t.device, dtype=torch.int32))

    def enable_repair(self, exact: "PagedCache") -> None:
        """Persistent repair: repair marks (one byte per page and KV head, all 0) and
        `exact` (the bf16 cache written by quantize_write_pair) as the exact store of
        marked pages."""
        if exact.kind != "bf16" or (exact.n_kv, exact.head_dim) != (self.n_kv, self.head_dim) or \
                exact.num_blocks < self.num_blocks:
            raise _lib.WitCertError("the exact store does not match the cache")
        self.tensors["repaired"] = torch.zeros((self.num_blocks, self.n_kv), dtype=torch.uint8,
                                               device=self.device)
        self.exact_store = exact

    def struct(self) -> WcCache:
        t = self.tensors
        ex = self.exact_store
        return WcCache(KINDS[self.kind], self.head_dim, self.n_kv, self.n_bands,
                       LAYOUTS[self.rope_layout], self.layer, self.num_blocks, self.seed,
                       _ptr(t["k_data"]), _ptr(t["v_data"]), _ptr(t["k_scale"]),
                       _ptr(t["v_scale"]), _ptr(t["k_witness"]), self.n_outlier_pairs,
                       1 if self.group_scales else 0, _ptr(t["outlier_pairs"]), _ptr(t["k_outlier"]),
                       _ptr(t["v_resid"]), _ptr(t["v_norm"]), _ptr(t.get("repaired")),
                       _ptr(ex.tensors["k_data"]) if ex is not None else None,
                       _ptr(ex.tensors["v_data"]) if ex is not None else None)


def quantize_write(cache: PagedCache, k: torch.Tensor, v: torch.Tensor, slots: torch.Tensor) -> None:
    """k, v [n_tok, n_kv, d] (fp32/bf16, post-RoPE keys); slots [n_tok] int64."""
    _dev_check(k, v, slots)
    assert slots.dtype == torch.int64 and k.shape == v.shape and k.dtype == v.dtype
    c = cache.struct()
    check(lib().wc_quantize_write(ctypes.byref(c), _ptr(k), _ptr(v), _dt(k), _ptr(slots),
                                  k.shape[0], _stream()), "wc_quantize_write")


def quantize_write_pair(cache: PagedCache, exact: PagedCache, k: torch.Tensor, v: torch.Tensor,
                        slots: torch.Tensor) -> None:
    """quantize_write into `cache` and a bf16 copy into `exact`, in one pass."""
    _dev_check(k, v, slots)
    assert slots.dtype == torch.int64 and k.shape == v.shape and k.dtype == v.dtype
    c, e = cache.struct(), exact.struct()
    check(lib().wc_quantize_write_pair(ctypes.byref(c), ctypes.byref(e), _ptr(k), _ptr(v), _dt(k),
                                       _ptr(slots), k.shape[0], _stream()), "wc_quantize_write_pair")


def select_outlier_pairs(k: torch.Tensor, m: int, rope_layout: str = "half",
                         out: torch.Tensor | None = None, ws: torch.Tensor | None = None) -> torch.Tensor:
    """The m RoPE pairs of largest energy of each KV head over the rows of
    k [n_tok, n_kv, d] -> int32 [n_kv, m], ascending."""
    _dev_check(k)
    n_tok, n_kv, d = k.shape
    if out is None:
        out = torch.empty((n_kv, m), dtype=torch.int32, device=k.device)
    if ws is None:
        n = lib().wc_select_workspace_size(n_tok, n_kv, d)
        ws = torch.empty(max(n, 8), dtype=torch.uint8, device=k.device)
    check(lib().wc_select_outlier_pairs(_ptr(k), _dt(k), n_tok, n_kv, d, LAYOUTS[rope_layout], m,
                                        _ptr(out), _ptr(ws), ws.numel(), _stream()),
          "wc_select_outlier_pairs")
    return out


def witness(x: torch.Tensor, xhat: torch.Tensor, n_bands: int, rope_layout: str = "half",
            out: torch.Tensor | None = None) -> torch.Tensor:
    """Band norms of xhat - x rounded up to fp16: [n_vec, n_bands] float16."""
    _dev_check(x, xhat)
    d = x.shape[-1]
    n = x.numel() // d
    if out is None:
        out = torch.empty((n, n_bands), dtype=torch.float16, device=x.device)
    check(lib().wc_witness(_ptr(x), _dt(x), _ptr(xhat), _dt(xhat), n, d, n_bands,
                           LAYOUTS[rope_layout], _ptr(out), _stream()), "wc_witness")
    return out


def decode_workspace(batch: int, n_q: int, n_kv: int, head_dim: int, max_seq_len: int,
                     split_tokens: int = 0, device="cuda") -> torch.Tensor:
    n = lib().wc_decode_workspace_size(batch, n_q, n_kv, head_dim, max_seq_len, split_tokens)
    if n == 0:
        raise _lib.WitCertError("bad workspace geometry")
    return torch.empty(n, dtype=torch.uint8, device=device)


def split_tokens_for(batch: int, n_kv: int, max_seq_len: int, split_tokens: int = 0,
                     total_tokens: int = 0) -> int:
    """Tokens per KV split of the decode calls (block repair's blocks are quarters);
    with total_tokens (the sum of the sequence lengths) balanced over the batch."""
    n = lib().wc_decode_split_tokens(batch, n_kv, max_seq_len, total_tokens, split_tokens)
    if n <= 0:
        raise _lib.WitCertError("bad split geometry")
    return n


def speculative_split_tokens(batch: int, n_kv: int, max_seq_len: int, split_tokens: int = 0,
                             total_tokens: int = 0) -> int:
    """Tokens per KV split for step_certified_decode_speculative: about half the
    decode calls' workgroups per split set, since its one launch holds both decodes'."""
    n = lib().wc_speculative_split_tokens(batch, n_kv, max_seq_len, total_tokens, split_tokens)
    if n <= 0:
        raise _lib.WitCertError("bad split geometry")
    return n


def metered_decode_attention(cache: PagedCache, q: torch.Tensor, block_table: torch.Tensor,
                             seq_lens: torch.Tensor, max_seq_len: int, sm_scale: float,
                             out_dtype=torch.float32, split_tokens: int = 0,
                             ws: torch.Tensor | None = None, out=None, meter=None, raw=None):
    """q [batch, n_q, d] -> (out [batch, n_q, d], meter [batch, n_q], raw [batch, n_q])."""
    _dev_check(q, block_table, seq_lens)
    batch, n_q, d = q.shape
    if ws is None:
        ws = decode_workspace(batch, n_q, cache.n_kv, d, max_seq_len, split_tokens, q.device)
    out = torch.empty((batch, n_q, d), dtype=out_dtype, device=q.device) if out is None else out
    meter = torch.empty((batch, n_q), dtype=torch.float32, device=q.device) if meter is None else meter
    raw = torch.empty((batch, n_q), dtype=torch.float32, device=q.device) if raw is None else raw
    c = cache.struct()
    check(lib().wc_metered_decode_attention(
        ctypes.byref(c), _ptr(q), _dt(q), batch, n_q, _ptr(block_table), block_table.shape[1],
        _ptr(seq_lens), max_seq_len, float(sm_scale), _ptr(out), _dt(out), _ptr(meter), _ptr(raw),
        split_tokens, _ptr(ws), ws.numel(), _stream()), "wc_metered_decode_attention")
    return out, meter, raw


def tierb_delta_loc(delta_req: float, n_layers: int, n_q_heads: int, n_steps: int) -> float:
    """Per-(layer, head, step) failure budget of Tier B (wc_tierb_delta_loc)."""
    d = lib().wc_tierb_delta_loc(float(delta_req), int(n_layers), int(n_q_heads), int(n_steps))
    if d <= 0.0:
        raise _lib.WitCertError("wc_tierb_delta_loc: invalid arguments")
    return float(d)


def tierb_decode_attention(cache: PagedCache, q: torch.Tensor, block_table: torch.Tensor,
                           seq_lens: torch.Tensor, max_seq_len: int, sm_scale: float, delta_loc: float,
                           out_dtype=torch.float32, split_tokens: int = 0, ws=None, out=None, meter=None,
                           raw=None):
    """Tier-B certified decode over an int8_dither cache -> (out, meter, raw)."""
    _dev_check(q, block_table, seq_lens)
    batch, n_q, d = q.shape
    if ws is None:
        ws = decode_workspace(batch, n_q, cache.n_kv, d, max_seq_len, split_tokens, q.device)
    out = torch.empty((batch, n_q, d), dtype=out_dtype, device=q.device) if out is None else out
    meter = torch.empty((batch, n_q), dtype=torch.float32, device=q.device) if meter is None else meter
    raw = torch.empty((batch, n_q), dtype=torch.float32, device=q.device) if raw is None else raw
    c = cache.struct()
    check(lib().wc_tierb_decode_attention(
        ctypes.byref(c), _ptr(q), _dt(q), batch, n_q, _ptr(block_table), block_table.shape[1],
        _ptr(seq_lens), max_seq_len, float(sm_scale), _ptr(out), _dt(out), _ptr(meter), _ptr(raw),
        split_tokens, float(delta_loc), _ptr(ws), ws.numel(), _stream()), "wc_tierb_decode_attention")
    return out, meter, raw


def metered_decode_gate(cache: PagedCache, q: torch.Tensor, block_table: torch.Tensor,
                        seq_lens: torch.Tensor, max_seq_len: int, sm_scale: float, tau: float,
                        out_dtype=torch.float32, split_tokens: int = 0, ws=None, out=None, meter=None,
                        raw=None, mask_q=None, mask_kv=None, n_gated=None):
    """metered_decode_attention then gate, fused: -> (out, meter, raw, mask_q, mask_kv)."""
    _dev_check(q, block_table, seq_lens)
    batch, n_q, d = q.shape
    if ws is None:
        ws = decode_workspace(batch, n_q, cache.n_kv, d, max_seq_len, split_tokens, q.device)
    out = torch.empty((batch, n_q, d), dtype=out_dtype, device=q.device) if out is None else out
    meter = torch.empty((batch, n_q), dtype=torch.float32, device=q.device) if meter is None else meter
    raw = torch.empty((batch, n_q), dtype=torch.float32, device=q.device) if raw is None else raw
    mask_q = torch.empty((batch, n_q), dtype=torch.uint8, device=q.device) if mask_q is None else mask_q
    mask_kv = (torch.empty((batch, cache.n_kv), dtype=torch.uint8, device=q.device)
               if mask_kv is None else mask_kv)
    c = cache.struct()
    check(lib().wc_metered_decode_gate(
        ctypes.byref(c), _ptr(q), _dt(q), batch, n_q, _ptr(block_table), block_table.shape[1],
        _ptr(seq_lens), max_seq_len, float(sm_scale), _ptr(out), _dt(out), _ptr(meter), _ptr(raw),
        split_tokens, float(tau), _ptr(mask_q), _ptr(mask_kv), _ptr(n_gated), _ptr(ws), ws.numel(),
        _stream()), "wc_metered_decode_gate")
    return out, meter, raw, mask_q, mask_kv


def step_metered_decode_gate(cache: PagedCache, exact: PagedCache, new_k: torch.Tensor, new_v: torch.Tensor,
                             new_slots: torch.Tensor, q: torch.Tensor, block_table: torch.Tensor,
                             seq_lens: torch.Tensor, max_seq_len: int, sm_scale: float, tau: float,
                             out_dtype=torch.float32, split_tokens: int = 0, ws=None, out=None, meter=None,
                             raw=None, mask_q=None, mask_kv=None, n_gated=None):
    """One decode step: quantize_write_pair of each sequence's new token (its last,
    new_k/new_v [batch, n_kv, d], new_slots [batch]) then metered_decode_gate, in one
    launch where the decode runs on the matrix cores -> (out, meter, raw, mask_q, mask_kv)."""
    _dev_check(q, block_table, seq_lens, new_k, new_v, new_slots)
    batch, n_q, d = q.shape
    assert new_slots.dtype == torch.int64 and new_k.shape == new_v.shape == (batch, cache.n_kv, d)
    assert new_k.dtype == new_v.dtype
    if ws is None:
        ws = decode_workspace(batch, n_q, cache.n_kv, d, max_seq_len, split_tokens, q.device)
    out = torch.empty((batch, n_q, d), dtype=out_dtype, device=q.device) if out is None else out
    meter = torch.empty((batch, n_q), dtype=torch.float32, device=q.device) if meter is None else meter
    raw = torch.empty((batch, n_q), dtype=torch.float32, device=q.device) if raw is None else raw
    mask_q = torch.empty((batch, n_q), dtype=torch.uint8, device=q.device) if mask_q is None else mask_q
    mask_kv = (torch.empty((batch, cache.n_kv), dtype=torch.uint8, device=q.device)
               if mask_kv is None else mask_kv)
    c, e = cache.struct(), exact.struct()
    check(lib().wc_step_metered_decode_gate(
        ctypes.byref(c), ctypes.byref(e), _ptr(new_k), _ptr(new_v), _dt(new_k), _ptr(new_slots), _ptr(q),
        _dt(q), batch, n_q, _ptr(block_table), block_table.shape[1], _ptr(seq_lens), max_seq_len,
        float(sm_scale), _ptr(out), _dt(out), _ptr(meter), _ptr(raw), split_tokens, float(tau),
        _ptr(mask_q), _ptr(mask_kv), _ptr(n_gated), _ptr(ws), ws.numel(), _stream()),
        "wc_step_metered_decode_gate")
    return out, meter, raw, mask_q, mask_kv


def certified_workspace(batch: int, n_q: int, n_kv: int, head_dim: int, max_seq_len: int,
                        split_tokens: int = 0, device="cuda") -> torch.Tensor:
    """Workspace of step_certified_decode (two regions of split records)."""
    n = lib().wc_certified_workspace_size(batch, n_q, n_kv, head_dim, max_seq_len, split_tokens)
    if n == 0:
        raise _lib.WitCertError("bad workspace geometry")
    return torch.empty(n, dtype=torch.uint8, device=device)


def _certified(fn_name, cache, exact, new_k, new_v, new_slots, q, block_table, seq_lens, max_seq_len, sm_scale,
               tau, out_dtype, split_tokens, ws, out, meter, raw, mask_q, mask_kv, n_gated):
    _dev_check(q, block_table, seq_lens, new_k, new_v, new_slots)
    batch, n_q, d = q.shape
    assert new_slots.dtype == torch.int64 and new_k.shape == new_v.shape == (batch, cache.n_kv, d)
    assert new_k.dtype == new_v.dtype
    if ws is None:
        ws = certified_workspace(batch, n_q, cache.n_kv, d, max_seq_len, split_tokens, q.device)
    out = torch.empty((batch, n_q, d), dtype=out_dtype, device=q.device) if out is None else out
    meter = torch.empty((batch, n_q), dtype=torch.float32, device=q.device) if meter is None else meter
    raw = torch.empty((batch, n_q), dtype=torch.float32, device=q.device) if raw is None else raw
    mask_q = torch.empty((batch, n_q), dtype=torch.uint8, device=q.device) if mask_q is None else mask_q
    mask_kv = (torch.empty((batch, cache.n_kv), dtype=torch.uint8, device=q.device)
               if mask_kv is None else mask_kv)
    c, e = cache.struct(), exact.struct()
    check(getattr(lib(), fn_name)(
        ctypes.byref(c), ctypes.byref(e), _ptr(new_k), _ptr(new_v), _dt(new_k), _ptr(new_slots), _ptr(q),
        _dt(q), batch, n_q, _ptr(block_table), block_table.shape[1], _ptr(seq_lens), max_seq_len,
        float(sm_scale), _ptr(out), _dt(out), _ptr(meter), _ptr(raw), split_tokens, float(tau),
        _ptr(mask_q), _ptr(mask_kv), _ptr(n_gated), _ptr(ws), ws.numel(), _stream()), fn_name)
    return out, meter, raw, mask_q, mask_kv


def step_certified_decode(cache: PagedCache, exact: PagedCache, new_k: torch.Tensor, new_v: torch.Tensor,
                          new_slots: torch.Tensor, q: torch.Tensor, block_table: torch.Tensor,
                          seq_lens: torch.Tensor, max_seq_len: int, sm_scale: float, tau: float,
                          out_dtype=torch.float32, split_tokens: int = 0, ws=None, out=None, meter=None,
                          raw=None, mask_q=None, mask_kv=None, n_gated=None):
    """One whole decode step: step_metered_decode_gate, then exact_decode_attention
    of the routed KV heads, in three launches (the gate decided in the exact
    fallback's prologue) -> (out, meter, raw, mask_q, mask_kv)."""
    return _certified("wc_step_certified_decode", cache, exact, new_k, new_v, new_slots, q, block_table, seq_lens,
                      max_seq_len, sm_scale, tau, out_dtype, split_tokens, ws, out, meter, raw, mask_q, mask_kv,
                      n_gated)


def step_certified_decode_speculative(cache: PagedCache, exact: PagedCache, new_k: torch.Tensor,
                                      new_v: torch.Tensor, new_slots: torch.Tensor, q: torch.Tensor,
                                      block_table: torch.Tensor, seq_lens: torch.Tensor, max_seq_len: int,
                                      sm_scale: float, tau: float, out_dtype=torch.float32, split_tokens: int = 0,
                                      ws=None, out=None, meter=None, raw=None, mask_q=None, mask_kv=None,
                                      n_gated=None):
    """step_certified_decode with the exact fallback of every KV head beside the
    metered decode (one launch where the kernels allow it) and the gate decided in
    the final merge: the same results, for steps where most KV heads are routed."""
    return _certified("wc_step_certified_decode_speculative", cache, exact, new_k, new_v, new_slots, q,
                      block_table, seq_lens, max_seq_len, sm_scale, tau, out_dtype, split_tokens, ws, out, meter,
                      raw, mask_q, mask_kv, n_gated)


def step_metered_decode_gate_noalloc(cache: PagedCache, exact: PagedCache, new_k: torch.Tensor,
                                     new_v: torch.Tensor, new_slots: torch.Tensor, q: torch.Tensor,
                                     block_table: torch.Tensor, seq_lens: torch.Tensor, max_seq_len: int,
                                     sm_scale: float, tau: float, out, meter, raw, mask_q, mask_kv,
                                     split_tokens: int = 0, n_gated=None):
    """step_metered_decode_gate for callers that cannot allocate: no workspace (the
    library's static per-GPU scratch holds the split records); every output is the
    caller's."""
    _dev_check(q, block_table, seq_lens, new_k, new_v, new_slots)
    batch, n_q, d = q.shape
    assert new_slots.dtype == torch.int64 and new_k.shape == new_v.shape == (batch, cache.n_kv, d)
    assert new_k.dtype == new_v.dtype
    c, e = cache.struct(), exact.struct()
    check(lib().wc_step_metered_decode_gate_noalloc(
        ctypes.byref(c), ctypes.byref(e), _ptr(new_k), _ptr(new_v), _dt(new_k), _ptr(new_slots), _ptr(q),
        _dt(q), batch, n_q, _ptr(block_table), block_table.shape[1], _ptr(seq_lens), max_seq_len,
        float(sm_scale), _ptr(out), _dt(out), _ptr(meter), _ptr(raw), split_tokens, float(tau),
        _ptr(mask_q), _ptr(mask_kv), _ptr(n_gated), _stream()),
        "wc_step_metered_decode_gate_noalloc")
    return out, meter, raw, mask_q, mask_kv


def joint_decode_gate(cache: PagedCache, q: torch.Tensor, block_table: torch.Tensor,
                      seq_lens: torch.Tensor, max_seq_len: int, sm_scale: float, tau: float = 0.2,
                      tau_v: float = 0.05, delta_loc: float = 0.0, out_dtype=torch.float32,
                      split_tokens: int = 0, ws=None, out=None, meter=None, raw=None, meter_v=None,
                      mask_q=None, mask_kv=None, n_gated=None):
    """Key meter (Tier A, or Tier B when delta_loc > 0), value meter and the joint
    gate -> (out, meter, raw, meter_v, mask_q, mask_kv)."""
    _dev_check(q, block_table, seq_lens)
    batch, n_q, d = q.shape
    dev = q.device
    if ws is None:
        ws = decode_workspace(batch, n_q, cache.n_kv, d, max_seq_len, split_tokens, dev)
    out = torch.empty((batch, n_q, d), dtype=out_dtype, device=dev) if out is None else out
    meter = torch.empty((batch, n_q), dtype=torch.float32, device=dev) if meter is None else meter
    raw = torch.empty((batch, n_q), dtype=torch.float32, device=dev) if raw is None else raw
    meter_v = torch.empty((batch, n_q), dtype=torch.float32, device=dev) if meter_v is None else meter_v
    mask_q = torch.empty((batch, n_q), dtype=torch.uint8, device=dev) if mask_q is None else mask_q
    mask_kv = torch.empty((batch, cache.n_kv), dtype=torch.uint8, device=dev) if mask_kv is None else mask_kv
    c = cache.struct()
    check(lib().wc_joint_decode_gate(
        ctypes.byref(c), _ptr(q), _dt(q), batch, n_q, _ptr(block_table), block_table.shape[1],
        _ptr(seq_lens), max_seq_len, float(sm_scale), _ptr(out), _dt(out), _ptr(meter), _ptr(raw),
        _ptr(meter_v), split_tokens, float(delta_loc), float(tau), float(tau_v), _ptr(mask_q),
        _ptr(mask_kv), _ptr(n_gated), _ptr(ws), ws.numel(), _stream()), "wc_joint_decode_gate")
    return out, meter, raw, meter_v, mask_q, mask_kv


def block_repair(cache: PagedCache, exact: PagedCache, q: torch.Tensor, block_table: torch.Tensor,
                 seq_lens: torch.Tensor, max_seq_len: int, sm_scale: float, tau: float, ws: torch.Tensor,
                 out: torch.Tensor, meter: torch.Tensor, raw: torch.Tensor, mask_kv: torch.Tensor,
                 delta_loc: float = 0.0, max_blocks: int = 16, split_tokens: int = 0,
                 repaired: torch.Tensor | None = None, n_repaired: torch.Tensor | None = None,
                 repair_ws: torch.Tensor | None = None):
    """Block repair (fixed 256-token blocks) of the KV heads a metered decode (same ws,
    split_tokens) routed:
    updates out, meter, raw and mask_kv in place -> (n_repaired [batch, n_kv],
    repaired [batch, n_kv, max_blocks])."""
    _dev_check(q, block_table, seq_lens, ws, out, meter, raw, mask_kv)
    batch, n_q, d = q.shape
    if repair_ws is None:
        repair_ws = repair_workspace(batch, n_q, cache.n_kv, d, max_blocks, device=q.device)
    if n_repaired is None:
        n_repaired = torch.empty((batch, cache.n_kv), dtype=torch.int32, device=q.device)
    if repaired is None:
        repaired = torch.empty((batch, cache.n_kv, max_blocks), dtype=torch.int32, device=q.device)
    c, e = cache.struct(), exact.struct()
    check(lib().wc_block_repair(
        ctypes.byref(c), ctypes.byref(e), _ptr(q), _dt(q), batch, n_q, _ptr(block_table),
        block_table.shape[1], _ptr(seq_lens), max_seq_len, float(sm_scale), split_tokens,
        float(delta_loc), float(tau), max_blocks, _ptr(ws), ws.numel(), _ptr(out), _dt(out),
        _ptr(meter), _ptr(raw), _ptr(mask_kv), _ptr(repaired), _ptr(n_repaired), _ptr(repair_ws),
        repair_ws.numel(), _stream()),
        "wc_block_repair")
    return n_repaired, repaired


def repair_write_back(cache: PagedCache, block_table: torch.Tensor, seq_lens: torch.Tensor,
                      repaired: torch.Tensor | None = None, n_repaired: torch.Tensor | None = None,
                      whole_kv: torch.Tensor | None = None) -> None:
    """Persistent repair: mark the pages of the blocks block_repair took (repaired
    [batch, n_kv, max_blocks], n_repaired [batch, n_kv]) and of the KV heads served by
    the whole-head fallback (whole_kv [batch, n_kv] uint8), zeroing their witness."""
    _dev_check(block_table, seq_lens)
    batch = seq_lens.shape[0]
    c = cache.struct()
    mb = repaired.shape[2] if repaired is not None else 0
    check(lib().wc_repair_write_back(ctypes.byref(c), batch, _ptr(block_table), block_table.shape[1],
                                     _ptr(seq_lens), _ptr(repaired), _ptr(n_repaired), mb, _ptr(whole_kv),
                                     _stream()), "wc_repair_write_back")


def repair_workspace(batch: int, n_q: int, n_kv: int, head_dim: int, max_blocks: int = 16,
                     device="cuda") -> torch.Tensor:
    """Device workspace of block_repair for these sizes."""
    n = lib().wc_block_repair_workspace_size(batch, n_q, n_kv, head_dim, max_blocks)
    if n == 0:
        raise _lib.WitCertError("bad repair workspace geometry")
    return torch.empty(n, dtype=torch.uint8, device=device)


def gate(meter: torch.Tensor, raw: torch.Tensor, group: int, tau: float,
         n_gated: torch.Tensor | None = None, mask_q=None, mask_kv=None):
    """-> (mask_q [batch, n_q] uint8, mask_kv [batch, n_kv] uint8)."""
    _dev_check(meter, raw)
    batch, n_q = meter.shape
    mask_q = torch.empty((batch, n_q), dtype=torch.uint8, device=meter.device) if mask_q is None else mask_q
    mask_kv = (torch.empty((batch, n_q // group), dtype=torch.uint8, device=meter.device)
               if mask_kv is None else mask_kv)
    check(lib().wc_gate(_ptr(meter), _ptr(raw), batch, n_q, group, float(tau), _ptr(mask_q),
                        _ptr(mask_kv), _ptr(n_gated), _stream()), "wc_gate")
    return mask_q, mask_kv


def exact_decode_attention(cache: PagedCache, q: torch.Tensor, block_table: torch.Tensor,
                           seq_lens: torch.Tensor, max_seq_len: int, sm_scale: float,
                           mask_kv: torch.Tensor, out: torch.Tensor, split_tokens: int = 0,
                           ws: torch.Tensor | None = None) -> torch.Tensor:
    """Overwrite out[b, heads of routed KV heads] with exact attention over a bf16 cache."""
    _dev_check(q, block_table, seq_lens, mask_kv, out)
    batch, n_q, d = q.shape
    if ws is None:
        ws = decode_workspace(batch, n_q, cache.n_kv, d, max_seq_len, split_tokens, q.device)
    c = cache.struct()
    check(lib().wc_exact_decode_attention(
        ctypes.byref(c), _ptr(q), _dt(q), batch, n_q, _ptr(block_table), block_table.shape[1],
        _ptr(seq_lens), max_seq_len, float(sm_scale), _ptr(mask_kv), _ptr(out), _dt(out),
        split_tokens, _ptr(ws), ws.numel(), _stream()), "wc_exact_decode_attention")
    return out
