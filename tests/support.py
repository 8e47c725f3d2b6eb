"""Shared helpers of the GPU parity tests: seeded cases from ``synth``, the HIP
path through the binding, the oracle on the same stored inputs."""
from __future__ import annotations

import sys

import numpy as np

import synth
from oracle import decode as odec
from oracle import fpformats as ofp

BLOCK = 16


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def make_case(wl, seq_lens, permute=True, layer=0, seed_key=0):
    """Stored K/V per sequence ([S_b, n_kv, d] float32 values), q [batch, n_q, d],
    block table and slots.  q of sequence b sits at position S_b - 1."""
    seq_lens = np.asarray(seq_lens, dtype=np.int64)
    table, nblocks = synth.block_table(np.maximum(seq_lens, 1), permute, seed_key)
    ks, vs, slots = [], [], []
    for b, S in enumerate(seq_lens):
        pos = np.arange(S)
        ks.append(np.stack([synth.gen_kv(wl, layer, h, b, "k", pos) for h in range(wl.n_kv)], 1)
                  if S else np.zeros((0, wl.n_kv, wl.d), np.float32))
        vs.append(np.stack([synth.gen_kv(wl, layer, h, b, "v", pos) for h in range(wl.n_kv)], 1)
                  if S else np.zeros((0, wl.n_kv, wl.d), np.float32))
        slots.append(synth.slots_of(table, b, pos))
    q = np.stack([synth.gen_q(wl, layer, b, 0, max(int(S) - 1, 0)) for b, S in enumerate(seq_lens)])
    return dict(wl=wl, seq_lens=seq_lens, table=table, nblocks=nblocks, k=ks, v=vs, slots=slots,
                q=q, layer=layer)


def torch_dtype(wl):
    import torch
    return torch.float32 if wl.dtype == "f32" else torch.bfloat16


def case_pairs(case, m):
    """Bypassed pairs [n_kv, m] chosen by the oracle from all keys of the case."""
    from oracle import bypass as obp
    wl = case["wl"]
    k = np.concatenate(case["k"])
    return np.stack([obp.select_pairs(k[:, h], m, wl.rope_layout) for h in range(wl.n_kv)])


def gpu_cache(case, kind, seed=None, pairs=None, value_side=False, group_scales=False):
    """Write every sequence of the case into a fresh GPU cache through wc_quantize_write
    (pairs [n_kv, m]: bypassed RoPE pairs of the keys; value_side: store the value
    residual and value norms; group_scales: one fp16 scale per 32-channel group)."""
    import torch

    import paper_2607_28699_amd as wc
    wl = case["wl"]
    m = 0 if pairs is None else int(np.asarray(pairs).shape[1])
    c = wc.PagedCache(kind, case["nblocks"], wl.n_kv, wl.d, wl.bands, layer=case["layer"],
                      seed=wl.philox_seed() if seed is None else seed, rope_layout=wl.rope_layout,
                      n_outlier_pairs=m, value_side=value_side, group_scales=group_scales)
    if m:
        c.set_outlier_pairs(torch.from_numpy(np.asarray(pairs, dtype=np.int32)))
    dt = torch_dtype(wl)
    k = np.concatenate(case["k"]) if len(case["k"]) else np.zeros((0, wl.n_kv, wl.d), np.float32)
    v = np.concatenate(case["v"])
    sl = np.concatenate(case["slots"]).astype(np.int64)
    if len(sl):
        wc.quantize_write(c, torch.from_numpy(k).to("cuda", dt), torch.from_numpy(v).to("cuda", dt),
                          torch.from_numpy(sl).cuda())
    return c


def gpu_decode(case, cache, split_tokens=0, out_dtype=None):
    import torch

    import paper_2607_28699_amd as wc
    wl = case["wl"]
    q = torch.from_numpy(case["q"]).to("cuda", torch_dtype(wl))
    table = torch.from_numpy(case["table"]).cuda()
    lens = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    out, meter, raw = wc.metered_decode_attention(
        cache, q, table, lens, int(case["seq_lens"].max()), 1 / np.sqrt(wl.d),
        out_dtype=out_dtype or torch.float32, split_tokens=split_tokens)
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64), meter.cpu().numpy(), raw.cpu().numpy()


def oracle_write(case, kind, pairs=None, group_scales=False):
    wl = case["wl"]
    return [odec.write_cache(kind, k, v, s, case["layer"], wl.philox_seed(), wl.bands, wl.rope_layout,
                             pairs=pairs, group_scales=group_scales)
            for k, v, s in zip(case["k"], case["v"], case["slots"])]


def oracle_decode(case, caches):
    wl = case["wl"]
    sm = 1 / np.sqrt(wl.d)
    res = []
    for b, c in enumerate(caches):
        if case["seq_lens"][b] == 0:
            res.append(None)
            continue
        r = odec.metered_decode(case["q"][b], c["khat"], c["vhat"], c["kw"], sm, wl.bands, wl.rope_layout)
        r["tv"] = odec.true_tv(case["q"][b], case["k"][b], c["khat"], sm)
        res.append(r)
    return res


def read_cache(cache, slots):
    """Host copies of one cache's arrays gathered at the given slots:
    dict(k [n, n_kv, d], v [n, n_kv, d], ks, vs [n, n_kv], kw [n, n_kv, B])."""
    t = {n: (x.cpu() if x is not None else None) for n, x in cache.tensors.items()}
    slots = np.asarray(slots, dtype=np.int64)
    blk, off = slots // BLOCK, slots % BLOCK
    out = {}
    kd = t["k_data"].numpy() if cache.kind != "bf16" else t["k_data"].view(__import__("torch").int16).numpy()
    vd = t["v_data"].numpy() if cache.kind != "bf16" else t["v_data"].view(__import__("torch").int16).numpy()
    # pages of 16-byte pieces [CL][4][16][16 bytes] (include/witcert.h): key row bytes
    # (g*CL + i)*16 .. of token t in piece (i, g, t); value quad q's row (channel c,
    # token t%4 at element 4c + t%4) bytes (r*CL + i)*16 .. in piece (i, q, r)
    esz = 2 if cache.kind == "bf16" else 1
    d = cache.head_dim
    cl = d * esz // 64
    c = np.arange(d)
    kb = c * esz
    ki, kg, kj = (kb // 16) % cl, (kb // 16) // cl, (kb % 16) // esz
    out["k"] = kd[blk[:, None], :, ki[None, :], kg[None, :], off[:, None], kj[None, :]].transpose(0, 2, 1)
    vb = (4 * c[None, :] + (off % 4)[:, None]) * esz
    vi, vr, vj = (vb // 16) % cl, (vb // 16) // cl, (vb % 16) // esz
    out["v"] = vd[blk[:, None], :, vi, (off // 4)[:, None], vr, vj].transpose(0, 2, 1)
    if cache.kind == "int8_dither":   # stored excess-128
        out["k"] = out["k"].astype(np.int16) - 128
        out["v"] = out["v"].astype(np.int16) - 128
    if t["k_scale"] is not None:   # [n, n_kv], or with group scales [n, n_kv, d/32]
        out["ks"] = ofp_f16(t["k_scale"].numpy()[blk, :, off])
        out["vs"] = ofp_f16(t["v_scale"].numpy()[blk, :, off])
    if t["k_witness"] is not None:
        out["kw"] = ofp_f16(t["k_witness"].numpy()[blk, :, off, :])
    if t.get("k_outlier") is not None:
        out["ko"] = ofp_f16(t["k_outlier"].numpy()[blk, :, off, :])
    if t.get("v_resid") is not None:
        out["vr"] = ofp_f16(t["v_resid"].numpy()[blk, :, off])
        out["vn"] = ofp_f16(t["v_norm"].numpy()[blk, :, off])
    return out


def ofp_f16(bits):
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def next_f16_up(x):
    h = np.asarray(x, dtype=np.float64).astype(np.float16)
    with np.errstate(over="ignore"):
        return np.nextafter(h, np.float16(np.inf)).astype(np.float64)


def rel_err(got, ref):
    ref = np.asarray(ref, dtype=np.float64)
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(np.asarray(got, dtype=np.float64) - ref)) / (den if den > 0 else 1.0))


def out_tol(wl):
    """Tolerance on outputs and meter: 1e-5 relative for fp32 workloads, 2e-3 for bf16."""
    return 1e-5 if wl.dtype == "f32" else 2e-3


_ = ofp  # the oracle's format helpers are the reference for fp16 values


def bf16_bits_to_f32(bits):
    """bf16 bit patterns (any integer dtype) -> float32 values."""
    return (np.asarray(bits).astype(np.uint16).astype(np.uint32) << 16).view(np.float32)
