"""A whole decode step in one call (GPU): wc_step_certified_decode against
wc_step_metered_decode_gate followed by wc_exact_decode_attention of the KV heads
the gate routes (the meter loop of Sec. 6: write, metered read, gate, exact
fallback).

The certified call decides each KV head's gate inside the exact fallback's
workgroups, from the metered decode's split records, and forms every output row
in one final merge.  Bar: bit-identical caches, outputs, meter, raw, gate masks
and counts, with thresholds that route some, none and all KV heads, on the
matrix-core and vector paths and with fp32 inputs; a captured step replayed
several times gives the same results; and against the oracle, the routed heads
match exact attention and the others the metered decode.
"""
import os

import numpy as np
import pytest

import synth
from oracle import decode as odec

from . import support as S

pytestmark = pytest.mark.gpu

W_GQA = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]
W_TINY = synth.WORKLOADS["tiny-d64-s256"]

CASES = [
    # name, workload, lengths (0: an empty sequence), split_tokens, kind, options
    ("int8", W_GQA, [700, 1, 129], 0, "int8_dither", {}),
    ("int8-split64-empty", W_GQA, [700, 0, 64, 65], 64, "int8_dither", {}),
    ("int8-bypass-groups-value", W_GQA, [513, 17], 64, "int8_dither",
     dict(pairs=4, group_scales=True, value_side=True)),
    ("fp8", W_GQA, [300, 33], 0, "fp8_raw", {}),
    ("group16", W_GQA.replace(n_q=32, n_kv=2), [400, 16], 64, "int8_dither", {}),
    ("vector-path", W_GQA, [300, 33], 64, "int8_dither", dict(force_valu=True)),
    ("fp32-inputs", W_GQA, [300, 33], 64, "int8_dither", dict(f32_inputs=True)),
    ("tiny-d64", W_TINY, [200, 0, 57], 64, "int8_dither", {}),
    ("many-splits", W_GQA, [2100, 5, 700], 64, "int8_dither", {}),
]
TAUS = ["median", "all", "none"]


def _setup(wl, lens, kind, opts, layer=3):
    """Two identical (quantized, exact) cache pairs holding every position but each
    sequence's last, and that step's tokens."""
    import torch

    import paper_2607_28699_amd as wc
    case = S.make_case(wl, lens, permute=True, layer=layer)
    pairs = S.case_pairs(case, opts["pairs"]) if opts.get("pairs") else None
    in_dt = torch.float32 if (opts.get("f32_inputs") or wl.dtype == "f32") else torch.bfloat16
    m = 0 if pairs is None else pairs.shape[1]
    caches = []
    for _ in range(2):
        c = wc.PagedCache(kind, case["nblocks"], wl.n_kv, wl.d, wl.bands, layer=case["layer"],
                          seed=wl.philox_seed(), rope_layout=wl.rope_layout, n_outlier_pairs=m,
                          value_side=opts.get("value_side", False), group_scales=opts.get("group_scales", False))
        if m:
            c.set_outlier_pairs(torch.from_numpy(pairs.astype(np.int32)))
        e = wc.PagedCache("bf16", case["nblocks"], wl.n_kv, wl.d, 0, layer=case["layer"])
        caches.append((c, e))
    batch = len(lens)
    for b, n in enumerate(lens):
        if n > 1:
            k = torch.from_numpy(case["k"][b][:n - 1]).to("cuda", in_dt)
            v = torch.from_numpy(case["v"][b][:n - 1]).to("cuda", in_dt)
            sl = torch.from_numpy(case["slots"][b][:n - 1].astype(np.int64)).cuda()
            for c, e in caches:
                wc.quantize_write_pair(c, e, k, v, sl)
    new_k = np.zeros((batch, wl.n_kv, wl.d), np.float32)
    new_v = np.zeros((batch, wl.n_kv, wl.d), np.float32)
    new_slots = np.full(batch, -1, np.int64)
    for b, n in enumerate(lens):
        if n > 0:
            new_k[b], new_v[b], new_slots[b] = case["k"][b][-1], case["v"][b][-1], case["slots"][b][-1]
    step_in = (torch.from_numpy(new_k).to("cuda", in_dt), torch.from_numpy(new_v).to("cuda", in_dt),
               torch.from_numpy(new_slots).cuda())
    return case, caches, step_in


def _tau(name, case, caches, step_in, split):
    """Thresholds that route some (the median raw of a probe run), all or none of the heads."""
    import torch

    import paper_2607_28699_amd as wc
    if name == "all":
        return 0.0
    if name == "none":
        return 3.0e38   # raw above it only on overflow (+inf)
    wl = case["wl"]
    c, e = caches[0]
    q = torch.from_numpy(case["q"]).to("cuda", torch.float32 if wl.dtype == "f32" else torch.bfloat16)
    table = torch.from_numpy(case["table"]).cuda()
    sl = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    _, _, raw = wc.metered_decode_attention(c, q, table, sl, max(int(case["seq_lens"].max()), 1),
                                            1 / np.sqrt(wl.d), split_tokens=split)
    r = raw.cpu().numpy()
    return float(np.quantile(r[case["seq_lens"] > 0], 0.5)) if np.any(case["seq_lens"] > 0) else 0.5


@pytest.mark.parametrize("tau_mode", TAUS)
@pytest.mark.parametrize("name,wl,lens,split,kind,opts", CASES)
def test_certified_equals_step_then_fallback(name, wl, lens, split, kind, opts, tau_mode):
    import torch

    import paper_2607_28699_amd as wc
    S.say(f"[certified] {name} tau={tau_mode} lens={lens} split={split}")
    case, caches, (nk, nv, ns) = _setup(wl, lens, kind, opts)
    q = torch.from_numpy(case["q"]).to("cuda", torch.float32 if wl.dtype == "f32" else torch.bfloat16)
    table = torch.from_numpy(case["table"]).cuda()
    sl = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L = max(int(case["seq_lens"].max()), 1)
    sm = 1 / np.sqrt(wl.d)
    if opts.get("force_valu"):
        os.environ["WITCERT_FORCE_VALU"] = "1"
    try:
        (c1, e1), (c2, e2) = caches
        # (the probe for the median threshold reads caches[0] before its step write)
        tau = _tau(tau_mode, case, caches, (nk, nv, ns), split)
        n1 = torch.zeros(2, dtype=torch.int32, device="cuda")
        got = wc.step_certified_decode(c1, e1, nk, nv, ns, q, table, sl, L, sm, tau, split_tokens=split,
                                       n_gated=n1)
        n2 = torch.zeros(2, dtype=torch.int32, device="cuda")
        ws = wc.decode_workspace(q.shape[0], wl.n_q, wl.n_kv, wl.d, L, split)
        ref = wc.step_metered_decode_gate(c2, e2, nk, nv, ns, q, table, sl, L, sm, tau, split_tokens=split,
                                          n_gated=n2, ws=ws)
        wc.exact_decode_attention(e2, q, table, sl, L, sm, ref[4], ref[0], ws=ws, split_tokens=split)
        torch.cuda.synchronize()
    finally:
        os.environ.pop("WITCERT_FORCE_VALU", None)
    for (x, y) in ((c1, c2), (e1, e2)):
        for n, t in x.tensors.items():
            if t is not None:
                assert torch.equal(t, y.tensors[n]), (name, n)
    for i, (x, y) in enumerate(zip(got, ref)):
        assert torch.equal(x, y), (name, tau_mode, i)
    assert torch.equal(n1, n2), (name, n1.tolist(), n2.tolist())
    routed = got[4].cpu().numpy()
    if tau_mode == "all":
        assert np.all(routed[case["seq_lens"] > 0] == 1)
    if tau_mode == "none":
        assert not np.any(routed)


def test_certified_against_oracle():
    """Routed KV heads match exact attention over the bf16 cache, the others the
    metered decode's output (oracle), meter and raw the oracle's."""
    import torch

    import paper_2607_28699_amd as wc
    wl = W_GQA
    lens = [700, 129, 40]
    S.say(f"[certified] oracle lens={lens}")
    case, caches, (nk, nv, ns) = _setup(wl, lens, "int8_dither", {})
    q = torch.from_numpy(case["q"]).to("cuda", torch.bfloat16)
    table = torch.from_numpy(case["table"]).cuda()
    sl = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L, sm = max(lens), 1 / np.sqrt(wl.d)
    c, e = caches[0]
    tau = _tau("median", case, caches, (nk, nv, ns), 64)
    out, meter, raw, mq, mk = wc.step_certified_decode(c, e, nk, nv, ns, q, table, sl, L, sm, tau, split_tokens=64)
    torch.cuda.synchronize()
    out, meter, raw, mq, mk = (x.cpu().numpy() for x in (out, meter, raw, mq, mk))
    refs = S.oracle_write(case, "int8_dither")
    res = S.oracle_decode(case, refs)
    g = wl.n_q // wl.n_kv
    tol = S.out_tol(wl)
    assert 0 < mk.sum() < mk.size
    for b in range(len(lens)):
        ex = odec.exact_decode(case["q"][b], synth.bf16_round(case["k"][b]), synth.bf16_round(case["v"][b]), sm)["out"]
        for kv in range(wl.n_kv):
            hs = slice(kv * g, (kv + 1) * g)
            want = ex[hs] if mk[b, kv] else res[b]["out"][hs]
            assert S.rel_err(out[b, hs], want) <= tol, (b, kv, int(mk[b, kv]))
        assert np.all(np.abs(raw[b] - res[b]["raw"]) <= tol * res[b]["raw"])
        assert np.all(meter[b] >= res[b]["tv"])
        assert np.array_equal(mq[b].astype(bool), (meter[b] > tau) if tau < 1 else (raw[b] > tau))


def test_certified_graph_replay():
    import torch

    import paper_2607_28699_amd as wc
    S.say("[certified] graph replay")
    wl = W_GQA
    lens = [900, 130]
    case, caches, (nk, nv, ns) = _setup(wl, lens, "int8_dither", {}, layer=5)
    c, e = caches[0]
    q = torch.from_numpy(case["q"]).to("cuda", torch.bfloat16)
    table = torch.from_numpy(case["table"]).cuda()
    sl = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L, sm = max(lens), 1 / np.sqrt(wl.d)
    tau = _tau("median", case, caches, (nk, nv, ns), 64)
    ws = wc.certified_workspace(len(lens), wl.n_q, wl.n_kv, wl.d, L, 64)
    out = torch.empty((len(lens), wl.n_q, wl.d), dtype=torch.float32, device="cuda")
    meter = torch.empty((len(lens), wl.n_q), dtype=torch.float32, device="cuda")
    raw, mq = torch.empty_like(meter), torch.empty((len(lens), wl.n_q), dtype=torch.uint8, device="cuda")
    mk = torch.empty((len(lens), wl.n_kv), dtype=torch.uint8, device="cuda")
    cnt = torch.zeros(2, dtype=torch.int32, device="cuda")
    kw = dict(split_tokens=64, ws=ws, out=out, meter=meter, raw=raw, mask_q=mq, mask_kv=mk, n_gated=cnt)
    args = (c, e, nk, nv, ns, q, table, sl, L, sm, tau)
    wc.step_certified_decode(*args, **kw)
    torch.cuda.synchronize()
    eager = [x.clone() for x in (out, meter, raw, mq, mk, cnt)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            wc.step_certified_decode(*args, **kw)
    torch.cuda.synchronize()
    for _ in range(3):
        for x in (out, meter, raw, mq, mk):
            x.zero_()
        cnt.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for x, y in zip((out, meter, raw, mq, mk, cnt), eager):
            assert torch.equal(x, y)


@pytest.mark.parametrize("tau_mode", TAUS)
@pytest.mark.parametrize("name,wl,lens,split,kind,opts", CASES)
def test_speculative_equals_certified(name, wl, lens, split, kind, opts, tau_mode):
    """wc_step_certified_decode_speculative (the exact fallback of every KV head
    beside the metered decode, the gate decided in the final merge) gives the
    certified step's caches, outputs, meter, raw, masks and counts bit for bit: in
    one launch for the plain Tier A caches with bf16 inputs, in two otherwise."""
    import torch

    import paper_2607_28699_amd as wc
    S.say(f"[speculative] {name} tau={tau_mode} lens={lens} split={split}")
    case, caches, (nk, nv, ns) = _setup(wl, lens, kind, opts)
    q = torch.from_numpy(case["q"]).to("cuda", torch.float32 if wl.dtype == "f32" else torch.bfloat16)
    table = torch.from_numpy(case["table"]).cuda()
    sl = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L = max(int(case["seq_lens"].max()), 1)
    sm = 1 / np.sqrt(wl.d)
    if opts.get("force_valu"):
        os.environ["WITCERT_FORCE_VALU"] = "1"
    try:
        (c1, e1), (c2, e2) = caches
        tau = _tau(tau_mode, case, caches, (nk, nv, ns), split)
        n1 = torch.zeros(2, dtype=torch.int32, device="cuda")
        got = wc.step_certified_decode_speculative(c1, e1, nk, nv, ns, q, table, sl, L, sm, tau,
                                                   split_tokens=split, n_gated=n1)
        n2 = torch.zeros(2, dtype=torch.int32, device="cuda")
        ref = wc.step_certified_decode(c2, e2, nk, nv, ns, q, table, sl, L, sm, tau, split_tokens=split, n_gated=n2)
        torch.cuda.synchronize()
    finally:
        os.environ.pop("WITCERT_FORCE_VALU", None)
    for (x, y) in ((c1, c2), (e1, e2)):
        for n, t in x.tensors.items():
            if t is not None:
                assert torch.equal(t, y.tensors[n]), (name, n)
    for i, (x, y) in enumerate(zip(got, ref)):
        assert torch.equal(x, y), (name, tau_mode, i)
    assert torch.equal(n1, n2), (name, n1.tolist(), n2.tolist())


def test_speculative_graph_replay():
    import torch

    import paper_2607_28699_amd as wc
    S.say("[speculative] graph replay")
    wl = W_GQA
    lens = [900, 130, 1]
    case, caches, (nk, nv, ns) = _setup(wl, lens, "int8_dither", {}, layer=5)
    c, e = caches[0]
    q = torch.from_numpy(case["q"]).to("cuda", torch.bfloat16)
    table = torch.from_numpy(case["table"]).cuda()
    sl = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L, sm = max(lens), 1 / np.sqrt(wl.d)
    tau = _tau("median", case, caches, (nk, nv, ns), 64)
    ws = wc.certified_workspace(len(lens), wl.n_q, wl.n_kv, wl.d, L, 64)
    out = torch.empty((len(lens), wl.n_q, wl.d), dtype=torch.float32, device="cuda")
    meter = torch.empty((len(lens), wl.n_q), dtype=torch.float32, device="cuda")
    raw, mq = torch.empty_like(meter), torch.empty((len(lens), wl.n_q), dtype=torch.uint8, device="cuda")
    mk = torch.empty((len(lens), wl.n_kv), dtype=torch.uint8, device="cuda")
    cnt = torch.zeros(2, dtype=torch.int32, device="cuda")
    kw = dict(split_tokens=64, ws=ws, out=out, meter=meter, raw=raw, mask_q=mq, mask_kv=mk, n_gated=cnt)
    args = (c, e, nk, nv, ns, q, table, sl, L, sm, tau)
    wc.step_certified_decode_speculative(*args, **kw)
    torch.cuda.synchronize()
    eager = [x.clone() for x in (out, meter, raw, mq, mk, cnt)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            wc.step_certified_decode_speculative(*args, **kw)
    torch.cuda.synchronize()
    for _ in range(3):
        for x in (out, meter, raw, mq, mk):
            x.zero_()
        cnt.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for x, y in zip((out, meter, raw, mq, mk, cnt), eager):
            assert torch.equal(x, y)
