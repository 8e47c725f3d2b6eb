"""One decode step in one call (GPU): wc_step_metered_decode_gate against
wc_quantize_write_pair of the step's tokens followed by wc_metered_decode_gate.

The step's token of each sequence is its last (position seq_len - 1); a sequence
without one passes slot -1.  Bar: bit-identical caches (codes, scales, witness,
group exponents, bypassed values, value side, exact copy) and bit-identical
outputs, meter, raw, gate masks and counts, on the fused matrix-core path (one
launch) and on the paths that run the two calls back to back (vector kernels,
fp32 inputs); a captured step replayed several times gives the same results.
"""
import os

import numpy as np
import pytest

import synth

from . import support as S

pytestmark = pytest.mark.gpu

W_GQA = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]
W_TINY = synth.WORKLOADS["tiny-d64-s256"]

CASES = [
    # name, workload, lengths (0: no token this step), split_tokens, kind, options
    ("int8", W_GQA, [700, 1, 129], 0, "int8_dither", {}),
    ("int8-split64", W_GQA, [700, 0, 64, 65], 64, "int8_dither", {}),
    ("int8-bypass-groups-value", W_GQA, [513, 17], 64, "int8_dither",
     dict(pairs=4, group_scales=True, value_side=True)),
    ("fp8", W_GQA, [300, 33], 0, "fp8_raw", {}),
    ("group16", W_GQA.replace(n_q=32, n_kv=2), [400, 16], 64, "int8_dither", {}),
    ("vector-path", W_GQA, [300, 33], 64, "int8_dither", dict(force_valu=True)),
    ("fp32-inputs", W_GQA, [300, 33], 64, "int8_dither", dict(f32_inputs=True)),
    ("tiny-d64", W_TINY, [200, 0, 57], 64, "int8_dither", {}),
    # sequence 1 has context but no token this step (slot -1, its context all written)
    ("no-token-row", W_GQA, [300, 40, 90], 64, "int8_dither", dict(idle=(1,))),
]


def _caches(case, kind, opts, pairs):
    import torch

    import paper_2607_28699_amd as wc
    wl = case["wl"]
    m = 0 if pairs is None else pairs.shape[1]
    c = wc.PagedCache(kind, case["nblocks"], wl.n_kv, wl.d, wl.bands, layer=case["layer"], seed=wl.philox_seed(),
                      rope_layout=wl.rope_layout, n_outlier_pairs=m, value_side=opts.get("value_side", False),
                      group_scales=opts.get("group_scales", False))
    if m:
        c.set_outlier_pairs(torch.from_numpy(pairs.astype(np.int32)))
    e = wc.PagedCache("bf16", case["nblocks"], wl.n_kv, wl.d, 0, layer=case["layer"])
    return c, e


@pytest.mark.parametrize("name,wl,lens,split,kind,opts", CASES)
def test_step_equals_write_then_decode(name, wl, lens, split, kind, opts):
    import torch

    import paper_2607_28699_amd as wc
    S.say(f"[step] {name} lens={lens} split={split}")
    case = S.make_case(wl, lens, permute=True, layer=3)
    pairs = S.case_pairs(case, opts["pairs"]) if opts.get("pairs") else None
    in_dt = torch.float32 if (opts.get("f32_inputs") or wl.dtype == "f32") else torch.bfloat16
    q_dt = torch.float32 if wl.dtype == "f32" else torch.bfloat16
    batch = len(lens)
    # everything but each sequence's last token is already in the caches
    caches = [_caches(case, kind, opts, pairs) for _ in range(2)]
    idle = opts.get("idle", ())
    for b, n in enumerate(lens):
        pre = n if b in idle else n - 1
        if pre > 0:
            k = torch.from_numpy(case["k"][b][:pre]).to("cuda", in_dt)
            v = torch.from_numpy(case["v"][b][:pre]).to("cuda", in_dt)
            sl = torch.from_numpy(case["slots"][b][:pre].astype(np.int64)).cuda()
            for c, e in caches:
                wc.quantize_write_pair(c, e, k, v, sl)
    new_k = np.zeros((batch, wl.n_kv, wl.d), np.float32)
    new_v = np.zeros((batch, wl.n_kv, wl.d), np.float32)
    new_slots = np.full(batch, -1, np.int64)
    for b, n in enumerate(lens):
        if n > 0 and b not in idle:
            new_k[b], new_v[b], new_slots[b] = case["k"][b][-1], case["v"][b][-1], case["slots"][b][-1]
    nk = torch.from_numpy(new_k).to("cuda", in_dt)
    nv = torch.from_numpy(new_v).to("cuda", in_dt)
    ns = torch.from_numpy(new_slots).cuda()
    q = torch.from_numpy(case["q"]).to("cuda", q_dt)
    table = torch.from_numpy(case["table"]).cuda()
    sl = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L = max(int(case["seq_lens"].max()), 1)
    sm = 1 / np.sqrt(wl.d)
    tau = 0.2
    if opts.get("force_valu"):
        os.environ["WITCERT_FORCE_VALU"] = "1"
    try:
        n1 = torch.zeros(2, dtype=torch.int32, device="cuda")
        (c1, e1), (c2, e2) = caches
        fused = wc.step_metered_decode_gate(c1, e1, nk, nv, ns, q, table, sl, L, sm, tau, split_tokens=split,
                                            n_gated=n1)
        n2 = torch.zeros(2, dtype=torch.int32, device="cuda")
        wc.quantize_write_pair(c2, e2, nk, nv, ns)
        ref = wc.metered_decode_gate(c2, q, table, sl, L, sm, tau, split_tokens=split, n_gated=n2)
        torch.cuda.synchronize()
    finally:
        os.environ.pop("WITCERT_FORCE_VALU", None)
    for (x, y) in ((c1, c2), (e1, e2)):
        for n, t in x.tensors.items():
            if t is not None:
                assert torch.equal(t, y.tensors[n]), (name, n)
    for i, (x, y) in enumerate(zip(fused, ref)):
        assert torch.equal(x, y), (name, i)
    assert torch.equal(n1, n2), (name, n1.tolist(), n2.tolist())


def test_step_graph_replay():
    import torch

    import paper_2607_28699_amd as wc
    S.say("[step] graph replay")
    wl = W_GQA
    lens = [900, 130]
    case = S.make_case(wl, lens, permute=True, layer=5)
    c, e = _caches(case, "int8_dither", {}, None)
    for b in range(len(lens)):
        wc.quantize_write_pair(c, e, torch.from_numpy(case["k"][b][:-1]).to("cuda", torch.bfloat16),
                               torch.from_numpy(case["v"][b][:-1]).to("cuda", torch.bfloat16),
                               torch.from_numpy(case["slots"][b][:-1].astype(np.int64)).cuda())
    nk = torch.from_numpy(np.stack([k[-1] for k in case["k"]])).to("cuda", torch.bfloat16)
    nv = torch.from_numpy(np.stack([v[-1] for v in case["v"]])).to("cuda", torch.bfloat16)
    ns = torch.from_numpy(np.array([s[-1] for s in case["slots"]], np.int64)).cuda()
    q = torch.from_numpy(case["q"]).to("cuda", torch.bfloat16)
    table = torch.from_numpy(case["table"]).cuda()
    sl = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L, sm = max(lens), 1 / np.sqrt(wl.d)
    ws = wc.decode_workspace(len(lens), wl.n_q, wl.n_kv, wl.d, L, 64)
    out = torch.empty((len(lens), wl.n_q, wl.d), dtype=torch.float32, device="cuda")
    meter = torch.empty((len(lens), wl.n_q), dtype=torch.float32, device="cuda")
    raw, mq = torch.empty_like(meter), torch.empty((len(lens), wl.n_q), dtype=torch.uint8, device="cuda")
    mk = torch.empty((len(lens), wl.n_kv), dtype=torch.uint8, device="cuda")

    def run():
        wc.step_metered_decode_gate(c, e, nk, nv, ns, q, table, sl, L, sm, 0.2, split_tokens=64, ws=ws, out=out,
                                    meter=meter, raw=raw, mask_q=mq, mask_kv=mk)

    run()
    torch.cuda.synchronize()
    want = [x.clone() for x in (out, meter, raw, mq, mk)] + [t.clone() for t in c.tensors.values() if t is not None]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    for rep in range(4):
        for x in (out, meter, raw):
            x.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        got = [out, meter, raw, mq, mk] + [t for t in c.tensors.values() if t is not None]
        for i, (x, y) in enumerate(zip(got, want)):
            assert torch.equal(x, y), (rep, i)
