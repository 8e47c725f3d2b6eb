"""GPU parity of the per-token 32-channel group scales (Sec. 6.2 storage side,
Table 4: one fp16 scale per token and group) against the oracle.

* write path: codes, group scales, witness, bypassed values and the value side
  bit-exact, both RoPE layouts, d = 64 and 128;
* decode on both paths (matrix cores for head_dim 128 and bf16 queries, the
  vector ALUs otherwise or when forced): Tier A (witness), Tier B (radius over the
  group steps) and the joint K + V gate: outputs within 1e-5 (fp32 workloads) /
  2e-3 (bf16) of the oracle, raw
  relative, the meter never below the true TV, the gate bit-exact;
* block repair over a group-scaled cache against the oracle's repaired state.
"""
import numpy as np
import pytest

import synth
from oracle import attention
from oracle import decode as odec
from oracle import gate as ogate
from oracle import groupscale as ogs
from oracle import meter as mt
from oracle import repair as orep

from . import support as S

pytestmark = pytest.mark.gpu

W_TINY = synth.WORKLOADS["tiny-d64-s256"]
W_GQA = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]
INFORMATIVE = W_GQA.replace(q_scale=1 / 16, n_outliers=0)
DLOC = 1e-6

CASES = [
    ("tiny", W_TINY, [272, 0, 33], 0),
    ("gqa", W_GQA, [700, 129, 1], 0),
    ("gqa-informative", INFORMATIVE, [777, 129], 0),
    ("gqa-bypass4", W_GQA, [333, 18], 4),
    ("gqa-group16", W_GQA.replace(n_q=32, n_kv=2), [400, 90], 0),
]


def _setup(wl, lens, m, layer=2):
    case = S.make_case(wl, lens, permute=True, layer=layer)
    pairs = S.case_pairs(case, m) if m else None
    refs = S.oracle_write(case, "int8_dither", pairs, group_scales=True)
    cache = S.gpu_cache(case, "int8_dither", pairs=pairs, value_side=True, group_scales=True)
    return case, pairs, refs, cache


@pytest.mark.parametrize("name,wl,lens,m", CASES)
@pytest.mark.parametrize("layout", ["half", "interleaved"])
def test_groupscale_write_bitexact(name, wl, lens, m, layout):
    wl = wl.replace(rope_layout=layout)
    S.say(f"[gs-write] {name} layout={layout} lens={lens} m={m}")
    case, pairs, refs, cache = _setup(wl, lens, m)
    n_grouped = 0
    for b, r in enumerate(refs):
        if case["seq_lens"][b] == 0:
            continue
        got = S.read_cache(cache, case["slots"][b])
        assert np.array_equal(got["k"].astype(np.int64), r["kcode"])
        assert np.array_equal(got["v"].astype(np.int64), r["vcode"])
        assert np.array_equal(got["ks"], r["ks"]) and np.array_equal(got["vs"], r["vs"])
        assert np.array_equal(got["kw"], r["kw"])
        assert np.array_equal(got["vr"], r["vr"]) and np.array_equal(got["vn"], r["vn"])
        if m:
            assert np.array_equal(got["ko"], r["ko"])
        n_grouped += int(np.sum(r["ks"].max(axis=-1) != r["ks"].min(axis=-1)))   # groups differ
    assert n_grouped > 0


def _decode(case, cache, tier, tau, tau_v, force_valu=False, joint=True):
    import os

    import torch

    import paper_2607_28699_amd as wc
    wl = case["wl"]
    q = torch.from_numpy(case["q"]).to("cuda", S.torch_dtype(wl))
    table = torch.from_numpy(case["table"]).cuda()
    lens = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L = max(int(case["seq_lens"].max()), 1)
    n = torch.zeros(2, dtype=torch.int32, device="cuda")
    sm = 1 / np.sqrt(wl.d)
    if force_valu:
        os.environ["WITCERT_FORCE_VALU"] = "1"
    try:
        if joint:
            res = wc.joint_decode_gate(cache, q, table, lens, L, sm, tau, tau_v,
                                       0.0 if tier == "A" else DLOC, n_gated=n)
        elif tier == "A":
            res = wc.metered_decode_gate(cache, q, table, lens, L, sm, tau, n_gated=n)
        else:
            o, m_, r_ = wc.tierb_decode_attention(cache, q, table, lens, L, sm, DLOC)
            mq, mk = wc.gate(m_, r_, wl.n_q // wl.n_kv, tau)
            res = (o, m_, r_, mq, mk)
    finally:
        os.environ.pop("WITCERT_FORCE_VALU", None)
    torch.cuda.synchronize()
    return [x.cpu().numpy() for x in res]


@pytest.mark.parametrize("name,wl,lens,m", CASES)
@pytest.mark.parametrize("tier", ["A", "B"])
@pytest.mark.parametrize("path", ["default", "vector"])
@pytest.mark.parametrize("joint", [True, False])
def test_groupscale_decode_parity(name, wl, lens, m, tier, path, joint):
    from oracle import value as ov
    if path == "vector" and wl.d != 128:
        pytest.skip("head_dim 64 always takes the vector path")
    S.say(f"[gs-decode] {name} tier={tier} path={path} joint={joint} lens={lens} m={m}")
    case, pairs, refs, cache = _setup(wl, lens, m)
    sm = 1 / np.sqrt(wl.d)
    tol = S.out_tol(wl)
    ref = []
    for b, c in enumerate(refs):
        if case["seq_lens"][b] == 0:
            ref.append(None)
            continue
        q = case["q"][b]
        if tier == "A":
            base = odec.metered_decode(q, c["khat"], c["vhat"], c["kw"], sm, wl.bands, wl.rope_layout)
            cb = base["c"]
        else:
            base = ogs.tierb_decode(q, c["khat"], c["vhat"], c["ks"], sm, DLOC,
                                    c.get("ko"), c.get("chans"))
            cb = base["u"]
        j = ov.joint_decode(q, c["khat"], c["vhat"], cb, c["vr"], c["vn"], sm)
        j["tv"] = odec.true_tv(q, case["k"][b], c["khat"], sm)
        ref.append(j)
    # thresholds inside the range of the oracle's values, so the gate goes both ways
    raws = np.concatenate([r["raw"] for r in ref if r is not None])
    mvs = np.concatenate([r["meter_v"] for r in ref if r is not None])
    tau = float(min(np.quantile(raws, 0.5), 0.9))
    tau_v = float(np.quantile(mvs, 0.5))
    if joint:
        out, meter, raw, mv, mq, mk = _decode(case, cache, tier, tau, tau_v, path == "vector")
    else:
        out, meter, raw, mq, mk = _decode(case, cache, tier, tau, tau_v, path == "vector", joint=False)
        mv = None
    for b, r in enumerate(ref):
        if r is None:
            assert np.all(meter[b] == 0) and np.all(mq[b] == 0)
            continue
        assert S.rel_err(out[b], r["out"]) <= tol, (b, S.rel_err(out[b], r["out"]))
        fin = r["raw"] < 1e30
        assert np.all(np.abs(raw[b][fin] - r["raw"][fin]) <= tol * np.maximum(r["raw"][fin], 1e-30)), \
            (b, np.max(np.abs(raw[b][fin] - r["raw"][fin]) / np.maximum(r["raw"][fin], 1e-30)))
        assert np.all(meter[b] >= r["tv"])
        if mv is None:   # the key gate alone
            exp_q = ogate.gate_q(meter[b], raw[b], tau)
        else:
            assert np.all(np.abs(mv[b] - r["meter_v"]) <= tol * np.maximum(r["meter_v"], 1e-30))
            # the joint gate as a function of the GPU's own meters, bit-exact
            exp_q = ov.joint_gate_q(meter[b], raw[b], mv[b], tau, tau_v)
        assert np.array_equal(mq[b].astype(bool), np.asarray(exp_q, dtype=bool))
        assert np.array_equal(mk[b].astype(bool), ogate.gate_kv(np.asarray(exp_q)[None], wl.n_q // wl.n_kv)[0].astype(bool))
    S.say(f"  tau={tau:.3g} tau_v={tau_v:.3g} gated q heads {int(mq.sum())}/{mq.size}")


def test_groupscale_block_repair():
    import torch

    import paper_2607_28699_amd as wc
    wl = INFORMATIVE
    lens = [1500, 700]
    split = 256
    S.say(f"[gs-repair] lens={lens}")
    case, _, refs, cache = _setup(wl, lens, 0)
    exact = S.gpu_cache(case, "bf16")
    sm = 1 / np.sqrt(wl.d)
    g = wl.n_q // wl.n_kv
    bounds, raws = [], []
    for b, c in enumerate(refs):
        cb = odec.metered_decode(case["q"][b], c["khat"], c["vhat"], c["kw"], sm, wl.bands, wl.rope_layout)["c"]
        bounds.append(cb)
        for h in range(wl.n_q):
            z = attention.logits(case["q"][b][h], c["khat"][:, h // g], sm)
            raws.append(mt.raw_from_am1(mt.a_minus_one_logits(z, cb[h])))
    tau = float(np.quantile(raws, 0.2))
    q = torch.from_numpy(case["q"]).to("cuda", S.torch_dtype(wl))
    table = torch.from_numpy(case["table"]).cuda()
    lens_t = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L = int(case["seq_lens"].max())
    ws = wc.decode_workspace(q.shape[0], wl.n_q, wl.n_kv, wl.d, L, split)
    out, meter, raw, mq, mk = wc.metered_decode_gate(cache, q, table, lens_t, L, sm, tau, ws=ws,
                                                     split_tokens=split)
    n_rep, rep = wc.block_repair(cache, exact, q, table, lens_t, L, sm, tau, ws, out, meter, raw, mk,
                                 max_blocks=16, split_tokens=split)
    torch.cuda.synchronize()
    out, raw, n_rep, rep = (x.cpu().numpy() for x in (out, raw, n_rep, rep))
    fixed = 0
    for b in range(len(lens)):
        for kv in range(wl.n_kv):
            if n_rep[b, kv] <= 0:
                continue
            hs = slice(kv * g, (kv + 1) * g)
            c = refs[b]
            kx = synth.bf16_round(case["k"][b][:, kv]).astype(np.float64)
            vx = synth.bf16_round(case["v"][b][:, kv]).astype(np.float64)
            ranges = orep.paper_blocks(int(case["seq_lens"][b]))
            st = orep.repaired_state(case["q"][b][hs], c["khat"][:, kv], c["vhat"][:, kv], kx, vx,
                                     bounds[b][hs], rep[b, kv, :n_rep[b, kv]], ranges, sm)
            assert S.rel_err(out[b, hs], st["out"]) <= S.out_tol(wl)
            assert np.all(np.abs(raw[b, hs] - st["raw"]) <= S.out_tol(wl) * np.maximum(st["raw"], 1e-30) + 1e-7)
            fixed += 1
    S.say(f"  repaired KV heads: {fixed}")
    assert fixed > 0


def test_groupscale_graph_replay_is_bit_identical():
    import torch

    import paper_2607_28699_amd as wc
    S.say("[gs-decode] graph replay")
    case, _, _, cache = _setup(W_GQA, [700, 300], 4)
    q = torch.from_numpy(case["q"]).to("cuda", torch.bfloat16)
    table = torch.from_numpy(case["table"]).cuda()
    lens = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    ws = wc.decode_workspace(2, 28, 4, 128, 700)
    out = torch.empty((2, 28, 128), device="cuda")
    meter = torch.empty((2, 28), device="cuda")
    raw = torch.empty((2, 28), device="cuda")
    mv = torch.empty((2, 28), device="cuda")
    mq = torch.empty((2, 28), dtype=torch.uint8, device="cuda")
    mk = torch.empty((2, 4), dtype=torch.uint8, device="cuda")
    args = (cache, q, table, lens, 700, 1 / np.sqrt(128), 0.2, 0.05, DLOC)
    kw = dict(ws=ws, out=out, meter=meter, raw=raw, meter_v=mv, mask_q=mq, mask_kv=mk)
    wc.joint_decode_gate(*args, **kw)
    torch.cuda.synchronize()
    eager = [x.clone() for x in (out, meter, raw, mv, mq, mk)]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            wc.joint_decode_gate(*args, **kw)
    torch.cuda.synchronize()
    for _ in range(3):
        for x in (out, meter, raw, mv, mq, mk):
            x.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip((out, meter, raw, mv, mq, mk), eager):
            assert torch.equal(a, b)
