"""GPU parity of persistent repair (the meter loop's gate, Sec. 6: repaired
slots keep their exact values and lose their witness; Sec. 6.3 gated evaluation
(c)) against the oracle.

* Decode over a cache whose pages carry repair marks (random marks, and every page
  marked): each decode variant serves the marked pages from the exact store with
  bound 0 -- outputs, raw and meter (and the value meter) against the oracle's
  mixed state (``repair.decode_repaired``) at 1e-5 (fp32) / 2e-3 (bf16) relative,
  on both decode paths, Tier A and Tier B keys, bypassed pairs, group scales and
  the fp8 cache; with every page marked the output is exact attention and raw 0.
* Two steps of one request: step 1 repairs (block repair, whole-head fallback
  where the budget does not suffice) and writes back -- the marks equal the
  oracle's ``persist`` / ``persist_all`` pages and the marked slots' witnesses are
  zero; step 2 writes new tokens (the last through the step call) and decodes the
  mixed state as the oracle does; its repair ranks only blocks that still hold an
  unmarked token and takes the oracle's blocks.
"""
import os
import zlib

import numpy as np
import pytest

import synth
from oracle import attention
from oracle import bypass as obp
from oracle import decode as odec
from oracle import groupscale as ogs
from oracle import meter as mt
from oracle import repair as orep
from oracle import tierb
from oracle import value as ov

from . import support as S

pytestmark = pytest.mark.gpu

W_TINY = synth.WORKLOADS["tiny-d64-s256"]
W_GQA = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]
INFORMATIVE = W_GQA.replace(q_scale=1 / 16, n_outliers=0)
DLOC = 1e-6
SPLIT = 256

# name, workload, lengths, kind, tier, bypassed pairs, value side, group scales
DEC_CASES = [
    ("tiny", W_TINY, [272, 0, 130], "int8_dither", "A", 0, False, False),
    ("gqa", W_GQA, [700, 129], "int8_dither", "A", 0, False, False),
    ("gqa-group8", W_GQA.replace(n_q=32, n_kv=4), [333, 18], "int8_dither", "A", 0, False, False),
    ("gqa-group16", W_GQA.replace(n_q=32, n_kv=2), [300, 47], "int8_dither", "A", 0, False, False),
    ("gqa-tierb", W_GQA.replace(q_scale=1 / 4), [600, 64], "int8_dither", "B", 0, False, False),
    ("gqa-bypass", W_GQA, [500, 33], "int8_dither", "A", 4, False, False),
    ("gqa-bypass-tierb", W_GQA.replace(q_scale=1 / 4), [400], "int8_dither", "B", 4, False, False),
    ("gqa-value", W_GQA, [450, 70], "int8_dither", "A", 0, True, False),
    ("gqa-group-scales", W_GQA, [380, 21], "int8_dither", "A", 0, False, True),
    ("gqa-group-scales-tierb", W_GQA.replace(q_scale=1 / 4), [420, 37], "int8_dither", "B", 0, False, True),
    ("gqa-group-scales-value-bypass", W_GQA, [360, 45], "int8_dither", "A", 4, True, True),
    ("gqa-fp8", W_GQA, [480, 17], "fp8_raw", "A", 0, False, False),
    ("tiny-fp8", W_TINY, [200, 31], "fp8_raw", "A", 0, False, False),
]


def _tensors(case, q=None, lens=None):
    import torch
    wl = case["wl"]
    q = case["q"] if q is None else q
    lens = case["seq_lens"] if lens is None else lens
    return (torch.from_numpy(np.asarray(q)).to("cuda", S.torch_dtype(wl)),
            torch.from_numpy(case["table"]).cuda(),
            torch.from_numpy(np.asarray(lens).astype(np.int32)).cuda())


def _rep_tokens(case, marks, b, S_):
    """bool [S_, n_kv]: position t of sequence b is served exactly when the physical
    page holding it is marked."""
    pos = np.arange(S_)
    return marks[case["table"][b][pos // S.BLOCK]].astype(bool)


def _bounds(case, c, b, tier, pairs, gs):
    """Per-token bounds [n_q, S] of the compressed keys (Tier A witness bound or Tier B radius)."""
    wl = case["wl"]
    sm = 1 / np.sqrt(wl.d)
    q = case["q"][b]
    if tier == "A":
        return odec.metered_decode(q, c["khat"], c["vhat"], c["kw"], sm, wl.bands, wl.rope_layout)["c"]
    if gs:
        return ogs.tierb_decode(q, c["khat"], c["vhat"], c["ks"], sm, DLOC)["u"]
    if pairs is None:
        return tierb.tierb_decode(q, c["khat"], c["vhat"], c["ks"], sm, DLOC)["u"]
    return obp.tierb_decode(q, c["khat"], c["vhat"], c["ks"], c["ko"], c["chans"], sm, DLOC)["u"]


@pytest.mark.parametrize("density", [0.35, 1.0])
@pytest.mark.parametrize("path", ["default", "vector"])
@pytest.mark.parametrize("name,wl,lens,kind,tier,m,vm,gs", DEC_CASES)
def test_decode_with_repair_marks(name, wl, lens, kind, tier, m, vm, gs, path, density):
    import torch

    import paper_2607_28699_amd as wc
    if path == "vector" and wl.d != 128:
        pytest.skip("this case always takes the vector path")
    S.say(f"[persistent decode] {name} path={path} density={density}")
    case = S.make_case(wl, lens, permute=True, layer=3)
    pairs = S.case_pairs(case, m) if m else None
    refs = S.oracle_write(case, kind, pairs, group_scales=gs)
    cache = S.gpu_cache(case, kind, pairs=pairs, value_side=vm, group_scales=gs)
    exact = S.gpu_cache(case, "bf16")
    cache.enable_repair(exact)
    rng = np.random.default_rng(zlib.crc32(f"{name}/{density}".encode()))
    marks = rng.random((case["nblocks"], wl.n_kv)) < density
    cache.tensors["repaired"].copy_(torch.from_numpy(marks.astype(np.uint8)))
    q, table, lens_t = _tensors(case)
    L = max(int(case["seq_lens"].max()), 1)
    sm = 1 / np.sqrt(wl.d)
    delta = 0.0 if tier == "A" else DLOC
    if path == "vector":
        os.environ["WITCERT_FORCE_VALU"] = "1"
    try:
        if vm:
            res = wc.joint_decode_gate(cache, q, table, lens_t, L, sm, float("inf"), float("inf"), delta)
            out, meter, raw, mv = (x.cpu().numpy() for x in res[:4])
        elif tier == "A":
            out, meter, raw = (x.cpu().numpy() for x in wc.metered_decode_attention(cache, q, table, lens_t, L, sm))
        else:
            out, meter, raw = (x.cpu().numpy() for x in wc.tierb_decode_attention(cache, q, table, lens_t, L, sm,
                                                                                   DLOC))
    finally:
        os.environ.pop("WITCERT_FORCE_VALU", None)
    tol = S.out_tol(wl)
    g = wl.n_q // wl.n_kv
    for b, c in enumerate(refs):
        S_ = int(case["seq_lens"][b])
        if S_ == 0:
            assert np.all(out[b] == 0) and np.all(raw[b] == 0)
            continue
        rep = _rep_tokens(case, marks, b, S_)
        kx = synth.bf16_round(case["k"][b]).astype(np.float64)
        vx = synth.bf16_round(case["v"][b]).astype(np.float64)
        cb = _bounds(case, c, b, tier, pairs, gs)
        r = orep.decode_repaired(case["q"][b], c["khat"], c["vhat"], kx, vx, cb, rep, sm)
        assert S.rel_err(out[b], r["out"]) <= tol, (b, S.rel_err(out[b], r["out"]))
        fin = r["raw"] < 1e30
        assert np.all(np.abs(raw[b][fin] - r["raw"][fin]) <= tol * np.maximum(r["raw"][fin], 1e-30) + 1e-30), \
            (b, raw[b], r["raw"])
        if rep.all():
            assert np.all(raw[b] == 0) and np.all(meter[b] == 0)
        # still sound: the meter bounds the TV between exact attention and the served mix
        # (bf16 workloads: the exact store holds the inputs exactly)
        for h in range(wl.n_q if wl.dtype != "f32" else 0):
            kv = h // g
            p = attention.softmax(attention.logits(case["q"][b][h], case["k"][b][:, kv], sm))
            kk = np.where(rep[:, kv, None], kx[:, kv], c["khat"][:, kv])
            pr = attention.softmax(attention.logits(case["q"][b][h], kk, sm))
            assert meter[b][h] >= attention.tv(p, pr) * (1 - 1e-6) - 1e-7
        if vm:
            for h in range(wl.n_q):
                kv = h // g
                want = ov.value_meter(r["ptilde"][h], np.where(rep[:, kv], 0.0, c["vr"][:, kv]), c["vn"][:, kv])
                assert abs(mv[b][h] - want) <= tol * max(want, 1e-30), (b, h, mv[b][h], want)


def _write(cache, exact, case, lo, hi):
    """Write positions lo[b] .. hi[b]-1 of every sequence b (quantized + exact copy)."""
    import torch

    import paper_2607_28699_amd as wc
    wl = case["wl"]
    dt = S.torch_dtype(wl)
    ks = np.concatenate([k[a:e] for k, a, e in zip(case["k"], lo, hi)])
    vs = np.concatenate([v[a:e] for v, a, e in zip(case["v"], lo, hi)])
    sl = np.concatenate([s[a:e] for s, a, e in zip(case["slots"], lo, hi)]).astype(np.int64)
    wc.quantize_write_pair(cache, exact, torch.from_numpy(ks).to("cuda", dt), torch.from_numpy(vs).to("cuda", dt),
                           torch.from_numpy(sl).cuda())


def _oracle_repair(case, refs, b, kv, q, S_, tau, max_blocks, rep_pages):
    """Oracle block repair of KV head kv of sequence b at length S_ over the
    repaired pages rep_pages (logical page flags)."""
    wl = case["wl"]
    g = wl.n_q // wl.n_kv
    sm = 1 / np.sqrt(wl.d)
    hs = slice(kv * g, (kv + 1) * g)
    c = refs[b]
    cb = odec.metered_decode(q, c["khat"][:S_], c["vhat"][:S_], c["kw"][:S_], sm, wl.bands, wl.rope_layout)["c"]
    kx = synth.bf16_round(case["k"][b][:S_, kv]).astype(np.float64)
    vx = synth.bf16_round(case["v"][b][:S_, kv]).astype(np.float64)
    base = orep.token_mask(rep_pages, S_)
    return orep.block_repair(q[hs], c["khat"][:S_, kv], c["vhat"][:S_, kv], kx, vx, cb[hs], orep.paper_blocks(S_),
                             sm, tau, max_blocks, base=base), cb


@pytest.mark.parametrize("path", ["default", "vector"])
def test_persistent_repair_two_steps(path):
    import torch

    import paper_2607_28699_amd as wc
    wl = INFORMATIVE
    S2 = np.array([1560, 760, 300])
    S1 = S2 - 40                   # step 2 adds 40 tokens per sequence (crossing pages)
    S.say(f"[persistent two steps] path={path}")
    case = S.make_case(wl, S2, permute=True, layer=5)
    refs = S.oracle_write(case, "int8_dither")
    g = wl.n_q // wl.n_kv
    sm = 1 / np.sqrt(wl.d)
    max_blocks = 3
    cache = wc.PagedCache("int8_dither", case["nblocks"], wl.n_kv, wl.d, wl.bands, layer=case["layer"],
                          seed=wl.philox_seed(), rope_layout=wl.rope_layout)
    exact = wc.PagedCache("bf16", case["nblocks"], wl.n_kv, wl.d, wl.bands, layer=case["layer"],
                          seed=wl.philox_seed(), rope_layout=wl.rope_layout)
    cache.enable_repair(exact)
    _write(cache, exact, case, np.zeros_like(S1), S1)
    # ---- step 1 over the first S1 tokens ----
    q1 = np.stack([synth.gen_q(wl, case["layer"], b, 0, int(s) - 1) for b, s in enumerate(S1)])
    raws = []
    for b in range(len(S1)):
        c = refs[b]
        cb = odec.metered_decode(q1[b], c["khat"][:S1[b]], c["vhat"][:S1[b]], c["kw"][:S1[b]], sm, wl.bands,
                                 wl.rope_layout)["c"]
        for h in range(wl.n_q):
            z = attention.logits(q1[b][h], c["khat"][:S1[b], h // g], sm)
            raws.append(mt.raw_from_am1(mt.a_minus_one_logits(z, cb[h])))
    tau = float(np.quantile(raws, 0.3))
    qt, table, lens1 = _tensors(case, q1, S1)
    if path == "vector":
        os.environ["WITCERT_FORCE_VALU"] = "1"
    try:
        ws = wc.decode_workspace(len(S1), wl.n_q, wl.n_kv, wl.d, int(S2.max()), SPLIT)
        out, meter, raw, mq, mk = wc.metered_decode_gate(cache, qt, table, lens1, int(S1.max()), sm, tau, ws=ws,
                                                         split_tokens=SPLIT)
        n_rep, rep = wc.block_repair(cache, exact, qt, table, lens1, int(S1.max()), sm, tau, ws, out, meter, raw,
                                     mk, max_blocks=max_blocks, split_tokens=SPLIT)
        wc.repair_write_back(cache, table, lens1, rep, n_rep, whole_kv=mk)
        torch.cuda.synchronize()
        n_rep1, rep1, mk1 = n_rep.cpu().numpy(), rep.cpu().numpy(), mk.cpu().numpy()
        marks = cache.tensors["repaired"].cpu().numpy().astype(bool)
        # oracle write-back of the GPU's decisions (the decisions themselves are
        # checked against the oracle by the block-repair tests)
        want = np.zeros_like(marks)
        pages_of = {}
        for b in range(len(S1)):
            for kv in range(wl.n_kv):
                rp = np.zeros(orep.pages_of(int(S2[b])), bool)
                if n_rep1[b, kv] > 0:
                    rp = orep.persist(rp, rep1[b, kv, :n_rep1[b, kv]], orep.paper_blocks(int(S1[b])), int(S1[b]))
                if mk1[b, kv]:
                    rp = orep.persist_all(rp, int(S1[b]))
                pages_of[(b, kv)] = rp
                want[case["table"][b][np.flatnonzero(rp)], kv] = True
        S.say(f"  step 1: repaired {n_rep1.ravel().tolist()}, whole-head {mk1.ravel().tolist()}, "
              f"marked pages {int(marks.sum())}")
        assert marks.sum() > 0 and np.array_equal(marks, want)
        wit = cache.tensors["k_witness"].cpu().numpy()
        assert np.all(wit[marks] == 0)
        assert np.any(wit[~marks] != 0)
        # ---- step 2: 39 more tokens written, the 40th through the step call ----
        _write(cache, exact, case, S1, S2 - 1)
        dt = S.torch_dtype(wl)
        q2 = np.stack([synth.gen_q(wl, case["layer"], b, 1, int(s) - 1) for b, s in enumerate(S2)])
        qt2, _, lens2 = _tensors(case, q2, S2)
        new_k = torch.from_numpy(np.stack([case["k"][b][S2[b] - 1] for b in range(len(S2))])).to("cuda", dt)
        new_v = torch.from_numpy(np.stack([case["v"][b][S2[b] - 1] for b in range(len(S2))])).to("cuda", dt)
        new_slots = torch.from_numpy(np.array([case["slots"][b][S2[b] - 1] for b in range(len(S2))],
                                              dtype=np.int64)).cuda()
        out2, meter2, raw2, mq2, mk2 = wc.step_metered_decode_gate(cache, exact, new_k, new_v, new_slots, qt2, table,
                                                                   lens2, int(S2.max()), sm, tau, ws=ws,
                                                                   split_tokens=SPLIT)
        torch.cuda.synchronize()
        o2, r2 = out2.cpu().numpy(), raw2.cpu().numpy()
        n_rep2, rep2 = wc.block_repair(cache, exact, qt2, table, lens2, int(S2.max()), sm, tau, ws, out2, meter2,
                                       raw2, mk2, max_blocks=max_blocks, split_tokens=SPLIT)
        torch.cuda.synchronize()
        n_rep2, rep2 = n_rep2.cpu().numpy(), rep2.cpu().numpy()
    finally:
        os.environ.pop("WITCERT_FORCE_VALU", None)
    tol = S.out_tol(wl)
    n_checked = 0
    for b in range(len(S2)):
        c = refs[b]
        S_ = int(S2[b])
        kx = synth.bf16_round(case["k"][b]).astype(np.float64)
        vx = synth.bf16_round(case["v"][b]).astype(np.float64)
        cb = odec.metered_decode(q2[b], c["khat"], c["vhat"], c["kw"], sm, wl.bands, wl.rope_layout)["c"]
        rep_tok = np.stack([orep.token_mask(pages_of[(b, kv)], S_) for kv in range(wl.n_kv)], 1)
        r = orep.decode_repaired(q2[b], c["khat"], c["vhat"], kx, vx, cb, rep_tok, sm)
        assert S.rel_err(o2[b], r["out"]) <= tol, (b, S.rel_err(o2[b], r["out"]))
        assert np.all(np.abs(r2[b] - r["raw"]) <= tol * np.maximum(r["raw"], 1e-30) + 1e-30)
        for kv in range(wl.n_kv):
            if rep_tok[:, kv].all():
                assert np.all(r2[b][kv * g:(kv + 1) * g] == 0)
            if n_rep2[b, kv] == 0:
                continue
            res, _ = _oracle_repair(case, refs, b, kv, q2[b], S_, tau, max_blocks, pages_of[(b, kv)])
            cand = orep.candidates(rep_tok[:, kv], orep.paper_blocks(S_))
            K = min(max_blocks, int(cand.sum()))
            got = rep2[b, kv, :K]
            assert all(cand[j] for j in got), (b, kv, got)
            tot = res["shares"].sum(axis=0)
            for i in range(min(K, res["order"].size)):
                if got[i] != res["order"][i]:
                    assert abs(tot[got[i]] - tot[res["order"][i]]) <= 1e-5 * tot.max(), (b, kv, i)
            n_checked += 1
    S.say(f"  step 2: repaired {n_rep2.ravel().tolist()}, checked {n_checked}")
    assert n_checked > 0
