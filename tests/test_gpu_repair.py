"""GPU parity of block-granular repair (Sec. 6.3, block-level paging) against the oracle.

After a metered decode with its gate, wc_block_repair takes the routed KV heads'
blocks (fixed 256-token runs of the sequence, Sec. 6.3) in decreasing order of
their meter shares until every query head passes tau:
* the number of blocks taken matches the oracle's minimal count (a count whose
  stopping state lies within 1e-3 relative of tau is accepted either way), and the
  block order matches (blocks whose totals are within 1e-5 relative may swap);
* repaired KV heads: outputs within 1e-5 (fp32) / 2e-3 (bf16) of the oracle's
  repaired state, raw and meter relative, mask cleared; heads the budget cannot
  repair and heads that were not routed are left untouched;
* both decode paths produced the records; Tier A and Tier B keys; bypassed pairs;
* the blocks do not depend on the decode's split: two split lengths take the same
  blocks in the same order and give the same repaired state within the merge's
  rounding.
"""
import os

import numpy as np
import pytest

import synth
from oracle import attention
from oracle import bypass as obp
from oracle import meter as mt
from oracle import decode as odec
from oracle import repair as orep
from oracle import tierb

from . import support as S

pytestmark = pytest.mark.gpu

W_TINY = synth.WORKLOADS["tiny-d64-s256"]
W_GQA = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]
INFORMATIVE = W_GQA.replace(q_scale=1 / 16, n_outliers=0)
DLOC = 1e-6
SPLIT = 256           # tokens per KV split of the decodes (repair blocks are 256 tokens regardless)

CASES = [
    ("tiny", W_TINY.replace(q_scale=1 / 8), [1000, 0, 300], "A", 0, 8),
    ("gqa-informative", INFORMATIVE, [1500, 700, 0, 300], "A", 0, 16),
    ("gqa-informative-tierb", INFORMATIVE, [1500, 700], "B", 0, 16),
    ("gqa-bypass-tierb", W_GQA.replace(q_scale=1 / 4), [900, 333], "B", 4, 16),
    ("gqa-small-budget", INFORMATIVE, [1500, 700], "A", 0, 2),
]


def _run(case, cache, exact, tier, tau, max_blocks, force_valu, round0=None, split=SPLIT):
    import torch

    import paper_2607_28699_amd as wc
    wl = case["wl"]
    q = torch.from_numpy(case["q"]).to("cuda", S.torch_dtype(wl))
    table = torch.from_numpy(case["table"]).cuda()
    lens = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L = max(int(case["seq_lens"].max()), 1)
    sm = 1 / np.sqrt(wl.d)
    delta = 0.0 if tier == "A" else DLOC
    if force_valu:
        os.environ["WITCERT_FORCE_VALU"] = "1"
    if round0 is not None:
        os.environ["WITCERT_REPAIR_ROUND0"] = str(round0)
    try:
        ws = wc.decode_workspace(q.shape[0], wl.n_q, wl.n_kv, wl.d, L, split)
        if tier == "A":
            out, meter, raw, mq, mk = wc.metered_decode_gate(cache, q, table, lens, L, sm, tau, ws=ws,
                                                             split_tokens=split)
        else:
            out, meter, raw = wc.tierb_decode_attention(cache, q, table, lens, L, sm, delta, ws=ws,
                                                        split_tokens=split)
            mq, mk = wc.gate(meter, raw, wl.group, tau)
        before = (out.clone(), meter.clone(), raw.clone(), mk.clone())
        n_rep, rep = wc.block_repair(cache, exact, q, table, lens, L, sm, tau, ws, out, meter, raw, mk,
                                     delta_loc=delta, max_blocks=max_blocks, split_tokens=split)
    finally:
        os.environ.pop("WITCERT_FORCE_VALU", None)
        os.environ.pop("WITCERT_REPAIR_ROUND0", None)
    torch.cuda.synchronize()
    cpu = lambda t: t.cpu().numpy()
    return ([cpu(x) for x in before], cpu(out).astype(np.float64), cpu(meter), cpu(raw), cpu(mk),
            cpu(n_rep), cpu(rep))


@pytest.mark.parametrize("name,wl,lens,tier,m,max_blocks", CASES)
@pytest.mark.parametrize("path", ["default", "vector"])
def test_block_repair_parity(name, wl, lens, tier, m, max_blocks, path):
    if path == "vector" and wl.d != 128:
        pytest.skip("head_dim 64 always takes the vector path")
    case = S.make_case(wl, lens, permute=True, layer=1)
    pairs = S.case_pairs(case, m) if m else None
    refs = S.oracle_write(case, "int8_dither", pairs)
    sm = 1 / np.sqrt(wl.d)
    g = wl.n_q // wl.n_kv
    # per (sequence, KV head): the bounds c of its query heads, from the oracle
    bounds = []
    for b, c in enumerate(refs):
        if case["seq_lens"][b] == 0:
            bounds.append(None)
            continue
        q = case["q"][b]
        if tier == "A":
            cb = odec.metered_decode(q, c["khat"], c["vhat"], c["kw"], sm, wl.bands, wl.rope_layout)["c"]
        elif pairs is None:
            cb = tierb.tierb_decode(q, c["khat"], c["vhat"], c["ks"], sm, DLOC)["u"]
        else:
            cb = obp.tierb_decode(q, c["khat"], c["vhat"], c["ks"], c["ko"], c["chans"], sm, DLOC)["u"]
        bounds.append(cb)
    # a threshold that routes most heads but that a few blocks can meet
    raws = []
    for b in range(len(refs)):
        if case["seq_lens"][b] == 0:
            continue
        for h in range(wl.n_q):
            z = attention.logits(case["q"][b][h], refs[b]["khat"][:, h // g], sm)
            raws.append(mt.raw_from_am1(mt.a_minus_one_logits(z, bounds[b][h])))
    tau = float(np.quantile(raws, 0.2))
    S.say(f"[repair] {name} path={path} tier={tier} tau={tau:.4g} max_blocks={max_blocks}")
    cache = S.gpu_cache(case, "int8_dither", pairs=pairs)
    exact = S.gpu_cache(case, "bf16")
    before, out, meter, raw, mk, n_rep, rep = _run(case, cache, exact, tier, tau, max_blocks, path == "vector")
    out0, meter0, raw0, mk0 = before
    tol = S.out_tol(wl)
    n_fixed = 0
    for b in range(len(lens)):
        for kv in range(wl.n_kv):
            hs = slice(kv * g, (kv + 1) * g)
            if case["seq_lens"][b] == 0 or mk0[b, kv] == 0:
                assert n_rep[b, kv] == 0
                assert np.array_equal(out[b, hs], out0[b, hs].astype(np.float64))
                continue
            c = refs[b]
            S_ = case["seq_lens"][b]
            # the exact store holds bf16 (the fallback cache): repaired blocks take those values
            kx = synth.bf16_round(case["k"][b][:, kv]).astype(np.float64)
            vx = synth.bf16_round(case["v"][b][:, kv]).astype(np.float64)
            ranges = orep.paper_blocks(S_)
            res = orep.block_repair(case["q"][b][hs], c["khat"][:, kv], c["vhat"][:, kv], kx, vx,
                                    bounds[b][hs], ranges, sm, tau, max_blocks)
            # the order: same blocks up to swaps of near-equal totals
            tot = res["shares"].sum(axis=0)
            K = min(max_blocks, len(ranges))
            got_order = rep[b, kv, :K]
            for i in range(K):
                if got_order[i] != res["order"][i]:
                    assert abs(tot[got_order[i]] - tot[res["order"][i]]) <= 1e-5 * tot.max(), (b, kv, i)
            n_o, n_g = res["n_blocks"], n_rep[b, kv]
            if n_g != n_o:
                # accepted only at a stopping state within 1e-3 of tau
                n_lo = min(x for x in (n_o, n_g) if x > 0) if max(n_o, n_g) > 0 else K
                st = orep.repaired_state(case["q"][b][hs], c["khat"][:, kv], c["vhat"][:, kv], kx, vx,
                                         bounds[b][hs], got_order[:n_lo], ranges, sm)
                val = st["raw"] if tau >= 1 else st["meter"]
                assert np.max(np.abs(val - tau)) <= 1e-3 * tau, (b, kv, n_o, n_g)
                continue
            if n_g == -1:
                assert mk[b, kv] == 1
                assert np.array_equal(out[b, hs], out0[b, hs].astype(np.float64))
                continue
            n_fixed += 1
            assert mk[b, kv] == 0
            st = orep.repaired_state(case["q"][b][hs], c["khat"][:, kv], c["vhat"][:, kv], kx, vx,
                                     bounds[b][hs], got_order[:n_g], ranges, sm)
            S.say(f"  ({b},{kv}) blocks {n_g}, output error {S.rel_err(out[b, hs], st['out']):.2e}")
            assert S.rel_err(out[b, hs], st["out"]) <= tol, (b, kv, S.rel_err(out[b, hs], st["out"]))
            assert np.all(np.abs(raw[b, hs] - st["raw"]) <= tol * np.maximum(st["raw"], 1e-30) + 1e-7)
            assert np.all(meter[b, hs] <= tau + 1e-6 if tau < 1 else raw[b, hs] <= tau * (1 + 1e-6))
    S.say(f"  repaired KV heads: {n_fixed}, left to the fallback: {int((n_rep == -1).sum())}")
    if name != "gqa-small-budget":
        assert n_fixed > 0


@pytest.mark.parametrize("round0", [1, 2])
def test_block_repair_rounds_do_not_change_the_result(round0):
    """The block corrections run in two rounds (the predicted count first); forcing
    a first round of 1 or 2 blocks moves work into the second round and must give
    the same repaired state bit for bit (the corrections are added in the repair
    order whatever round computed them)."""
    name, wl, lens, tier, m, max_blocks = CASES[1]
    case = S.make_case(wl, lens, permute=True, layer=1)
    refs = S.oracle_write(case, "int8_dither")
    sm = 1 / np.sqrt(wl.d)
    g = wl.n_q // wl.n_kv
    raws = []
    for b in range(len(lens)):
        if case["seq_lens"][b] == 0:
            continue
        c = refs[b]
        cb = odec.metered_decode(case["q"][b], c["khat"], c["vhat"], c["kw"], sm, wl.bands, wl.rope_layout)["c"]
        for h in range(wl.n_q):
            z = attention.logits(case["q"][b][h], c["khat"][:, h // g], sm)
            raws.append(mt.raw_from_am1(mt.a_minus_one_logits(z, cb[h])))
    tau = 1e-3 * float(np.min(raws))   # low enough that most of the 256-token blocks are taken
    cache = S.gpu_cache(case, "int8_dither")
    exact = S.gpu_cache(case, "bf16")
    ref = _run(case, cache, exact, tier, tau, max_blocks, False)
    got = _run(case, cache, exact, tier, tau, max_blocks, False, round0=round0)
    S.say(f"[repair rounds] round0={round0} blocks {ref[5].ravel().tolist()}")
    assert np.any(ref[5] > round0), "no KV head needed the second round"
    for x, y in zip(ref[1:], got[1:]):
        assert np.array_equal(x, y)


def test_block_repair_graph_replay_is_bit_identical():
    """Metered decode with the gate and block repair captured in one HIP graph:
    every replay (eager work and synchronizations in between) equals the eager run."""
    import torch

    import paper_2607_28699_amd as wc
    name, wl, lens, tier, m, max_blocks = CASES[1]
    S.say("[repair] graph replay")
    case = S.make_case(wl, lens, permute=True, layer=1)
    cache = S.gpu_cache(case, "int8_dither")
    exact = S.gpu_cache(case, "bf16")
    q = torch.from_numpy(case["q"]).to("cuda", S.torch_dtype(wl))
    table = torch.from_numpy(case["table"]).cuda()
    lens_t = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L = int(case["seq_lens"].max())
    sm = 1 / np.sqrt(wl.d)
    B = q.shape[0]
    ws = wc.decode_workspace(B, wl.n_q, wl.n_kv, wl.d, L, SPLIT)
    rws = wc.repair_workspace(B, wl.n_q, wl.n_kv, wl.d, max_blocks)
    out = torch.empty((B, wl.n_q, wl.d), device="cuda")
    meter = torch.empty((B, wl.n_q), device="cuda")
    raw = torch.empty_like(meter)
    mq = torch.empty((B, wl.n_q), dtype=torch.uint8, device="cuda")
    mk = torch.empty((B, wl.n_kv), dtype=torch.uint8, device="cuda")
    nrep = torch.empty((B, wl.n_kv), dtype=torch.int32, device="cuda")
    rl = torch.empty((B, wl.n_kv, max_blocks), dtype=torch.int32, device="cuda")
    # a threshold that routes most heads but that a few blocks can meet
    _, _, r0 = wc.metered_decode_attention(cache, q, table, lens_t, L, sm, split_tokens=SPLIT)
    r0 = r0.cpu().numpy()[case["seq_lens"] > 0]
    tau = float(np.quantile(r0, 0.2))

    def step():
        wc.metered_decode_gate(cache, q, table, lens_t, L, sm, tau, ws=ws, out=out, meter=meter, raw=raw,
                               mask_q=mq, mask_kv=mk, split_tokens=SPLIT)
        wc.block_repair(cache, exact, q, table, lens_t, L, sm, tau, ws, out, meter, raw, mk,
                        max_blocks=max_blocks, split_tokens=SPLIT, repaired=rl, n_repaired=nrep, repair_ws=rws)
    step()
    torch.cuda.synchronize()
    eager = [x.clone() for x in (out, meter, raw, mk, nrep, rl)]
    assert int((eager[4] > 0).sum()) > 0, "nothing repaired"
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    g = torch.cuda.CUDAGraph()
    with torch.cuda.stream(s):
        with torch.cuda.graph(g, stream=s):
            step()
    torch.cuda.synchronize()
    for _ in range(3):
        for x in (out, meter, raw):
            x.zero_()
        mk.fill_(7)
        nrep.fill_(-9)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip((out, meter, raw, mk, nrep, rl), eager):
            assert torch.equal(a, b)


@pytest.mark.parametrize("path", ["default", "vector"])
def test_block_repair_does_not_depend_on_the_split(path):
    """Repair blocks are fixed 256-token runs: decodes with 64-, 256- and 1088-token
    splits (block segments recorded from different wave and split boundaries) take
    the same blocks in the same order (blocks whose totals are within 1e-5 relative
    may swap) and give the same repaired outputs within the split merge's rounding."""
    name, wl, lens, tier, m, max_blocks = CASES[1]
    case = S.make_case(wl, lens, permute=True, layer=2)
    refs = S.oracle_write(case, "int8_dither")
    sm = 1 / np.sqrt(wl.d)
    g = wl.n_q // wl.n_kv
    raws = []
    for b in range(len(lens)):
        if case["seq_lens"][b] == 0:
            continue
        c = refs[b]
        cb = odec.metered_decode(case["q"][b], c["khat"], c["vhat"], c["kw"], sm, wl.bands, wl.rope_layout)["c"]
        for h in range(wl.n_q):
            z = attention.logits(case["q"][b][h], c["khat"][:, h // g], sm)
            raws.append(mt.raw_from_am1(mt.a_minus_one_logits(z, cb[h])))
    tau = float(np.quantile(raws, 0.2))
    cache = S.gpu_cache(case, "int8_dither")
    exact = S.gpu_cache(case, "bf16")
    runs = {sp: _run(case, cache, exact, tier, tau, max_blocks, path == "vector", split=sp) for sp in (64, 256, 1088)}
    _, out0, meter0, raw0, mk0, nrep0, rep0 = runs[256]
    S.say(f"[repair split] path={path} blocks {nrep0.ravel().tolist()}")
    assert int((nrep0 > 0).sum()) > 0, "nothing repaired"
    for sp in (64, 1088):
        _, out1, meter1, raw1, mk1, nrep1, rep1 = runs[sp]
        for b in range(len(lens)):
            for kv in range(wl.n_kv):
                if nrep0[b, kv] != nrep1[b, kv]:
                    pytest.fail(f"split {sp}: ({b},{kv}) took {nrep1[b, kv]} blocks, split 256 took {nrep0[b, kv]}")
                n = max(int(nrep0[b, kv]), 0)
                if n and not np.array_equal(rep0[b, kv, :n], rep1[b, kv, :n]):
                    assert sorted(rep0[b, kv, :n].tolist()) == sorted(rep1[b, kv, :n].tolist()), (sp, b, kv)
        assert np.array_equal(mk0, mk1)
        assert S.rel_err(out1, out0) <= 2e-3
