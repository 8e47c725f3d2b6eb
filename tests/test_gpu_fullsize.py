"""Parity at the full workload sizes, in the launch configuration bench.py times.

One layer of each long-context workload is prefilled through
wc_quantize_write_pair (quantized cache and bf16 exact copy), then one decode step
runs through wc_step_metered_decode_gate -- the step's token written by the
decode kernel itself -- and through wc_step_certified_decode and its speculative
form, the calls bench.py times (the same step with the exact fallback: meters and
masks bit-identical, a routed head's output exact attention; the speculative form
bit-identical to the certified one), with bench.py's split choice
(max_seq_len = prefill + steps + warmup, the split balanced over the batch's
total tokens; the serving mix with all 64 sequences).  Sampled (sequence, query
head) cells, the shortest and the longest sequence among them, are recomputed by
the oracle one by one from the stored inputs of that cell, and sampled tokens'
codes are compared bit-exactly.  Also: the matrix-core and vector-ALU decode
paths agree on the same cache.
"""
import os

import numpy as np
import pytest

import synth
from oracle import decode as odec
from oracle import quantizer as oq
from oracle import tierb

from . import support as S

pytestmark = pytest.mark.gpu

BENCH_STEPS, BENCH_WARMUP = 8, 2


def _setup(name):
    import torch

    import paper_2607_28699_amd as wc
    from synth import torch_gen
    wl = synth.WORKLOADS[name]
    lens0 = (synth.serving_lengths(wl.batch, wl.len_lo, wl.ctx) if wl.ragged
             else np.full(wl.batch, wl.ctx, dtype=np.int64))
    extra = BENCH_STEPS + BENCH_WARMUP
    table, nblocks = synth.block_table(lens0 + extra, permute=wl.ragged, seed_key=wl.wid)
    layer = 5
    cache = wc.PagedCache("int8_dither", nblocks, wl.n_kv, wl.d, wl.bands, layer=layer,
                          seed=wl.philox_seed(), rope_layout=wl.rope_layout)
    exact = wc.PagedCache("bf16", nblocks, wl.n_kv, wl.d, 0, layer=layer)
    kv, new_k, new_v, new_slots = [], [], [], []
    for b, L in enumerate(lens0):
        pos = torch.arange(int(L) + 1, device="cuda")
        k, v = torch_gen.gen_kv_layer(wl, layer, b, pos)
        sl = synth.slots_of(table, b, np.arange(int(L) + 1))
        wc.quantize_write_pair(cache, exact, k[:-1], v[:-1], torch.from_numpy(sl[:-1]).cuda())
        kv.append((k, v, sl))
        new_k.append(k[-1])
        new_v.append(v[-1])
        new_slots.append(int(sl[-1]))
    pos = torch.from_numpy(lens0).cuda()
    q = torch_gen.gen_q_batch(wl, layer, 0, pos)
    lens = torch.from_numpy((lens0 + 1).astype(np.int32)).cuda()
    tab = torch.from_numpy(table).cuda()
    max_len = int(lens0.max() + extra)
    # bench.py's split: balanced over the batch's total tokens at the last timed step
    st = wc.split_tokens_for(len(lens0), wl.n_kv, max_len, total_tokens=int((lens0 + extra).sum()))
    step = (torch.stack(new_k), torch.stack(new_v), torch.tensor(new_slots, dtype=torch.int64, device="cuda"))
    return wl, lens0, cache, exact, kv, q, tab, lens, max_len, layer, st, step


def _cell_check(wl, kv, q, b, h, layer):
    """Oracle result for query head h of sequence b from that cell's stored inputs."""
    k, v, sl = kv[b]
    g = h // wl.group
    kb = k[:, g].float().cpu().numpy().astype(np.float64)
    vb = v[:, g].float().cpu().numpy().astype(np.float64)
    qb = q[b, h:h + 1].float().cpu().numpy().astype(np.float64)
    kc, ks, _, kh = oq.int8_quantize_slots(kb, sl, layer, g, wl.philox_seed())
    vc, vs, _, vh = oq.int8_quantize_slots(vb, sl, layer, g, wl.philox_seed())
    kw = oq.witness(kb, kh, wl.bands, wl.rope_layout)
    sm = 1 / np.sqrt(wl.d)
    res = odec.metered_decode(qb, kh[:, None], vh[:, None], kw[:, None], sm, wl.bands, wl.rope_layout)
    tv = odec.true_tv(qb, kb[:, None], kh[:, None], sm)
    res["khat"], res["vhat"] = kh, vh
    return res, tv, kc, vc, ks


@pytest.mark.parametrize("name", ["gqa-28x4-d128-s32k-b4", "gqa-28x4-d128-s131k-b1", "serving-64seq-paged"])
def test_fullsize_sampled_cells(name):
    import torch

    import paper_2607_28699_amd as wc
    S.say(f"[fullsize] {name}")
    wl, lens0, cache, exact, kv, q, tab, lens, max_len, layer, st, (nk, nv, ns) = _setup(name)
    sm = 1 / np.sqrt(wl.d)
    tau = 0.2
    out, meter, raw, mask_q, mask_kv = wc.step_metered_decode_gate(cache, exact, nk, nv, ns, q, tab, lens,
                                                                   max_len, sm, tau, split_tokens=st)
    dloc = wc.tierb_delta_loc(1e-2, wl.n_layers, wl.n_q, 256)
    _, meter_b, raw_b = wc.tierb_decode_attention(cache, q, tab, lens, max_len, sm, dloc, split_tokens=st)
    torch.cuda.synchronize()
    out, meter, raw = out.cpu().numpy(), meter.cpu().numpy(), raw.cpu().numpy()
    mask_q, mask_kv = mask_q.cpu().numpy(), mask_kv.cpu().numpy()
    meter_b, raw_b = meter_b.cpu().numpy(), raw_b.cpu().numpy()
    # the gate as a function of the GPU's meter (the end-to-end decision is in the gate tests)
    assert np.array_equal(mask_q, (meter > tau).astype(np.uint8))
    assert np.array_equal(mask_kv, mask_q.reshape(len(lens0), wl.n_kv, wl.group).max(-1))
    rng = np.random.default_rng(17)
    seqs = sorted({int(np.argmin(lens0)), int(np.argmax(lens0)), int(rng.integers(len(lens0)))})
    cells = [(b, int(rng.integers(wl.n_q))) for b in seqs]
    oracle_cells = {}
    for b, h in cells:
        S.say(f"  cell b={b} h={h} L={int(lens0[b]) + 1} split={st}")
        res, tv, kc, vc, ks = _cell_check(wl, kv, q, b, h, layer)
        oracle_cells[(b, h)] = (res, tv)
        assert S.rel_err(out[b, h], res["out"][0]) <= 2e-3
        assert abs(raw[b, h] - res["raw"][0]) <= 2e-3 * res["raw"][0]
        assert meter[b, h] >= tv[0]
        # the Tier-B certificate of the same cell (Sec. 4.2)
        rb = tierb.tierb_decode(q[b, h:h + 1].float().cpu().numpy().astype(np.float64), res["khat"][:, None],
                                res["vhat"][:, None], ks[:, None], sm, dloc)
        assert abs(raw_b[b, h] - rb["raw"][0]) <= 2e-3 * rb["raw"][0]
        assert meter_b[b, h] >= tv[0]
        # codes of sampled tokens of this cell (the step's token among them), bit-exact
        sl = kv[b][2]
        pick = np.unique(np.concatenate([rng.choice(len(sl), min(512, len(sl)), replace=False), [len(sl) - 1]]))
        got = S.read_cache(cache, sl[pick])
        g = h // wl.group
        assert np.array_equal(got["k"][:, g].astype(np.int64), kc[pick])
        assert np.array_equal(got["v"][:, g].astype(np.int64), vc[pick])
        assert np.array_equal(got["ks"][:, g], ks[pick])
        # the exact copy holds the bf16 inputs
        gx = S.read_cache(exact, sl[pick])
        kin = kv[b][0][:, g].float().cpu().numpy()[pick]
        assert np.array_equal(S.bf16_bits_to_f32(gx["k"][:, g]), kin)
    # the certified step (what bench.py times) on the same caches: the step's token is
    # written again with the same bytes; meters and masks as above, bit for bit; a
    # routed KV head's rows are exact attention, the others the metered rows
    ws = wc.certified_workspace(len(lens0), wl.n_q, wl.n_kv, wl.d, max_len, st)
    c_out, c_meter, c_raw, c_mq, c_mk = wc.step_certified_decode(cache, exact, nk, nv, ns, q, tab, lens, max_len, sm,
                                                                 tau, split_tokens=st, ws=ws)
    torch.cuda.synchronize()
    c_out = c_out.cpu().numpy()
    assert np.array_equal(c_meter.cpu().numpy(), meter) and np.array_equal(c_raw.cpu().numpy(), raw)
    assert np.array_equal(c_mq.cpu().numpy(), mask_q) and np.array_equal(c_mk.cpu().numpy(), mask_kv)
    unrouted = np.repeat(mask_kv == 0, wl.group, axis=1)
    assert np.array_equal(c_out[unrouted], out[unrouted])
    for b, h in cells:
        if mask_kv[b, h // wl.group]:
            k, v, _ = kv[b]
            g = h // wl.group
            ex = odec.exact_decode(q[b, h:h + 1].float().cpu().numpy().astype(np.float64),
                                   k[:, g:g + 1].float().cpu().numpy().astype(np.float64),
                                   v[:, g:g + 1].float().cpu().numpy().astype(np.float64), sm)["out"]
            assert S.rel_err(c_out[b, h], ex[0]) <= 2e-3, (b, h)
    # its speculative form (what bench.py times when the first step routes at least
    # half of the KV heads): the certified step's results bit for bit
    nq_ = torch.zeros(2, dtype=torch.int32, device="cuda")
    s_res = wc.step_certified_decode_speculative(cache, exact, nk, nv, ns, q, tab, lens, max_len, sm, tau,
                                                 split_tokens=st, ws=ws, n_gated=nq_)
    torch.cuda.synchronize()
    for x, y in zip(s_res, (c_out, c_meter, c_raw, c_mq, c_mk)):
        y = y if isinstance(y, np.ndarray) else y.cpu().numpy()
        assert np.array_equal(x.cpu().numpy(), y)
    # and at the split bench.py gives that form (about half the decode calls'
    # workgroups per split set): the sampled cells against the oracle, the gate as a
    # function of its own meter
    st_s = wc.speculative_split_tokens(len(lens0), wl.n_kv, max_len, total_tokens=int((lens0 + max_len - lens0.max()).sum()))
    S.say(f"  speculative split {st_s} (decode split {st})")
    s_out, s_meter, s_raw, s_mq, s_mk = (x.cpu().numpy() for x in wc.step_certified_decode_speculative(
        cache, exact, nk, nv, ns, q, tab, lens, max_len, sm, tau, split_tokens=st_s, ws=ws))
    assert np.array_equal(s_mq, (s_meter > tau).astype(np.uint8))
    assert np.array_equal(s_mk, s_mq.reshape(len(lens0), wl.n_kv, wl.group).max(-1))
    for (b, h), (res, tv) in oracle_cells.items():
        assert abs(s_raw[b, h] - res["raw"][0]) <= 2e-3 * res["raw"][0]
        assert s_meter[b, h] >= tv[0]
        if s_mk[b, h // wl.group]:
            k, v, _ = kv[b]
            g = h // wl.group
            want = odec.exact_decode(q[b, h:h + 1].float().cpu().numpy().astype(np.float64),
                                     k[:, g:g + 1].float().cpu().numpy().astype(np.float64),
                                     v[:, g:g + 1].float().cpu().numpy().astype(np.float64), sm)["out"][0]
        else:
            want = res["out"][0]
        assert S.rel_err(s_out[b, h], want) <= 2e-3, (b, h)


def test_matrix_core_and_vector_paths_agree():
    import torch

    import paper_2607_28699_amd as wc
    S.say("[fullsize] mfma vs valu")
    wl = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]
    case = S.make_case(wl, [4097, 1000, 33, 1], permute=True)
    out = {}
    for kind in ("int8_dither", "fp8_raw"):
        cache = S.gpu_cache(case, kind)
        a = S.gpu_decode(case, cache)
        os.environ["WITCERT_FORCE_VALU"] = "1"
        try:
            bv = S.gpu_decode(case, cache)
        finally:
            del os.environ["WITCERT_FORCE_VALU"]
        assert S.rel_err(a[0], bv[0]) <= 2e-3
        assert np.all(np.abs(a[2] - bv[2]) <= 2e-3 * np.abs(bv[2]))
        out[kind] = a
    _ = torch


def test_fullsize_bypass_group_scales():
    """The bench's third cache at full size (32k context, batch 4): pairs chosen on
    the GPU from the layer's keys, 32-channel group scales, value side; sampled
    cells of Tier A, Tier B and the value meter against the oracle."""
    import torch

    import paper_2607_28699_amd as wc
    from oracle import bypass as obp
    from oracle import groupscale as ogs
    from oracle import philox as oph
    from oracle import value as ov
    from synth import torch_gen
    name = "gqa-28x4-d128-s32k-b4"
    S.say(f"[fullsize] {name} bypass + group scales")
    wl = synth.WORKLOADS[name]
    lens0 = np.full(wl.batch, wl.ctx, dtype=np.int64)
    extra = BENCH_STEPS + BENCH_WARMUP
    table, nblocks = synth.block_table(lens0 + extra, permute=False, seed_key=wl.wid)
    layer, m = 3, 4
    kv = []
    for b, L in enumerate(lens0):
        k, v = torch_gen.gen_kv_layer(wl, layer, b, torch.arange(int(L) + 1, device="cuda"))
        kv.append((k, v, synth.slots_of(table, b, np.arange(int(L) + 1))))
    kall = torch.cat([k for k, _, _ in kv])
    pairs = wc.select_outlier_pairs(kall, m, wl.rope_layout)
    ka = kall.float().cpu().numpy().astype(np.float64)
    ref_pairs = np.stack([obp.select_pairs(ka[:, h], m, wl.rope_layout) for h in range(wl.n_kv)])
    assert np.array_equal(pairs.cpu().numpy(), ref_pairs)
    del ka
    cache = wc.PagedCache("int8_dither", nblocks, wl.n_kv, wl.d, wl.bands, layer=layer, seed=wl.philox_seed(),
                          rope_layout=wl.rope_layout, n_outlier_pairs=m, value_side=True, group_scales=True)
    cache.set_outlier_pairs(pairs)
    for k, v, sl in kv:
        wc.quantize_write(cache, k, v, torch.from_numpy(sl).cuda())
    q = torch_gen.gen_q_batch(wl, layer, 0, torch.from_numpy(lens0).cuda())
    lens = torch.from_numpy((lens0 + 1).astype(np.int32)).cuda()
    tab = torch.from_numpy(table).cuda()
    max_len = int(lens0.max() + extra)
    sm = 1 / np.sqrt(wl.d)
    dloc = wc.tierb_delta_loc(1e-2, wl.n_layers, wl.n_q, 256)
    out, meter, raw, mv, _, _ = wc.joint_decode_gate(cache, q, tab, lens, max_len, sm, 0.2, 0.05)
    _, meter_b, raw_b = wc.tierb_decode_attention(cache, q, tab, lens, max_len, sm, dloc)
    torch.cuda.synchronize()
    out, meter, raw, mv = (x.cpu().numpy() for x in (out, meter, raw, mv))
    meter_b, raw_b = meter_b.cpu().numpy(), raw_b.cpu().numpy()
    rng = np.random.default_rng(23)
    for b, h in [(int(rng.integers(wl.batch)), int(rng.integers(wl.n_q))) for _ in range(2)]:
        S.say(f"  cell b={b} h={h}")
        k, v, sl = kv[b]
        g = h // wl.group
        kb = k[:, g].float().cpu().numpy().astype(np.float64)
        vb = v[:, g].float().cpu().numpy().astype(np.float64)
        qb = q[b, h:h + 1].float().cpu().numpy().astype(np.float64)
        chans = obp.bypass_channels(ref_pairs[g], wl.d, wl.rope_layout)
        xi = oph.dither_values(sl, wl.d, layer, g, wl.philox_seed())
        kc, ks, ko, kh = ogs.quantize(kb, xi, chans)
        vc, vs, _, vh = ogs.quantize(vb, xi)
        kw = oq.witness(kb, kh, wl.bands, wl.rope_layout)
        ra = odec.metered_decode(qb, kh[:, None], vh[:, None], kw[:, None], sm, wl.bands, wl.rope_layout)
        rb = ogs.tierb_decode(qb, kh[:, None], vh[:, None], ks[:, None], sm, dloc, ko[:, None],
                              chans[None])
        tv = odec.true_tv(qb, kb[:, None], kh[:, None], sm)
        j = ov.joint_decode(qb, kh[:, None], vh[:, None], ra["c"], ov.value_residual(vb[:, None], vh[:, None]),
                            ov.value_norm(vb[:, None]), sm)
        assert S.rel_err(out[b, h], ra["out"][0]) <= 2e-3
        assert abs(raw[b, h] - ra["raw"][0]) <= 2e-3 * ra["raw"][0]
        assert abs(raw_b[b, h] - rb["raw"][0]) <= 2e-3 * rb["raw"][0]
        assert abs(mv[b, h] - j["meter_v"][0]) <= 2e-3 * j["meter_v"][0]
        assert meter[b, h] >= tv[0] and meter_b[b, h] >= tv[0]
        pick = rng.choice(len(sl), 512, replace=False)
        got = S.read_cache(cache, sl[pick])
        assert np.array_equal(got["k"][:, g].astype(np.int64), kc[pick])
        assert np.array_equal(got["v"][:, g].astype(np.int64), vc[pick])
        assert np.array_equal(got["ks"][:, g], ks[pick]) and np.array_equal(got["vs"][:, g], vs[pick])
