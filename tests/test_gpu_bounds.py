"""Inputs that point outside the cache (GPU): the kernels never touch memory
outside it, and the other sequences' results do not change.

* a slot at or beyond num_blocks * 16 (like a negative slot) is skipped by the
  write: the cache is byte-identical to a write of the valid tokens only;
* a block-table entry outside [0, num_blocks) (here num_blocks itself and -5)
  in one sequence leaves the outputs, meter, raw and gates of the other
  sequences bit-identical, on the matrix-core path, the vector path, the exact
  fallback and block repair (the affected sequence's result is unspecified).
"""
import os

import numpy as np
import pytest

import synth

from . import support as S

pytestmark = pytest.mark.gpu

W_GQA = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]
W_TINY = synth.WORKLOADS["tiny-d64-s256"]


def test_write_skips_slots_outside_the_cache():
    import torch

    import paper_2607_28699_amd as wc
    S.say("[bounds] write slots")
    wl = W_GQA
    case = S.make_case(wl, [300], permute=True, layer=1)
    k = torch.from_numpy(case["k"][0]).to("cuda", torch.bfloat16)
    v = torch.from_numpy(case["v"][0]).to("cuda", torch.bfloat16)
    slots = torch.from_numpy(case["slots"][0].astype(np.int64)).cuda()
    cap = case["nblocks"] * 16
    bad = slots.clone()
    bad[5], bad[17], bad[100] = cap, cap + 12345, -3

    def fresh():
        return (wc.PagedCache("int8_dither", case["nblocks"], wl.n_kv, wl.d, wl.bands, layer=1,
                              seed=wl.philox_seed(), rope_layout=wl.rope_layout),
                wc.PagedCache("bf16", case["nblocks"], wl.n_kv, wl.d, 0, layer=1))

    a_c, a_e = fresh()
    b_c, b_e = fresh()
    wc.quantize_write_pair(a_c, a_e, k, v, bad)
    keep = torch.ones(len(slots), dtype=torch.bool, device="cuda")
    keep[[5, 17, 100]] = False
    wc.quantize_write_pair(b_c, b_e, k[keep].contiguous(), v[keep].contiguous(), slots[keep].contiguous())
    torch.cuda.synchronize()
    for x, y in ((a_c, b_c), (a_e, b_e)):
        for n, t in x.tensors.items():
            if t is not None:
                assert torch.equal(t, y.tensors[n]), n


def _decode_all(case, cache, exact, table, vector, tau=0.2):
    import torch

    import paper_2607_28699_amd as wc
    wl = case["wl"]
    dt = S.torch_dtype(wl)
    q = torch.from_numpy(case["q"]).to("cuda", dt if vector else torch.bfloat16)
    lens = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L = int(case["seq_lens"].max())
    sm = 1 / np.sqrt(wl.d)
    if vector:
        os.environ["WITCERT_FORCE_VALU"] = "1"
    try:
        o, m, r, mq, mk = wc.metered_decode_gate(cache, q, table, lens, L, sm, tau, split_tokens=64)
        fb = o.clone()
        wc.exact_decode_attention(exact, q, table, lens, L, sm, mk, fb, split_tokens=64)
        res = [o, m, r, mq, mk, fb]
        if not vector and wl.d == 128:
            mq2, mk2 = mq.clone(), mk.clone()
            ws = wc.decode_workspace(q.shape[0], wl.n_q, wl.n_kv, wl.d, L, 64)
            o2, m2, r2, mq2, mk2 = wc.metered_decode_gate(cache, q, table, lens, L, sm, tau, ws=ws,
                                                          split_tokens=64, mask_q=mq2, mask_kv=mk2)
            rep = torch.full((q.shape[0], wl.n_kv, 8), -1, dtype=torch.int32, device="cuda")
            nrep = torch.zeros((q.shape[0], wl.n_kv), dtype=torch.int32, device="cuda")
            wc.block_repair(cache, exact, q, table, lens, L, sm, tau, ws, o2, m2, r2, mk2, max_blocks=8,
                            split_tokens=64, repaired=rep, n_repaired=nrep)
            res += [o2, m2, r2, mk2, rep, nrep]
    finally:
        os.environ.pop("WITCERT_FORCE_VALU", None)
    torch.cuda.synchronize()
    return [x.clone() for x in res]


@pytest.mark.parametrize("wl,vector", [(W_GQA, False), (W_GQA, True), (W_TINY, True)],
                         ids=["mfma", "vector", "vector-d64"])
def test_table_entries_outside_the_cache(wl, vector):
    import torch
    S.say(f"[bounds] table entries vector={vector} d={wl.d}")
    case = S.make_case(wl, [300, 200, 150], permute=True, layer=2)
    cache = S.gpu_cache(case, "int8_dither")
    exact = S.gpu_cache(case, "bf16")
    good = torch.from_numpy(case["table"]).cuda()
    bad = good.clone()
    bad[1, 2] = case["nblocks"]          # one past the last block
    bad[1, 7] = -5
    ref = _decode_all(case, cache, exact, good, vector)
    got = _decode_all(case, cache, exact, bad, vector)
    keep = [0, 2]                        # the sequences whose tables are intact
    for i, (x, y) in enumerate(zip(ref, got)):
        assert torch.equal(x[keep], y[keep]), i
