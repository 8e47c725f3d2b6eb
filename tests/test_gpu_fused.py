"""Fused entry points against the calls they fuse (GPU).

wc_quantize_write_pair must leave both caches bit-identical to two separate
wc_quantize_write calls; wc_metered_decode_gate must give bit-identical outputs,
meter, raw, masks and counts to wc_metered_decode_attention followed by wc_gate.
"""
import numpy as np
import pytest

import synth

from . import support as S

pytestmark = pytest.mark.gpu

W_TINY = synth.WORKLOADS["tiny-d64-s256"]
W_GQA = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]


@pytest.mark.parametrize("kind", ["int8_dither", "fp8_raw"])
def test_write_pair_equals_two_writes(kind):
    import torch

    import paper_2607_28699_amd as wc
    S.say(f"[fused] write pair {kind}")
    wl = W_GQA
    case = S.make_case(wl, [300, 17], permute=True, layer=4)
    dt = S.torch_dtype(wl)

    def fresh():
        return (wc.PagedCache(kind, case["nblocks"], wl.n_kv, wl.d, wl.bands, layer=4,
                              seed=wl.philox_seed(), rope_layout=wl.rope_layout),
                wc.PagedCache("bf16", case["nblocks"], wl.n_kv, wl.d, 0, layer=4))

    a_c, a_e = fresh()
    b_c, b_e = fresh()
    for k, v, sl in zip(case["k"], case["v"], case["slots"]):
        kt, vt = torch.from_numpy(k).to("cuda", dt), torch.from_numpy(v).to("cuda", dt)
        st = torch.from_numpy(sl).cuda()
        wc.quantize_write_pair(a_c, a_e, kt, vt, st)
        wc.quantize_write(b_c, kt, vt, st)
        wc.quantize_write(b_e, kt, vt, st)
    torch.cuda.synchronize()
    for x, y in ((a_c, b_c), (a_e, b_e)):
        for n, t in x.tensors.items():
            if t is not None:
                assert torch.equal(t, y.tensors[n]), n


FUSED_CASES = [
    ("gqa", W_GQA, [700, 0, 129], 0.2),
    ("gqa-raw", W_GQA, [700, 0, 129], 40.0),
    ("gqa-informative", W_GQA.replace(q_scale=1 / 16, n_outliers=0), [777, 129], 0.05),
    ("gqa-group16", W_GQA.replace(n_q=32, n_kv=2), [300, 64], 0.1),
    ("tiny-vector-path", W_TINY, [257, 1, 0, 130], 0.2),
]


@pytest.mark.parametrize("name,wl,lens,tau", FUSED_CASES)
def test_decode_gate_equals_decode_then_gate(name, wl, lens, tau):
    import torch

    import paper_2607_28699_amd as wc
    S.say(f"[fused] decode+gate {name} tau={tau}")
    case = S.make_case(wl, lens, permute=True, layer=2)
    cache = S.gpu_cache(case, "int8_dither")
    q = torch.from_numpy(case["q"]).to("cuda", S.torch_dtype(wl))
    table = torch.from_numpy(case["table"]).cuda()
    sl = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L = max(int(case["seq_lens"].max()), 1)
    sm = 1 / np.sqrt(wl.d)
    o1, m1, r1 = wc.metered_decode_attention(cache, q, table, sl, L, sm)
    n1 = torch.zeros(2, dtype=torch.int32, device="cuda")
    mq1, mk1 = wc.gate(m1, r1, wl.group, tau, n_gated=n1)
    # twice, the masks primed with garbage: the fused call must clear what it sets
    ws = wc.decode_workspace(q.shape[0], wl.n_q, wl.n_kv, wl.d, L)
    for rep in range(2):
        mq2 = torch.full_like(mq1, 0xAB)
        mk2 = torch.full_like(mk1, 0xCD)
        n2 = torch.zeros(2, dtype=torch.int32, device="cuda")
        o2, m2, r2, mq2, mk2 = wc.metered_decode_gate(cache, q, table, sl, L, sm, tau, ws=ws,
                                                      mask_q=mq2, mask_kv=mk2, n_gated=n2)
        torch.cuda.synchronize()
        assert torch.equal(o1, o2) and torch.equal(m1, m2) and torch.equal(r1, r2), rep
        assert torch.equal(mq1, mq2) and torch.equal(mk1, mk2), rep
        assert torch.equal(n1, n2), (rep, n1.tolist(), n2.tolist())
