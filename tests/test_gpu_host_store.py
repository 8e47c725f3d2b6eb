"""An exact store in pinned host memory (GPU): the kernels read the paper's CPU copy
of the cache (Sec. 6.3) over the host link, with the same results as from device
memory.

The exact fallback and block repair take a bf16 cache whose arrays live in pinned
host memory (PagedCache(host=True), or host_copy() of a device cache); both are
bit-identical to the same calls on the device copy.
"""
import numpy as np
import pytest

import synth

from . import support as S

pytestmark = pytest.mark.gpu

W_GQA = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]
INFORMATIVE = W_GQA.replace(q_scale=1 / 16, n_outliers=0)


def test_host_store_fallback_and_repair_bit_identical():
    import torch

    import paper_2607_28699_amd as wc
    wl = INFORMATIVE
    lens = [1500, 700, 33]
    split = 256
    S.say(f"[host store] lens={lens}")
    case = S.make_case(wl, lens, permute=True, layer=2)
    cache = S.gpu_cache(case, "int8_dither")
    exact = S.gpu_cache(case, "bf16")
    exact_h = exact.host_copy()
    assert not exact_h.tensors["k_data"].is_cuda and exact_h.tensors["k_data"].is_pinned()
    q = torch.from_numpy(case["q"]).to("cuda", torch.bfloat16)
    table = torch.from_numpy(case["table"]).cuda()
    lens_t = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L, sm = max(lens), 1 / np.sqrt(wl.d)
    ws = wc.decode_workspace(len(lens), wl.n_q, wl.n_kv, wl.d, L, split)
    out, meter, raw, mq, mk = wc.metered_decode_gate(cache, q, table, lens_t, L, sm, 0.0, ws=ws, split_tokens=split)
    assert int(mk.sum()) == mk.numel()   # tau 0: every KV head routed (no sequence is empty)
    res = {}
    for name, ex in (("device", exact), ("host", exact_h)):
        o = out.clone()
        wc.exact_decode_attention(ex, q, table, lens_t, L, sm, mk, o, ws=ws, split_tokens=split)
        torch.cuda.synchronize()
        res[name] = o
    assert torch.equal(res["device"], res["host"])
    # block repair from the host store: the same blocks, outputs and meters
    tau = float(torch.quantile(raw.flatten(), 0.3).item())
    rep = {}
    for name, ex in (("device", exact), ("host", exact_h)):
        o, m_, r_, q_, k_ = wc.metered_decode_gate(cache, q, table, lens_t, L, sm, tau, ws=ws, split_tokens=split)
        n_rep, lst = wc.block_repair(cache, ex, q, table, lens_t, L, sm, tau, ws, o, m_, r_, k_, max_blocks=16,
                                     split_tokens=split)
        torch.cuda.synchronize()
        rep[name] = (o, m_, r_, k_, n_rep, lst)
    for x, y in zip(rep["device"], rep["host"]):
        assert torch.equal(x, y)
    assert int((rep["host"][4] > 0).sum()) > 0, "nothing repaired"
