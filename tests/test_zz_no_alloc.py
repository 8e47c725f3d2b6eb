"""The allocation-free decode step (GPU): wc_step_metered_decode_gate_noalloc,
whose split records live in the library's static per-GPU scratch, against
wc_step_metered_decode_gate with a caller workspace on twin caches.

Two calls in a row, the second with a smaller input (fewer, shorter sequences,
so the scratch still holds the first call's records past the second's); the
bar is bit-identical caches, outputs, meter, raw, gate masks and counts, on the
fused matrix-core path and on the vector path (write kernel then decode).
"""
import os

import numpy as np
import pytest

import synth

from . import support as S

pytestmark = pytest.mark.gpu

W_GQA = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]


def _step_pair(wl, lens, layer, split):
    """Twin caches holding all but each sequence's last token, and the step's inputs."""
    import torch

    import paper_2607_28699_amd as wc
    case = S.make_case(wl, lens, permute=True, layer=layer)
    caches = []
    for _ in range(2):
        c = wc.PagedCache("int8_dither", case["nblocks"], wl.n_kv, wl.d, wl.bands, layer=layer,
                          seed=wl.philox_seed(), rope_layout=wl.rope_layout)
        e = wc.PagedCache("bf16", case["nblocks"], wl.n_kv, wl.d, 0, layer=layer)
        for b in range(len(lens)):
            wc.quantize_write_pair(c, e, torch.from_numpy(case["k"][b][:-1]).to("cuda", torch.bfloat16),
                                   torch.from_numpy(case["v"][b][:-1]).to("cuda", torch.bfloat16),
                                   torch.from_numpy(case["slots"][b][:-1].astype(np.int64)).cuda())
        caches.append((c, e))
    inp = dict(
        nk=torch.from_numpy(np.stack([k[-1] for k in case["k"]])).to("cuda", torch.bfloat16),
        nv=torch.from_numpy(np.stack([v[-1] for v in case["v"]])).to("cuda", torch.bfloat16),
        ns=torch.from_numpy(np.array([s[-1] for s in case["slots"]], np.int64)).cuda(),
        q=torch.from_numpy(case["q"]).to("cuda", torch.bfloat16),
        table=torch.from_numpy(case["table"]).cuda(),
        lens=torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda(),
        L=max(lens), split=split)
    return caches, inp


def _outputs(batch, wl):
    import torch
    dev = "cuda"
    return dict(out=torch.full((batch, wl.n_q, wl.d), float("nan"), device=dev),
                meter=torch.full((batch, wl.n_q), float("nan"), device=dev),
                raw=torch.full((batch, wl.n_q), float("nan"), device=dev),
                mask_q=torch.full((batch, wl.n_q), 7, dtype=torch.uint8, device=dev),
                mask_kv=torch.full((batch, wl.n_kv), 7, dtype=torch.uint8, device=dev),
                n_gated=torch.zeros(2, dtype=torch.int32, device=dev))


@pytest.mark.parametrize("vector_path", [False, True])
def test_noalloc_step_equals_workspace_step(vector_path):
    import torch

    import paper_2607_28699_amd as wc
    wl = W_GQA
    sm, tau = 1 / np.sqrt(wl.d), 0.2
    if vector_path:
        os.environ["WITCERT_FORCE_VALU"] = "1"
    try:
        # the second call is smaller: fewer and shorter sequences, another split
        for i, (lens, split) in enumerate((([3000, 700, 129], 0), ([300, 77], 64))):
            S.say(f"[noalloc] call {i} lens={lens} split={split} vector_path={vector_path}")
            pair, inp = _step_pair(wl, lens, 6 + i, split)
            (c1, e1), (c2, e2) = pair
            o1, o2 = _outputs(len(lens), wl), _outputs(len(lens), wl)
            wc.step_metered_decode_gate_noalloc(c1, e1, inp["nk"], inp["nv"], inp["ns"], inp["q"], inp["table"],
                                                inp["lens"], inp["L"], sm, tau, o1["out"], o1["meter"],
                                                o1["raw"], o1["mask_q"], o1["mask_kv"], split_tokens=split,
                                                n_gated=o1["n_gated"])
            wc.step_metered_decode_gate(c2, e2, inp["nk"], inp["nv"], inp["ns"], inp["q"], inp["table"],
                                        inp["lens"], inp["L"], sm, tau, split_tokens=split, out=o2["out"],
                                        meter=o2["meter"], raw=o2["raw"], mask_q=o2["mask_q"],
                                        mask_kv=o2["mask_kv"], n_gated=o2["n_gated"])
            torch.cuda.synchronize()
            for x, y in ((c1, c2), (e1, e2)):
                for n, t in x.tensors.items():
                    if t is not None:
                        assert torch.equal(t, y.tensors[n]), (i, n)
            for n in o1:
                assert torch.equal(o1[n], o2[n]), (i, n)
            assert not torch.isnan(o1["out"]).any()
    finally:
        os.environ.pop("WITCERT_FORCE_VALU", None)


def test_noalloc_refuses_oversized_request():
    import torch

    import paper_2607_28699_amd as wc
    from paper_2607_28699_amd import _lib
    wl = W_GQA
    pair, inp = _step_pair(wl, [100], 9, 0)
    c, e = pair[0]
    o = _outputs(1, wl)
    big = 1 << 22   # tokens: with 16-token splits the records exceed the scratch
    table = torch.zeros((1, big // 16), dtype=torch.int32, device="cuda")
    with pytest.raises(wc.WitCertError, match="static scratch"):
        wc.step_metered_decode_gate_noalloc(c, e, inp["nk"], inp["nv"], inp["ns"], inp["q"], table, inp["lens"],
                                            big, 0.1, 0.2, o["out"], o["meter"], o["raw"], o["mask_q"],
                                            o["mask_kv"], split_tokens=64)
    torch.cuda.synchronize()
    assert torch.isnan(o["out"]).all()   # nothing was enqueued
    assert _lib.WC_ESCRATCH == -5
