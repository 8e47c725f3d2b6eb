"""GPU parity of the Tier-B certified decode (Sec. 4.2, Tier B) against the oracle.

Same bar as the Tier-A decode: outputs within 1e-5 (fp32 workloads) / 2e-3 (bf16)
of the oracle, raw and meter relative to the oracle's Tier-B values, the meter
above the true TV (at delta_loc = 1e-6 a violation has probability <= 1e-6 per
call); both decode paths; a cache without a witness; and, on the informative
family, the Tier-B raw below the Tier-A raw on the same cache.
"""
import os

import numpy as np
import pytest

import synth
from oracle import decode as odec
from oracle import tierb

from . import support as S

pytestmark = pytest.mark.gpu

W_TINY = synth.WORKLOADS["tiny-d64-s256"]
W_GQA = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]
INFORMATIVE = W_GQA.replace(q_scale=1 / 16, n_outliers=0)
DLOC = 1e-6

CASES = [
    ("tiny", W_TINY, [272, 0, 33], 0),
    ("gqa", W_GQA, [700, 129, 1], 0),
    ("gqa-split64", W_GQA, [300, 64], 64),
    ("gqa-informative", INFORMATIVE, [777, 129], 128),
    ("gqa-group16", W_GQA.replace(n_q=32, n_kv=2), [400, 90], 0),
]


def _run(case, cache, split=0, force_valu=False):
    import torch

    import paper_2607_28699_amd as wc
    wl = case["wl"]
    q = torch.from_numpy(case["q"]).to("cuda", S.torch_dtype(wl))
    table = torch.from_numpy(case["table"]).cuda()
    lens = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    if force_valu:
        os.environ["WITCERT_FORCE_VALU"] = "1"
    try:
        out, meter, raw = wc.tierb_decode_attention(cache, q, table, lens, max(int(case["seq_lens"].max()), 1),
                                                    1 / np.sqrt(wl.d), DLOC, split_tokens=split)
    finally:
        os.environ.pop("WITCERT_FORCE_VALU", None)
    torch.cuda.synchronize()
    return out.cpu().numpy().astype(np.float64), meter.cpu().numpy(), raw.cpu().numpy()


def _oracle(case):
    wl = case["wl"]
    res = []
    for b, c in enumerate(S.oracle_write(case, "int8_dither")):
        if case["seq_lens"][b] == 0:
            res.append(None)
            continue
        r = tierb.tierb_decode(case["q"][b], c["khat"], c["vhat"], c["ks"], 1 / np.sqrt(wl.d), DLOC)
        r["tv"] = odec.true_tv(case["q"][b], case["k"][b], c["khat"], 1 / np.sqrt(wl.d))
        res.append(r)
    return res


def _check(case, res, out, meter, raw):
    tol = S.out_tol(case["wl"])
    for b, r in enumerate(res):
        if r is None:
            assert np.all(out[b] == 0) and np.all(meter[b] == 0) and np.all(raw[b] == 0)
            continue
        assert S.rel_err(out[b], r["out"]) <= tol, (b, S.rel_err(out[b], r["out"]))
        fin = r["raw"] < 1e30
        rr = np.abs(raw[b][fin] - r["raw"][fin]) / np.maximum(r["raw"][fin], 1e-30)
        assert np.all(rr <= tol), (b, rr.max())
        assert np.all(np.abs(meter[b] - r["meter"]) <= tol * np.maximum(r["meter"], 1e-30))
        assert np.all(meter[b] >= r["tv"]), "Tier-B meter below the true TV"


@pytest.mark.parametrize("name,wl,lens,split", CASES)
@pytest.mark.parametrize("path", ["default", "vector"])
def test_tierb_parity(name, wl, lens, split, path):
    if path == "vector" and wl.d != 128:
        pytest.skip("head_dim 64 always takes the vector path")
    S.say(f"[tierb] {name} path={path} lens={lens} split={split}")
    case = S.make_case(wl, lens, permute=True, layer=2)
    cache = S.gpu_cache(case, "int8_dither")
    out, meter, raw = _run(case, cache, split, force_valu=(path == "vector"))
    _check(case, _oracle(case), out, meter, raw)


def test_tierb_needs_no_witness_and_is_tighter():
    S.say("[tierb] no witness; tighter than tier A on the informative family")
    case = S.make_case(INFORMATIVE, [900, 257], permute=True, layer=1)
    cache = S.gpu_cache(case, "int8_dither")
    _, _, raw_a = S.gpu_decode(case, cache)
    out1, meter1, raw1 = _run(case, cache)
    cache.tensors["k_witness"] = None          # Tier B reads no witness
    out2, meter2, raw2 = _run(case, cache)
    assert np.array_equal(out1, out2) and np.array_equal(raw1, raw2)
    assert np.all(raw1 < raw_a)
    _check(case, _oracle(case), out2, meter2, raw2)
