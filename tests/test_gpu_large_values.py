"""Large value magnitudes on the matrix-core decode paths (GPU).

The PV products take fp16 operands.  The INT8 weight operand p s^v 2^8 carries
2^-ve, ve a running exponent raised whenever a page's largest value scale passes
2^ve, and the bf16 exact cache's values enter as v 2^-ve, ve raised when a page's
largest |v| passes 2^(15 + ve); the accumulators are rescaled by the exact power
of two.  Values from the fp16-safe range up to value scales of 3e4 (|v| about
4e6) give finite outputs that match the oracle; below the old limits (value
scale 1, |v| 32768) the results do not change at all (covered by every other
decode test).  A group-scaled cache puts s 2^-ve into the value operand instead,
with ve starting at -14: group scales from fp16 subnormals to 3e4, mixed inside
one token, give outputs that match the oracle.
"""
import numpy as np
import pytest

import synth
from oracle import decode as odec

from . import support as S

pytestmark = pytest.mark.gpu

W_GQA = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]


def _scaled_case(mode, layer):
    case = S.make_case(W_GQA, [700, 333, 50], permute=True, layer=layer)
    rng = np.random.default_rng(11 + layer)
    for b, v in enumerate(case["v"]):
        amax = np.abs(v).max(axis=2, keepdims=True)
        if mode == "uniform-4e3":
            target = np.full_like(amax, 4e3)
        elif mode == "uniform-5e4":
            target = np.full_like(amax, 5e4)
        else:   # per token and head: value scales 10^U[0, log10 3e4], i.e. |v| up to ~3.8e6
            target = 126.5 * 10.0 ** rng.uniform(0.0, np.log10(3e4), size=amax.shape)
        case["v"][b] = synth.bf16_round(v / np.maximum(amax, 1e-30) * target).astype(np.float32)
    return case


@pytest.mark.parametrize("mode", ["uniform-4e3", "uniform-5e4", "per-token-1-to-3e4"])
def test_large_values_metered_and_exact(mode):
    import torch

    import paper_2607_28699_amd as wc
    S.say(f"[large values] {mode}")
    wl = W_GQA
    case = _scaled_case(mode, {"uniform-4e3": 1, "uniform-5e4": 2}.get(mode, 3))
    cache = S.gpu_cache(case, "int8_dither")
    out, meter, raw = S.gpu_decode(case, cache)
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(raw))
    res = S.oracle_decode(case, S.oracle_write(case, "int8_dither"))
    for b, r in enumerate(res):
        assert S.rel_err(out[b], r["out"]) <= 2e-3, b
        assert np.all(np.abs(raw[b] - r["raw"]) <= 2e-3 * r["raw"]), b
        assert np.all(meter[b] >= r["tv"])
    # the exact bf16 fallback of every KV head over the same values
    exact = S.gpu_cache(case, "bf16")
    q = torch.from_numpy(case["q"]).to("cuda", torch.bfloat16)
    table = torch.from_numpy(case["table"]).cuda()
    lens = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    mkv = torch.ones((len(case["seq_lens"]), wl.n_kv), dtype=torch.uint8, device="cuda")
    o = torch.zeros((len(case["seq_lens"]), wl.n_q, wl.d), dtype=torch.float32, device="cuda")
    wc.exact_decode_attention(exact, q, table, lens, int(case["seq_lens"].max()), 1 / np.sqrt(wl.d), mkv, o)
    torch.cuda.synchronize()
    o = o.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(o))
    for b in range(len(case["seq_lens"])):
        ex = odec.exact_decode(case["q"][b], case["k"][b], case["v"][b], 1 / np.sqrt(wl.d))["out"]
        assert S.rel_err(o[b], ex) <= 2e-3, b


def _group_case(mode, layer):
    """Values whose 32-channel groups carry their own magnitudes: every (token, KV
    head, group) has value scale 10^U[lo, hi] (mixed: 1e-6 .. 3e4 inside one token;
    tiny: 1e-7 .. 1e-5, fp16 subnormal scales included)."""
    case = S.make_case(W_GQA, [700, 333, 50], permute=True, layer=layer)
    rng = np.random.default_rng(23 + layer)
    lo, hi = (-6.0, np.log10(3e4)) if mode == "groups-1e-6-to-3e4" else (-7.0, -5.0)
    for b, v in enumerate(case["v"]):
        n, h, d = v.shape
        vg = v.reshape(n, h, d // 32, 32)
        amax = np.abs(vg).max(axis=3, keepdims=True)
        target = 126.5 * 10.0 ** rng.uniform(lo, hi, size=amax.shape)
        case["v"][b] = synth.bf16_round((vg / np.maximum(amax, 1e-30) * target).reshape(n, h, d)).astype(np.float32)
    return case


@pytest.mark.parametrize("mode", ["groups-1e-6-to-3e4", "groups-tiny"])
def test_group_scaled_values_across_the_fp16_range(mode):
    """Group-scaled INT8 cache on the matrix cores: the value operand s 2^-ve (code + E)
    stays finite and normal for value scales anywhere in the fp16 range (ve starts
    at -14 and rises with the largest scale); outputs match the oracle."""
    S.say(f"[large values] {mode}")
    case = _group_case(mode, 4 if mode == "groups-tiny" else 5)
    refs = S.oracle_write(case, "int8_dither", group_scales=True)
    cache = S.gpu_cache(case, "int8_dither", group_scales=True)
    out, meter, raw = S.gpu_decode(case, cache)
    assert np.all(np.isfinite(out)) and np.all(np.isfinite(raw))
    res = S.oracle_decode(case, refs)
    for b, r in enumerate(res):
        assert S.rel_err(out[b], r["out"]) <= 2e-3, (b, S.rel_err(out[b], r["out"]))
        assert np.all(np.abs(raw[b] - r["raw"]) <= 2e-3 * r["raw"]), b
        assert np.all(meter[b] >= r["tv"])
