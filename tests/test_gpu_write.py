"""GPU parity of the write path against the oracle: codes, scales and witness
bit-exact (the witness is the fp16 round-up of the float64 band norm)."""
import numpy as np
import pytest

import synth
from oracle import decode as odec
from oracle import fpformats as ofp
from oracle import quantizer as oq

from . import support as S

pytestmark = pytest.mark.gpu

CASES = [
    ("tiny-d64-s256", [37]),
    ("tiny-d64-s256", [256, 1, 17]),
    ("gqa-28x4-d128-s4k-b8", [300, 45]),
]


@pytest.mark.parametrize("name,lens", CASES)
@pytest.mark.parametrize("layout", ["half", "interleaved"])
def test_int8_write_bitexact(name, lens, layout):
    wl = synth.WORKLOADS[name].replace(rope_layout=layout)
    S.say(f"[write-int8] {name} lens={lens} layout={layout}")
    case = S.make_case(wl, lens, permute=True, layer=3)
    cache = S.gpu_cache(case, "int8_dither")
    ref = S.oracle_write(case, "int8_dither")
    for b, r in enumerate(ref):
        got = S.read_cache(cache, case["slots"][b])
        assert np.array_equal(got["k"].astype(np.int64), r["kcode"])
        assert np.array_equal(got["v"].astype(np.int64), r["vcode"])
        assert np.array_equal(got["ks"], r["ks"])
        assert np.array_equal(got["vs"], r["vs"])
        assert np.array_equal(got["kw"], r["kw"])
        # the stored witness bounds the residual of the stored reconstruction
        assert np.all(got["kw"] >= oq.band_norms(r["khat"] - case["k"][b], wl.bands, layout) * (1 - 1e-12))


@pytest.mark.parametrize("name,lens", CASES[1:])
def test_fp8_write_bitexact(name, lens):
    wl = synth.WORKLOADS[name]
    S.say(f"[write-fp8] {name} lens={lens}")
    case = S.make_case(wl, lens, permute=True, layer=1)
    cache = S.gpu_cache(case, "fp8_raw")
    ref = S.oracle_write(case, "fp8_raw")
    for b, r in enumerate(ref):
        got = S.read_cache(cache, case["slots"][b])
        assert np.array_equal(got["k"], ofp.e4m3_encode(case["k"][b]))
        assert np.array_equal(got["v"], ofp.e4m3_encode(case["v"][b]))
        assert np.array_equal(got["kw"], r["kw"])


def test_fp8_cast_saturates_and_keeps_sign():
    import torch

    import paper_2607_28699_amd as wc
    wl = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"].replace(n_kv=1, n_q=7, dtype="f32")
    S.say("[write-fp8] extremes")
    x = np.zeros((4, 1, 128), np.float32)
    x[0, 0, :4] = [448.0, -448.0, 447.9, -1e-12]
    x[1, 0, :4] = [600.0, -2000.0, 2.0 ** -9, 2.0 ** -10]    # beyond 448: saturating reading
    x[2, 0] = np.linspace(-300, 300, 128)
    x[3, 0] = np.linspace(-1e-3, 1e-3, 128)
    c = wc.PagedCache("fp8_raw", 1, 1, 128, 8)
    wc.quantize_write(c, torch.from_numpy(x).cuda(), torch.from_numpy(x).cuda(),
                      torch.arange(4, dtype=torch.int64).cuda())
    torch.cuda.synchronize()
    got = S.read_cache(c, np.arange(4))
    assert np.array_equal(got["k"][:, 0], ofp.e4m3_encode(x[:, 0]))
    _ = wl


def test_bf16_write_is_exact_copy():
    import torch
    wl = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]
    S.say("[write-bf16]")
    case = S.make_case(wl, [50, 7], permute=True)
    cache = S.gpu_cache(case, "bf16")
    for b in range(2):
        got = S.read_cache(cache, case["slots"][b])
        want_k = synth.to_bf16_bits(case["k"][b]).view(np.int16)
        want_v = synth.to_bf16_bits(case["v"][b]).view(np.int16)
        assert np.array_equal(got["k"], want_k) and np.array_equal(got["v"], want_v)
    _ = torch


def test_zero_token_has_zero_scale_codes_and_witness():
    import torch

    import paper_2607_28699_amd as wc
    S.say("[write-int8] zero rows")
    x = np.zeros((3, 2, 128), np.float32)
    x[1, 1, 5] = 1.0
    c = wc.PagedCache("int8_dither", 1, 2, 128, 8, seed=5)
    wc.quantize_write(c, torch.from_numpy(x).cuda(), torch.from_numpy(x).cuda(),
                      torch.tensor([3, 9, 15], dtype=torch.int64).cuda())
    torch.cuda.synchronize()
    got = S.read_cache(c, np.array([3, 9, 15]))
    assert np.all(got["ks"][0] == 0) and np.all(got["k"][0] == 0) and np.all(got["kw"][0] == 0)
    ref = odec.write_cache("int8_dither", x[1:2], x[1:2], np.array([9]), 0, 5, 8)
    assert np.array_equal(got["k"][1:2].astype(np.int64), ref["kcode"])
    assert np.array_equal(got["kw"][1:2], ref["kw"])


@pytest.mark.parametrize("dts", [("f32", "f32"), ("bf16", "f32"), ("f32", "f16"), ("bf16", "bf16")])
@pytest.mark.parametrize("layout", ["half", "interleaved"])
def test_blackbox_witness(dts, layout):
    import torch

    import paper_2607_28699_amd as wc
    S.say(f"[witness] {dts} {layout}")
    rng = np.random.default_rng(3)
    tmap = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
    x = torch.from_numpy(rng.standard_normal((333, 128)).astype(np.float32) * 3).to(tmap[dts[0]])
    xh = (x.float() + torch.from_numpy(rng.standard_normal((333, 128)).astype(np.float32)) * 0.05).to(tmap[dts[1]])
    w = wc.witness(x.cuda(), xh.cuda(), 16, layout)
    torch.cuda.synchronize()
    ref = oq.witness(x.double().numpy(), xh.double().numpy(), 16, layout)
    got = w.cpu().double().numpy()
    assert np.array_equal(got, ref)


def test_witness_round_up_at_fp16_boundaries():
    """Band norms at and next to fp16 values round up as in the oracle: norms that
    are fp16 values, one part in 2^20 above and below them, norms within 2^-50 of a
    square (where the kernels take the float64 root), zero, fp16 subnormals, tiny
    residuals whose squares leave the float32 range, and norms past 65504."""
    import torch

    import paper_2607_28699_amd as wc
    d, B = 128, 16
    band = oq.band_index(d, B, "half")
    chans = [np.flatnonzero(band == b) for b in range(B)]
    rng = np.random.default_rng(11)
    fp16 = np.unique(np.abs(rng.standard_normal(200).astype(np.float16)).astype(np.float64))
    special = [1.0, 1.5, 2.0 ** -14, 2.0 ** -24, 3 * 2.0 ** -24, 2048.0, 65504.0]
    cases = []   # the nonzero residuals of one band
    for h in list(fp16[fp16 > 0][:60]) + special:
        cases += [(h,), (h * (1 + 2.0 ** -20),), (h * (1 - 2.0 ** -20),)]
    cases += [(1.0, 2.0 ** -25), (2.0, 2.0 ** -24), (1 - 2.0 ** -24,), (0.0,), (2.0 ** -30,), (2.0 ** -70,),
              (2.0 ** -100,), (3.0, 4.0), (70000.0,), (65504.0, 256.0), (65504.0 * (1 + 2.0 ** -20),)]
    rows = (len(cases) + B - 1) // B
    xh = np.zeros((rows, d), np.float32)
    for i, c in enumerate(cases):
        r, b = divmod(i, B)
        for j, val in enumerate(c):
            xh[r, chans[b][j]] = np.float32(val)
    x = np.zeros_like(xh)
    S.say(f"[witness] fp16 boundaries: {len(cases)} bands")
    w = wc.witness(torch.from_numpy(x).cuda(), torch.from_numpy(xh).cuda(), B, "half")
    torch.cuda.synchronize()
    ref = oq.witness(x.astype(np.float64), xh.astype(np.float64), B, "half")
    got = w.cpu().double().numpy()
    assert np.array_equal(got, ref), np.argwhere(got != ref)[:8]



def _codes_next_to_half(x, xi):
    """Rows x [n, d] (float32) whose channels 1.. are moved, where possible, to the
    float32 next to (sign(xi)/2 - xi) * s at which rounding x * inv to fp32 before
    adding the dither xi gives code 0 and one fused multiply-add would give +-1
    (the scaled value is then below 1/2 in magnitude, where its fp32 spacing is finer
    than that of the sum); channel 0 holds the row's amax, so the scale is the
    row's.  Returns the rows and the number of channels where the two roundings differ."""
    x = np.array(x, dtype=np.float32)
    n, d = x.shape
    s = oq.int8_scale(x)
    inv = (1.0 / s).astype(np.float32).astype(np.float64)
    split = 0
    steps = np.arange(-64, 65)
    for r in range(n):
        for c in range(1, d):
            x0 = np.float32((np.sign(xi[r, c]) * 0.5 - xi[r, c]) / inv[r])
            cand = (x0 + steps.astype(np.float32) * np.spacing(np.abs(x0))).astype(np.float32)
            y = cand.astype(np.float64) * inv[r]                 # exact product
            unfused = np.rint(np.float32(np.float32(y) + np.float32(xi[r, c])))
            fused = np.rint(np.float32(y + xi[r, c]))            # y + xi is exact in float64
            hit = np.flatnonzero(unfused != fused)
            if len(hit):
                x[r, c] = cand[hit[0]]
                split += 1
    return x, split


def test_int8_code_decided_before_the_dither_is_added():
    """The code 0 / +-1 of a channel whose scaled value x / s lies just off
    +-1/2 - xi is decided as the quantizer defines it -- x / s rounded to fp32, then
    the dither added -- not by one fused multiply-add, which there gives +-1 where
    the definition gives 0: keys and values built so that the two roundings part in
    about a third of the channels are written bit-exactly as in the oracle."""
    from oracle.philox import dither_values

    wl = synth.WORKLOADS["tiny-d64-s256"]
    S.say("[write-int8] codes next to +-1/2")
    case = S.make_case(wl, [48], permute=True, layer=3)
    xi = dither_values(case["slots"][0], wl.d, 3, 0, wl.philox_seed())
    split = 0
    for name in ("k", "v"):
        rows = np.clip(case[name][0][:, 0, :], -2.5, 2.5)
        rows[:, 0] = 3.0
        rows, n_split = _codes_next_to_half(rows, xi)
        case[name][0][:, 0, :] = rows
        split += n_split
    assert split > 48 * wl.d // 2, split   # a third of the channels sit where the two roundings part
    cache = S.gpu_cache(case, "int8_dither")
    ref = S.oracle_write(case, "int8_dither")[0]
    got = S.read_cache(cache, case["slots"][0])
    assert np.array_equal(got["k"].astype(np.int64), ref["kcode"]), np.argwhere(got["k"] != ref["kcode"])[:8]
    assert np.array_equal(got["v"].astype(np.int64), ref["vcode"]), np.argwhere(got["v"] != ref["vcode"])[:8]
    assert np.array_equal(got["ks"], ref["ks"]) and np.array_equal(got["kw"], ref["kw"])
