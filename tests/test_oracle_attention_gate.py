"""Pins of the oracle's attention, gate and composed decode (CPU).

* attention equals torch's float64 scaled_dot_product_attention (a library routine);
* TV is a metric bounded by 1;
* gate: strict ">", certified meter below tau = 1, raw risk score from tau = 1 on,
  any-of-G routing; the fallback swaps exactly the routed groups;
* composed decode: the meter is never below the true TV (Theorems black-box
  logit bound + sound replacement) for dithered INT8 and raw fp8 caches, both in
  the informative and in the saturated regime of the synthetic workloads; an
  exact cache (zero witness) gives meter 0.
"""
import numpy as np
import pytest
import torch

import synth
from oracle import attention, decode, gate


def test_attention_matches_torch_sdpa_float64():
    rng = np.random.default_rng(0)
    for S, d in ((1, 64), (17, 64), (300, 128)):
        q = rng.standard_normal((7, d)) * 3
        k = rng.standard_normal((S, d))
        v = rng.standard_normal((S, d))
        p, y = attention.attend(q, k, v, 1 / np.sqrt(d))
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.from_numpy(q)[None, :, None], torch.from_numpy(k)[None, None].expand(1, 7, S, d),
            torch.from_numpy(v)[None, None].expand(1, 7, S, d))[0, :, 0].numpy()
        assert np.allclose(y, ref, rtol=1e-12, atol=1e-12)
        assert np.allclose(p.sum(-1), 1)


def test_tv_properties():
    rng = np.random.default_rng(1)
    a = rng.dirichlet(np.ones(20), size=50)
    b = rng.dirichlet(np.ones(20), size=50)
    t = attention.tv(a, b)
    assert np.all((t >= 0) & (t <= 1))
    assert np.allclose(t, attention.tv(b, a))
    assert np.all(attention.tv(a, a) == 0)
    one_hot = np.eye(20)
    assert np.isclose(attention.tv(one_hot[0], one_hot[1]), 1.0)


def test_gate_thresholds_and_routing():
    meter = np.array([[0.2, 0.2000001, 1.0, 0.0]])
    raw = np.array([[0.2, 0.2000001, 3.0, 0.0]])
    assert gate.gate_q(meter, raw, 0.2).tolist() == [[False, True, True, False]]
    # tau >= 1: raw score (risk-ranked); the saturated meter can never exceed 1
    assert gate.gate_q(meter, raw, 1.0).tolist() == [[False, False, True, False]]
    assert gate.gate_q(meter, raw, 3.0).tolist() == [[False, False, False, False]]
    assert gate.gate_q(meter, np.array([[0, 0, np.inf, 0]]), 5.0).tolist() == [[False, False, True, False]]
    mq = np.array([[False, False, True, False, False, False]])
    assert gate.gate_kv(mq, 3).tolist() == [[True, False]]
    assert gate.gate_kv(mq, 2).tolist() == [[False, True, False]]
    oc = np.zeros((1, 6, 4))
    oe = np.ones((1, 6, 4))
    f = gate.apply_fallback(oc, oe, np.array([[True, False]]), 3)
    assert f[0, :3].min() == 1 and f[0, 3:].max() == 0


def _cell(wl, S, layer=0, seq=0, kind="int8_dither"):
    k = np.stack([synth.gen_kv(wl, layer, h, seq, "k", np.arange(S)) for h in range(wl.n_kv)], 1)
    v = np.stack([synth.gen_kv(wl, layer, h, seq, "v", np.arange(S)) for h in range(wl.n_kv)], 1)
    q = synth.gen_q(wl, layer, seq, 0, S - 1)
    cache = decode.write_cache(kind, k, v, np.arange(S) + 1000, layer, wl.philox_seed(),
                               wl.bands, wl.rope_layout)
    return q, k, v, cache


@pytest.mark.parametrize("kind", ["int8_dither", "fp8_raw"])
@pytest.mark.parametrize("qscale,outliers", [(1.0, 2), (1 / 16, 0), (1 / 64, 0)])
def test_meter_never_below_true_tv(kind, qscale, outliers):
    base = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]
    wl = base.replace(q_scale=qscale, n_outliers=outliers)
    S = 300
    for layer in range(2):
        q, k, v, cache = _cell(wl, S, layer=layer, kind=kind)
        sm = 1 / np.sqrt(wl.d)
        res = decode.metered_decode(q, cache["khat"], cache["vhat"], cache["kw"], sm, wl.bands)
        t = decode.true_tv(q, k, cache["khat"], sm)
        assert np.all(res["raw"] >= t)
        assert np.all(res["meter"] >= t)
        if qscale < 1:
            assert np.all(res["raw"] < 1)           # informative regime really is informative


def test_exact_cache_has_zero_meter_and_exact_output():
    wl = synth.WORKLOADS["tiny-d64-s256"]
    q, k, v, cache = _cell(wl, 64, kind="bf16")
    sm = 1 / np.sqrt(wl.d)
    res = decode.metered_decode(q, cache["khat"], cache["vhat"], cache["kw"], sm, wl.bands)
    assert np.all(res["raw"] == 0) and np.all(res["meter"] == 0)
    ex = decode.exact_decode(q, k, v, sm)
    assert np.allclose(res["out"], ex["out"], rtol=0, atol=0)
