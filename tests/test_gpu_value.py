"""GPU parity of the value side and the joint K+V gate (Sec. 3 output bound;
Sec. 4.2 value side and joint event) against the oracle.

* write path: stored value residual (up) and value norm (down) bit-exact, both
  quantized kinds, with and without the key bypass;
* wc_joint_decode_gate on both decode paths and both key tiers: outputs, raw and
  meter as the single-meter calls; meter_v within 1e-5 (fp32 workloads) / 2e-3
  (bf16) of the oracle and never below the true ratio; the joint gate bit-exact
  (decisions within 1e-5 relative of a threshold accepted either way);
* the output bound with the GPU's own meters against exact attention;
* tau_v = inf gives the key-only fused gate bit for bit.
"""
import os

import numpy as np
import pytest

import synth
from oracle import attention
from oracle import bypass as obp
from oracle import decode as odec
from oracle import gate as ogate
from oracle import tierb
from oracle import value as ov

from . import support as S

pytestmark = pytest.mark.gpu

W_TINY = synth.WORKLOADS["tiny-d64-s256"]
W_GQA = synth.WORKLOADS["gqa-28x4-d128-s4k-b8"]
INFORMATIVE = W_GQA.replace(q_scale=1 / 16, n_outliers=0)
DLOC = 1e-6

CASES = [
    ("tiny", W_TINY, [272, 0, 33], "int8_dither", 0),
    ("gqa", W_GQA, [700, 129, 1], "int8_dither", 0),
    ("gqa-informative", INFORMATIVE, [777, 129], "int8_dither", 0),
    ("gqa-bypass4", W_GQA, [333, 18], "int8_dither", 4),
    ("gqa-group16", W_GQA.replace(n_q=32, n_kv=2), [400, 90], "int8_dither", 0),
    ("gqa-fp8", W_GQA, [300, 65], "fp8_raw", 0),
]


def _joint(case, cache, delta, tau, tau_v, force_valu=False):
    import torch

    import paper_2607_28699_amd as wc
    wl = case["wl"]
    q = torch.from_numpy(case["q"]).to("cuda", S.torch_dtype(wl))
    table = torch.from_numpy(case["table"]).cuda()
    lens = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    n = torch.zeros(2, dtype=torch.int32, device="cuda")
    if force_valu:
        os.environ["WITCERT_FORCE_VALU"] = "1"
    try:
        res = wc.joint_decode_gate(cache, q, table, lens, max(int(case["seq_lens"].max()), 1),
                                   1 / np.sqrt(wl.d), tau, tau_v, delta, n_gated=n)
    finally:
        os.environ.pop("WITCERT_FORCE_VALU", None)
    torch.cuda.synchronize()
    out, meter, raw, mv, mq, mk = (x.cpu().numpy() for x in res)
    return out.astype(np.float64), meter, raw, mv, mq, mk, n.cpu().numpy()


def _oracle(case, refs, delta, pairs):
    wl = case["wl"]
    sm = 1 / np.sqrt(wl.d)
    res = []
    for b, c in enumerate(refs):
        if case["seq_lens"][b] == 0:
            res.append(None)
            continue
        q = case["q"][b]
        if delta == 0:
            base = odec.metered_decode(q, c["khat"], c["vhat"], c["kw"], sm, wl.bands, wl.rope_layout)
            cb = base["c"]
        elif pairs is None:
            base = tierb.tierb_decode(q, c["khat"], c["vhat"], c["ks"], sm, delta)
            cb = base["u"]
        else:
            base = obp.tierb_decode(q, c["khat"], c["vhat"], c["ks"], c["ko"], c["chans"], sm, delta)
            cb = base["u"]
        j = ov.joint_decode(q, c["khat"], c["vhat"], cb, c["vr"], c["vn"], sm)
        # the true value-side ratio: ptilde with the true residuals and norms
        g = wl.n_q // wl.n_kv
        vtrue = np.empty(wl.n_q)
        for h in range(wl.n_q):
            kv = h // g
            pt = attention.softmax(attention.logits(q[h], c["khat"][:, kv], sm))
            rho = np.linalg.norm(c["vhat"][:, kv] - case["v"][b][:, kv], axis=1)
            vtrue[h] = (pt @ rho) / np.linalg.norm(case["v"][b][:, kv], axis=1).max()
        j["vtrue"] = vtrue
        j["tv"] = odec.true_tv(q, case["k"][b], c["khat"], sm)
        res.append(j)
    return res


def _check(case, res, out, meter, raw, mv, mq, mk, tau, tau_v):
    wl = case["wl"]
    tol = S.out_tol(wl)
    for b, r in enumerate(res):
        if r is None:
            assert np.all(out[b] == 0) and np.all(meter[b] == 0) and np.all(mv[b] == 0)
            assert np.all(mq[b] == 0) and np.all(mk[b] == 0)
            continue
        assert S.rel_err(out[b], r["out"]) <= tol
        fin = r["raw"] < 1e30
        assert np.all(np.abs(raw[b][fin] - r["raw"][fin]) <= tol * np.maximum(r["raw"][fin], 1e-30))
        assert np.all(np.abs(mv[b] - r["meter_v"]) <= tol * np.maximum(r["meter_v"], 1e-30)), \
            (b, np.max(np.abs(mv[b] - r["meter_v"]) / r["meter_v"]))
        assert np.all(meter[b] >= r["tv"]), "key meter below the true TV"
        assert np.all(mv[b] >= r["vtrue"] * (1 - 1e-6)), "value meter below the true ratio"
        want = ov.joint_gate_q(r["meter"], r["raw"], r["meter_v"], tau, tau_v)
        ties = (np.abs((r["raw"] if tau >= 1 else r["meter"]) - tau) <= 1e-5 * tau) | \
               (np.abs(r["meter_v"] - tau_v) <= 1e-5 * tau_v)
        assert np.array_equal(mq[b].astype(bool)[~ties], want[~ties])
        assert np.array_equal(mk[b].astype(bool), ogate.gate_kv(mq[b].astype(bool)[None], wl.group)[0])


@pytest.mark.parametrize("name,wl,lens,kind,m", CASES)
def test_value_side_write_bitexact(name, wl, lens, kind, m):
    S.say(f"[value-write] {name} kind={kind} m={m}")
    case = S.make_case(wl, lens, permute=True, layer=1)
    pairs = S.case_pairs(case, m) if m else None
    cache = S.gpu_cache(case, kind, pairs=pairs, value_side=True)
    for b, r in enumerate(S.oracle_write(case, kind, pairs)):
        if case["seq_lens"][b] == 0:
            continue
        got = S.read_cache(cache, case["slots"][b])
        assert np.array_equal(got["vr"], r["vr"])
        assert np.array_equal(got["vn"], r["vn"])


@pytest.mark.parametrize("name,wl,lens,kind,m", CASES)
@pytest.mark.parametrize("tier", ["A", "B"])
@pytest.mark.parametrize("path", ["default", "vector"])
def test_joint_decode_parity(name, wl, lens, kind, m, tier, path):
    if path == "vector" and wl.d != 128:
        pytest.skip("head_dim 64 always takes the vector path")
    if tier == "B" and kind != "int8_dither":
        pytest.skip("Tier B is defined for the dithered INT8 cache")
    tau, tau_v = (0.2, 0.05) if "informative" not in name else (0.05, 0.005)
    S.say(f"[joint] {name} tier={tier} path={path} lens={lens}")
    case = S.make_case(wl, lens, permute=True, layer=1)
    pairs = S.case_pairs(case, m) if m else None
    cache = S.gpu_cache(case, kind, pairs=pairs, value_side=True)
    delta = 0.0 if tier == "A" else DLOC
    out, meter, raw, mv, mq, mk, n = _joint(case, cache, delta, tau, tau_v, force_valu=(path == "vector"))
    res = _oracle(case, S.oracle_write(case, kind, pairs), delta, pairs)
    _check(case, res, out, meter, raw, mv, mq, mk, tau, tau_v)
    assert n[0] == mq.sum() and n[1] == mk.sum()


def test_output_bound_with_gpu_meters():
    """||y - yhat|| <= (2 meter + meter_v) max_t ||v_t|| with the GPU's meters and output."""
    S.say("[joint] output bound with GPU meters")
    for wl in (INFORMATIVE, W_GQA):
        case = S.make_case(wl, [600, 77], permute=True, layer=3)
        cache = S.gpu_cache(case, "int8_dither", value_side=True)
        out, meter, raw, mv, mq, mk, _ = _joint(case, cache, 0.0, 0.2, 0.05)
        sm = 1 / np.sqrt(wl.d)
        for b in range(2):
            ex = odec.exact_decode(case["q"][b], case["k"][b], case["v"][b], sm)["out"]
            g = wl.n_q // wl.n_kv
            for h in range(wl.n_q):
                vmax = np.linalg.norm(case["v"][b][:, h // g], axis=1).max()
                err = np.linalg.norm(ex[h] - out[b][h])
                assert err <= (2 * meter[b][h] + mv[b][h]) * vmax * (1 + 1e-3), (b, h)


def test_tau_v_infinite_is_the_key_gate():
    import torch

    import paper_2607_28699_amd as wc
    S.say("[joint] tau_v = inf")
    wl = INFORMATIVE
    case = S.make_case(wl, [500, 0, 129], permute=True, layer=2)
    cache = S.gpu_cache(case, "int8_dither", value_side=True)
    q = torch.from_numpy(case["q"]).to("cuda", S.torch_dtype(wl))
    table = torch.from_numpy(case["table"]).cuda()
    sl = torch.from_numpy(case["seq_lens"].astype(np.int32)).cuda()
    L = int(case["seq_lens"].max())
    sm = 1 / np.sqrt(wl.d)
    o1, m1, r1, mq1, mk1 = wc.metered_decode_gate(cache, q, table, sl, L, sm, 0.05)
    o2, m2, r2, _, mq2, mk2 = wc.joint_decode_gate(cache, q, table, sl, L, sm, 0.05, float("inf"))
    torch.cuda.synchronize()
    for a_, b_ in ((o1, o2), (m1, m2), (r1, r2), (mq1, mq2), (mk1, mk2)):
        assert torch.equal(a_, b_)
