"""Pins of the value-side oracle (Sec. 3 output bound; Sec. 4.2 value side and
joint event) against the mathematics.

* The output bound ||y - yhat|| <= 2 TV max_t ||v_t|| + sum_t ptilde_t rho_t holds
  with the true quantities on random cells of both quantized caches, in the
  informative and the saturated regime, and in units of the largest value norm
  with the stored meters (2 meter_K + meter_V).
* It is attained: two exact values v, -v with moved attention give equality in
  the first term (so TV alone, without the factor 2, is violated), one token with
  a value error gives equality in the second.
* The stored residual is never below the true one and the stored norm never
  above the true one (round-down brute force over fp16), so the value meter is
  never below the true ratio; its special cases (0/0, x/0).
* Joint gate: routed exactly when pass_K and pass_V do not both hold.
"""
import numpy as np

from oracle import attention, decode as odec, fpformats as fp, gate as ogate, value as ov

ALL_F16 = np.sort(np.arange(0, 0x7C00, dtype=np.uint16).view(np.float16).astype(np.float64))


def test_f16_round_down_is_largest_fp16_not_above():
    rng = np.random.default_rng(30)
    x = np.concatenate([
        np.exp(rng.uniform(np.log(1e-9), np.log(6e4), 20000)),
        ALL_F16[1:2000],
        ALL_F16[1:2000] * (1 - 1e-9),
        [0.0, 65504.0, 1e5],
    ])
    got = fp.f16_round_down(x)
    idx = np.searchsorted(ALL_F16, np.minimum(x, 65504.0), side="right") - 1   # last value <= x
    assert np.array_equal(got, ALL_F16[idx])


def _cells(rng, kind, q_scale):
    S, n_kv, d = 120, 2, 32
    k = rng.normal(size=(S, n_kv, d)) * rng.uniform(0.5, 3, size=(n_kv, d))
    v = rng.normal(size=(S, n_kv, d)) * rng.uniform(0.5, 3, size=(n_kv, d))
    q = rng.normal(size=(6, d)) * q_scale
    c = odec.write_cache(kind, k, v, np.arange(S), 0, int(rng.integers(1 << 30)), 4)
    return q, k, v, c


def test_output_bound_holds():
    rng = np.random.default_rng(31)
    sm = 1 / np.sqrt(32)
    for kind in ("int8_dither", "fp8_raw"):
        for q_scale in (1.0, 1 / 8):
            for _ in range(6):
                q, k, v, c = _cells(rng, kind, q_scale)
                ex = odec.exact_decode(q, k, v, sm)
                res = odec.metered_decode(q, c["khat"], c["vhat"], c["kw"], sm, 4)
                tv = odec.true_tv(q, k, c["khat"], sm)
                for h in range(q.shape[0]):
                    kv = h // 3
                    p_t = attention.softmax(attention.logits(q[h], c["khat"][:, kv], sm))
                    vmax = np.max(np.linalg.norm(v[:, kv], axis=1))
                    rho = np.linalg.norm(c["vhat"][:, kv] - v[:, kv], axis=1)
                    err = np.linalg.norm(ex["out"][h] - res["out"][h])
                    assert err <= 2 * tv[h] * vmax + p_t @ rho + 1e-12
                    mv = ov.value_meter(p_t, c["vr"][:, kv], c["vn"][:, kv])
                    assert err <= ov.output_bound_units(res["meter"][h], mv) * vmax * (1 + 1e-12)


def test_output_bound_is_attained():
    a = np.array([3.0, -4.0])          # ||a|| = 5
    v = np.stack([a, -a])
    p = np.array([0.8, 0.2])
    pt = np.array([0.3, 0.7])
    err = np.linalg.norm(p @ v - pt @ v)      # exact values: rho = 0
    tv = attention.tv(p, pt)
    assert np.isclose(err, 2 * tv * 5.0)
    assert err > tv * 5.0                     # the factor 2 is needed
    assert np.isclose(err, ov.output_bound_units(tv, 0.0) * 5.0)   # and the oracle's form is tight
    r = np.array([0.25, 0.5])                 # one token: the whole error is its value error
    assert np.isclose(np.linalg.norm(np.array([1.0]) @ (a[None] + r[None]) - a), 1.0 * np.linalg.norm(r))


def test_stored_value_quantities_and_meter_are_upper_bounds():
    rng = np.random.default_rng(32)
    for kind in ("int8_dither", "fp8_raw"):
        q, k, v, c = _cells(rng, kind, 1.0)
        rho = np.linalg.norm(c["vhat"] - v, axis=-1)
        nrm = np.linalg.norm(v, axis=-1)
        assert np.all(c["vr"] >= rho) and np.all(c["vr"] <= rho * (1 + 2.0 ** -10) + 2.0 ** -24)
        assert np.all(c["vn"] <= nrm) and np.all(c["vn"] >= nrm * (1 - 2.0 ** -10))
        for kv in range(2):
            pt = rng.dirichlet(np.ones(v.shape[0]))
            true = (pt @ rho[:, kv]) / nrm[:, kv].max()
            assert ov.value_meter(pt, c["vr"][:, kv], c["vn"][:, kv]) >= true
    assert ov.value_meter(np.array([1.0]), np.array([0.0]), np.array([0.0])) == 0.0
    assert ov.value_meter(np.array([1.0]), np.array([1e-3]), np.array([0.0])) == np.inf
    # an exact value cache (bf16 kind stores no value side; a zero residual gives 0)
    assert ov.value_meter(np.array([0.5, 0.5]), np.zeros(2), np.array([1.0, 2.0])) == 0.0


def test_joint_gate():
    mk = np.array([0.1, 0.3, 0.1, 0.3, 1.0])
    raw = np.array([0.1, 0.3, 0.1, 0.3, 7.0])
    mv = np.array([0.01, 0.01, 0.06, 0.06, 0.0])
    got = ov.joint_gate_q(mk, raw, mv, 0.2, 0.05)
    assert list(got) == [False, True, True, True, True]
    # tau_K >= 1 compares the raw key-side score, as the key-side gate alone does
    assert list(ov.joint_gate_q(mk, raw, mv * 0, 5.0, 0.05)) == list(ogate.gate_q(mk, raw, 5.0))
    # the joint decode agrees with its parts
    rng = np.random.default_rng(33)
    q, k, v, c = _cells(rng, "int8_dither", 1 / 4)
    sm = 1 / np.sqrt(32)
    ref = odec.metered_decode(q, c["khat"], c["vhat"], c["kw"], sm, 4)
    j = ov.joint_decode(q, c["khat"], c["vhat"], ref["c"], c["vr"], c["vn"], sm)
    assert np.array_equal(j["out"], ref["out"]) and np.array_equal(j["raw"], ref["raw"])
    for h in range(q.shape[0]):
        assert j["meter_v"][h] == ov.value_meter(ref["ptilde"][h], c["vr"][:, h // 3], c["vn"][:, h // 3])
