"""Pins of the block-repair oracle (Sec. 6.3, block-level paging).

* The shares of the blocks add up to A - 1 (block decomposability), and when the
  exact logits of the repaired blocks equal the compressed ones the repaired
  certificate is A - (sum of their shares) exactly: the paper's statement.
* Repairing every block gives the exact output and raw 0.
* After any repair the certificate still bounds the true TV between the exact
  distribution and the repaired one.
* The order equals a brute-force sort, and the stop rule is minimal: the first
  n - 1 blocks of the order do not pass, the first n do.
"""
import numpy as np

from oracle import attention, decode as odec, meter as mt, repair as orep


def _case(rng, S=300, d=32, G=3, q_scale=0.5):
    k = rng.normal(size=(S, d)) * rng.uniform(0.5, 3, size=d)
    v = rng.normal(size=(S, d))
    c = odec.write_cache("int8_dither", k[:, None], v[:, None], np.arange(S), 0, int(rng.integers(1 << 30)), 4)
    q = rng.normal(size=(G, d)) * q_scale
    cb = np.stack([mt.logit_bound(q[h], c["kw"][:, 0], 1 / np.sqrt(d), 4) for h in range(G)])
    return q, k, v, c["khat"][:, 0], c["vhat"][:, 0], cb


def test_shares_sum_and_decomposability():
    rng = np.random.default_rng(40)
    q, k, v, kh, vh, cb = _case(rng)
    sm = 1 / np.sqrt(q.shape[1])
    ranges = orep.block_ranges(kh.shape[0], 64)
    assert ranges[-1] == (256, 300) and len(ranges) == 5
    for h in range(q.shape[0]):
        z = attention.logits(q[h], kh, sm)
        p = attention.softmax(z)
        sh = orep.block_shares(p, cb[h], ranges)
        assert np.isclose(sh.sum(), mt.a_minus_one_logits(z, cb[h]), rtol=1e-12)
    # exact logits equal to the compressed ones on the repaired blocks: A' = A - shares
    for R in ([0], [1, 3], [4], [0, 1, 2, 3]):
        st = orep.repaired_state(q, kh, vh, kh, vh, cb, R, ranges, sm)
        for h in range(q.shape[0]):
            z = attention.logits(q[h], kh, sm)
            sh = orep.block_shares(attention.softmax(z), cb[h], ranges)
            a = 1 + mt.a_minus_one_logits(z, cb[h])
            a_rep = np.sqrt(1 + 2 * st["raw"][h])     # A' from raw' = (A'^2 - 1)/2
            assert np.isclose(a_rep, a - sh[R].sum(), rtol=1e-10)


def test_full_repair_is_exact_and_repair_stays_sound():
    rng = np.random.default_rng(41)
    q, k, v, kh, vh, cb = _case(rng)
    sm = 1 / np.sqrt(q.shape[1])
    ranges = orep.block_ranges(kh.shape[0], 64)
    st = orep.repaired_state(q, kh, vh, k, v, cb, range(len(ranges)), ranges, sm)
    ex = np.stack([attention.attend(q[h], k, v, sm)[1] for h in range(q.shape[0])])
    assert np.allclose(st["out"], ex, rtol=0, atol=1e-12) and np.all(st["raw"] == 0)
    for R in ([0], [2, 4], [1, 2, 3]):
        st = orep.repaired_state(q, kh, vh, k, v, cb, R, ranges, sm)
        kk = np.where(st["repaired"][:, None], k, kh)
        for h in range(q.shape[0]):
            p = attention.softmax(attention.logits(q[h], k, sm))
            pr = attention.softmax(attention.logits(q[h], kk, sm))
            assert st["raw"][h] >= attention.tv(p, pr)


def test_order_and_minimal_stop():
    rng = np.random.default_rng(42)
    for trial in range(10):
        q, k, v, kh, vh, cb = _case(rng, q_scale=rng.uniform(0.2, 1.0))
        sm = 1 / np.sqrt(q.shape[1])
        ranges = orep.block_ranges(kh.shape[0], 32)
        res = orep.block_repair(q, kh, vh, k, v, cb, ranges, sm, 0.05, len(ranges))
        tot = res["shares"].sum(axis=0)
        assert np.all(np.diff(tot[res["order"]]) <= 0)
        n = res["n_blocks"]
        assert n >= 1
        st = orep.repaired_state(q, kh, vh, k, v, cb, res["order"][:n], ranges, sm)
        assert np.all(st["meter"] <= 0.05) and np.array_equal(st["out"], res["out"])
        if n > 1:
            prev = orep.repaired_state(q, kh, vh, k, v, cb, res["order"][:n - 1], ranges, sm)
            assert np.any(prev["meter"] > 0.05)
    # a budget too small to pass leaves the head to the whole-head fallback
    q, k, v, kh, vh, cb = _case(np.random.default_rng(43), q_scale=2.0)
    res = orep.block_repair(q, kh, vh, k, v, cb, orep.block_ranges(300, 32), 1 / np.sqrt(32), 1e-6, 2)
    assert res["n_blocks"] == -1


def test_paper_blocks():
    """Sec. 6.3's blocks: S = 32768 tokens give n_b = 128 blocks of 256 tokens; any
    length is covered once by consecutive blocks, only the last one shorter, and
    the partition depends on nothing but the sequence length."""
    bl = orep.paper_blocks(32768)
    assert len(bl) == 128 and all(t1 - t0 == 256 for t0, t1 in bl)
    for S in (1, 255, 256, 257, 300, 4106, 32770, 131073):
        bl = orep.paper_blocks(S)
        assert len(bl) == -(-S // 256)
        covered = np.zeros(S, dtype=int)
        for j, (t0, t1) in enumerate(bl):
            assert t0 == 256 * j and 0 < t1 - t0 <= 256
            covered[t0:t1] += 1
        assert np.all(covered == 1) and bl[-1][1] == S
        assert all(t1 - t0 == 256 for t0, t1 in bl[:-1])
