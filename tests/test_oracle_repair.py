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


def test_split_blocks_partition():
    """The decode's blocks: four page-aligned parts per split, covering [0, S) once;
    quarters of a full split; a last split divided as evenly as pages allow."""
    for S, st in ((300, 256), (4106, 256), (32770, 1088), (600, 3904), (1, 256), (16, 64), (33, 64)):
        bl = orep.split_blocks(S, st)
        assert len(bl) == 4 * (-(-S // st))
        covered = np.zeros(S, dtype=int)
        prev = 0
        for t0, t1 in bl:
            assert t0 == prev and t0 <= t1          # in order, contiguous, possibly empty
            covered[t0:t1] += 1
            prev = t1
            if t1 > t0:
                assert t0 % 16 == 0                 # page-aligned starts
        assert prev == S and np.all(covered == 1)
        for j in range(S // st):                    # full splits: exact quarters
            assert bl[4 * j:4 * j + 4] == [(j * st + w * st // 4, j * st + (w + 1) * st // 4) for w in range(4)]
    # a 600-token sequence in one 3904-token split: 38 pages -> 10, 10, 10, 8 pages
    assert [t1 - t0 for t0, t1 in orep.split_blocks(600, 3904)] == [160, 160, 160, 120]
    # a single page: the first part takes it
    assert [t1 - t0 for t0, t1 in orep.split_blocks(10, 256)] == [10, 0, 0, 0]
