"""Pins of the block-repair oracle (Sec. 6.3, block-level paging).

* The shares of the blocks add up to A - 1 (block decomposability), and when the
  exact logits of the repaired blocks equal the compressed ones the repaired
  certificate is A - (sum of their shares) exactly: the paper's statement.
* Repairing every block gives the exact output and raw 0.
* After any repair the certificate still bounds the true TV between the exact
  distribution and the repaired one.
* The order equals a brute-force sort, and the stop rule is minimal: the first
  n - 1 blocks of the order do not pass, the first n do.
* Persistent repair (Sec. 6 gate; Sec. 6.3 gated evaluation (c)): the mixed state
  reduces to the plain decode (nothing repaired) and to exact attention with
  raw 0 (everything repaired), equals the split merge of its two token sets under
  the LSE weights, and still bounds the true TV; the written-back pages follow a
  brute-force count; over two steps the written-back state reproduces the repair,
  later repairs rank only blocks with unrepaired tokens (their shares of repaired
  tokens are 0), and no token is paged in twice.
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


# ---- incremental persistent repair (Sec. 6 gate; Sec. 6.3 gated evaluation (c)) ----

def _split_merge(q, kh, vh, k, v, c, rep, sm):
    """The mixed state by another route: the repaired and the compressed tokens as two
    splits, each reduced on its own, merged under the LSE weights (Sec. 6.2)."""
    G = q.shape[0]
    out = np.empty((G, v.shape[1]))
    raw = np.empty(G)
    for h in range(G):
        parts = []
        for sel, kk, vv, cc in ((~rep, kh, vh, c[h]), (rep, k, v, np.zeros_like(c[h]))):
            if not sel.any():
                continue
            z = np.array([sm * float(np.dot(q[h], kk[t])) for t in np.flatnonzero(sel)])
            m = z.max()
            w = np.exp(z - m)
            parts.append((m, w.sum(), w @ vv[sel], float(np.sum(w * np.expm1(cc[sel])))))
        M = max(p[0] for p in parts)
        L = sum(np.exp(p[0] - M) * p[1] for p in parts)
        out[h] = sum(np.exp(p[0] - M) * p[2] for p in parts) / L
        am1 = sum(np.exp(p[0] - M) * p[3] for p in parts) / L
        raw[h] = am1 * (am1 + 2) / 2
    return out, raw


def test_mixed_state_special_cases_and_split_merge():
    rng = np.random.default_rng(43)
    q, k, v, kh, vh, cb = _case(rng, S=200)
    sm = 1 / np.sqrt(q.shape[1])
    S = kh.shape[0]
    # nothing repaired: the plain metered decode of the compressed cache
    st = orep.mixed_state(q, kh, vh, k, v, cb, np.zeros(S, bool), sm)
    ref = odec.metered_decode(q, kh[:, None], vh[:, None], np.zeros((S, 1, 4)), sm, 4)
    assert np.allclose(st["out"], ref["out"], rtol=0, atol=1e-13)
    for h in range(q.shape[0]):
        z = attention.logits(q[h], kh, sm)
        assert np.isclose(st["raw"][h], mt.raw_from_am1(mt.a_minus_one_logits(z, cb[h])), rtol=1e-12)
    # everything repaired: exact attention, A = 1
    st = orep.mixed_state(q, kh, vh, k, v, cb, np.ones(S, bool), sm)
    ex = odec.exact_decode(q, k[:, None], v[:, None], sm)["out"]
    assert np.allclose(st["out"], ex, rtol=0, atol=1e-13) and np.all(st["raw"] == 0)
    # random page masks against the split merge
    for trial in range(6):
        pages = rng.random(orep.pages_of(S)) < rng.uniform(0.1, 0.9)
        rep = orep.token_mask(pages, S)
        st = orep.mixed_state(q, kh, vh, k, v, cb, rep, sm)
        o2, r2 = _split_merge(q, kh, vh, k, v, cb, rep, sm)
        assert np.allclose(st["out"], o2, rtol=0, atol=1e-12)
        assert np.allclose(st["raw"], r2, rtol=1e-10, atol=0)


def test_mixed_state_stays_sound():
    rng = np.random.default_rng(44)
    for trial in range(8):
        q, k, v, kh, vh, cb = _case(rng, S=180, q_scale=rng.uniform(0.3, 1.5))
        sm = 1 / np.sqrt(q.shape[1])
        rep = orep.token_mask(rng.random(orep.pages_of(180)) < 0.5, 180)
        st = orep.mixed_state(q, kh, vh, k, v, cb, rep, sm)
        kk = np.where(rep[:, None], k, kh)
        for h in range(q.shape[0]):
            p = attention.softmax(attention.logits(q[h], k, sm))
            pr = attention.softmax(attention.logits(q[h], kk, sm))
            assert attention.tv(p, pr) <= st["meter"][h] + 1e-15


def test_persist_pages_brute_force():
    ranges = orep.block_ranges(300, 64)
    for S in (1, 15, 16, 17, 64, 100, 255, 300):
        for blocks in ([0], [4], [1, 3], [0, 1, 2, 3, 4]):
            pages = orep.persist(np.zeros(orep.pages_of(320), bool), blocks, ranges, S)
            want = {t // 16 for j in blocks for t in range(*ranges[j]) if t < S}
            assert set(np.flatnonzero(pages)) == want
    p = orep.persist_all(np.zeros(25, bool), 300)
    assert np.flatnonzero(p).tolist() == list(range(19))          # pages 0 .. 18 hold 0 .. 299
    m = orep.token_mask(np.array([False, True, False]), 40)
    assert m.tolist() == [False] * 16 + [True] * 16 + [False] * 8
    assert orep.candidates(m, orep.block_ranges(40, 16)).tolist() == [True, False, True]


def test_persistent_repair_two_steps():
    """Step 1 repairs and writes back; step 2, three pages longer, decodes the mixed
    state, ranks only blocks with unrepaired tokens, and never pages a token in twice."""
    rng = np.random.default_rng(45)
    d, G, S1, S2 = 32, 3, 296, 340
    kf = rng.normal(size=(S2, d)) * rng.uniform(0.5, 3, size=d)
    vf = rng.normal(size=(S2, d))
    seed = int(rng.integers(1 << 30))
    cache = odec.write_cache("int8_dither", kf[:, None], vf[:, None], np.arange(S2), 0, seed, 4)
    kh, vh = cache["khat"][:, 0], cache["vhat"][:, 0]
    q = rng.normal(size=(G, d)) * 0.7
    sm = 1 / np.sqrt(d)
    cb = np.stack([mt.logit_bound(q[h], cache["kw"][:, 0], sm, 4) for h in range(G)])
    ranges1 = orep.block_ranges(S1, 64)
    r1 = orep.block_repair(q, kh[:S1], vh[:S1], kf[:S1], vf[:S1], cb[:, :S1], ranges1, sm, 0.05, len(ranges1))
    assert r1["n_blocks"] >= 1
    taken = r1["order"][:r1["n_blocks"]]
    pages = orep.persist(np.zeros(orep.pages_of(S2), bool), taken, ranges1, S1)
    # step 1's state read back from the written-back pages equals the repair's result
    st1 = orep.mixed_state(q, kh[:S1], vh[:S1], kf[:S1], vf[:S1], cb[:, :S1], orep.token_mask(pages, S1), sm)
    assert np.allclose(st1["out"], r1["out"], rtol=0, atol=1e-13) and np.allclose(st1["raw"], r1["raw"])
    # step 2: tokens S1 .. S2-1 join; the marked pages stay exact (S1 = 296 lies in page 18)
    rep2 = orep.token_mask(pages, S2)
    assert rep2[S1:S2].sum() == (16 - S1 % 16 if pages[S1 // 16] else 0)
    ranges2 = orep.block_ranges(S2, 64)
    r2 = orep.block_repair(q, kh, vh, kf, vf, cb, ranges2, sm, 0.02, len(ranges2), base=rep2)
    cand = orep.candidates(rep2, ranges2)
    assert all(cand[j] for j in r2["order"])
    full = {j for j in range(len(ranges2)) if rep2[ranges2[j][0]:ranges2[j][1]].all()}
    assert full and not full & set(r2["order"].tolist())
    # shares of the mixed state: a repaired token contributes nothing
    for h in range(G):
        for j in full:
            assert r2["shares"][h, j] == 0.0
    if r2["n_blocks"] >= 1:
        pages2 = orep.persist(pages, r2["order"][:r2["n_blocks"]], ranges2, S2)
        newly = orep.token_mask(pages2, S2) & ~rep2
        assert not (newly & rep2).any()
        assert np.array_equal(orep.token_mask(pages2, S2), rep2 | newly)
