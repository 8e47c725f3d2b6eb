"""Block-granular repair of gated heads (Sec. 6.3, block-level paging).

TEST INFRASTRUCTURE ONLY (see the package header).

The certificate is block decomposable: A - 1 = sum_t ptilde_t (e^{c_t} - 1) splits
into per-block shares, share_j = sum_{t in block j} ptilde_t (e^{c_t} - 1).  A gated
head can therefore be repaired by taking a few blocks from the exact store:
blocks are taken in decreasing order of their share, and after each block the
certificate is recomputed, until it falls back to the threshold (Sec. 6.3).

Definitions followed, with our readings where the paper leaves a choice:

* Blocks: fixed runs of BLOCK_TOKENS = 256 consecutive tokens of the sequence,
  block j holding positions 256j .. 256j + 255 (the last one shorter): Sec. 6.3
  divides S = 32768 into n_b = 128 blocks (``paper_blocks``).  The definitions
  below take any partition into consecutive ranges (``block_ranges``), so the
  pins can use small blocks on small cases.
* Order: for a KV head with G query heads, blocks are ranked by the sum over the
  G heads of their shares, largest first, ties to the lower block index (the
  exact values of a block serve every query head of its KV head).
* Repaired state after taking a set R of blocks: on the tokens of R the logits,
  values and bounds are the exact ones (logit error 0, so c = 0 there);
  elsewhere the compressed ones.  The compressed distribution, the output and
  the certificate are recomputed from that mixed state:
      ptilde'_t = softmax over t of (exact logit on R, compressed logit off R),
      out' = sum_t ptilde'_t v'_t (v' exact on R, vhat off R),
      A' = sum_t ptilde'_t e^{c'_t},  raw' = (A'^2 - 1)/2,  meter' = min(1, raw').
  (When the exact logits of R equal the compressed ones, A' = A - sum_{j in R}
  share_j exactly, which is the paper's statement.)
* Stop: blocks are added in order until every query head's gate value (meter',
  or raw' when tau >= 1) is at most tau; at most max_blocks blocks, otherwise the
  KV head is left to the whole-head exact fallback.

Incremental persistent repair (the meter loop's gate, Sec. 6: the flagged blocks or
head come back from the exact store, the head is recomputed, the exact values are
kept and their witnesses cleared; Sec. 6.3 gated evaluation (c): un-repaired slots are
paged in once, and repaired slots are filtered out by their zero witness).
Readings:

* The repaired state is kept per cache page (PAGE_TOKENS = 16 consecutive
  positions) and KV head: writing back block j marks the pages that hold its
  positions below the current length (``persist``); the whole-head fallback
  marks every page of the sequence (``persist_all``).  A marked page is served
  from the exact store from then on, for every token it holds, including tokens
  written into it later; its bound is 0 (the zeroed witness).
* Every later decode is the mixed state over the marked tokens (``mixed_state``,
  ``decode_repaired``), and a later repair ranks and takes only blocks that still
  hold a token outside the marked pages (``candidates``: the witness-nonzero
  filter); the shares of a repair are those of the mixed state.
"""
from __future__ import annotations

import numpy as np

from . import attention, meter as mt


def block_ranges(seq_len: int, block_tokens: int) -> list:
    """[(t0, t1)]: consecutive blocks of block_tokens tokens (the last one shorter)."""
    return [(t, min(t + block_tokens, seq_len)) for t in range(0, seq_len, block_tokens)]


BLOCK_TOKENS = 256


def paper_blocks(seq_len: int) -> list:
    """The repair blocks of a sequence: consecutive 256-token runs (Sec. 6.3)."""
    return block_ranges(seq_len, BLOCK_TOKENS)


def block_shares(ptilde: np.ndarray, c: np.ndarray, ranges: list) -> np.ndarray:
    """share_j = sum_{t in j} ptilde_t (e^{c_t} - 1); sums to A - 1."""
    term = np.asarray(ptilde, dtype=np.float64) * np.expm1(np.asarray(c, dtype=np.float64))
    return np.array([term[t0:t1].sum() for t0, t1 in ranges])


def repair_order(shares: np.ndarray) -> np.ndarray:
    """Block indices by decreasing sum over the query heads (rows), ties to the lower index."""
    tot = np.asarray(shares, dtype=np.float64).sum(axis=0)
    return np.array(sorted(range(tot.size), key=lambda j: (-tot[j], j)), dtype=np.int64)


PAGE_TOKENS = 16


def mixed_state(q: np.ndarray, khat: np.ndarray, vhat: np.ndarray, k: np.ndarray, v: np.ndarray,
                c: np.ndarray, rep: np.ndarray, sm_scale: float) -> dict:
    """q [G, d] of one KV head; khat, vhat, k, v [S, d]; c [G, S]; rep bool [S]: tokens
    served exactly (exact logit and value, bound 0), the others compressed."""
    rep = np.asarray(rep, dtype=bool)
    kk = np.where(rep[:, None], k, khat)
    vv = np.where(rep[:, None], v, vhat)
    G = q.shape[0]
    out = np.empty((G, vv.shape[1]))
    raw = np.empty(G)
    pt = np.empty((G, rep.size))
    for h in range(G):
        z = attention.logits(q[h], kk, sm_scale)
        p = attention.softmax(z)
        out[h] = p @ vv
        raw[h] = mt.raw_from_am1(mt.a_minus_one_logits(z, np.where(rep, 0.0, c[h])))
        pt[h] = p
    return {"out": out, "raw": raw, "meter": mt.meter(raw), "repaired": rep, "ptilde": pt}


def block_tokens_mask(S: int, blocks, ranges: list) -> np.ndarray:
    """bool [S]: the tokens of the given blocks."""
    rep = np.zeros(S, dtype=bool)
    for j in blocks:
        t0, t1 = ranges[j]
        rep[t0:t1] = True
    return rep


def repaired_state(q: np.ndarray, khat: np.ndarray, vhat: np.ndarray, k: np.ndarray, v: np.ndarray,
                   c: np.ndarray, blocks, ranges: list, sm_scale: float, base=None) -> dict:
    """The mixed state with the tokens of `blocks` (and of the mask `base`) repaired."""
    rep = block_tokens_mask(khat.shape[0], blocks, ranges)
    if base is not None:
        rep |= np.asarray(base, dtype=bool)
    return mixed_state(q, khat, vhat, k, v, c, rep, sm_scale)


def candidates(rep: np.ndarray, ranges: list) -> np.ndarray:
    """bool [n_blocks]: blocks holding a token that is not yet repaired."""
    rep = np.asarray(rep, dtype=bool)
    return np.array([not rep[t0:t1].all() for t0, t1 in ranges])


def block_repair(q: np.ndarray, khat: np.ndarray, vhat: np.ndarray, k: np.ndarray, v: np.ndarray,
                 c: np.ndarray, ranges: list, sm_scale: float, tau: float, max_blocks: int,
                 base=None) -> dict:
    """Repair one KV head: returns order, n_blocks (-1 when max_blocks do not suffice),
    and the repaired out, raw, meter (those of the last state tried).  With `base`
    (bool [S], tokens already repaired) the shares are those of the mixed state and
    only candidate blocks are ranked."""
    G = q.shape[0]
    S = khat.shape[0]
    base = np.zeros(S, dtype=bool) if base is None else np.asarray(base, dtype=bool)
    cur = mixed_state(q, khat, vhat, k, v, c, base, sm_scale)
    shares = np.empty((G, len(ranges)))
    for h in range(G):
        shares[h] = block_shares(cur["ptilde"][h], np.where(base, 0.0, c[h]), ranges)
    cand = candidates(base, ranges)
    order = np.array([j for j in repair_order(shares) if cand[j]], dtype=np.int64)
    res = None
    for n in range(1, min(max_blocks, order.size) + 1):
        res = repaired_state(q, khat, vhat, k, v, c, order[:n], ranges, sm_scale, base)
        val = res["raw"] if tau >= 1.0 else res["meter"]
        if np.all(val <= tau):
            return {"order": order, "shares": shares, "n_blocks": n, **res}
    return {"order": order, "shares": shares, "n_blocks": -1, **(res or {})}


def pages_of(S: int) -> int:
    """Pages that hold positions 0 .. S-1."""
    return -(-S // PAGE_TOKENS)


def token_mask(rep_pages: np.ndarray, S: int) -> np.ndarray:
    """bool [S]: position t is repaired when its page t // 16 is marked."""
    rep_pages = np.asarray(rep_pages, dtype=bool)
    return np.array([t // PAGE_TOKENS < rep_pages.size and rep_pages[t // PAGE_TOKENS] for t in range(S)],
                    dtype=bool)


def persist(rep_pages: np.ndarray, blocks, ranges: list, S: int) -> np.ndarray:
    """Write-back of taken blocks: the pages holding their positions below S are marked."""
    out = np.array(rep_pages, dtype=bool, copy=True)
    for j in blocks:
        t0, t1 = ranges[j]
        for t in range(t0, min(t1, S)):
            out[t // PAGE_TOKENS] = True
    return out


def persist_all(rep_pages: np.ndarray, S: int) -> np.ndarray:
    """Write-back after the whole-head fallback: every page of positions 0 .. S-1."""
    out = np.array(rep_pages, dtype=bool, copy=True)
    out[:pages_of(S)] = True
    return out


def decode_repaired(q: np.ndarray, khat: np.ndarray, vhat: np.ndarray, k: np.ndarray, v: np.ndarray,
                    c: np.ndarray, rep: np.ndarray, sm_scale: float) -> dict:
    """Decode of all query heads over a cache with repaired tokens: q [n_q, d]; khat,
    vhat, k, v [S, n_kv, d]; c [n_q, S] per-token bounds of the compressed keys; rep
    bool [S, n_kv].  Returns out, raw, meter [n_q] and ptilde [n_q, S]."""
    q = np.asarray(q, dtype=np.float64)
    n_q, d = q.shape
    n_kv = khat.shape[1]
    g = n_q // n_kv
    out = np.empty((n_q, d))
    raw = np.empty(n_q)
    pt = np.empty((n_q, khat.shape[0]))
    for kv in range(n_kv):
        hs = slice(kv * g, (kv + 1) * g)
        st = mixed_state(q[hs], khat[:, kv], vhat[:, kv], k[:, kv], v[:, kv], c[hs], rep[:, kv], sm_scale)
        out[hs], raw[hs], pt[hs] = st["out"], st["raw"], st["ptilde"]
    return {"out": out, "raw": raw, "meter": mt.meter(raw), "ptilde": pt}
