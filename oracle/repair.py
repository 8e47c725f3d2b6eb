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


def repaired_state(q: np.ndarray, khat: np.ndarray, vhat: np.ndarray, k: np.ndarray, v: np.ndarray,
                   c: np.ndarray, blocks, ranges: list, sm_scale: float) -> dict:
    """q [G, d] of one KV head; khat, vhat, k, v [S, d]; c [G, S]; blocks: repaired block ids."""
    S = khat.shape[0]
    rep = np.zeros(S, dtype=bool)
    for j in blocks:
        t0, t1 = ranges[j]
        rep[t0:t1] = True
    kk = np.where(rep[:, None], k, khat)
    vv = np.where(rep[:, None], v, vhat)
    G = q.shape[0]
    out = np.empty((G, vv.shape[1]))
    raw = np.empty(G)
    for h in range(G):
        z = attention.logits(q[h], kk, sm_scale)
        p = attention.softmax(z)
        out[h] = p @ vv
        raw[h] = mt.raw_from_am1(mt.a_minus_one_logits(z, np.where(rep, 0.0, c[h])))
    return {"out": out, "raw": raw, "meter": mt.meter(raw), "repaired": rep}


def block_repair(q: np.ndarray, khat: np.ndarray, vhat: np.ndarray, k: np.ndarray, v: np.ndarray,
                 c: np.ndarray, ranges: list, sm_scale: float, tau: float, max_blocks: int) -> dict:
    """Repair one KV head: returns order, n_blocks (-1 when max_blocks do not suffice),
    and the repaired out, raw, meter (those of the last state tried)."""
    G = q.shape[0]
    shares = np.empty((G, len(ranges)))
    for h in range(G):
        z = attention.logits(q[h], khat, sm_scale)
        shares[h] = block_shares(attention.softmax(z), c[h], ranges)
    order = repair_order(shares)
    res = None
    for n in range(1, min(max_blocks, len(ranges)) + 1):
        res = repaired_state(q, khat, vhat, k, v, c, order[:n], ranges, sm_scale)
        val = res["raw"] if tau >= 1.0 else res["meter"]
        if np.all(val <= tau):
            return {"order": order, "shares": shares, "n_blocks": n, **res}
    return {"order": order, "shares": shares, "n_blocks": -1, **(res or {})}
