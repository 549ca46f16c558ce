"""Oracle of the content-adaptive top-k key-tile selection (test infrastructure only).

What the paper fixes (Sec. 2.3.1 (b), Eq. 4; App. L, Eq. 10): queries and keys
are mean-pooled within each block, a block score is the dot product of a pooled
query with a pooled key divided by sqrt(d_h), a softmax runs over each query
block's row of scores, and each head keeps, per query block, the key blocks
that the top-k budget admits; the result is intersected with the structural
masks.  The budget grows linearly with the sequence length (Eq. 10).

Readings taken here, where the paper leaves the arithmetic open:

* Blocks are the T-token tiles (each chunk tiled on its own from its first
  token); a pooled vector is the mean over the tile's valid tokens.
* The threshold tau_k of Eq. 4 is read as the count k: the k best-scoring
  candidate tiles of a row are kept.  The softmax and the positive factor
  1/sqrt(d_h) are monotone, so the ranking uses the raw pooled dot products.
  Equal scores go to the lower logical tile index.
* The tiles of the pinned chunk and of the current chunk may be forced (kept
  outside the ranking, as the structural part of the Bernoulli rule in
  ``keep``); with both flags off the rule is Eq. 4's top-k over the whole
  causal window.
* The arithmetic is IEEE float32 in a fixed order, so that this oracle and
  the GPU make the same integer decision:

      mean[d]  = (((x_0[d] + x_1[d]) + x_2[d]) + ... + x_{n-1}[d]) / n
      score    = ((qm[0]*km[0] + qm[1]*km[1]) + ... ) + qm[D-1]*km[D-1]

  every sum, product and the division rounded to float32 (no fused
  multiply-add).  Scores are ordered through the unsigned key that orders
  float32 values like the real line (sign bit set: all bits flipped; else the
  sign bit set), highest first.

Parity of this reading against the paper is unpinned: the paper defines
tau_k both as a probability threshold (Eq. 4) and as a count (Eq. 10), and its
Eq. 10 gives a budget above the number of blocks at the 1K and 2K shapes.
"""

import math
from dataclasses import dataclass

import numpy as np

from .keep import tile_geometry


@dataclass(frozen=True)
class TopkRule:
    budget: int                # k: kept tiles per row among the ranked candidates
    keep_sink: bool = True     # force the pinned chunk's tiles
    keep_current: bool = True  # force the current chunk's tiles


def topk_budget(rho: float, seq_len: int, seq_ref: int, n_blocks: int, k_min: int = 4) -> int:
    """Eq. 10: max(k_min, floor(rho * S / S_ref * N_blocks)), evaluated in double."""
    return max(int(k_min), int(math.floor(float(rho) * float(seq_len) / float(seq_ref) * float(n_blocks))))


def pooled_means(x, T: int) -> np.ndarray:
    """Per-tile means [NT, D] float32 of x [L, D] (bf16 values), valid tokens only.

    Sequential float32 sum over the tile's tokens in order, then one division.
    Rows past the chunk end are zero and add nothing (x + 0 == x exactly).
    """
    x32 = np.asarray(x, dtype=np.float32)
    L, D = x32.shape
    nt, tail = tile_geometry(L, T)
    xp = np.zeros((nt * T, D), dtype=np.float32)
    xp[:L] = x32
    xp = xp.reshape(nt, T, D)
    acc = np.zeros((nt, D), dtype=np.float32)
    for r in range(T):
        acc = (acc + xp[:, r, :]).astype(np.float32)
    n = np.full((nt, 1), T, dtype=np.float32)
    n[-1, 0] = tail
    return (acc / n).astype(np.float32)


def block_scores(qm: np.ndarray, km: np.ndarray) -> np.ndarray:
    """Scores [NQ, NK] float32: products rounded to float32, added in order of d."""
    qm = np.asarray(qm, dtype=np.float32)
    km = np.asarray(km, dtype=np.float32)
    acc = np.zeros((qm.shape[0], km.shape[0]), dtype=np.float32)
    for d in range(qm.shape[1]):
        prod = (qm[:, d, None] * km[None, :, d]).astype(np.float32)
        acc = (acc + prod).astype(np.float32)
    return acc


def order_key(s: np.ndarray) -> np.ndarray:
    """uint32 key that orders float32 values like the real line."""
    u = np.asarray(s, dtype=np.float32).view(np.uint32)
    return np.where((u & np.uint32(0x80000000)) != 0, ~u, u | np.uint32(0x80000000)).astype(np.uint32)


def select_topk(scores: np.ndarray, candidate: np.ndarray, k: int) -> np.ndarray:
    """Boolean [NK]: the k candidates with the highest scores, ties to the lower index."""
    keep = np.zeros(scores.shape[0], dtype=bool)
    cand = np.nonzero(candidate)[0]
    if k <= 0 or cand.size == 0:
        return keep
    key = order_key(scores[cand]).astype(np.int64)
    order = np.lexsort((cand, -key))       # highest key first, then ascending index
    keep[cand[order[:k]]] = True
    return keep


def topk_scores(ring, q, T: int):
    """Block scores [B, H, NQ, NK] float32 of the current chunk's queries q [B, L, H, D]."""
    chunks = ring.logical_chunks()
    q = np.asarray(q)
    B, L, H, _ = q.shape
    nt, _ = tile_geometry(L, T)
    out = np.empty((B, H, nt, nt * len(chunks)), dtype=np.float32)
    for b in range(B):
        for h in range(H):
            qm = pooled_means(q[b, :, h, :], T)
            km = np.concatenate([pooled_means(c.k[b, :, h, :], T) for c in chunks], axis=0)
            out[b, h] = block_scores(qm, km)
    return out


def topk_bits(ring, q, T: int, rule: TopkRule, scores=None) -> np.ndarray:
    """Boolean keep set [B, H, NQ, NK]: forced tiles plus the top ``rule.budget`` of the rest."""
    chunks = ring.logical_chunks()
    cur = ring.current
    s = topk_scores(ring, q, T) if scores is None else scores
    B, H, nq, nk = s.shape
    nt = nq
    forced = np.zeros(nk, dtype=bool)
    for pos, c in enumerate(chunks):
        if (c.sink and rule.keep_sink) or (c.seq == cur.seq and rule.keep_current):
            forced[pos * nt:(pos + 1) * nt] = True
    bits = np.zeros((B, H, nq, nk), dtype=bool)
    for b in range(B):
        for h in range(H):
            for i in range(nq):
                bits[b, h, i] = forced | select_topk(s[b, h, i], ~forced, int(rule.budget))
    return bits
