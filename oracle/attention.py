"""Oracle of block-sparse chunk-causal attention (test infrastructure only).

Definition (Sec. 2.3.1, Eq. 4 and the sentence after it): for each head, the
current chunk's queries attend, with ordinary scaled softmax attention, over
the keys of the kept key blocks only; every other key is excluded from the
softmax.  Under the temporal causal mask the key set is the cache window of
earlier chunks plus the current chunk, and inside the current chunk there is
no token-level triangle (the mask is chunk-granular, Sec. 2.3.1(a)).

For one query row r of query tile i, with K, V the concatenation over the
window's chunks in logical order and ``kept(i)`` the union of the token spans
of the kept key tiles:

    s_c = scale * <q_r, k_c>                  for c in kept(i)
    m   = max_c s_c
    l   = sum_c exp(s_c - m)
    o_r = sum_c exp(s_c - m) * v_c / l
    lse = m + log(l)

An empty kept set gives o_r = 0 and lse = -inf (a degenerate case the keep
rule never produces, since the current chunk is always kept).

Computed in float64 over the window's keys with a keep mask per row: the
scores of excluded keys take no part in the row maximum and are never
exponentiated, so their weights are exactly zero.  Inputs are the bf16 values
widened exactly.
"""

import numpy as np

from .keep import tile_geometry


def dense_keys(ring, b: int, h: int):
    """(K, V) [Sk, D] float64 of head (b, h): the window's chunks in logical order."""
    chunks = ring.logical_chunks()
    K = np.concatenate([c.k[b, :, h, :] for c in chunks], axis=0)
    V = np.concatenate([c.v[b, :, h, :] for c in chunks], axis=0)
    return K, V


def _kept_columns(kept_tiles, L: int, T: int, nt: int, sk: int) -> np.ndarray:
    cols = np.zeros(sk, dtype=bool)
    for j in kept_tiles:
        pos, t = divmod(int(j), nt)
        lo = pos * L + t * T
        hi = pos * L + min((t + 1) * T, L)
        cols[lo:hi] = True
    return cols


def _attend_rows(Q, K, V, cols, scale):
    """Softmax attention of query rows Q [n, D] over the keys where cols is True.

    cols is [Sk] (one keep set for every row) or [n, Sk] (one per row).  A row
    with no kept key gives o = 0, lse = -inf and a row sum of 0.
    """
    n = Q.shape[0]
    M = np.broadcast_to(np.asarray(cols, dtype=bool), (n, K.shape[0]))
    S = (Q @ K.T) * scale
    m = np.max(S, axis=1, where=M, initial=-np.inf)
    P = np.zeros_like(S)
    np.exp(S - m[:, None], out=P, where=M)
    l = P.sum(axis=1)
    has = l > 0
    ls = np.where(has, l, 1.0)
    O = (P @ V) / ls[:, None]
    lse = np.where(has, m + np.log(ls), -np.inf)
    rowsum = (P / ls[:, None]).sum(axis=1)
    return O, lse, rowsum


def sparse_causal_attention(ring, q, bits, T: int, scale: float, heads=None, qtiles=None,
                            with_rowsum: bool = False):
    """Attention of the current chunk's queries over the kept key tiles.

    q: [B, L, H, D] (bf16 values); bits: [B, H, NQ, NK] bool keep set.
    Returns O [B, L, H, D] float64 and LSE [B, H, L] float64 (and, on request,
    the row sums of the normalised weights).  ``heads`` / ``qtiles`` restrict
    the work to a subset (other entries are left as NaN).
    """
    q = np.asarray(q, np.float64)
    B, L, H, D = q.shape
    nt, _ = tile_geometry(L, T)
    sk = ring.n_live * L
    O = np.full((B, L, H, D), np.nan)
    LSE = np.full((B, H, L), np.nan)
    RS = np.full((B, H, L), np.nan)
    heads = range(H) if heads is None else heads
    qtiles = range(nt) if qtiles is None else qtiles
    for b in range(B):
        for h in heads:
            K, V = dense_keys(ring, b, h)
            for i in qtiles:
                r0, r1 = i * T, min((i + 1) * T, L)
                cols = _kept_columns(np.nonzero(bits[b, h, i])[0], L, T, nt, sk)
                o, lse, rs = _attend_rows(q[b, r0:r1, h, :], K, V, cols, scale)
                O[b, r0:r1, h, :] = o
                LSE[b, h, r0:r1] = lse
                RS[b, h, r0:r1] = rs
    if with_rowsum:
        return O, LSE, RS
    return O, LSE


def sparse_causal_attention_rows(ring, q, bits, T: int, scale: float, samples):
    """Same definition, evaluated only at sampled (b, h, row) triples.

    samples: iterable of (b, h, r).  Returns O [n, D] and LSE [n] float64.
    The rows of one head are evaluated together, each over its own keep set.
    """
    q = np.asarray(q, np.float64)
    B, L, H, D = q.shape
    nt, _ = tile_geometry(L, T)
    sk = ring.n_live * L
    samples = list(samples)
    O = np.zeros((len(samples), D))
    LSE = np.zeros(len(samples))
    by_head = {}
    for n, (b, h, r) in enumerate(samples):
        by_head.setdefault((b, h), []).append(n)
    for (b, h), ns in by_head.items():
        K, V = dense_keys(ring, b, h)
        rows = [samples[n][2] for n in ns]
        cols = {}
        for r in rows:
            if r // T not in cols:
                cols[r // T] = _kept_columns(np.nonzero(bits[b, h, r // T])[0], L, T, nt, sk)
        M = np.stack([cols[r // T] for r in rows])
        o, lse, _ = _attend_rows(q[b, rows, h, :], K, V, M, scale)
        O[ns] = o
        LSE[ns] = lse
    return O, LSE
