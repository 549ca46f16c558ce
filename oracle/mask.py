"""Oracle of the composed block mask of Eq. 4 (test infrastructure only).

What the paper fixes (Sec. 2.3.1 (a) and (b), Eq. 4; App. C): each head's
block mask is the intersection of three masks over (query block, key block)
pairs of the window: the content rule (the top-k selection over pooled block
scores), the spatial local window M_local (an r x r window of blocks) and the
temporal causal mask M_causal (a chunk sees itself and earlier chunks).

Readings taken here:

* M_causal holds for every key block of the window: the window only ever
  contains the current chunk and earlier ones, and inside the current chunk
  the mask is chunk-granular (no token-level triangle).
* The content rule is either the top-k rule of ``topk`` or the seeded
  Bernoulli stand-in of ``keep``; both may force the pinned chunk's and the
  current chunk's blocks (kept outside the draw or the ranking).
* The rule is applied first, over every candidate of the window; M_local is
  intersected afterwards, forced blocks included.  A top-k pick that falls
  outside the window is therefore lost and not replaced by the next-best
  block inside it, as the literal intersection of Eq. 4 says.
* Blocks are either the T-token tiles of each chunk (raster tiles; M_local
  needs a 2-D block grid and is not defined for them) or the 3-D blocks of a
  ``BlockGeom`` (tile = b_t * b_h * b_w rows, blocks in raster order of
  block time, block row, block column; pooled means over each block's
  valid tokens).
"""

import numpy as np

from .blocks import BlockGeom, block_means, local_mask
from .keep import KeepRule, keep_bits
from .ring import Chunk, RingModel
from .topk import TopkRule, block_scores, select_topk, topk_bits


def _forced(chunks, cur, keep_sink: bool, keep_current: bool, nb: int) -> np.ndarray:
    forced = np.zeros(nb * len(chunks), dtype=bool)
    for pos, c in enumerate(chunks):
        if (c.sink and keep_sink) or (c.seq == cur.seq and keep_current):
            forced[pos * nb:(pos + 1) * nb] = True
    return forced


def _metadata_ring(ring: RingModel, B: int, rows: int, H: int) -> RingModel:
    """The ring's chunk sequence with chunks of ``rows`` token rows (no data)."""
    meta = RingModel(ring.max_chunks, ring.pin_sink)
    z = np.broadcast_to(np.zeros(1), (B, rows, H, 1))
    meta.live = [Chunk(c.seq, c.sink, z, None) for c in ring.live]
    return meta


def block_sparse_mask(ring: RingModel, rule, q=None, T: int = None, geom: BlockGeom = None,
                      local_r: int = 0) -> np.ndarray:
    """Keep set [B, H, NQ, NK] of Eq. 4 for the ring's current chunk.

    ring   -- the window (raster-order chunks [B, tokens, H, D]); the keys are
              read only by the top-k rule.
    rule   -- ``KeepRule`` (Bernoulli stand-in) or ``TopkRule``.
    q      -- the current chunk's queries [B, tokens, H, D] (top-k only).
    T      -- tile size of raster tiles, or None with ``geom``.
    geom   -- 3-D block geometry of every chunk, or None with ``T``.
    local_r -- r of M_local (0: no local window); needs ``geom``.

    NQ = blocks of the current chunk; NK = n_live * blocks per chunk, in
    logical order (key block j is block j % NB of the chunk at position
    j // NB).
    """
    if (T is None) == (geom is None):
        raise ValueError("give exactly one of T (raster tiles) and geom (3-D blocks)")
    if local_r and geom is None:
        raise ValueError("M_local needs the 2-D block grid of a BlockGeom")
    chunks = ring.logical_chunks()
    cur = ring.current
    B, _, H, _ = cur.k.shape
    if isinstance(rule, KeepRule):
        if geom is None:
            bits = keep_bits(_metadata_ring(ring, B, cur.k.shape[1], H), T, rule)
        else:
            bits = keep_bits(_metadata_ring(ring, B, geom.padded_tokens, H), geom.tile, rule)
    elif isinstance(rule, TopkRule):
        if q is None:
            raise ValueError("the top-k rule ranks pooled queries: q is required")
        if geom is None:
            bits = topk_bits(ring, q, T, rule)
        else:
            nb = geom.n_blocks
            forced = _forced(chunks, cur, rule.keep_sink, rule.keep_current, nb)
            qv = np.asarray(q)
            bits = np.zeros((B, H, nb, nb * len(chunks)), dtype=bool)
            for b in range(B):
                for h in range(H):
                    qm = block_means(qv[b, :, h], geom)
                    km = np.concatenate([block_means(c.k[b, :, h], geom) for c in chunks])
                    s = block_scores(qm, km)
                    for i in range(nb):
                        bits[b, h, i] = forced | select_topk(s[i], ~forced, int(rule.budget))
    else:
        raise TypeError("rule must be a KeepRule or a TopkRule")
    if local_r:
        local = np.tile(local_mask(geom, local_r), (1, len(chunks)))
        bits = bits & local[None, None]
    return bits
