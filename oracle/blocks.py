"""Oracle of the 3-D block tiling and the structural local mask (test infrastructure only).

What the paper fixes (Sec. 2.3.1, block-sparse causal attention (a);
App. C): the token grid (t, h, w) of a chunk is divided into non-overlapping
(b_t, b_h, b_w) blocks, (2, 8, 8) in the paper's model; a spatial locality
mask confines each block's receptive field to an r x r sliding window of
blocks; the temporal causal mask lets a chunk see itself and earlier chunks.

Readings taken here:

* A chunk of F latent frames on a gh x gw grid has blocks
  (ceil(F/b_t), ceil(gh/b_h), ceil(gw/b_w)) in raster order (block time,
  then block row, then block column); edge blocks hold fewer tokens.
* Block order of tokens: block after block, and inside a block the valid
  tokens in raster (t, h, w) order, the block padded to b_t*b_h*b_w rows (one
  tile) with rows that count as no token.
* M_local keeps key block j for query block i when their block rows and
  block columns both differ by at most floor(r/2) (an r x r window centred
  on the query block, clipped at the grid edge), in every chunk of the
  window and at every block time.  It intersects whatever keep rule is used,
  forced tiles included (Eq. 4: rule, M_local and M_causal are intersected).
"""

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class BlockGeom:
    frames: int
    grid_h: int
    grid_w: int
    bt: int = 2
    bh: int = 8
    bw: int = 8

    @property
    def tile(self) -> int:
        return self.bt * self.bh * self.bw

    @property
    def nblocks3(self):
        return (-(-self.frames // self.bt), -(-self.grid_h // self.bh), -(-self.grid_w // self.bw))

    @property
    def n_blocks(self) -> int:
        a, b, c = self.nblocks3
        return a * b * c

    @property
    def tokens(self) -> int:
        return self.frames * self.grid_h * self.grid_w

    @property
    def padded_tokens(self) -> int:
        return self.n_blocks * self.tile

    def block_coords(self, j):
        """(block time, block row, block column) of block index j (raster order)."""
        _, nbh, nbw = self.nblocks3
        j = np.asarray(j)
        return j // (nbh * nbw), (j // nbw) % nbh, j % nbw

    def valid_counts(self) -> np.ndarray:
        """Tokens of every block, in block order."""
        bti, bhi, bwi = self.block_coords(np.arange(self.n_blocks))
        nt = np.minimum(self.bt, self.frames - bti * self.bt)
        nh = np.minimum(self.bh, self.grid_h - bhi * self.bh)
        nw = np.minimum(self.bw, self.grid_w - bwi * self.bw)
        return (nt * nh * nw).astype(np.int64)


def block_order(g: BlockGeom) -> np.ndarray:
    """src[k] = raster token index at block-order row k, or -1 for a padding row."""
    src = np.full(g.padded_tokens, -1, dtype=np.int64)
    for j in range(g.n_blocks):
        bti, bhi, bwi = (int(x) for x in g.block_coords(j))
        row = j * g.tile
        for t in range(bti * g.bt, min((bti + 1) * g.bt, g.frames)):
            for h in range(bhi * g.bh, min((bhi + 1) * g.bh, g.grid_h)):
                for w in range(bwi * g.bw, min((bwi + 1) * g.bw, g.grid_w)):
                    src[row] = (t * g.grid_h + h) * g.grid_w + w
                    row += 1
    return src


def block_of_token(g: BlockGeom) -> np.ndarray:
    """Block index of every raster token."""
    t, h, w = np.unravel_index(np.arange(g.tokens), (g.frames, g.grid_h, g.grid_w))
    _, nbh, nbw = g.nblocks3
    return ((t // g.bt) * nbh + h // g.bh) * nbw + w // g.bw


def local_mask(g: BlockGeom, r: int) -> np.ndarray:
    """M_local [n_blocks, n_blocks]: block rows and columns within floor(r/2)."""
    _, bhi, bwi = g.block_coords(np.arange(g.n_blocks))
    half = int(r) // 2
    return (np.abs(bhi[:, None] - bhi[None, :]) <= half) & (np.abs(bwi[:, None] - bwi[None, :]) <= half)


def attention_in_raster(chunks_k, chunks_v, q, g: BlockGeom, bits, scale: float):
    """Attention of one head in raster token order.

    chunks_k, chunks_v: lists (logical order) of [tokens, D] arrays; q [tokens, D];
    bits [n_blocks, n_live * n_blocks] keep set of query block i over the
    window's (chunk, block) pairs.  A query token of block i attends to every
    token of every kept (chunk, block); float64 masked softmax.
    Returns (O [tokens, D], LSE [tokens]).
    """
    nb = g.n_blocks
    blk = block_of_token(g)
    K = np.concatenate(chunks_k, axis=0)
    V = np.concatenate(chunks_v, axis=0)
    key_block = np.concatenate([pos * nb + blk for pos in range(len(chunks_k))])
    O = np.zeros_like(q, dtype=np.float64)
    LSE = np.full(q.shape[0], -np.inf)
    for i in range(nb):
        rows = np.nonzero(blk == i)[0]
        cols = np.nonzero(bits[i][key_block])[0]
        if rows.size == 0 or cols.size == 0:
            continue
        S = (q[rows] @ K[cols].T) * scale
        m = S.max(axis=1)
        P = np.exp(S - m[:, None])
        l = P.sum(axis=1)
        O[rows] = (P @ V[cols]) / l[:, None]
        LSE[rows] = m + np.log(l)
    return O, LSE


def block_means(x, g: BlockGeom) -> np.ndarray:
    """Per-block means [n_blocks, D] float32 of raster tokens x [tokens, D]: the
    block's valid tokens in block order, summed sequentially in float32, then
    divided once by their count (the pooling of Eq. 4 on 3-D blocks)."""
    x32 = np.asarray(x, dtype=np.float32)
    src = block_order(g).reshape(g.n_blocks, g.tile)
    D = x32.shape[1]
    acc = np.zeros((g.n_blocks, D), dtype=np.float32)
    for r in range(g.tile):
        idx = src[:, r]
        rows = np.where(idx[:, None] >= 0, x32[np.maximum(idx, 0)], np.float32(0))
        acc = (acc + rows).astype(np.float32)
    n = g.valid_counts().astype(np.float32)[:, None]
    return (acc / n).astype(np.float32)


def attention_in_raster_bwd(chunks_k, chunks_v, q, do, g: BlockGeom, bits, scale: float):
    """Gradients of ``attention_in_raster`` for an upstream gradient do [tokens, D]:
    per query block, the kept tokens' softmax P, delta = <do, o>, dS = P (do V^T -
    delta); dq = scale dS K, dK += scale dS^T q, dV += P^T do (float64).
    Returns (dq [tokens, D], dk list, dv list) with the chunks' shapes."""
    nb = g.n_blocks
    blk = block_of_token(g)
    K = np.concatenate(chunks_k, axis=0)
    V = np.concatenate(chunks_v, axis=0)
    key_block = np.concatenate([pos * nb + blk for pos in range(len(chunks_k))])
    dq = np.zeros_like(q, dtype=np.float64)
    dK = np.zeros_like(K, dtype=np.float64)
    dV = np.zeros_like(V, dtype=np.float64)
    for i in range(nb):
        rows = np.nonzero(blk == i)[0]
        cols = np.nonzero(bits[i][key_block])[0]
        if rows.size == 0 or cols.size == 0:
            continue
        S = (q[rows] @ K[cols].T) * scale
        P = np.exp(S - S.max(axis=1, keepdims=True))
        P /= P.sum(axis=1, keepdims=True)
        O = P @ V[cols]
        dP = do[rows] @ V[cols].T
        dS = P * (dP - (do[rows] * O).sum(axis=1, keepdims=True))
        dq[rows] = scale * (dS @ K[cols])
        dK[cols] += scale * (dS.T @ q[rows])
        dV[cols] += P.T @ do[rows]
    n = chunks_k[0].shape[0]
    return dq, [dK[p * n:(p + 1) * n] for p in range(len(chunks_k))], [dV[p * n:(p + 1) * n] for p in range(len(chunks_k))]
