"""Oracle of the per-(head, query tile) key-tile keep set (test infrastructure only).

What the paper fixes (Sec. 2.3.1, block-sparse causal attention, Eq. 4): the
token grid is split into non-overlapping blocks; each head gets a block-level
mask that is the intersection of the temporal causal mask (a chunk
attends only to itself and to earlier chunks) with a content-dependent top-k
keep set; attention is then evaluated over the kept blocks only.

What stands in for the content rule here (not in the paper, so parity against
the paper is unpinned): for every (batch b, head h, query tile i) and every key
tile (chunk c, tile t) of the window,

* keep when c is the pinned first chunk and ``keep_sink``;
* keep when c is the current chunk and ``keep_current``;
* otherwise keep with probability ``p_prior``, decided by a counter hash:
  ``x = seed; for f in (b, h, seq(current), i, seq(c), t): x = splitmix64(x ^ f)``
  and keep iff ``(x >> 32) < thr`` with ``thr = 2**32`` for ``p >= 1`` else
  ``floor(p * 2**32)`` evaluated in IEEE double.

The hash is keyed on append sequence numbers, never on storage slots, so the
keep set depends only on the logical content of the window.

``splitmix64`` is one step of the SplitMix64 generator of Steele, Lea and Flood
("Fast splittable pseudorandom number generators", OOPSLA 2014): add the
golden-ratio increment 0x9E3779B97F4A7C15 to the state, then apply the 64-bit
finaliser z ^= z >> 30; z *= 0xBF58476D1CE4E5B9; z ^= z >> 27;
z *= 0x94D049BB133111EB; z ^= z >> 31 (all modulo 2**64).

Tiles: each chunk of L tokens is tiled on its own from its first token into
``NT = ceil(L / T)`` tiles; the last holds ``L - (NT - 1) * T`` tokens.  Key
tile ``j`` of the window is tile ``j % NT`` of the chunk at logical position
``j // NT``; query tile ``i`` covers tokens ``[i*T, min((i+1)*T, L))`` of the
current chunk.
"""

from dataclasses import dataclass

import numpy as np

_GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


@dataclass(frozen=True)
class KeepRule:
    seed: int
    p_prior: float
    keep_sink: bool = True
    keep_current: bool = True


def splitmix64(x):
    """One SplitMix64 step from state ``x`` (uint64 array or int); returns uint64."""
    z = np.asarray(x, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = z + _GAMMA
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
        z = z ^ (z >> np.uint64(31))
    return z


def keep_threshold(p: float) -> int:
    """Integer threshold on the upper 32 hash bits for keep probability p."""
    p = float(p)
    if not (0.0 <= p <= 1.0):
        raise ValueError("p_prior must lie in [0, 1]")
    if p >= 1.0:
        return 1 << 32
    return int(np.floor(p * 4294967296.0))


def tile_geometry(L: int, T: int):
    """(number of tiles per chunk, valid tokens in the last tile)."""
    if L < 1 or T < 1:
        raise ValueError("L and T must be >= 1")
    nt = -(-L // T)
    return nt, L - (nt - 1) * T


def keep_bits(ring, T: int, rule: KeepRule) -> np.ndarray:
    """Boolean keep set [B, H, NQ, NK] for the ring's current chunk.

    NQ = tiles of the current chunk; NK = n_live * NT logical key tiles.
    """
    chunks = ring.logical_chunks()
    cur = ring.current
    B, L, H, _ = cur.k.shape
    nt, _ = tile_geometry(L, T)
    thr = np.uint64(keep_threshold(rule.p_prior))
    b = np.arange(B, dtype=np.uint64)[:, None, None, None, None]
    h = np.arange(H, dtype=np.uint64)[None, :, None, None, None]
    i = np.arange(nt, dtype=np.uint64)[None, None, :, None, None]
    seqs = np.array([c.seq for c in chunks], dtype=np.uint64)[None, None, None, :, None]
    t = np.arange(nt, dtype=np.uint64)[None, None, None, None, :]
    x = np.full((1, 1, 1, 1, 1), rule.seed & 0xFFFFFFFFFFFFFFFF, dtype=np.uint64)
    for field in (b, h, np.uint64(cur.seq), i, seqs, t):
        x = splitmix64(x ^ field)
    x = np.broadcast_to(x, (B, H, nt, len(chunks), nt))
    bits = (x >> np.uint64(32)) < thr
    for pos, c in enumerate(chunks):
        forced = (c.sink and rule.keep_sink) or (c.seq == cur.seq and rule.keep_current)
        if forced:
            bits[:, :, :, pos, :] = True
    return bits.reshape(B, H, nt, len(chunks) * nt)


def lists_from_bits(bits: np.ndarray, nk_cap: int):
    """(counts, idx, mask) in the list layout: row stride nk_cap, words ceil(nk_cap/32).

    counts [B,H,NQ] int32; idx [B,H,NQ,nk_cap] int32 ascending, padded with -1;
    mask [B,H,NQ,ceil(nk_cap/32)] uint32, bit (j % 32) of word j // 32 set iff kept.
    """
    B, H, NQ, NK = bits.shape
    if NK > nk_cap:
        raise ValueError("more key tiles than the list capacity")
    nw = -(-nk_cap // 32)
    counts = bits.sum(axis=-1).astype(np.int32)
    idx = np.full((B, H, NQ, nk_cap), -1, dtype=np.int32)
    for bb in range(B):
        for hh in range(H):
            for ii in range(NQ):
                kept = np.nonzero(bits[bb, hh, ii])[0]
                idx[bb, hh, ii, : kept.size] = kept
    padded = np.zeros((B, H, NQ, nw * 32), dtype=bool)
    padded[..., :NK] = bits
    # little bit order: key tile j lands in bit (j % 32) of little-endian word j // 32
    mask = np.packbits(padded, axis=-1, bitorder="little").view("<u4").astype(np.uint32)
    return counts, idx, mask
