"""Pins of the composed Eq. 4 block mask (oracle.block_sparse_mask).

Hand-derived keep sets on grids small enough to write out: the content rule
is applied over every candidate first and M_local intersected afterwards
(Sec. 2.3.1 (a)(b), Eq. 4), so a top-k pick outside the r x r window is lost
rather than replaced, and forced blocks are clipped by the window too; block
time does not enter the spatial window.  On raster tiles without a local
window the composition reduces to the plain rules.
"""

import numpy as np
import pytest

import oracle
from oracle import BlockGeom, KeepRule, RingModel, TopkRule


def _ring_with_keys(keys, pin_sink):
    """One chunk per entry of ``keys`` ([tokens, D] arrays), B = H = 1."""
    ring = RingModel(len(keys), pin_sink)
    for k in keys:
        ring.append(k[None, :, None, :], np.zeros_like(k)[None, :, None, :])
    return ring


def _row(*bits):
    return [bool(b) for b in bits]


def test_topk_pick_outside_window_is_lost_and_forced_blocks_are_clipped():
    # one frame on a 1 x 24 grid, blocks (1, 1, 8): three blocks in a row
    g = BlockGeom(1, 1, 24, 1, 1, 8)
    assert g.nblocks3 == (1, 1, 3)
    D = 4
    prior = np.zeros((24, D))
    prior[:, 0] = np.repeat([1.0, 2.0, 3.0], 8)       # pooled scores 1, 2, 3: block 2 ranks first
    current = np.zeros((24, D))
    ring = _ring_with_keys([prior, current], pin_sink=False)
    q = np.zeros((1, 24, 1, D))
    q[..., 0] = 1.0
    rule = TopkRule(budget=1, keep_sink=False, keep_current=True)

    # no local window: the prior chunk's block 2 plus every current block
    full = oracle.block_sparse_mask(ring, rule, q=q, geom=g)
    assert full[0, 0].tolist() == [_row(0, 0, 1, 1, 1, 1)] * 3

    # r = 1: only the same block column; query block 0 loses its top-k pick
    # (prior block 2) and does not get prior block 0 in its place
    r1 = oracle.block_sparse_mask(ring, rule, q=q, geom=g, local_r=1)
    assert r1[0, 0].tolist() == [_row(0, 0, 0, 1, 0, 0),
                                 _row(0, 0, 0, 0, 1, 0),
                                 _row(0, 0, 1, 0, 0, 1)]

    # r = 3: neighbouring columns; current blocks outside the window are clipped
    r3 = oracle.block_sparse_mask(ring, rule, q=q, geom=g, local_r=3)
    assert r3[0, 0].tolist() == [_row(0, 0, 0, 1, 1, 0),
                                 _row(0, 0, 1, 1, 1, 1),
                                 _row(0, 0, 1, 0, 1, 1)]


def test_forced_sink_and_current_clipped_across_block_times():
    # two frames with b_t = 1 (two block times) on a 1 x 16 grid, b_w = 8:
    # blocks 0 (t0, c0), 1 (t0, c1), 2 (t1, c0), 3 (t1, c1)
    g = BlockGeom(2, 1, 16, 1, 1, 8)
    assert g.nblocks3 == (2, 1, 2)
    z = np.zeros((32, 2))
    ring = _ring_with_keys([z, z], pin_sink=True)
    same_col = [_row(1, 0, 1, 0, 1, 0, 1, 0), _row(0, 1, 0, 1, 0, 1, 0, 1)]
    want = [same_col[0], same_col[1], same_col[0], same_col[1]]
    # p = 0: only the forced sink and current blocks, then the window
    forced = oracle.block_sparse_mask(ring, KeepRule(7, 0.0), geom=g, local_r=1)
    assert forced[0, 0].tolist() == want
    # p = 1 with nothing forced: every draw keeps, the window decides alone
    drawn = oracle.block_sparse_mask(ring, KeepRule(7, 1.0, False, False), geom=g, local_r=1)
    assert drawn[0, 0].tolist() == want
    # without the window everything is kept
    assert oracle.block_sparse_mask(ring, KeepRule(7, 0.0), geom=g).all()


def test_raster_tiles_reduce_to_the_plain_rules():
    rng = np.random.default_rng(5)
    ring = RingModel(4, True)
    for _ in range(4):
        ring.append(rng.standard_normal((2, 300, 3, 8)), rng.standard_normal((2, 300, 3, 8)))
    q = rng.standard_normal((2, 300, 3, 8))
    kr = KeepRule(11, 0.4)
    assert np.array_equal(oracle.block_sparse_mask(ring, kr, T=128), oracle.keep_bits(ring, 128, kr))
    tr = TopkRule(2)
    assert np.array_equal(oracle.block_sparse_mask(ring, tr, q=q, T=128), oracle.topk_bits(ring, q, 128, tr))


def test_block_bernoulli_draws_follow_the_block_index():
    """With 3-D blocks the Bernoulli draw of (query block i, chunk, block t) is the
    one of tile indices i and t: the same bits as raster tiles of one block each."""
    g = BlockGeom(3, 10, 12, 2, 4, 8)
    rng = np.random.default_rng(6)
    ring = RingModel(3, True)
    for _ in range(3):
        ring.append(rng.standard_normal((1, g.tokens, 2, 4)), rng.standard_normal((1, g.tokens, 2, 4)))
    rule = KeepRule(13, 0.5)
    got = oracle.block_sparse_mask(ring, rule, geom=g)
    # a ring whose chunks have exactly n_blocks rows, tiled by 1, draws the same bits
    meta = RingModel(3, True)
    for c in ring.logical_chunks():
        meta.live.append(oracle.ring.Chunk(c.seq, c.sink, np.zeros((1, g.n_blocks, 2, 1)), None))
    assert np.array_equal(got, oracle.keep_bits(meta, 1, rule))


def test_argument_errors():
    ring = _ring_with_keys([np.zeros((8, 2))], pin_sink=False)
    with pytest.raises(ValueError):
        oracle.block_sparse_mask(ring, KeepRule(1, 0.5), T=8, local_r=3)
    with pytest.raises(ValueError):
        oracle.block_sparse_mask(ring, KeepRule(1, 0.5))
    with pytest.raises(ValueError):
        oracle.block_sparse_mask(ring, TopkRule(1), T=8)
