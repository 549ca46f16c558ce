"""Pins of the 3-D block tiling oracle (Sec. 2.3.1 (a), Eq. 4 structural masks).

Hand-derived block orders, counts and window masks on small grids; the block
order is a bijection; attention in raster order equals plain dense attention
when every block is kept and equals attention over exactly the tokens of the
kept blocks otherwise; block means follow the fixed float32 rule.
"""

import numpy as np

import oracle
from oracle import blocks


def test_block_order_hand_example():
    # 3 frames on a 3 x 5 grid, blocks (2, 2, 2): block grid (2, 2, 3), 8 rows per block
    g = oracle.BlockGeom(3, 3, 5, 2, 2, 2)
    assert g.nblocks3 == (2, 2, 3) and g.n_blocks == 12 and g.tile == 8
    src = oracle.block_order(g)
    # raster index = t*15 + h*5 + w
    assert src[0:8].tolist() == [0, 1, 5, 6, 15, 16, 20, 21]            # t 0-1, h 0-1, w 0-1
    assert src[16:24].tolist() == [4, 9, 19, 24, -1, -1, -1, -1]        # w = 4 only
    assert src[24:32].tolist() == [10, 11, 25, 26, -1, -1, -1, -1]      # h = 2 only
    assert src[48:56].tolist() == [30, 31, 35, 36, -1, -1, -1, -1]      # t = 2 only
    assert src[88:96].tolist() == [44] + [-1] * 7                       # t 2, h 2, w 4
    assert g.valid_counts().tolist() == [8, 8, 4, 4, 4, 2, 4, 4, 2, 2, 2, 1]


def test_block_order_is_a_bijection_onto_valid_rows():
    for g in (oracle.BlockGeom(3, 68, 120), oracle.BlockGeom(3, 30, 52), oracle.BlockGeom(1, 9, 17, 1, 4, 4)):
        src = oracle.block_order(g)
        valid = src[src >= 0]
        assert np.array_equal(np.sort(valid), np.arange(g.tokens))
        counts = (src.reshape(g.n_blocks, g.tile) >= 0).sum(1)
        assert np.array_equal(counts, g.valid_counts())
        # valid rows first inside every block
        per = src.reshape(g.n_blocks, g.tile) >= 0
        assert all(np.all(row[:c]) and not np.any(row[c:]) for row, c in zip(per, counts))
        assert np.array_equal(oracle.block_of_token(g)[valid], np.repeat(np.arange(g.n_blocks), counts))


def test_local_mask_hand_example():
    g = oracle.BlockGeom(1, 4, 4, 1, 1, 1)          # 4 x 4 block grid, blocks = tokens
    m = oracle.local_mask(g, 3)                      # half-width 1
    assert m[0].reshape(4, 4).astype(int).tolist() == [[1, 1, 0, 0], [1, 1, 0, 0], [0, 0, 0, 0], [0, 0, 0, 0]]
    assert m[5].reshape(4, 4).astype(int).tolist() == [[1, 1, 1, 0], [1, 1, 1, 0], [1, 1, 1, 0], [0, 0, 0, 0]]
    assert np.array_equal(m, m.T)
    assert oracle.local_mask(g, 7).all()
    assert np.array_equal(oracle.local_mask(g, 1), np.eye(16, dtype=bool))
    # block time does not enter the spatial window
    g2 = oracle.BlockGeom(4, 2, 2, 2, 1, 1)          # 2 block times, 2 x 2 block grid
    m2 = oracle.local_mask(g2, 1)
    assert m2[0].astype(int).tolist() == [1, 0, 0, 0, 1, 0, 0, 0]


def _rand(shape, rng):
    return rng.standard_normal(shape)


def test_attention_in_raster_dense_and_single_block():
    rng = np.random.default_rng(4)
    g = oracle.BlockGeom(3, 3, 5, 2, 2, 2)
    D = 8
    ks = [_rand((g.tokens, D), rng) for _ in range(2)]
    vs = [_rand((g.tokens, D), rng) for _ in range(2)]
    q = _rand((g.tokens, D), rng)
    scale = 0.3
    nb = g.n_blocks
    O, LSE = oracle.attention_in_raster(ks, vs, q, g, np.ones((nb, 2 * nb), bool), scale)
    K, V = np.concatenate(ks), np.concatenate(vs)
    S = q @ K.T * scale
    P = np.exp(S - S.max(1, keepdims=True))
    assert np.allclose(O, (P / P.sum(1, keepdims=True)) @ V, atol=1e-12)
    assert np.allclose(LSE, np.log(np.exp(S).sum(1)), atol=1e-12)
    # only block 5 of chunk 1 kept: exactly its tokens
    bits = np.zeros((nb, 2 * nb), bool)
    bits[:, nb + 5] = True
    O1, _ = oracle.attention_in_raster(ks, vs, q, g, bits, scale)
    toks = np.nonzero(oracle.block_of_token(g) == 5)[0]
    S1 = q @ ks[1][toks].T * scale
    P1 = np.exp(S1 - S1.max(1, keepdims=True))
    assert np.allclose(O1, (P1 / P1.sum(1, keepdims=True)) @ vs[1][toks], atol=1e-12)


def test_block_means_float32_rule():
    g = oracle.BlockGeom(3, 3, 5, 2, 2, 2)
    x = np.arange(g.tokens, dtype=np.float64)[:, None] * np.ones((1, 2))
    m = oracle.block_means(x, g)
    src = oracle.block_order(g).reshape(g.n_blocks, g.tile)
    want = np.array([[x[s[s >= 0], 0].mean()] * 2 for s in src], dtype=np.float32)
    assert np.array_equal(m, want)                   # small integers: exact in float32
    row = np.float32([1.5, -2.25, 3.0])
    eq = oracle.block_means(np.tile(row, (g.tokens, 1)), g)
    assert np.array_equal(eq, np.tile(row, (g.n_blocks, 1)))


def test_attention_in_raster_bwd_central_differences():
    """Gradients of raster-order block attention against central differences
    of attention_in_raster, with a partial block set and the local mask."""
    rng = np.random.default_rng(8)
    g = oracle.BlockGeom(3, 3, 5, 2, 2, 2)
    D, nb = 3, g.n_blocks
    ks = [_rand((g.tokens, D), rng) for _ in range(2)]
    vs = [_rand((g.tokens, D), rng) for _ in range(2)]
    q = _rand((g.tokens, D), rng)
    do = _rand((g.tokens, D), rng)
    bits = (rng.random((nb, 2 * nb)) < 0.5) & np.tile(oracle.local_mask(g, 3), (1, 2))
    bits[nb - 1] = False                            # a query block with no kept block
    scale = 0.6
    dq, dk, dv = oracle.attention_in_raster_bwd(ks, vs, q, do, g, bits, scale)

    def f():
        O, _ = oracle.attention_in_raster(ks, vs, q, g, bits, scale)
        return float((O * do).sum())

    eps = 1e-6
    for arr, grad in [(q, dq), (ks[0], dk[0]), (ks[1], dk[1]), (vs[0], dv[0]), (vs[1], dv[1])]:
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            keep = arr[idx]
            arr[idx] = keep + eps
            fp = f()
            arr[idx] = keep - eps
            fm = f()
            arr[idx] = keep
            num[idx] = (fp - fm) / (2 * eps)
        assert np.allclose(grad, num, atol=1e-7, rtol=1e-6)
    assert np.all(dq[oracle.block_of_token(g) == nb - 1] == 0)
