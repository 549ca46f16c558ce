"""Pins of the top-k oracle (Eq. 4 content-adaptive selection; App. L, Eq. 10).

Each pin checks the oracle against something outside it:
* means and scores worked out by hand on small integers;
* float32 facts: the order of the additions and unfused products change
  these results, so a float64 or a fused evaluation fails;
* the selection rule on hand-made score rows (highest first, lower index on
  ties, candidates only, budget extremes);
* agreement with a float64 evaluation of the same definition wherever the
  k-th and (k+1)-th scores of a row are not near-tied;
* invariances: exact power-of-two scaling of Q or K changes no bit.
Planted mistakes at the end must each fail at least one of them.
"""

import numpy as np
import pytest

import oracle
import oracle.topk as topk

F32 = np.float32


def _ring(B, L, H, T, n_chunks, pin, seed, max_chunks=None, d=8):
    rng = np.random.default_rng(seed)
    ring = oracle.RingModel(max_chunks or n_chunks, pin)
    for _ in range(n_chunks):
        # bf16-representable values: N(0,1) rounded to 8 significant bits
        k = rng.standard_normal((B, L, H, d)).astype(np.float32)
        k = (k.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32).astype(np.float64)
        ring.append(k, np.zeros_like(k))
    q = rng.standard_normal((B, L, H, d)).astype(np.float32)
    q = (q.view(np.uint32) & np.uint32(0xFFFF0000)).view(np.float32).astype(np.float64)
    return ring, q


def test_pooled_means_hand_values():
    x = np.array([[1, 2], [3, 4], [5, 6]], dtype=np.float64)     # L = 3, D = 2
    m = topk.pooled_means(x, 2)                                   # tiles {0,1}, {2}
    assert m.dtype == np.float32
    assert np.array_equal(m, np.array([[2, 3], [5, 6]], dtype=F32))


def test_pooled_mean_of_equal_rows_is_the_row():
    # n copies of one bf16 row sum exactly; the mean divides by the VALID count
    rng = np.random.default_rng(3)
    row = (rng.standard_normal(16).astype(F32).view(np.uint32) & np.uint32(0xFFFF0000)).view(F32)
    for L, T in ((7, 4), (9, 4), (1, 8), (130, 64)):
        m = topk.pooled_means(np.tile(row, (L, 1)), T)
        assert np.array_equal(m, np.tile(row, (m.shape[0], 1))), (L, T)


def test_block_scores_hand_values():
    qm = np.array([[1, 2], [-1, 0]], dtype=F32)
    km = np.array([[3, 4], [5, -6], [0, 1]], dtype=F32)
    assert np.array_equal(topk.block_scores(qm, km), np.array([[11, -7, 2], [-3, -5, 0]], dtype=F32))


def test_block_scores_are_float32_in_order_without_fusion():
    # order of the additions in float32: (1e8 - 1e8) + 1 = 1, but (1 + 1e8) - 1e8 = 0
    # (1 + 1e8 rounds to 1e8); a float64 or reordered evaluation gives 1 for both
    assert topk.block_scores(np.ones((1, 3), F32), np.array([[1e8, -1e8, 1]], F32))[0, 0] == 1.0
    assert topk.block_scores(np.ones((1, 3), F32), np.array([[1, 1e8, -1e8]], F32))[0, 0] == 0.0
    # rounded products: fl(a*a) - fl(a*a) = 0, while a fused evaluation leaves -2^-24
    a = F32(1 + 2.0 ** -12)
    s = topk.block_scores(np.array([[a, a]], F32), np.array([[a, -a]], F32))[0, 0]
    assert s == 0.0 and np.float64(a) * np.float64(a) != np.float64(F32(np.float64(a) * np.float64(a)))


def test_select_topk_rule():
    s = np.array([5, 7, 7, 1, 9], dtype=F32)
    allc = np.ones(5, dtype=bool)
    assert np.nonzero(topk.select_topk(s, allc, 3))[0].tolist() == [1, 2, 4]
    assert np.nonzero(topk.select_topk(s, allc, 2))[0].tolist() == [1, 4]           # tie -> lower index
    no4 = allc.copy()
    no4[4] = False
    assert np.nonzero(topk.select_topk(s, no4, 2))[0].tolist() == [1, 2]            # candidates only
    assert np.nonzero(topk.select_topk(np.full(4, 2, F32), np.ones(4, bool), 2))[0].tolist() == [0, 1]
    assert not topk.select_topk(s, allc, 0).any()
    assert topk.select_topk(s, allc, 99).all()
    neg = np.array([-3, -1, -2, -np.inf, np.inf], dtype=F32)
    assert np.nonzero(topk.select_topk(neg, allc, 2))[0].tolist() == [1, 4]
    # the order key orders like the real line, with -0 just below +0
    vals = np.array([-np.inf, -2, -0.5, -0.0, 0.0, 1e-30, 3, np.inf], dtype=F32)
    assert np.all(np.diff(topk.order_key(vals).astype(np.int64)) > 0)


def test_topk_bits_forced_tiles_and_budget_extremes():
    ring, q = _ring(1, 10, 2, 4, 4, True, seed=11)                 # NT = 3, NK = 12
    nt = 3
    forced = np.zeros(12, bool)
    forced[0:3] = True                                              # pinned chunk
    forced[9:12] = True                                             # current chunk
    b0 = topk.topk_bits(ring, q, 4, oracle.TopkRule(0))
    assert np.array_equal(b0, np.broadcast_to(forced, b0.shape))
    assert topk.topk_bits(ring, q, 4, oracle.TopkRule(6)).all()
    assert topk.topk_bits(ring, q, 4, oracle.TopkRule(12, False, False)).all()
    b3 = topk.topk_bits(ring, q, 4, oracle.TopkRule(3))
    assert np.all(b3.sum(-1) == 6 + 3) and np.all(b3[..., forced])
    bn = topk.topk_bits(ring, q, 4, oracle.TopkRule(5, False, False))
    assert np.all(bn.sum(-1) == 5)
    assert nt * ring.n_live == b0.shape[-1]


def test_topk_agrees_with_float64_away_from_near_ties():
    ring, q = _ring(2, 37, 3, 8, 5, True, seed=5, d=16)
    k = 4
    bits = topk.topk_bits(ring, q, 8, oracle.TopkRule(k))
    nt = 5
    checked = 0
    for b in range(2):
        for h in range(3):
            qm = np.stack([q[b, i * 8:(i + 1) * 8, h].mean(0) for i in range(nt)])
            km = np.concatenate([np.stack([c.k[b, i * 8:(i + 1) * 8, h].mean(0) for i in range(nt)])
                                 for c in ring.logical_chunks()])
            s = qm @ km.T                                               # float64 reference scores
            for i in range(nt):
                cand = np.arange(nt, 4 * nt)                             # earlier non-pinned chunks
                order = cand[np.argsort(-s[i, cand], kind="stable")]
                gap = s[i, order[k - 1]] - s[i, order[k]]
                if gap > 1e-3:
                    assert set(np.nonzero(bits[b, h, i, nt:4 * nt])[0] + nt) == set(order[:k].tolist())
                    checked += 1
    assert checked >= 20


def test_topk_exact_power_of_two_scaling_changes_nothing():
    ring, q = _ring(1, 40, 2, 8, 4, False, seed=9, d=16)
    rule = oracle.TopkRule(3, False, False)
    base = topk.topk_bits(ring, q, 8, rule)
    assert np.array_equal(base, topk.topk_bits(ring, q * 4.0, 8, rule))
    for c in ring.live:
        c.k = c.k * 0.5
    assert np.array_equal(base, topk.topk_bits(ring, q, 8, rule))


def test_topk_budget_eq10():
    # S = S_ref gives rho * N; the budget scales linearly with S; k_min is a floor
    assert topk.topk_budget(1.0, 1560, 1560, 200) == 200
    assert topk.topk_budget(0.5, 3120, 1560, 200) == 200
    assert topk.topk_budget(1.0, 780, 1560, 201) == 100
    assert topk.topk_budget(1.0, 10, 1560, 100) == 4
    assert topk.topk_budget(0.7, 1560, 1560, 10, k_min=0) == 7


# ---- planted mistakes ------------------------------------------------------

TOPK_PINS = [
    test_pooled_means_hand_values,
    test_pooled_mean_of_equal_rows_is_the_row,
    test_block_scores_hand_values,
    test_block_scores_are_float32_in_order_without_fusion,
    test_select_topk_rule,
    test_topk_bits_forced_tiles_and_budget_extremes,
    test_topk_agrees_with_float64_away_from_near_ties,
]


def _fails_some(tests):
    for t in tests:
        try:
            t()
        except AssertionError:
            return True
    return False


def _means_over_T(x, T):
    x32 = np.asarray(x, dtype=np.float32)
    L, D = x32.shape
    nt, _ = oracle.tile_geometry(L, T)
    xp = np.zeros((nt * T, D), np.float32)
    xp[:L] = x32
    return (xp.reshape(nt, T, D).sum(1, dtype=np.float32) / F32(T)).astype(np.float32)


def _scores_f64(qm, km):
    return (np.asarray(qm, np.float64) @ np.asarray(km, np.float64).T).astype(np.float32)


_REAL_SCORES = topk.block_scores


def _scores_reversed_columns(qm, km):
    return _REAL_SCORES(qm, km)[:, ::-1]


def _select_high_index_ties(scores, candidate, k):
    keep = np.zeros(scores.shape[0], dtype=bool)
    cand = np.nonzero(candidate)[0]
    if k <= 0 or cand.size == 0:
        return keep
    key = topk.order_key(scores[cand]).astype(np.int64)
    order = np.lexsort((-cand, -key))
    keep[cand[order[:k]]] = True
    return keep


def _select_lowest(scores, candidate, k):
    keep = np.zeros(scores.shape[0], dtype=bool)
    cand = np.nonzero(candidate)[0]
    order = np.lexsort((cand, topk.order_key(scores[cand]).astype(np.int64)))
    keep[cand[order[:max(k, 0)]]] = True
    return keep


@pytest.mark.parametrize("name,attr,slip", [
    ("mean divides by T", "pooled_means", _means_over_T),
    ("float64 scores", "block_scores", _scores_f64),
    ("reversed key columns", "block_scores", _scores_reversed_columns),
    ("ties to the higher index", "select_topk", _select_high_index_ties),
    ("lowest scores kept", "select_topk", _select_lowest),
])
def test_topk_slips_are_caught(monkeypatch, name, attr, slip):
    monkeypatch.setattr(topk, attr, slip)
    assert _fails_some(TOPK_PINS), name
