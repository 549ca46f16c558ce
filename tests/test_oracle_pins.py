"""Pins of the CPU oracle against facts that do not come from the oracle itself.

* brute force: per-query, per-key float64 loops with math.exp over every keep
  mask of a micro shape (Eq. 4: attention restricted to the kept blocks);
* a library routine: torch's scaled_dot_product_attention in float64 with a
  boolean mask expanded from the kept tiles, and without a mask when every
  tile is kept (dense attention over the window = the all-kept special case);
* closed forms: identical keys (or a zero query) give uniform weights, so the
  output is the mean of V over exactly the kept, valid keys and the LSE is
  log(number of kept keys); V == 1 gives O == 1;
* invariants: softmax rows sum to one, token order inside a tile does not
  matter, and the window's eviction history does not matter;
* the published SplitMix64 outputs and the binomial statistics of the
  Bernoulli keep stand-in; the workload tile geometry.
"""

import itertools
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import KeepRule, RingModel

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def _bf16_values(rng, shape):
    x = torch.from_numpy(rng.standard_normal(shape).astype(np.float32)).to(torch.bfloat16)
    return x.double().numpy()


def _ring(rng, B, L, H, D, n_chunks, max_chunks, pin_sink, evict_each=True):
    ring = RingModel(max_chunks, pin_sink)
    for _ in range(n_chunks):
        if ring.n_live == max_chunks:
            ring.evict(1)
        ring.append(_bf16_values(rng, (B, L, H, D)), _bf16_values(rng, (B, L, H, D)))
    return ring


# --------------------------------------------------------------------------
# SplitMix64, thresholds, geometry
# --------------------------------------------------------------------------

def _golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return [ln.split("#")[0].strip() for ln in f if ln.split("#")[0].strip()]


def test_splitmix64_published_outputs():
    want = [int(x, 16) for x in _golden_lines("splitmix64_seed0.txt")]
    gamma = 0x9E3779B97F4A7C15
    got = [int(oracle.splitmix64((k * gamma) % (1 << 64))) for k in range(4)]
    assert got == want
    # vectorised form agrees with the scalar form
    arr = oracle.splitmix64(np.array([(k * gamma) % (1 << 64) for k in range(4)], dtype=np.uint64))
    assert [int(v) for v in arr] == want


def test_keep_threshold():
    assert oracle.keep_threshold(0.0) == 0
    assert oracle.keep_threshold(1.0) == 1 << 32
    assert oracle.keep_threshold(0.25) == 1 << 30
    assert oracle.keep_threshold(0.5) == 1 << 31
    assert oracle.keep_threshold(0.15) == math.floor(0.15 * 2**32)
    with pytest.raises(ValueError):
        oracle.keep_threshold(1.5)
    with pytest.raises(ValueError):
        oracle.keep_threshold(-0.1)


def test_workload_geometry_golden():
    import synth
    rows = [ln.split() for ln in _golden_lines("workload_geometry.txt")]
    assert len(rows) == 4
    for name, gh, gw, L, T, nt, tail in rows:
        wl = synth.WORKLOADS[name]
        assert (wl.grid_h, wl.grid_w, wl.chunk_tokens, wl.tile) == (int(gh), int(gw), int(L), int(T))
        assert oracle.tile_geometry(int(L), int(T)) == (int(nt), int(tail))
    assert 30 * 52 == 1560  # S_ref of the adaptive budget is the 480P frame grid


# --------------------------------------------------------------------------
# Ring model
# --------------------------------------------------------------------------

def test_ring_capacity_and_sink():
    rng = _rng(1)
    ring = RingModel(3, pin_sink=True)
    for _ in range(3):
        ring.append(np.zeros((1, 2, 1, 4)), np.zeros((1, 2, 1, 4)))
    with pytest.raises(oracle.RingCapacityError):
        ring.append(np.zeros((1, 2, 1, 4)), np.zeros((1, 2, 1, 4)))
    ring.evict(1)
    assert [c.seq for c in ring.logical_chunks()] == [0, 2]
    assert ring.logical_chunks()[0].sink
    ring.evict(1)
    assert [c.seq for c in ring.logical_chunks()] == [0]
    with pytest.raises(oracle.RingEmptyError):
        ring.evict(1)
    assert ring.current.seq == 0
    del rng


def test_ring_no_sink_evicts_oldest():
    ring = RingModel(2, pin_sink=False)
    for _ in range(2):
        ring.append(np.zeros((1, 1, 1, 1)), np.zeros((1, 1, 1, 1)))
    ring.evict(1)
    assert [c.seq for c in ring.logical_chunks()] == [1]
    ring.append(np.zeros((1, 1, 1, 1)), np.zeros((1, 1, 1, 1)))
    assert [c.seq for c in ring.logical_chunks()] == [1, 2]


# --------------------------------------------------------------------------
# Keep set and lists
# --------------------------------------------------------------------------

def test_keep_forced_tiles_and_extremes():
    rng = _rng(2)
    ring = _ring(rng, 1, 40, 3, 4, n_chunks=5, max_chunks=4, pin_sink=True)
    nt, _ = oracle.tile_geometry(40, 16)
    bits = oracle.keep_bits(ring, 16, KeepRule(seed=7, p_prior=0.0))
    assert bits.shape == (1, 3, nt, 4 * nt)
    assert bits[..., :nt].all()            # pinned first chunk
    assert bits[..., 3 * nt:].all()        # current chunk
    assert not bits[..., nt:3 * nt].any()  # p = 0: no earlier tile
    bits1 = oracle.keep_bits(ring, 16, KeepRule(seed=7, p_prior=1.0))
    assert bits1.all()
    bits2 = oracle.keep_bits(ring, 16, KeepRule(seed=7, p_prior=0.0, keep_sink=False))
    assert not bits2[..., :nt].any()


def test_keep_statistics_1k_shape():
    """Kept fraction of earlier-chunk tiles within 5 sigma of p on the 1K shape."""
    B, H, L, T = 1, 12, 24480, 128
    ring = RingModel(5, pin_sink=True)
    z = np.broadcast_to(np.zeros(1), (B, L, H, 1))  # the keep set depends on metadata only
    for _ in range(5):
        ring.append(z, z)
    bits = oracle.keep_bits(ring, T, KeepRule(seed=0x5EED0002, p_prior=0.25))
    nt = 192
    prior = bits[..., nt:4 * nt]
    n = prior.size
    frac = prior.mean()
    sigma = math.sqrt(0.25 * 0.75 / n)
    assert abs(frac - 0.25) < 5 * sigma
    # rows are independent draws, not copies of one another
    rows = prior.reshape(-1, prior.shape[-1])
    assert not (rows[0] == rows[1]).all()
    # per-row counts spread like a binomial(576, 0.25): variance within 30 %
    var = rows.sum(axis=1).var()
    assert 0.7 * 576 * 0.25 * 0.75 < var < 1.3 * 576 * 0.25 * 0.75


def test_keep_eviction_history_invariance():
    """Same logical window reached by different append/evict interleavings."""
    z = np.zeros((1, 1, 2, 1))
    a = RingModel(5, True)
    for _ in range(8):
        if a.n_live == 5:
            a.evict(1)
        a.append(z, z)
    b = RingModel(5, True)
    for _ in range(5):
        b.append(z, z)
    b.evict(3)
    for _ in range(3):
        b.append(z, z)
    assert [c.seq for c in a.logical_chunks()] == [c.seq for c in b.logical_chunks()] == [0, 4, 5, 6, 7]
    rule = KeepRule(seed=99, p_prior=0.3)
    assert np.array_equal(oracle.keep_bits(a, 4, rule), oracle.keep_bits(b, 4, rule))


def test_lists_from_bits_layout():
    rng = _rng(3)
    bits = rng.random((1, 2, 3, 45)) < 0.4
    counts, idx, mask = oracle.lists_from_bits(bits, nk_cap=70)
    assert idx.shape == (1, 2, 3, 70) and mask.shape == (1, 2, 3, 3)
    for h in range(2):
        for i in range(3):
            kept = [j for j in range(45) if bits[0, h, i, j]]
            assert counts[0, h, i] == len(kept)
            assert list(idx[0, h, i, :len(kept)]) == kept
            assert (idx[0, h, i, len(kept):] == -1).all()
            words = mask[0, h, i]
            got = [j for j in range(96) if (int(words[j // 32]) >> (j % 32)) & 1]
            assert got == kept
            assert sum(bin(int(w)).count("1") for w in words) == counts[0, h, i]


# --------------------------------------------------------------------------
# Attention: brute force, library routine, closed forms, invariants
# --------------------------------------------------------------------------

def _brute_force(ring, q, bits, T, scale):
    """Explicit per-query / per-key loops with math.exp (no matrix algebra)."""
    B, L, H, D = q.shape
    nt = -(-L // T)
    chunks = ring.logical_chunks()
    O = np.zeros((B, L, H, D))
    LSE = np.zeros((B, H, L))
    for b in range(B):
        for h in range(H):
            for r in range(L):
                i = r // T
                keys = []
                for pos, c in enumerate(chunks):
                    for tok in range(L):
                        if bits[b, h, i, pos * nt + tok // T]:
                            keys.append((c.k[b, tok, h], c.v[b, tok, h]))
                if not keys:
                    LSE[b, h, r] = -math.inf
                    continue
                s = [scale * sum(q[b, r, h, d] * k[d] for d in range(D)) for k, _ in keys]
                m = max(s)
                w = [math.exp(x - m) for x in s]
                tot = sum(w)
                for d in range(D):
                    O[b, r, h, d] = sum(wi * v[d] for wi, (_, v) in zip(w, keys)) / tot
                LSE[b, h, r] = m + math.log(tot)
    return O, LSE


def test_brute_force_all_masks_micro():
    """Every one of the 2**12 keep masks of a micro shape (L=3, T=2, 3 chunks)."""
    rng = _rng(4)
    B, L, H, D, T = 1, 3, 1, 4, 2
    ring = _ring(rng, B, L, H, D, n_chunks=4, max_chunks=3, pin_sink=True)
    assert [c.seq for c in ring.logical_chunks()] == [0, 2, 3]
    q = _bf16_values(rng, (B, L, H, D))
    nq, nk = 2, 6
    scale = 0.5
    worst = 0.0
    for m in range(1 << (nq * nk)):
        bits = np.array([(m >> k) & 1 for k in range(nq * nk)], dtype=bool).reshape(1, 1, nq, nk)
        O, LSE = oracle.sparse_causal_attention(ring, q, bits, T, scale)
        Ob, LSEb = _brute_force(ring, q, bits, T, scale)
        assert np.array_equal(np.isneginf(LSE), np.isneginf(LSEb))
        fin = np.isfinite(LSEb)
        worst = max(worst, float(np.abs(O - Ob).max()), float(np.abs(LSE[fin] - LSEb[fin]).max(initial=0)))
    assert worst < 1e-12


def test_brute_force_ragged_tiles():
    """L=7 with T=3 (tail 1), four chunks, random keep rule, two heads, batch 2."""
    rng = _rng(5)
    B, L, H, D, T = 2, 7, 2, 5, 3
    ring = _ring(rng, B, L, H, D, n_chunks=6, max_chunks=4, pin_sink=True)
    q = _bf16_values(rng, (B, L, H, D))
    bits = oracle.keep_bits(ring, T, KeepRule(seed=11, p_prior=0.4))
    O, LSE = oracle.sparse_causal_attention(ring, q, bits, T, 0.3)
    Ob, LSEb = _brute_force(ring, q, bits, T, 0.3)
    assert np.abs(O - Ob).max() < 1e-12
    assert np.abs(LSE - LSEb).max() < 1e-12


def _sdpa_mask(ring, bits, L, T):
    B, H, nq, nk = bits.shape
    nt = -(-L // T)
    sk = ring.n_live * L
    mask = np.zeros((B, H, L, sk), dtype=bool)
    for b in range(B):
        for h in range(H):
            for i in range(nq):
                for j in np.nonzero(bits[b, h, i])[0]:
                    pos, t = divmod(int(j), nt)
                    mask[b, h, i * T:min((i + 1) * T, L), pos * L + t * T:pos * L + min((t + 1) * T, L)] = True
    return mask


def _sdpa(ring, q, mask, scale):
    B, L, H, D = q.shape
    Q = torch.from_numpy(q).permute(0, 2, 1, 3)
    K = torch.from_numpy(np.stack([np.concatenate([c.k[b] for c in ring.logical_chunks()], 0) for b in range(B)])).permute(0, 2, 1, 3)
    V = torch.from_numpy(np.stack([np.concatenate([c.v[b] for c in ring.logical_chunks()], 0) for b in range(B)])).permute(0, 2, 1, 3)
    m = None if mask is None else torch.from_numpy(mask)
    O = torch.nn.functional.scaled_dot_product_attention(Q, K.contiguous(), V.contiguous(), attn_mask=m, scale=scale)
    return O.permute(0, 2, 1, 3).numpy()


def test_library_sdpa_masked_tiny_shape():
    rng = _rng(6)
    B, L, H, D, T = 1, 192, 2, 128, 64
    ring = _ring(rng, B, L, H, D, n_chunks=4, max_chunks=3, pin_sink=True)
    q = _bf16_values(rng, (B, L, H, D))
    bits = oracle.keep_bits(ring, T, KeepRule(seed=12, p_prior=0.5))
    O, _ = oracle.sparse_causal_attention(ring, q, bits, T, 1 / math.sqrt(D))
    Ot = _sdpa(ring, q, _sdpa_mask(ring, bits, L, T), 1 / math.sqrt(D))
    assert np.abs(O - Ot).max() < 1e-10


def test_all_kept_is_dense_attention():
    rng = _rng(7)
    B, L, H, D, T = 1, 100, 3, 16, 32   # ragged: NT = 4, tail 4
    ring = _ring(rng, B, L, H, D, n_chunks=3, max_chunks=3, pin_sink=False)
    q = _bf16_values(rng, (B, L, H, D))
    bits = oracle.keep_bits(ring, T, KeepRule(seed=1, p_prior=1.0))
    assert bits.all()
    O, _ = oracle.sparse_causal_attention(ring, q, bits, T, 0.25)
    Ot = _sdpa(ring, q, None, 0.25)
    assert np.abs(O - Ot).max() < 1e-10


def test_closed_form_uniform_weights_pick_exact_keys():
    """Identical key rows: weights are uniform over the kept, valid keys only."""
    rng = _rng(8)
    B, L, H, D, T = 1, 10, 2, 4, 4        # NT = 3, tail 2
    ring = RingModel(3, pin_sink=True)
    krow = rng.standard_normal(D)
    vals = []
    for _ in range(3):
        k = np.broadcast_to(krow, (B, L, H, D)).copy()
        v = _bf16_values(rng, (B, L, H, D))
        vals.append(v)
        ring.append(k, v)
    q = _bf16_values(rng, (B, L, H, D))
    bits = oracle.keep_bits(ring, T, KeepRule(seed=3, p_prior=0.5))
    O, LSE = oracle.sparse_causal_attention(ring, q, bits, T, 0.7)
    nt = 3
    for h in range(H):
        for r in range(L):
            i = r // T
            sel = []
            for j in np.nonzero(bits[0, h, i])[0]:
                pos, t = divmod(int(j), nt)
                for tok in range(t * T, min((t + 1) * T, L)):
                    sel.append(vals[pos][0, tok, h])
            want = np.mean(sel, axis=0)
            assert np.abs(O[0, r, h] - want).max() < 1e-12
            s = 0.7 * float(q[0, r, h] @ krow)
            assert abs(LSE[0, h, r] - (s + math.log(len(sel)))) < 1e-12


def test_v_ones_and_row_sums():
    rng = _rng(9)
    B, L, H, D, T = 1, 50, 2, 8, 16
    ring = RingModel(4, pin_sink=True)
    for _ in range(4):
        ring.append(_bf16_values(rng, (B, L, H, D)), np.ones((B, L, H, D)))
    q = _bf16_values(rng, (B, L, H, D)) * 4
    bits = oracle.keep_bits(ring, T, KeepRule(seed=5, p_prior=0.3))
    O, LSE, RS = oracle.sparse_causal_attention(ring, q, bits, T, 0.35, with_rowsum=True)
    assert np.abs(O - 1).max() < 1e-12
    assert np.abs(RS - 1).max() < 1e-12
    # LSE is the log of the sum of exponentiated kept scores
    K, _ = oracle.dense_keys(ring, 0, 1)
    cols = oracle.attention._kept_columns(np.nonzero(bits[0, 1, 2])[0], L, T, 4, 4 * L)
    s = 0.35 * (q[0, 40, 1] @ K[cols].T)
    assert abs(LSE[0, 1, 40] - math.log(np.exp(s).sum())) < 1e-12


def test_token_order_inside_tiles_does_not_matter():
    rng = _rng(10)
    B, L, H, D, T = 1, 20, 2, 8, 8        # NT = 3, tail 4
    ring_a = RingModel(3, True)
    ring_b = RingModel(3, True)
    for _ in range(3):
        k = _bf16_values(rng, (B, L, H, D))
        v = _bf16_values(rng, (B, L, H, D))
        perm = np.concatenate([t * T + rng.permutation(min(T, L - t * T)) for t in range(3)])
        ring_a.append(k, v)
        ring_b.append(k[:, perm], v[:, perm])
    q = _bf16_values(rng, (B, L, H, D))
    rule = KeepRule(seed=8, p_prior=0.5)
    bits = oracle.keep_bits(ring_a, T, rule)
    assert np.array_equal(bits, oracle.keep_bits(ring_b, T, rule))
    Oa, La = oracle.sparse_causal_attention(ring_a, q, bits, T, 0.3)
    Ob, Lb = oracle.sparse_causal_attention(ring_b, q, bits, T, 0.3)
    assert np.abs(Oa - Ob).max() < 1e-12 and np.abs(La - Lb).max() < 1e-12


def test_eviction_history_invariance_of_outputs():
    rng = _rng(11)
    B, L, H, D, T = 1, 12, 1, 4, 4
    chunks = [(_bf16_values(rng, (B, L, H, D)), _bf16_values(rng, (B, L, H, D))) for _ in range(7)]
    a = RingModel(4, True)
    for k, v in chunks:
        if a.n_live == 4:
            a.evict(1)
        a.append(k, v)
    b = RingModel(4, True)
    for k, v in chunks[:4]:
        b.append(k, v)
    b.evict(3)
    for k, v in chunks[4:]:
        b.append(k, v)
    q = _bf16_values(rng, (B, L, H, D))
    rule = KeepRule(seed=4, p_prior=0.5)
    bits = oracle.keep_bits(a, T, rule)
    Oa, _ = oracle.sparse_causal_attention(a, q, bits, T, 0.5)
    Ob, _ = oracle.sparse_causal_attention(b, q, oracle.keep_bits(b, T, rule), T, 0.5)
    assert np.array_equal(Oa, Ob)


def test_empty_keep_row_is_zero_with_neg_inf_lse():
    rng = _rng(12)
    ring = _ring(rng, 1, 6, 1, 4, n_chunks=2, max_chunks=2, pin_sink=False)
    q = _bf16_values(rng, (1, 6, 1, 4))
    bits = np.zeros((1, 1, 2, 4), dtype=bool)
    bits[0, 0, 1, 2] = True
    O, LSE = oracle.sparse_causal_attention(ring, q, bits, 3, 0.5)
    assert (O[0, :3] == 0).all() and np.isneginf(LSE[0, 0, :3]).all()
    assert np.isfinite(LSE[0, 0, 3:]).all()


def test_sampled_rows_match_full():
    rng = _rng(13)
    B, L, H, D, T = 2, 33, 3, 8, 8
    ring = _ring(rng, B, L, H, D, n_chunks=5, max_chunks=4, pin_sink=True)
    q = _bf16_values(rng, (B, L, H, D))
    bits = oracle.keep_bits(ring, T, KeepRule(seed=21, p_prior=0.35))
    O, LSE = oracle.sparse_causal_attention(ring, q, bits, T, 0.4)
    samples = [(b, h, r) for b, h, r in itertools.product(range(B), range(H), [0, 7, 8, 31, 32])]
    Os, Ls = oracle.sparse_causal_attention_rows(ring, q, bits, T, 0.4, samples)
    for n, (b, h, r) in enumerate(samples):
        # same definition; only the BLAS blocking of one row vs a tile differs
        assert np.abs(Os[n] - O[b, r, h]).max() < 1e-13 and abs(Ls[n] - LSE[b, h, r]) < 1e-13
