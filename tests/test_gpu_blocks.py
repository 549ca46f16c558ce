"""3-D block tiling on the GPU (block order of tokens, per-block valid rows,
the local window M_local) against the CPU oracle.

The GPU path permutes raster tokens into block order (uf_block_permute),
runs the window with block geometry, and permutes the output back; the oracle
evaluates the same attention directly in raster order over the tokens of the
kept blocks, so the two share nothing but the definition.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_common import REL_TOL, f64, log, lse_tol, require_gpu, row_errors, row_rel_err

pytestmark = pytest.mark.gpu


def _permute(P, g, x, inverse):
    B, _, H, D = x.shape
    n = g.tokens if inverse else g.padded_tokens
    out = torch.empty((B, n, H, D), dtype=x.dtype, device=x.device)
    P.uf_block_permute(P.uf_block_geom(g.frames, g.grid_h, g.grid_w, g.bt, g.bh, g.bw), B, H, x, out, inverse)
    return out


@pytest.mark.parametrize("geom", [(3, 10, 12, 2, 4, 8), (3, 68, 120, 2, 8, 8), (1, 9, 17, 1, 8, 8)])
def test_block_permute_matches_oracle_order(geom):
    P = require_gpu()
    g = oracle.BlockGeom(*geom)
    x = synth.custom_tensor((2, g.tokens, 3, 128), 31, 0, "k").cuda()
    y = _permute(P, g, x, 0)
    torch.cuda.synchronize()
    src = torch.from_numpy(oracle.block_order(g)).cuda()
    want = torch.zeros_like(y)
    valid = src >= 0
    want[:, valid] = x[:, src[valid]]
    assert torch.equal(y, want)
    back = _permute(P, g, y, 1)
    torch.cuda.synchronize()
    assert torch.equal(back, x)


class BlockCase:
    """A blocked window on the GPU and the same chunks, in raster order, for the oracle."""

    def __init__(self, P, g, B, H, max_chunks, pin_sink, seed):
        self.P, self.g, self.B, self.H, self.seed = P, g, B, H, seed
        self.win = P.KVWindow(B, H, g.padded_tokens, g.tile, max_chunks, pin_sink)
        self.win.set_block_geom(g.frames, g.grid_h, g.grid_w, g.bt, g.bh, g.bw)
        self.ring = oracle.RingModel(max_chunks, pin_sink)
        self.n = 0

    def draw(self, chunk, name):
        return synth.custom_tensor((self.B, self.g.tokens, self.H, 128), self.seed, chunk, name, device="cuda")

    def append(self):
        if self.win.info().n_live == self.win.desc.max_chunks:
            self.win.evict(1)
            self.ring.evict(1)
        k, v = self.draw(self.n, "k"), self.draw(self.n, "v")
        self.win.append(_permute(self.P, self.g, k, 0), _permute(self.P, self.g, v, 0))
        self.ring.append(f64(k), f64(v))
        self.n += 1

    def oracle_bernoulli(self, p, r):
        """Eq. 4 keep set from the oracle: Bernoulli stand-in, then M_local."""
        return oracle.block_sparse_mask(self.ring, oracle.KeepRule(self.seed, p), geom=self.g, local_r=r)

    def oracle_topk(self, q, budget, r):
        """Eq. 4 keep set from the oracle: top-k over pooled blocks, then M_local."""
        return oracle.block_sparse_mask(self.ring, oracle.TopkRule(budget), q=f64(q), geom=self.g, local_r=r)

    def gpu_lists(self):
        torch.cuda.synchronize()
        c, i, m = self.win.lists_views()
        return c.cpu().numpy(), i.cpu().numpy(), m.cpu().numpy().view(np.uint32)

    def compare_lists(self, bits):
        want = oracle.lists_from_bits(bits, self.win.info().nk_cap)
        for got, exp in zip(self.gpu_lists(), want):
            assert np.array_equal(got, exp)

    def attention(self, q, blocks=None):
        """GPU O and LSE in raster order; (optional) only the query blocks listed are checked."""
        o, lse = self.win.attention(_permute(self.P, self.g, q, 0))
        o_r = _permute(self.P, self.g, o, 1)
        torch.cuda.synchronize()
        src = oracle.block_order(self.g)
        lse_r = np.empty((self.B, self.H, self.g.tokens))
        lb = lse.cpu().numpy()
        lse_r[:, :, src[src >= 0]] = lb[:, :, np.nonzero(src >= 0)[0]]
        return f64(o_r), lse_r

    def check_attention(self, q, bits, heads=None, blocks=None):
        o, lse = self.attention(q)
        qh = f64(q)
        blk = oracle.block_of_token(self.g)
        worst, lworst = 0.0, 0.0
        for b in range(self.B):
            for h in (range(self.H) if heads is None else heads):
                ks = [c.k[b, :, h] for c in self.ring.logical_chunks()]
                vs = [c.v[b, :, h] for c in self.ring.logical_chunks()]
                bb = bits[b, h].copy()
                if blocks is not None:
                    keep_rows = np.zeros(self.g.n_blocks, bool)
                    keep_rows[list(blocks)] = True
                    bb[~keep_rows] = False
                O, LSE = oracle.attention_in_raster(ks, vs, qh[b, :, h], self.g, bb, 1 / math.sqrt(128))
                rows = np.nonzero(np.isin(blk, list(blocks)))[0] if blocks is not None else np.arange(self.g.tokens)
                worst = max(worst, row_rel_err(o[b, rows, h], O[rows]))
                lworst = max(lworst, float(np.abs(lse[b, h, rows] - LSE[rows]).max()))
        log(f"  rel_err={worst:.3e} lse_err={lworst:.3e}")
        assert worst <= REL_TOL and lworst <= lse_tol(self.g.tile)


SMALL = oracle.BlockGeom(3, 10, 12, 2, 4, 8)     # 12 blocks of 64, edge blocks partial


@pytest.mark.parametrize("r", [0, 1, 3])
def test_blocked_bernoulli_lists_and_attention(r):
    P = require_gpu()
    log(f"blocks bernoulli r={r}")
    case = BlockCase(P, SMALL, 2, 3, 4, True, seed=41)
    for _ in range(5):
        case.append()
    case.win.build_lists(case.seed, 0.5, local_r=r)
    bits = case.oracle_bernoulli(0.5, r)
    case.compare_lists(bits)
    case.check_attention(case.draw(99, "q"), bits)


@pytest.mark.parametrize("r", [0, 3])
def test_blocked_topk_lists_and_attention(r):
    P = require_gpu()
    log(f"blocks topk r={r}")
    case = BlockCase(P, SMALL, 1, 2, 4, True, seed=43)
    for _ in range(4):
        case.append()
    q = case.draw(98, "q")
    case.win.build_topk_lists(_permute(P, SMALL, q, 0), 5, local_r=r)
    bits = case.oracle_topk(q, 5, r)
    case.compare_lists(bits)
    case.check_attention(q, bits)


def test_blocked_pooled_keys_follow_block_counts():
    P = require_gpu()
    case = BlockCase(P, SMALL, 1, 2, 3, False, seed=45)
    for _ in range(2):
        case.append()
    torch.cuda.synchronize()
    km = case.win.kmean_view().cpu().numpy()
    for pos, c in enumerate(case.ring.logical_chunks()):
        slot, _ = case.win.logical(pos)
        for h in range(2):
            assert np.array_equal(km[slot, 0, h], oracle.block_means(c.k[0, :, h], SMALL))


def test_paper_geometry_1k_local_window():
    """The paper's (2, 8, 8) blocks on the 1K grid (3 x 68 x 120, 270 blocks with
    partial edge blocks), r = 9: lists bit for bit on every head, attention on
    sampled query blocks of two heads."""
    P = require_gpu()
    g = oracle.BlockGeom(3, 68, 120, 2, 8, 8)
    log("blocks 1k geometry r=9")
    case = BlockCase(P, g, 1, 4, 5, True, seed=47)
    for _ in range(5):
        case.append()
    case.win.build_lists(case.seed, 0.25, local_r=9)
    bits = case.oracle_bernoulli(0.25, 9)
    case.compare_lists(bits)
    q = case.draw(97, "q")
    case.check_attention(q, bits, heads=[0, 3], blocks=[0, 14, 134, 269])


G128 = oracle.BlockGeom(3, 10, 12, 2, 8, 8)     # 8 blocks of 128 tokens, edge blocks partial


@pytest.mark.parametrize("r", [0, 1])
def test_blocked_128_attention_skips_empty_key_halves(r):
    """128-token blocks (valid counts 128, 64, 32, 16 at the first block time and
    64, 32, 16, 8 at the second): the attention walks only the 64-key units that
    hold a valid key; against the oracle in raster order, whole and split."""
    P = require_gpu()
    log(f"blocks 128 attention r={r}")
    case = BlockCase(P, G128, 2, 2, 4, True, seed=51)
    for _ in range(5):
        case.append()
    case.win.build_lists(case.seed, 0.5, local_r=r)
    bits = case.oracle_bernoulli(0.5, r)
    case.compare_lists(bits)
    q = case.draw(96, "q")
    case.check_attention(q, bits)
    qb = _permute(P, G128, q, 0)
    o1, l1 = case.win.attention(qb)
    o3, l3 = case.win.attention(qb, split=3)
    torch.cuda.synchronize()
    src = oracle.block_order(G128)
    valid = torch.from_numpy(src >= 0).cuda()
    assert row_rel_err(f64(o3[:, valid]), f64(o1[:, valid])) <= REL_TOL
    assert float((l3[:, :, valid] - l1[:, :, valid]).abs().max()) <= lse_tol(128)


@pytest.mark.parametrize("g", [G128, SMALL], ids=["blocks128", "blocks64"])
@pytest.mark.parametrize("r", [0, 1])
def test_blocked_backward(r, g):
    """dQ, dK, dV on block-ordered tokens (uf_sparse_causal_attn_bwd with block
    geometry) mapped back to raster order, against the oracle's raster-order
    gradients; padding rows are exactly zero.  Bar: per gradient row,
    max_d|diff| / max_d|ref| <= 1e-2, as for the raster backward."""
    P = require_gpu()
    log(f"blocks backward r={r} tile={g.tile}")
    case = BlockCase(P, g, 2, 2, 4, True, seed=49)
    for _ in range(5):
        case.append()
    case.win.build_lists(case.seed, 0.5, local_r=r)
    bits = case.oracle_bernoulli(0.5, r)
    q, do = case.draw(99, "q"), case.draw(99, "do")
    qb, dob = _permute(P, g, q, 0), _permute(P, g, do, 0)
    o, lse = case.win.attention(qb)
    dq, dk, dv = case.win.attention_bwd(qb, o, lse, dob)
    torch.cuda.synchronize()
    src = oracle.block_order(g)
    valid = src >= 0
    gq, gk, gv = dq.cpu().numpy(), dk.cpu().numpy(), dv.cpu().numpy()
    assert np.all(gq[:, ~valid] == 0) and np.all(gk[:, :, ~valid] == 0) and np.all(gv[:, :, ~valid] == 0)
    rq = np.zeros((case.B, g.tokens, case.H, 128))
    rq[:, src[valid]] = gq[:, valid]
    rk = np.zeros((gk.shape[0], case.B, g.tokens, case.H, 128))
    rv = np.zeros_like(rk)
    rk[:, :, src[valid]] = gk[:, :, valid]
    rv[:, :, src[valid]] = gv[:, :, valid]
    qh, doh = f64(q), f64(do)
    chunks = case.ring.logical_chunks()
    worst = 0.0
    for b in range(case.B):
        for h in range(case.H):
            wq, wk, wv = oracle.attention_in_raster_bwd([c.k[b, :, h] for c in chunks], [c.v[b, :, h] for c in chunks],
                                                        qh[b, :, h], doh[b, :, h], g, bits[b, h], 1 / math.sqrt(128))
            for got, want in ((rq[b, :, h], wq), (rk[:, b, :, h], np.stack(wk)), (rv[:, b, :, h], np.stack(wv))):
                worst = max(worst, float(row_errors(got, want).max()))
    log(f"  per-row={worst:.3e}")
    assert worst <= 1e-2
