"""GPU content-adaptive top-k (pooled keys written by uf_kv_append, lists by
uf_build_topk_lists through the C ABI) against the CPU oracle: bit for bit.

Both sides evaluate the same float32 arithmetic in the same order (the rule's
definition in include/uf.h), so pooled keys, and therefore the integer keep
decisions, must agree exactly.  The attention over top-k lists is then
compared with the oracle's attention over the oracle's top-k keep set.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_common import REL_TOL, Case, f64, log, lse_tol, require_gpu, row_rel_err

pytestmark = pytest.mark.gpu


def _pooled_check(case):
    km = case.win.kmean_view().cpu().numpy()                       # [slots, B, H, NT, D]
    for pos, c in enumerate(case.ring.logical_chunks()):
        slot, seq = case.win.logical(pos)
        assert seq == c.seq
        for b in range(case.B):
            for h in range(case.H):
                want = oracle.pooled_means(c.k[b, :, h, :], case.T)
                assert np.array_equal(km[slot, b, h], want), (pos, b, h)


def _topk_compare(case, q, rule):
    bits = oracle.topk_bits(case.ring, case._host(q), case.T, rule)
    info = case.win.info()
    want_c, want_i, want_m = oracle.lists_from_bits(bits, info.nk_cap)
    case.win.build_topk_lists(q, rule.budget, rule.keep_sink, rule.keep_current)
    torch.cuda.synchronize()
    c, i, m = case.win.lists_views()
    got_c, got_i, got_m = c.cpu().numpy(), i.cpu().numpy(), m.cpu().numpy().view(np.uint32)
    assert np.array_equal(got_c, want_c)
    assert np.array_equal(got_i, want_i)
    assert np.array_equal(got_m, want_m)
    return bits


SHAPES = [
    # B, L, H, T, max_chunks, pin_sink, n_appended
    (1, 192, 2, 64, 3, False, 3),
    (2, 300, 3, 128, 4, True, 6),
    (1, 130, 2, 64, 5, True, 7),
    (1, 1, 1, 128, 3, True, 3),
    (1, 1000, 2, 128, 5, True, 5),
]


@pytest.mark.parametrize("B,L,H,T,mc,pin,n", SHAPES)
def test_pooled_keys_bit_exact(B, L, H, T, mc, pin, n):
    P = require_gpu()
    log(f"topk pooled B={B} L={L} H={H} T={T} max={mc} pin={pin} n={n}")
    case = Case(P, B, L, H, T, mc, pin, seed=3000 + L + H)
    for _ in range(n):
        case.append()
    torch.cuda.synchronize()
    _pooled_check(case)


def test_pooled_keys_ignore_padding():
    P = require_gpu()
    outs = []
    for flags in (0, P._lib.UF_F_POISON_PAD):
        c = Case(P, 1, 300, 2, 128, 3, True, seed=17, flags=flags)
        for _ in range(3):
            c.append()
        torch.cuda.synchronize()
        outs.append(c.win.kmean_view().clone())
    assert torch.equal(outs[0], outs[1])


@pytest.mark.parametrize("B,L,H,T,mc,pin,n", SHAPES)
@pytest.mark.parametrize("budget,keep_sink,keep_current", [(0, True, True), (3, True, True), (2, False, True),
                                                           (5, False, False), (10 ** 6, True, False)])
def test_topk_lists_bit_exact(B, L, H, T, mc, pin, n, budget, keep_sink, keep_current):
    P = require_gpu()
    log(f"topk lists B={B} L={L} H={H} T={T} n={n} budget={budget} sink={keep_sink} cur={keep_current}")
    case = Case(P, B, L, H, T, mc, pin, seed=4000 + L + H)
    for _ in range(n):
        case.append()
    _topk_compare(case, case.query(), oracle.TopkRule(budget, keep_sink, keep_current))


@pytest.mark.parametrize("name,frac", [("1k", 0.25), ("2k", 0.15)])
def test_topk_lists_workloads(name, frac):
    """Full-size windows in the bench's configuration, every head, bit for bit."""
    P = require_gpu()
    wl = synth.WORKLOADS[name]
    log(f"topk workload={name}")
    case = Case(P, 1, wl.chunk_tokens, wl.heads, wl.tile, wl.max_chunks, wl.pin_sink, wl.seed, gen_device="cuda")
    for _ in range(wl.window_chunks):
        case.append()
    nt = -(-wl.chunk_tokens // wl.tile)
    budget = int(frac * wl.prior_chunks * nt)
    bits = _topk_compare(case, case.query(), oracle.TopkRule(budget))
    assert np.all(bits.sum(-1) == budget + (1 + 1) * nt)


def test_topk_eviction_history_gives_identical_lists():
    P = require_gpu()
    lists = []
    for script in ("one_by_one", "batch"):
        c = Case(P, 1, 300, 2, 128, 5, True, seed=21)
        if script == "one_by_one":
            for _ in range(4):
                c.append()
            for _ in range(3):
                c.win.evict(1)
                c.ring.evict(1)
                c.append(evict_when_full=False)
        else:
            for _ in range(4):
                c.append()
            c.win.evict(3)
            c.ring.evict(3)
            for _ in range(3):
                c.append(evict_when_full=False)
        q = synth.custom_tensor((1, 300, 2, 128), 21, 99, "q").cuda()
        _topk_compare(c, q, oracle.TopkRule(2))
        lists.append([t.clone() for t in c.win.lists_views()])   # the sections, not the alignment gaps
    for a, b in zip(*lists):
        assert torch.equal(a, b)


def test_attention_over_topk_lists():
    P = require_gpu()
    case = Case(P, 2, 700, 3, 128, 5, True, seed=55)
    for _ in range(6):
        case.append()
    q = case.query()
    rule = oracle.TopkRule(4)
    bits = _topk_compare(case, q, rule)
    o, lse = case.attention(q)
    O, LSE = oracle.sparse_causal_attention(case.ring, case._host(q), bits, 128, 1 / math.sqrt(128))
    err = row_rel_err(case._host(o), O)
    lerr = float(np.abs(f64(lse) - LSE).max())
    log(f"  rel_err={err:.3e} lse_err={lerr:.3e}")
    assert err <= REL_TOL and lerr <= lse_tol(case.T)


def test_replace_newest_equals_appending_the_refreshed_chunk():
    """A refreshed current chunk (Sec. 2.3.2 (ii)) gives the same pages, pooled keys,
    lists and attention as a window that appended the refreshed K/V directly."""
    P = require_gpu()
    shape = (1, 300, 2, 128)
    kv = [(synth.custom_tensor(shape, 8, c, "k").cuda(), synth.custom_tensor(shape, 8, c, "v").cuda())
          for c in range(5)]
    q = synth.custom_tensor(shape, 8, 9, "q").cuda()
    wa = P.KVWindow(1, 2, 300, 128, 4, True)
    wb = P.KVWindow(1, 2, 300, 128, 4, True)
    for c in range(4):
        wa.append(*kv[c])
    wa.replace_newest(*kv[4])                   # chunk 3 refreshed with chunk 4's K/V
    for c in (0, 1, 2, 4):
        wb.append(*kv[c])
    assert torch.equal(wa.pool, wb.pool)
    outs = []
    for w in (wa, wb):
        w.build_topk_lists(q, 2)
        lists = [t.clone() for t in w.lists_views()]
        o, lse = w.attention(q)
        torch.cuda.synchronize()
        outs.append((lists, o, lse))
    for a, b in zip(outs[0][0], outs[1][0]):
        assert torch.equal(a, b)
    assert torch.equal(outs[0][1], outs[1][1]) and torch.equal(outs[0][2], outs[1][2])
