"""GPU backward (uf_sparse_causal_attn_bwd through the C ABI) against the CPU
oracle on the same seeded inputs, element by element.

Bar: per row of each gradient (a query row of dQ, a key row of dK or dV),
max_d |g_gpu - g_ref| / max_d |g_ref| <= 1e-2; a row whose exact gradient is
zero (a key that no query row keeps) must be exactly zero.  Derivation: Q, K,
V and dO are bf16 inputs, exact on both sides; the kernels round P and dS to
bf16 (dS is formed from the bf16 P) before the products that give dV, dK and
dQ, each rounding within a relative 2^-8, and take delta from the bf16
forward output, all with fp32 accumulation.  An element of a gradient row is
a sum of such rounded terms with independent errors, so its error is a small
multiple of the typical rounding (about 2^-8/sqrt(3)) of the row's scale; 1e-2
leaves that margin and equals the forward's bar.  Full comparison at sizes
the oracle finishes in seconds (ragged tails, batch 2, evictions, a one-token
chunk) and on two heads of the 480p window; at the 1K and 2K windows (the
launches that bench.py times) one full head element by element, one dQ row in
every query tile of every head, and, on every head, identities that the exact
gradients satisfy at any size.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_common import Case, f64, head_ring, log, require_gpu, row_errors, row_errors_scaled

pytestmark = pytest.mark.gpu

GRAD_TOL = 1e-2


def _normwise(g, r):
    den = np.linalg.norm(r)
    if den == 0:
        return float(np.linalg.norm(g))
    return float(np.linalg.norm(g - r) / den)


def _rows(g, r):
    """Worst per-row error of gradient rows (last axis = D)."""
    e = row_errors(g, r)
    return float(e.max()) if e.size else 0.0


def _run(case, rule, scale=None):
    scale = 1 / math.sqrt(128) if scale is None else scale
    case.gpu_lists(rule)
    q = case.query()
    o, lse = case.win.attention(q, scale)
    do = case._draw(case.n_appended - 1, "do")
    dq, dk, dv = case.win.attention_bwd(q, o, lse, do, scale)
    torch.cuda.synchronize()
    return q, o, lse, do, dq, dk, dv


def _compare_heads(gq, gk, gv, rq, rk, rv, pairs, B):
    """pairs: (GPU head, oracle head index).  Returns the worst per-row error
    of each gradient; asserts the bar."""
    worst = {"dq": 0.0, "dk": 0.0, "dv": 0.0}
    for b in range(B):
        for h, n in pairs:
            worst["dq"] = max(worst["dq"], _rows(gq[b, :, h], rq[b, :, n]))
            worst["dk"] = max(worst["dk"], _rows(gk[:, b, :, h], rk[:, b, :, n]))
            worst["dv"] = max(worst["dv"], _rows(gv[:, b, :, h], rv[:, b, :, n]))
    log("  per-row " + " ".join(f"{k}={v:.3e}" for k, v in worst.items()))
    assert max(worst.values()) <= GRAD_TOL, worst
    return worst


def _full_compare(case, rule, heads=None, scale=None):
    scale = 1 / math.sqrt(128) if scale is None else scale
    q, o, lse, do, dq, dk, dv = _run(case, rule, scale)
    bits = case.oracle_bits(rule)
    hsel = list(range(case.H)) if heads is None else heads
    bits = bits[:, hsel]
    rq, rk, rv = oracle.sparse_causal_attention_bwd(case.ring, case._host(q), case._host(do), bits, case.T, scale)
    gq, gk, gv = dq.cpu().numpy(), dk.cpu().numpy(), dv.cpu().numpy()
    _compare_heads(gq, gk, gv, rq, rk, rv, [(h, n) for n, h in enumerate(hsel)], case.B)
    return dq, dk, dv


SMALL = [
    # B, L, H, max_chunks, pin_sink, n_chunks, p
    (2, 300, 3, 4, True, 6, 0.5),
    (1, 1, 1, 3, True, 3, 0.5),
    (1, 1000, 2, 5, True, 7, 0.25),
    (1, 256, 1, 1, False, 1, 0.0),
    (1, 640, 4, 3, False, 4, 0.0),
    (1, 700, 2, 5, False, 5, 1.0),
]


@pytest.mark.parametrize("T", [128, 64])
@pytest.mark.parametrize("B,L,H,mc,pin,n,p", SMALL)
def test_small_backward_parity(B, L, H, mc, pin, n, p, T):
    P = require_gpu()
    log(f"bwd small T={T} B={B} L={L} H={H} max={mc} pin={pin} n={n} p={p}")
    case = Case(P, B, L, H, T, mc, pin, seed=2000 + L + H)
    for _ in range(n):
        case.append()
    _full_compare(case, case.rule(p))


def test_backward_tiny_workload():
    """The tiny window (64-token tiles, 2 heads, 384 keys, every tile kept) in full."""
    P = require_gpu()
    wl = synth.WORKLOADS["tiny"]
    log("bwd workload=tiny")
    case = Case(P, wl.batch, wl.chunk_tokens, wl.heads, wl.tile, wl.max_chunks, wl.pin_sink, wl.seed)
    for _ in range(wl.window_chunks):
        case.append()
    _full_compare(case, case.rule(wl.p_prior))


def test_backward_large_logits():
    """Peaked rows (q and k scaled by 3): P near one-hot, so dP - delta cancels
    for the dominant key and the exact dQ and dK rows of such queries shrink
    towards zero while the rounding of the kernel's factors (delta from the
    bf16 O, P and dS in bf16) does not.  Bar: per row, max_d|diff| over the
    larger of max_d|ref| and the largest scale of the row's summands
    (oracle.sparse_causal_attention_bwd_scales) <= 1e-2; the plain per-row
    form must still hold for dV, which has no such cancellation."""
    P = require_gpu()
    log("bwd large logits")
    case = Case(P, 1, 500, 2, 128, 4, True, seed=2101, gain=lambda c, n: 3.0 if n in ("q", "k") else 1.0)
    for _ in range(4):
        case.append()
    rule = case.rule(0.5)
    scale = 1 / math.sqrt(128)
    q, o, lse, do, dq, dk, dv = _run(case, rule, scale)
    bits = case.oracle_bits(rule)
    hq, hdo = case._host(q), case._host(do)
    rq, rk, rv = oracle.sparse_causal_attention_bwd(case.ring, hq, hdo, bits, case.T, scale)
    sq, sk, sv = oracle.sparse_causal_attention_bwd_scales(case.ring, hq, hdo, bits, case.T, scale)
    gq, gk, gv = dq.cpu().numpy(), dk.cpu().numpy(), dv.cpu().numpy()
    worst = {"dq": 0.0, "dk": 0.0, "dv": 0.0, "dv_plain": 0.0, "dq_plain": 0.0}
    for h in range(case.H):
        worst["dq"] = max(worst["dq"], float(row_errors_scaled(gq[0, :, h], rq[0, :, h], sq[0, :, h]).max()))
        worst["dk"] = max(worst["dk"], float(row_errors_scaled(gk[:, 0, :, h], rk[:, 0, :, h], sk[:, 0, :, h]).max()))
        worst["dv"] = max(worst["dv"], float(row_errors_scaled(gv[:, 0, :, h], rv[:, 0, :, h], sv[:, 0, :, h]).max()))
        worst["dv_plain"] = max(worst["dv_plain"], _rows(gv[:, 0, :, h], rv[:, 0, :, h]))
        worst["dq_plain"] = max(worst["dq_plain"], _rows(gq[0, :, h], rq[0, :, h]))
    log("  " + " ".join(f"{k}={v:.3e}" for k, v in worst.items()))
    assert max(worst["dq"], worst["dk"], worst["dv"], worst["dv_plain"]) <= GRAD_TOL, worst


@pytest.mark.parametrize("T", [128, 64])
def test_backward_poisoned_padding_and_determinism(T):
    """Padding keys (bf16 9984.0 in the pool) never count, bit for bit, and two
    runs give identical gradients (no atomics)."""
    P = require_gpu()
    log(f"bwd poison pad + determinism T={T}")
    outs = []
    for flags in (0, P._lib.UF_F_POISON_PAD):
        case = Case(P, 1, 300, 2, T, 3, True, seed=2102, flags=flags)
        for _ in range(3):
            case.append()
        outs.append(_run(case, case.rule(0.5))[4:])
        outs.append(_run(case, case.rule(0.5))[4:])
    for a, b in zip(outs[0], outs[1]):
        assert torch.equal(a, b)
    for a, b in zip(outs[0], outs[2]):
        assert torch.equal(a, b)


def test_backward_480p_full_two_heads():
    P = require_gpu()
    wl = synth.WORKLOADS["480p"]
    log("bwd workload=480p heads 0, 7")
    case = Case(P, 1, wl.chunk_tokens, wl.heads, wl.tile, wl.max_chunks, wl.pin_sink, wl.seed,
                gen_device="cuda", oracle_heads=[0, 7])
    for _ in range(wl.window_chunks):
        case.append()
    _full_compare(case, case.rule(wl.p_prior), heads=[0, 7])


FULL_HEAD = {"1k": 5, "2k": 10}


@pytest.mark.parametrize("name", ["1k", "2k"])
def test_backward_full_head_every_tile_and_identities(name):
    P = require_gpu()
    wl = synth.WORKLOADS[name]
    h_full = FULL_HEAD[name]
    log(f"bwd workload={name}: full head {h_full}, one dQ row per query tile, identities")
    case = Case(P, 1, wl.chunk_tokens, wl.heads, wl.tile, wl.max_chunks, wl.pin_sink, wl.seed, gen_device="cuda")
    for _ in range(wl.window_chunks):
        case.append()
    rule = case.rule(wl.p_prior)
    scale = 1 / math.sqrt(128)
    q, o, lse, do, dq, dk, dv = _run(case, rule, scale)
    for t in (dq, dk, dv):
        assert torch.isfinite(t).all()
    bits = case.oracle_bits(rule)
    hq, hdo = f64(q), f64(do)
    gq = dq.cpu().numpy()
    gk = dk[:, :, :, h_full:h_full + 1].cpu().numpy()
    gv = dv[:, :, :, h_full:h_full + 1].cpu().numpy()

    # one head in full: every dQ query row and every dK, dV key row of the window
    rq, rk, rv = oracle.sparse_causal_attention_bwd(head_ring(case.ring, [h_full]), hq[:, :, [h_full]],
                                                    hdo[:, :, [h_full]], bits[:, [h_full]], wl.tile, scale)
    _compare_heads(gq[:, :, h_full:h_full + 1], gk, gv, rq, rk, rv, [(0, 0)], 1)

    # one random dQ row in every query tile of every head
    rng = np.random.default_rng(wl.seed + 7)
    L, T = wl.chunk_tokens, wl.tile
    nt = -(-L // T)
    samples = [(0, h, int(i * T + rng.integers(0, min(T, L - i * T)))) for h in range(wl.heads) for i in range(nt)]
    samples += [(0, h, r) for h in range(wl.heads) for r in (0, T - 1, L - 1)]
    want = oracle.sparse_causal_attention_bwd_rows(case.ring, hq, hdo, bits, T, scale, samples)
    got = np.stack([gq[b, r, h] for b, h, r in samples])
    err = _rows(got, want)
    log(f"  sampled dq rows={len(samples)} worst per-row={err:.3e}")
    assert err <= GRAD_TOL

    # identities of the exact gradients, per head, over the whole window
    gk, gv, go = dk.cpu().numpy(), dv.cpu().numpy(), f64(o)
    ks = np.stack([c.k[0] for c in case.ring.logical_chunks()])     # [n_live, L, H, D]
    vs = np.stack([c.v[0] for c in case.ring.logical_chunks()])
    for h in range(wl.heads):
        s_dk = np.linalg.norm(gk[:, 0, :, h].sum(axis=(0, 1)))
        assert s_dk <= GRAD_TOL * np.linalg.norm(gk[:, 0, :, h])
        tk = (gk[:, 0, :, h] * ks[:, :, h]).sum(-1)
        tq = (gq[0, :, h] * hq[0, :, h]).sum(-1)
        assert abs(tk.sum() - tq.sum()) <= GRAD_TOL * (np.abs(tk).sum() + np.abs(tq).sum())
        tv = (gv[:, 0, :, h] * vs[:, :, h]).sum(-1)
        to = (hdo[0, :, h] * go[0, :, h]).sum(-1)
        assert abs(tv.sum() - to.sum()) <= GRAD_TOL * (np.abs(tv).sum() + np.abs(to).sum())


@pytest.mark.parametrize("T", [128, 64])
def test_backward_empty_rows_and_stale_entries(T):
    """A row with no kept tile gets zero gradients and gives none; a list entry
    outside the window counts no key (hand-made lists, index and mask sections
    kept consistent)."""
    P = require_gpu()
    log(f"bwd empty rows + stale entries T={T}")
    case = Case(P, 1, 300, 2, T, 4, True, seed=2103)
    for _ in range(3):
        case.append()
    counts, idx, mask = case.gpu_lists(case.rule(1.0))
    nt = -(-300 // T)
    nk = 3 * nt
    counts, idx, mask = counts.copy(), idx.copy(), mask.copy()
    counts[0, 0, 1] = 0                          # empty row
    idx[0, 0, 1, :] = -1
    mask[0, 0, 1, :] = 0
    idx[0, 1, 2, :] = -1                         # row keeps tiles 0, 4 and a stale 50
    idx[0, 1, 2, :3] = [0, 4, 50]
    counts[0, 1, 2] = 3
    mask[0, 1, 2, :] = 0
    mask[0, 1, 2, 0] = (1 << 0) | (1 << 4)
    c_v, i_v, m_v = case.win.lists_views()
    c_v.copy_(torch.from_numpy(counts))
    i_v.copy_(torch.from_numpy(idx))
    m_v.copy_(torch.from_numpy(mask.view(np.int32)))
    scale = 1 / math.sqrt(128)
    q = case.query()
    o, lse = case.win.attention(q, scale)
    do = case._draw(case.n_appended - 1, "do")
    dq, dk, dv = case.win.attention_bwd(q, o, lse, do, scale)
    torch.cuda.synchronize()
    bits = np.ones((1, 2, nt, nk), dtype=bool)
    bits[0, 0, 1] = False
    bits[0, 1, 2] = False
    bits[0, 1, 2, [0, 4]] = True
    rq, rk, rv = oracle.sparse_causal_attention_bwd(case.ring, case._host(q), case._host(do), bits, T, scale)
    gq, gk, gv = dq.cpu().numpy(), dk.cpu().numpy(), dv.cpu().numpy()
    assert np.all(gq[0, T:2 * T, 0] == 0)
    _compare_heads(gq, gk, gv, rq, rk, rv, [(0, 0), (1, 1)], 1)
