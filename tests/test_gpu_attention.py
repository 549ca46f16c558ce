"""GPU attention (uf_sparse_causal_attn_fwd through the C ABI) against the
CPU oracle on the same seeded inputs.

Bar: per (b, h, row) max_d|O_gpu - O_ref| / max_d|O_ref| <= 1e-2 on the bf16
output, |LSE_gpu - LSE_ref| <= 5e-3 (64-token tiles) or 1e-3 (128-token
tiles).  Full comparison at sizes the oracle finishes in seconds (several
tiles, ragged tails, T = 64 and 128, batch 2) and on the whole tiny and 480p
windows; at the 1K and 2K windows, in the launch configuration that bench.py
times, one full head element by element plus one row in every query tile of
every head; the streaming workload on a fixed head subset at four steps, with
one of its heads in full at two steps once the window is full.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_common import REL_TOL, Case, f64, head_ring, log, lse_tol, require_gpu, row_rel_err

pytestmark = pytest.mark.gpu


def _full_check(case, rule, q, scale=None):
    scale = 1 / math.sqrt(128) if scale is None else scale
    o, lse = case.attention(q, scale)
    bits = case.oracle_bits(rule)
    if case.oracle_heads is not None:
        bits = bits[:, case.oracle_heads]
    O, LSE = oracle.sparse_causal_attention(case.ring, case._host(q), bits, case.T, scale)
    og, lg = case._host(o), f64(lse)
    if case.oracle_heads is not None:
        lg = lg[:, case.oracle_heads]
    err = row_rel_err(og, O)
    lerr = float(np.abs(lg - LSE).max())
    log(f"  rel_err={err:.3e} lse_err={lerr:.3e}")
    assert err <= REL_TOL
    assert lerr <= lse_tol(case.T)
    return o, lse


SMALL = [
    # B, L, H, T, max_chunks, pin_sink, n_chunks, p
    (1, 192, 2, 64, 2, False, 2, 1.0),
    (2, 300, 3, 128, 4, True, 6, 0.5),
    (1, 130, 2, 64, 3, True, 5, 0.4),
    (1, 1, 1, 128, 3, True, 3, 0.5),
    (1, 1000, 2, 128, 5, True, 7, 0.25),
    (1, 256, 1, 128, 1, False, 1, 0.0),
    (1, 640, 4, 128, 3, False, 4, 0.0),
    # one tile per chunk: every row keeps a single tile (two 64-key units) ...
    (1, 100, 2, 128, 1, False, 1, 0.0),
    # ... or the pinned tile and the current one (four units)
    (2, 100, 2, 128, 2, True, 2, 1.0),
    # 64-token tiles with long lists (up to 188 tiles per row) and with more
    # rows (320) than compute units
    (1, 3000, 3, 64, 4, True, 5, 0.4),
    (2, 2500, 4, 64, 3, False, 3, 1.0),
]


@pytest.mark.parametrize("B,L,H,T,mc,pin,n,p", SMALL)
def test_small_full_parity(B, L, H, T, mc, pin, n, p):
    P = require_gpu()
    log(f"attn small B={B} L={L} H={H} T={T} max={mc} pin={pin} n={n} p={p}")
    case = Case(P, B, L, H, T, mc, pin, seed=1000 + L + H)
    for _ in range(n):
        case.append()
    rule = case.rule(p)
    case.gpu_lists(rule)
    _full_check(case, rule, case.query())


# Score magnitudes far from N(0,1) data: K of chunk c (logical order = append
# order) multiplied by a per-chunk gain, Q by q_gain.  Rising gains make the
# row maximum grow from tile to tile by more than the exponent range of fp32
# (weights against a stale offset overflow to inf and must be recomputed);
# falling gains make later tiles underflow against the first tile's maximum.
LOGIT_CASES = [
    # name, q_gain, k_gain(c)
    ("rising", 4.0, lambda c: 1.0 + 2.0 * c),
    ("falling", 4.0, lambda c: 9.0 - 2.0 * c),
    ("huge", 16.0, lambda c: 4.0 + 4.0 * (c % 2)),
    ("tiny", 0.01, lambda c: 0.5),
]


@pytest.mark.parametrize("T", [128, 64])
@pytest.mark.parametrize("name,q_gain,k_gain", LOGIT_CASES, ids=[c[0] for c in LOGIT_CASES])
def test_large_and_shifting_logits(name, q_gain, k_gain, T):
    P = require_gpu()
    log(f"attn logits case={name} T={T}")

    def gain(chunk, tensor):
        return q_gain if tensor == "q" else (k_gain(chunk) if tensor == "k" else 1.0)

    case = Case(P, 1, 700, 2, T, 5, True, seed=4242, gain=gain)
    for _ in range(5):
        case.append()
    rule = case.rule(0.6)
    case.gpu_lists(rule)
    _full_check(case, rule, case.query())


def _workload_case(P, name, gen_device, oracle_heads=None):
    wl = synth.WORKLOADS[name]
    case = Case(P, 1, wl.chunk_tokens, wl.heads, wl.tile, wl.max_chunks, wl.pin_sink, wl.seed,
                gen_device=gen_device, oracle_heads=oracle_heads)
    return wl, case


@pytest.mark.parametrize("name", ["tiny", "480p"])
def test_workload_full_parity(name):
    P = require_gpu()
    log(f"attn workload={name} full")
    wl, case = _workload_case(P, name, "cpu" if name == "tiny" else "cuda")
    for _ in range(wl.window_chunks):
        case.append()
    rule = case.rule(wl.p_prior)
    case.gpu_lists(rule)
    _full_check(case, rule, case.query())


def _sample_rows(rng, L, T, H, per_head):
    nt = -(-L // T)
    fixed = [0, 1, T - 1, T, L - 1, (nt - 1) * T, L // 2]
    out = []
    for h in range(H):
        rows = sorted(set(fixed + list(rng.integers(0, L, per_head))))
        out += [(0, h, r) for r in rows]
    return out


def _tile_rows(rng, L, T, heads):
    """One random valid row in every query tile of every listed head."""
    nt = -(-L // T)
    out = []
    for h in heads:
        for i in range(nt):
            out.append((0, h, int(i * T + rng.integers(0, min(T, L - i * T)))))
    return out


def _sampled_check(case, rule, q, samples, heads_map=None, o=None, lse=None):
    scale = 1 / math.sqrt(128)
    if o is None:
        o, lse = case.attention(q, scale)
    bits = case.oracle_bits(rule)
    hq = case._host(q)
    if heads_map is not None:
        bits = bits[:, heads_map]
    O, LSE = oracle.sparse_causal_attention_rows(case.ring, hq, bits, case.T, scale, samples)
    og = case._host(o)
    lg = f64(lse)
    if heads_map is not None:
        lg = lg[:, heads_map]
    got = np.stack([og[b, r, h] for b, h, r in samples])
    gl = np.array([lg[b, h, r] for b, h, r in samples])
    err = row_rel_err(got, O)
    lerr = float(np.abs(gl - LSE).max())
    log(f"  sampled rows={len(samples)} rel_err={err:.3e} lse_err={lerr:.3e}")
    assert err <= REL_TOL
    assert lerr <= lse_tol(case.T)
    return o, lse


def _full_head_check(case, rule, q, o, lse, h, hi=None):
    """Every row of head h (index hi of the oracle's heads) element by element."""
    scale = 1 / math.sqrt(128)
    hi = h if hi is None else hi
    bits = case.oracle_bits(rule)[:, [h]]
    ring = head_ring(case.ring, [hi])
    O, LSE = oracle.sparse_causal_attention(ring, case._host(q)[:, :, [hi]], bits, case.T, scale)
    og = f64(o[:, :, h:h + 1])
    lg = f64(lse[:, h:h + 1])
    err = row_rel_err(og, O)
    lerr = float(np.abs(lg - LSE).max())
    log(f"  full head {h}: rows={O.shape[1]} rel_err={err:.3e} lse_err={lerr:.3e}")
    assert err <= REL_TOL
    assert lerr <= lse_tol(case.T)


FULL_HEAD = {"1k": 7, "2k": 3, "1k_stream": 13}


@pytest.mark.parametrize("name", ["1k", "2k"])
def test_workload_full_head_and_every_tile(name):
    P = require_gpu()
    log(f"attn workload={name}: one full head, one row per query tile of every head")
    wl, case = _workload_case(P, name, "cuda")
    for _ in range(wl.window_chunks):
        case.append()
    rule = case.rule(wl.p_prior)
    counts, _, _ = case.gpu_lists(rule)
    q = case.query()
    o, lse = case.attention(q)
    assert torch.isfinite(o.float()).all() and torch.isfinite(lse).all()
    assert counts.min() >= (1 + int(wl.pin_sink)) * -(-wl.chunk_tokens // wl.tile)
    rng = np.random.default_rng(wl.seed)
    samples = _tile_rows(rng, wl.chunk_tokens, wl.tile, range(wl.heads))
    samples += _sample_rows(rng, wl.chunk_tokens, wl.tile, wl.heads, per_head=2)
    _sampled_check(case, rule, q, samples, o=o, lse=lse)
    _full_head_check(case, rule, q, o, lse, FULL_HEAD[name])


def test_stream_head_subset_parity():
    P = require_gpu()
    heads = [0, 13, 26, 39]
    full = FULL_HEAD["1k_stream"]
    wl, case = _workload_case(P, "1k_stream", "cuda", oracle_heads=heads)
    rng = np.random.default_rng(wl.seed)
    for step in range(wl.stream_chunks):
        case.append()
        assert case.win.info().n_live == min(step + 1, wl.max_chunks)
        rule = case.rule(wl.p_prior)
        case.gpu_lists(rule)
        q = case.query()
        if step in (0, 3, 4, 11):
            log(f"attn stream step={step}")
            o, lse = case.attention(q)
            samples = _tile_rows(rng, wl.chunk_tokens, wl.tile, range(len(heads)))
            samples += [(0, i, r) for i, _ in enumerate(heads)
                        for r in sorted(set([0, 127, 128, wl.chunk_tokens - 1] + list(rng.integers(0, wl.chunk_tokens, 6))))]
            _sampled_check(case, rule, q, samples, heads_map=heads, o=o, lse=lse)
            if step in (4, 11):
                _full_head_check(case, rule, q, o, lse, full, hi=heads.index(full))
        else:
            case.attention(q)


# ---------------------------------------------------------------------------
# invariances and degenerate cases
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("T", [128, 64])
def test_eviction_history_gives_bitwise_identical_output(T):
    P = require_gpu()
    a = Case(P, 1, 700, 3, T, 5, True, seed=42)
    b = Case(P, 1, 700, 3, T, 5, True, seed=42)
    for _ in range(8):
        a.append()
    for _ in range(4):
        b.append()
    b.win.evict(3)
    b.ring.evict(3)
    for _ in range(4):
        b.append(evict_when_full=False)
    assert [a.win.logical(p)[1] for p in range(5)] == [b.win.logical(p)[1] for p in range(5)]
    assert [a.win.logical(p)[0] for p in range(5)] != [b.win.logical(p)[0] for p in range(5)]
    rule = a.rule(0.4)
    a.gpu_lists(rule)
    b.gpu_lists(rule)
    q = a.query()
    oa, la = a.attention(q)
    ob, lb = b.attention(q)
    assert torch.equal(oa, ob) and torch.equal(la, lb)
    # and run-to-run determinism
    oa2, la2 = a.attention(q)
    assert torch.equal(oa, oa2) and torch.equal(la, la2)


@pytest.mark.parametrize("T", [128, 64])
def test_poisoned_padding_never_counts(T):
    P = require_gpu()
    outs = []
    for flags in (0, P._lib.UF_F_POISON_PAD):
        c = Case(P, 1, 300, 2, T, 3, True, seed=7, flags=flags)
        for _ in range(4):
            c.append()
        c.gpu_lists(c.rule(0.6))
        outs.append(c.attention(c.query()))
    assert torch.equal(outs[0][0], outs[1][0]) and torch.equal(outs[0][1], outs[1][1])


@pytest.mark.parametrize("T", [128, 64])
def test_v_ones_gives_ones(T):
    P = require_gpu()
    win = P.KVWindow(1, 2, 300, T, 3, True)
    for c in range(3):
        k = synth.custom_tensor((1, 300, 2, 128), 5, c, "k").cuda()
        win.append(k, torch.ones_like(k))
    win.build_lists(3, 0.5)
    q = synth.custom_tensor((1, 300, 2, 128), 5, 2, "q").cuda() * 3
    o, lse = win.attention(q)
    assert (o.float() - 1).abs().max().item() <= 1e-2


@pytest.mark.parametrize("T", [128, 64])
def test_empty_rows_and_stale_entries(T):
    """Rows with no kept tile give O = 0, LSE = -inf; list entries outside the
    window are skipped (hand-made lists, not producible by the builder)."""
    P = require_gpu()
    log(f"attn empty rows + stale entries T={T}")
    case = Case(P, 1, 300, 2, T, 4, True, seed=3)
    for _ in range(3):
        case.append()
    rule = case.rule(1.0)
    counts, idx, mask = case.gpu_lists(rule)
    nt = -(-300 // T)
    nk = 3 * nt
    counts = counts.copy()
    idx = idx.copy()
    counts[0, 0, 1] = 0                      # empty row
    idx[0, 1, 2, :] = -1                     # row keeps tiles 0, 4 and a stale 50
    idx[0, 1, 2, :3] = [0, 4, 50]
    counts[0, 1, 2] = 3
    c_v, i_v, _ = case.win.lists_views()
    c_v.copy_(torch.from_numpy(counts))
    i_v.copy_(torch.from_numpy(idx))
    q = case.query()
    o, lse = case.attention(q)
    of, lf = f64(o), f64(lse)
    assert (of[0, T:2 * T, 0] == 0).all() and np.isneginf(lf[0, 0, T:2 * T]).all()
    bits = np.ones((1, 2, nt, nk), dtype=bool)
    bits[0, 0, 1] = False
    bits[0, 1, 2] = False
    bits[0, 1, 2, [0, 4]] = True
    O, LSE = oracle.sparse_causal_attention(case.ring, case._host(q), bits, T, 1 / math.sqrt(128))
    fin = np.isfinite(LSE)
    assert row_rel_err(of[:, :, 1:], O[:, :, 1:]) <= REL_TOL
    assert np.abs(lf[fin] - LSE[fin]).max() <= lse_tol(T)


def test_lse_optional_and_outputs_untouched_beyond_shape():
    P = require_gpu()
    case = Case(P, 1, 200, 2, 128, 2, False, seed=9)
    for _ in range(2):
        case.append()
    case.gpu_lists(case.rule(1.0))
    q = case.query()
    big = torch.full((1, 210, 2, 128), 7.0, dtype=torch.bfloat16, device="cuda")
    o = big[:, :200]
    assert o.is_contiguous()
    o1 = case.win.attention(q, out=o, lse=False)
    torch.cuda.synchronize()
    assert (big[:, 200:] == 7.0).all()
    o2, _ = case.attention(q)
    assert torch.equal(o1, o2)


@pytest.mark.parametrize("n_split", [1, 2, 3, 7])
def test_split_kv_parity(n_split):
    """Split-KV: list slices attended by separate workgroups and merged; the oracle's
    bar, and agreement with the unsplit kernel up to rounding order."""
    P = require_gpu()
    log(f"attn split n_split={n_split}")
    case = Case(P, 2, 700, 3, 128, 5, True, seed=77)
    for _ in range(6):
        case.append()
    rule = case.rule(0.5)
    case.gpu_lists(rule)
    q = case.query()
    o1, l1 = case.attention(q)
    os_, ls_ = case.win.attention(q, split=n_split)
    torch.cuda.synchronize()
    bits = case.oracle_bits(rule)
    O, LSE = oracle.sparse_causal_attention(case.ring, case._host(q), bits, 128, 1 / math.sqrt(128))
    err = row_rel_err(case._host(os_), O)
    lerr = float(np.abs(f64(ls_) - LSE).max())
    log(f"  rel_err={err:.3e} lse_err={lerr:.3e}")
    assert err <= REL_TOL and lerr <= lse_tol(128)
    assert row_rel_err(case._host(os_), case._host(o1)) <= REL_TOL
    assert float((ls_ - l1).abs().max()) <= lse_tol(128)


def test_split_kv_more_slices_than_tiles():
    """Rows with fewer kept tiles than slices leave empty slices, which the merge skips."""
    P = require_gpu()
    case = Case(P, 1, 200, 2, 128, 3, True, seed=78)
    for _ in range(3):
        case.append()
    rule = case.rule(0.3)
    case.gpu_lists(rule)
    q = case.query()
    o, lse = case.win.attention(q, split=64)
    torch.cuda.synchronize()
    bits = case.oracle_bits(rule)
    O, LSE = oracle.sparse_causal_attention(case.ring, case._host(q), bits, 128, 1 / math.sqrt(128))
    assert row_rel_err(case._host(o), O) <= REL_TOL
    assert float(np.abs(f64(lse) - LSE).max()) <= lse_tol(128)


def test_split_kv_480p_full():
    P = require_gpu()
    log("attn split 480p full, n_split=4")
    wl, case = _workload_case(P, "480p", "cuda")
    for _ in range(wl.window_chunks):
        case.append()
    rule = case.rule(wl.p_prior)
    case.gpu_lists(rule)
    q = case.query()
    o, lse = case.win.attention(q, split=4)
    torch.cuda.synchronize()
    bits = case.oracle_bits(rule)
    O, LSE = oracle.sparse_causal_attention(case.ring, case._host(q), bits, wl.tile, 1 / math.sqrt(128))
    err = row_rel_err(case._host(o), O)
    lerr = float(np.abs(f64(lse) - LSE).max())
    log(f"  rel_err={err:.3e} lse_err={lerr:.3e}")
    assert err <= REL_TOL and lerr <= lse_tol(128)


def test_split_rows_parity_and_plan():
    """Split-KV of the rows from split_from on only (the tail of the last
    round): a small window with a mid split point against the oracle and the
    unsplit kernel, then the 480p window with rows 256.. of its 444 cut into 4
    slices (the last round on 256 CUs; the plan declines it, the fixed costs
    outweighing the saving) in full against the oracle."""
    P = require_gpu()
    L = P._lib
    log("attn split rows B=2 L=700 H=3 split_from=20 n_split=3")
    case = Case(P, 2, 700, 3, 128, 5, True, seed=79)
    for _ in range(6):
        case.append()
    rule = case.rule(0.5)
    case.gpu_lists(rule)
    q = case.query()
    o1, l1 = case.attention(q)
    o = torch.empty_like(q)
    lse = torch.empty_like(l1)
    work = torch.empty(L.uf_attn_split_rows_work_bytes(case.win.handle, 20, 3), dtype=torch.uint8, device="cuda")
    L.uf_sparse_causal_attn_fwd_split_rows(case.win.handle, q, case.win.lists, 1 / math.sqrt(128), o, lse, 20, 3, work)
    torch.cuda.synchronize()
    bits = case.oracle_bits(rule)
    O, LSE = oracle.sparse_causal_attention(case.ring, case._host(q), bits, 128, 1 / math.sqrt(128))
    err = row_rel_err(case._host(o), O)
    lerr = float(np.abs(f64(lse) - LSE).max())
    log(f"  rel_err={err:.3e} lse_err={lerr:.3e}")
    assert err <= REL_TOL and lerr <= lse_tol(128)
    # the binding's split=(split_from, n_split) is the same call
    o2, l2 = case.win.attention(q, 1 / math.sqrt(128), split=(20, 3))
    torch.cuda.synchronize()
    assert torch.equal(o2, o) and torch.equal(l2, lse)
    # rows before split_from run the unsplit code: bit-identical to the plain kernel
    rows_whole = 20                  # rows (b*H + h)*NT + i with NT = 6
    for r in range(rows_whole):
        b, rem = divmod(r, 3 * 6)
        h, i = divmod(rem, 6)
        assert torch.equal(o[b, 128 * i:128 * (i + 1), h], o1[b, 128 * i:128 * (i + 1), h])

    wl, case = _workload_case(P, "480p", "cuda")
    for _ in range(wl.window_chunks):
        case.append()
    assert L.uf_attn_tail_plan(case.win.handle, 256) == (444, 1)
    log("attn split rows 480p (256, 4)")
    rule = case.rule(wl.p_prior)
    case.gpu_lists(rule)
    q = case.query()
    o = torch.empty_like(q)
    lse = torch.empty((1, wl.heads, wl.chunk_tokens), dtype=torch.float32, device="cuda")
    work = torch.empty(L.uf_attn_split_rows_work_bytes(case.win.handle, 256, 4), dtype=torch.uint8, device="cuda")
    L.uf_sparse_causal_attn_fwd_split_rows(case.win.handle, q, case.win.lists, 1 / math.sqrt(128), o, lse, 256, 4,
                                           work)
    torch.cuda.synchronize()
    bits = case.oracle_bits(rule)
    O, LSE = oracle.sparse_causal_attention(case.ring, case._host(q), bits, wl.tile, 1 / math.sqrt(128))
    err = row_rel_err(case._host(o), O)
    lerr = float(np.abs(f64(lse) - LSE).max())
    log(f"  rel_err={err:.3e} lse_err={lerr:.3e}")
    assert err <= REL_TOL and lerr <= lse_tol(128)


@pytest.mark.parametrize("n_split", [2, 3, 5])
def test_split_kv_parity_t64(n_split):
    """Split-KV with 64-token tiles (ragged tail, evictions, a pinned chunk)
    against the oracle and the unsplit 64-token kernel."""
    P = require_gpu()
    log(f"attn split t64 n_split={n_split}")
    case = Case(P, 1, 130, 2, 64, 3, True, seed=80)
    for _ in range(5):
        case.append()
    rule = case.rule(0.4)
    case.gpu_lists(rule)
    q = case.query()
    o1, l1 = case.attention(q)
    os_, ls_ = case.win.attention(q, split=n_split)
    torch.cuda.synchronize()
    bits = case.oracle_bits(rule)
    O, LSE = oracle.sparse_causal_attention(case.ring, case._host(q), bits, 64, 1 / math.sqrt(128))
    err = row_rel_err(case._host(os_), O)
    lerr = float(np.abs(f64(ls_) - LSE).max())
    log(f"  rel_err={err:.3e} lse_err={lerr:.3e}")
    assert err <= REL_TOL and lerr <= lse_tol(64)
    assert row_rel_err(case._host(os_), case._host(o1)) <= REL_TOL


def test_tiny_workload_split_rows():
    """The tiny workload (6 rows of 64-token tiles, too short for the plan to
    split) with every row cut into one slice per key tile, in full against the
    oracle."""
    P = require_gpu()
    L = P._lib
    wl, case = _workload_case(P, "tiny", "cpu")
    for _ in range(wl.window_chunks):
        case.append()
    assert L.uf_attn_tail_plan(case.win.handle, 256) == (6, 1)
    log("attn tiny split rows (0, 6)")
    rule = case.rule(wl.p_prior)
    case.gpu_lists(rule)
    q = case.query()
    o = torch.empty_like(q)
    lse = torch.empty((1, wl.heads, wl.chunk_tokens), dtype=torch.float32, device="cuda")
    work = torch.empty(L.uf_attn_split_rows_work_bytes(case.win.handle, 0, 6), dtype=torch.uint8, device="cuda")
    L.uf_sparse_causal_attn_fwd_split_rows(case.win.handle, q, case.win.lists, 1 / math.sqrt(128), o, lse, 0, 6, work)
    torch.cuda.synchronize()
    bits = case.oracle_bits(rule)
    O, LSE = oracle.sparse_causal_attention(case.ring, case._host(q), bits, wl.tile, 1 / math.sqrt(128))
    err = row_rel_err(case._host(o), O)
    lerr = float(np.abs(f64(lse) - LSE).max())
    log(f"  rel_err={err:.3e} lse_err={lerr:.3e}")
    assert err <= REL_TOL and lerr <= lse_tol(64)


def test_plan_chosen_split_long_window_few_rows():
    """A window of 32 chunks whose 5 rows (one head, 5 query tiles) fill few
    CUs: the plan cuts every row into 51 slices, and the attention with
    split="tail" (plan, split launch, merge) matches the oracle in full."""
    P = require_gpu()
    L = P._lib
    log("attn plan-chosen split: 32 chunks, 5 rows")
    case = Case(P, 1, 640, 1, 128, 32, True, seed=83)
    for _ in range(32):
        case.append()
    assert L.uf_attn_tail_plan(case.win.handle, 256) == (0, 51)
    rule = case.rule(0.6)
    case.gpu_lists(rule)
    q = case.query()
    o, lse = case.win.attention(q, split="tail")
    o1, l1 = case.win.attention(q)
    torch.cuda.synchronize()
    bits = case.oracle_bits(rule)
    O, LSE = oracle.sparse_causal_attention(case.ring, case._host(q), bits, 128, 1 / math.sqrt(128))
    err = row_rel_err(case._host(o), O)
    lerr = float(np.abs(f64(lse) - LSE).max())
    log(f"  rel_err={err:.3e} lse_err={lerr:.3e}")
    assert err <= REL_TOL and lerr <= lse_tol(128)
    assert row_rel_err(case._host(o), case._host(o1)) <= REL_TOL
