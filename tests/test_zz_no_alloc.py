"""The no-allocation backward (uf_sparse_causal_attn_bwd_noalloc through the C
ABI) against the allocating entry point, uf_sparse_causal_attn_bwd.

Both run the same kernels on the same query-tile records, the first from the
library's own device scratch and the second from the caller's workspace, so
the gradients must agree bit for bit.  Three no-allocation calls run in a
row, each later one on a smaller window (the last with 64-token tiles), so
that they read the scratch after an earlier call left its records there; the outputs start as NaN so that any element a
call leaves unwritten shows.
"""

import math

import pytest
import torch

from tests.gpu_common import Case, log, require_gpu

pytestmark = pytest.mark.gpu

CASES = [
    # B, L, H, max_chunks, n_chunks, p, seed, tile: 48 list rows, then 3, then 6
    (2, 1000, 3, 5, 6, 0.4, 3001, 128),
    (1, 300, 1, 3, 3, 0.6, 3002, 128),
    (1, 192, 2, 2, 2, 1.0, 3003, 64),
]


def _prepared(P, B, L, H, mc, n, p, seed, T):
    case = Case(P, B, L, H, T, mc, True, seed)
    for _ in range(n):
        case.append()
    case.gpu_lists(case.rule(p))
    scale = 1 / math.sqrt(128)
    q = case.query()
    o, lse = case.win.attention(q, scale)
    do = case._draw(case.n_appended - 1, "do")
    return case, q, o, lse, do, scale


def test_noalloc_backward_matches_the_allocating_entry_point():
    P = require_gpu()
    L = P._lib
    runs = [_prepared(P, *c) for c in CASES]
    got = []
    for case, q, o, lse, do, scale in runs:
        n_live = case.win.info().n_live
        dq = torch.full((case.B, case.L, case.H, 128), float("nan"), dtype=torch.float32, device="cuda")
        dk = torch.full((n_live, case.B, case.L, case.H, 128), float("nan"), dtype=torch.float32, device="cuda")
        dv = torch.full_like(dk, float("nan"))
        log(f"noalloc bwd B={case.B} L={case.L} H={case.H} T={case.T} rows={case.win.layout.rows}")
        L.uf_sparse_causal_attn_bwd_noalloc(case.win.handle, q, o, do, lse, case.win.lists, scale, dq, dk, dv)
        got.append((dq, dk, dv))
    torch.cuda.synchronize()
    for (case, q, o, lse, do, scale), g in zip(runs, got):
        want = case.win.attention_bwd(q, o, lse, do, scale)
        torch.cuda.synchronize()
        for a, b in zip(g, want):
            assert torch.equal(a, b)
    # a window beyond the scratch is refused before any device work
    big = P.KVWindow(1, 12, 24480, 128, 2, True)
    k = torch.zeros((1, 24480, 12, 128), dtype=torch.bfloat16, device="cuda")
    big.append(k, k)
    with pytest.raises(P.UfError) as ei:
        L.uf_sparse_causal_attn_bwd_noalloc(big.handle, k, k, k, torch.zeros((1, 12, 24480), device="cuda"),
                                            big.lists, 0.1, None, None, None)
    assert ei.value.status == L.UF_ERR_CAPACITY
