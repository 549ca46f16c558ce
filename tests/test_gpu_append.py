"""uf_kv_append: pages read back bit for bit against the layout documented in
include/uf.h (K and V transposed, in 64-column blocks for 128-token pages;
swap23 key order; padded tails)."""

import numpy as np
import pytest
import torch

import synth
from tests.gpu_common import log, require_gpu

pytestmark = pytest.mark.gpu


def _page_views(raw, T, D):
    """Logical K [T][D] and V^T [D][T] of a page (uf.h: 128-token pages keep
    both as two blocks of 64 columns, 64-token pages as plain rows)."""
    half = raw.size // 2
    k = raw[:half].view(np.uint16)
    v = raw[half:].view(np.uint16)
    if T == 128:
        k = k.reshape(2, T, 64).transpose(1, 0, 2).reshape(T, D)
        v = v.reshape(2, D, 64).transpose(1, 0, 2).reshape(D, T)
    else:
        k = k.reshape(T, D)
        v = v.reshape(D, T)
    return k, v


def _swap23(p):
    return (p & ~12) | ((p & 4) << 1) | ((p & 8) >> 1)


def _bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


@pytest.mark.parametrize("B,L,H,T,poison", [(1, 192, 2, 64, False), (2, 300, 3, 128, False),
                                            (1, 300, 2, 128, True), (1, 130, 1, 64, True)])
def test_pages_read_back(B, L, H, T, poison):
    P = require_gpu()
    log(f"append B={B} L={L} H={H} T={T} poison={poison}")
    flags = P._lib.UF_F_POISON_PAD if poison else 0
    win = P.KVWindow(B, H, L, T, 3, True, flags=flags)
    chunks = {}
    for c in range(5):
        if win.info().n_live == 3:
            win.evict(1)
        k = synth.custom_tensor((B, L, H, 128), 99, c, "k").cuda()
        v = synth.custom_tensor((B, L, H, 128), 99, c, "v").cuda()
        win.append(k, v)
        chunks[c] = (_bits(k), _bits(v))
    torch.cuda.synchronize()
    pool = win.pool.cpu().numpy()
    info = win.info()
    nt, tail = info.nq_tiles, info.tail_valid
    pad = 0x461C if poison else 0
    D = 128
    page = 4 * T * D
    assert info.n_live == 3
    for pos in range(info.n_live):
        slot, seq = win.logical(pos)
        kb, vb = chunks[seq]
        for b in range(B):
            for h in range(H):
                for t in range(nt):
                    off = (((slot * B + b) * H + h) * nt + t) * page
                    kpage, vpage = _page_views(pool[off:off + page], T, D)
                    valid = tail if t == nt - 1 else T
                    assert np.array_equal(kpage[:valid], kb[b, t * T:t * T + valid, h, :])
                    assert (kpage[valid:] == pad).all()
                    keys = np.array([_swap23(p) for p in range(T)])
                    want_v = np.full((D, T), pad, dtype=np.uint16)
                    ok = keys < valid
                    want_v[:, ok] = vb[b, t * T + keys[ok], h, :].T
                    assert np.array_equal(vpage, want_v)


def test_pages_read_back_1k_sampled():
    """The 1K workload's shape (12 heads, 24,480-token chunks, 128-token
    pages, five-slot ring): sampled pages of two appended chunks, bit for bit,
    including the partial last tile."""
    P = require_gpu()
    wl = synth.WORKLOADS["1k"]
    L, H, T, D = wl.chunk_tokens, wl.heads, wl.tile, 128
    log(f"append 1k sampled pages L={L} H={H} T={T}")
    win = P.KVWindow(1, H, L, T, wl.max_chunks, wl.pin_sink)
    chunks = {}
    for c in range(2):
        k = synth.custom_tensor((1, L, H, D), 7, c, "k", device="cuda")
        v = synth.custom_tensor((1, L, H, D), 7, c, "v", device="cuda")
        win.append(k, v)
        chunks[c] = (_bits(k), _bits(v))
    torch.cuda.synchronize()
    info = win.info()
    nt, tail = info.nq_tiles, info.tail_valid
    assert nt == -(-L // T) and tail == L - (nt - 1) * T
    page = 4 * T * D
    keys = np.array([_swap23(p) for p in range(T)])
    for pos in range(info.n_live):
        slot, seq = win.logical(pos)
        kb, vb = chunks[seq]
        for h in (0, 5, H - 1):
            for t in (0, 1, nt // 2, nt - 2, nt - 1):
                off = ((slot * H + h) * nt + t) * page
                raw = win.pool[off:off + page].cpu().numpy()
                kpage, vpage = _page_views(raw, T, D)
                valid = tail if t == nt - 1 else T
                assert np.array_equal(kpage[:valid], kb[0, t * T:t * T + valid, h, :])
                assert (kpage[valid:] == 0).all()
                want_v = np.zeros((D, T), dtype=np.uint16)
                ok = keys < valid
                want_v[:, ok] = vb[0, t * T + keys[ok], h, :].T
                assert np.array_equal(vpage, want_v)
