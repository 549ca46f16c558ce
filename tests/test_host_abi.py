"""Host-side tests of the C ABI (no GPU): exported symbols, the window's
metadata against the oracle's window model under random append/evict
scripts (dry-run mode), and every error path that the host can force."""

import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "uf.h")


@pytest.fixture(scope="module")
def P():
    import paper_2606_09150_amd as pkg
    from paper_2606_09150_amd import _lib
    if not os.path.exists(_lib.LIB_PATH):
        pytest.fail("libuf.so is not built (python -m paper_2606_09150_amd.build)")
    pkg.load()
    return pkg


def _declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:int|const char\*)\s+(uf_\w+)\s*\(", text, re.M)))


def test_library_exports_every_declared_symbol(P):
    from paper_2606_09150_amd import _lib
    names = _declared()
    assert len(names) == 27
    lib = ctypes.CDLL(_lib.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", _lib.LIB_PATH], capture_output=True, text=True).stdout
    exported = sorted(set(re.findall(r"\sT\s(uf_\w+)$", out, re.M)))
    assert exported == names
    assert set(_lib._SIGNATURES) == set(names)


def _dry(P, max_chunks=5, pin_sink=True, L=300, T=128, B=1, H=2):
    return P.KVWindow(B, H, L, T, max_chunks, pin_sink, flags=P._lib.UF_F_DRYRUN)


@pytest.mark.parametrize("pin_sink", [True, False])
@pytest.mark.parametrize("seed", range(6))
def test_dry_run_window_matches_oracle_model(P, pin_sink, seed):
    rng = np.random.default_rng(seed)
    max_chunks = int(rng.integers(1, 7))
    w = _dry(P, max_chunks=max_chunks, pin_sink=pin_sink)
    model = oracle.RingModel(max_chunks, pin_sink)
    z = np.zeros((1, 1, 1, 1))
    for _ in range(60):
        if rng.random() < 0.6:
            try:
                model.append(z, z)
                want = None
            except oracle.RingCapacityError:
                want = P._lib.UF_ERR_CAPACITY
            try:
                w.append(None, None)
                got = None
            except P.UfError as e:
                got = e.status
        else:
            n = int(rng.integers(0, 4))
            try:
                model.evict(n)
                want = None
            except oracle.RingEmptyError:
                want = P._lib.UF_ERR_EMPTY
            try:
                w.evict(n)
                got = None
            except P.UfError as e:
                got = e.status
        assert got == want
        info = w.info()
        chunks = model.logical_chunks()
        assert info.n_live == len(chunks)
        assert info.nk_tiles == len(chunks) * info.nq_tiles
        seqs = [w.logical(p)[1] for p in range(info.n_live)]
        assert seqs == [c.seq for c in chunks]
        slots = [w.logical(p)[0] for p in range(info.n_live)]
        assert len(set(slots)) == len(slots) and all(0 <= s < max_chunks for s in slots)
        assert info.has_sink == int(bool(chunks) and chunks[0].sink)
        assert info.first_seq == (chunks[0].seq if chunks else -1)
        assert info.last_seq == (chunks[-1].seq if chunks else -1)


def test_geometry_and_layout(P):
    w = _dry(P, max_chunks=5, L=24480, T=128, H=12)
    info = w.info()
    assert (info.nq_tiles, info.tail_valid, info.nk_cap) == (192, 32, 960)
    lay = w.layout
    rows = 12 * 192
    assert lay.rows == rows and lay.nk_cap == 960 and lay.mask_words == 30
    assert lay.counts_offset == 0 and lay.idx_offset % 256 == 0 and lay.mask_offset % 256 == 0
    assert lay.idx_offset >= 4 * rows
    assert lay.mask_offset >= lay.idx_offset + 4 * rows * 960
    assert lay.scratch_offset % 256 == 0 and lay.scratch_offset >= lay.mask_offset + 4 * rows * 30
    assert lay.total_bytes >= lay.scratch_offset + 4 * rows * 128
    assert w.pool_bytes == 5 * 12 * 192 * (4 * 128 * 128 + 4 * 128)   # pages, then pooled keys


def test_error_paths(P):
    L = P._lib
    E = P.UfError

    def status(fn, *a):
        with pytest.raises(E) as ei:
            fn(*a)
        return ei.value.status

    base = dict(batch=1, heads=2, chunk_tokens=100, tile=128, max_chunks=3, pin_sink=1, head_dim=128, flags=0)
    bad = [
        (dict(batch=0), L.UF_ERR_ARG), (dict(heads=0), L.UF_ERR_ARG), (dict(chunk_tokens=0), L.UF_ERR_ARG),
        (dict(max_chunks=0), L.UF_ERR_ARG), (dict(max_chunks=65), L.UF_ERR_ARG), (dict(pin_sink=2), L.UF_ERR_ARG),
        (dict(flags=8), L.UF_ERR_ARG), (dict(head_dim=64), L.UF_ERR_UNSUPPORTED),
        (dict(tile=32), L.UF_ERR_UNSUPPORTED), (dict(batch=1 << 20, heads=1 << 10), L.UF_ERR_ARG),
    ]
    for change, code in bad:
        d = L.make_desc(**{**base, **change})
        assert status(L.uf_kv_pool_bytes, d) == code
    d = L.make_desc(**base)
    need = L.uf_kv_pool_bytes(d)

    class FakePtr:  # an aligned address that is never dereferenced on these paths
        def __init__(self, p):
            self.p = p

        def data_ptr(self):
            return self.p

    assert status(L.uf_kv_create, d, None, need) == L.UF_ERR_ARG
    assert status(L.uf_kv_create, d, FakePtr(0x10000 + 8), need) == L.UF_ERR_ARG
    assert status(L.uf_kv_create, d, FakePtr(0x10000), need - 1) == L.UF_ERR_CAPACITY
    h = L.uf_kv_create(d, FakePtr(0x10000), need)
    try:
        # no chunk yet
        assert status(L.uf_sparse_causal_attn_fwd, h, FakePtr(0x20000), FakePtr(0x30000), 0.1,
                      FakePtr(0x40000), None, 0) == L.UF_ERR_EMPTY
        rule = L.uf_keep_rule(1, 0.5, 1, 1)
        assert status(L.uf_build_tile_lists, h, rule, FakePtr(0x30000), 1 << 20, 0) == L.UF_ERR_EMPTY
        assert status(L.uf_kv_evict, h, 1) == L.UF_ERR_EMPTY
        assert status(L.uf_kv_evict, h, -1) == L.UF_ERR_ARG
        # append argument checks happen before any launch
        assert status(L.uf_kv_append, h, None, FakePtr(0x20000), 0) == L.UF_ERR_ARG
        assert status(L.uf_kv_append, h, FakePtr(0x20008), FakePtr(0x20000), 0) == L.UF_ERR_ARG
        assert L.uf_kv_get_info(h).n_live == 0
        assert status(L.uf_kv_logical, h, 0) == L.UF_ERR_ARG
    finally:
        L.uf_kv_destroy(h)
    # rule and scale checks on a dry-run window that holds a chunk
    w = _dry(P, max_chunks=2)
    w.append(None, None)
    for p in (-0.1, 1.5, float("nan")):
        assert status(L.uf_build_tile_lists, w.handle, L.uf_keep_rule(1, p, 1, 1), None, 0) == L.UF_ERR_ARG
    assert status(L.uf_build_tile_lists, w.handle, L.uf_keep_rule(1, 0.5, 2, 1), None, 0) == L.UF_ERR_ARG
    L.uf_build_tile_lists(w.handle, L.uf_keep_rule(1, 0.5, 1, 1), None, 0)
    for bad in (float("inf"), float("nan"), 0.0, -0.1, 1e-45):
        assert status(L.uf_sparse_causal_attn_fwd, w.handle, None, None, bad, None) == L.UF_ERR_ARG
    L.uf_sparse_causal_attn_fwd(w.handle, None, None, 0.1, None)
    w.append(None, None)
    assert status(L.uf_kv_append, w.handle, None, None) == L.UF_ERR_CAPACITY
    assert status(L.uf_kv_evict, w.handle, 2) == L.UF_ERR_EMPTY   # the pinned chunk is not evictable
    w.evict(1)
    assert w.info().n_live == 1 and w.info().has_sink == 1
    # status strings and the null handle
    assert L.uf_status_string(0) == "UF_OK"
    for code in (L.UF_ERR_ARG, L.UF_ERR_UNSUPPORTED, L.UF_ERR_CAPACITY, L.UF_ERR_EMPTY, L.UF_ERR_HIP):
        assert L.uf_status_string(code).startswith("UF_ERR_")
    assert status(L.uf_kv_evict, None, 1) == L.UF_ERR_ARG
    assert "null" in L.uf_last_error()


def test_topk_host_paths(P):
    """Top-k builder checks that need no device, and Eq. 10's budget helper."""
    L = P._lib
    E = P.UfError

    def status(fn, *a):
        with pytest.raises(E) as ei:
            fn(*a)
        return ei.value.status

    w = _dry(P, max_chunks=4, L=300, T=128)
    assert status(L.uf_build_topk_lists, w.handle, None, L.uf_topk_rule(3, 1, 1, 0), None, 0) == L.UF_ERR_EMPTY
    w.append(None, None)
    w.append(None, None)
    L.uf_build_topk_lists(w.handle, None, L.uf_topk_rule(3, 1, 1, 0), None, 0)      # dry run: no device work
    for rule in (L.uf_topk_rule(-1, 1, 1, 0), L.uf_topk_rule(1, 2, 1, 0), L.uf_topk_rule(1, 1, -1, 0),
                 L.uf_topk_rule(1, 1, 1, 7)):
        assert status(L.uf_build_topk_lists, w.handle, None, rule, None, 0) == L.UF_ERR_ARG
    # more ranked candidates per row than the builder supports
    big = _dry(P, max_chunks=4, L=128 * 8200, T=128, H=1)
    for _ in range(3):
        big.append(None, None)
    assert status(L.uf_build_topk_lists, big.handle, None, L.uf_topk_rule(5, 0, 0, 0), None, 0) == L.UF_ERR_UNSUPPORTED
    L.uf_build_topk_lists(big.handle, None, L.uf_topk_rule(5, 1, 1, 0), None, 0)     # 8200 candidates: fine
    # Eq. 10 through the C helper agrees with the oracle's helper
    for rho, S, Sr, n, kmin in ((1.0, 1560, 1560, 200, 4), (1.0, 8160, 1560, 960, 4), (0.25, 1560, 1560, 576, 4),
                                (0.7, 100, 1560, 10, 4), (2.0, 14400, 1560, 1352, 0), (0.0, 5, 7, 9, 3)):
        assert L.uf_topk_budget(rho, S, Sr, n, kmin) == oracle.topk_budget(rho, S, Sr, n, kmin)
    assert L.uf_topk_budget(1e9, 10 ** 9, 1, 10 ** 9, 0) == 2 ** 31 - 1                 # clamped
    for args in ((-1.0, 1, 1, 1, 0), (float("nan"), 1, 1, 1, 0), (1.0, 1, 0, 1, 0), (1.0, -1, 1, 1, 0),
                 (1.0, 1, 1, 1, -1)):
        assert status(L.uf_topk_budget, *args) == L.UF_ERR_ARG


def test_replace_newest_keeps_window_metadata(P):
    L = P._lib
    w = _dry(P, max_chunks=3)
    with pytest.raises(P.UfError) as ei:
        w.replace_newest(None, None)
    assert ei.value.status == L.UF_ERR_EMPTY
    for _ in range(3):
        w.append(None, None)
    before = [w.logical(p) for p in range(3)], (w.info().first_seq, w.info().last_seq, w.info().n_live)
    w.replace_newest(None, None)
    after = [w.logical(p) for p in range(3)], (w.info().first_seq, w.info().last_seq, w.info().n_live)
    assert before == after


def test_split_kv_host_paths(P):
    L = P._lib
    E = P.UfError

    def status(fn, *a):
        with pytest.raises(E) as ei:
            fn(*a)
        return ei.value.status

    w = _dry(P, max_chunks=4, L=300, T=128, H=2)
    rows = 2 * 3
    assert L.uf_attn_split_work_bytes(w.handle, 4) == rows * 4 * 128 * 130 * 4
    for n in (0, -1, 65):
        assert status(L.uf_attn_split_work_bytes, w.handle, n) == L.UF_ERR_ARG
    assert status(L.uf_sparse_causal_attn_fwd_split, w.handle, None, None, 0.1, None, None, 2, None, 0) == L.UF_ERR_EMPTY
    w.append(None, None)
    L.uf_sparse_causal_attn_fwd_split(w.handle, None, None, 0.1, None, None, 2, None, 0)   # dry run
    assert status(L.uf_sparse_causal_attn_fwd_split, w.handle, None, None, 0.1, None, None, 0, None, 0) == L.UF_ERR_ARG
    # 64-token tiles: partials of 64 rows per slice
    w64 = _dry(P, max_chunks=2, L=300, T=64)
    w64.append(None, None)
    assert L.uf_attn_split_work_bytes(w64.handle, 2) == (2 * 5) * 2 * 64 * 130 * 4
    L.uf_sparse_causal_attn_fwd_split(w64.handle, None, None, 0.1, None, None, 2, None, 0)   # dry run


def test_backward_host_paths(P):
    L = P._lib
    E = P.UfError

    def status(fn, *a):
        with pytest.raises(E) as ei:
            fn(*a)
        return ei.value.status

    w = _dry(P, max_chunks=4, L=300, T=128, H=2)
    rows = 2 * 3
    # per row: Q and dO rows (32 KB each) + LSE and delta
    assert L.uf_attn_bwd_work_bytes(w.handle) == rows * (2 * 32768 + 1024)
    bwd = L.uf_sparse_causal_attn_bwd
    args = (None, None, None, None, None, 0.1, None, None, None, None, 0)
    assert status(bwd, w.handle, *args) == L.UF_ERR_EMPTY
    w.append(None, None)
    bwd(w.handle, *args)                                                   # dry run: no device work
    for bad in (0.0, -1.0, float("inf"), float("nan")):
        assert status(bwd, w.handle, None, None, None, None, None, bad, None, None, None, None, 0) == L.UF_ERR_ARG
    # 64-token tiles: one record per list row as well (2 heads x 5 query tiles)
    w64 = _dry(P, max_chunks=2, L=300, T=64)
    w64.append(None, None)
    assert L.uf_attn_bwd_work_bytes(w64.handle) == 10 * 66560
    bwd(w64.handle, *args)
    many = _dry(P, max_chunks=2, L=2049 * 64, T=64)                      # 2,049 query tiles per chunk
    many.append(None, None)
    assert status(bwd, many.handle, *args) == L.UF_ERR_UNSUPPORTED

    # the no-allocation variant: same checks, no workspace, and a capacity
    # limit of its own scratch (66,560 bytes per list row, 64 MiB in all)
    na = L.uf_sparse_causal_attn_bwd_noalloc
    nargs = (None, None, None, None, None, 0.1, None, None, None)
    wn = _dry(P, max_chunks=4, L=300, T=128, H=2)
    assert status(na, wn.handle, *nargs) == L.UF_ERR_EMPTY
    wn.append(None, None)
    na(wn.handle, *nargs)                                                  # dry run: no device work
    na(w64.handle, *nargs)
    fits = _dry(P, max_chunks=2, L=1008 * 128, T=128, H=1)               # 1,008 rows: exactly the scratch
    fits.append(None, None)
    na(fits.handle, *nargs)
    big = _dry(P, max_chunks=2, L=24480, T=128, H=12)                    # the 1K window: 2,304 rows
    big.append(None, None)
    assert status(na, big.handle, *nargs) == L.UF_ERR_CAPACITY
    assert "1008 rows" in L.uf_last_error()


def test_tail_plan_and_split_rows_host_paths(P):
    L = P._lib
    E = P.UfError

    def status(fn, *a):
        with pytest.raises(E) as ei:
            fn(*a)
        return ei.value.status

    def plan(B, L_, H, n_cu, T=128, chunks=1):
        w = _dry(P, max_chunks=max(2, chunks), L=L_, T=T, H=H, B=B)
        for _ in range(chunks):
            w.append(None, None)
        return L.uf_attn_tail_plan(w.handle, n_cu)

    # 480p: 444 rows on 256 CUs; 4 slices of rows 256.. would take 1.75
    # row-times plus three slices' and the merge's fixed costs (2.03 against
    # 2 whole), so no split
    assert plan(1, 4680, 12, 256, chunks=4) == (444, 1)
    # 1K: 2,304 rows are nine whole rounds; 2K: 4,056 rows leave 216 in the last
    # round, where no slice count saves a fifth of a row-time
    assert plan(1, 24480, 12, 256, chunks=5) == (2304, 1)
    assert plan(1, 43200, 12, 256, chunks=4) == (4056, 1)
    # fewer rows than CUs: every row split, at most into as many slices as the
    # window has key tiles (160 here), when rows are long enough to repay it
    w = _dry(P, max_chunks=32, L=640, T=128, H=1)
    for _ in range(32):
        w.append(None, None)
    assert L.uf_attn_tail_plan(w.handle, 256) == (0, 51)
    # short rows (5 or 6 key tiles) are not split
    assert plan(1, 640, 1, 256) == (5, 1)
    assert plan(1, 192, 2, 256, T=64, chunks=2) == (6, 1)
    w = _dry(P, max_chunks=4, L=300, T=128, H=2)
    rows = 2 * 3
    assert L.uf_attn_split_rows_work_bytes(w.handle, 2, 3) == (rows - 2) * 3 * 128 * 130 * 4
    assert L.uf_attn_split_rows_work_bytes(w.handle, rows, 3) == 0
    assert status(L.uf_attn_split_rows_work_bytes, w.handle, rows + 1, 3) == L.UF_ERR_ARG
    assert status(L.uf_attn_split_rows_work_bytes, w.handle, 0, 0) == L.UF_ERR_ARG
    assert status(L.uf_attn_tail_plan, w.handle, 0) == L.UF_ERR_ARG
    fn = L.uf_sparse_causal_attn_fwd_split_rows
    assert status(fn, w.handle, None, None, 0.1, None, None, 0, 2, None, 0) == L.UF_ERR_EMPTY
    w.append(None, None)
    fn(w.handle, None, None, 0.1, None, None, 2, 3, None, 0)             # dry run
    assert status(fn, w.handle, None, None, 0.1, None, None, -1, 3, None, 0) == L.UF_ERR_ARG
    assert status(fn, w.handle, None, None, 0.1, None, None, 0, 65, None, 0) == L.UF_ERR_ARG
