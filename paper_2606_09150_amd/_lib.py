"""ctypes binding of libuf.so: the C ABI entry points under the same names.

Argument marshalling only: torch tensors supply device pointers and the
current HIP stream; every step of the path runs in the library's kernels.
A missing library is an error, never a fallback.
"""

import ctypes
import os

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libuf.so")

UF_OK = 0
UF_ERR_ARG = -1
UF_ERR_UNSUPPORTED = -2
UF_ERR_CAPACITY = -3
UF_ERR_EMPTY = -4
UF_ERR_HIP = -5
UF_F_DRYRUN = 1
UF_F_POISON_PAD = 2
UF_MAX_CHUNKS = 64


class UfError(RuntimeError):
    def __init__(self, status: int, detail: str):
        self.status = status
        super().__init__(f"{_status_text(status)}: {detail}")


class uf_kv_desc(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("chunk_tokens", ctypes.c_int32), ("tile", ctypes.c_int32), ("max_chunks", ctypes.c_int32),
                ("pin_sink", ctypes.c_int32), ("flags", ctypes.c_uint32)]


class uf_keep_rule(ctypes.Structure):
    _fields_ = [("seed", ctypes.c_uint64), ("p_prior", ctypes.c_double),
                ("keep_sink", ctypes.c_int32), ("keep_current", ctypes.c_int32),
                ("local_r", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class uf_block_geom(ctypes.Structure):
    _fields_ = [("frames", ctypes.c_int32), ("grid_h", ctypes.c_int32), ("grid_w", ctypes.c_int32),
                ("bt", ctypes.c_int32), ("bh", ctypes.c_int32), ("bw", ctypes.c_int32)]


class uf_topk_rule(ctypes.Structure):
    _fields_ = [("budget", ctypes.c_int32), ("keep_sink", ctypes.c_int32),
                ("keep_current", ctypes.c_int32), ("local_r", ctypes.c_int32)]


class uf_kv_info(ctypes.Structure):
    _fields_ = [("n_live", ctypes.c_int32), ("nq_tiles", ctypes.c_int32), ("nk_tiles", ctypes.c_int32),
                ("tail_valid", ctypes.c_int32), ("first_seq", ctypes.c_int64), ("last_seq", ctypes.c_int64),
                ("has_sink", ctypes.c_int32), ("nk_cap", ctypes.c_int32)]


class uf_lists_layout(ctypes.Structure):
    _fields_ = [("counts_offset", ctypes.c_size_t), ("idx_offset", ctypes.c_size_t),
                ("mask_offset", ctypes.c_size_t), ("scratch_offset", ctypes.c_size_t),
                ("total_bytes", ctypes.c_size_t),
                ("rows", ctypes.c_int32), ("nk_cap", ctypes.c_int32), ("mask_words", ctypes.c_int32),
                ("reserved", ctypes.c_int32)]


_P = ctypes.c_void_p
_SIGNATURES = {
    "uf_kv_pool_bytes": (ctypes.c_int, [ctypes.POINTER(uf_kv_desc), ctypes.POINTER(ctypes.c_size_t)]),
    "uf_kv_create": (ctypes.c_int, [ctypes.POINTER(uf_kv_desc), _P, ctypes.c_size_t, ctypes.POINTER(_P)]),
    "uf_kv_destroy": (ctypes.c_int, [_P]),
    "uf_kv_append": (ctypes.c_int, [_P, _P, _P, _P]),
    "uf_kv_evict": (ctypes.c_int, [_P, ctypes.c_int32]),
    "uf_block_geom_tokens": (ctypes.c_int, [ctypes.POINTER(uf_block_geom), ctypes.POINTER(ctypes.c_int32),
                                            ctypes.POINTER(ctypes.c_int32)]),
    "uf_kv_set_block_geom": (ctypes.c_int, [_P, ctypes.POINTER(uf_block_geom)]),
    "uf_block_permute": (ctypes.c_int, [ctypes.POINTER(uf_block_geom), ctypes.c_int32, ctypes.c_int32,
                                        ctypes.c_int32, _P, _P, ctypes.c_int32, _P]),
    "uf_kv_replace_newest": (ctypes.c_int, [_P, _P, _P, _P]),
    "uf_kv_get_info": (ctypes.c_int, [_P, ctypes.POINTER(uf_kv_info)]),
    "uf_kv_logical": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32),
                                     ctypes.POINTER(ctypes.c_int64)]),
    "uf_tile_lists_layout": (ctypes.c_int, [_P, ctypes.POINTER(uf_lists_layout)]),
    "uf_tile_lists_bytes": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_size_t)]),
    "uf_build_tile_lists": (ctypes.c_int, [_P, ctypes.POINTER(uf_keep_rule), _P, ctypes.c_size_t, _P]),
    "uf_build_topk_lists": (ctypes.c_int, [_P, _P, ctypes.POINTER(uf_topk_rule), _P, ctypes.c_size_t, _P]),
    "uf_topk_budget": (ctypes.c_int, [ctypes.c_double, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                      ctypes.c_int32, ctypes.POINTER(ctypes.c_int32)]),
    "uf_sparse_causal_attn_fwd": (ctypes.c_int, [_P, _P, _P, ctypes.c_float, _P, _P, _P]),
    "uf_attn_split_work_bytes": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)]),
    "uf_sparse_causal_attn_fwd_split": (ctypes.c_int, [_P, _P, _P, ctypes.c_float, _P, _P, ctypes.c_int32, _P,
                                                       ctypes.c_size_t, _P]),
    "uf_attn_tail_plan": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.POINTER(ctypes.c_int32),
                                         ctypes.POINTER(ctypes.c_int32)]),
    "uf_attn_split_rows_work_bytes": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_int32,
                                                     ctypes.POINTER(ctypes.c_size_t)]),
    "uf_sparse_causal_attn_fwd_split_rows": (ctypes.c_int, [_P, _P, _P, ctypes.c_float, _P, _P, ctypes.c_int32,
                                                            ctypes.c_int32, _P, ctypes.c_size_t, _P]),
    "uf_attn_bwd_work_bytes": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_size_t)]),
    "uf_sparse_causal_attn_bwd": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, _P,
                                                 ctypes.c_size_t, _P]),
    "uf_sparse_causal_attn_bwd_noalloc": (ctypes.c_int, [_P, _P, _P, _P, _P, _P, ctypes.c_float, _P, _P, _P, _P]),
    "uf_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "uf_last_error": (ctypes.c_char_p, []),
}

_lib = None


def load():
    """Load libuf.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2606_09150_amd.build`")
        lib = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


def _status_text(status: int) -> str:
    return load().uf_status_string(status).decode()


def _check(status: int) -> None:
    if status != UF_OK:
        raise UfError(status, load().uf_last_error().decode())


def _stream_ptr(stream):
    """hipStream_t of a torch stream (None: the current stream of the current device)."""
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _ptr(t):
    return None if t is None else t.data_ptr()


# --------------------------------------------------------------------------
# Entry points (same names as the C ABI)
# --------------------------------------------------------------------------

def make_desc(batch, heads, chunk_tokens, tile, max_chunks, pin_sink, head_dim=128, flags=0) -> uf_kv_desc:
    return uf_kv_desc(batch, heads, head_dim, chunk_tokens, tile, max_chunks, int(pin_sink), flags)


def uf_kv_pool_bytes(desc: uf_kv_desc) -> int:
    out = ctypes.c_size_t()
    _check(load().uf_kv_pool_bytes(ctypes.byref(desc), ctypes.byref(out)))
    return out.value


def uf_kv_create(desc: uf_kv_desc, pool, pool_bytes: int = None):
    """pool: a device tensor (or None under UF_F_DRYRUN). Returns the opaque handle."""
    h = _P()
    ptr = _ptr(pool)
    nbytes = pool_bytes if pool_bytes is not None else (0 if pool is None else pool.numel() * pool.element_size())
    _check(load().uf_kv_create(ctypes.byref(desc), ptr, nbytes, ctypes.byref(h)))
    return h


def uf_kv_destroy(handle) -> None:
    _check(load().uf_kv_destroy(handle))


def uf_kv_append(handle, k, v, stream=None) -> None:
    s = None if (k is None and v is None) else _stream_ptr(stream)
    _check(load().uf_kv_append(handle, _ptr(k), _ptr(v), s))


def uf_kv_replace_newest(handle, k, v, stream=None) -> None:
    s = None if k is None else _stream_ptr(stream)
    _check(load().uf_kv_replace_newest(handle, _ptr(k), _ptr(v), s))


def uf_block_geom_tokens(geom: uf_block_geom):
    padded, nb = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(load().uf_block_geom_tokens(ctypes.byref(geom), ctypes.byref(padded), ctypes.byref(nb)))
    return padded.value, nb.value


def uf_kv_set_block_geom(handle, geom: uf_block_geom) -> None:
    _check(load().uf_kv_set_block_geom(handle, ctypes.byref(geom)))


def uf_block_permute(geom: uf_block_geom, batch: int, heads: int, src, dst, inverse: int, head_dim: int = 128,
                     stream=None) -> None:
    s = None if src is None else _stream_ptr(stream)
    _check(load().uf_block_permute(ctypes.byref(geom), batch, heads, head_dim, _ptr(src), _ptr(dst), int(inverse), s))


def uf_kv_evict(handle, n_chunks: int) -> None:
    _check(load().uf_kv_evict(handle, n_chunks))


def uf_kv_get_info(handle) -> uf_kv_info:
    info = uf_kv_info()
    _check(load().uf_kv_get_info(handle, ctypes.byref(info)))
    return info


def uf_kv_logical(handle, pos: int):
    slot, seq = ctypes.c_int32(), ctypes.c_int64()
    _check(load().uf_kv_logical(handle, pos, ctypes.byref(slot), ctypes.byref(seq)))
    return slot.value, seq.value


def uf_tile_lists_layout(handle) -> uf_lists_layout:
    lay = uf_lists_layout()
    _check(load().uf_tile_lists_layout(handle, ctypes.byref(lay)))
    return lay


def uf_tile_lists_bytes(handle) -> int:
    out = ctypes.c_size_t()
    _check(load().uf_tile_lists_bytes(handle, ctypes.byref(out)))
    return out.value


def uf_build_tile_lists(handle, rule: uf_keep_rule, lists, nbytes: int = None, stream=None) -> None:
    n = nbytes if nbytes is not None else (0 if lists is None else lists.numel() * lists.element_size())
    s = None if lists is None else _stream_ptr(stream)
    _check(load().uf_build_tile_lists(handle, ctypes.byref(rule), _ptr(lists), n, s))


def uf_build_topk_lists(handle, q, rule: uf_topk_rule, lists, nbytes: int = None, stream=None) -> None:
    n = nbytes if nbytes is not None else (0 if lists is None else lists.numel() * lists.element_size())
    s = None if lists is None else _stream_ptr(stream)
    _check(load().uf_build_topk_lists(handle, _ptr(q), ctypes.byref(rule), _ptr(lists), n, s))


def uf_topk_budget(rho: float, seq_len: int, seq_ref: int, n_blocks: int, k_min: int = 4) -> int:
    out = ctypes.c_int32(0)
    _check(load().uf_topk_budget(ctypes.c_double(rho), seq_len, seq_ref, n_blocks, k_min, ctypes.byref(out)))
    return out.value


def uf_sparse_causal_attn_fwd(handle, q, lists, scale: float, o, lse=None, stream=None) -> None:
    s = None if q is None else _stream_ptr(stream)
    _check(load().uf_sparse_causal_attn_fwd(handle, _ptr(q), _ptr(lists), ctypes.c_float(scale),
                                            _ptr(o), _ptr(lse), s))


def uf_attn_split_work_bytes(handle, n_split: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load().uf_attn_split_work_bytes(handle, n_split, ctypes.byref(out)))
    return out.value


def uf_sparse_causal_attn_fwd_split(handle, q, lists, scale: float, o, lse, n_split: int, work,
                                    work_bytes: int = None, stream=None) -> None:
    n = work_bytes if work_bytes is not None else (0 if work is None else work.numel() * work.element_size())
    s = None if q is None else _stream_ptr(stream)
    _check(load().uf_sparse_causal_attn_fwd_split(handle, _ptr(q), _ptr(lists), ctypes.c_float(scale), _ptr(o),
                                                  _ptr(lse), n_split, _ptr(work), n, s))


def uf_attn_tail_plan(handle, n_cu: int):
    """(split_from, n_split) that balances the last round of rows over n_cu compute units."""
    f, s = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(load().uf_attn_tail_plan(handle, n_cu, ctypes.byref(f), ctypes.byref(s)))
    return f.value, s.value


def uf_attn_split_rows_work_bytes(handle, split_from: int, n_split: int) -> int:
    out = ctypes.c_size_t(0)
    _check(load().uf_attn_split_rows_work_bytes(handle, split_from, n_split, ctypes.byref(out)))
    return out.value


def uf_sparse_causal_attn_fwd_split_rows(handle, q, lists, scale: float, o, lse, split_from: int, n_split: int,
                                         work, work_bytes: int = None, stream=None) -> None:
    n = work_bytes if work_bytes is not None else (0 if work is None else work.numel() * work.element_size())
    s = None if q is None else _stream_ptr(stream)
    _check(load().uf_sparse_causal_attn_fwd_split_rows(handle, _ptr(q), _ptr(lists), ctypes.c_float(scale), _ptr(o),
                                                       _ptr(lse), split_from, n_split, _ptr(work), n, s))


def uf_attn_bwd_work_bytes(handle) -> int:
    out = ctypes.c_size_t(0)
    _check(load().uf_attn_bwd_work_bytes(handle, ctypes.byref(out)))
    return out.value


def uf_sparse_causal_attn_bwd(handle, q, o, do, lse, lists, scale: float, dq, dk, dv, work,
                              work_bytes: int = None, stream=None) -> None:
    n = work_bytes if work_bytes is not None else (0 if work is None else work.numel() * work.element_size())
    s = None if q is None else _stream_ptr(stream)
    _check(load().uf_sparse_causal_attn_bwd(handle, _ptr(q), _ptr(o), _ptr(do), _ptr(lse), _ptr(lists),
                                            ctypes.c_float(scale), _ptr(dq), _ptr(dk), _ptr(dv), _ptr(work), n, s))


def uf_sparse_causal_attn_bwd_noalloc(handle, q, o, do, lse, lists, scale: float, dq, dk, dv, stream=None) -> None:
    s = None if q is None else _stream_ptr(stream)
    _check(load().uf_sparse_causal_attn_bwd_noalloc(handle, _ptr(q), _ptr(o), _ptr(do), _ptr(lse), _ptr(lists),
                                                    ctypes.c_float(scale), _ptr(dq), _ptr(dk), _ptr(dv), s))


def uf_status_string(status: int) -> str:
    return _status_text(status)


def uf_last_error() -> str:
    return load().uf_last_error().decode()
