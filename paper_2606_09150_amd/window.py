"""A torch-facing wrapper over one KV window of the C ABI.

Holds the caller-side device buffers (the page pool and the list buffer, both
plain torch allocations) and checks tensor shapes, dtypes and devices before
each call, since the C ABI receives bare pointers.  All computation happens in
libuf.so's kernels.
"""

import math

import torch

from . import _lib as L


def _check_chunk(t, name, B, Lc, H, D):
    if t is None:
        raise ValueError(f"{name} is None")
    if t.dtype != torch.bfloat16:
        raise TypeError(f"{name} must be bfloat16 (got {t.dtype})")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if tuple(t.shape) != (B, Lc, H, D):
        raise ValueError(f"{name} must have shape {(B, Lc, H, D)} (got {tuple(t.shape)})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


class KVWindow:
    """Window of at most ``max_chunks`` chunks of ``chunk_tokens`` tokens."""

    def __init__(self, batch, heads, chunk_tokens, tile=128, max_chunks=4, pin_sink=True,
                 head_dim=128, flags=0, device=None):
        self.desc = L.make_desc(batch, heads, chunk_tokens, tile, max_chunks, pin_sink, head_dim, flags)
        self.B, self.H, self.L, self.D, self.T = batch, heads, chunk_tokens, head_dim, tile
        self.dry = bool(flags & L.UF_F_DRYRUN)
        self.pool_bytes = L.uf_kv_pool_bytes(self.desc)
        if self.dry:
            self.pool = None
            self.handle = L.uf_kv_create(self.desc, None, 0)
        else:
            dev = torch.device("cuda") if device is None else torch.device(device)
            self.pool = torch.empty(self.pool_bytes, dtype=torch.uint8, device=dev)
            self.handle = L.uf_kv_create(self.desc, self.pool, self.pool_bytes)
        self.layout = L.uf_tile_lists_layout(self.handle)
        self.lists = None
        if not self.dry:
            self.lists = torch.empty(self.layout.total_bytes, dtype=torch.uint8, device=self.pool.device)

    def close(self):
        if getattr(self, "handle", None) is not None:
            L.uf_kv_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- window -------------------------------------------------------------
    def append(self, k, v, stream=None):
        if not self.dry:
            _check_chunk(k, "k", self.B, self.L, self.H, self.D)
            _check_chunk(v, "v", self.B, self.L, self.H, self.D)
        L.uf_kv_append(self.handle, k, v, stream)

    def replace_newest(self, k, v, stream=None):
        """Refresh the current chunk's K and V in place (same sequence number)."""
        if not self.dry:
            _check_chunk(k, "k", self.B, self.L, self.H, self.D)
            _check_chunk(v, "v", self.B, self.L, self.H, self.D)
        L.uf_kv_replace_newest(self.handle, k, v, stream)

    def set_block_geom(self, frames, grid_h, grid_w, bt=2, bh=8, bw=8):
        """Tiles become (bt, bh, bw) blocks of a frames x grid_h x grid_w chunk (before any append)."""
        L.uf_kv_set_block_geom(self.handle, L.uf_block_geom(frames, grid_h, grid_w, bt, bh, bw))

    def evict(self, n=1):
        L.uf_kv_evict(self.handle, n)

    def info(self):
        return L.uf_kv_get_info(self.handle)

    def logical(self, pos):
        return L.uf_kv_logical(self.handle, pos)

    # -- lists --------------------------------------------------------------
    def build_lists(self, seed, p_prior, keep_sink=True, keep_current=True, stream=None, local_r=0):
        rule = L.uf_keep_rule(seed & 0xFFFFFFFFFFFFFFFF, float(p_prior), int(keep_sink), int(keep_current),
                              int(local_r), 0)
        L.uf_build_tile_lists(self.handle, rule, self.lists, None, stream)
        return self.lists

    def build_topk_lists(self, q, budget, keep_sink=True, keep_current=True, stream=None, local_r=0):
        """Lists by content-adaptive top-k from the current chunk's queries q [B, L, H, D] bf16."""
        if not self.dry:
            _check_chunk(q, "q", self.B, self.L, self.H, self.D)
        rule = L.uf_topk_rule(int(budget), int(keep_sink), int(keep_current), int(local_r))
        L.uf_build_topk_lists(self.handle, q, rule, self.lists, None, stream)
        return self.lists

    def kmean_view(self):
        """Pooled keys [max_chunks, B, H, NT, D] float32 (the pool's tail section)."""
        nt = -(-self.L // self.T)
        pages = self.desc.max_chunks * self.B * self.H * nt
        off = pages * 4 * self.T * self.D
        return self.pool[off:off + pages * self.D * 4].view(torch.float32).view(
            self.desc.max_chunks, self.B, self.H, nt, self.D)

    def lists_views(self, lists=None):
        """(counts [B,H,NT], idx [B,H,NT,nk_cap], mask [B,H,NT,words]) views of a list buffer."""
        buf = self.lists if lists is None else lists
        lay = self.layout
        nt = -(-self.L // self.T)
        shp = (self.B, self.H, nt)
        counts = buf[lay.counts_offset:lay.counts_offset + 4 * lay.rows].view(torch.int32).view(shp)
        idx = buf[lay.idx_offset:lay.idx_offset + 4 * lay.rows * lay.nk_cap].view(torch.int32).view(*shp, lay.nk_cap)
        mask = buf[lay.mask_offset:lay.mask_offset + 4 * lay.rows * lay.mask_words].view(torch.int32).view(
            *shp, lay.mask_words)
        return counts, idx, mask

    # -- attention ----------------------------------------------------------
    def attention(self, q, scale=None, out=None, lse=True, lists=None, stream=None, split=None, work=None):
        """O [B,L,H,D] bf16 (and LSE [B,H,L] fp32 when ``lse``) for the current chunk.

        ``split`` > 0 selects split-KV attention with that many list slices per
        row; ``split="tail"`` splits only the rows of the last, partly filled
        round of one workgroup per compute unit as uf_attn_tail_plan chooses,
        and ``split=(split_from, n_split)`` rows split_from.. into n_split
        slices; ``work`` is the scratch buffer (allocated here when None)."""
        _check_chunk(q, "q", self.B, self.L, self.H, self.D)
        if scale is None:
            scale = 1.0 / math.sqrt(self.D)
        if out is None:
            out = torch.empty_like(q)
        else:
            _check_chunk(out, "out", self.B, self.L, self.H, self.D)
        lse_t = None
        if lse is True:
            lse_t = torch.empty((self.B, self.H, self.L), dtype=torch.float32, device=q.device)
        elif lse is not False and lse is not None:
            lse_t = lse
            if lse_t.dtype != torch.float32 or tuple(lse_t.shape) != (self.B, self.H, self.L) or not lse_t.is_contiguous():
                raise ValueError("lse must be a contiguous float32 [B, H, L] tensor")
        buf = self.lists if lists is None else lists
        if buf.numel() < self.layout.total_bytes:
            raise ValueError("list buffer too small")
        if split == "tail" or isinstance(split, tuple):
            if split == "tail":
                n_cu = torch.cuda.get_device_properties(q.device).multi_processor_count
                split_from, n_split = L.uf_attn_tail_plan(self.handle, n_cu)
            else:
                split_from, n_split = (int(x) for x in split)
            need = L.uf_attn_split_rows_work_bytes(self.handle, split_from, n_split)
            if work is None and need > 0:
                work = torch.empty(need, dtype=torch.uint8, device=q.device)
            L.uf_sparse_causal_attn_fwd_split_rows(self.handle, q, buf, scale, out, lse_t, split_from, n_split, work,
                                                   None, stream)
        elif split:
            need = L.uf_attn_split_work_bytes(self.handle, int(split))
            if work is None:
                work = torch.empty(need, dtype=torch.uint8, device=q.device)
            L.uf_sparse_causal_attn_fwd_split(self.handle, q, buf, scale, out, lse_t, int(split), work, None, stream)
        else:
            L.uf_sparse_causal_attn_fwd(self.handle, q, buf, scale, out, lse_t, stream)
        return (out, lse_t) if lse_t is not None else out

    def attention_bwd(self, q, o, lse, do, scale=None, lists=None, stream=None, work=None):
        """(dQ [B,L,H,D], dK, dV [n_live,B,L,H,D]) fp32 of the attention of the
        current chunk, from the forward's O and LSE on the same lists."""
        for t, name in ((q, "q"), (o, "o"), (do, "do")):
            _check_chunk(t, name, self.B, self.L, self.H, self.D)
        if lse.dtype != torch.float32 or tuple(lse.shape) != (self.B, self.H, self.L) or not lse.is_contiguous():
            raise ValueError("lse must be a contiguous float32 [B, H, L] tensor")
        if scale is None:
            scale = 1.0 / math.sqrt(self.D)
        buf = self.lists if lists is None else lists
        if buf.numel() < self.layout.total_bytes:
            raise ValueError("list buffer too small")
        n_live = self.info().n_live
        dq = torch.empty((self.B, self.L, self.H, self.D), dtype=torch.float32, device=q.device)
        dk = torch.empty((n_live, self.B, self.L, self.H, self.D), dtype=torch.float32, device=q.device)
        dv = torch.empty_like(dk)
        if work is None:
            work = torch.empty(L.uf_attn_bwd_work_bytes(self.handle), dtype=torch.uint8, device=q.device)
        L.uf_sparse_causal_attn_bwd(self.handle, q, o, do, lse, buf, scale, dq, dk, dv, work, None, stream)
        return dq, dk, dv
