"""MI355X (gfx950) block-sparse chunk-causal attention over a streaming KV window.

The path of Ultra Flash's single-step SR DiT attention (arXiv 2606.09150,
Sec. 2.3.1 (block-sparse causal attention), Eq. 4; Sec. 2.3.2 dynamic
cache management (iii)), behind the C ABI of ``include/uf.h`` (``libuf.so``):

* ``uf_kv_append`` / ``uf_kv_evict``  -- paged bf16 KV window with a pinned
  first chunk and oldest-first eviction;
* ``uf_build_tile_lists``             -- per (b, h, query tile) key-tile keep lists;
* ``uf_sparse_causal_attn_fwd``       -- the attention kernel (bf16 MFMA).

``_lib`` binds the entry points under the same names; ``KVWindow`` adds
shape checks and torch-allocated buffers.
"""

from . import _lib
from ._lib import (
    UfError,
    load,
    make_desc,
    uf_build_tile_lists,
    uf_build_topk_lists,
    uf_keep_rule,
    uf_topk_budget,
    uf_topk_rule,
    uf_kv_append,
    uf_kv_create,
    uf_kv_desc,
    uf_kv_destroy,
    uf_kv_evict,
    uf_block_geom,
    uf_block_geom_tokens,
    uf_block_permute,
    uf_kv_set_block_geom,
    uf_kv_replace_newest,
    uf_kv_get_info,
    uf_kv_logical,
    uf_kv_pool_bytes,
    uf_last_error,
    uf_attn_split_work_bytes,
    uf_sparse_causal_attn_fwd,
    uf_sparse_causal_attn_fwd_split,
    uf_attn_bwd_work_bytes,
    uf_attn_split_rows_work_bytes,
    uf_attn_tail_plan,
    uf_sparse_causal_attn_fwd_split_rows,
    uf_sparse_causal_attn_bwd,
    uf_sparse_causal_attn_bwd_noalloc,
    uf_status_string,
    uf_tile_lists_bytes,
    uf_tile_lists_layout,
)
from .window import KVWindow

__all__ = [
    "UfError", "load", "make_desc", "uf_build_tile_lists", "uf_build_topk_lists", "uf_keep_rule",
    "uf_topk_budget", "uf_topk_rule", "uf_kv_append",
    "uf_kv_create", "uf_kv_desc", "uf_kv_destroy", "uf_kv_evict", "uf_block_geom", "uf_block_geom_tokens", "uf_block_permute", "uf_kv_set_block_geom", "uf_kv_replace_newest", "uf_kv_get_info", "uf_kv_logical",
    "uf_kv_pool_bytes", "uf_last_error", "uf_sparse_causal_attn_fwd", "uf_sparse_causal_attn_fwd_split", "uf_attn_split_work_bytes",
    "uf_attn_bwd_work_bytes", "uf_attn_split_rows_work_bytes", "uf_attn_tail_plan",
    "uf_sparse_causal_attn_fwd_split_rows", "uf_sparse_causal_attn_bwd", "uf_sparse_causal_attn_bwd_noalloc", "uf_status_string",
    "uf_tile_lists_bytes", "uf_tile_lists_layout", "KVWindow",
]
