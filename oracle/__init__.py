"""CPU oracle for chunk-wise block-sparse causal attention over a streaming KV cache.

TEST INFRASTRUCTURE ONLY. Nothing in the product path may import, call or link
anything in this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.

It is a plain, slow, obviously correct restatement of what the method computes
(Ultra Flash, arXiv 2606.09150):

* ``ring``      -- the KV cache window of earlier chunks plus the current chunk
                   (Sec. 2.3.2, dynamic cache management (iii): the cache
                   length of the SR model adapted to a compact window; App. C
                   gives its size in chunks), with a pinned first ("sink")
                   chunk and oldest-first eviction.
* ``keep``      -- the per-(head, query tile) key-tile keep set: the temporal
                   causal mask of Sec. 2.3.1(a) intersected with a seeded
                   Bernoulli content stand-in for the top-k rule of Eq. 4.
                   The Bernoulli rule and its SplitMix64 counter hash are not in
                   the paper: their parity against the paper is unpinned; they
                   are pinned to the published SplitMix64 outputs and to
                   binomial statistics.
* ``topk``      -- the content-adaptive top-k keep set of Eq. 4: mean-pooled
                   query and key tiles, block scores, top-k per (head, query
                   tile) with forced pinned/current chunks; fixed float32
                   arithmetic (parity against the paper unpinned).
* ``blocks``    -- the 3-D (b_t, b_h, b_w) block tiling of a chunk's token
                   grid, the block order of tokens, the r x r local window
                   mask M_local, and attention evaluated in raster order.
* ``mask``      -- the composed block mask of Eq. 4: the content rule (top-k
                   or the Bernoulli stand-in, forced chunks included), then
                   M_local, over raster tiles or 3-D blocks.
* ``backward``  -- gradients dq, dk, dv of the masked attention (the training
                   side of the same forward), float64.
* ``attention`` -- softmax attention of the current chunk's queries over the
                   union of kept key tiles (Eq. 4 mask semantics), computed as
                   masked dense attention in float64.

It shares no code with the HIP path (``paper_2606_09150_amd``) and imports
nothing from it.
"""

from .ring import RingModel, RingCapacityError, RingEmptyError
from .keep import (
    KeepRule,
    splitmix64,
    keep_threshold,
    tile_geometry,
    keep_bits,
    lists_from_bits,
)
from .topk import (
    TopkRule,
    topk_budget,
    pooled_means,
    block_scores,
    order_key,
    select_topk,
    topk_scores,
    topk_bits,
)
from .blocks import (
    BlockGeom,
    block_order,
    block_of_token,
    block_means,
    local_mask,
    attention_in_raster,
    attention_in_raster_bwd,
)
from .mask import block_sparse_mask
from .backward import (
    sparse_causal_attention_bwd,
    sparse_causal_attention_bwd_rows,
    sparse_causal_attention_bwd_scales,
)
from .attention import (
    sparse_causal_attention,
    sparse_causal_attention_rows,
    dense_keys,
)

__all__ = [
    "RingModel",
    "RingCapacityError",
    "RingEmptyError",
    "KeepRule",
    "splitmix64",
    "keep_threshold",
    "tile_geometry",
    "keep_bits",
    "lists_from_bits",
    "BlockGeom",
    "block_order",
    "block_of_token",
    "block_means",
    "local_mask",
    "attention_in_raster",
    "attention_in_raster_bwd",
    "block_sparse_mask",
    "TopkRule",
    "topk_budget",
    "pooled_means",
    "block_scores",
    "order_key",
    "select_topk",
    "topk_scores",
    "topk_bits",
    "sparse_causal_attention_bwd",
    "sparse_causal_attention_bwd_rows",
    "sparse_causal_attention_bwd_scales",
    "sparse_causal_attention",
    "sparse_causal_attention_rows",
    "dense_keys",
]
