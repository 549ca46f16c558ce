"""Oracle model of the streaming KV cache window (test infrastructure only).

The paper keeps, per attention layer of the single-step SR DiT, a KV cache of
earlier chunks that the current chunk's queries attend over (App. C gives its
size, a few chunks), and at inference selects a compact cache window
(Sec. 2.3.2, dynamic cache management (iii); Alg. 3, inference part, the step
that picks the SR model's window).  This model realises that window as:

* a list of live chunks in *logical order* = ascending append sequence number;
* an optional pinned first chunk (the "sink", not named by the paper; it is the
  reading chosen for the first-chunk-always-kept configurations), which is
  never evicted and therefore always sits at logical position 0;
* ``evict(n)`` drops the ``n`` oldest non-sink chunks; ``append`` fails when
  the window already holds ``max_chunks`` chunks.

The *current* chunk is the most recently appended live chunk; its queries are
the ones that attend.  Only metadata and the chunk tensors are kept: there are
no slots or pages here, because the result may not depend on physical
placement.
"""

from dataclasses import dataclass

import numpy as np


class RingCapacityError(RuntimeError):
    """append() on a window that already holds max_chunks chunks."""


class RingEmptyError(RuntimeError):
    """evict(n) with fewer than n evictable chunks, or a query on no chunks."""


@dataclass
class Chunk:
    seq: int          # append sequence number, 0-based, never reused
    sink: bool        # pinned first chunk
    k: np.ndarray     # [B, L, H, D] float64 (bf16 values)
    v: np.ndarray     # [B, L, H, D] float64 (bf16 values)


class RingModel:
    def __init__(self, max_chunks: int, pin_sink: bool):
        if max_chunks < 1:
            raise ValueError("max_chunks must be >= 1")
        self.max_chunks = int(max_chunks)
        self.pin_sink = bool(pin_sink)
        self.live: list[Chunk] = []
        self.next_seq = 0

    # -- mutation ---------------------------------------------------------
    def append(self, k, v) -> int:
        if len(self.live) >= self.max_chunks:
            raise RingCapacityError("window full")
        seq = self.next_seq
        sink = self.pin_sink and seq == 0
        self.live.append(Chunk(seq, sink, np.asarray(k, np.float64), np.asarray(v, np.float64)))
        self.next_seq += 1
        return seq

    def evict(self, n: int) -> None:
        if n < 0:
            raise ValueError("n must be >= 0")
        evictable = [c for c in self.live if not c.sink]
        if n > len(evictable):
            raise RingEmptyError("not enough evictable chunks")
        drop = {c.seq for c in sorted(evictable, key=lambda c: c.seq)[:n]}
        self.live = [c for c in self.live if c.seq not in drop]

    # -- queries ----------------------------------------------------------
    @property
    def n_live(self) -> int:
        return len(self.live)

    @property
    def current(self) -> Chunk:
        if not self.live:
            raise RingEmptyError("no live chunk")
        return self.live[-1]

    def logical_chunks(self) -> list:
        """Live chunks in logical order: [sink][oldest prior .. newest prior][current]."""
        return sorted(self.live, key=lambda c: c.seq)
