"""Seeded synthetic inputs and workload shapes.

This module holds no arithmetic of the attention method: it only draws seeded
i.i.d. N(0, 1) values, rounds them to bf16 (round to nearest even, torch's
conversion) and describes the workload shapes.  Both the HIP path's tests and
bench and the CPU oracle's callers take their inputs from here; neither side
imports the other.

Workloads (B = 1 and D = 128 throughout; a chunk is 3 latent frames of one
token grid, so the chunk length is 3 * grid_h * grid_w):

* ``tiny``      8x8 grid, 192 tokens per chunk, 64-token tiles, one earlier
                chunk plus the current one, every tile kept.
* ``480p``      30x52 grid (1560 tokens per frame; the paper's reference
                length S_ref = 1560 of Eq. 10 is this grid), 4680-token chunks,
                three earlier chunks plus the current one, every tile kept.
* ``1k``        68x120 grid, 24480-token chunks, a pinned first chunk plus
                three earlier chunks plus the current one, earlier-chunk tiles
                kept with probability 0.25.
* ``2k``        90x160 grid, 43200-token chunks, pinned first chunk plus two
                earlier chunks plus the current one, p = 0.15.
* ``1k_stream`` the 1k grid with 40 heads, twelve successive chunks through a
                window of at most five chunks (pinned first chunk plus the
                four most recent, the current one included), p = 0.25.

The paper's model has 12 heads of dimension 128 (App. C); 40 heads is a wide
synthetic stress shape.
"""

from dataclasses import dataclass

import numpy as np
import torch

BASE_SEED = 0x5EED0000


@dataclass(frozen=True)
class Workload:
    name: str
    index: int
    heads: int
    grid_h: int
    grid_w: int
    frames: int
    tile: int
    prior_chunks: int      # earlier chunks in the window besides the pinned one
    pin_sink: bool
    p_prior: float
    max_chunks: int
    stream_chunks: int = 0  # >0: chunks pushed through the window one by one
    batch: int = 1
    head_dim: int = 128

    @property
    def chunk_tokens(self) -> int:
        return self.frames * self.grid_h * self.grid_w

    @property
    def seed(self) -> int:
        return BASE_SEED + self.index

    @property
    def window_chunks(self) -> int:
        """Chunks in the window when the current one is attended (steady state)."""
        return (1 if self.pin_sink else 0) + self.prior_chunks + 1


WORKLOADS = {
    "tiny": Workload("tiny", 0, heads=2, grid_h=8, grid_w=8, frames=3, tile=64,
                     prior_chunks=1, pin_sink=False, p_prior=1.0, max_chunks=2),
    "480p": Workload("480p", 1, heads=12, grid_h=30, grid_w=52, frames=3, tile=128,
                     prior_chunks=3, pin_sink=False, p_prior=1.0, max_chunks=4),
    "1k": Workload("1k", 2, heads=12, grid_h=68, grid_w=120, frames=3, tile=128,
                   prior_chunks=3, pin_sink=True, p_prior=0.25, max_chunks=5),
    "2k": Workload("2k", 3, heads=12, grid_h=90, grid_w=160, frames=3, tile=128,
                   prior_chunks=2, pin_sink=True, p_prior=0.15, max_chunks=4),
    "1k_stream": Workload("1k_stream", 4, heads=40, grid_h=68, grid_w=120, frames=3, tile=128,
                          prior_chunks=3, pin_sink=True, p_prior=0.25, max_chunks=5,
                          stream_chunks=12),
}

TENSOR_ID = {"q": 0, "k": 1, "v": 2, "do": 3}


def derive_seed(*key: int) -> int:
    """A 63-bit generator seed from a tuple of non-negative integers."""
    state = np.random.SeedSequence([int(k) for k in key]).generate_state(2, np.uint32)
    return int((int(state[0]) << 32 | int(state[1])) & 0x7FFFFFFFFFFFFFFF)


def normal_bf16(shape, *key: int, device="cpu") -> torch.Tensor:
    """i.i.d. N(0,1) drawn in float32 by torch's generator for ``device``, rounded to bf16.

    The values differ between the CPU and the GPU generators; a caller that
    needs the same values on both sides draws once and copies.
    """
    g = torch.Generator(device=device)
    g.manual_seed(derive_seed(*key))
    x = torch.randn(tuple(shape), generator=g, device=device, dtype=torch.float32)
    return x.to(torch.bfloat16)


def chunk_tensor(wl: Workload, chunk: int, name: str, device="cpu", seed=None) -> torch.Tensor:
    """Q, K or V [B, L, H, D] bf16 of chunk number ``chunk`` of workload ``wl``."""
    shape = (wl.batch, wl.chunk_tokens, wl.heads, wl.head_dim)
    return normal_bf16(shape, wl.seed if seed is None else seed, chunk, TENSOR_ID[name], device=device)


def custom_tensor(shape, seed: int, chunk: int, name: str, device="cpu") -> torch.Tensor:
    """Same draw for an arbitrary [B, L, H, D] shape (small parity cases)."""
    return normal_bf16(shape, seed, chunk, TENSOR_ID[name], device=device)
