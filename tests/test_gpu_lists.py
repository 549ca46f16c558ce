"""GPU tile lists versus the oracle's keep set: bit for bit."""

import numpy as np
import pytest
import torch

import oracle
import synth
from tests.gpu_common import Case, log, require_gpu

pytestmark = pytest.mark.gpu


def _compare(case, rule):
    bits = case.oracle_bits(rule)
    info = case.win.info()
    want_c, want_i, want_m = oracle.lists_from_bits(bits, info.nk_cap)
    got_c, got_i, got_m = case.gpu_lists(rule)
    assert np.array_equal(got_c, want_c)
    assert np.array_equal(got_i, want_i)
    assert np.array_equal(got_m, want_m)
    return bits


class ZeroCase(Case):
    """Lists depend only on metadata: append zero chunks (no generation cost)."""

    def _draw(self, chunk, name):
        return torch.zeros((self.B, self.L, self.H, 128), dtype=torch.bfloat16, device="cuda")

    def _host(self, t):
        return np.broadcast_to(np.zeros(1), (self.B, self.L, self.H, 1))


@pytest.mark.parametrize("name", ["tiny", "480p", "1k", "2k"])
def test_lists_bit_exact_workloads(name):
    P = require_gpu()
    wl = synth.WORKLOADS[name]
    log(f"lists workload={name}")
    case = ZeroCase(P, 1, wl.chunk_tokens, wl.heads, wl.tile, wl.max_chunks, wl.pin_sink, wl.seed)
    for _ in range(wl.window_chunks):
        case.append()
    bits = _compare(case, case.rule(wl.p_prior))
    nt = -(-wl.chunk_tokens // wl.tile)
    if wl.p_prior < 1:
        prior = bits[..., nt:(wl.window_chunks - 1) * nt]
        sigma = np.sqrt(wl.p_prior * (1 - wl.p_prior) / prior.size)
        assert abs(prior.mean() - wl.p_prior) < 5 * sigma
    else:
        assert bits.all()


def test_lists_stream_steps():
    P = require_gpu()
    wl = synth.WORKLOADS["1k_stream"]
    case = ZeroCase(P, 1, wl.chunk_tokens, wl.heads, wl.tile, wl.max_chunks, wl.pin_sink, wl.seed)
    for step in range(wl.stream_chunks):
        case.append()
        if step in (0, 1, 4, 5, 11):
            log(f"lists stream step={step}")
            _compare(case, case.rule(wl.p_prior))


@pytest.mark.parametrize("T,L,B,H", [(128, 300, 2, 3), (64, 130, 1, 2), (128, 128, 1, 1), (64, 1, 1, 1)])
def test_lists_rules_and_ragged_shapes(T, L, B, H):
    P = require_gpu()
    case = ZeroCase(P, B, L, H, T, 6, True, 17)
    for step in range(9):
        case.append()
        for rule in (case.rule(0.37, seed=0xFFFFFFFFFFFFFFF1), case.rule(0.0), case.rule(1.0),
                     case.rule(0.5, keep_sink=False), case.rule(0.5, keep_current=False),
                     case.rule(0.9, keep_sink=False, keep_current=False)):
            _compare(case, rule)


def test_lists_eviction_history_invariance():
    P = require_gpu()
    a = ZeroCase(P, 1, 500, 2, 128, 5, True, 5)
    b = ZeroCase(P, 1, 500, 2, 128, 5, True, 5)
    for _ in range(8):
        a.append()
    for _ in range(4):
        b.append()
    b.win.evict(3)
    b.ring.evict(3)
    for _ in range(4):
        b.append(evict_when_full=False)
    slots_a = [a.win.logical(p) for p in range(5)]
    slots_b = [b.win.logical(p) for p in range(5)]
    assert [s for _, s in slots_a] == [s for _, s in slots_b]      # same logical content
    assert [s for s, _ in slots_a] != [s for s, _ in slots_b]      # different physical slots
    rule = a.rule(0.3)
    la = a.gpu_lists(rule)
    lb = b.gpu_lists(rule)
    for x, y in zip(la, lb):
        assert np.array_equal(x, y)
