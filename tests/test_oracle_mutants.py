"""Planted mistakes in the oracle (on the CPU) must each fail at least one pin.

Each mutant swaps one oracle helper for a copy with a plausible slip (a tail
span that runs into the next chunk, a dropped scale, a flipped sign, a
transposed operand, a dropped LSE term, a sink that is not forced) and runs
the pins of ``test_oracle_pins`` against it.
"""

import numpy as np
import pytest

import oracle
import oracle.attention as att
import oracle.keep as keep
from tests import test_oracle_pins as pins

ATTENTION_PINS = [
    pins.test_brute_force_ragged_tiles,
    pins.test_closed_form_uniform_weights_pick_exact_keys,
    pins.test_all_kept_is_dense_attention,
    pins.test_v_ones_and_row_sums,
]


def _fails_some(tests):
    for t in tests:
        try:
            t()
        except AssertionError:
            return True
    return False


def _spans_no_tail_clip(kept_tiles, L, T, nt, sk):
    cols = np.zeros(sk, dtype=bool)
    for j in kept_tiles:
        pos, t = divmod(int(j), nt)
        cols[pos * L + t * T: pos * L + (t + 1) * T] = True   # slip: no min(., L)
    return cols


def _make_attend(slip):
    def _attend(Q, K, V, cols, scale):
        n = Q.shape[0]
        M = np.broadcast_to(np.asarray(cols, dtype=bool), (n, K.shape[0]))
        S = (Q @ K.T) * (1.0 if slip == "scale" else scale)
        m = np.max(S, axis=1, where=M, initial=-np.inf)
        P = np.zeros_like(S)
        if slip == "sign":
            np.exp(-(S - m[:, None]), out=P, where=M)
        else:
            np.exp(S - m[:, None], out=P, where=M)
        l = P.sum(axis=1)
        has = l > 0
        ls = np.where(has, l, 1.0)
        O = (P @ (K if slip == "operand" else V)) / ls[:, None]
        lse = np.where(has, (0.0 if slip == "lse" else m) + np.log(ls), -np.inf)
        return O, lse, (P / ls[:, None]).sum(axis=1)
    return _attend


@pytest.mark.parametrize("slip", ["scale", "sign", "operand", "lse"])
def test_attention_slips_are_caught(monkeypatch, slip):
    monkeypatch.setattr(att, "_attend_rows", _make_attend(slip))
    assert _fails_some(ATTENTION_PINS)


def test_tail_spill_is_caught(monkeypatch):
    monkeypatch.setattr(att, "_kept_columns", _spans_no_tail_clip)
    assert _fails_some(ATTENTION_PINS)


def test_unforced_sink_is_caught(monkeypatch):
    real = keep.keep_bits

    def slip(ring, T, rule):
        return real(ring, T, oracle.KeepRule(rule.seed, rule.p_prior, keep_sink=False,
                                             keep_current=rule.keep_current))
    monkeypatch.setattr(oracle, "keep_bits", slip)
    assert _fails_some([pins.test_keep_forced_tiles_and_extremes])


def test_splitmix_constant_slip_is_caught(monkeypatch):
    monkeypatch.setattr(keep, "_M2", np.uint64(0x94D049BB133111EA))
    assert _fails_some([pins.test_splitmix64_published_outputs])
