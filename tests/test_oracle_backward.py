"""Pins of the backward oracle: central finite differences of the forward
oracle, autograd of an independently written masked softmax attention in
float64, and closed-form special cases."""

import numpy as np
import torch

import oracle


def _ring(B, L, H, D, n, pin, seed):
    rng = np.random.default_rng(seed)
    ring = oracle.RingModel(n, pin)
    for _ in range(n):
        ring.append(rng.standard_normal((B, L, H, D)), rng.standard_normal((B, L, H, D)))
    q = rng.standard_normal((B, L, H, D))
    do = rng.standard_normal((B, L, H, D))
    return ring, q, do, rng


def _bits(rng, B, H, nt, nk):
    bits = rng.random((B, H, nt, nk)) < 0.6
    bits[..., -1] = True          # every row keeps at least one tile
    return bits


def test_backward_matches_central_differences():
    B, L, H, D, T = 1, 5, 1, 4, 2
    ring, q, do, rng = _ring(B, L, H, D, 3, True, 1)
    nt = 3
    bits = _bits(rng, B, H, nt, 3 * nt)
    scale = 0.7
    dq, dk, dv = oracle.sparse_causal_attention_bwd(ring, q, do, bits, T, scale)

    def f():
        O, _ = oracle.sparse_causal_attention(ring, q, bits, T, scale)
        return float((O * do).sum())

    eps = 1e-6
    for arr, grad in [(q, dq)] + [(c.k, dk[p]) for p, c in enumerate(ring.logical_chunks())] + \
                     [(c.v, dv[p]) for p, c in enumerate(ring.logical_chunks())]:
        num = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            keep = arr[idx]
            arr[idx] = keep + eps
            fp = f()
            arr[idx] = keep - eps
            fm = f()
            arr[idx] = keep
            num[idx] = (fp - fm) / (2 * eps)
        assert np.allclose(grad, num, atol=1e-7, rtol=1e-6)


def test_backward_matches_autograd_of_masked_attention():
    B, L, H, D, T = 2, 7, 2, 8, 3
    ring, q, do, rng = _ring(B, L, H, D, 4, False, 2)
    nt = 3
    bits = _bits(rng, B, H, nt, 4 * nt)
    scale = 0.35
    dq, dk, dv = oracle.sparse_causal_attention_bwd(ring, q, do, bits, T, scale)
    chunks = ring.logical_chunks()
    for b in range(B):
        for h in range(H):
            Q = torch.tensor(q[b, :, h], requires_grad=True)
            Ks = [torch.tensor(c.k[b, :, h], requires_grad=True) for c in chunks]
            Vs = [torch.tensor(c.v[b, :, h], requires_grad=True) for c in chunks]
            K, V = torch.cat(Ks), torch.cat(Vs)
            # token-level mask from the tile bits: query token r in tile r // T,
            # key token (pos, t) in logical tile pos * nt + t // T
            key_tile = torch.tensor([p * nt + t // T for p in range(len(chunks)) for t in range(L)])
            qt = torch.arange(L) // T
            mask = torch.tensor(bits[b, h])[qt][:, key_tile]
            S = (Q @ K.T) * scale
            S = S.masked_fill(~mask, float("-inf"))
            O = torch.softmax(S, dim=1) @ V
            (O * torch.tensor(do[b, :, h])).sum().backward()
            assert np.allclose(Q.grad.numpy(), dq[b, :, h], atol=1e-10)
            for p in range(len(chunks)):
                assert np.allclose(Ks[p].grad.numpy(), dk[p, b, :, h], atol=1e-10)
                assert np.allclose(Vs[p].grad.numpy(), dv[p, b, :, h], atol=1e-10)


def test_backward_closed_forms():
    B, L, H, D, T = 1, 6, 1, 4, 2
    ring, q, do, rng = _ring(B, L, H, D, 2, False, 3)
    bits = _bits(rng, B, H, 3, 6)
    # equal values: dp = delta for every key, so ds = 0 and dq = dk = 0
    v0 = ring.live[0].v[:, :1].copy()
    for c in ring.live:
        c.v = np.broadcast_to(v0, c.v.shape).copy()
    dq, dk, dv = oracle.sparse_causal_attention_bwd(ring, q, do, bits, T, 0.5)
    assert np.allclose(dq, 0, atol=1e-12) and np.allclose(dk, 0, atol=1e-12)
    # shifting every key by one vector leaves dq unchanged (rows of ds sum to 0)
    ring2, q2, do2, rng2 = _ring(B, L, H, D, 2, False, 4)
    bits2 = _bits(rng2, B, H, 3, 6)
    dq1, _, _ = oracle.sparse_causal_attention_bwd(ring2, q2, do2, bits2, T, 0.5)
    shift = rng2.standard_normal(D)
    for c in ring2.live:
        c.k = c.k + shift
    dq2, _, _ = oracle.sparse_causal_attention_bwd(ring2, q2, do2, bits2, T, 0.5)
    assert not np.allclose(dq1, 0) and np.allclose(dq1, dq2, atol=1e-10)
    # keys no row keeps get zero gradients
    bits3 = np.zeros((1, 1, 3, 6), bool)
    bits3[..., 4] = True
    _, dk3, dv3 = oracle.sparse_causal_attention_bwd(ring2, q2, do2, bits3, T, 0.5)
    assert np.all(dk3[0] == 0) and np.all(dv3[0] == 0) and np.any(dv3[1] != 0)


def test_backward_identities():
    """Properties of the exact gradients at any size: rows of dS sum to zero,
    so the dK of a head sum to zero over the window's keys; sum_c <dK_c, k_c>
    = sum_r <dQ_r, q_r> (both equal sum dS * S); sum_c <dV_c, v_c> =
    sum_r <dO_r, O_r>."""
    B, L, H, D, T = 2, 9, 2, 6, 4
    ring, q, do, rng = _ring(B, L, H, D, 3, True, 5)
    nt = 3
    bits = _bits(rng, B, H, nt, 3 * nt)
    scale = 0.4
    dq, dk, dv = oracle.sparse_causal_attention_bwd(ring, q, do, bits, T, scale)
    O, _ = oracle.sparse_causal_attention(ring, q, bits, T, scale)
    ks = np.stack([c.k for c in ring.logical_chunks()])
    vs = np.stack([c.v for c in ring.logical_chunks()])
    for b in range(B):
        for h in range(H):
            assert np.allclose(dk[:, b, :, h].sum(axis=(0, 1)), 0, atol=1e-12)
            lhs = (dk[:, b, :, h] * ks[:, b, :, h]).sum()
            assert np.isclose(lhs, (dq[b, :, h] * q[b, :, h]).sum(), atol=1e-12)
            assert np.isclose((dv[:, b, :, h] * vs[:, b, :, h]).sum(), (do[b, :, h] * O[b, :, h]).sum(), atol=1e-12)


def test_sampled_rows_match_full_backward():
    B, L, H, D, T = 2, 10, 2, 5, 4
    ring, q, do, rng = _ring(B, L, H, D, 3, False, 6)
    nt = 3
    bits = _bits(rng, B, H, nt, 3 * nt)
    bits[1, 0, 2] = False                    # a row with no kept tile: zero gradient
    dq, _, _ = oracle.sparse_causal_attention_bwd(ring, q, do, bits, T, 0.3)
    samples = [(0, 0, 0), (0, 1, 9), (1, 0, 3), (1, 0, 8), (1, 1, 5)]
    got = oracle.sparse_causal_attention_bwd_rows(ring, q, do, bits, T, 0.3, samples)
    want = np.stack([dq[b, r, h] for b, h, r in samples])
    assert np.allclose(got, want, atol=1e-12)
    assert np.all(got[3] == 0)


def _brute_scales(ring, q, do, bits, T, scale):
    """Element-by-element loops over the definition of the summand scales."""
    chunks = ring.logical_chunks()
    B, L, H, D = q.shape
    nt = -(-L // T)
    keys = [(p, t) for p in range(len(chunks)) for t in range(L)]
    sq = np.zeros_like(q)
    sk = np.zeros((len(chunks), B, L, H, D))
    sv = np.zeros_like(sk)
    for b in range(B):
        for h in range(H):
            for r in range(L):
                kept = [(p, t) for (p, t) in keys if bits[b, h, r // T, p * nt + t // T]]
                s = [scale * sum(q[b, r, h, d] * chunks[p].k[b, t, h, d] for d in range(D)) for p, t in kept]
                mx = max(s)
                e = [np.exp(x - mx) for x in s]
                pr = [x / sum(e) for x in e]
                o = [sum(pr[n] * chunks[p].v[b, t, h, d] for n, (p, t) in enumerate(kept)) for d in range(D)]
                dp = [sum(do[b, r, h, d] * chunks[p].v[b, t, h, d] for d in range(D)) for p, t in kept]
                delta = sum(do[b, r, h, d] * o[d] for d in range(D))
                dsum = sum(abs(do[b, r, h, d] * o[d]) for d in range(D))
                for n, (p, t) in enumerate(kept):
                    m = pr[n] * (abs(dp[n] - delta) + dsum)
                    for d in range(D):
                        sq[b, r, h, d] += (scale * m * chunks[p].k[b, t, h, d]) ** 2
                        sk[p, b, t, h, d] += (scale * m * q[b, r, h, d]) ** 2
                        sv[p, b, t, h, d] += (pr[n] * do[b, r, h, d]) ** 2
    return np.sqrt(sq), np.sqrt(sk), np.sqrt(sv)


def test_summand_scales_brute_force():
    B, L, H, D, T = 1, 5, 2, 3, 2
    ring, q, do, rng = _ring(B, L, H, D, 3, True, 11)
    bits = _bits(rng, B, H, 3, 9)
    got = oracle.sparse_causal_attention_bwd_scales(ring, q, do, bits, T, 0.6)
    want = _brute_scales(ring, q, do, bits, T, 0.6)
    for g, w in zip(got, want):
        assert np.allclose(g, w, rtol=1e-12, atol=1e-14)


def test_summand_scales_single_key_closed_form():
    """One kept key: p = 1 and o = v, so dp - delta = 0 and the exact dq and dk
    vanish, while the scales keep the size of delta's terms."""
    rng = np.random.default_rng(12)
    ring = oracle.RingModel(1, False)
    k, v = rng.standard_normal((1, 1, 1, 4)), rng.standard_normal((1, 1, 1, 4))
    ring.append(k, v)
    q, do = rng.standard_normal((1, 1, 1, 4)), rng.standard_normal((1, 1, 1, 4))
    bits = np.ones((1, 1, 1, 1), bool)
    dq, dk, dv = oracle.sparse_causal_attention_bwd(ring, q, do, bits, 1, 0.5)
    sq, sk, sv = oracle.sparse_causal_attention_bwd_scales(ring, q, do, bits, 1, 0.5)
    assert np.allclose(dq, 0, atol=1e-15) and np.allclose(dk, 0, atol=1e-15)
    assert np.allclose(dv[0], do)
    dsum = np.abs(do * v).sum()
    assert np.allclose(sq[0, 0, 0], 0.5 * dsum * np.abs(k[0, 0, 0]))
    assert np.allclose(sk[0, 0, 0, 0], 0.5 * dsum * np.abs(q[0, 0, 0]))
    assert np.allclose(sv[0, 0, 0, 0], np.abs(do[0, 0, 0]))


def test_summand_scales_bound_perturbed_factors():
    """Relative perturbations of size u in p, in dp - delta's factors and in
    delta's terms move every gradient element by a few u times its scale."""
    B, L, H, D, T = 1, 40, 1, 16, 8
    ring, q, do, rng = _ring(B, L, H, D, 3, True, 13)
    for c in ring.live:          # peaked rows
        c.k *= 3.0
    q = q * 3.0
    bits = _bits(rng, B, H, 5, 15)
    scale, u = 0.5, 1e-3
    sq, sk, sv = oracle.sparse_causal_attention_bwd_scales(ring, q, do, bits, T, scale)
    K = np.concatenate([c.k[0, :, 0] for c in ring.logical_chunks()])
    V = np.concatenate([c.v[0, :, 0] for c in ring.logical_chunks()])
    cols = np.zeros((5, 15 * T), bool)
    for i in range(5):
        for j in np.nonzero(bits[0, 0, i])[0]:
            p, t = divmod(j, 5)
            cols[i, p * L + t * T:p * L + t * T + T] = True
    exact = np.zeros((L, D)), np.zeros((3 * L, D)), np.zeros((3 * L, D))
    pert = np.zeros((L, D)), np.zeros((3 * L, D)), np.zeros((3 * L, D))
    for i in range(5):
        rows = slice(i * T, (i + 1) * T)
        c = cols[i]
        Qi, dOi = q[0, rows, 0], do[0, rows, 0]
        S = Qi @ K[c].T * scale
        P = np.exp(S - S.max(1, keepdims=True))
        P /= P.sum(1, keepdims=True)
        O = P @ V[c]
        for out, noisy in ((exact, False), (pert, True)):
            e = (lambda shape: 1 + u * rng.uniform(-1, 1, shape)) if noisy else (lambda shape: 1.0)
            Pn = P * e(P.shape)
            delta = (dOi * O * e(O.shape)).sum(1, keepdims=True)
            dS = Pn * (dOi @ V[c].T - delta) * e(P.shape)
            out[0][rows] += scale * dS @ K[c]
            out[1][c] += scale * dS.T @ Qi
            out[2][c] += Pn.T @ dOi
    for g, x, s_ in ((pert[0], exact[0], sq[0, :, 0]), (pert[1], exact[1], np.concatenate(sk[:, 0, :, 0])),
                     (pert[2], exact[2], np.concatenate(sv[:, 0, :, 0]))):
        assert np.all(np.abs(g - x) <= 6 * u * s_ + 1e-15)
