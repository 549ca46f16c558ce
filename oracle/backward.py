"""Oracle of the block-sparse chunk-causal attention backward (test infrastructure only).

The student of Phase I is trained through sparse causal attention (Sec. 2.3.1:
the same Eq. 4 mask in the generator that DMD updates), so the training side
needs the gradients of the forward defined in ``attention``: for one head and
query row r with kept key set C(r),

    p_rc  = exp(s_rc - lse_r),  s_rc = scale * <q_r, k_c>     (c in C(r))
    o_r   = sum_c p_rc v_c

and an upstream gradient do_r, the chain rule gives

    dv_c  = sum_{r: c in C(r)} p_rc do_r
    dp_rc = <do_r, v_c>
    delta_r = sum_c p_rc dp_rc = <do_r, o_r>
    ds_rc = p_rc (dp_rc - delta_r)
    dq_r  = scale * sum_c ds_rc k_c
    dk_c  = scale * sum_{r: c in C(r)} ds_rc q_r

Keys outside every kept set get zero gradients; padding never exists here
(chunks hold exactly their tokens).  Evaluated in float64 as masked dense
products over the window's keys in logical order.
"""

import numpy as np

from .attention import dense_keys, _kept_columns
from .keep import tile_geometry


def sparse_causal_attention_bwd(ring, q, do, bits, T: int, scale: float, heads=None):
    """Gradients of the forward oracle.

    q, do: [B, L, H, D] (current chunk queries and upstream gradient of O);
    bits: [B, H, NQ, NK] keep set.  Returns (dq [B, L, H, D],
    dk, dv [n_live, B, L, H, D] in logical chunk order), float64.
    """
    chunks = ring.logical_chunks()
    B, L, H, D = q.shape
    n_live = len(chunks)
    nt, _ = tile_geometry(L, T)
    sk = L * n_live
    dq = np.zeros((B, L, H, D))
    dk = np.zeros((n_live, B, L, H, D))
    dv = np.zeros((n_live, B, L, H, D))
    for b in range(B):
        for h in (range(H) if heads is None else heads):
            K, V = dense_keys(ring, b, h)
            dK = np.zeros((sk, D))
            dV = np.zeros((sk, D))
            for i in range(nt):
                r0, r1 = i * T, min((i + 1) * T, L)
                cols = _kept_columns(np.nonzero(bits[b, h, i])[0], L, T, nt, sk)
                if not cols.any():
                    continue
                Q = q[b, r0:r1, h].astype(np.float64)
                dO = do[b, r0:r1, h].astype(np.float64)
                Kc, Vc = K[cols], V[cols]
                S = (Q @ Kc.T) * scale
                P = np.exp(S - S.max(axis=1, keepdims=True))
                P /= P.sum(axis=1, keepdims=True)
                O = P @ Vc
                dP = dO @ Vc.T
                delta = (dO * O).sum(axis=1, keepdims=True)
                dS = P * (dP - delta)
                dq[b, r0:r1, h] = scale * (dS @ Kc)
                dK[cols] += scale * (dS.T @ Q)
                dV[cols] += P.T @ dO
            dk[:, b, :, h] = dK.reshape(n_live, L, D)
            dv[:, b, :, h] = dV.reshape(n_live, L, D)
    return dq, dk, dv


def sparse_causal_attention_bwd_scales(ring, q, do, bits, T: int, scale: float, heads=None):
    """Scale of the summands of every gradient element (float64), for error bars.

    Each gradient element is a sum over keys (dq) or query rows (dk, dv) of
    products of the definition's factors.  Bounding each factor by its
    magnitude, with ds_rc = p_rc (dp_rc - delta_r) bounded by
    m_rc = p_rc (|dp_rc - delta_r| + sum_d |do_rd o_rd|) -- the second term is
    the size of delta's own terms, so that a relative error in those terms is
    covered where dp_rc - delta_r cancels (a near one-hot row) --, the scale of
    an element is the root sum of squares of its summands' bounds:

        sdq_rd = scale * sqrt(sum_c m_rc^2 k_cd^2)
        sdk_cd = scale * sqrt(sum_r m_rc^2 q_rd^2)
        sdv_cd =         sqrt(sum_r p_rc^2 do_rd^2)

    Independent relative errors of size u in the factors change an element by
    about u times its scale.  Same shapes and head selection as
    ``sparse_causal_attention_bwd``.
    """
    chunks = ring.logical_chunks()
    B, L, H, D = q.shape
    n_live = len(chunks)
    nt, _ = tile_geometry(L, T)
    sk = L * n_live
    sq = np.zeros((B, L, H, D))
    sk2 = np.zeros((n_live, B, L, H, D))
    sv2 = np.zeros((n_live, B, L, H, D))
    for b in range(B):
        for h in (range(H) if heads is None else heads):
            K, V = dense_keys(ring, b, h)
            aK = np.zeros((sk, D))
            aV = np.zeros((sk, D))
            for i in range(nt):
                r0, r1 = i * T, min((i + 1) * T, L)
                cols = _kept_columns(np.nonzero(bits[b, h, i])[0], L, T, nt, sk)
                if not cols.any():
                    continue
                Q = q[b, r0:r1, h].astype(np.float64)
                dO = do[b, r0:r1, h].astype(np.float64)
                Kc, Vc = K[cols], V[cols]
                S = (Q @ Kc.T) * scale
                P = np.exp(S - S.max(axis=1, keepdims=True))
                P /= P.sum(axis=1, keepdims=True)
                O = P @ Vc
                dP = dO @ Vc.T
                delta = (dO * O).sum(axis=1, keepdims=True)
                M2 = (P * (np.abs(dP - delta) + np.abs(dO * O).sum(axis=1, keepdims=True))) ** 2
                sq[b, r0:r1, h] = scale * np.sqrt(M2 @ (Kc * Kc))
                aK[cols] += scale * scale * (M2.T @ (Q * Q))
                aV[cols] += (P * P).T @ (dO * dO)
            sk2[:, b, :, h] = aK.reshape(n_live, L, D)
            sv2[:, b, :, h] = aV.reshape(n_live, L, D)
    return sq, np.sqrt(sk2), np.sqrt(sv2)


def sparse_causal_attention_bwd_rows(ring, q, do, bits, T: int, scale: float, samples):
    """dq of the same definition at sampled (b, h, r) query rows only: each row
    needs just its own kept keys (its softmax, o_r and delta_r).  The rows of
    one head are evaluated together, each over its own keep set.  Returns
    dq [n, D] float64."""
    q = np.asarray(q, np.float64)
    do = np.asarray(do, np.float64)
    B, L, H, D = q.shape
    nt, _ = tile_geometry(L, T)
    sk = ring.n_live * L
    samples = list(samples)
    out = np.zeros((len(samples), D))
    by_head = {}
    for n, (b, h, r) in enumerate(samples):
        by_head.setdefault((b, h), []).append(n)
    for (b, h), ns in by_head.items():
        K, V = dense_keys(ring, b, h)
        rows = [samples[n][2] for n in ns]
        M = np.stack([_kept_columns(np.nonzero(bits[b, h, r // T])[0], L, T, nt, sk) for r in rows])
        Q, dO = q[b, rows, h], do[b, rows, h]
        S = (Q @ K.T) * scale
        m = np.max(S, axis=1, where=M, initial=-np.inf)
        P = np.zeros_like(S)
        np.exp(S - m[:, None], out=P, where=M)
        l = P.sum(axis=1, keepdims=True)
        P /= np.where(l > 0, l, 1.0)
        O = P @ V
        dP = dO @ V.T
        delta = (dO * O).sum(axis=1, keepdims=True)
        dS = P * (dP - delta)
        out[ns] = scale * (dS @ K)
    return out
