"""Closed-form masked softmax attention and its forward-mode tangent in fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What is computed (paper, App. B, "FlashAttention-2 JVP kernel with custom
masks", the masked-attention equation, the score-tangent equation and the
tangent-output equation), for every batch b and head h independently:

    S   = s * Q K^T,        S[a,b]  = -inf where the mask forbids (a,b)
    P   = softmax_rows(S)   (m = row max, l = sum exp(S - m), P = exp(S - m)/l)
    LSE = m + ln l          (natural log, in the scaled-score domain)
    O   = P V
    dS  = s * (dQ K^T + Q dK^T),  dS[a,b] = 0 where the mask forbids (a,b)
    mu  = rowsum(P o dS)
    dO  = (P o (dS - mu)) V + P dV

with s = 1/sqrt(D) unless a positive ``scale`` overrides it.  A row with no
allowed key gets O = 0, dO = 0, LSE = -inf.

This is the plain definition: the whole row of scores is materialised, there
is no online recurrence, no tiling of keys, and no range list.  Query rows are
processed in blocks only to bound memory; each row's arithmetic is independent
of the blocking.
"""
import numpy as np

from .masks import MASK_TEACHER_FORCING, allowed_mask


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def _softmax_rows(S, allowed):
    """Masked row softmax. Returns (P, m, l) with P = 0 on forbidden entries."""
    S = np.where(allowed, S, -np.inf)
    m = S.max(axis=1)
    empty = ~np.isfinite(m)
    m_safe = np.where(empty, 0.0, m)
    E = np.where(allowed, np.exp(S - m_safe[:, None]), 0.0)
    l = E.sum(axis=1)
    P = E / np.where(empty, 1.0, l)[:, None]
    return P, m, l, empty


def _one_head(q, k, v, dq, dk, dv, allowed, s, want_tangent):
    S = s * (q @ k.T)
    P, m, l, empty = _softmax_rows(S, allowed)
    O = P @ v
    with np.errstate(divide="ignore"):
        lse = np.where(empty, -np.inf, m + np.log(np.where(empty, 1.0, l)))
    if not want_tangent:
        return O, None, lse
    dS = s * (dq @ k.T + q @ dk.T)
    dS = np.where(allowed, dS, 0.0)
    mu = (P * dS).sum(axis=1, keepdims=True)
    dP = P * (dS - mu)
    dO = dP @ v + P @ dv
    return O, dO, lse


def _run(Q, K, V, dQ, dK, dV, kind, offsets, scale, rows, block, want_tangent):
    Q, K, V = _f64(Q), _f64(K), _f64(V)
    if want_tangent:
        dQ, dK, dV = _f64(dQ), _f64(dK), _f64(dV)
    B, H, L, D = Q.shape
    s = float(scale) if (scale is not None and scale > 0) else 1.0 / np.sqrt(D)
    rows = np.arange(L) if rows is None else np.asarray(rows, dtype=np.int64)
    R = rows.size
    O = np.zeros((B, H, R, D))
    dO = np.zeros((B, H, R, D)) if want_tangent else None
    LSE = np.zeros((B, H, R))
    for r0 in range(0, R, block):
        sel = rows[r0:r0 + block]
        allowed = allowed_mask(kind, offsets, L, sel)
        for b in range(B):
            for h in range(H):
                o, do, lse = _one_head(
                    Q[b, h, sel], K[b, h], V[b, h],
                    dQ[b, h, sel] if want_tangent else None,
                    dK[b, h] if want_tangent else None,
                    dV[b, h] if want_tangent else None,
                    allowed, s, want_tangent)
                O[b, h, r0:r0 + sel.size] = o
                LSE[b, h, r0:r0 + sel.size] = lse
                if want_tangent:
                    dO[b, h, r0:r0 + sel.size] = do
    return O, dO, LSE


def attention_jvp(Q, K, V, dQ, dK, dV, kind, offsets=None, scale=None, rows=None, block=256):
    """(O, dO, LSE) in fp64 for inputs of shape [B, H, L, D].

    ``rows`` optionally restricts the query rows computed (outputs then have
    len(rows) rows); every key is always used.
    """
    O, dO, LSE = _run(Q, K, V, dQ, dK, dV, kind, offsets, scale, rows, block, True)
    return O, dO, LSE


def attention_fwd(Q, K, V, kind, offsets=None, scale=None, rows=None, block=256):
    """(O, LSE) in fp64: the primal part of :func:`attention_jvp`."""
    O, _, LSE = _run(Q, K, V, None, None, None, kind, offsets, scale, rows, block, False)
    return O, LSE


def attention_jvp_zero_clean(Q, K, V, dQn, dKn, dVn, offsets, scale=None, rows=None, block=256):
    """(O, dO, LSE) in fp64 of teacher-forcing attention whose clean half has zero tangent.

    Paper Sec. 3.1.2, the TF-sCM tangent equation: the JVP runs through the packed
    [clean | noisy] forward with input tangent [0^clean, t^noisy].  Q, K, V are
    [B, H, L, D] over the packed sequence; dQn, dKn, dVn are [B, H, L - L/2, D], the
    tangents of the noisy rows.  This is the definition written out: the tangents
    are padded with zeros over the clean rows and :func:`attention_jvp` is taken
    with the teacher-forcing mask.  dO is returned for every row (``rows`` selects
    sequence rows, as in :func:`attention_jvp`); its clean rows come out zero.
    """
    Q = _f64(Q)
    half = Q.shape[2] // 2
    pad = lambda t: np.concatenate([np.zeros(Q.shape[:2] + (half, Q.shape[3])), _f64(t)], axis=2)
    return attention_jvp(Q, K, V, pad(dQn), pad(dKn), pad(dVn), MASK_TEACHER_FORCING, offsets, scale,
                         rows, block)
