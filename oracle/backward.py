"""Closed-form gradient (vector-Jacobian product) of masked softmax attention in fp64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The map is the masked-attention equation of the paper's App. B ("FlashAttention-2
JVP kernel with custom masks"), O = softmax(s Q K^T + M) V, per batch b and head h.
Training the student through the packed teacher-forcing forward (Sec. 3.1.2, the
TF-sCM objective, whose gradient flows through the TF-masked student pass) needs
the reverse-mode derivative of that map: for a cotangent gO of O,

    P     = softmax_rows(s Q K^T + M)          (P = 0 on forbidden pairs)
    O     = P V
    Delta = rowsum(gO o O)
    gV    = P^T gO
    gP    = gO V^T
    gS    = P o (gP - Delta)                   (0 on forbidden pairs, since P is)
    gQ    = s gS K
    gK    = s gS^T Q

This is that definition written out on whole score rows: no tiling of keys, no
range lists, no online recurrence.  Query rows are processed in blocks only to
bound memory, and a block's score rows leave out the keys none of its rows admits
(their P is exactly zero).  A row with no admissible key has P = 0 and contributes
nothing.
"""
import numpy as np

from .masks import allowed_mask


def _f64(x):
    return np.asarray(x, dtype=np.float64)


def attention_vjp(Q, K, V, gO, kind, offsets=None, scale=None, rows=None, keys=None, block=256):
    """(gQ, gK, gV, Delta) in fp64 for inputs of shape [B, H, L, D].

    ``rows`` restricts the query rows of gQ and Delta, ``keys`` the key rows of gK and
    gV (outputs then have len(rows) / len(keys) rows); every pair of the mask that
    touches them is always used.
    """
    Q, K, V, gO = _f64(Q), _f64(K), _f64(V), _f64(gO)
    B, H, L, D = Q.shape
    s = float(scale) if (scale is not None and scale > 0) else 1.0 / np.sqrt(D)
    rows = np.arange(L) if rows is None else np.asarray(rows, dtype=np.int64)
    keys = np.arange(L) if keys is None else np.asarray(keys, dtype=np.int64)
    want_row = np.zeros(L, dtype=bool)
    want_row[rows] = True
    row_pos = np.full(L, -1, dtype=np.int64)
    row_pos[rows] = np.arange(rows.size)
    # gQ and Delta need the requested rows; gK and gV every row that admits a requested
    # key (the other rows contribute exactly zero to them)
    visit_mask = want_row.copy()
    if keys.size:
        visit_mask |= allowed_mask(kind, offsets, L, cols=keys).any(axis=1)
    visit = np.flatnonzero(visit_mask)
    gQ = np.zeros((B, H, rows.size, D))
    Delta = np.zeros((B, H, rows.size))
    gK = np.zeros((B, H, keys.size, D))
    gV = np.zeros((B, H, keys.size, D))
    key_mask = np.zeros(L, dtype=bool)
    key_mask[keys] = True
    key_pos = np.full(L, -1, dtype=np.int64)
    key_pos[keys] = np.arange(keys.size)
    for r0 in range(0, visit.size, block):
        sel = visit[r0:r0 + block]
        allowed = allowed_mask(kind, offsets, L, sel)
        # columns no row of the block admits hold P = 0 and are left out (exact zeros)
        cols = np.flatnonzero(allowed.any(axis=0))
        a = allowed[:, cols]
        kc = cols[key_mask[cols]]  # requested keys among them
        for b in range(B):
            for h in range(H):
                q, k, v, g = Q[b, h, sel], K[b, h, cols], V[b, h, cols], gO[b, h, sel]
                S = np.where(a, s * (q @ k.T), -np.inf)
                m = S.max(axis=1) if cols.size else np.full(sel.size, -np.inf)
                empty = ~np.isfinite(m)
                E = np.where(a, np.exp(S - np.where(empty, 0.0, m)[:, None]), 0.0)
                l = E.sum(axis=1)
                P = E / np.where(empty, 1.0, l)[:, None]
                O = P @ v
                delta = (g * O).sum(axis=1)
                gS = P * (g @ v.T - delta[:, None])
                mine = want_row[sel]
                if mine.any():
                    pos = row_pos[sel[mine]]
                    gQ[b, h, pos] = s * (gS[mine] @ k)
                    Delta[b, h, pos] = delta[mine]
                if kc.size:
                    j = np.searchsorted(cols, kc)
                    gK[b, h, key_pos[kc]] += s * (gS[:, j].T @ q)
                    gV[b, h, key_pos[kc]] += P[:, j].T @ g
    return gQ, gK, gV, Delta
