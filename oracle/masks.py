"""Attention masks materialised from their definition.  TEST INFRASTRUCTURE ONLY.

Mask kinds (paper, Sec. 3.1.1 on the packed teacher-forcing forward, and the
background section on TF / DF training):

* ``full``            -- every query attends every key (bidirectional teacher).
* ``block_causal``    -- diffusion-forcing mask on a sequence of N chunks: a
                         query in chunk i attends keys in chunks j <= i.
* ``teacher_forcing`` -- the packed sequence [clean c_1..c_N | noisy c_1..c_N].
                         A clean query in chunk j attends clean chunks <= j; a
                         noisy query in chunk i attends clean chunks < i and
                         the noisy chunk i itself (bidirectional inside it).
* ``ranges``          -- the mask given directly as query groups with key ranges
                         (paper App. B, sparse custom-mask representation): a list
                         of groups (q0, q1, K) where the query interval [q0, q1)
                         admits every key of every interval [k0, k1) in the list
                         K = [(k0, k1), ...] (any number R_g >= 0 of ranges).
                         Passed in place of ``offsets``.

A chunk layout is the prefix array ``offsets`` = [o_0=0 < o_1 < ... < o_N] of
chunk boundaries within ONE half (TF) or within the whole sequence
(block-causal).  Nothing here builds ranges or tiles: for a chunk layout each
(row, column) pair is decided from the two tokens' chunk ids and halves, and for
a range list from the row's group and the column's membership in that group's
key intervals, one comparison at a time.
"""
import numpy as np

MASK_FULL = "full"
MASK_BLOCK_CAUSAL = "block_causal"
MASK_TEACHER_FORCING = "teacher_forcing"
MASK_RANGES = "ranges"


def _chunk_of(tok, offsets):
    """Chunk index of each token position ``tok`` (positions within one half)."""
    offsets = np.asarray(offsets, dtype=np.int64)
    return np.searchsorted(offsets, tok, side="right") - 1


def check_groups(groups, L):
    """Validate a query-group / key-range list against a sequence of L tokens.

    The App. B representation gives each query group g a contiguous interval
    Q_g = [q0, q1) and a list K_g of key intervals [k0, k1).  The passage leaves two
    things implicit, read here as requirements: the query intervals of different
    groups are disjoint (each task of Algorithm 1 writes the output rows of its
    group, so a row in two groups would be written twice), and the key intervals of
    one group are disjoint (Algorithm 1 streams every interval of K_g, so a key in
    two of them would enter the softmax twice).  Empty intervals (k0 == k1), groups
    with no key interval and rows in no group are allowed: such rows admit no key.
    Returns the groups as [(q0, q1, [(k0, k1), ...]), ...].
    """
    out = []
    for g in groups:
        q0, q1, K = int(g[0]), int(g[1]), [(int(a), int(b)) for a, b in g[2]]
        if not 0 <= q0 < q1 <= L:
            raise ValueError(f"query interval [{q0}, {q1}) is not inside [0, {L})")
        for k0, k1 in K:
            if not 0 <= k0 <= k1 <= L:
                raise ValueError(f"key interval [{k0}, {k1}) is not inside [0, {L}]")
        nonempty = sorted((k0, k1) for k0, k1 in K if k1 > k0)
        for (a0, a1), (b0, b1) in zip(nonempty, nonempty[1:]):
            if b0 < a1:
                raise ValueError(f"key intervals [{a0}, {a1}) and [{b0}, {b1}) of one group overlap")
        out.append((q0, q1, K))
    spans = sorted((q0, q1) for q0, q1, _ in out)
    for (a0, a1), (b0, b1) in zip(spans, spans[1:]):
        if b0 < a1:
            raise ValueError(f"query intervals [{a0}, {a1}) and [{b0}, {b1}) overlap")
    return out


def allowed_mask(kind, offsets, L, rows=None, cols=None):
    """Boolean matrix allowed[a, b] for query rows ``rows`` and keys ``cols`` (default all)."""
    rows = np.arange(L, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    cols = np.arange(L, dtype=np.int64) if cols is None else np.asarray(cols, dtype=np.int64)
    if kind == MASK_FULL:
        return np.ones((rows.size, cols.size), dtype=bool)
    if kind == MASK_RANGES:
        # M[a, b] admits (a, b) iff some group g has a in Q_g and b in one of K_g's intervals
        out = np.zeros((rows.size, cols.size), dtype=bool)
        for q0, q1, K in check_groups(offsets, L):
            in_q = (rows >= q0) & (rows < q1)
            for k0, k1 in K:
                in_k = (cols >= k0) & (cols < k1)
                out |= in_q[:, None] & in_k[None, :]
        return out
    if kind == MASK_BLOCK_CAUSAL:
        assert L == int(offsets[-1]), "block-causal layout must cover the sequence"
        cq = _chunk_of(rows, offsets)[:, None]
        ck = _chunk_of(cols, offsets)[None, :]
        return ck <= cq
    if kind == MASK_TEACHER_FORCING:
        half = int(offsets[-1])
        assert L == 2 * half, "TF layout must cover [clean | noisy]"
        q_noisy = (rows >= half)[:, None]
        k_noisy = (cols >= half)[None, :]
        cq = _chunk_of(rows - half * (rows >= half), offsets)[:, None]
        ck = _chunk_of(cols - half * (cols >= half), offsets)[None, :]
        clean_to_clean = ~q_noisy & ~k_noisy & (ck <= cq)
        noisy_to_clean = q_noisy & ~k_noisy & (ck < cq)
        noisy_to_noisy = q_noisy & k_noisy & (ck == cq)
        return clean_to_clean | noisy_to_clean | noisy_to_noisy
    raise ValueError(f"unknown mask kind {kind!r}")


def count_allowed_pairs(kind, offsets, L, block=4096):
    """Number of allowed (query, key) pairs, by materialising the mask block by block."""
    total = 0
    for r0 in range(0, L, block):
        rows = np.arange(r0, min(L, r0 + block))
        total += int(allowed_mask(kind, offsets, L, rows).sum())
    return total
