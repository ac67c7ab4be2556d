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
                         of (q_end, a0, a1, b0, b1); group g owns query rows
                         [q_end of g-1, q_end) and admits keys in [a0, a1) and
                         [b0, b1).  Passed in place of ``offsets``.

A chunk layout is the prefix array ``offsets`` = [o_0=0 < o_1 < ... < o_N] of
chunk boundaries within ONE half (TF) or within the whole sequence
(block-causal).  Nothing here builds ranges or tiles: each (row, column) pair
is decided from the two tokens' chunk ids and halves, one comparison at a time.
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


def expected_length(kind, offsets):
    """Sequence length implied by a layout (None for the full mask)."""
    if kind == MASK_FULL:
        return None
    if kind == MASK_RANGES:
        return int(offsets[-1][0])
    half = int(offsets[-1])
    return 2 * half if kind == MASK_TEACHER_FORCING else half


def allowed_mask(kind, offsets, L, rows=None, cols=None):
    """Boolean matrix allowed[a, b] for query rows ``rows`` and keys ``cols`` (default all)."""
    rows = np.arange(L, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    cols = np.arange(L, dtype=np.int64) if cols is None else np.asarray(cols, dtype=np.int64)
    if kind == MASK_FULL:
        return np.ones((rows.size, cols.size), dtype=bool)
    if kind == MASK_RANGES:
        groups = [tuple(int(v) for v in g) for g in offsets]
        assert groups[-1][0] == L, "query groups must cover the sequence"
        q_end = np.array([g[0] for g in groups])
        g_of_row = np.searchsorted(q_end, rows, side="right")
        out = np.zeros((rows.size, cols.size), dtype=bool)
        for i, g in enumerate(g_of_row):
            _, a0, a1, b0, b1 = groups[g]
            out[i] = ((cols >= a0) & (cols < a1)) | ((cols >= b0) & (cols < b1))
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
