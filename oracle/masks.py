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

A chunk layout is the prefix array ``offsets`` = [o_0=0 < o_1 < ... < o_N] of
chunk boundaries within ONE half (TF) or within the whole sequence
(block-causal).  Nothing here builds ranges or tiles: each (row, column) pair
is decided from the two tokens' chunk ids and halves, one comparison at a time.
"""
import numpy as np

MASK_FULL = "full"
MASK_BLOCK_CAUSAL = "block_causal"
MASK_TEACHER_FORCING = "teacher_forcing"


def _chunk_of(tok, offsets):
    """Chunk index of each token position ``tok`` (positions within one half)."""
    offsets = np.asarray(offsets, dtype=np.int64)
    return np.searchsorted(offsets, tok, side="right") - 1


def expected_length(kind, offsets):
    """Sequence length implied by a layout (None for the full mask)."""
    if kind == MASK_FULL:
        return None
    half = int(offsets[-1])
    return 2 * half if kind == MASK_TEACHER_FORCING else half


def allowed_mask(kind, offsets, L, rows=None):
    """Boolean matrix allowed[a, b] for query rows ``rows`` (default all) and all L keys."""
    rows = np.arange(L, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)
    cols = np.arange(L, dtype=np.int64)
    if kind == MASK_FULL:
        return np.ones((rows.size, L), dtype=bool)
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
