"""Host checks of the LDS address arithmetic of the bf16 matrix-core kernels (CPU only).

The kernels swizzle the 16-byte chunks of every LDS row (D bf16 values = D/8 chunks) as
chunk ^ swz(row), with swz(row) = 4 (row mod 4) + (row / 4 mod 4) for D = 128 and
4 (row / 2 mod 2) + (row / 4 mod 4) for D = 64 (two 128-byte rows per 64 banks), and form the
per-step operand offsets by XOR from per-lane bases instead of holding every offset in a
register:

* b128 score-operand reads: chunk 2s + hh of a row lies at lds_off(row, hh) ^ 32 s;
* transposed reads (ds_read_b64_tr_b16) for k step t, key half p and d tile dt lie at
  16 t ROWB + (trx[p] ^ 64 dt).

Both identities need the tile base to be a multiple of the row size (the kernels assert
1 KiB alignment).  This file restates the swizzle and checks the identities for every lane
and step, that the swizzle is a bijection of each row's chunks, and that the reads are free
of LDS bank conflicts (64 banks of 4 bytes; a b128 read serves 16 lanes per pass, a
transposed b64 read 32 lanes).
"""
import pytest


def swz(D, row):
    if D == 128:
        return ((row & 3) << 2) | ((row >> 2) & 3)
    return (((row >> 1) & 1) << 2) | ((row >> 2) & 3)


def lds_off(D, row, chunk):
    return row * (2 * D) + ((chunk ^ swz(D, row)) << 4)


def tr_offset(D, lane, t, p, dt):
    """Per-lane offset of the transposed read as the kernels first computed it."""
    g16, s16 = lane >> 4, lane & 15
    r = 16 * t + 8 * p + 4 * (g16 >> 1) + (s16 >> 2)
    chunk = 4 * dt + 2 * (g16 & 1) + ((s16 & 3) >> 1)
    return lds_off(D, r, chunk) + 8 * (s16 & 1)


def tr_base(D, lane, p):
    g16, s16 = lane >> 4, lane & 15
    r = 4 * (g16 >> 1) + (s16 >> 2)
    chunk = 2 * (g16 & 1) + ((s16 & 3) >> 1)
    return lds_off(D, 8 * p + r, chunk) + 8 * (s16 & 1)


@pytest.mark.parametrize("D", [64, 128])
def test_swizzle_is_a_bijection_of_each_row(D):
    for row in range(64):
        assert sorted(c ^ swz(D, row) for c in range(D // 8)) == list(range(D // 8))


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("base", [0, 8192, 3 * 32768])
def test_score_operand_offsets_by_xor(D, base):
    for lane in range(64):
        hh, krow = lane >> 5, lane & 31
        for s in range(D // 16):
            assert base + lds_off(D, krow, 2 * s + hh) == (base + lds_off(D, krow, hh)) ^ (32 * s)


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("base", [0, 8192, 3 * 32768])
def test_transposed_offsets_by_xor(D, base):
    rowb = 2 * D
    for lane in range(64):
        for p in range(2):
            for t in range(2):
                for dt in range(D // 32):
                    want = base + tr_offset(D, lane, t, p, dt)
                    assert want == ((base + tr_base(D, lane, p)) ^ (64 * dt)) + 16 * t * rowb


def test_xor_identity_needs_row_aligned_bases():
    # a base that is not a multiple of the row size breaks the identity (the kernels assert
    # 1 KiB-aligned tiles for this reason)
    D, base = 128, 32
    broken = any(base + lds_off(D, lane & 31, 2 * s + (lane >> 5)) !=
                 (base + lds_off(D, lane & 31, lane >> 5)) ^ (32 * s)
                 for lane in range(64) for s in range(D // 16))
    assert broken


def _banks(addrs_bytes, width):
    """Bank-conflict degree of one pass: max number of distinct 4-byte words per bank."""
    words = {}
    for a in addrs_bytes:
        for w in range(width // 4):
            word = a // 4 + w
            words.setdefault(word % 64, set()).add(word)
    return max(len(v) for v in words.values())


@pytest.mark.parametrize("D", [64, 128])
def test_score_operand_reads_are_conflict_free(D):
    # ds_read_b128: lane l reads row l % 32, chunk 2s + l / 32; 16 lanes per pass
    for s in range(D // 16):
        addrs = [lds_off(D, lane & 31, 2 * s + (lane >> 5)) for lane in range(64)]
        for p0 in range(0, 64, 16):
            assert _banks(addrs[p0:p0 + 16], 16) == 1


@pytest.mark.parametrize("D", [64, 128])
def test_transposed_reads_are_conflict_free(D):
    # ds_read_b64_tr_b16: 8 bytes per lane, 32 lanes per pass
    for t in range(2):
        for p in range(2):
            for dt in range(D // 32):
                addrs = [tr_offset(D, lane, t, p, dt) for lane in range(64)]
                for p0 in range(0, 64, 32):
                    assert _banks(addrs[p0:p0 + 32], 8) == 1
