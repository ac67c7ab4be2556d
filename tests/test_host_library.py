"""CPU tests of the C-ABI library: symbols, host-side layout logic and error paths.

No kernel runs here.  Every call either is host-only (pair counts, group table,
tile plans) or fails argument validation, which happens before any HIP call.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from oracle import (MASK_BLOCK_CAUSAL, MASK_FULL, MASK_RANGES, MASK_TEACHER_FORCING, allowed_mask,
                    count_allowed_pairs)
from paper_2606_25473_amd import binding
from paper_2606_25473_amd.binding import make_layout
from paper_2606_25473_amd.workloads import WORKLOADS

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "attn_jvp.h")

LAYOUTS = [
    (MASK_TEACHER_FORCING, [0, 16, 32, 48, 64], 128),
    (MASK_TEACHER_FORCING, [0, 100, 200, 300], 600),
    (MASK_TEACHER_FORCING, [0, 1, 3, 7, 40, 41, 90, 200], 400),
    (MASK_TEACHER_FORCING, list(range(65)), 128),          # C = 1, N = 64
    (MASK_TEACHER_FORCING, [0, 300], 600),                  # N = 1
    (MASK_BLOCK_CAUSAL, [0, 50, 77, 200, 333], 333),
    (MASK_FULL, None, 1000),
    (MASK_FULL, None, 7),
    (MASK_RANGES, [(0, 100, []), (100, 300, [(0, 50), (250, 300)]), (300, 301, [(0, 301)]),
                   (301, 520, [(400, 520), (10, 20)])], 520),
    (MASK_RANGES, [(0, 7, [(3, 5)])], 7),
    # several key ranges per group, adjacent ones, an empty one, out of order
    (MASK_RANGES, [(0, 40, [(0, 5), (30, 33), (60, 90), (100, 101)]), (40, 41, []),
                   (41, 200, [(10, 20), (20, 40), (150, 200)]), (200, 300, [(299, 300), (0, 1), (50, 50), (120, 180)])],
     300),
]


def random_ranges(L, G, seed, max_ranges=5):
    """Seeded random query groups tiling [0, L), each with 0..max_ranges disjoint key ranges
    (some empty, some touching, in random order)."""
    rng = np.random.default_rng(seed)
    cuts = [0] + sorted(int(c) for c in rng.choice(np.arange(1, L), size=G - 1, replace=False)) + [L]
    groups = []
    for q0, q1 in zip(cuts, cuts[1:]):
        n = int(rng.integers(0, max_ranges + 1))
        pts = sorted(int(v) for v in rng.integers(0, L + 1, size=2 * n))
        ks = [(pts[2 * i], pts[2 * i + 1]) for i in range(n)]
        if n >= 2 and rng.random() < 0.3:  # make two neighbours touch
            ks[1] = (ks[0][1], max(ks[0][1], ks[1][1]))
        rng.shuffle(ks)
        groups.append((q0, q1, [tuple(k) for k in ks]))
    return groups


@pytest.fixture(scope="module")
def lib():
    return binding.load_library()


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return re.findall(r"^\s*(?:const\s+)?[a-z0-9_]+\s*\*?\s*(attn_[a-z_]+)\s*\(", text, flags=re.M)


def test_library_exports_every_declared_symbol(lib):
    names = _declared_functions()
    assert {"attn_jvp_fwd", "attn_fwd", "attn_count_unmasked_pairs", "attn_last_error"} <= set(names)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in attn_jvp.h but not exported"


@pytest.mark.parametrize("kind,offsets,L", LAYOUTS)
def test_unmasked_pair_count_matches_brute_force(lib, kind, offsets, L):
    assert binding.count_unmasked_pairs(kind, offsets, L) == count_allowed_pairs(kind, offsets, L)


@pytest.mark.parametrize("name", ["tiny_tf", "wan1.3b_chunkwise_tf", "wan1.3b_framewise_tf",
                                  "wan1.3b_bidirectional", "wan14b_chunkwise_tf"])
def test_workload_pair_counts_closed_form(lib, name):
    w = WORKLOADS[name]
    n = binding.count_unmasked_pairs(w.kind, list(w.offsets) or None, w.L)
    if w.kind == MASK_FULL:
        assert n == w.L * w.L
    else:
        C, N = w.offsets[1], w.num_chunks
        assert n == C * C * N * (N + 1)


def _table_mask(groups, L):
    """Mask of a library table [(q0, q1, [(k0, k1), ...]), ...], checking its normal form:
    the groups tile [0, L); each group's ranges are non-empty, increasing, not touching."""
    m = np.zeros((L, L), dtype=bool)
    prev = 0
    for q0, q1, ks in groups:
        assert q0 == prev and q1 > q0
        prev = q1
        for (a0, a1), (b0, b1) in zip(ks, ks[1:]):
            assert a1 < b0
        for k0, k1 in ks:
            assert 0 <= k0 < k1 <= L
            m[q0:q1, k0:k1] = True
    assert prev == L
    return m


@pytest.mark.parametrize("kind,offsets,L", LAYOUTS)
def test_query_groups_reproduce_mask(lib, kind, offsets, L):
    groups = binding.query_groups(kind, offsets, L)
    assert np.array_equal(_table_mask(groups, L), allowed_mask(kind, offsets, L))


@pytest.mark.parametrize("kind,offsets,L", LAYOUTS)
def test_key_tile_plans_cover_transposed_mask(lib, kind, offsets, L):
    """The backward's key tiles visit every query block with an admissible pair, once, in
    order, and skip the mask only on blocks where every (query, key) pair is admissible."""
    KT, QB = 128, 64
    mask = allowed_mask(kind, offsets, L)
    for t in range((L + KT - 1) // KT):
        keys = slice(t * KT, min(L, t * KT + KT))
        plan = binding.key_tile_plan(kind, offsets, L, t)
        blocks = [b for b, _ in plan]
        assert blocks == sorted(set(blocks))
        visited = np.zeros(L, dtype=bool)
        for b, full in plan:
            visited[b * QB:(b + 1) * QB] = True
            if full:
                assert b * QB + QB <= L and mask[b * QB:b * QB + QB, keys].all()
        assert not (mask[:, keys] & ~visited[:, None]).any()


def test_key_tile_plan_of_teacher_forcing(lib):
    # keys 0..127 of 4 chunks x 64 tokens: clean chunks 0 and 1, seen by clean rows 0..255
    # (all of them admit every key of the tile from row 64 on) and noisy rows 320..511
    plan = binding.key_tile_plan("teacher_forcing", [0, 64, 128, 192, 256], 512, 0)
    assert [b for b, _ in plan] == [0, 1, 2, 3, 5, 6, 7]
    assert [f for _, f in plan] == [False, True, True, True, False, True, True]


def _many_runs():
    """128 two-row query groups; group g admits keys g and 128 + g: each key is seen by one
    group, and a key tile by 128 separate query runs."""
    return [(2 * g, 2 * g + 2, [(g, g + 1), (128 + g, 129 + g)]) for g in range(128)]


def test_key_tile_plan_with_many_query_runs(lib):
    test_key_tile_plans_cover_transposed_mask(lib, MASK_RANGES, _many_runs(), 256)
    assert len(binding.query_groups("ranges", _many_runs(), 256)) == 128


@pytest.mark.parametrize("seed", range(10))
def test_random_range_lists(lib, seed):
    L = int(np.random.default_rng(seed).integers(40, 900))
    groups = random_ranges(L, 1 + seed * 5, seed)
    assert binding.count_unmasked_pairs("ranges", groups, L) == count_allowed_pairs(MASK_RANGES, groups, L)
    test_query_groups_reproduce_mask(lib, MASK_RANGES, groups, L)
    test_key_tile_plans_cover_transposed_mask(lib, MASK_RANGES, groups, L)
    test_tile_plans_cover_mask_and_full_blocks_are_full(lib, MASK_RANGES, groups, L)


@pytest.mark.parametrize("kind,offsets,L", LAYOUTS)
def test_tile_plans_cover_mask_and_full_blocks_are_full(lib, kind, offsets, L):
    R, C = binding.tile_shape()
    mask = allowed_mask(kind, offsets, L)
    computed = 0
    for t in range((L + R - 1) // R):
        rows = slice(t * R, min(L, t * R + R))
        plan = binding.tile_plan(kind, offsets, L, t)
        blocks = [b for b, _ in plan]
        assert blocks == sorted(set(blocks)), "blocks visited once, in key order"
        visited = np.zeros(L, dtype=bool)
        for b, full in plan:
            visited[b * C:(b + 1) * C] = True
            if full:
                assert b * C + C <= L and mask[rows, b * C:b * C + C].all()
            computed += (rows.stop - rows.start) * min(C, L - b * C)
        # every admissible pair of the tile lies in a visited block
        assert not (mask[rows] & ~visited[None, :]).any()
    assert computed == binding.count_computed_pairs(kind, offsets, L)


def test_computed_pair_overhead_on_wan_chunkwise(lib):
    w = WORKLOADS["wan1.3b_chunkwise_tf"]
    un = binding.count_unmasked_pairs(w.kind, w.offsets, w.L)
    comp = binding.count_computed_pairs(w.kind, w.offsets, w.L)
    assert 1.0 <= comp / un < 1.02


def _tile_cost(kind, offsets, L, t, zero_clean):
    """Key-block contractions of tile t: 2 (scores, output) per block for a primal-only
    tile, 4 per block of clean keys and 6 per block with noisy keys otherwise."""
    R, C = binding.tile_shape()
    half = L // 2
    blocks = [b for b, _ in binding.tile_plan(kind, offsets, L, t)]
    if not zero_clean:
        return 6 * len(blocks)
    if (t + 1) * R <= half:
        return 2 * len(blocks)
    return sum(6 if b * C + C > half else 4 for b in blocks)


@pytest.mark.parametrize("kind,offsets,L", LAYOUTS)
def test_tile_order_is_a_permutation(lib, kind, offsets, L):
    R, _ = binding.tile_shape()
    nt = (L + R - 1) // R
    assert sorted(binding.tile_order(kind, offsets, L)) == list(range(nt))
    if kind == MASK_TEACHER_FORCING:
        assert sorted(binding.tile_order(kind, offsets, L, zero_clean=True)) == list(range(nt))


@pytest.mark.parametrize("name", ["wan1.3b_chunkwise_tf", "wan1.3b_framewise_tf"])
def test_zero_clean_tile_order_is_heaviest_first(lib, name):
    """The zero-clean order starts with one of the heaviest tiles and ends with the
    lightest ones: every tile of the last quarter costs at most what the lightest
    tile of the first quarter costs (the tiles straddling two noisy chunks are the
    only ones out of monotone order, and only slightly)."""
    w = WORKLOADS[name]
    order = binding.tile_order(w.kind, w.offsets, w.L, zero_clean=True)
    costs = [_tile_cost(w.kind, w.offsets, w.L, t, True) for t in order]
    q = len(costs) // 4
    assert costs[0] >= 0.9 * max(costs) and costs[-1] == min(costs)
    assert max(costs[-q:]) <= min(costs[:q])


def test_tile_order_rejects_zero_clean_without_teacher_forcing(lib):
    with pytest.raises(binding.AttnError):
        binding.tile_order("block_causal", [0, 300, 600], 600, zero_clean=True)


# ----------------------------------------------------------------------------- error paths

FAKE = 1 << 40          # never dereferenced: every call below fails validation first

# Belt and braces: these calls pass fake device pointers, so never run them where a
# GPU could actually receive a launch if a case were wrongly accepted.
_no_gpu = pytest.mark.skipif(__import__("torch").cuda.is_available(),
                             reason="fake-pointer validation tests run on CPU-only hosts")


def _ptrs(n=9, dtype_bytes=2, B=1, H=1, L=64, D=64):
    span = B * H * L * D * dtype_bytes
    return [FAKE + i * (span + 4096) for i in range(n)]


def _with(i, value):
    """The 9 pointers Q, K, V, dQ, dK, dV, O, dO, LSE with entry i replaced."""
    p = _ptrs()
    p[i] = value
    return p


def _raw(bounds, roffs, flat):
    """An ATTN_MASK_RANGES layout built directly from its three arrays (no binding checks)."""
    arrs = [None if a is None else (ctypes.c_int32 * max(1, len(a)))(*a) for a in (bounds, roffs, flat)]
    lay = binding._Layout(3, len(bounds) - 1, *arrs)
    lay._keep = arrs
    return lay


def _call(lib, **kw):
    dtype, B, H, L, D = kw.get("dtype", 1), kw.get("B", 1), kw.get("H", 1), kw.get("L", 64), kw.get("D", 64)
    es = 4 if dtype == 0 else 2
    p = kw.get("ptrs") or _ptrs(9, es, B, H, L, D)
    layout = kw.get("layout") or make_layout("full")
    return lib.attn_jvp_fwd(dtype, B, H, L, D, p[0], p[1], p[2], p[3], p[4], p[5],
                            ctypes.byref(layout), 0.0, p[6], p[7], p[8], None)


@pytest.mark.parametrize("kw,code,needle", [
    (dict(dtype=7), 2, "dtype"),
    (dict(D=96), 2, "head_dim"),
    (dict(L=0), 1, "positive"),
    (dict(B=-1), 1, "positive"),
    (dict(ptrs=_with(0, 0)), 1, "NULL"),
    (dict(ptrs=_with(5, 0)), 1, "NULL"),
    (dict(ptrs=_with(0, FAKE + 2)), 1, "aligned"),
    # fp32 tensors too are moved in 16-byte pieces: a 4-byte aligned Q or dV is refused
    (dict(dtype=0, ptrs=_with(0, FAKE + 4)), 1, "16-byte aligned"),
    (dict(dtype=0, ptrs=_with(5, FAKE + 5 * (64 * 64 * 4 + 4096) + 8)), 1, "16-byte aligned"),
    (dict(ptrs=_with(6, _ptrs()[0])), 1, "overlaps input"),
    (dict(ptrs=_with(7, _ptrs()[6] + 64)), 1, "overlap"),
    (dict(layout=make_layout("teacher_forcing", [0, 16, 40])), 1, "L = 2"),
    (dict(layout=make_layout("teacher_forcing", [0, 16, 16, 32]), L=64), 1, "increasing"),
    (dict(layout=make_layout("teacher_forcing", [5, 16, 32]), L=64), 1, "must be 0"),
    (dict(layout=make_layout("block_causal", [0, 10, 20]), L=64), 1, "block-causal"),
    (dict(layout=make_layout("teacher_forcing", list(range(66))), L=130), 1, "num_chunks"),
    (dict(layout=make_layout(9)), 1, "kind"),
    (dict(layout=_raw([0, 30, 64], [0, 2, 3], [0, 10, 5, 20, 0, 64])), 1, "overlap"),
    (dict(layout=_raw([0, 30, 60], [0, 1, 2], [0, 10, 0, 64])), 1, "cover"),
    (dict(layout=_raw([0, 30, 30, 64], [0, 1, 1, 2], [0, 10, 0, 64])), 1, "increasing"),
    (dict(layout=_raw([5, 64], [0, 1], [0, 10])), 1, "row 0"),
    (dict(layout=_raw([0, 64], [0, 1], [0, 65])), 1, "begin <= end <= L"),
    (dict(layout=_raw([0, 64], [0, 1], [9, 3])), 1, "begin <= end <= L"),
    (dict(layout=_raw([0, 32, 64], [0, 2, 1], [0, 1, 2, 3])), 1, "must not decrease"),
    (dict(layout=_raw([0, 64], [1, 1], [0, 1])), 1, "range_offsets[0]"),
    (dict(layout=_raw([0, 64], None, [0, 1])), 1, "range_offsets is NULL"),
    (dict(layout=_raw([0, 64], [0, 1], None)), 1, "ranges is NULL"),
    (dict(layout=_raw([0], [0], [])), 1, "query groups"),
    (dict(layout=_raw(list(range(0, 130)), list(range(130)), list(range(2 * 129))), L=129), 1,
     "query groups"),
    # 257 disjoint, non-touching ranges in one group: more than the table holds
    (dict(layout=_raw([0, 1024], [0, 257], [v for i in range(257) for v in (3 * i, 3 * i + 1)]), L=1024), 1,
     "ATTN_MAX_RANGES"),
    # size limits: 32-bit offsets within a bf16 head, work-groups per launch, fp32 grid rows
    (dict(L=(1 << 24) + 2, D=128, layout=make_layout("teacher_forcing", [0, (1 << 23) + 1])), 1, "2^31"),
    (dict(L=(1 << 25) + 2, D=64, layout=make_layout("teacher_forcing", [0, (1 << 24) + 1])), 1, "2^31"),
    (dict(B=1024, H=1024, L=1 << 18, D=64), 1, "work-groups"),
    (dict(B=2, H=1 << 20), 1, "B * H too large"),
    (dict(dtype=0, L=(1 << 23) + 2, D=128, layout=make_layout("teacher_forcing", [0, (1 << 22) + 1])), 1,
     "2^30"),
])
@_no_gpu
def test_invalid_arguments_are_rejected_before_any_hip_call(lib, kw, code, needle):
    rc = _call(lib, **kw)
    assert rc == code
    assert needle in binding.last_error()


@_no_gpu
def test_zero_clean_entry_point_validates(lib):
    # tangents of the noisy half: [1, 1, 32, 64] bf16 buffers
    p = _ptrs(9)
    lay = make_layout("full")
    rc = lib.attn_jvp_fwd_zero_clean(1, 1, 1, 64, 64, p[0], p[1], p[2], p[3], p[4], p[5], ctypes.byref(lay),
                                     0.0, p[6], p[7], p[8], None)
    assert rc == 1 and "teacher-forcing" in binding.last_error()
    lay = make_layout("teacher_forcing", [0, 16, 32])
    # dOn overlapping dKn (both are half-length buffers: 4096 bytes)
    q = list(p)
    q[7] = q[4] + 2048
    rc = lib.attn_jvp_fwd_zero_clean(1, 1, 1, 64, 64, q[0], q[1], q[2], q[3], q[4], q[5], ctypes.byref(lay),
                                     0.0, q[6], q[7], q[8], None)
    assert rc == 1 and "overlaps input dK" in binding.last_error()
    # a dOn right after a half-length dKn does not overlap it (the buffers are half-length);
    # a layout error is then the first failure
    q[7] = q[4] + 4096
    rc = lib.attn_jvp_fwd_zero_clean(1, 1, 1, 64, 64, q[0], q[1], q[2], q[3], q[4], q[5],
                                     ctypes.byref(make_layout("teacher_forcing", [0, 16, 40])), 0.0,
                                     q[6], q[7], q[8], None)
    assert rc == 1 and "L = 2" in binding.last_error()


@_no_gpu
def test_backward_entry_point_validates(lib):
    # Q, K, V, O, gO, LSE, gQ, gK, gV, Delta as fake bf16 [1, 1, 64, 64] / fp32 [1, 1, 64]
    p = _ptrs(10)

    def call(ptrs, layout=None, dtype=1, D=64):
        lay = layout or make_layout("full")
        return lib.attn_bwd(dtype, 1, 1, 64, D, *ptrs[:6], ctypes.byref(lay), 0.0, *ptrs[6:], None)

    q = list(p); q[4] = 0
    assert call(q) == 1 and "NULL pointer gO" in binding.last_error()
    q = list(p); q[9] = q[0]
    assert call(q) == 1 and "overlaps input Q" in binding.last_error()
    q = list(p); q[7] = q[6] + 1024
    assert call(q) == 1 and "overlap" in binding.last_error()
    q = list(p); q[0] = q[0] + 4  # fp32 inputs need 16-byte alignment too
    assert call(q, dtype=0) == 1 and "misaligned" in binding.last_error()
    assert call(p, D=80) == 2 and "head_dim" in binding.last_error()
    assert call(p, layout=make_layout("teacher_forcing", [0, 16, 40])) == 1 and "L = 2" in binding.last_error()


@_no_gpu
def test_largest_accepted_sizes_pass_the_size_checks(lib):
    # the largest bf16 head (L * D = 2^31), the largest fp32 head (L * D = 2^30) and fp32
    # launches over 2^20 (batch, head) pairs pass the size checks: the first failure is then
    # a deliberately bad layout (checked later)
    bad = make_layout("teacher_forcing", [0, 16, 40])
    assert _call(lib, L=1 << 24, D=128, layout=bad) == 1 and "L = 2" in binding.last_error()
    assert _call(lib, dtype=0, L=1 << 23, D=128, layout=bad) == 1 and "L = 2" in binding.last_error()
    assert _call(lib, dtype=0, B=1024, H=1024, L=16, layout=bad) == 1 and "L = 2" in binding.last_error()
    p = _ptrs(10, 2, 1, 1, 1 << 24, 128)
    rc = lib.attn_bwd(1, 1, 1, (1 << 24) + 2, 128, *p[:6], ctypes.byref(make_layout("full")), 0.0, *p[6:], None)
    assert rc == 1 and "2^31" in binding.last_error()
    # and so does an fp32 backward over 2^20 (batch, head) pairs
    p = _ptrs(10, 4, 1024, 1024, 16, 64)
    rc = lib.attn_bwd(0, 1024, 1024, 16, 64, *p[:6], ctypes.byref(bad), 0.0, *p[6:], None)
    assert rc == 1 and "L = 2" in binding.last_error()


@_no_gpu
def test_forward_entry_point_validates_too(lib):
    p = _ptrs(5)
    rc = lib.attn_fwd(1, 1, 1, 64, 80, p[0], p[1], p[2], ctypes.byref(make_layout("full")), 0.0, p[3], p[4], None)
    assert rc == 2 and "head_dim" in binding.last_error()


def test_host_queries_reject_bad_layouts(lib):
    with pytest.raises(binding.AttnError):
        binding.count_unmasked_pairs("teacher_forcing", [0, 10, 5], 20)
    with pytest.raises(binding.AttnError):
        binding.tile_plan("full", None, 100, 1)
    assert lib.attn_count_computed_pairs(ctypes.byref(make_layout("full")), 100, 32) == -1


def test_python_binding_refuses_cpu_tensors():
    import torch
    x = torch.zeros(1, 1, 8, 64)
    with pytest.raises(ValueError):
        binding.attn_jvp_fwd(x, x, x, x, x, x, "full")


def test_header_compiles_as_c_and_links(lib, tmp_path):
    """The ABI is usable from plain C: tests/c/abi_check.c compiled with gcc -std=c99
    against include/attn_jvp.h, linked to the library, run (host-only calls)."""
    import shutil
    import subprocess
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    libdir = os.path.dirname(binding.library_path())
    exe = str(tmp_path / "abi_check")
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(root, "include"),
                    os.path.join(root, "tests", "c", "abi_check.c"), "-L", libdir, "-lattnjvp",
                    "-Wl,-rpath," + libdir, "-o", exe], check=True)
    out = subprocess.run([exe], capture_output=True, text=True)
    assert out.returncode == 0 and out.stdout.strip() == "OK", out.stdout + out.stderr


def test_schedule_helpers_on_the_host(tmp_path):
    """The work-group -> (batch-head, tile) slots and the tile orders that the kernels
    evaluate (schedule.hpp, compiled here with g++) are permutations."""
    import shutil
    import subprocess
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    exe = str(tmp_path / "schedule_check")
    subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-Werror",
                    "-I", os.path.join(root, "paper_2606_25473_amd", "csrc"),
                    os.path.join(root, "tests", "c", "schedule_check.cpp"), "-o", exe], check=True)
    out = subprocess.run([exe], capture_output=True, text=True)
    assert out.returncode == 0 and out.stdout.strip() == "OK", out.stdout + out.stderr


def test_binding_checks_caller_supplied_outputs():
    """Outputs passed in `out` must have the shape, dtype, device and layout the call
    writes; the check runs before any library call (here on CPU tensors, q's device)."""
    import torch
    q = torch.zeros(1, 2, 8, 64, dtype=torch.bfloat16)
    good = [("O", q.shape, q.dtype), ("LSE", (1, 2, 8), torch.float32)]
    binding._check_outs([torch.empty_like(q), torch.empty(1, 2, 8)], good, q)
    bad_sets = [
        [torch.empty(1, 2, 7, 64, dtype=torch.bfloat16), torch.empty(1, 2, 8)],   # short O
        [torch.empty_like(q, dtype=torch.float32), torch.empty(1, 2, 8)],         # O dtype
        [torch.empty_like(q), torch.empty(1, 2, 8, dtype=torch.bfloat16)],        # LSE dtype
        [torch.empty_like(q), torch.empty(1, 2, 16)[..., ::2]],                    # LSE not contiguous
        [torch.empty_like(q)],                                                     # missing LSE
    ]
    for outs in bad_sets:
        with pytest.raises(ValueError):
            binding._check_outs(outs, good, q)
