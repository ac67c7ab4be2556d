"""GPU parity of the HIP path against the fp64 CPU oracle (marked ``gpu``).

Small and edge-case shapes are compared element by element over every output;
the full Wan-shaped workloads are run in the launch configuration the bench
times and compared on sampled rows (chunk and tile boundaries plus seeded
random rows), which the oracle evaluates one by one.

Tolerance: relative L2 error ||x - x_ref|| / ||x_ref|| per output (O, dO, LSE),
<= 1e-2 for bf16 inputs/outputs and <= 1e-4 for the fp32 path.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import attention_jvp
from paper_2606_25473_amd import attn_fwd, attn_jvp_fwd
from paper_2606_25473_amd.workloads import (MASK_BLOCK_CAUSAL, MASK_FULL, MASK_TEACHER_FORCING, WORKLOADS,
                                            custom_workload, make_inputs)

pytestmark = pytest.mark.gpu

TOL = {"bf16": 1e-2, "f32": 1e-4}


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def _rel(x, ref):
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(x - ref) / max(np.linalg.norm(ref), 1e-300))


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _offsets(w):
    return list(w.offsets) if w.offsets else None


def _run_gpu(w, x):
    g = {k: v.cuda() for k, v in x.items()}
    o, do, lse = attn_jvp_fwd(g["Q"], g["K"], g["V"], g["dQ"], g["dK"], g["dV"], w.kind, _offsets(w))
    torch.cuda.synchronize()
    return o, do, lse


def _check_full(w, seed=0):
    _say(f"[parity] {w.name} B={w.B} H={w.H} L={w.L} D={w.D} {w.dtype} {w.kind} offsets={w.offsets[:6]}")
    x = make_inputs(w, "cpu", seed)
    o, do, lse = _run_gpu(w, x)
    O, dO, LSE = attention_jvp(*[_np(x[k]) for k in ("Q", "K", "V", "dQ", "dK", "dV")], w.kind, _offsets(w))
    errs = (_rel(_np(o), O), _rel(_np(do), dO), _rel(_np(lse), LSE))
    _say(f"[parity] {w.name} rel-L2 O={errs[0]:.3e} dO={errs[1]:.3e} LSE={errs[2]:.3e}")
    tol = TOL[w.dtype]
    assert max(errs) <= tol, errs
    return x, (o, do, lse)


EDGE = [
    custom_workload("tf_ragged_bf16", 2, 2, 128, "bf16", MASK_TEACHER_FORCING, 3, 100, tangent_std=0.5),
    custom_workload("tf_several_tiles_bf16", 1, 3, 128, "bf16", MASK_TEACHER_FORCING, 4, 300, tangent_std=0.5),
    # 3 x 3 = 9 (batch, head) pairs: two full groups of four heads and a group of one in the
    # work-group order
    custom_workload("tf_nine_heads_bf16", 3, 3, 128, "bf16", MASK_TEACHER_FORCING, 2, 170, tangent_std=0.5),
    custom_workload("tf_one_token_chunks_bf16", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 64, 1, tangent_std=0.5),
    custom_workload("tf_one_chunk_bf16", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 1, 300, tangent_std=0.5),
    custom_workload("tf_nonuniform_bf16", 1, 2, 128, "bf16", MASK_TEACHER_FORCING,
                    offsets=[0, 1, 3, 7, 40, 41, 90, 200], tangent_std=0.5),
    custom_workload("tf_d64_bf16", 1, 2, 64, "bf16", MASK_TEACHER_FORCING, 4, 50, tangent_std=0.5),
    custom_workload("block_causal_bf16", 1, 2, 128, "bf16", MASK_BLOCK_CAUSAL,
                    offsets=[0, 50, 77, 200, 333], tangent_std=0.5),
    custom_workload("full_1000_bf16", 1, 2, 128, "bf16", MASK_FULL, L=1000, tangent_std=0.5),
    custom_workload("full_below_one_tile_bf16", 1, 1, 128, "bf16", MASK_FULL, L=7, tangent_std=0.5),
    custom_workload("full_single_token_bf16", 1, 1, 128, "bf16", MASK_FULL, L=1, tangent_std=0.5),
    custom_workload("full_d64_bf16", 2, 1, 64, "bf16", MASK_FULL, L=333, tangent_std=0.5),
    custom_workload("tf_f32_d128", 1, 2, 128, "f32", MASK_TEACHER_FORCING, 3, 20),
    custom_workload("full_f32_d64", 1, 2, 64, "f32", MASK_FULL, L=50),
    custom_workload("block_causal_f32", 1, 1, 64, "f32", MASK_BLOCK_CAUSAL, offsets=[0, 3, 10, 31]),
    # the fp32 kernels' own tiling (128-row tiles, 16 rows per wave, 32-key blocks): ragged
    # tails, several tiles, a partial head group, one-token and single chunks, uneven offsets
    custom_workload("tf_ragged_f32", 2, 2, 128, "f32", MASK_TEACHER_FORCING, 3, 100),
    custom_workload("tf_several_tiles_f32", 1, 3, 128, "f32", MASK_TEACHER_FORCING, 4, 300),
    custom_workload("tf_nine_heads_f32", 3, 3, 64, "f32", MASK_TEACHER_FORCING, 2, 170),
    custom_workload("tf_one_token_chunks_f32", 1, 2, 128, "f32", MASK_TEACHER_FORCING, 64, 1),
    custom_workload("tf_one_chunk_f32", 1, 2, 64, "f32", MASK_TEACHER_FORCING, 1, 300),
    custom_workload("tf_nonuniform_f32", 1, 2, 128, "f32", MASK_TEACHER_FORCING, offsets=[0, 1, 3, 7, 40, 41, 90, 200]),
    custom_workload("block_causal_uneven_f32", 1, 2, 128, "f32", MASK_BLOCK_CAUSAL, offsets=[0, 50, 77, 200, 333]),
    custom_workload("full_1000_f32", 1, 2, 128, "f32", MASK_FULL, L=1000),
    custom_workload("full_below_one_tile_f32", 1, 1, 128, "f32", MASK_FULL, L=7),
    custom_workload("full_single_token_f32", 1, 1, 64, "f32", MASK_FULL, L=1),
]


def test_tiny_tf_fp32_workload():
    """The 4-chunk x 16-token fp32 TF workload, seed 0, against the oracle to 1e-4."""
    _check_full(WORKLOADS["tiny_tf"])


@pytest.mark.parametrize("w", EDGE, ids=[w.name for w in EDGE])
def test_edge_shapes(w):
    _check_full(w, seed=1)


def test_zero_tangents_give_exact_zero():
    for dt in ("bf16", "f32"):
        w = custom_workload(f"zero_tangent_{dt}", 1, 2, 128, dt, MASK_TEACHER_FORCING, 3, 100)
        _say(f"[invariant] zero tangents {dt}")
        x = make_inputs(w, "cpu", 3)
        for k in ("dQ", "dK", "dV"):
            x[k] = torch.zeros_like(x[k])
        _, do, _ = _run_gpu(w, x)
        assert torch.count_nonzero(do).item() == 0


def test_forward_matches_jvp_primal_and_oracle():
    w = custom_workload("fwd_vs_jvp", 2, 2, 128, "bf16", MASK_TEACHER_FORCING, 3, 100, tangent_std=0.5)
    _say("[invariant] attn_fwd vs attn_jvp_fwd primal")
    x = make_inputs(w, "cpu", 4)
    o, _, lse = _run_gpu(w, x)
    g = {k: v.cuda() for k, v in x.items()}
    of, lsef = attn_fwd(g["Q"], g["K"], g["V"], w.kind, _offsets(w))
    torch.cuda.synchronize()
    # same operations in the same order for the primal part
    assert _rel(_np(of), _np(o)) < 1e-3
    assert _rel(_np(lsef), _np(lse)) < 1e-6
    O, _, LSE = attention_jvp(*[_np(x[k]) for k in ("Q", "K", "V", "dQ", "dK", "dV")], w.kind, _offsets(w))
    assert _rel(_np(of), O) < TOL["bf16"] and _rel(_np(lsef), LSE) < TOL["bf16"]


def test_deterministic_run_to_run():
    w = custom_workload("determinism", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 4, 150, tangent_std=0.5)
    _say("[invariant] determinism")
    x = make_inputs(w, "cpu", 5)
    a = _run_gpu(w, x)
    b = _run_gpu(w, x)
    for u, v in zip(a, b):
        assert torch.equal(u, v)


def test_clean_half_independent_of_noisy_inputs():
    w = custom_workload("clean_half", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 3, 100, tangent_std=0.5)
    _say("[invariant] clean half independent of noisy inputs")
    x = make_inputs(w, "cpu", 6)
    a = _run_gpu(w, x)
    half = w.L // 2
    y = {k: v.clone() for k, v in x.items()}
    gen = torch.Generator().manual_seed(99)
    for k in y:
        y[k][:, :, half:] = torch.randn(y[k][:, :, half:].shape, generator=gen).to(y[k].dtype)
    b = _run_gpu(w, y)
    for u, v in zip(a, b):
        assert torch.equal(u[:, :, :half], v[:, :, :half])


def test_tangent_linearity():
    w = custom_workload("linearity", 1, 2, 128, "f32", MASK_TEACHER_FORCING, 3, 40)
    _say("[invariant] linearity (fp32 path)")
    x = make_inputs(w, "cpu", 7)
    _, d1, _ = _run_gpu(w, x)
    y = dict(x)
    for k in ("dQ", "dK", "dV"):
        y[k] = 2.5 * x[k]
    _, d2, _ = _run_gpu(w, y)
    assert _rel(_np(d2), 2.5 * _np(d1)) < 1e-5


# ----------------------------------------------------------------------------- full-size workloads

def _sample_rows(w, n_random=24, seed=0):
    """Rows that cover every boundary the kernels treat specially: the first and last row
    of every query tile (256 rows for the JVP, 128 for the forward), the rows around every
    chunk boundary of both halves, the ends of the sequence, plus seeded random rows."""
    L = w.L
    rows = {0, L - 1}
    for t in range(0, L, 128):
        rows.update((t, min(L, t + 128) - 1))
    if w.kind == MASK_TEACHER_FORCING:
        half = w.offsets[-1]
        for o in w.offsets:
            for base in (0, half):
                for d in (-1, 0, 1):
                    r = base + o + d
                    if 0 <= r < L:
                        rows.add(r)
    rng = np.random.default_rng(seed)
    rows.update(int(r) for r in rng.integers(0, L, n_random))
    return np.array(sorted(rows))


def _sample_heads(w, n):
    """n (batch, head) pairs spread over the launch (every pair when n >= B * H)."""
    pairs = [(b, h) for b in range(w.B) for h in range(w.H)]
    if n >= len(pairs):
        return pairs
    idx = np.unique(np.linspace(0, len(pairs) - 1, n).round().astype(int))
    return [pairs[i] for i in idx]


FULL_SIZE = ["wan1.3b_chunkwise_tf", "wan1.3b_framewise_tf", "wan1.3b_bidirectional", "wan14b_chunkwise_tf"]
# heads compared with the oracle: every one of the 1.3B shapes, 16 of the 80 of the 14B shape
FULL_SIZE_HEADS = {"wan1.3b_chunkwise_tf": 12, "wan1.3b_framewise_tf": 12, "wan1.3b_bidirectional": 12,
                   "wan14b_chunkwise_tf": 16}


@pytest.mark.parametrize("name", FULL_SIZE)
def test_full_size_sampled_rows(name):
    w = WORKLOADS[name]
    _say(f"[full-size] {name} B={w.B} H={w.H} L={w.L}: generating inputs on the GPU")
    x = make_inputs(w, "cuda", 0)
    o, do, lse = attn_jvp_fwd(x["Q"], x["K"], x["V"], x["dQ"], x["dK"], x["dV"], w.kind, _offsets(w))
    torch.cuda.synchronize()
    _say(f"[full-size] {name}: kernel done, checking finiteness and sampled rows")
    assert torch.isfinite(o).all() and torch.isfinite(do).all() and torch.isfinite(lse).all()
    rows = _sample_rows(w)
    heads = _sample_heads(w, FULL_SIZE_HEADS[name])
    fwd = attn_fwd(x["Q"], x["K"], x["V"], w.kind, _offsets(w)) if name == "wan14b_chunkwise_tf" else None
    torch.cuda.synchronize()
    ridx = torch.from_numpy(rows).cuda()
    worst = [0.0, 0.0, 0.0]
    for b, h in heads:
        sl = {k: _np(v[b:b + 1, h:h + 1]) for k, v in x.items()}
        O, dO, LSE = attention_jvp(sl["Q"], sl["K"], sl["V"], sl["dQ"], sl["dK"], sl["dV"], w.kind,
                                   _offsets(w), rows=rows)
        got = (_np(o[b, h].index_select(0, ridx)), _np(do[b, h].index_select(0, ridx)),
               _np(lse[b, h].index_select(0, ridx)))
        errs = (_rel(got[0], O[0, 0]), _rel(got[1], dO[0, 0]), _rel(got[2], LSE[0, 0]))
        worst = [max(a, e) for a, e in zip(worst, errs)]
        assert max(errs) <= TOL["bf16"], ((b, h), errs)
        if fwd is not None:
            ef = (_rel(_np(fwd[0][b, h].index_select(0, ridx)), O[0, 0]),
                  _rel(_np(fwd[1][b, h].index_select(0, ridx)), LSE[0, 0]))
            assert max(ef) <= TOL["bf16"], ((b, h), ef)
    _say(f"[full-size] {name} {len(heads)} heads x {len(rows)} rows: worst rel-L2 O={worst[0]:.3e} "
         f"dO={worst[1]:.3e} LSE={worst[2]:.3e}")


def test_whole_head_bidirectional():
    """One whole head of the Wan-shaped bidirectional workload (bf16, L = 32760, D = 128),
    every row of O, dO and LSE (and of the forward's O and LSE) against the oracle."""
    w = WORKLOADS["wan1.3b_bidirectional"]
    b, h = 0, 5
    _say(f"[whole head] {w.name} B={w.B} H={w.H} L={w.L}: generating inputs on the GPU")
    x = make_inputs(w, "cuda", 0)
    o, do, lse = attn_jvp_fwd(x["Q"], x["K"], x["V"], x["dQ"], x["dK"], x["dV"], w.kind, _offsets(w))
    of, lsef = attn_fwd(x["Q"], x["K"], x["V"], w.kind, _offsets(w))
    torch.cuda.synchronize()
    _say(f"[whole head] kernels done; oracle over all {w.L} rows of head ({b}, {h})")
    sl = {k: _np(v[b:b + 1, h:h + 1]) for k, v in x.items()}
    O, dO, LSE = attention_jvp(sl["Q"], sl["K"], sl["V"], sl["dQ"], sl["dK"], sl["dV"], w.kind, _offsets(w))
    errs = {"O": _rel(_np(o[b, h]), O[0, 0]), "dO": _rel(_np(do[b, h]), dO[0, 0]),
            "LSE": _rel(_np(lse[b, h]), LSE[0, 0]), "fwd O": _rel(_np(of[b, h]), O[0, 0]),
            "fwd LSE": _rel(_np(lsef[b, h]), LSE[0, 0])}
    worst_row = float(np.max(np.linalg.norm(_np(do[b, h]) - dO[0, 0], axis=1) /
                             np.maximum(np.linalg.norm(dO[0, 0], axis=1), 1e-300)))
    _say(f"[whole head] rel-L2 " + " ".join(f"{n}={e:.3e}" for n, e in errs.items()) +
         f"; worst single dO row {worst_row:.3e}")
    assert max(errs.values()) <= TOL["bf16"], errs


# ----------------------------------------------------------------------------- rescale stress

def _scaled_inputs(w, seed, key_gain):
    """Inputs whose key norms grow along the sequence (gain per key position), so that
    the running row maximum keeps increasing and the reference max must move often."""
    x = make_inputs(w, "cpu", seed)
    L = w.L
    g = torch.exp(torch.linspace(0.0, float(np.log(key_gain)), L))[None, None, :, None]
    for k in ("K", "dK"):
        x[k] = (x[k].float() * g).to(x[k].dtype)
    return x


@pytest.mark.parametrize("dt,gain,qscale", [("bf16", 12.0, 1.0), ("bf16", 3.0, 4.0), ("f32", 12.0, 1.0)])
def test_growing_scores_force_rescales(dt, gain, qscale):
    """Scores rise along the keys (up to ~gain x), so blocks keep exceeding the stored
    reference max: exercises the rescale path on every kind of row and block."""
    w = custom_workload(f"rescale_{dt}_{gain}_{qscale}", 1, 2, 128, dt, MASK_TEACHER_FORCING, 3, 130,
                        tangent_std=0.5)
    _say(f"[rescale] {w.name}")
    x = _scaled_inputs(w, 8, gain)
    x["Q"] = (x["Q"].float() * qscale).to(x["Q"].dtype)
    o, do, lse = _run_gpu(w, x)
    O, dO, LSE = attention_jvp(*[_np(x[k]) for k in ("Q", "K", "V", "dQ", "dK", "dV")], w.kind, _offsets(w))
    errs = (_rel(_np(o), O), _rel(_np(do), dO), _rel(_np(lse), LSE))
    _say(f"[rescale] {w.name} rel-L2 O={errs[0]:.3e} dO={errs[1]:.3e} LSE={errs[2]:.3e}")
    assert np.isfinite(_np(o)).all() and np.isfinite(_np(do)).all()
    assert max(errs) <= TOL[dt], errs


def test_full_mask_growing_scores():
    w = custom_workload("rescale_full_bf16", 1, 1, 128, "bf16", MASK_FULL, L=777, tangent_std=0.5)
    _say("[rescale] full mask, growing key norms")
    x = _scaled_inputs(w, 9, 20.0)
    o, do, lse = _run_gpu(w, x)
    O, dO, LSE = attention_jvp(*[_np(x[k]) for k in ("Q", "K", "V", "dQ", "dK", "dV")], w.kind, None)
    errs = (_rel(_np(o), O), _rel(_np(do), dO), _rel(_np(lse), LSE))
    _say(f"[rescale] full rel-L2 O={errs[0]:.3e} dO={errs[1]:.3e} LSE={errs[2]:.3e}")
    assert max(errs) <= TOL["bf16"], errs


# ----------------------------------------------------------------------------- explicit range lists

def _random_ranges(L, G, seed, max_ranges=5):
    """Seeded query groups tiling [0, L), each with 0..max_ranges disjoint key ranges in
    random order (some empty, some touching)."""
    rng = np.random.default_rng(seed)
    cuts = [0] + sorted(int(c) for c in rng.choice(np.arange(1, L), size=G - 1, replace=False)) + [L]
    groups = []
    for q0, q1 in zip(cuts, cuts[1:]):
        n = int(rng.integers(0, max_ranges + 1))
        pts = sorted(int(v) for v in rng.integers(0, L + 1, size=2 * n))
        ks = [(pts[2 * i], pts[2 * i + 1]) for i in range(n)]
        if n >= 2 and rng.random() < 0.3:
            ks[1] = (ks[0][1], max(ks[0][1], ks[1][1]))
        rng.shuffle(ks)
        groups.append((q0, q1, [tuple(k) for k in ks]))
    return groups


def _striped(L, G, stripes, width, seed):
    """Groups of L/G rows, each admitting `stripes` narrow key ranges spread over the whole
    sequence: more separate block runs per query tile than a tile plan holds, so the plan
    merges runs and masks the blocks in between."""
    rng = np.random.default_rng(seed)
    groups = []
    bounds = [round(i * L / G) for i in range(G + 1)]
    for q0, q1 in zip(bounds, bounds[1:]):
        starts = sorted(int(v) for v in rng.choice(np.arange(0, L - width, 2 * width), size=stripes, replace=False))
        groups.append((q0, q1, [(a, a + int(rng.integers(1, width + 1))) for a in starts]))
    return groups


def _check_ranges(w, seed):
    x = make_inputs(w, "cpu", seed)
    o, do, lse = _run_gpu(w, x)
    O, dO, LSE = attention_jvp(*[_np(x[k]) for k in ("Q", "K", "V", "dQ", "dK", "dV")], w.kind, _offsets(w))
    lse_g = _np(lse)
    dead = ~np.isfinite(LSE)
    # rows with no admissible key: O = dO = 0 and LSE = -inf exactly
    assert np.array_equal(np.isneginf(lse_g), dead)
    assert np.all(_np(o)[np.broadcast_to(dead[..., None], O.shape)] == 0)
    assert np.all(_np(do)[np.broadcast_to(dead[..., None], dO.shape)] == 0)
    errs = (_rel(_np(o), O), _rel(_np(do), dO), _rel(lse_g[~dead], LSE[~dead]))
    _say(f"[ranges] {w.name} dead rows={int(dead.sum())} rel-L2 O={errs[0]:.3e} dO={errs[1]:.3e} LSE={errs[2]:.3e}")
    assert max(errs) <= TOL[w.dtype], errs


@pytest.mark.parametrize("dt,D,L,G,seed", [("bf16", 128, 700, 9, 1), ("bf16", 128, 1500, 40, 2),
                                           ("bf16", 64, 333, 5, 3), ("f32", 128, 200, 6, 4),
                                           ("f32", 64, 97, 12, 5), ("bf16", 128, 2100, 25, 6),
                                           ("bf16", 64, 900, 60, 7), ("f32", 128, 300, 30, 8)])
def test_random_range_lists(dt, D, L, G, seed):
    groups = _random_ranges(L, G, seed)
    if seed == 1:
        groups[0] = (groups[0][0], groups[0][1], [])  # guarantee a fully masked group
    if seed == 6:
        groups[1] = (groups[1][0], groups[1][1], [(0, 5), (40, 41), (300, 700), (900, 901), (2000, 2100)])
    w = custom_workload(f"ranges_{dt}_{D}_{L}_{G}", 1, 2, D, dt, "ranges", offsets=groups, tangent_std=0.5)
    _say(f"[ranges] {w.name} groups={groups[:3]}...")
    _check_ranges(w, seed)


@pytest.mark.parametrize("dt,D,L,G,stripes,seed", [("bf16", 128, 3000, 6, 9, 21), ("bf16", 64, 1200, 3, 12, 22),
                                                    ("f32", 128, 700, 4, 7, 23)])
def test_range_lists_with_more_runs_than_a_tile_plan_holds(dt, D, L, G, stripes, seed):
    groups = _striped(L, G, stripes, 40, seed)
    w = custom_workload(f"stripes_{dt}_{D}_{L}_{G}x{stripes}", 1, 2, D, dt, "ranges", offsets=groups,
                        tangent_std=0.5)
    _say(f"[ranges] {w.name} group 0 ranges={groups[0][2]}")
    _check_ranges(w, seed)


def test_ranges_equal_to_tf_layout_match_tf_bitwise():
    """The TF mask given as an explicit group table runs the same schedule, so the
    outputs are bit-identical to the teacher-forcing layout."""
    N, C = 3, 100
    half = N * C
    groups = [(j * C, (j + 1) * C, [(0, (j + 1) * C)]) for j in range(N)]
    groups += [(half + i * C, half + (i + 1) * C, [(0, i * C), (half + i * C, half + (i + 1) * C)]) for i in range(N)]
    w_tf = custom_workload("tf_as_tf", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, N, C, tangent_std=0.5)
    w_rg = custom_workload("tf_as_ranges", 1, 2, 128, "bf16", "ranges", offsets=groups, tangent_std=0.5)
    _say("[ranges] TF table vs TF layout")
    x = make_inputs(w_tf, "cpu", 11)
    a = _run_gpu(w_tf, x)
    b = _run_gpu(w_rg, x)
    for u, v in zip(a, b):
        assert torch.equal(u, v)


def test_wrong_output_tensors_are_refused():
    """Caller-supplied outputs of the wrong shape or dtype raise before the library runs."""
    w = custom_workload("out_check", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 2, 64, tangent_std=0.5)
    g = {k: v.cuda() for k, v in make_inputs(w, "cpu", 3).items()}
    q = g["Q"]
    lse = torch.empty(q.shape[:3], device=q.device)
    for out in [(torch.empty_like(q)[:, :, :-1], torch.empty_like(q), lse),
                (torch.empty_like(q), torch.empty_like(q, dtype=torch.float32), lse),
                (torch.empty_like(q), torch.empty_like(q), lse.to(torch.bfloat16))]:
        with pytest.raises(ValueError):
            attn_jvp_fwd(q, g["K"], g["V"], g["dQ"], g["dK"], g["dV"], w.kind, list(w.offsets), out=out)
    o, do, lse2 = attn_jvp_fwd(q, g["K"], g["V"], g["dQ"], g["dK"], g["dV"], w.kind, list(w.offsets),
                               out=(torch.empty_like(q), torch.empty_like(q), lse))
    torch.cuda.synchronize()
    assert lse2.data_ptr() == lse.data_ptr() and torch.isfinite(o.float()).all()
