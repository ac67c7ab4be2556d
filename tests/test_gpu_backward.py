"""GPU parity of the masked-attention backward (attn_bwd) against the fp64 oracle (marked ``gpu``).

O and LSE fed to the kernels come from the oracle's forward (O rounded to the input
dtype, LSE in fp32), so these tests isolate the backward; one test chains the HIP
forward into the HIP backward.  Outputs gQ, gK, gV and Delta are compared by relative
L2 error over every element (<= 1e-2 for bf16, <= 1e-4 for fp32; a reference whose
norm is below 1e-3 of the cotangent's, as for L = 1 where gQ = gK = 0, is compared
against that floor) on shapes with
ragged tails, several key tiles and query blocks, one-token and single chunks, D = 64,
block-causal, full and explicit range masks (including rows with no key and keys no
row sees); the full Wan2.1-1.3B chunk-wise workload is checked on sampled rows and
keys; and two launches must agree bit for bit.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import attention_fwd, attention_vjp
from paper_2606_25473_amd import attn_bwd, attn_fwd
from paper_2606_25473_amd.workloads import (MASK_BLOCK_CAUSAL, MASK_FULL, MASK_RANGES, MASK_TEACHER_FORCING,
                                            WORKLOADS, custom_workload, make_inputs)

pytestmark = pytest.mark.gpu

TOL = {"bf16": 1e-2, "f32": 1e-4}


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def _rel(x, ref, floor=1e-300):
    """||x - ref|| / ||ref||, with ||ref|| floored (gradients that vanish exactly, as gQ
    and gK do for a row with one key, are compared against the cotangent's scale)."""
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(x - ref) / max(np.linalg.norm(ref), floor))


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _offsets(w):
    return list(w.offsets) if w.kind == MASK_RANGES else (list(w.offsets) if w.offsets else None)


def _inputs(w, seed):
    """Q, K, V, gO (the dV draw of the seeded recipe serves as the cotangent)."""
    x = make_inputs(w, "cpu", seed)
    return x["Q"], x["K"], x["V"], x["dV"]


def _oracle_fwd(w, q, k, v):
    O, LSE = attention_fwd(_np(q), _np(k), _np(v), w.kind, _offsets(w))
    return torch.from_numpy(O).to(q.dtype), torch.from_numpy(LSE).float()


SHAPES = [
    custom_workload("bwd_tiny_tf_f32", 1, 2, 64, "f32", MASK_TEACHER_FORCING, 4, 16),
    custom_workload("bwd_tf_f32_d128", 1, 2, 128, "f32", MASK_TEACHER_FORCING, 3, 20),
    custom_workload("bwd_tf_ragged_bf16", 2, 2, 128, "bf16", MASK_TEACHER_FORCING, 3, 100, tangent_std=0.5),
    custom_workload("bwd_tf_several_tiles_bf16", 1, 3, 128, "bf16", MASK_TEACHER_FORCING, 4, 300, tangent_std=0.5),
    custom_workload("bwd_tf_five_heads_bf16", 1, 5, 128, "bf16", MASK_TEACHER_FORCING, 3, 150, tangent_std=0.5),
    custom_workload("bwd_tf_one_token_chunks_bf16", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 64, 1,
                    tangent_std=0.5),
    custom_workload("bwd_tf_one_chunk_bf16", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 1, 300, tangent_std=0.5),
    custom_workload("bwd_tf_nonuniform_bf16", 1, 2, 128, "bf16", MASK_TEACHER_FORCING,
                    offsets=[0, 1, 3, 7, 40, 41, 90, 200], tangent_std=0.5),
    custom_workload("bwd_tf_d64_bf16", 1, 2, 64, "bf16", MASK_TEACHER_FORCING, 4, 50, tangent_std=0.5),
    custom_workload("bwd_block_causal_bf16", 1, 2, 128, "bf16", MASK_BLOCK_CAUSAL,
                    offsets=[0, 50, 77, 200, 333], tangent_std=0.5),
    custom_workload("bwd_full_1000_bf16", 1, 2, 128, "bf16", MASK_FULL, L=1000, tangent_std=0.5),
    custom_workload("bwd_full_below_one_tile_bf16", 1, 1, 128, "bf16", MASK_FULL, L=7, tangent_std=0.5),
    custom_workload("bwd_full_single_token_bf16", 1, 1, 128, "bf16", MASK_FULL, L=1, tangent_std=0.5),
    custom_workload("bwd_full_d64_f32", 1, 2, 64, "f32", MASK_FULL, L=50),
    custom_workload("bwd_tf_ragged_f32", 2, 2, 128, "f32", MASK_TEACHER_FORCING, 3, 100),
    custom_workload("bwd_tf_several_tiles_f32", 1, 3, 64, "f32", MASK_TEACHER_FORCING, 4, 300),
    custom_workload("bwd_tf_nonuniform_f32", 1, 2, 128, "f32", MASK_TEACHER_FORCING, offsets=[0, 1, 3, 7, 40, 41, 90, 200]),
    custom_workload("bwd_block_causal_f32", 1, 2, 128, "f32", MASK_BLOCK_CAUSAL, offsets=[0, 50, 77, 200, 333]),
    custom_workload("bwd_full_below_one_tile_f32", 1, 1, 128, "f32", MASK_FULL, L=7),
    custom_workload("bwd_full_single_token_f32", 1, 1, 64, "f32", MASK_FULL, L=1),
    # rows 100..149 see no key; keys 450..499 are seen by no row
    custom_workload("bwd_ranges_bf16", 1, 2, 128, "bf16", MASK_RANGES,
                    offsets=[(0, 100, [(0, 100), (300, 350)]), (100, 150, []), (150, 400, [(0, 450)]),
                             (400, 500, [(100, 200)])], tangent_std=0.5),
    custom_workload("bwd_ranges_f32", 1, 1, 64, "f32", MASK_RANGES,
                    offsets=[(0, 10, [(0, 10), (30, 35)]), (10, 15, []), (15, 40, [(0, 20)])]),
    # several key ranges per group (touching, out of order), a group admitted by keys that
    # three separate query runs see
    custom_workload("bwd_ranges_many_bf16", 1, 2, 128, "bf16", MASK_RANGES,
                    offsets=[(0, 300, [(0, 40), (100, 101), (500, 700), (900, 1000)]), (300, 333, []),
                             (333, 700, [(950, 1000), (0, 40), (40, 80), (600, 650)]),
                             (700, 1000, [(0, 1), (200, 260), (690, 1000)])], tangent_std=0.5),
    custom_workload("bwd_ranges_many_d64_bf16", 1, 2, 64, "bf16", MASK_RANGES,
                    offsets=[(0, 64, [(0, 10), (64, 65), (128, 130)]), (64, 128, [(0, 10)]),
                             (128, 200, [(0, 10), (120, 200)])], tangent_std=0.5),
    custom_workload("bwd_ranges_many_f32", 1, 1, 128, "f32", MASK_RANGES,
                    offsets=[(0, 20, [(0, 3), (5, 8), (30, 40)]), (20, 30, [(0, 3)]), (30, 60, [(0, 60)])]),
]


def _check(w, q, k, v, go, o, lse, label):
    g = [t.cuda() for t in (q, k, v, o, go)]
    gq, gk, gv, delta = attn_bwd(*g, lse.cuda(), w.kind, _offsets(w))
    torch.cuda.synchronize()
    ref = attention_vjp(_np(q), _np(k), _np(v), _np(go), w.kind, _offsets(w))
    floor = 1e-3 * float(np.linalg.norm(_np(go)))
    errs = [_rel(_np(a), b, floor) for a, b in zip((gq, gk, gv, delta), ref)]
    _say(f"[backward] {w.name} {label} rel-L2 gQ={errs[0]:.3e} gK={errs[1]:.3e} gV={errs[2]:.3e} "
         f"Delta={errs[3]:.3e}")
    for t in (gq, gk, gv, delta):
        assert torch.isfinite(t).all()
    assert max(errs) <= TOL[w.dtype], errs
    return gq, gk, gv, delta, ref


def _random_groups(L, G, seed, max_ranges=5):
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


def _striped_groups(L, G, stripes, width, seed):
    """Groups of L/G rows, each admitting `stripes` narrow key ranges spread over the
    sequence: more separate runs per key tile than a plan holds (merged and masked)."""
    rng = np.random.default_rng(seed)
    bounds = [round(i * L / G) for i in range(G + 1)]
    return [(q0, q1, [(a, a + int(rng.integers(1, width + 1)))
                      for a in sorted(int(v) for v in rng.choice(np.arange(0, L - width, 2 * width), size=stripes,
                                                                   replace=False))])
            for q0, q1 in zip(bounds, bounds[1:])]


@pytest.mark.parametrize("dt,D,L,G,seed,stripes", [("bf16", 128, 700, 9, 31, 0), ("bf16", 64, 1500, 40, 32, 0),
                                                   ("bf16", 128, 2100, 25, 35, 0), ("f32", 128, 300, 12, 33, 0),
                                                   ("f32", 64, 500, 30, 34, 0), ("bf16", 128, 3000, 6, 36, 9),
                                                   ("f32", 128, 900, 4, 37, 7)])
def test_backward_random_range_lists(dt, D, L, G, seed, stripes):
    """Seeded random range-list masks (fully masked groups, keys no row sees, touching and
    unsorted ranges; or striped groups with more runs per tile than a plan holds)."""
    groups = _striped_groups(L, G, stripes, 40, seed) if stripes else _random_groups(L, G, seed)
    w = custom_workload(f"bwd_random_ranges_{dt}_{D}_{L}_{G}_{seed}", 1, 2, D, dt, MASK_RANGES, offsets=groups,
                        tangent_std=0.5)
    _say(f"[backward] {w.name} groups={groups[:2]}...")
    q, k, v, go = _inputs(w, seed)
    o, lse = _oracle_fwd(w, q, k, v)
    _check(w, q, k, v, go, o, lse, "oracle O/LSE")


@pytest.mark.parametrize("w", SHAPES, ids=[w.name for w in SHAPES])
def test_backward_vs_oracle(w):
    _say(f"[backward] {w.name} B={w.B} H={w.H} L={w.L} D={w.D} {w.dtype} {w.kind}")
    q, k, v, go = _inputs(w, 11)
    o, lse = _oracle_fwd(w, q, k, v)
    gq, gk, gv, delta, ref = _check(w, q, k, v, go, o, lse, "oracle O/LSE")
    if w.kind == MASK_RANGES:
        # fully masked rows and unseen keys get exactly zero
        m = np.zeros(w.L, dtype=bool)
        for q0g, q1g, ks in w.offsets:
            if all(k1 == k0 for k0, k1 in ks):
                m[q0g:q1g] = True
        assert (gq[:, :, torch.from_numpy(np.flatnonzero(m)).cuda()] == 0).all()
        unseen = np.flatnonzero(~np.abs(ref[2]).sum(axis=(0, 1, 3)).astype(bool))
        if unseen.size:
            idx = torch.from_numpy(unseen).cuda()
            assert (gk[:, :, idx] == 0).all() and (gv[:, :, idx] == 0).all()


def test_backward_after_hip_forward():
    """The HIP forward's O and LSE feed the HIP backward (the training pipeline)."""
    w = custom_workload("bwd_chain_bf16", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 4, 300, tangent_std=0.5)
    _say("[backward] chained after attn_fwd")
    q, k, v, go = _inputs(w, 12)
    o, lse = attn_fwd(q.cuda(), k.cuda(), v.cuda(), w.kind, list(w.offsets))
    torch.cuda.synchronize()
    _check(w, q, k, v, go, o.cpu(), lse.cpu(), "HIP O/LSE")


def test_backward_deterministic():
    w = custom_workload("bwd_determinism", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 4, 300, tangent_std=0.5)
    _say("[backward] run-to-run determinism")
    q, k, v, go = _inputs(w, 13)
    o, lse = _oracle_fwd(w, q, k, v)
    g = [t.cuda() for t in (q, k, v, o, go)] + [lse.cuda()]
    a = attn_bwd(*g, w.kind, list(w.offsets))
    b = attn_bwd(*g, w.kind, list(w.offsets))
    torch.cuda.synchronize()
    for u, t in zip(a, b):
        assert torch.equal(u, t)


def _cheap_keys(w, rng):
    """Keys whose gradients the oracle can form from few query rows: for teacher forcing,
    the last clean chunk (seen by its own clean rows only) and the first noisy chunk (seen
    by its own noisy rows, which admit no other key); for the full mask any key (every row
    sees it, so the oracle runs the whole head once)."""
    L = w.L
    if w.kind == MASK_FULL:
        return np.unique(np.concatenate([[0, L // 2, L - 1], rng.integers(0, L, 9)]))
    offs = list(w.offsets)
    half = L // 2
    pools = [np.arange(offs[-2], half), half + np.arange(offs[0], offs[1])]
    return np.unique(np.concatenate([[offs[-2], half - 1, half, half + offs[1] - 1]] +
                                    [rng.choice(p, 6) for p in pools]))


@pytest.mark.parametrize("name,heads", [("wan1.3b_chunkwise_tf", ((0, 0), (0, 11))),
                                        ("wan1.3b_framewise_tf", ((0, 5),)),
                                        ("wan1.3b_bidirectional", ((0, 7),)),
                                        ("wan14b_chunkwise_tf", ((0, 3), (1, 39)))])
def test_backward_full_size_sampled(name, heads):
    """The Wan-shaped workloads (bf16, D = 128) in the launch configuration the bench
    times: HIP forward, then backward; sampled rows of gQ and Delta (tile and chunk
    boundaries included) and sampled keys of gK, gV against the oracle."""
    w = WORKLOADS[name]
    _say(f"[backward] full size {w.name} B={w.B} H={w.H} L={w.L}: generating inputs on the GPU")
    x = make_inputs(w, "cuda", 0)
    q, k, v, go = x["Q"], x["K"], x["V"], x["dV"]
    offs = list(w.offsets) if w.offsets else None
    o, lse = attn_fwd(q, k, v, w.kind, offs)
    gq, gk, gv, delta = attn_bwd(q, k, v, o, go, lse, w.kind, offs)
    torch.cuda.synchronize()
    _say("[backward] full size: kernels done, checking sampled rows and keys")
    for t in (gq, gk, gv, delta):
        assert torch.isfinite(t).all()
    rng = np.random.default_rng(0)
    half = w.L // 2
    rows = np.unique(np.concatenate([[0, half - 1, half, w.L - 1], np.arange(0, w.L, 256 * 16),
                                     np.arange(255, w.L, 256 * 16), rng.integers(0, w.L, 16)]))
    keys = _cheap_keys(w, rng)
    for b, h in heads:
        sl = [_np(t[b:b + 1, h:h + 1]) for t in (q, k, v, go)]
        rq, rk, rv, rd = attention_vjp(*sl, w.kind, offs, rows=rows, keys=keys)
        ri, ki = torch.from_numpy(rows).cuda(), torch.from_numpy(keys).cuda()
        errs = (_rel(_np(gq[b, h].index_select(0, ri)), rq[0, 0]), _rel(_np(gk[b, h].index_select(0, ki)), rk[0, 0]),
                _rel(_np(gv[b, h].index_select(0, ki)), rv[0, 0]), _rel(_np(delta[b, h].index_select(0, ri)), rd[0, 0]))
        _say(f"[backward] full size (b={b}, h={h}) {len(rows)} rows / {len(keys)} keys rel-L2 gQ={errs[0]:.3e} "
             f"gK={errs[1]:.3e} gV={errs[2]:.3e} Delta={errs[3]:.3e}")
        assert max(errs) <= TOL["bf16"], errs
