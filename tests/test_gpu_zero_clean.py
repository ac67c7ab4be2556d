"""GPU tests of the zero-clean-tangent JVP (marked ``gpu``).

attn_jvp_fwd_zero_clean takes the tangents of the noisy half of a teacher-forcing
sequence only (the clean context has zero tangent, paper Sec. 3.1.2).  Checked:

* parity with the fp64 oracle (oracle.attention_jvp_zero_clean) over every output,
  rel-L2 <= 1e-2 (bf16) / 1e-4 (fp32), on shapes with ragged tails, tiles and key
  blocks straddling the clean/noisy boundary, one-token and single chunks, D = 64;
* equality with the dense attn_jvp_fwd on the zero-padded tangents: the variant
  only skips products with exact zeros, so O, LSE and the noisy dO must be equal
  value for value, and the dense kernel's clean dO must be exactly zero;
* the same at the full Wan2.1-1.3B chunk-wise size (plus sampled oracle rows),
  under growing scores (rescale path), and run-to-run determinism.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import attention_jvp_zero_clean
from paper_2606_25473_amd import attn_jvp_fwd, attn_jvp_fwd_zero_clean
from paper_2606_25473_amd.workloads import MASK_TEACHER_FORCING, WORKLOADS, custom_workload, make_inputs

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


def _noisy(x):
    """(Q, K, V, dQn, dKn, dVn): the tangents cut to the noisy half."""
    half = x["Q"].shape[2] // 2
    return (x["Q"], x["K"], x["V"]) + tuple(x[k][:, :, half:].contiguous() for k in ("dQ", "dK", "dV"))


def _padded(x):
    """The dense tangents with the clean half set to zero."""
    half = x["Q"].shape[2] // 2
    out = dict(x)
    for k in ("dQ", "dK", "dV"):
        t = x[k].clone()
        t[:, :, :half] = 0
        out[k] = t
    return out


SHAPES = [
    custom_workload("zc_ragged_bf16", 2, 2, 128, "bf16", MASK_TEACHER_FORCING, 3, 100, tangent_std=0.5),
    custom_workload("zc_several_tiles_bf16", 1, 3, 128, "bf16", MASK_TEACHER_FORCING, 4, 300, tangent_std=0.5),
    custom_workload("zc_six_heads_bf16", 2, 3, 128, "bf16", MASK_TEACHER_FORCING, 3, 150, tangent_std=0.5),
    custom_workload("zc_tile_aligned_bf16", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 4, 128, tangent_std=0.5),
    custom_workload("zc_one_token_chunks_bf16", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 64, 1, tangent_std=0.5),
    custom_workload("zc_one_chunk_bf16", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 1, 300, tangent_std=0.5),
    custom_workload("zc_nonuniform_bf16", 1, 2, 128, "bf16", MASK_TEACHER_FORCING,
                    offsets=[0, 1, 3, 7, 40, 41, 90, 200], tangent_std=0.5),
    custom_workload("zc_d64_bf16", 1, 2, 64, "bf16", MASK_TEACHER_FORCING, 4, 50, tangent_std=0.5),
    custom_workload("zc_f32_d128", 1, 2, 128, "f32", MASK_TEACHER_FORCING, 3, 20),
    custom_workload("zc_f32_d64", 2, 1, 64, "f32", MASK_TEACHER_FORCING, offsets=[0, 5, 6, 30]),
    # t0 = L/2 inside a 32-key block and a 128-row tile of the fp32 kernel, and on their bounds
    custom_workload("zc_ragged_f32", 2, 2, 128, "f32", MASK_TEACHER_FORCING, 3, 100),
    custom_workload("zc_tile_aligned_f32", 1, 2, 128, "f32", MASK_TEACHER_FORCING, 4, 128),
    custom_workload("zc_nonuniform_f32", 1, 2, 64, "f32", MASK_TEACHER_FORCING, offsets=[0, 1, 3, 7, 40, 41, 90, 200]),
]


def _check_oracle(w, x, o, don, lse):
    O, dO, LSE = attention_jvp_zero_clean(*[_np(t) for t in _noisy(x)], list(w.offsets))
    half = w.L // 2
    errs = (_rel(_np(o), O), _rel(_np(don), dO[:, :, half:]), _rel(_np(lse), LSE))
    _say(f"[zero-clean] {w.name} rel-L2 O={errs[0]:.3e} dOn={errs[1]:.3e} LSE={errs[2]:.3e}")
    assert max(errs) <= TOL[w.dtype], errs


def _check_dense_equal(w, x, o, don, lse):
    p = {k: v.cuda() for k, v in _padded(x).items()}
    o2, do2, lse2 = attn_jvp_fwd(p["Q"], p["K"], p["V"], p["dQ"], p["dK"], p["dV"], w.kind, list(w.offsets))
    torch.cuda.synchronize()
    half = w.L // 2
    assert torch.equal(o, o2), "O differs from the dense kernel"
    assert torch.equal(lse, lse2), "LSE differs from the dense kernel"
    assert torch.equal(don, do2[:, :, half:]), "noisy dO differs from the dense kernel"
    assert (do2[:, :, :half] == 0).all(), "dense kernel: clean dO is not exactly zero"


@pytest.mark.parametrize("w", SHAPES, ids=[w.name for w in SHAPES])
def test_zero_clean_vs_oracle_and_dense(w):
    _say(f"[zero-clean] {w.name} B={w.B} H={w.H} L={w.L} D={w.D} {w.dtype} offsets={list(w.offsets)[:6]}")
    x = make_inputs(w, "cpu", 5)
    g = [t.cuda() for t in _noisy(x)]
    o, don, lse = attn_jvp_fwd_zero_clean(*g, list(w.offsets))
    torch.cuda.synchronize()
    assert don.shape == (w.B, w.H, w.L - w.L // 2, w.D)
    _check_oracle(w, x, o, don, lse)
    _check_dense_equal(w, {k: v.cuda() for k, v in x.items()}, o, don, lse)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_zero_clean_growing_scores(dt):
    """Key norms grow along the sequence (x12), so blocks keep raising the row max:
    the rescale path in both the primal-only and the tangent tiles."""
    w = custom_workload(f"zc_rescale_{dt}", 1, 2, 128, dt, MASK_TEACHER_FORCING, 3, 130, tangent_std=0.5)
    _say(f"[zero-clean] {w.name}: growing key norms")
    x = make_inputs(w, "cpu", 8)
    gain = torch.exp(torch.linspace(0.0, float(np.log(12.0)), w.L))[None, None, :, None]
    for k in ("K", "dK"):
        x[k] = (x[k].float() * gain).to(x[k].dtype)
    g = [t.cuda() for t in _noisy(x)]
    o, don, lse = attn_jvp_fwd_zero_clean(*g, list(w.offsets))
    torch.cuda.synchronize()
    _check_oracle(w, x, o, don, lse)
    _check_dense_equal(w, {k: v.cuda() for k, v in x.items()}, o, don, lse)


def test_zero_clean_deterministic():
    w = custom_workload("zc_determinism", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 4, 300, tangent_std=0.5)
    _say("[zero-clean] run-to-run determinism")
    g = [t.cuda() for t in _noisy(make_inputs(w, "cpu", 6))]
    a = attn_jvp_fwd_zero_clean(*g, list(w.offsets))
    b = attn_jvp_fwd_zero_clean(*g, list(w.offsets))
    torch.cuda.synchronize()
    for u, v in zip(a, b):
        assert torch.equal(u, v)


@pytest.mark.parametrize("name,nheads", [("wan1.3b_chunkwise_tf", 4), ("wan1.3b_framewise_tf", 4),
                                         ("wan14b_chunkwise_tf", 8)])
def test_zero_clean_full_size(name, nheads):
    """The Wan-shaped workloads (L = 65520, D = 128, bf16) in the launch configuration the
    bench times: equal to the dense kernel on zero-padded tangents over the whole tensors,
    and sampled rows of both halves (every tile boundary and chunk boundary) of spread
    heads against the oracle."""
    w = WORKLOADS[name]
    _say(f"[zero-clean] full size {w.name} B={w.B} H={w.H}: generating inputs on the GPU")
    x = make_inputs(w, "cuda", 0)
    g = _noisy(x)
    o, don, lse = attn_jvp_fwd_zero_clean(*g, list(w.offsets))
    torch.cuda.synchronize()
    _say("[zero-clean] full size: kernel done, comparing with the dense kernel")
    assert torch.isfinite(o).all() and torch.isfinite(don).all() and torch.isfinite(lse).all()
    _check_dense_equal(w, x, o, don, lse)
    del x
    half = w.L // 2
    rows = sorted({0, half - 1, half, half + 1, w.L - 1} |
                  {t for t in range(0, w.L, 128)} | {min(w.L, t + 128) - 1 for t in range(0, w.L, 128)} |
                  {half + o_ + d for o_ in w.offsets[1:-1] for d in (-1, 0)} |
                  {o_ + d for o_ in w.offsets[1:-1] for d in (-1, 0)} |
                  set(int(r) for r in np.random.default_rng(0).integers(0, w.L, 16)))
    rows = np.array(rows)
    ridx = torch.from_numpy(rows).cuda()
    pairs = [(b, h) for b in range(w.B) for h in range(w.H)]
    heads = [pairs[i] for i in np.unique(np.linspace(0, len(pairs) - 1, nheads).round().astype(int))]
    for b, h in heads:
        sl = [_np(t[b:b + 1, h:h + 1]) for t in g]
        O, dO, LSE = attention_jvp_zero_clean(*sl, list(w.offsets), rows=rows)
        noisy = rows >= half
        got_do = _np(don[b, h].index_select(0, torch.from_numpy(rows[noisy] - half).cuda()))
        errs = (_rel(_np(o[b, h].index_select(0, ridx)), O[0, 0]), _rel(got_do, dO[0, 0][noisy]),
                _rel(_np(lse[b, h].index_select(0, ridx)), LSE[0, 0]))
        assert np.all(dO[0, 0][~noisy] == 0.0)
        _say(f"[zero-clean] full size (b={b}, h={h}) {len(rows)} rows rel-L2 O={errs[0]:.3e} "
             f"dOn={errs[1]:.3e} LSE={errs[2]:.3e}")
        assert max(errs) <= TOL["bf16"], errs
