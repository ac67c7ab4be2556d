"""fp32 at full size (marked ``gpu``): the Wan2.1-1.3B chunk-wise teacher-forcing and
bidirectional shapes (B = 1, H = 12, D = 128, L = 65520 / 32760) with fp32 inputs.

The JVP, the forward and the backward run over every head; sampled query rows (every
128-row tile boundary of the fp32 kernels, the chunk boundaries, seeded random rows) of O,
dO, LSE, gQ and Delta, and sampled keys of gK and gV, are compared with the fp64 oracle on
two heads, element by element, at the fp32 bar (relative L2 1e-4).
"""
import sys

import numpy as np
import pytest
import torch

from oracle import attention_jvp, attention_vjp
from paper_2606_25473_amd import attn_bwd, attn_fwd, attn_jvp_fwd
from paper_2606_25473_amd.workloads import MASK_FULL, MASK_TEACHER_FORCING, WORKLOADS, custom_workload, make_inputs

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _rel(x, ref):
    return float(np.linalg.norm(np.asarray(x) - np.asarray(ref)) / max(np.linalg.norm(ref), 1e-300))


def _fp32_copy(name):
    w = WORKLOADS[name]
    return custom_workload(name + "_f32", w.B, w.H, w.D, "f32", w.kind, offsets=list(w.offsets) or None,
                           L=w.L_full, tangent_std=w.tangent_std)


def _rows(w, rng):
    L = w.L
    rows = {0, L - 1}
    for t in range(0, L, 128):  # the fp32 kernels' query tiles
        rows.update((t, min(L, t + 128) - 1))
    if w.kind == MASK_TEACHER_FORCING:
        half = w.offsets[-1]
        for o in w.offsets:
            for base in (0, half):
                rows.update(r for r in (base + o - 1, base + o) if 0 <= r < L)
    rows.update(int(r) for r in rng.integers(0, L, 16))
    return np.array(sorted(rows))


def _keys(w, rng):
    """Keys whose gradients the oracle forms from few rows (see the bf16 full-size test):
    teacher forcing, the last clean chunk and the first noisy chunk; full mask, any key."""
    L = w.L
    if w.kind == MASK_FULL:
        return np.unique(np.concatenate([[0, 127, 128, L // 2, L - 1], rng.integers(0, L, 9)]))
    offs = list(w.offsets)
    half = L // 2
    pools = [np.arange(offs[-2], half), half + np.arange(offs[0], offs[1])]
    return np.unique(np.concatenate([[offs[-2], half - 1, half, half + offs[1] - 1]] +
                                    [rng.choice(p, 6) for p in pools]))


@pytest.mark.parametrize("name,heads", [("wan1.3b_chunkwise_tf", ((0, 0), (0, 11))),
                                        ("wan1.3b_bidirectional", ((0, 6),))])
def test_f32_full_size_sampled(name, heads):
    w = _fp32_copy(name)
    offs = list(w.offsets) or None
    _say(f"[f32 full size] {w.name} B={w.B} H={w.H} L={w.L}: generating inputs on the GPU")
    x = make_inputs(w, "cuda", 3)
    q, k, v, dq, dk, dv = (x[n] for n in ("Q", "K", "V", "dQ", "dK", "dV"))
    assert q.dtype == torch.float32
    o, do, lse = attn_jvp_fwd(q, k, v, dq, dk, dv, w.kind, offs)
    of, lsef = attn_fwd(q, k, v, w.kind, offs)
    gq, gk, gv, delta = attn_bwd(q, k, v, of, dv, lsef, w.kind, offs)  # cotangent: the dV draw
    torch.cuda.synchronize()
    _say(f"[f32 full size] {w.name}: kernels done, checking sampled rows and keys")
    for t in (o, do, lse, of, lsef, gq, gk, gv, delta):
        assert torch.isfinite(t).all()
    rng = np.random.default_rng(1)
    rows, keys = _rows(w, rng), _keys(w, rng)
    ri, ki = torch.from_numpy(rows).cuda(), torch.from_numpy(keys).cuda()
    for b, h in heads:
        s = {n: _np(t[b:b + 1, h:h + 1]) for n, t in x.items()}
        O, dO, LSE = attention_jvp(s["Q"], s["K"], s["V"], s["dQ"], s["dK"], s["dV"], w.kind, offs, rows=rows)
        rq, rk, rv, rd = attention_vjp(s["Q"], s["K"], s["V"], s["dV"], w.kind, offs, rows=rows, keys=keys)
        sel = lambda t, idx: _np(t[b, h].index_select(0, idx))  # noqa: E731
        errs = {"O": _rel(sel(o, ri), O[0, 0]), "dO": _rel(sel(do, ri), dO[0, 0]), "LSE": _rel(sel(lse, ri), LSE[0, 0]),
                "fwd O": _rel(sel(of, ri), O[0, 0]), "fwd LSE": _rel(sel(lsef, ri), LSE[0, 0]),
                "gQ": _rel(sel(gq, ri), rq[0, 0]), "Delta": _rel(sel(delta, ri), rd[0, 0]),
                "gK": _rel(sel(gk, ki), rk[0, 0]), "gV": _rel(sel(gv, ki), rv[0, 0])}
        _say(f"[f32 full size] (b={b}, h={h}) {len(rows)} rows / {len(keys)} keys rel-L2 " +
             " ".join(f"{n}={e:.2e}" for n, e in errs.items()))
        assert max(errs.values()) <= TOL, errs
