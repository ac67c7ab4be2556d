"""A softmax scale other than 1/sqrt(D) on every entry point (marked ``gpu``).

The boundary takes ``softmax_scale`` (<= 0 selects 1/sqrt(D)); the kernels fold it into
the exp2 argument of the scores, into the score tangents and into gQ, gK.  Checked
against the fp64 oracle with the same scale, element by element, for the JVP, the forward,
the zero-clean JVP and the backward, at a small scale (flat softmax), a moderate one and
s = 1 with D = 128 (score standard deviation ~11: nearly one-hot rows, frequent moves of the
reference max).  Tolerance: relative L2 1e-2 for bf16, 1e-4 for fp32.  Also peaked rows
from Q and K drawn with standard deviation 2-3.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import attention_fwd, attention_jvp, attention_jvp_zero_clean, attention_vjp
from paper_2606_25473_amd import attn_bwd, attn_fwd, attn_jvp_fwd, attn_jvp_fwd_zero_clean
from paper_2606_25473_amd.workloads import MASK_TEACHER_FORCING, custom_workload, make_inputs

pytestmark = pytest.mark.gpu

TOL = {"bf16": 1e-2, "f32": 1e-4}
SCALES = [0.05, 0.3, 1.0]


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _rel(x, ref):
    x, ref = np.asarray(x, np.float64), np.asarray(ref, np.float64)
    return float(np.linalg.norm(x - ref) / max(np.linalg.norm(ref), 1e-300))


def _workload(dt):
    return custom_workload(f"scale_{dt}", 1, 2, 128, dt, MASK_TEACHER_FORCING, 3, 100 if dt == "bf16" else 20,
                           tangent_std=0.5)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("s", SCALES)
def test_jvp_and_forward_with_scale(dt, s):
    w = _workload(dt)
    offs = list(w.offsets)
    _say(f"[scale] JVP and forward, {dt}, s = {s}")
    x = make_inputs(w, "cpu", 41)
    g = {k: v.cuda() for k, v in x.items()}
    o, do, lse = attn_jvp_fwd(g["Q"], g["K"], g["V"], g["dQ"], g["dK"], g["dV"], w.kind, offs, scale=s)
    of, lsef = attn_fwd(g["Q"], g["K"], g["V"], w.kind, offs, scale=s)
    torch.cuda.synchronize()
    xs = [_np(x[k]) for k in ("Q", "K", "V", "dQ", "dK", "dV")]
    O, dO, LSE = attention_jvp(*xs, w.kind, offs, scale=s)
    errs = (_rel(_np(o), O), _rel(_np(do), dO), _rel(_np(lse), LSE), _rel(_np(of), O), _rel(_np(lsef), LSE))
    _say(f"[scale] {dt} s={s} rel-L2 O={errs[0]:.2e} dO={errs[1]:.2e} LSE={errs[2]:.2e} "
         f"fwd O={errs[3]:.2e} fwd LSE={errs[4]:.2e}")
    assert max(errs) <= TOL[dt], errs


@pytest.mark.parametrize("s", SCALES)
def test_zero_clean_with_scale(s):
    w = _workload("bf16")
    offs = list(w.offsets)
    half = w.L // 2
    _say(f"[scale] zero-clean JVP, s = {s}")
    x = make_inputs(w, "cpu", 42)
    tn = {k: x[k][:, :, half:].contiguous() for k in ("dQ", "dK", "dV")}
    o, don, lse = attn_jvp_fwd_zero_clean(x["Q"].cuda(), x["K"].cuda(), x["V"].cuda(), tn["dQ"].cuda(),
                                          tn["dK"].cuda(), tn["dV"].cuda(), offs, scale=s)
    torch.cuda.synchronize()
    O, dO, LSE = attention_jvp_zero_clean(*[_np(t) for t in (x["Q"], x["K"], x["V"], tn["dQ"], tn["dK"], tn["dV"])],
                                          offs, scale=s)
    errs = (_rel(_np(o), O), _rel(_np(don), dO[:, :, half:]), _rel(_np(lse), LSE))
    _say(f"[scale] zero-clean s={s} rel-L2 O={errs[0]:.2e} dOn={errs[1]:.2e} LSE={errs[2]:.2e}")
    assert max(errs) <= TOL["bf16"], errs


@pytest.mark.parametrize("dt", ["bf16", "f32"])
@pytest.mark.parametrize("s", SCALES)
def test_backward_with_scale(dt, s):
    w = _workload(dt)
    offs = list(w.offsets)
    _say(f"[scale] backward, {dt}, s = {s}")
    x = make_inputs(w, "cpu", 43)
    q, k, v, go = x["Q"], x["K"], x["V"], x["dV"]
    O, LSE = attention_fwd(_np(q), _np(k), _np(v), w.kind, offs, scale=s)
    o = torch.from_numpy(O).to(q.dtype)
    lse = torch.from_numpy(LSE).float()
    gq, gk, gv, delta = attn_bwd(q.cuda(), k.cuda(), v.cuda(), o.cuda(), go.cuda(), lse.cuda(), w.kind, offs,
                                 scale=s)
    torch.cuda.synchronize()
    rq, rk, rv, rd = attention_vjp(_np(q), _np(k), _np(v), _np(go), w.kind, offs, scale=s)
    errs = (_rel(_np(gq), rq), _rel(_np(gk), rk), _rel(_np(gv), rv), _rel(_np(delta), rd))
    _say(f"[scale] backward {dt} s={s} rel-L2 gQ={errs[0]:.2e} gK={errs[1]:.2e} gV={errs[2]:.2e} "
         f"Delta={errs[3]:.2e}")
    assert max(errs) <= TOL[dt], errs


# Peaked rows (the stress variant of Q and K drawn with standard deviation 2-3, and a softmax
# scale of 1): the tangent dO = (T - r O) / l subtracts nearly equal terms there, which
# magnifies the bf16 rounding of H~; the errors stay inside the bf16 bar.


def _peaked_inputs(w, seed, qk_std):
    x = make_inputs(w, "cpu", seed)
    for k in ("Q", "K"):
        x[k] = (x[k].float() * qk_std).to(x[k].dtype)
    return x


@pytest.mark.parametrize("qk_std,s", [(1.0, 1.0), (2.5, None), (3.0, None), (2.0, 0.3)])
def test_peaked_rows_tangent_error(qk_std, s):
    w = _workload("bf16")
    offs = list(w.offsets)
    half = w.L // 2
    _say(f"[peaked] Q, K std {qk_std}, scale {s or '1/sqrt(D)'}")
    x = _peaked_inputs(w, 44, qk_std)
    g = {k: v.cuda() for k, v in x.items()}
    o, do, lse = attn_jvp_fwd(g["Q"], g["K"], g["V"], g["dQ"], g["dK"], g["dV"], w.kind, offs, scale=s)
    tn = [g[k][:, :, half:].contiguous() for k in ("dQ", "dK", "dV")]
    oz, don, lsez = attn_jvp_fwd_zero_clean(g["Q"], g["K"], g["V"], *tn, offs, scale=s)
    torch.cuda.synchronize()
    xs = [_np(x[k]) for k in ("Q", "K", "V", "dQ", "dK", "dV")]
    O, dO, LSE = attention_jvp(*xs, w.kind, offs, scale=s)
    xz = xs[:3] + [t[:, :, half:] for t in xs[3:]]
    Oz, dOz, LSEz = attention_jvp_zero_clean(*xz, offs, scale=s)
    errs = (_rel(_np(o), O), _rel(_np(do), dO), _rel(_np(lse), LSE), _rel(_np(don), dOz[:, :, half:]),
            _rel(_np(oz), Oz))
    _say(f"[peaked] std {qk_std} s={s} rel-L2 O={errs[0]:.2e} dO={errs[1]:.2e} LSE={errs[2]:.2e} "
         f"zero-clean dOn={errs[3]:.2e} O={errs[4]:.2e}")
    assert max(errs) <= TOL["bf16"], errs
