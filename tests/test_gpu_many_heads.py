"""The largest head counts the boundary accepts (marked ``gpu``).

B * H = 2^20 (batch 1024 x 1024 heads of 32 tokens, D = 64) in bf16 and in fp32: about a
million work-groups per launch, mapped through the head-group / position order.  The JVP, the forward and the backward are checked
on sampled (batch, head) pairs -- the first, the last, and seeded random ones -- against the
oracle, element by element; every output must be finite.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import attention_fwd, attention_jvp, attention_vjp
from paper_2606_25473_amd import attn_bwd, attn_fwd, attn_jvp_fwd
from paper_2606_25473_amd.workloads import MASK_TEACHER_FORCING, custom_workload, make_inputs

pytestmark = pytest.mark.gpu

TOL = {"bf16": 1e-2, "f32": 1e-4}


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _rel(x, ref):
    return float(np.linalg.norm(np.asarray(x) - np.asarray(ref)) / max(np.linalg.norm(ref), 1e-300))


@pytest.mark.parametrize("dt,B,H,C", [("bf16", 1024, 1024, 8), ("f32", 1024, 1024, 8)])
def test_largest_head_count(dt, B, H, C):
    w = custom_workload(f"many_heads_{dt}", B, H, 64, dt, MASK_TEACHER_FORCING, 2, C, tangent_std=0.5)
    offs = list(w.offsets)
    _say(f"[many-heads] {dt} B={B} H={H} (B*H = {B * H}) L={w.L} D=64: generating inputs on the GPU")
    x = make_inputs(w, "cuda", 61)
    o, do, lse = attn_jvp_fwd(x["Q"], x["K"], x["V"], x["dQ"], x["dK"], x["dV"], w.kind, offs)
    of, lsef = attn_fwd(x["Q"], x["K"], x["V"], w.kind, offs)
    gq, gk, gv, delta = attn_bwd(x["Q"], x["K"], x["V"], o, x["dV"], lse, w.kind, offs)
    torch.cuda.synchronize()
    _say(f"[many-heads] {dt}: kernels done")
    for t in (o, do, lse, of, lsef, gq, gk, gv, delta):
        assert torch.isfinite(t).all()
    rng = np.random.default_rng(6)
    pairs = {(0, 0), (B - 1, H - 1)} | {(int(rng.integers(B)), int(rng.integers(H))) for _ in range(6)}
    errs = []
    for b, h in sorted(pairs):
        s = {k: _np(v[b:b + 1, h:h + 1]) for k, v in x.items()}
        O, dO, LSE = attention_jvp(s["Q"], s["K"], s["V"], s["dQ"], s["dK"], s["dV"], w.kind, offs)
        # the backward from the GPU's own O and LSE of this head, against the oracle's gradient
        rq, rk, rv, rd = attention_vjp(s["Q"], s["K"], s["V"], s["dV"], w.kind, offs)
        errs.append((_rel(_np(o[b, h]), O[0, 0]), _rel(_np(do[b, h]), dO[0, 0]), _rel(_np(lse[b, h]), LSE[0, 0]),
                     _rel(_np(of[b, h]), O[0, 0]), _rel(_np(gq[b, h]), rq[0, 0]), _rel(_np(gk[b, h]), rk[0, 0]),
                     _rel(_np(gv[b, h]), rv[0, 0]), _rel(_np(delta[b, h]), rd[0, 0])))
    worst = np.max(np.array(errs), axis=0)
    _say(f"[many-heads] {dt} {len(pairs)} heads, worst rel-L2 O={worst[0]:.2e} dO={worst[1]:.2e} "
         f"LSE={worst[2]:.2e} fwd O={worst[3]:.2e} gQ={worst[4]:.2e} gK={worst[5]:.2e} gV={worst[6]:.2e} "
         f"Delta={worst[7]:.2e}")
    del x, o, do, lse, of, lsef, gq, gk, gv, delta
    torch.cuda.empty_cache()
    assert worst.max() <= TOL[dt], worst
