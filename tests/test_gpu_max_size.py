"""The largest heads the boundary accepts (marked ``gpu``).

The kernels address a head with 32-bit byte offsets, and the boundary admits L * D up to
2^31 in bf16 and 2^30 in fp32: L = 2^24 (bf16) or 2^23 (fp32) tokens at D = 128, where key
and query rows near the end lie within 512 bytes of the 4 GiB limit.  Attention over the
whole sequence at that length is far too slow for a test, so the mask is an explicit range
list that keeps every row's work small and still reaches both ends of the key space: 64
query groups, group g admitting the first 256 keys and the 256 keys [L - 256 (g + 1),
L - 256 g) (2^33 or 2^32 admissible pairs).

Checked: the JVP and the forward on sampled rows (first and last rows, group boundaries,
seeded random rows) against the oracle, evaluated exactly on each row's 512 admissible keys
gathered into a small problem (masked keys contribute nothing, so the function is the same);
and the backward through the adjoint identity with the JVP over the whole head, plus gQ of
the sampled rows against the oracle on the same gathered problems.

The identity's fp32 bound is wider than the element-wise one.  The first 256 keys are
admitted by every row, so their gK and gV are sums over all L = 2^23 rows: 2^21 dependent
fp32 additions per output element (four rows per matrix instruction).  For the random-signed
terms here, the rounding error of such a sum grows like sqrt(2^21) 2^-24 = 8.7e-5 relative,
and these keys carry a large share of <gK, dK> + <gV, dV>.  The bound is 5e-4, a little over
five times that estimate; every element-wise comparison keeps the fp32 bar of 1e-4.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import attention_jvp, attention_vjp
from paper_2606_25473_amd import attn_bwd, attn_fwd, attn_jvp_fwd
from paper_2606_25473_amd.workloads import MASK_RANGES, custom_workload, make_inputs

pytestmark = pytest.mark.gpu

D, W, G = 128, 256, 64
# dtype: sequence length (the largest with L * D within the 32-bit byte offsets), tolerance
CASES = {"bf16": (1 << 24, 1e-2), "f32": (1 << 23, 1e-4)}
ADJOINT_TOL = {"bf16": 1e-2, "f32": 5e-4}


def _groups(L):
    R = L // G
    return [(g * R, (g + 1) * R, [(0, W), (L - W * (g + 1), L - W * g)]) for g in range(G)]


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def _np(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def _rel(x, ref):
    return float(np.linalg.norm(np.asarray(x) - np.asarray(ref)) / max(np.linalg.norm(ref), 1e-300))


def _dot(a, b, chunk=1 << 27):
    a, b = a.reshape(-1), b.reshape(-1)
    return sum(float((a[i:i + chunk].double() * b[i:i + chunk].double()).sum()) for i in range(0, a.numel(), chunk))


def _keys_of(r, L):
    g = r // (L // G)
    return np.concatenate([np.arange(W), np.arange(L - W * (g + 1), L - W * g)])


def _gathered(x, r, L):
    """The row r problem on its 512 admissible keys: query row r first, full mask."""
    keys = torch.from_numpy(_keys_of(r, L)).cuda()
    n = keys.numel()
    out = {}
    for name in ("Q", "dQ"):
        row = _np(x[name][0:1, 0:1, r:r + 1])
        out[name] = np.concatenate([row, np.zeros((1, 1, n - 1, D))], axis=2)
    for name in ("K", "V", "dK", "dV"):
        out[name] = _np(x[name][0:1, 0:1].index_select(2, keys))
    return out


def _rows(L):
    R = L // G
    rows = {0, 1, R - 1, R, L // 2, L - R, L - 2, L - 1}
    rows.update(int(r) for r in np.random.default_rng(5).integers(0, L, 8))
    return sorted(rows)


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_largest_head_jvp_forward_backward(dt):
    L, tol = CASES[dt]
    groups = _groups(L)
    w = custom_workload(f"max_head_ranges_{dt}", 1, 1, D, dt, MASK_RANGES, offsets=groups, tangent_std=0.5)
    assert w.L == L and L * D * (2 if dt == "bf16" else 4) == 1 << 32
    _say(f"[max-size] {dt} L = 2^{L.bit_length() - 1}, D = 128 (4 GiB per tensor), {G} query groups: "
         "generating inputs on the GPU")
    x = make_inputs(w, "cuda", 51)
    o, do, lse = attn_jvp_fwd(x["Q"], x["K"], x["V"], x["dQ"], x["dK"], x["dV"], w.kind, groups)
    of, lsef = attn_fwd(x["Q"], x["K"], x["V"], w.kind, groups)
    torch.cuda.synchronize()
    _say("[max-size] JVP and forward done; checking sampled rows")
    for t in (o, do, lse, of, lsef):
        assert torch.isfinite(t).all()
    rows = _rows(L)
    got = {k: [] for k in ("O", "dO", "LSE", "fO", "fLSE")}
    ref = {k: [] for k in ("O", "dO", "LSE")}
    for r in rows:
        p = _gathered(x, r, L)
        O, dO, LSE = attention_jvp(p["Q"], p["K"], p["V"], p["dQ"], p["dK"], p["dV"], "full", None, rows=[0])
        ref["O"].append(O[0, 0, 0]); ref["dO"].append(dO[0, 0, 0]); ref["LSE"].append(LSE[0, 0, 0])
        got["O"].append(_np(o[0, 0, r])); got["dO"].append(_np(do[0, 0, r])); got["LSE"].append(float(lse[0, 0, r]))
        got["fO"].append(_np(of[0, 0, r])); got["fLSE"].append(float(lsef[0, 0, r]))
    errs = (_rel(got["O"], ref["O"]), _rel(got["dO"], ref["dO"]), _rel(got["LSE"], ref["LSE"]),
            _rel(got["fO"], ref["O"]), _rel(got["fLSE"], ref["LSE"]))
    _say(f"[max-size] {len(rows)} rows rel-L2 O={errs[0]:.2e} dO={errs[1]:.2e} LSE={errs[2]:.2e} "
         f"fwd O={errs[3]:.2e} fwd LSE={errs[4]:.2e}")
    assert max(errs) <= tol, errs
    del of, lsef

    _say("[max-size] backward with gO = dO")
    gq, gk, gv, _ = attn_bwd(x["Q"], x["K"], x["V"], o, do, lse, w.kind, groups)
    torch.cuda.synchronize()
    for t in (gq, gk, gv):
        assert torch.isfinite(t).all()
    lhs = _dot(do, do)
    rhs = _dot(gq, x["dQ"]) + _dot(gk, x["dK"]) + _dot(gv, x["dV"])
    rel = abs(lhs - rhs) / abs(lhs)
    _say(f"[max-size] adjoint identity: <dO, dO> = {lhs:.6e}, <g, t> = {rhs:.6e}, rel diff {rel:.2e}")
    assert rel <= ADJOINT_TOL[dt]
    gq_ref, gq_got = [], []
    for r in rows[:8]:
        p = _gathered(x, r, L)
        go = np.concatenate([_np(do[0:1, 0:1, r:r + 1]), np.zeros((1, 1, 2 * W - 1, D))], axis=2)
        rq, _, _, _ = attention_vjp(p["Q"], p["K"], p["V"], go, "full", None, rows=[0], keys=[0])
        gq_ref.append(rq[0, 0, 0]); gq_got.append(_np(gq[0, 0, r]))
    e = _rel(gq_got, gq_ref)
    _say(f"[max-size] gQ of {len(gq_ref)} rows rel-L2 {e:.2e}")
    del x, o, do, lse, gq, gk, gv
    torch.cuda.empty_cache()
    assert e <= tol
