"""Invariants of the HIP kernels that hold at any size (marked ``gpu``).

These tests compare the kernels with properties the mathematics fixes rather than with
the oracle, so they also run at the full Wan2.1-1.3B chunk-wise shape (B=1, H=12,
L=65520, D=128), which the oracle cannot evaluate whole:

* value tangent only (dQ = dK = 0): the tangent of O is attention applied to dV, so
  dO = attn_fwd(Q, K, dV); the JVP kernel's tangent accumulator then receives the same
  matrix-core products as the forward kernel's output accumulator (H~ is exactly zero),
  so the two agree bit for bit;
* dV = V, dQ = dK = 0: dO = O bit for bit (same products in both accumulators);
* one tangent u for every key (dK_b = u, dQ = dV = 0): the scores of a row move by the
  same amount s Q_a . u, which softmax ignores, so dO = 0; on the GPU what remains is the
  bf16 rounding of H~ = P~ (s Q_a . u), a few 2^-9 of |s Q_a . u| |O_a|;
* rows with exactly one admissible key a (teacher forcing with one-token chunks: the
  first clean row and the first noisy row): O = V_a bit for bit, LSE = s Q_a . K_a,
  and dO = dV_a up to the bf16 rounding of H~ (bounded element by element);
* the adjoint identity between the JVP and the backward kernels for the same (Q, K, V):
  <gO, dO(t)> = <gQ, dQ> + <gK, dK> + <gV, dV>, with the cotangent gO = dO(t), so that
  both sides equal ||dO||^2 (a sign or term error in either kernel moves one side by
  order one; bf16 rounding moves it by far less than the 1e-2 allowed).
"""
import sys

import pytest
import torch

from paper_2606_25473_amd import attn_bwd, attn_fwd, attn_jvp_fwd
from paper_2606_25473_amd.workloads import (HEADLINE, MASK_FULL, MASK_TEACHER_FORCING, WORKLOADS,
                                            custom_workload, make_inputs)

pytestmark = pytest.mark.gpu

SHAPES = [
    custom_workload("inv_tf_ragged", 2, 3, 128, "bf16", MASK_TEACHER_FORCING, 3, 170, tangent_std=0.5),
    custom_workload("inv_tf_d64", 1, 2, 64, "bf16", MASK_TEACHER_FORCING, 4, 100, tangent_std=0.5),
    custom_workload("inv_full_ragged", 1, 2, 128, "bf16", MASK_FULL, L=1000, tangent_std=0.5),
    WORKLOADS[HEADLINE],
]


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def _offs(w):
    return list(w.offsets) if w.offsets else None


def _rel(x, ref):
    x, ref = x.double(), ref.double()
    return float((x - ref).norm() / ref.norm().clamp_min(1e-300))


def _dot(a, b):
    return float((a.double() * b.double()).sum())


@pytest.mark.parametrize("w", SHAPES, ids=lambda w: w.name)
def test_value_tangent_only_is_attention_of_dv(w):
    _say(f"[invariant] dQ = dK = 0: dO = attn_fwd(Q, K, dV) on {w.name} B={w.B} H={w.H} L={w.L} D={w.D}")
    x = make_inputs(w, "cuda", 31)
    z = torch.zeros_like(x["dQ"])
    o, do, lse = attn_jvp_fwd(x["Q"], x["K"], x["V"], z, z, x["dV"], w.kind, _offs(w))
    o2, lse2 = attn_fwd(x["Q"], x["K"], x["dV"], w.kind, _offs(w))
    torch.cuda.synchronize()
    _say(f"[invariant] {w.name} rel-L2(dO, attn_fwd(Q, K, dV)) = {_rel(do, o2):.3e}")
    assert torch.equal(do, o2)
    assert torch.equal(lse, lse2)


@pytest.mark.parametrize("w", SHAPES, ids=lambda w: w.name)
def test_value_tangent_equal_to_v_gives_do_equal_o(w):
    _say(f"[invariant] dV = V, dQ = dK = 0: dO = O on {w.name}")
    x = make_inputs(w, "cuda", 32)
    z = torch.zeros_like(x["dQ"])
    o, do, _ = attn_jvp_fwd(x["Q"], x["K"], x["V"], z, z, x["V"], w.kind, _offs(w))
    torch.cuda.synchronize()
    _say(f"[invariant] {w.name} rel-L2(dO, O) = {_rel(do, o):.3e}")
    assert torch.equal(do, o)


@pytest.mark.parametrize("w", SHAPES[:3], ids=lambda w: w.name)
def test_uniform_key_tangent_gives_zero_do(w):
    _say(f"[invariant] dK_b = u for every key: dO = 0 on {w.name}")
    x = make_inputs(w, "cuda", 33)
    g = torch.Generator(device="cuda")
    g.manual_seed(7)
    u = torch.randn((w.B, w.H, 1, w.D), generator=g, device="cuda").mul_(0.5).to(x["Q"].dtype)
    dk = u.expand_as(x["K"]).contiguous()
    z = torch.zeros_like(x["dQ"])
    o, do, _ = attn_jvp_fwd(x["Q"], x["K"], x["V"], z, dk, z, w.kind, _offs(w))
    torch.cuda.synchronize()
    # the score shift of each row, and the size dO would have without the cancellation
    shift = (x["Q"].double() @ u.double().transpose(-1, -2).contiguous()) / w.D ** 0.5  # [B, H, L, 1]
    scale = (shift * o.double()).norm()
    frac = float(do.double().norm() / scale)
    _say(f"[invariant] {w.name} ||dO|| / ||shift * O|| = {frac:.3e}")
    assert frac <= 1e-2


@pytest.mark.parametrize("D", [64, 128])
def test_single_admissible_key_rows(D):
    N = 64  # one-token chunks: row 0 sees key 0 only, row N (first noisy) sees key N only
    w = custom_workload("inv_one_key", 2, 2, D, "bf16", MASK_TEACHER_FORCING, N, 1, tangent_std=0.5)
    _say(f"[invariant] single-key rows, TF N={N} C=1, D={D}")
    x = make_inputs(w, "cuda", 34)
    o, do, lse = attn_jvp_fwd(x["Q"], x["K"], x["V"], x["dQ"], x["dK"], x["dV"], w.kind, _offs(w))
    torch.cuda.synchronize()
    for a in (0, N):
        assert torch.equal(o[:, :, a], x["V"][:, :, a])
        ref_lse = (x["Q"][:, :, a].double() * x["K"][:, :, a].double()).sum(-1) / D ** 0.5
        err = float((lse[:, :, a].double() - ref_lse).abs().max())
        assert err <= 1e-5 * (1.0 + float(ref_lse.abs().max())), err
        # dO_a = dV_a + V_a (bf16(h) - h), h = s (dQ_a . K_a + Q_a . dK_a): at most half a
        # bf16 unit of h times |V_a|, plus the rounding of dO itself (2^-7 covers both)
        h = ((x["dQ"][:, :, a].double() * x["K"][:, :, a].double()).sum(-1, keepdim=True) +
             (x["Q"][:, :, a].double() * x["dK"][:, :, a].double()).sum(-1, keepdim=True)) / D ** 0.5
        dva, va = x["dV"][:, :, a].double(), x["V"][:, :, a].double()
        dev = (do[:, :, a].double() - dva).abs()
        bound = 2.0 ** -7 * (h.abs() * va.abs() + dva.abs()) + 1e-6
        _say(f"[invariant] row {a}: LSE err {err:.2e}, max |dO - dV_a| / bound = {float((dev / bound).max()):.3f}")
        assert bool((dev <= bound).all())


@pytest.mark.parametrize("w", [SHAPES[0], SHAPES[2], SHAPES[3]], ids=lambda w: w.name)
def test_adjoint_identity_jvp_vs_backward(w):
    _say(f"[invariant] <dO, dO(t)> = <(gQ, gK, gV), t> on {w.name} B={w.B} H={w.H} L={w.L}")
    x = make_inputs(w, "cuda", 35)
    q, k, v, dq, dk, dv = (x[n] for n in ("Q", "K", "V", "dQ", "dK", "dV"))
    o, do, lse = attn_jvp_fwd(q, k, v, dq, dk, dv, w.kind, _offs(w))
    gq, gk, gv, _ = attn_bwd(q, k, v, o, do, lse, w.kind, _offs(w))
    torch.cuda.synchronize()
    lhs = _dot(do, do)
    rhs = _dot(gq, dq) + _dot(gk, dk) + _dot(gv, dv)
    rel = abs(lhs - rhs) / abs(lhs)
    _say(f"[invariant] {w.name} <gO, dO> = {lhs:.6e}, <g, t> = {rhs:.6e}, rel diff {rel:.2e}")
    assert rel <= 1e-2
