"""Pins of the fp64 backward oracle (oracle.attention_vjp) to things other than itself (CPU only).

* PyTorch autograd through scaled_dot_product_attention (fp64, math backend) on
  the full, token-causal and teacher-forcing masks (the TF mask rebuilt here from
  chunk ids with torch ops, not from the oracle);
* the adjoint identity with the independently pinned JVP oracle:
  <gO, JVP(t)> = <VJP(gO), t> for random tangents t;
* central finite differences of f = sum(gO o O);
* invariants: keys' gradients sum to zero (softmax is shift invariant in the
  scores), the value gradients sum to the cotangents of rows that see any key,
  Delta = rowsum(gO o O) with O from the forward oracle, row/key subsets, and
  gradients of keys no row admits are exactly zero.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from torch.nn.attention import SDPBackend, sdpa_kernel

from oracle import (MASK_BLOCK_CAUSAL, MASK_FULL, MASK_RANGES, MASK_TEACHER_FORCING, attention_fwd,
                    attention_jvp, attention_vjp)


def _rand(shape, seed, scale=1.0):
    return np.random.default_rng(seed).standard_normal(shape) * scale


def _tf(N, C):
    return [i * C for i in range(N + 1)]


def _torch_grads(q, k, v, g, mask=None, is_causal=False):
    q, k, v = (t.clone().requires_grad_(True) for t in (q, k, v))
    with sdpa_kernel(SDPBackend.MATH):
        o = F.scaled_dot_product_attention(q, k, v, attn_mask=mask, is_causal=is_causal)
    o.backward(g)
    return q.grad.numpy(), k.grad.numpy(), v.grad.numpy()


def _tf_mask_torch(N, C):
    """Boolean TF mask from chunk ids with torch ops: clean j sees clean <= j; noisy i sees
    clean < i and noisy i."""
    half = N * C
    idx = torch.arange(2 * half)
    noisy = idx >= half
    chunk = (idx % half) // C
    cq, ck = chunk[:, None], chunk[None, :]
    nq, nk = noisy[:, None], noisy[None, :]
    return (~nq & ~nk & (ck <= cq)) | (nq & ~nk & (ck < cq)) | (nq & nk & (ck == cq))


@pytest.mark.parametrize("case", ["full", "causal", "tf"])
def test_vjp_vs_torch_autograd(case):
    B, H, D = 1, 2, 16
    if case == "tf":
        N, C = 3, 5
        L = 2 * N * C
    else:
        L = 37
    x = [torch.from_numpy(_rand((B, H, L, D), 200 + s)) for s in range(4)]
    if case == "full":
        ref = _torch_grads(*x)
        got = attention_vjp(*[t.numpy() for t in x], MASK_FULL)
    elif case == "causal":
        ref = _torch_grads(*x, is_causal=True)
        got = attention_vjp(*[t.numpy() for t in x], MASK_BLOCK_CAUSAL, list(range(L + 1)))
    else:
        ref = _torch_grads(*x, mask=_tf_mask_torch(N, C))
        got = attention_vjp(*[t.numpy() for t in x], MASK_TEACHER_FORCING, _tf(N, C))
    for a, b in zip(got[:3], ref):
        np.testing.assert_allclose(a, b, rtol=1e-11, atol=1e-12)


LAYOUTS = [
    (MASK_TEACHER_FORCING, _tf(3, 4), 24),
    (MASK_BLOCK_CAUSAL, [0, 3, 7, 10], 10),
    (MASK_FULL, None, 13),
    (MASK_RANGES, [(0, 5, [(0, 3), (9, 12)]), (5, 9, []), (9, 14, [(2, 6), (7, 14)])], 14),  # group 1: no keys
    # three key intervals in one group, adjacent intervals, a row in no group
    (MASK_RANGES, [(0, 4, [(0, 2), (5, 6), (9, 11)]), (4, 10, [(3, 5), (5, 8)]), (11, 13, [(12, 13), (0, 1)])], 13),
]


@pytest.mark.parametrize("kind,offsets,L", LAYOUTS)
def test_adjoint_identity_with_jvp_oracle(kind, offsets, L):
    B, H, D = 1, 2, 8
    Q, K, V, dQ, dK, dV, gO = [_rand((B, H, L, D), 210 + s) for s in range(7)]
    _, dO, _ = attention_jvp(Q, K, V, dQ, dK, dV, kind, offsets)
    gQ, gK, gV, _ = attention_vjp(Q, K, V, gO, kind, offsets)
    lhs = float((gO * dO).sum())
    rhs = float((gQ * dQ).sum() + (gK * dK).sum() + (gV * dV).sum())
    assert lhs == pytest.approx(rhs, rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("kind,offsets,L", LAYOUTS[:3])
def test_vjp_vs_central_finite_differences(kind, offsets, L):
    B, H, D = 1, 1, 8
    Q, K, V, gO = [_rand((B, H, L, D), 220 + s) for s in range(4)]
    dirs = [_rand((B, H, L, D), 230 + s) for s in range(3)]
    gQ, gK, gV, _ = attention_vjp(Q, K, V, gO, kind, offsets)

    def f(eps):
        O, _ = attention_fwd(Q + eps * dirs[0], K + eps * dirs[1], V + eps * dirs[2], kind, offsets)
        return float((gO * O).sum())

    h = 1e-5
    fd = (f(h) - f(-h)) / (2 * h)
    exact = float((gQ * dirs[0]).sum() + (gK * dirs[1]).sum() + (gV * dirs[2]).sum())
    assert fd == pytest.approx(exact, rel=1e-7, abs=1e-9)


def test_vjp_invariants_and_subsets():
    N, C, D = 3, 5, 8
    L = 2 * N * C
    Q, K, V, gO = [_rand((1, 2, L, D), 240 + s) for s in range(4)]
    offs = _tf(N, C)
    gQ, gK, gV, Delta = attention_vjp(Q, K, V, gO, MASK_TEACHER_FORCING, offs)
    # softmax is invariant to a per-row shift of the scores: the key gradients sum to zero
    np.testing.assert_allclose(gK.sum(axis=2), 0.0, atol=1e-12)
    # every row of a TF mask sees a key, and each row's P sums to one
    np.testing.assert_allclose(gV.sum(axis=2), gO.sum(axis=2), rtol=1e-12, atol=1e-12)
    O, _ = attention_fwd(Q, K, V, MASK_TEACHER_FORCING, offs)
    np.testing.assert_allclose(Delta, (gO * O).sum(axis=3), rtol=1e-13, atol=1e-13)
    rows, keys = np.array([0, 7, 15, 16, 29]), np.array([1, 14, 15, 22])
    a = attention_vjp(Q, K, V, gO, MASK_TEACHER_FORCING, offs, rows=rows, keys=keys, block=4)
    np.testing.assert_allclose(a[0], gQ[:, :, rows], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(a[1], gK[:, :, keys], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(a[2], gV[:, :, keys], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(a[3], Delta[:, :, rows], rtol=1e-13, atol=1e-14)


def test_unseen_keys_and_empty_rows_get_zero_gradient():
    # keys 10..13 are admitted by no group; rows 5..8 admit no key
    groups = [(0, 5, [(0, 4), (6, 10)]), (5, 9, []), (9, 14, [(0, 10)])]
    L, D = 14, 8
    Q, K, V, gO = [_rand((1, 1, L, D), 250 + s) for s in range(4)]
    gQ, gK, gV, Delta = attention_vjp(Q, K, V, gO, MASK_RANGES, groups)
    assert np.all(gK[0, 0, 10:] == 0.0) and np.all(gV[0, 0, 10:] == 0.0)
    assert np.all(gQ[0, 0, 5:9] == 0.0) and np.all(Delta[0, 0, 5:9] == 0.0)
    # single-key row: a row that sees only key j has P = e_j, so gV_j gets its cotangent
    g2 = [(0, 1, [(3, 4)]), (1, L, [(0, L)])]
    Z = np.zeros_like(gO)
    Z[0, 0, 0] = gO[0, 0, 0]
    _, _, gV2, _ = attention_vjp(Q, K, V, Z, MASK_RANGES, g2)
    np.testing.assert_allclose(gV2[0, 0, 3], gO[0, 0, 0], rtol=1e-14)
    assert np.all(np.delete(gV2[0, 0], 3, axis=0) == 0.0)
    assert math.isfinite(float(np.abs(gV2).sum()))
