"""Pins of the fp64 CPU oracle to things other than itself (CPU only).

* hand-written masks and hand-derived worked examples (tests/golden/),
* closed-form pair counts,
* PyTorch's scaled_dot_product_attention and torch.func.jvp (fp64, CPU),
* central finite differences of the oracle's own primal,
* a pure-Python dual-number evaluation (oracle/dual.py),
* the paper's two-pass TF identity and algebraic invariants of the tangent.
"""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from torch.nn.attention import SDPBackend, sdpa_kernel

from oracle import (MASK_BLOCK_CAUSAL, MASK_FULL, MASK_RANGES, MASK_TEACHER_FORCING, allowed_mask,
                    attention_fwd, attention_jvp, attention_jvp_zero_clean, count_allowed_pairs)
from oracle.dual import attention_dual

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _read_mask(name):
    rows, offsets = [], None
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line.startswith("# offsets:"):
                offsets = [int(x) for x in line.split(":")[1].split()]
            if not line or line.startswith("#"):
                continue
            rows.append([c == "1" for c in line])
    return np.array(rows, dtype=bool), offsets


def _rand(shape, seed, scale=1.0):
    g = np.random.default_rng(seed)
    return g.standard_normal(shape) * scale


def _tf(N, C):
    return [i * C for i in range(N + 1)]


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


# ----------------------------------------------------------------------------- masks

def test_tf_mask_matches_hand_written():
    m, _ = _read_mask("tf_mask_N3_C2.txt")
    assert np.array_equal(allowed_mask(MASK_TEACHER_FORCING, _tf(3, 2), 12), m)


def test_block_causal_mask_matches_hand_written():
    m, _ = _read_mask("block_causal_N3_C2.txt")
    assert np.array_equal(allowed_mask(MASK_BLOCK_CAUSAL, _tf(3, 2), 6), m)


def test_nonuniform_tf_mask_matches_hand_written():
    m, offsets = _read_mask("tf_mask_nonuniform.txt")
    assert offsets == [0, 1, 3]
    assert np.array_equal(allowed_mask(MASK_TEACHER_FORCING, offsets, 6), m)


def test_ranges_mask_reproduces_hand_written_tf_mask():
    # the TF mask of the golden fixture, given as query groups with key ranges
    m, _ = _read_mask("tf_mask_N3_C2.txt")
    groups = [(0, 2, [(0, 2)]), (2, 4, [(0, 4)]), (4, 6, [(0, 6)]),
              (6, 8, [(0, 0), (6, 8)]), (8, 10, [(0, 2), (8, 10)]), (10, 12, [(0, 4), (10, 12)])]
    assert np.array_equal(allowed_mask(MASK_RANGES, groups, 12), m)


def test_ranges_mask_with_empty_group_and_two_ranges():
    groups = [(0, 1, []), (1, 3, [(1, 2), (4, 5)]), (3, 5, [(0, 5)])]
    want = np.array([[0, 0, 0, 0, 0], [0, 1, 0, 0, 1], [0, 1, 0, 0, 1], [1, 1, 1, 1, 1], [1, 1, 1, 1, 1]], bool)
    assert np.array_equal(allowed_mask(MASK_RANGES, groups, 5), want)


def _read_groups(name):
    """The query groups of a golden range-list fixture ('# group: q0 q1 : k0 k1 ...' lines)."""
    groups = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            if line.startswith("# group:"):
                q, k = line.split(":", 1)[1].split(":")
                q0, q1 = (int(v) for v in q.split())
                ks = [int(v) for v in k.split()]
                groups.append((q0, q1, list(zip(ks[0::2], ks[1::2]))))
    return groups


GENERAL_GROUPS = _read_groups("ranges_general.txt")


def test_general_range_list_mask_matches_hand_written():
    """Groups with four key intervals, none, adjacent ones, an empty one, rows in no group."""
    m, _ = _read_mask("ranges_general.txt")
    assert len(GENERAL_GROUPS) == 4 and len(GENERAL_GROUPS[0][2]) == 4 and GENERAL_GROUPS[1][2] == []
    assert np.array_equal(allowed_mask(MASK_RANGES, GENERAL_GROUPS, 12), m)
    # the same mask with the adjacent intervals merged, the empty one dropped, groups reordered
    merged = [GENERAL_GROUPS[3][:2] + ([(0, 3), (11, 12)],), (4, 7, [(2, 6), (9, 10)]), GENERAL_GROUPS[0]]
    assert np.array_equal(allowed_mask(MASK_RANGES, merged, 12), m)
    assert count_allowed_pairs(MASK_RANGES, GENERAL_GROUPS, 12) == int(m.sum()) == 2 * 6 + 3 * 5 + 3 * 4


@pytest.mark.parametrize("groups,msg", [
    ([(0, 4, [(0, 3), (2, 5)])], "overlap"),             # key intervals of one group overlap
    ([(0, 4, [(0, 3)]), (3, 6, [(0, 1)])], "overlap"),    # query intervals overlap
    ([(0, 4, [(0, 9)])], "inside"),                       # key interval past the end
    ([(2, 2, [(0, 1)])], "inside"),                       # empty query interval
    ([(0, 9, [(0, 1)])], "inside"),                       # query interval past the end
])
def test_range_lists_outside_the_representation_are_rejected(groups, msg):
    with pytest.raises(ValueError, match=msg):
        allowed_mask(MASK_RANGES, groups, 8)


def test_fully_masked_rows_give_zero_and_minus_inf():
    groups = [(0, 2, []), (2, 5, [(0, 5)])]
    x = [_rand((1, 1, 5, 4), 200 + s) for s in range(6)]
    O, dO, LSE = attention_jvp(*x, MASK_RANGES, groups)
    assert np.all(O[0, 0, :2] == 0) and np.all(dO[0, 0, :2] == 0) and np.all(LSE[0, 0, :2] == -np.inf)
    assert np.all(np.isfinite(O[0, 0, 2:])) and np.all(np.isfinite(LSE[0, 0, 2:]))


@pytest.mark.parametrize("N,C", [(1, 1), (3, 5), (4, 16), (7, 13), (21, 3)])
def test_tf_pair_count_closed_form(N, C):
    # clean chunk j: C rows x (j+1)C keys; noisy chunk i: C rows x (i+1)C keys -> C^2 N (N+1)
    assert count_allowed_pairs(MASK_TEACHER_FORCING, _tf(N, C), 2 * N * C) == C * C * N * (N + 1)


@pytest.mark.parametrize("N,C", [(1, 4), (5, 3)])
def test_block_causal_and_full_pair_counts(N, C):
    assert count_allowed_pairs(MASK_BLOCK_CAUSAL, _tf(N, C), N * C) == C * C * N * (N + 1) // 2
    assert count_allowed_pairs(MASK_FULL, None, 37) == 37 * 37


def test_tf_mask_row_subsets_agree():
    full = allowed_mask(MASK_TEACHER_FORCING, _tf(5, 7), 70)
    rows = np.array([0, 6, 7, 34, 35, 36, 41, 69])
    assert np.array_equal(allowed_mask(MASK_TEACHER_FORCING, _tf(5, 7), 70, rows), full[rows])


# ----------------------------------------------------------------------------- worked examples

def _ev(x):
    if isinstance(x, str):
        return float(eval(x, {"__builtins__": {}}, {"ln": math.log}))
    return float(x)


def _arr(rows):
    return np.array([[_ev(v) for v in r] for r in rows], dtype=np.float64)


with open(os.path.join(GOLDEN, "worked_examples.json")) as _f:
    _EXAMPLES = json.load(_f)["examples"]


@pytest.mark.parametrize("ex", _EXAMPLES, ids=[e["name"] for e in _EXAMPLES])
def test_hand_derived_worked_examples(ex):
    t = {k: _arr(ex[k])[None, None] for k in ("Q", "K", "V", "dQ", "dK", "dV")}
    O, dO, LSE = attention_jvp(t["Q"], t["K"], t["V"], t["dQ"], t["dK"], t["dV"],
                               ex["kind"], ex["offsets"], scale=ex["scale"])
    np.testing.assert_allclose(O[0, 0], _arr(ex["O"]), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(dO[0, 0], _arr(ex["dO"]), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(LSE[0, 0], [_ev(v) for v in ex["LSE"]], rtol=1e-13, atol=1e-13)


# ----------------------------------------------------------------------------- torch SDPA / jvp

def _sdpa(q, k, v, mask=None, scale=None):
    return F.scaled_dot_product_attention(q, k, v, attn_mask=mask, scale=scale)


def _torch_jvp(q, k, v, dq, dk, dv, mask=None, is_causal=False):
    # forward-mode AD through PyTorch's own SDPA (math backend: the fused CPU kernel has no jvp rule)
    f = lambda a, b, c: F.scaled_dot_product_attention(a, b, c, attn_mask=mask, is_causal=is_causal)
    with sdpa_kernel(SDPBackend.MATH):
        return torch.func.jvp(f, (q, k, v), (dq, dk, dv))


def test_full_mask_vs_torch_sdpa_and_jvp():
    B, H, L, D = 2, 3, 40, 16
    x = [torch.from_numpy(_rand((B, H, L, D), s)) for s in range(6)]
    O, dO, LSE = attention_jvp(*[t.numpy() for t in x], MASK_FULL)
    o_ref, do_ref = _torch_jvp(*x)
    np.testing.assert_allclose(O, o_ref.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dO, do_ref.numpy(), rtol=1e-11, atol=1e-12)
    lse_ref = torch.logsumexp((x[0] @ x[1].transpose(-1, -2)) / math.sqrt(D), dim=-1)
    np.testing.assert_allclose(LSE, lse_ref.numpy(), rtol=1e-13, atol=1e-12)


def test_block_causal_one_token_chunks_is_token_causal_sdpa():
    B, H, L, D = 1, 2, 33, 8
    x = [torch.from_numpy(_rand((B, H, L, D), 10 + s)) for s in range(6)]
    O, dO, _ = attention_jvp(*[t.numpy() for t in x], MASK_BLOCK_CAUSAL, list(range(L + 1)))
    o_ref, do_ref = _torch_jvp(*x, is_causal=True)
    np.testing.assert_allclose(O, o_ref.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dO, do_ref.numpy(), rtol=1e-11, atol=1e-12)


def test_scale_override_vs_sdpa():
    B, H, L, D = 1, 1, 17, 8
    x = [torch.from_numpy(_rand((B, H, L, D), 20 + s)) for s in range(3)]
    O, LSE = attention_fwd(*[t.numpy() for t in x], MASK_FULL, scale=0.37)
    np.testing.assert_allclose(O, _sdpa(*x, scale=0.37).numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("N,C", [(3, 4), (4, 3), (1, 5)])
def test_tf_two_pass_identity(N, C):
    """Paper Sec. 3.1.1: TF equals (1) block-causal attention over the clean half and
    (2) noisy chunk i attending [clean chunks < i | noisy chunk i] without a mask."""
    B, H, D = 1, 2, 8
    half = N * C
    L = 2 * half
    x = [torch.from_numpy(_rand((B, H, L, D), 30 + s)) for s in range(6)]
    O, dO, _ = attention_jvp(*[t.numpy() for t in x], MASK_TEACHER_FORCING, _tf(N, C))
    # (1) clean rows: block-causal mask built as kron(tril(ones N), ones C)
    bc = torch.kron(torch.tril(torch.ones(N, N)), torch.ones(C, C)).bool()
    o1, do1 = _torch_jvp(*[t[:, :, :half] for t in x], mask=bc)
    np.testing.assert_allclose(O[:, :, :half], o1.numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dO[:, :, :half], do1.numpy(), rtol=1e-11, atol=1e-12)
    # (2) noisy rows of chunk i: dense attention over gathered keys
    for i in range(N):
        q_sl = slice(half + i * C, half + (i + 1) * C)
        keys = torch.cat([torch.arange(0, i * C), torch.arange(half + i * C, half + (i + 1) * C)])
        q, k, v, dq, dk, dv = x
        o2, do2 = _torch_jvp(q[:, :, q_sl], k[:, :, keys], v[:, :, keys],
                             dq[:, :, q_sl], dk[:, :, keys], dv[:, :, keys])
        np.testing.assert_allclose(O[:, :, q_sl], o2.numpy(), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(dO[:, :, q_sl], do2.numpy(), rtol=1e-11, atol=1e-12)


# ----------------------------------------------------------------------------- finite differences

@pytest.mark.parametrize("kind,offsets,L", [(MASK_TEACHER_FORCING, _tf(3, 4), 24),
                                            (MASK_BLOCK_CAUSAL, [0, 3, 7, 10], 10),
                                            (MASK_FULL, None, 13),
                                            (MASK_RANGES, GENERAL_GROUPS, 12)])
def test_tangent_vs_central_finite_differences(kind, offsets, L):
    B, H, D = 1, 2, 8
    x = [_rand((B, H, L, D), 40 + s) for s in range(6)]
    Q, K, V, dQ, dK, dV = x
    _, dO, _ = attention_jvp(Q, K, V, dQ, dK, dV, kind, offsets)
    h = 1e-5
    Op, _ = attention_fwd(Q + h * dQ, K + h * dK, V + h * dV, kind, offsets)
    Om, _ = attention_fwd(Q - h * dQ, K - h * dK, V - h * dV, kind, offsets)
    fd = (Op - Om) / (2 * h)
    assert _rel(dO, fd) < 1e-8


# ----------------------------------------------------------------------------- dual numbers

@pytest.mark.parametrize("kind,offsets,L,D", [(MASK_TEACHER_FORCING, _tf(2, 3), 12, 4),
                                              (MASK_TEACHER_FORCING, [0, 1, 4, 6], 12, 3),
                                              (MASK_BLOCK_CAUSAL, [0, 2, 5], 5, 4),
                                              (MASK_FULL, None, 7, 5),
                                              (MASK_RANGES, GENERAL_GROUPS, 12, 3)])
def test_closed_form_vs_dual_numbers(kind, offsets, L, D):
    B, H = 1, 2
    x = [_rand((B, H, L, D), 50 + s) for s in range(6)]
    O, dO, LSE = attention_jvp(*x, kind, offsets)
    Od, dOd, LSEd, _ = attention_dual(*[a.tolist() for a in x], kind, offsets)
    np.testing.assert_allclose(O, np.array(Od), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dO, np.array(dOd), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(LSE, np.array(LSEd), rtol=1e-13, atol=1e-13)


def test_dual_numbers_on_tiny_tf_heads():
    """The 4-chunk x 16-token TF layout at head_dim 16 (one head), closed form vs duals."""
    L, D = 128, 16
    x = [_rand((1, 1, L, D), 60 + s) for s in range(6)]
    O, dO, LSE = attention_jvp(*x, MASK_TEACHER_FORCING, _tf(4, 16))
    Od, dOd, LSEd, _ = attention_dual(*[a.tolist() for a in x], MASK_TEACHER_FORCING, _tf(4, 16))
    np.testing.assert_allclose(O, np.array(Od), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dO, np.array(dOd), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(LSE, np.array(LSEd), rtol=1e-13, atol=1e-13)


# ----------------------------------------------------------------------------- invariants

def _tf_inputs(N=3, C=5, D=8, seed=70):
    L = 2 * N * C
    return [_rand((1, 2, L, D), seed + s) for s in range(6)], _tf(N, C)


def test_zero_tangents_give_exact_zero():
    (Q, K, V, *_), offs = _tf_inputs()
    z = np.zeros_like(Q)
    _, dO, _ = attention_jvp(Q, K, V, z, z, z, MASK_TEACHER_FORCING, offs)
    assert np.all(dO == 0.0)


def test_tangent_is_linear():
    (Q, K, V, dQ, dK, dV), offs = _tf_inputs()
    t2 = [_rand(Q.shape, 90 + s) for s in range(3)]
    a, b = 0.7, -1.3
    _, d1, _ = attention_jvp(Q, K, V, dQ, dK, dV, MASK_TEACHER_FORCING, offs)
    _, d2, _ = attention_jvp(Q, K, V, *t2, MASK_TEACHER_FORCING, offs)
    mix = [a * u + b * w for u, w in zip((dQ, dK, dV), t2)]
    _, d12, _ = attention_jvp(Q, K, V, *mix, MASK_TEACHER_FORCING, offs)
    np.testing.assert_allclose(d12, a * d1 + b * d2, rtol=1e-12, atol=1e-12)


def test_value_tangent_only_is_attention_of_dV():
    (Q, K, V, _, _, dV), offs = _tf_inputs()
    z = np.zeros_like(Q)
    _, dO, _ = attention_jvp(Q, K, V, z, z, dV, MASK_TEACHER_FORCING, offs)
    O_dv, _ = attention_fwd(Q, K, dV, MASK_TEACHER_FORCING, offs)
    np.testing.assert_allclose(dO, O_dv, rtol=1e-13, atol=1e-13)
    _, dO2, _ = attention_jvp(Q, K, V, z, z, V, MASK_TEACHER_FORCING, offs)
    O, _ = attention_fwd(Q, K, V, MASK_TEACHER_FORCING, offs)
    np.testing.assert_allclose(dO2, O, rtol=1e-13, atol=1e-13)


def test_uniform_key_shift_has_zero_tangent():
    (Q, K, V, *_), offs = _tf_inputs()
    u = _rand((1, 2, 1, Q.shape[-1]), 99)
    dK = np.broadcast_to(u, K.shape).copy()
    z = np.zeros_like(Q)
    _, dO, _ = attention_jvp(Q, K, V, z, dK, z, MASK_TEACHER_FORCING, offs)
    assert np.abs(dO).max() < 1e-12


def test_single_allowed_key_rows():
    # TF with one-token chunks: the first noisy token sees only itself
    N, C, D = 4, 1, 8
    L = 2 * N * C
    Q, K, V, dQ, dK, dV = [_rand((1, 1, L, D), 110 + s) for s in range(6)]
    O, dO, LSE = attention_jvp(Q, K, V, dQ, dK, dV, MASK_TEACHER_FORCING, _tf(N, C))
    for a in (0, N):   # clean token 0 and noisy token 0 each see exactly one key (themselves)
        np.testing.assert_allclose(O[0, 0, a], V[0, 0, a], rtol=1e-14, atol=1e-14)
        np.testing.assert_allclose(dO[0, 0, a], dV[0, 0, a], rtol=1e-13, atol=1e-13)
        assert LSE[0, 0, a] == pytest.approx(Q[0, 0, a] @ K[0, 0, a] / math.sqrt(D), rel=1e-14)


def test_clean_half_independent_of_noisy_inputs():
    (Q, K, V, dQ, dK, dV), offs = _tf_inputs()
    half = Q.shape[2] // 2
    O1, dO1, L1 = attention_jvp(Q, K, V, dQ, dK, dV, MASK_TEACHER_FORCING, offs)
    X = [a.copy() for a in (Q, K, V, dQ, dK, dV)]
    for a in X:
        a[:, :, half:] = _rand(a[:, :, half:].shape, 123)
    O2, dO2, L2 = attention_jvp(*X, MASK_TEACHER_FORCING, offs)
    assert np.array_equal(O1[:, :, :half], O2[:, :, :half])
    assert np.array_equal(dO1[:, :, :half], dO2[:, :, :half])
    assert np.array_equal(L1[:, :, :half], L2[:, :, :half])


def test_row_subset_matches_full_evaluation():
    (Q, K, V, dQ, dK, dV), offs = _tf_inputs()
    rows = np.array([0, 4, 15, 16, 29])
    O, dO, LSE = attention_jvp(Q, K, V, dQ, dK, dV, MASK_TEACHER_FORCING, offs)
    Os, dOs, LSEs = attention_jvp(Q, K, V, dQ, dK, dV, MASK_TEACHER_FORCING, offs, rows=rows, block=2)
    # BLAS may round a differently-shaped product differently in the last bit
    np.testing.assert_allclose(Os, O[:, :, rows], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(dOs, dO[:, :, rows], rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(LSEs, LSE[:, :, rows], rtol=1e-14, atol=1e-14)


# ----------------------------------------------------------------------------- zero clean tangents

@pytest.mark.parametrize("N,C", [(3, 4), (4, 3), (1, 5)])
def test_zero_clean_tangent_vs_torch_jvp(N, C):
    """Paper Sec. 3.1.2 (TF-sCM tangent [0^clean, t^noisy]): clean rows have dO = 0
    exactly, and noisy chunk i equals torch's JVP of dense attention over
    [clean chunks < i | noisy chunk i] with zero tangents on the clean keys."""
    B, H, D = 1, 2, 8
    half = N * C
    L = 2 * half
    q, k, v = [torch.from_numpy(_rand((B, H, L, D), 130 + s)) for s in range(3)]
    dqn, dkn, dvn = [torch.from_numpy(_rand((B, H, half, D), 140 + s)) for s in range(3)]
    O, dO, LSE = attention_jvp_zero_clean(q.numpy(), k.numpy(), v.numpy(), dqn.numpy(), dkn.numpy(),
                                          dvn.numpy(), _tf(N, C))
    assert dO.shape == (B, H, L, D)
    assert np.all(dO[:, :, :half] == 0.0)
    O_fwd, LSE_fwd = attention_fwd(q.numpy(), k.numpy(), v.numpy(), MASK_TEACHER_FORCING, _tf(N, C))
    np.testing.assert_array_equal(O, O_fwd)
    np.testing.assert_array_equal(LSE, LSE_fwd)
    z = torch.zeros(B, H, half, D, dtype=torch.float64)
    dq, dk, dv = [torch.cat([z, t], dim=2) for t in (dqn, dkn, dvn)]
    for i in range(N):
        q_sl = slice(half + i * C, half + (i + 1) * C)
        keys = torch.cat([torch.arange(0, i * C), torch.arange(half + i * C, half + (i + 1) * C)])
        o2, do2 = _torch_jvp(q[:, :, q_sl], k[:, :, keys], v[:, :, keys],
                             dq[:, :, q_sl], dk[:, :, keys], dv[:, :, keys])
        np.testing.assert_allclose(O[:, :, q_sl], o2.numpy(), rtol=1e-12, atol=1e-12)
        np.testing.assert_allclose(dO[:, :, q_sl], do2.numpy(), rtol=1e-11, atol=1e-12)


def test_zero_clean_tangent_noisy_rows_drop_clean_key_terms():
    """Over clean keys only the dQ term of the score tangent and the V term of the
    output tangent survive: perturbing the clean part of padded dK, dV changes the
    noisy dO, while the zero-clean JVP is blind to it by construction."""
    (Q, K, V, dQ, dK, dV), offs = _tf_inputs()
    half = Q.shape[2] // 2
    O, dO, _ = attention_jvp_zero_clean(Q, K, V, dQ[:, :, half:], dK[:, :, half:], dV[:, :, half:], offs)
    X = [a.copy() for a in (dQ, dK, dV)]
    for a in X:
        a[:, :, :half] = 0.0
    _, dO_pad, _ = attention_jvp(Q, K, V, *X, MASK_TEACHER_FORCING, offs)
    np.testing.assert_array_equal(dO, dO_pad)
    _, dO_dense, _ = attention_jvp(Q, K, V, dQ, dK, dV, MASK_TEACHER_FORCING, offs)
    assert _rel(dO[:, :, half:], dO_dense[:, :, half:]) > 1e-3   # the clean tangents did matter
