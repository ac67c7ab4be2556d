"""HIP graph capture and concurrent streams (marked ``gpu``).

The entry points only launch kernels on the caller's stream (no allocation, no copy,
no memset, no synchronisation; the mask schedule travels in the kernel arguments),
so a call can be captured in a HIP graph and calls on different streams may overlap.
Checked here:

* the JVP, zero-clean JVP and backward calls captured in a graph (torch.cuda.CUDAGraph
  on a side stream), replayed several times with eager work between the replays: every
  replay equals the eager result bit for bit (the kernels are deterministic); after the
  inputs change in place, a replay follows the new inputs;
* two JVP calls on two streams without synchronisation between them equal the same calls
  made one after the other;
* the same for the fp32 kernels: every fp32 entry point in one graph, and an fp32 call
  beside a bf16 call on two streams.
"""
import sys

import pytest
import torch

from paper_2606_25473_amd import attn_bwd, attn_fwd, attn_jvp_fwd, attn_jvp_fwd_zero_clean
from paper_2606_25473_amd.workloads import MASK_FULL, MASK_TEACHER_FORCING, custom_workload, make_inputs

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, file=sys.stderr, flush=True)


def _capture(fn):
    """Capture fn() in a graph (after one warm-up call on the side stream); returns the
    graph and the outputs it writes."""
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        out = fn()
    torch.cuda.synchronize()
    return g, out


def _replays_equal(g, out, eager, x):
    for rep in range(3):
        # eager work of the program between the replays
        _ = float((x["Q"].float() * 0.5).abs().max())
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(out, eager):
            assert torch.equal(a, b), f"replay {rep} differs from the eager call"


def test_jvp_in_a_graph():
    w = custom_workload("graph_tf", 1, 2, 128, "bf16", MASK_TEACHER_FORCING, 3, 200, tangent_std=0.5)
    _say("[graph] attn_jvp_fwd captured and replayed")
    x = make_inputs(w, "cuda", 21)
    offs = list(w.offsets)
    args = lambda: (x["Q"], x["K"], x["V"], x["dQ"], x["dK"], x["dV"], w.kind, offs)
    eager = attn_jvp_fwd(*args())
    torch.cuda.synchronize()
    eager = [t.clone() for t in eager]
    g, out = _capture(lambda: attn_jvp_fwd(*args()))
    _replays_equal(g, out, eager, x)
    # new input values in the same buffers: the replay computes on them
    x["dV"].mul_(-2.0)
    x["Q"].mul_(0.5)
    g.replay()
    torch.cuda.synchronize()
    fresh = attn_jvp_fwd(*args())
    torch.cuda.synchronize()
    for a, b in zip(out, fresh):
        assert torch.equal(a, b)
    assert not torch.equal(out[1], eager[1])


def test_zero_clean_and_forward_in_a_graph():
    w = custom_workload("graph_zc", 2, 2, 128, "bf16", MASK_TEACHER_FORCING, 3, 150, tangent_std=0.5)
    _say("[graph] attn_jvp_fwd_zero_clean + attn_fwd captured in one graph")
    x = make_inputs(w, "cuda", 22)
    half = w.L // 2
    offs = list(w.offsets)
    tn = {k: x[k][:, :, half:].contiguous() for k in ("dQ", "dK", "dV")}

    def both():
        zc = attn_jvp_fwd_zero_clean(x["Q"], x["K"], x["V"], tn["dQ"], tn["dK"], tn["dV"], offs)
        fw = attn_fwd(x["Q"], x["K"], x["V"], w.kind, offs)
        return (*zc, *fw)

    eager = [t.clone() for t in both()]
    torch.cuda.synchronize()
    g, out = _capture(both)
    _replays_equal(g, out, eager, x)


def test_backward_in_a_graph():
    w = custom_workload("graph_bwd", 1, 3, 128, "bf16", MASK_TEACHER_FORCING, 3, 120, tangent_std=0.5)
    _say("[graph] attn_fwd + attn_bwd captured in one graph")
    x = make_inputs(w, "cuda", 23)
    offs = list(w.offsets)

    def fwd_bwd():
        o, lse = attn_fwd(x["Q"], x["K"], x["V"], w.kind, offs)
        return attn_bwd(x["Q"], x["K"], x["V"], o, x["dV"], lse, w.kind, offs)

    eager = [t.clone() for t in fwd_bwd()]
    torch.cuda.synchronize()
    g, out = _capture(fwd_bwd)
    _replays_equal(g, out, eager, x)


def test_two_streams_overlap():
    wa = custom_workload("streams_tf", 1, 4, 128, "bf16", MASK_TEACHER_FORCING, 4, 300, tangent_std=0.5)
    wb = custom_workload("streams_full", 2, 2, 128, "bf16", MASK_FULL, L=900, tangent_std=0.5)
    _say("[streams] two JVP calls on two streams")
    xa, xb = make_inputs(wa, "cuda", 24), make_inputs(wb, "cuda", 25)

    def call(w, x, stream=None):
        return attn_jvp_fwd(x["Q"], x["K"], x["V"], x["dQ"], x["dK"], x["dV"], w.kind,
                            list(w.offsets) if w.offsets else None, stream=stream)

    ra = [t.clone() for t in call(wa, xa)]
    rb = [t.clone() for t in call(wb, xb)]
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    s1.wait_stream(torch.cuda.current_stream())
    s2.wait_stream(torch.cuda.current_stream())
    for _ in range(3):
        with torch.cuda.stream(s1):
            oa = call(wa, xa, s1)
        with torch.cuda.stream(s2):
            ob = call(wb, xb, s2)
        torch.cuda.synchronize()
        for a, b in zip(oa, ra):
            assert torch.equal(a, b)
        for a, b in zip(ob, rb):
            assert torch.equal(a, b)


def test_fp32_calls_in_a_graph():
    w = custom_workload("graph_f32", 1, 2, 128, "f32", MASK_TEACHER_FORCING, 3, 150)
    _say("[graph] fp32 attn_jvp_fwd, attn_jvp_fwd_zero_clean, attn_fwd and attn_bwd in one graph")
    x = make_inputs(w, "cuda", 26)
    half = w.L // 2
    offs = list(w.offsets)
    tn = {k: x[k][:, :, half:].contiguous() for k in ("dQ", "dK", "dV")}

    def calls():
        jvp = attn_jvp_fwd(x["Q"], x["K"], x["V"], x["dQ"], x["dK"], x["dV"], w.kind, offs)
        zc = attn_jvp_fwd_zero_clean(x["Q"], x["K"], x["V"], tn["dQ"], tn["dK"], tn["dV"], offs)
        o, lse = attn_fwd(x["Q"], x["K"], x["V"], w.kind, offs)
        bwd = attn_bwd(x["Q"], x["K"], x["V"], o, x["dV"], lse, w.kind, offs)
        return (*jvp, *zc, o, lse, *bwd)

    eager = [t.clone() for t in calls()]
    torch.cuda.synchronize()
    g, out = _capture(calls)
    _replays_equal(g, out, eager, x)


def test_bf16_and_fp32_on_two_streams():
    wa = custom_workload("streams_bf16", 1, 4, 128, "bf16", MASK_TEACHER_FORCING, 4, 300, tangent_std=0.5)
    wb = custom_workload("streams_f32", 2, 2, 64, "f32", MASK_FULL, L=700)
    _say("[streams] a bf16 and an fp32 JVP call on two streams")
    xa, xb = make_inputs(wa, "cuda", 27), make_inputs(wb, "cuda", 28)

    def call(w, x, stream=None):
        return attn_jvp_fwd(x["Q"], x["K"], x["V"], x["dQ"], x["dK"], x["dV"], w.kind,
                            list(w.offsets) if w.offsets else None, stream=stream)

    ra = [t.clone() for t in call(wa, xa)]
    rb = [t.clone() for t in call(wb, xb)]
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    s1.wait_stream(torch.cuda.current_stream())
    s2.wait_stream(torch.cuda.current_stream())
    for _ in range(3):
        with torch.cuda.stream(s1):
            oa = call(wa, xa, s1)
        with torch.cuda.stream(s2):
            ob = call(wb, xb, s2)
        torch.cuda.synchronize()
        for a, b in zip(oa, ra):
            assert torch.equal(a, b)
        for a, b in zip(ob, rb):
            assert torch.equal(a, b)
