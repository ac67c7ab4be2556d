"""Throughput of the fused masked attention forward + JVP on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--forward | --zero-clean | --backward] [--no-cpu]

One step = one ``attn_jvp_fwd`` call over the whole batch of the workload
(default: Wan2.1-1.3B chunk-wise teacher forcing, B=1, H=12, L=65520, D=128,
bf16), inputs already resident in HBM.  Work is counted over admissible
(query, key) pairs only: 12*D flop per pair for the JVP, 4*D for the forward.
``--zero-clean`` times ``attn_jvp_fwd_zero_clean`` instead (teacher-forcing
workloads: tangents of the noisy half only) and counts the work that variant
must do: 4*D per pair of a clean query, 8*D per (noisy query, clean key) pair
(scores, dQ term, output, H~ term), 12*D per (noisy query, noisy key) pair; it
also reports the dense JVP's time on the same inputs.  ``--backward`` times
``attn_bwd`` (both of its launches) for a cotangent gO, with O and LSE from an
untimed ``attn_fwd``, and counts 10*D flop per pair (scores recomputed, gP, gV,
gK, gQ).
Prints ONE JSON line.  The ``cpu_baseline`` leg times the fp64 CPU oracle on a
bounded sample of query rows of the same workload (and checks the sampled GPU
rows against it).
"""
import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2606_25473_amd import (attn_bwd, attn_fwd, attn_jvp_fwd, attn_jvp_fwd_zero_clean,  # noqa: E402
                                  count_computed_pairs, count_unmasked_pairs, query_groups)
from paper_2606_25473_amd.workloads import HEADLINE, WORKLOADS, custom_workload, make_inputs  # noqa: E402

METRIC = "masked attention fwd+JVP TFLOP/s (unmasked pairs) and % bf16 MFMA peak"
# the line printed by the non-default modes names what they measure
MODE_METRIC = {
    "jvp": METRIC,
    "fwd": "masked attention forward TFLOP/s (unmasked pairs, 4*D each) and % bf16 MFMA peak",
    "zc": "masked attention zero-clean-tangent fwd+JVP TFLOP/s (required flop) and % bf16 MFMA peak",
    "bwd": "masked attention backward TFLOP/s (unmasked pairs, 10*D each) and % bf16 MFMA peak",
}
# MI355X dense bf16 matrix peak: 256 CUs x 2.4 GHz x 4096 flop/clk/CU
PEAK_BF16_TFLOPS = 256 * 2.4e9 * 4096 / 1e12
PEAK_FP32_TFLOPS = 157.3
KERNEL_SOURCES = ["paper_2606_25473_amd/csrc/attn_mfma.hip", "paper_2606_25473_amd/csrc/attn_bwd.hip",
                  "paper_2606_25473_amd/csrc/mfma_common.hpp", "paper_2606_25473_amd/csrc/schedule.hpp",
                  "paper_2606_25473_amd/csrc/kernels.hpp"]
# the fp32 kernels' sources (their counter records are kept apart from the bf16 ones)
KERNEL_SOURCES_F32 = ["paper_2606_25473_amd/csrc/attn_f32.hip", "paper_2606_25473_amd/csrc/mfma_common.hpp",
                      "paper_2606_25473_amd/csrc/schedule.hpp", "paper_2606_25473_amd/csrc/kernels.hpp"]


def kernel_source_hash(dtype="bf16"):
    h = hashlib.sha256()
    for p in KERNEL_SOURCES if dtype == "bf16" else KERNEL_SOURCES_F32:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def record_key(workload, mode, dtype="bf16"):
    """Key of a counter record in profiles/hbm_traffic.json."""
    return f"{workload}:{mode}" if dtype == "bf16" else f"{workload}:{mode}:{dtype}"


def zero_clean_flop(groups, half, D):
    """Flop per (batch, head) of the zero-clean JVP from the query-group table
    [(q0, q1, [(k0, k1), ...])]: 4D per pair of a clean query, 8D per (noisy query,
    clean key) pair, 12D per (noisy query, noisy key) pair."""
    total = 0
    for q0, q1, ks in groups:
        for r0, r1 in ((q0, min(q1, half)), (max(q0, half), q1)):
            if r1 <= r0:
                continue
            for k0, k1 in ks:
                clean_keys = max(0, min(k1, half) - k0)
                noisy_keys = max(0, k1 - max(k0, half))
                if r1 <= half:
                    total += (r1 - r0) * (clean_keys + noisy_keys) * 4 * D
                else:
                    total += (r1 - r0) * (clean_keys * 8 + noisy_keys * 12) * D
    return total


def profile_record(workload, mode, dtype="bf16"):
    """The committed rocprofv3 counter record of this workload (HBM bytes per launch,
    shader clock, MFMA busy fraction), if it was taken on the current kernel source;
    else an empty dict."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    if not os.path.exists(path):
        return {}
    with open(path) as f:
        rec = json.load(f)
    ent = rec.get(record_key(workload, mode, dtype))
    if not ent or ent.get("kernel_source_hash") != kernel_source_hash(dtype):
        return {}
    return ent


def cpu_baseline(w, x, out, mode, budget_s=15.0):
    """Time the fp64 CPU oracle on a bounded sample of rows of head (0, 0)."""
    # the oracle is only used on this leg
    from oracle import allowed_mask, attention_fwd, attention_jvp, attention_jvp_zero_clean
    try:
        from threadpoolctl import threadpool_info
        blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        cores = int(blas[0]["num_threads"]) if blas else os.cpu_count()
        blas_name = blas[0].get("internal_api", "?") if blas else "?"
    except Exception:  # threadpoolctl missing
        cores, blas_name = os.cpu_count(), "?"
    L, D = w.L, w.D
    half = L // 2
    h = {k: v[0:1, 0:1].float().cpu().numpy() for k, v in x.items()}
    offs = list(w.offsets) or None
    # rows spread evenly over the sequence so the per-row key-count mix matches the workload
    order = np.random.default_rng(0).permutation(L)
    done, t_used, pairs, flop = 0, 0.0, 0, 0
    errs = []
    got_o, got_do = out[0][0, 0], (None if mode == "fwd" else out[1][0, 0])
    batch = 256
    while t_used < budget_s and done < L:
        rows = np.sort(order[done:done + batch])
        t0 = time.perf_counter()
        if mode == "fwd":
            O, _ = attention_fwd(h["Q"], h["K"], h["V"], w.kind, offs, rows=rows)
            dO = None
        elif mode == "zc":
            O, dO, _ = attention_jvp_zero_clean(h["Q"], h["K"], h["V"], h["dQn"], h["dKn"], h["dVn"], offs,
                                                rows=rows)
        else:
            O, dO, _ = attention_jvp(h["Q"], h["K"], h["V"], h["dQ"], h["dK"], h["dV"], w.kind, offs, rows=rows)
        t_used += time.perf_counter() - t0
        done += len(rows)
        m = allowed_mask(w.kind, offs, L, rows)
        pairs += int(m.sum())
        if mode == "zc":
            clean_q = rows < half
            ck, nk = m[:, :half].sum(1), m[:, half:].sum(1)
            flop += int((4 * (ck + nk))[clean_q].sum() + (8 * ck + 12 * nk)[~clean_q].sum()) * D
        else:
            flop += int(m.sum()) * (4 if mode == "fwd" else 12) * D
        r = torch.from_numpy(rows).to(got_o.device)
        g = got_o.index_select(0, r).float().cpu().numpy()
        errs.append((np.linalg.norm(g - O[0, 0]) ** 2, np.linalg.norm(O[0, 0]) ** 2))
        if dO is not None:
            if mode == "zc":   # the GPU's dO holds the noisy rows only; the clean rows' is zero
                sel = rows >= half
                gd = np.zeros_like(dO[0, 0])
                gd[sel] = got_do.index_select(0, torch.from_numpy(rows[sel] - half).to(got_do.device)) \
                    .float().cpu().numpy()
            else:
                gd = got_do.index_select(0, r).float().cpu().numpy()
            errs.append((np.linalg.norm(gd - dO[0, 0]) ** 2, np.linalg.norm(dO[0, 0]) ** 2))
    rel = float(np.sqrt(sum(e for e, _ in errs) / max(sum(n for _, n in errs), 1e-300)))
    value = flop / t_used / 1e12
    return {"value": value, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": f"{done} query rows of head (0,0) spread over the {L}-token sequence "
                      f"({pairs} admissible pairs, {t_used:.1f} s, fp64 numpy/{blas_name})",
            "sample_rel_l2_vs_gpu": rel}


def cpu_baseline_bwd(w, x, out, budget_s=15.0):
    """Time the fp64 backward oracle on a bounded sample of query rows (gQ) of head (0, 0)."""
    from oracle import allowed_mask, attention_vjp  # the oracle is only used on this leg
    try:
        from threadpoolctl import threadpool_info
        blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        cores = int(blas[0]["num_threads"]) if blas else os.cpu_count()
    except Exception:
        cores = os.cpu_count()
    L, D = w.L, w.D
    h = {k: v[0:1, 0:1].float().cpu().numpy() for k, v in x.items()}
    offs = list(w.offsets) or None
    order = np.random.default_rng(0).permutation(L)
    done, t_used, pairs, errs = 0, 0.0, 0, []
    empty = np.array([], dtype=np.int64)
    while t_used < budget_s and done < L:
        rows = np.sort(order[done:done + 256])
        t0 = time.perf_counter()
        gQ, _, _, _ = attention_vjp(h["Q"], h["K"], h["V"], h["gO"], w.kind, offs, rows=rows, keys=empty)
        t_used += time.perf_counter() - t0
        done += len(rows)
        pairs += int(allowed_mask(w.kind, offs, L, rows).sum())
        g = out[0][0, 0].index_select(0, torch.from_numpy(rows).to(out[0].device)).float().cpu().numpy()
        errs.append((np.linalg.norm(g - gQ[0, 0]) ** 2, np.linalg.norm(gQ[0, 0]) ** 2))
    rel = float(np.sqrt(sum(e for e, _ in errs) / max(sum(n for _, n in errs), 1e-300)))
    # per pair the oracle evaluates the same five contractions (10 D flop) as the metric counts
    return {"value": pairs * 10 * D / t_used / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": f"gQ of {done} query rows of head (0,0) spread over the {L}-token sequence "
                      f"({pairs} admissible pairs, {t_used:.1f} s, fp64 numpy)",
            "sample_rel_l2_vs_gpu": rel}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=HEADLINE, choices=sorted(WORKLOADS))
    ap.add_argument("--forward", action="store_true", help="time attn_fwd instead of attn_jvp_fwd")
    ap.add_argument("--zero-clean", action="store_true",
                    help="time attn_jvp_fwd_zero_clean (teacher forcing, zero clean-half tangents)")
    ap.add_argument("--backward", action="store_true", help="time attn_bwd (gradients for a cotangent of O)")
    ap.add_argument("--dtype", choices=["bf16", "f32"],
                    help="run the workload's shape with inputs of this dtype (default: the workload's)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="first run one plain device copy of this many MiB (HBM counter calibration)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the kernels run on one "
              "GPU's share of heads; a multi-GPU (head-sharded) run is not implemented.", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)

    w = WORKLOADS[args.workload]
    if args.dtype and args.dtype != w.dtype:  # the same shape, mask and recipe in another dtype
        w = custom_workload(w.name, w.B, w.H, w.D, args.dtype, w.kind, offsets=list(w.offsets) or None,
                            L=w.L_full, tangent_std=w.tangent_std)
    if args.forward + args.zero_clean + args.backward > 1:
        ap.error("--forward, --zero-clean and --backward are exclusive")
    if args.zero_clean and w.kind != "teacher_forcing":
        ap.error("--zero-clean needs a teacher-forcing workload")
    mode = "fwd" if args.forward else ("zc" if args.zero_clean else ("bwd" if args.backward else "jvp"))
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    x = make_inputs(w, "cuda", seed=0)
    offs = list(w.offsets) or None
    q, k, v, dq, dk, dv = (x[n] for n in ("Q", "K", "V", "dQ", "dK", "dV"))
    B, H, L, D = q.shape
    o = torch.empty_like(q)
    do = torch.empty_like(q)
    lse = torch.empty((B, H, L), device=dev, dtype=torch.float32)
    half = L // 2
    if mode == "zc":  # tangents of the noisy half only
        for n in ("dQ", "dK", "dV"):
            x[n + "n"] = x.pop(n)[:, :, half:].contiguous()
        dqn, dkn, dvn = x["dQn"], x["dKn"], x["dVn"]
        del dq, dk, dv
        don = torch.empty_like(dqn)
    if mode == "bwd":  # cotangent: the dV draw; O and LSE from the forward (untimed)
        go = x.pop("dV")
        for n in ("dQ", "dK"):
            del x[n]
        del dq, dk, dv
        x["gO"] = go
        attn_fwd(q, k, v, w.kind, offs, out=(o, lse))
        gq, gk, gv = torch.empty_like(q), torch.empty_like(q), torch.empty_like(q)
        delta = torch.empty_like(lse)

    def step():
        if mode == "fwd":
            attn_fwd(q, k, v, w.kind, offs, out=(o, lse))
        elif mode == "zc":
            attn_jvp_fwd_zero_clean(q, k, v, dqn, dkn, dvn, offs, out=(o, don, lse))
        elif mode == "bwd":
            attn_bwd(q, k, v, o, go, lse, w.kind, offs, out=(gq, gk, gv, delta))
        else:
            attn_jvp_fwd(q, k, v, dq, dk, dv, w.kind, offs, out=(o, do, lse))

    if args.copy_calibration_mib:
        n = args.copy_calibration_mib * (1 << 20)
        src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)  # reads n bytes, writes n bytes
        torch.cuda.synchronize()
        del src, dst

    def outputs():
        if mode == "fwd":
            return (o, lse)
        if mode == "zc":
            return (o, don, lse)
        if mode == "bwd":
            return (gq, gk, gv, delta)
        return (o, do, lse)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # outputs of the first launch (untimed copy), compared bit for bit with the last timed one
    first = [t.clone() for t in outputs()] if args.warmup > 0 else None
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream(dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(args.steps):
        step()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    deterministic = None if first is None else all(torch.equal(a, b) for a, b in zip(first, outputs()))
    del first
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(args.steps)]
    kernel_ms = ev[0].elapsed_time(ev[-1]) / args.steps
    ms_per_step = wall * 1e3 / args.steps

    pairs = count_unmasked_pairs(w.kind, offs, L)
    computed = count_computed_pairs(w.kind, offs, L, D)
    if mode == "zc":
        flop = zero_clean_flop(query_groups(w.kind, offs, L), half, D) * B * H
    else:
        flop = pairs * {"fwd": 4, "bwd": 10, "jvp": 12}[mode] * D * B * H
    value = flop / (ms_per_step * 1e-3) / 1e12
    achieved = flop / (kernel_ms * 1e-3) / 1e12
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_FP32_TFLOPS
    prof = profile_record(w.name, mode, w.dtype)
    traffic = prof.get("hbm_bytes_per_launch")
    if mode == "bwd" and traffic is not None:
        # a backward call is two launches; the record of the first (query-tile) pass is separate
        traffic = traffic + profile_record(w.name, "bwd_dq", w.dtype).get("hbm_bytes_per_launch", float("nan"))
    res = {
        "metric": MODE_METRIC[mode] if w.dtype == "bf16" else MODE_METRIC[mode].replace("bf16", "fp32"),
        "value": round(value, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": dict(w.describe(), op={"fwd": "attn_fwd", "zc": "attn_jvp_fwd_zero_clean",
                                         "bwd": "attn_bwd"}.get(mode, "attn_jvp_fwd")),
        "pct_peak": round(100 * achieved / peak, 2),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": round(peak, 1),
                     "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                     "traffic": None if traffic is None else round(traffic)},
        "kernel_ms": {"mean": round(kernel_ms, 4), "median": round(float(np.median(per)), 4),
                      "min": round(min(per), 4)},
        "unmasked_pairs_per_head": pairs,
        # pairs the bf16 JVP kernel's 256-row tile plans evaluate, masked lanes included (the
        # other kernels tile differently: not reported for them)
        "computed_over_unmasked": round(computed / pairs, 4) if w.dtype == "bf16" and mode == "jvp" else None,
        # every output of the last timed launch equals the first launch's bit for bit
        "deterministic": deterministic,
    }
    if prof.get("clock_ghz") and prof.get("trace_kernel_ms"):
        # The committed profile run of this kernel source (possibly on another box, whose shader
        # clock under this load may differ): its mean launch time, its clock (the nominal peak
        # assumes 2.4 GHz) and its matrix-core busy fraction, and the roofline fraction at that
        # clock from that run's own launch time.
        clk, pms = prof["clock_ghz"], prof["trace_kernel_ms"]
        if mode == "bwd":  # a call is two launches: add the query-tile pass's time
            pms += profile_record(w.name, "bwd_dq", w.dtype).get("trace_kernel_ms", float("nan"))
        res["roofline"]["profile"] = {
            "kernel_ms": round(pms, 4), "clock_ghz": round(clk, 3),
            "frac_at_clock": round(flop / (pms * 1e-3) / 1e12 / (peak * clk / 2.4), 4),
            "mfma_busy_cycles_frac": round(prof.get("mfma_busy", 0.0), 4)}
    if mode == "zc":
        # the dense JVP of the same function (tangents zero-padded over the clean half)
        pad = {n: torch.cat([torch.zeros_like(x[n + "n"]), x[n + "n"]], dim=2) for n in ("dQ", "dK", "dV")}
        o2, do2 = torch.empty_like(q), torch.empty_like(q)
        for _ in range(args.warmup):
            attn_jvp_fwd(q, k, v, pad["dQ"], pad["dK"], pad["dV"], w.kind, offs, out=(o2, do2, lse))
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(args.steps):
            attn_jvp_fwd(q, k, v, pad["dQ"], pad["dK"], pad["dV"], w.kind, offs, out=(o2, do2, lse))
        e1.record(stream)
        torch.cuda.synchronize()
        dense_ms = e0.elapsed_time(e1) / args.steps
        res["dense_jvp_kernel_ms"] = round(dense_ms, 4)
        res["speedup_vs_dense_jvp"] = round(dense_ms / kernel_ms, 3)
        res["zero_clean_flop_over_dense"] = round(flop / (pairs * 12 * D * B * H), 4)
        del pad, o2, do2
        step()  # restore the outputs the CPU leg compares against
        torch.cuda.synchronize()
    if not args.no_cpu and mode != "bwd":
        res["cpu_baseline"] = cpu_baseline(w, x, (o, don if mode == "zc" else do, lse), mode, args.cpu_budget)
    if not args.no_cpu and mode == "bwd":
        res["cpu_baseline"] = cpu_baseline_bwd(w, x, (gq, gk, gv), args.cpu_budget)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
