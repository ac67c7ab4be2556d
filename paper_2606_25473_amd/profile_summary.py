"""Summarise rocprofv3 CSV output of a bench.py run into a short text report.

    python -m paper_2606_25473_amd.profile_summary --trace DIR [--fetch DIR --write DIR]
        [--copy-mib N] [--workload NAME] [--op jvp|fwd|zc|bwd|bwd_dq] [--dtype bf16|f32]
        [--record profiles/hbm_traffic.json]

--trace: a ``rocprofv3 --kernel-trace --stats -f csv`` output directory;
--fetch/--write: ``rocprofv3 --pmc FETCH_SIZE`` / ``--pmc WRITE_SIZE`` output
directories of a bench run that also did ``--copy-calibration-mib N``.  The
copy kernel of N MiB (N MiB read, N MiB written) calibrates the counters: the
attention kernel's bytes = its counter value x (N MiB / the copy's counter).
With --record, the per-launch HBM bytes are stored for bench.py together with
a hash of the kernel sources (bench.py ignores the record once they change).
"""
import argparse
import csv
import glob
import json
import os
import re
import statistics

# the bf16 kernel whose counters stand for each op: attn_mfma_kernel<D, mode, waves> for the
# forward, JVP and zero-clean JVP; the key-tile pass (the longer one) for the backward
OP_KERNEL = {"fwd": r"attn_mfma_kernel<\d+, 0, \d+>", "jvp": r"attn_mfma_kernel<\d+, 1, \d+>",
             "zc": r"attn_mfma_kernel<\d+, 2, \d+>", "bwd": r"attn_bwd_dkdv_kernel<\d+>",
             "bwd_dq": r"attn_bwd_dq_kernel<\d+>"}
# the fp32 kernels (one kernel serves the dense and the zero-clean JVP)
OP_KERNEL_F32 = {"fwd": r"attn_f32_kernel<\d+, false>", "jvp": r"attn_f32_kernel<\d+, true>",
                 "zc": r"attn_f32_kernel<\d+, true>", "bwd": r"attn_f32_bwd_dkdv_kernel<\d+>",
                 "bwd_dq": r"attn_f32_bwd_dq_kernel<\d+>"}


# matrix-core flop per admissible (query, key) pair in each op's kernel (the zero-clean JVP's
# varies with the pair's halves)
OP_FLOP_PER_PAIR = {"fwd": 4, "jvp": 12, "zc": None, "bwd": 8, "bwd_dq": 6}


def matrix_flop_line(op, workload, mflop, dtype="bf16"):
    """The counted matrix-core flop of one dispatch against the flop of the admissible pairs
    (and, for the bf16 JVP, of the pairs its 256-row tile plans compute, masked lanes
    included)."""
    from .binding import count_computed_pairs, count_unmasked_pairs
    from .workloads import WORKLOADS
    w = WORKLOADS[workload]
    offs = list(w.offsets) or None
    line = f"matrix-core flop ({mops_counter(dtype)} x 512): {mflop:.4g} per dispatch"
    f = OP_FLOP_PER_PAIR[op]
    if f:
        pairs = count_unmasked_pairs(w.kind, offs, w.L) * w.B * w.H
        line += f" = {mflop / (pairs * f * w.D):.4f} x the {f} D flop of the admissible pairs"
        if op == "jvp" and dtype == "bf16":
            comp = count_computed_pairs(w.kind, offs, w.L, w.D) * w.B * w.H
            line += f", {mflop / (comp * f * w.D):.4f} x that of the pairs the tile plans compute"
    return line


def mops_counter(dtype):
    """The counter of matrix-core operations (512 flop each) of the dtype's kernels."""
    return "SQ_INSTS_VALU_MFMA_MOPS_BF16" if dtype == "bf16" else "SQ_INSTS_VALU_MFMA_MOPS_F32"


def attn_kernel_of(op, dtype="bf16"):
    """Predicate on rocprofv3 kernel names selecting the kernel of ``op`` for ``dtype``."""
    pat = re.compile((OP_KERNEL if dtype == "bf16" else OP_KERNEL_F32)[op])
    return lambda name: bool(pat.search(name))


def _rows(d, suffix):
    out = []
    for f in glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True):
        with open(f, newline="") as fh:
            out.extend(csv.DictReader(fh))
    return out


def kernel_stats(d):
    rows = _rows(d, "kernel_stats.csv")
    return [(r["Name"], int(r["Calls"]), float(r["AverageNs"]), float(r["MinNs"]), float(r["MaxNs"]),
             float(r.get("Percentage", 0) or 0)) for r in rows]


def counter_per_dispatch(d, counter):
    """{kernel name: [value per dispatch]} for one counter."""
    res = {}
    for r in _rows(d, "counter_collection.csv"):
        if r.get("Counter_Name") != counter:
            continue
        res.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return res


def _pick(d, key):
    """First (name, values) whose name contains ``key`` (a string) or satisfies it (a predicate)."""
    for name, vals in d.items():
        if (key(name) if callable(key) else key in name):
            return name, vals
    return None, []


def main(argv=None):
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-mib", type=int, default=0)
    ap.add_argument("--workload", default="wan1.3b_chunkwise_tf")
    ap.add_argument("--op", default="jvp", choices=sorted(OP_KERNEL))
    ap.add_argument("--dtype", default="bf16", choices=["bf16", "f32"])
    ap.add_argument("--record")
    ap.add_argument("--pmc", nargs="*", default=[], help="counter-collection output dirs to list")
    a = ap.parse_args(argv)
    lines = []
    derived = {}
    if a.trace:
        st = sorted(kernel_stats(a.trace), key=lambda r: -r[2] * r[1])
        mine = [r for r in st if attn_kernel_of(a.op, a.dtype)(r[0])]
        if mine:
            derived["trace_kernel_ms"] = mine[0][2] / 1e6  # mean launch time under the tracer
        lines.append("| kernel | calls | avg ms | min ms | max ms | % time |")
        lines.append("|---|---|---|---|---|---|")
        for name, calls, avg, mn, mx, pct in st[:8]:
            lines.append(f"| {name[:90]} | {calls} | {avg / 1e6:.4f} | {mn / 1e6:.4f} | {mx / 1e6:.4f} | {pct:.1f} |")
    traffic = None
    if a.fetch and a.write and a.copy_mib:
        nbytes = a.copy_mib * (1 << 20)
        out = {}
        for label, d, cnt in (("read", a.fetch, "FETCH_SIZE"), ("write", a.write, "WRITE_SIZE")):
            per = counter_per_dispatch(d, cnt)
            # the calibration copy is a device-to-device hipMemcpy (runtime blit kernel)
            cname, cvals = _pick(per, "copyBuffer")
            kname, kvals = _pick(per, attn_kernel_of(a.op, a.dtype))
            if not cvals or not kvals:
                lines.append(f"{cnt}: copy or attention kernel missing in {d}")
                continue
            copy_kib = max(cvals)          # the largest blit is the calibration copy
            factor = nbytes / copy_kib      # bytes per counter unit
            att = statistics.median(kvals) * factor
            out[label] = att
            lines.append(f"{cnt}: copy kernel `{cname[:60]}` {copy_kib:.0f} units for {nbytes} B "
                         f"-> {factor:.1f} B/unit; attention kernel median {statistics.median(kvals):.0f} "
                         f"units/dispatch over {len(kvals)} dispatches = {att / 1e9:.3f} GB")
        if len(out) == 2:
            traffic = out["read"] + out["write"]
            lines.append(f"HBM traffic per launch: {traffic / 1e9:.3f} GB "
                         f"(read {out['read'] / 1e9:.3f} + write {out['write'] / 1e9:.3f})")
    is_attn = attn_kernel_of(a.op, a.dtype)
    for d in a.pmc:
        per, dur = {}, []
        for r in _rows(d, "counter_collection.csv"):
            if is_attn(r["Kernel_Name"]):
                per.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
                if r["Counter_Name"] == "GRBM_GUI_ACTIVE":
                    dur.append(float(r["End_Timestamp"]) - float(r["Start_Timestamp"]))
        xcc = 8
        for info in _rows(d, "agent_info.csv"):
            if info.get("Num_Xcc", "0") not in ("", "0"):
                xcc = int(info["Num_Xcc"])
        for cnt in sorted(per):
            lines.append(f"{cnt}: median {statistics.median(per[cnt]):.6g} per dispatch ({len(per[cnt])} dispatches)")
        if "GRBM_GUI_ACTIVE" in per and dur:
            # the counter is summed over the XCDs; per-XCD cycles / dispatch time = shader clock
            cyc = statistics.median(per["GRBM_GUI_ACTIVE"]) / xcc
            derived["clock_ghz"] = cyc / statistics.median(dur)
            lines.append(f"shader clock during the kernel: {derived['clock_ghz']:.3f} GHz "
                         f"(GRBM_GUI_ACTIVE / {xcc} XCDs / dispatch time {statistics.median(dur) / 1e6:.3f} ms)")
            if mops_counter(a.dtype) in per:
                mflop = statistics.median(per[mops_counter(a.dtype)]) * 512
                lines.append(matrix_flop_line(a.op, a.workload, mflop, a.dtype))
            if "SQ_VALU_MFMA_BUSY_CYCLES" in per:
                simds = 1024
                util = statistics.median(per["SQ_VALU_MFMA_BUSY_CYCLES"]) / (cyc * simds)
                derived["mfma_busy"] = util
                lines.append(f"MFMA busy: {100 * util:.1f} % of SIMD cycles "
                             f"(SQ_VALU_MFMA_BUSY_CYCLES / (per-XCD GRBM_GUI_ACTIVE x {simds} SIMDs))")
    print("\n".join(lines))
    if a.record and traffic is not None:
        import importlib.util
        root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
        spec = importlib.util.spec_from_file_location("bench", os.path.join(root, "bench.py"))
        bench = importlib.util.module_from_spec(spec)
        spec.loader.exec_module(bench)
        rec = {}
        if os.path.exists(a.record):
            with open(a.record) as f:
                rec = json.load(f)
        ent = {"hbm_bytes_per_launch": traffic, "kernel_source_hash": bench.kernel_source_hash(a.dtype)}
        ent.update(derived)
        rec[bench.record_key(a.workload, a.op, a.dtype)] = ent
        with open(a.record, "w") as f:
            json.dump(rec, f, indent=1, sort_keys=True)


if __name__ == "__main__":
    main()
