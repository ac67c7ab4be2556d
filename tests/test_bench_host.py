"""Host logic of the measurement (CPU only).

* bench.py's flop count of the zero-clean JVP against brute-force counting over the mask
  built from its definition (4 D per pair of a clean query, 8 D per (noisy query, clean
  key) pair, 12 D per (noisy query, noisy key) pair), and its dense counts against the
  closed form of the pair count;
* bench.py refuses more than one GPU with a message, before touching any device;
* a counter record taken on other kernel sources is ignored (traffic reported as null);
* profile_summary's calibration of FETCH_SIZE / WRITE_SIZE by the copy kernel, on
  synthetic rocprofv3 CSV output.
"""
import csv
import json
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
from oracle import allowed_mask
from paper_2606_25473_amd import count_unmasked_pairs, profile_summary, query_groups

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _brute_zero_clean_flop(offsets, D):
    L = 2 * offsets[-1]
    half = L // 2
    m = allowed_mask("teacher_forcing", offsets, L)
    clean_q = m[:half].sum()
    noisy_clean = m[half:, :half].sum()
    noisy_noisy = m[half:, half:].sum()
    return int(4 * D * clean_q + 8 * D * noisy_clean + 12 * D * noisy_noisy)


@pytest.mark.parametrize("offsets", [[0, 5, 10, 15], [0, 1, 3, 7, 40, 41, 90], [0, 64], [0, 1, 2, 3, 4]])
def test_zero_clean_flop_matches_brute_force(offsets):
    L = 2 * offsets[-1]
    for D in (64, 128):
        got = bench.zero_clean_flop(query_groups("teacher_forcing", offsets, L), L // 2, D)
        assert got == _brute_zero_clean_flop(offsets, D)


@pytest.mark.parametrize("N,C", [(7, 4680), (21, 1560), (3, 5)])
def test_dense_pair_count_closed_form(N, C):
    offsets = [C * i for i in range(N + 1)]
    assert count_unmasked_pairs("teacher_forcing", offsets, 2 * N * C) == C * C * N * (N + 1)


def test_zero_clean_flop_ratio_on_the_headline_layout():
    # 4 x 28 + 8 x 21 + 12 x 7 = 364 of 12 x 56 = 672 units of C^2 D
    C, N = 4680, 7
    offsets = [C * i for i in range(N + 1)]
    zc = bench.zero_clean_flop(query_groups("teacher_forcing", offsets, 2 * N * C), N * C, 128)
    dense = 12 * 128 * count_unmasked_pairs("teacher_forcing", offsets, 2 * N * C)
    assert zc * 672 == dense * 364


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, cwd=ROOT, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_counter_record_of_other_sources_is_ignored(tmp_path, monkeypatch):
    (tmp_path / "profiles").mkdir()
    rec = {"w:jvp": {"hbm_bytes_per_launch": 123.0, "kernel_source_hash": "current"},
           "w:fwd": {"hbm_bytes_per_launch": 456.0, "kernel_source_hash": "older"},
           "w:bwd:f32": {"hbm_bytes_per_launch": 789.0, "kernel_source_hash": "current"}}
    (tmp_path / "profiles" / "hbm_traffic.json").write_text(json.dumps(rec))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_hash", lambda dtype="bf16": "current")
    assert bench.profile_record("w", "jvp")["hbm_bytes_per_launch"] == 123.0
    assert bench.profile_record("w", "fwd") == {}
    assert bench.profile_record("w", "zc") == {}
    # fp32 records sit under their own keys
    assert bench.profile_record("w", "bwd", "f32")["hbm_bytes_per_launch"] == 789.0
    assert bench.profile_record("w", "bwd") == {} and bench.profile_record("w", "jvp", "f32") == {}


def test_kernel_source_hash_covers_the_kernel_sources():
    assert all(os.path.exists(os.path.join(ROOT, p)) for p in bench.KERNEL_SOURCES + bench.KERNEL_SOURCES_F32)
    assert len(bench.kernel_source_hash()) == 16
    # the bf16 and fp32 records depend on different sources and are kept apart
    assert bench.kernel_source_hash("f32") != bench.kernel_source_hash("bf16")
    assert bench.record_key("w", "jvp") == "w:jvp" and bench.record_key("w", "jvp", "f32") == "w:jvp:f32"


def _counter_csv(path, rows):
    path.mkdir(parents=True)
    with open(path / "x_counter_collection.csv", "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Kernel_Name", "Counter_Name", "Counter_Value",
                                          "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        for r in rows:
            w.writerow(r)


def test_profile_summary_calibrates_counters_with_the_copy(tmp_path, capsys):
    kern = "void attn::(anonymous namespace)::attn_mfma_kernel<128, 1, 8>(attn::AttnArgs)"
    copy = "__amd_rocclr_copyBuffer"
    mib = 64
    # the copy moves 64 MiB each way: FETCH_SIZE reads 32768 units (2 KiB each), WRITE_SIZE
    # 65536 units (1 KiB each); the attention kernel's three dispatches read 1000, 1100, 900
    # units and write 10, 12, 11 units
    _counter_csv(tmp_path / "fetch", [dict(Kernel_Name=copy, Counter_Name="FETCH_SIZE", Counter_Value=32768,
                                           Start_Timestamp=0, End_Timestamp=1)] +
                 [dict(Kernel_Name=kern, Counter_Name="FETCH_SIZE", Counter_Value=v, Start_Timestamp=0,
                       End_Timestamp=1) for v in (1000, 1100, 900)])
    _counter_csv(tmp_path / "write", [dict(Kernel_Name=copy, Counter_Name="WRITE_SIZE", Counter_Value=65536,
                                           Start_Timestamp=0, End_Timestamp=1)] +
                 [dict(Kernel_Name=kern, Counter_Name="WRITE_SIZE", Counter_Value=v, Start_Timestamp=0,
                       End_Timestamp=1) for v in (10, 12, 11)])
    profile_summary.main(["--fetch", str(tmp_path / "fetch"), "--write", str(tmp_path / "write"),
                          "--copy-mib", str(mib), "--op", "jvp"])
    out = capsys.readouterr().out
    read, write = 1000 * 2048, 11 * 1024  # medians x bytes per unit
    assert f"HBM traffic per launch: {(read + write) / 1e9:.3f} GB" in out
    assert "2048.0 B/unit" in out and "1024.0 B/unit" in out


def test_profile_summary_picks_the_kernel_of_the_op():
    names = {"fwd": "attn_mfma_kernel<128, 0, 4>", "jvp": "attn_mfma_kernel<128, 1, 8>",
             "zc": "attn_mfma_kernel<64, 2, 8>", "bwd": "attn_bwd_dkdv_kernel<128>",
             "bwd_dq": "attn_bwd_dq_kernel<64>"}
    for op, name in names.items():
        pick = profile_summary.attn_kernel_of(op)
        assert pick(f"void attn::(anonymous namespace)::{name}(attn::AttnArgs)")
        assert not any(pick(n) for o, n in names.items() if o != op)
    f32 = {"fwd": "attn_f32_kernel<128, false>", "jvp": "attn_f32_kernel<64, true>",
           "bwd": "attn_f32_bwd_dkdv_kernel<128>", "bwd_dq": "attn_f32_bwd_dq_kernel<64>"}
    for op, name in f32.items():
        pick = profile_summary.attn_kernel_of(op, "f32")
        assert pick(f"void attn::(anonymous namespace)::{name}(attn::AttnArgs)")
        assert not any(pick(n) for o, n in f32.items() if o != op)
        assert not any(pick(n) for n in names.values())
    assert profile_summary.attn_kernel_of("zc", "f32")("attn_f32_kernel<128, true>(attn::AttnArgs)")


def test_matrix_flop_line_compares_with_the_computed_pairs():
    from paper_2606_25473_amd import count_computed_pairs, count_unmasked_pairs
    from paper_2606_25473_amd.profile_summary import matrix_flop_line
    from paper_2606_25473_amd.workloads import WORKLOADS
    w = WORKLOADS["wan1.3b_chunkwise_tf"]
    offs = list(w.offsets)
    comp = count_computed_pairs(w.kind, offs, w.L, w.D) * w.B * w.H
    pairs = count_unmasked_pairs(w.kind, offs, w.L) * w.B * w.H
    line = matrix_flop_line("jvp", w.name, comp * 12 * w.D)
    assert "1.0000 x that of the pairs the tile plans compute" in line
    assert f"{comp / pairs:.4f} x the 12 D flop of the admissible pairs" in line
    assert "admissible" in matrix_flop_line("bwd", w.name, pairs * 8 * w.D)
    assert "x the" not in matrix_flop_line("zc", w.name, 1.0e13)

