"""Host logic of bench.py, on the CPU: the refusal of more than one GPU, the arithmetic of the
counter summaries (calibration by the device copy, grouping of dispatches and instances, which
dispatches count), and the source-digest guard on the committed traffic figures.

The counter files here are synthetic, in the layout rocprofv3 writes (one row per counter
instance of a dispatch), with values chosen so that every expected figure is a plain product."""
import argparse
import csv
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

FIELDS = ["Dispatch_Id", "Kernel_Name", "Grid_Size", "Counter_Name", "Counter_Value", "Start_Timestamp"]
COPY = "__amd_rocclr_copyBuffer"
STREAM = "void curvefp::quantize_rows_kernel<curvefp::Fmt<4, 3, 1, 1>, true, 2, true, true>(args)"
QP = "void curvefp::quantize_prepare_kernel<curvefp::Fmt<3, 3, 1, 1>, true, 4, 1>(args)"
GEMM = "void curvefp::gemm_ws_kernel<24, false>(args)"
VENDOR = "Cijk_Ailk_Bljk_HHS_BH_MT256x256x64"


def write_counters(d, counter, dispatches):
    """dispatches: (id, kernel, grid, [instance values]); each instance is one row."""
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "pmc_counter_collection.csv"), "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=FIELDS)
        w.writeheader()
        for did, kernel, grid, values in dispatches:
            for i, v in enumerate(values):
                w.writerow({"Dispatch_Id": did, "Kernel_Name": kernel, "Grid_Size": grid, "Counter_Name": counter,
                            "Counter_Value": v, "Start_Timestamp": 1000 * did + i})


def key_values(text):
    return dict(l.split("=", 1) for l in text.splitlines() if "=" in l and " " not in l.split("=", 1)[0])


def test_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], cwd=ROOT,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_stream_summary_calibration(tmp_path, capsys):
    # the copy moves 256 MiB each way; FETCH_SIZE reports half of it, WRITE_SIZE all of it
    copy_kib = bench.COPY_BYTES / 1024
    fetch, write = str(tmp_path / "fetch"), str(tmp_path / "write")
    write_counters(fetch, "FETCH_SIZE", [
        (1, COPY, 512, [7.0]),                              # a small staging copy: not the calibration
        (2, COPY, 131072, [copy_kib / 4, copy_kib / 4]),    # two instances summed: 0.5x
        (3, COPY, 131072, [copy_kib / 2]),
        (4, STREAM, 2097152, [5.0]),                        # a smaller launch of the same kernel
        (5, STREAM, 8388608, [300000.0, 200000.0]),
        (6, STREAM, 8388608, [500000.0]),
        (6, STREAM, 8388608, [500000.0]),                   # the same record repeated: counted once
    ])
    write_counters(write, "WRITE_SIZE", [
        (2, COPY, 131072, [copy_kib]),
        (5, STREAM, 8388608, [250000.0, 250000.0]),
        (6, STREAM, 8388608, [600000.0]),
    ])
    bench.summarize_stream_pmc(argparse.Namespace(summarize_stream_pmc=[fetch, write], gemm="prepared"))
    kv = key_values(capsys.readouterr().out)
    assert float(kv["fetch_bytes"]) == pytest.approx(500000.0 * 1024 / 0.5, rel=1e-9)
    assert float(kv["write_bytes"]) == pytest.approx(550000.0 * 1024, rel=1e-9)
    assert kv["kernel_source_sha256"] == bench.kernel_source_digest(bench.QUANTIZE_SOURCES)


def test_prepared_summary_attribution(tmp_path, capsys):
    # inference workload, 2048 x 4096 x 4096 bf16 -> E3C3: one wave per row of 4096, four rows per
    # workgroup, so a quantize-prepare grid is 64 workgroups of 256 work-items per tile of 256 rows
    from paper_2608_10010_amd import curvefp as cf
    from paper_2608_10010_amd import workloads as W
    w = W.get("inference")
    per_tile = 64 * 256
    g_act, g_wt = (w.M // 256) * per_tile, (w.N // 256) * per_tile
    g_pair = g_act + g_wt
    copy_kib = bench.COPY_BYTES / 1024
    fetch, write = str(tmp_path / "fetch"), str(tmp_path / "write")
    write_counters(fetch, "FETCH_SIZE", [
        (1, COPY, 131072, [copy_kib / 2]),
        (2, QP, g_pair, [1000.0, 1000.0]),
        (3, QP, g_pair, [2000.0]),
        (4, GEMM, 65536, [40000.0]),
        (5, GEMM, 65536, [20000.0, 20000.0]),
        (6, GEMM, 2048, [9.0]),            # another configuration's GEMM: fewer dispatches, ignored
        (7, QP, g_act, [300.0]),
        (8, QP, g_wt, [700.0]),
        (9, VENDOR, 65536, [80000.0]),
    ])
    write_counters(write, "WRITE_SIZE", [
        (1, COPY, 131072, [copy_kib]),
        (2, QP, g_pair, [5000.0]),
        (3, QP, g_pair, [5000.0]),
        (4, GEMM, 65536, [8000.0]),
        (5, GEMM, 65536, [8000.0]),
        (6, GEMM, 2048, [1.0]),
        (7, QP, g_act, [3000.0]),
        (8, QP, g_wt, [2000.0]),
        (9, VENDOR, 65536, [4000.0]),
    ])
    bench.summarize_pmc_prepared(argparse.Namespace(summarize_pmc=[fetch, write], gemm="prepared",
                                                    workload="inference"))
    out = capsys.readouterr().out
    kv = key_values(out)
    gemm_fetch, gemm_write = 40000.0 * 1024 / 0.5, 8000.0 * 1024
    pair = 2000.0 * 1024 / 0.5 + 5000.0 * 1024
    assert float(kv["fetch_bytes_per_launch"]) == pytest.approx(gemm_fetch, rel=1e-9)
    assert float(kv["write_bytes_per_launch"]) == pytest.approx(gemm_write, rel=1e-9)
    assert float(kv["traffic_bytes_per_launch"]) == pytest.approx(gemm_fetch + gemm_write, rel=1e-9)
    # the step: the pair launch, then the GEMM (the one-operand launches are not part of it)
    assert float(kv["call_traffic_bytes"]) == pytest.approx(pair + gemm_fetch + gemm_write, rel=1e-9)
    assert kv["kernel_source_sha256"] == bench.kernel_source_digest()
    # algorithmic bytes of the pair row: both sources, codes, scales, planes and row maxima, and the
    # activations' fp32 reconstruction
    bpe = bench.quantize_bytes_per_elem(w.fmt, w.dtype)
    alg = (w.M * w.K * (bpe + 4.0) + cf.curvefp_prepared_bytes(w.M, w.K)
           + w.N * w.K * bpe + cf.curvefp_prepared_bytes(w.N, w.K))
    pair_row = next(l for l in out.splitlines() if l.startswith("| `quantize_prepare_pair"))
    assert pair_row.rstrip(" |").endswith(f"{alg / 1e6:.1f}")


def test_committed_traffic_matches_sources():
    t = bench.measured_traffic("sweep8b_gateup_e4c3_8192x14336x4096", "prepared")
    assert t is not None and t > 0
    s = bench.measured_stream_traffic()
    assert s is not None and s > 0


def test_traffic_void_when_sources_change(monkeypatch):
    monkeypatch.setattr(bench, "kernel_source_digest", lambda sources=None: "0" * 64)
    assert bench.measured_traffic("sweep8b_gateup_e4c3_8192x14336x4096", "prepared") is None
    assert bench.measured_stream_traffic() is None


def test_profile_commands_are_the_bench_commands():
    """The committed counter summaries name the commands bench.py would give for them today."""
    for name in ("gemm_prepared_sweep8b_gateup_e4c3_8192x14336x4096_traffic.md",
                 "quantize_stream_e4c3_1gib_traffic.md"):
        text = open(os.path.join(ROOT, "profiles", name)).read()
        for cmd in bench.pmc_commands("prepared"):
            assert cmd in text, (name, cmd)
