"""Benchmark of the CurveFP hot path on one MI355X.

One step = one pass of the whole path over one batch of the largest workload,
the 8B-shaped gate/up projection in CurveFP8 E4C3 (activations 8192 x 4096 bf16
N(0,1), weights 14336 x 4096 bf16 N(0, 0.02), both block 32; 962.1 GFLOP):

    quantize(activations) -> quantize(weights) -> CurveFP GEMM -> dequantize(activation codes)

Prints one JSON line.  `value` is whole-step throughput in GEMM TFLOP/s
(2 M N K per step over the measured step time, inputs resident in HBM).
The GEMM is curvefp_gemm_ws by default (codes expanded once into a workspace
that is allocated before the timed region, like C); --gemm fused times the
allocation-free curvefp_gemm instead.  Per-call times come from HIP events
recorded on the stream the library launches on.  The roofline object is for the
GEMM call (the dominant part: its expansion and GEMM kernels together).

Also reported, each in a key of its own:
  configs          every configuration of the workload set timed on its own: the tiny
                   E4C3 case, the E3C3 inference GEMM, the 7B up-projection forward
                   (E4C3, weights quantize-transposed), its E5C2 dgrad and wgrad, and the
                   12 GEMMs of the 8B layer sweep (QKV, O, gate/up, down x E4C3, E5C2,
                   E3C3): quantize GB/s of both operands and GEMM TFLOP/s and roofline
                   fraction, each the median of individually timed calls;
  quantize_stream  a 1 GiB bf16 source (larger than the 256 MB Infinity Cache)
                   quantized to E4C3, against 8 TB/s and against a measured 1 GiB
                   device copy in the same run;
  backward_mixed   the two backward GEMMs of the 7B up-projection as the paper runs
                   them (E5C2 output gradients times the reused E4C3 forward codes);
  radix_variants, static_scales, requant, block_sizes
                   the inference workload in the E4C3 radix variants, with
                   reconstruction-error scale search, with its output requantized in
                   the epilogue, and with one scale per 32, 64, 512 or K elements;
  cpu_baseline     the CPU oracle on a bounded row sample of the headline workload,
                   with the host's CPU model, affinity and thread count.
--cpu-baseline-table times the oracle on every configuration instead (full size
for the two smallest, every 32nd row of A for the rest) and prints that table.
"""

import argparse
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "CurveFP GEMM TFLOP/s + quantize GB/s (1×MI355X, % roofline), oracle-exact"
# the largest single-GPU configuration: the 8B gate/up projection in the forward format
HEADLINE = "sweep_gateup_E4C3"
SWEEPS = [f"sweep_{layer}_{fmt}" for layer in ("qkv", "o", "gateup", "down") for fmt in ("E4C3", "E5C2", "E3C3")]
# every configuration of the workload set, in order: tiny, inference, 7B forward, dgrad, wgrad, 8B sweep
CONFIGS = ["tiny", "inference", "fwd", "dgrad", "wgrad"] + SWEEPS
HBM_PEAK_GBS = 8000.0
F16_DENSE_PEAK_TFLOPS = 2500.0   # MI355X dense fp16/bf16 MFMA


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default=HEADLINE)
    p.add_argument("--gemm", choices=["prepared", "ws", "fused"], default="prepared",
                   help="prepared: both operands quantized and expanded for the GEMM by one "
                        "curvefp_quantize_prepare_pair launch (--separate-step: quantize, prepare and "
                        "dequantize calls on two streams), then curvefp_gemm_prepared; ws: quantize calls, then "
                        "curvefp_gemm_ws (both expansions "
                        "and the GEMM in one call) with a workspace allocated before the timed region; "
                        "fused: curvefp_gemm (expansion inside the GEMM kernel)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-stream", action="store_true")
    p.add_argument("--no-backward", action="store_true",
                   help="skip the mixed-format backward GEMMs (E5C2 gradients x reused E4C3 codes)")
    p.add_argument("--no-requant", action="store_true",
                   help="skip the GEMM with output requantization (fused epilogue vs GEMM + quantize)")
    p.add_argument("--no-blocks", action="store_true",
                   help="skip the block-size sweep (G = 32, 64, 512, K) of the inference workload")
    p.add_argument("--no-static", action="store_true",
                   help="skip the static-scale (reconstruction-MSE search) quantize of the inference weight")
    p.add_argument("--no-radix", action="store_true",
                   help="skip the E4C3 radix variants (r = 2, 2^(8/9), 2^(3/4)) on the inference operands")
    p.add_argument("--serial-step", action="store_true",
                   help="run the step's calls one after another on one stream")
    p.add_argument("--separate-step", action="store_true",
                   help="prepared path: quantize, dequantize and prepare as separate calls instead of "
                        "curvefp_quantize_prepare (one launch per operand)")
    p.add_argument("--no-reference", action="store_true",
                   help="skip the vendor fp16 GEMM (torch.matmul) of the same M, N and 3K")
    p.add_argument("--no-configs", action="store_true",
                   help="skip the per-configuration timings (every workload of the set)")
    p.add_argument("--cpu-seconds", type=float, default=15.0)
    p.add_argument("--cpu-baseline-table", action="store_true",
                   help="time the CPU oracle on every configuration (full size for the tiny and "
                        "inference cases, every 32nd row of A otherwise), print the table, then exit")
    p.add_argument("--copy-calibration", action="store_true",
                   help="also run a plain 256 MiB device copy three times (counter calibration)")
    p.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                   help="print the traffic summary of two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) "
                        "of this script with --copy-calibration, then exit")
    p.add_argument("--summarize-stream-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                   help="the same for the streaming quantize of the same runs, then exit")
    return p.parse_args()


COPY_BYTES = 256 << 20
KERNEL_SOURCES = ("gemm.hip", "curvefp_internal.hpp", "device_util.hpp", "planes.hpp", "codec.hpp")


QUANTIZE_SOURCES = ("quantize.hip", "curvefp_internal.hpp", "device_util.hpp", "planes.hpp", "codec.hpp")
STREAM_TRAFFIC = os.path.join(ROOT, "profiles", "quantize_stream_e4c3_1gib_traffic.md")


def kernel_source_digest(sources=None) -> str:
    """sha256 over a kernel's sources (the GEMM's by default): a traffic figure is void once
    they change."""
    import hashlib
    h = hashlib.sha256()
    for name in (sources or KERNEL_SOURCES):
        with open(os.path.join(ROOT, "paper_2608_10010_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def traffic_file(workload: str, path: str = "ws") -> str:
    return os.path.join(ROOT, "profiles", f"gemm_{path}_{workload}_traffic.md")


# the kernels one GEMM call launches, by path
CALL_KERNELS = {"ws": ("prep_kernel", "expand_kernel", "gemm_ws_kernel"),
                "prepared": ("prep_kernel", "expand_kernel", "gemm_ws_kernel"),
                "fused": ("zero_rows_kernel", "gemm_kernel")}
# the kernel whose traffic the roofline carries: the whole call, or (prepared operands) the
# GEMM kernel alone, the expansions being calls of their own
ROOFLINE_KERNELS = {"ws": CALL_KERNELS["ws"], "prepared": ("gemm_ws_kernel",), "fused": CALL_KERNELS["fused"]}


def pmc_per_dispatch(d: str, counter: str, path: str):
    """Mean per dispatch of `counter` (summed over its instances) for each kernel of one GEMM call
    and for the calibration copy; "gemm" is their sum (bytes of one whole call)."""
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    per = {}
    copy_grid = 0
    rows = []
    for f in files:
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            kind = next((k for k in CALL_KERNELS[path] if k + "<" in name or k + "(" in name), None)
            if kind is None and "copyBuffer" in name:
                kind = "copy"
            if kind is None and name.startswith("Cijk_"):
                kind = "vendor"      # the vendor fp16 GEMM of the same matrix-core work
            if kind is None:
                continue
            rows.append((kind, r))
            if kind == "copy":
                copy_grid = max(copy_grid, int(r["Grid_Size"]))
    # the calibration copies are the largest copy dispatches (the others stage small inputs)
    seen = set()
    for kind, r in rows:
        if kind == "copy" and int(r["Grid_Size"]) != copy_grid:
            continue
        key = (kind, r["Dispatch_Id"])
        inst = (key, r.get("Counter_Value"), r.get("Start_Timestamp"))
        if inst in seen:      # the same record repeated
            continue
        seen.add(inst)
        per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    out = {}
    # per GEMM call: a kernel's total over its dispatches / the GEMM kernel's dispatch count (the
    # prepared path launches prep_kernel and expand_kernel once per operand, twice per call)
    main_kernel = CALL_KERNELS[path][-1]
    ncalls = len([1 for (k, _) in per if k == main_kernel])
    if ncalls == 0:
        raise SystemExit(f"no {main_kernel} dispatches with {counter} in {d}")
    for kind in CALL_KERNELS[path] + ("copy",):
        vals = [v for (k, _), v in per.items() if k == kind]
        if not vals:
            # zero_rows_kernel runs only when K is split (fused path)
            if kind == "zero_rows_kernel":
                out[kind] = (0.0, 0)
                continue
            raise SystemExit(f"no {kind} dispatches with {counter} in {d}")
        out[kind] = (sum(vals) / (len(vals) if kind == "copy" else ncalls), len(vals))
    out["gemm"] = (sum(out[k][0] for k in CALL_KERNELS[path]), ncalls)
    out["roofline"] = (sum(out[k][0] for k in ROOFLINE_KERNELS[path]), ncalls)
    vend = [v for (k, _), v in per.items() if k == "vendor"]
    if vend:
        out["vendor"] = (sum(vend) / len(vend), len(vend))
    return out


def pmc_dir(kind: str, gemm: str, workload: str = HEADLINE) -> str:
    return f"gpurun_out/pmc_{kind}_{gemm}" + ("" if workload == HEADLINE else f"_{workload}")


def pmc_commands(gemm: str, workload: str = HEADLINE):
    """The two counter runs a traffic summary comes from (on the headline workload: the GEMM call's
    and the streaming quantize's)."""
    other = "" if workload == HEADLINE else f" --workload {workload} --no-stream --no-reference"
    run = (f"python bench.py --steps 3 --warmup 1 --no-cpu-baseline --no-backward --no-radix --no-static --no-requant "
           f"--no-blocks --no-configs "
           f"--copy-calibration --gemm {gemm}{other}")
    return [f"rocprofv3 --pmc {c} --output-format csv -d {pmc_dir(d, gemm, workload)} -o pmc -- {run}"
            for c, d in (("FETCH_SIZE", "fetch"), ("WRITE_SIZE", "write"))]


# the bf16 -> E4C3 rows kernel with 2 chunks per thread (demangled with or without the default
# radix arguments of Fmt)
STREAM_KERNEL = re.compile(r"quantize_rows_kernel<curvefp::Fmt<4, 3(, 1, 1)?>, true, 2,")


def stream_per_dispatch(d: str, counter: str):
    """Mean per dispatch of `counter` for the streaming quantize and the calibration copy."""
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    per, copy_grid, stream_grid, rows = {}, 0, 0, []
    for f in files:
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            kind = "stream" if STREAM_KERNEL.search(name) else ("copy" if "copyBuffer" in name else None)
            if kind is None:
                continue
            rows.append((kind, r))
            if kind == "copy":
                copy_grid = max(copy_grid, int(r["Grid_Size"]))
            else:
                stream_grid = max(stream_grid, int(r["Grid_Size"]))
    seen = set()
    for kind, r in rows:
        # the streaming case is the largest launch of its kernel (the step's own quantizes of
        # bf16 -> E4C3 operands use the same instantiation with smaller grids)
        if int(r["Grid_Size"]) != (copy_grid if kind == "copy" else stream_grid):
            continue
        inst = ((kind, r["Dispatch_Id"]), r.get("Counter_Value"), r.get("Start_Timestamp"))
        if inst in seen:
            continue
        seen.add(inst)
        key = (kind, r["Dispatch_Id"])
        per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    out = {}
    for kind in ("stream", "copy"):
        vals = [v for (k, _), v in per.items() if k == kind]
        if not vals:
            raise SystemExit(f"no {kind} dispatches with {counter} in {d}")
        out[kind] = (sum(vals) / len(vals), len(vals))
    return out


def summarize_stream_pmc(args):
    fetch = stream_per_dispatch(args.summarize_stream_pmc[0], "FETCH_SIZE")
    write = stream_per_dispatch(args.summarize_stream_pmc[1], "WRITE_SIZE")
    f_fetch = fetch["copy"][0] * 1024.0 / COPY_BYTES
    f_write = write["copy"][0] * 1024.0 / COPY_BYTES
    fb = fetch["stream"][0] * 1024.0 / f_fetch
    wb = write["stream"][0] * 1024.0 / f_write
    elems = 32768 * 16384
    lines = [
        "# HBM traffic of the 1 GiB streaming quantize (32768 x 16384 bf16 -> E4C3)",
        "",
        "Commands (from the repository root on one MI355X, `export TMPDIR=/tmp` first; each pass is its own run):",
        "",
        "```",
        *pmc_commands(args.gemm),
        f"python bench.py --summarize-stream-pmc {pmc_dir('fetch', args.gemm)} {pmc_dir('write', args.gemm)}",
        "```",
        "",
        "Kernel: `quantize_rows_kernel<Fmt<4, 3>, true, 2, ...>` (bf16 -> E4C3, 2 chunks per thread), the "
        "`quantize_stream` case of bench.py.",
        "",
        "| dispatch | count | FETCH_SIZE KiB/dispatch | WRITE_SIZE KiB/dispatch |",
        "|---|---|---|---|",
        f"| streaming quantize | {fetch['stream'][1]} + {write['stream'][1]} | {fetch['stream'][0]:.1f} | "
        f"{write['stream'][0]:.1f} |",
        f"| `__amd_rocclr_copyBuffer`, {COPY_BYTES >> 20} MiB device copy | {fetch['copy'][1]} + {write['copy'][1]} | "
        f"{fetch['copy'][0]:.1f} | {write['copy'][0]:.1f} |",
        "",
        f"Calibration (same runs): the copy reads and writes {COPY_BYTES >> 20} MiB once each; the counters report "
        f"{f_fetch:.4f}x (FETCH_SIZE) and {f_write:.4f}x (WRITE_SIZE) those bytes.",
        f"Streaming quantize, calibrated: {fb / 1e6:.1f} MB read (algorithmic: the 1 GiB source, "
        f"{elems * 2 / 1e6:.1f} MB) and {wb / 1e6:.1f} MB written (algorithmic: codes + scales, "
        f"{elems * (1 + 1 / 32) / 1e6:.1f} MB).",
        "",
        f"fetch_bytes={fb:.0f}",
        f"write_bytes={wb:.0f}",
        f"kernel_source_sha256={kernel_source_digest(QUANTIZE_SOURCES)}",
    ]
    print("\n".join(lines))


def pmc_by_grid(d: str, counter: str, kinds):
    """Mean per dispatch of `counter` (summed over its instances) for each (kernel, grid size) of the
    given kernels, for the vendor GEMM and for the largest copy (the calibration copy)."""
    import csv
    import glob
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    per, seen, copy_grid, rows = {}, set(), 0, []
    for f in files:
        for r in csv.DictReader(open(f)):
            if r["Counter_Name"] != counter:
                continue
            name = r["Kernel_Name"]
            kind = next((k for k in kinds if k + "<" in name or k + "(" in name), None)
            if kind is None and "copyBuffer" in name:
                kind = "copy"
                copy_grid = max(copy_grid, int(r["Grid_Size"]))
            if kind is None and name.startswith("Cijk_"):
                kind = "vendor"
            if kind is not None:
                rows.append((kind, r))
    for kind, r in rows:
        if kind == "copy" and int(r["Grid_Size"]) != copy_grid:
            continue
        inst = ((kind, r["Dispatch_Id"]), r.get("Counter_Value"), r.get("Start_Timestamp"))
        if inst in seen:
            continue
        seen.add(inst)
        key = (kind, int(r["Grid_Size"]), r["Dispatch_Id"])
        per[key] = per.get(key, 0.0) + float(r["Counter_Value"])
    out = {}
    for (kind, grid, _), v in per.items():
        s, n = out.get((kind, grid), (0.0, 0))
        out[(kind, grid)] = (s + v, n + 1)
    return {k: (s / n, n) for k, (s, n) in out.items()}


def summarize_pmc_prepared(args):
    """The prepared step's kernels: one curvefp_quantize_prepare per operand (quantize, expansion and,
    for the activations, reconstruction in one launch) and the GEMM kernel on the prepared operands."""
    from paper_2608_10010_amd import curvefp as cf
    from paper_2608_10010_amd import workloads as W
    w = W.get(args.workload)
    kinds = ("quantize_prepare_kernel", "gemm_ws_kernel")
    fetch = pmc_by_grid(args.summarize_pmc[0], "FETCH_SIZE", kinds)
    write = pmc_by_grid(args.summarize_pmc[1], "WRITE_SIZE", kinds)
    cf_ = [v for (k, _), v in fetch.items() if k == "copy"][0]
    cw_ = [v for (k, _), v in write.items() if k == "copy"][0]
    f_fetch, f_write = cf_[0] * 1024.0 / COPY_BYTES, cw_[0] * 1024.0 / COPY_BYTES
    rt = lambda rows: (rows + 255) // 256
    # the quantize_prepare grids (a workgroup per 4 rows, or per row for rows longer than 4096 bf16
    # elements): one operand alone, or both in one launch (the step), told apart by their tiles
    qp_grids = {}
    for (k, grid) in fetch:
        if k == "quantize_prepare_kernel":
            tiles = grid // (64 * 256)
            for nm, t in (("act", rt(w.M)), ("weight", rt(w.N)), ("pair", rt(w.M) + rt(w.N))):
                if tiles in (t, 4 * t):
                    qp_grids[nm] = grid
    bpe = quantize_bytes_per_elem(w.fmt, w.dtype)
    alg = {"act": w.M * w.K * (bpe + 4.0) + cf.curvefp_prepared_bytes(w.M, w.K),
           "weight": w.N * w.K * bpe + cf.curvefp_prepared_bytes(w.N, w.K)}
    alg["pair"] = alg["act"] + alg["weight"]
    lines = [
        f"# Memory traffic of the prepared step's kernels, {args.workload} workload",
        "",
        "Commands (from the repository root on one MI355X; each pass is its own run):",
        "",
        "```",
        *pmc_commands(args.gemm, args.workload),
        f"python bench.py --summarize-pmc {pmc_dir('fetch', args.gemm, args.workload)} "
        f"{pmc_dir('write', args.gemm, args.workload)} --gemm prepared"
        + ("" if args.workload == HEADLINE else f" --workload {args.workload}"),
        "```",
        "",
        "Per dispatch, each counter summed over its instances; MB = the counter scaled by what it reads for "
        f"the {COPY_BYTES >> 20} MiB device copy of the same run ({f_fetch:.4f}x FETCH_SIZE, {f_write:.4f}x "
        "WRITE_SIZE of the bytes the copy moves).  FETCH_SIZE / WRITE_SIZE count the L2s' requests to the "
        "fabric, served by the 256 MB MALL or by HBM.",
        "",
        "| kernel | grid (work-items) | dispatches | FETCH_SIZE KiB | WRITE_SIZE KiB | MB read | MB written | "
        "algorithmic MB |",
        "|---|---|---|---|---|---|---|---|",
    ]
    step = 0.0
    for nm in ("pair", "weight", "act"):
        g = qp_grids.get(nm)
        if g is None:
            continue
        fb, wb = fetch[("quantize_prepare_kernel", g)][0] * 1024 / f_fetch, write[("quantize_prepare_kernel", g)][0] * 1024 / f_write
        if nm == "pair" or "pair" not in qp_grids:
            step += fb + wb                   # the step's launch(es)
        what = {"pair": "quantize_prepare_pair (both operands, the activations with their reconstruction: the step)",
                "act": "quantize_prepare (act, with its fp32 reconstruction)",
                "weight": "quantize_prepare (weight)"}[nm]
        lines.append(f"| `{what}` | {g} | {fetch[('quantize_prepare_kernel', g)][1]} | "
                     f"{fetch[('quantize_prepare_kernel', g)][0]:.1f} | {write[('quantize_prepare_kernel', g)][0]:.1f} | "
                     f"{fb / 1e6:.1f} | {wb / 1e6:.1f} | {alg[nm] / 1e6:.1f} |")
    gk = [k for k in fetch if k[0] == "gemm_ws_kernel"]
    gk = max(gk, key=lambda k: fetch[k][1])          # the headline GEMM's grid: the most dispatches
    gf, gw = fetch[gk][0] * 1024 / f_fetch, write[gk][0] * 1024 / f_write
    step += gf + gw
    planes = cf.curvefp_prepared_bytes(w.M, w.K) + cf.curvefp_prepared_bytes(w.N, w.K)
    lines.append(f"| `gemm_ws_kernel` (curvefp_gemm_prepared) | {gk[1]} | {fetch[gk][1]} | {fetch[gk][0]:.1f} | "
                 f"{write[gk][0]:.1f} | {gf / 1e6:.1f} | {gw / 1e6:.1f} | {(planes + 4.0 * w.M * w.N) / 1e6:.1f} |")
    lines += [
        "",
        "Algorithmic bytes: quantize_prepare reads the source and writes codes, scales, the prepared planes "
        "and row maxima (4 bytes per element of the rows padded to 256) and, for the activations, the fp32 "
        "reconstruction; the GEMM's column is its prepared operands read once and C written once.  The GEMM "
        "kernel reads its planes repeatedly (each 256-row panel once per output tile that needs it; the L2s "
        "serve most re-reads): its traffic is what the roofline carries.",
        "",
    ]
    vend = fetch.get(next((k for k in fetch if k[0] == "vendor"), None))
    vendw = write.get(next((k for k in write if k[0] == "vendor"), None))
    if vend and vendw:
        vf, vw = vend[0] * 1024.0 / f_fetch, vendw[0] * 1024.0 / f_write
        valg = 2.0 * (w.M * 3 * w.K + 3 * w.K * w.N + w.M * w.N)
        lines += [
            f"For comparison, the vendor fp16 GEMM of the same matrix-core work in the same runs (torch.matmul "
            f"{w.M} x {w.N} x {3 * w.K}, `Cijk_...`, {vend[1]} dispatches): {vf / 1e6:.2f} MB read + "
            f"{vw / 1e6:.2f} MB written per call, {(vf + vw) / valg:.2f}x its own algorithmic bytes (fp16 A, B and "
            f"C, {valg / 1e6:.1f} MB).",
            "",
        ]
    lines += [
        f"traffic_bytes_per_launch={gf + gw:.0f}",
        f"fetch_bytes_per_launch={gf:.0f}",
        f"write_bytes_per_launch={gw:.0f}",
        f"call_traffic_bytes={step:.0f}",
        f"kernel_source_sha256={kernel_source_digest()}",
    ]
    print("\n".join(lines))


def summarize_pmc(args):
    if args.gemm == "prepared":
        summarize_pmc_prepared(args)
        return
    fetch = pmc_per_dispatch(args.summarize_pmc[0], "FETCH_SIZE", args.gemm)
    write = pmc_per_dispatch(args.summarize_pmc[1], "WRITE_SIZE", args.gemm)
    # KiB the counter reads per byte a plain copy moves (read and written once each)
    f_fetch = fetch["copy"][0] * 1024.0 / COPY_BYTES
    f_write = write["copy"][0] * 1024.0 / COPY_BYTES
    gemm_fetch = fetch["gemm"][0] * 1024.0 / f_fetch
    gemm_write = write["gemm"][0] * 1024.0 / f_write
    kernels = CALL_KERNELS[args.gemm]
    flag = f" --gemm {args.gemm}" + ("" if args.workload == HEADLINE else f" --workload {args.workload}")
    roof_fetch = fetch["roofline"][0] * 1024.0 / f_fetch
    roof_write = write["roofline"][0] * 1024.0 / f_write
    lines = [
        f"# Memory traffic of one CurveFP GEMM call ({args.gemm} path), {args.workload} workload",
        "",
        "Commands (from the repository root on one MI355X; each pass is its own run):",
        "",
        "```",
        *pmc_commands(args.gemm, args.workload),
        f"python bench.py --summarize-pmc {pmc_dir('fetch', args.gemm, args.workload)} "
        f"{pmc_dir('write', args.gemm, args.workload)}{flag}",
        "```",
        "",
        "| kernel | dispatches | FETCH_SIZE KiB per call | WRITE_SIZE KiB per call |",
        "|---|---|---|---|",
    ]
    for k in kernels:
        if fetch[k][1] == 0:
            continue                           # not launched by this call
        lines.append(f"| `{k}` | {fetch[k][1]} | {fetch[k][0]:.1f} | {write[k][0]:.1f} |")
    lines += [
        f"| one GEMM call (sum) | {fetch['gemm'][1]} | {fetch['gemm'][0]:.1f} | {write['gemm'][0]:.1f} |",
        f"| `__amd_rocclr_copyBuffer` ({COPY_BYTES >> 20} MiB copy) | {fetch['copy'][1]} | "
        f"{fetch['copy'][0]:.1f} | {write['copy'][0]:.1f} |",
        "",
        f"Calibration: the copy reads and writes {COPY_BYTES >> 20} MiB once each; the counters "
        f"report {f_fetch:.4f}x (FETCH_SIZE) and {f_write:.4f}x (WRITE_SIZE) those bytes, and the "
        f"GEMM's counts are divided by the same factors.",
        f"Traffic past the L2s per GEMM call (FETCH_SIZE / WRITE_SIZE count the L2s' requests to the "
        f"fabric, served by the 256 MB MALL or by HBM): {gemm_fetch / 1e6:.2f} MB read + "
        f"{gemm_write / 1e6:.2f} MB written.",
        "",
    ]
    if args.gemm == "prepared":
        lines += [
            f"The prepared path's call is curvefp_prepare of A, curvefp_prepare of B (one `prep_kernel` and one "
            f"`expand_kernel` each: two dispatches of each per call, summed above) and curvefp_gemm_prepared "
            f"(`gemm_ws_kernel`). The GEMM kernel alone, whose traffic the roofline carries: "
            f"{roof_fetch / 1e6:.2f} MB read + {roof_write / 1e6:.2f} MB written.",
            "",
        ]
    if "vendor" in fetch and "vendor" in write:
        from paper_2608_10010_amd import workloads as W
        w = W.get(args.workload)
        vf, vw = fetch["vendor"][0] * 1024.0 / f_fetch, write["vendor"][0] * 1024.0 / f_write
        alg = 2.0 * (w.M * 3 * w.K + 3 * w.K * w.N + w.M * w.N)
        lines += [
            f"For comparison, the vendor fp16 GEMM of the same matrix-core work in the same runs (torch.matmul "
            f"{w.M} x {w.N} x {3 * w.K}, `Cijk_...`, {fetch['vendor'][1]} dispatches): {vf / 1e6:.2f} MB read + "
            f"{vw / 1e6:.2f} MB written per call, {(vf + vw) / alg:.2f}x its own algorithmic bytes (fp16 A, B and "
            f"C, {alg / 1e6:.1f} MB).",
            "",
        ]
    lines += [
        f"traffic_bytes_per_launch={roof_fetch + roof_write:.0f}",
        f"fetch_bytes_per_launch={roof_fetch:.0f}",
        f"write_bytes_per_launch={roof_write:.0f}",
        f"call_traffic_bytes={gemm_fetch + gemm_write:.0f}",
        f"kernel_source_sha256={kernel_source_digest()}",
    ]
    print("\n".join(lines))


def measured_traffic(workload: str, path: str):
    """HBM bytes per GEMM call from the committed counter summary, or None when there is none
    or the kernel sources changed since it was taken."""
    try:
        text = open(traffic_file(workload, path)).read()
    except OSError:
        return None
    kv = dict(l.split("=", 1) for l in text.splitlines() if "=" in l and " " not in l.split("=", 1)[0])
    if kv.get("kernel_source_sha256") != kernel_source_digest():
        return None
    return float(kv["traffic_bytes_per_launch"])


def measured_stream_traffic():
    """HBM bytes of one streaming-quantize launch from the committed counter summary, or None
    when there is none or the quantize sources changed since it was taken."""
    try:
        text = open(STREAM_TRAFFIC).read()
    except OSError:
        return None
    kv = dict(l.split("=", 1) for l in text.splitlines() if "=" in l and " " not in l.split("=", 1)[0])
    if kv.get("kernel_source_sha256") != kernel_source_digest(QUANTIZE_SOURCES):
        return None
    return float(kv["fetch_bytes"]) + float(kv["write_bytes"])


def quantize_bytes_per_elem(fmt: str, dtype: str) -> float:
    src = 2.0 if dtype == "bf16" else 4.0
    code = 7.0 / 8.0 if fmt == "E3C3" else 1.0
    return src + code + 1.0 / 32.0


def dequantize_bytes_per_elem(fmt: str) -> float:
    return (7.0 / 8.0 if fmt == "E3C3" else 1.0) + 1.0 / 32.0 + 4.0


def host_cpu():
    """The host the oracle runs on: CPU model, cores this process may use, nproc."""
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = os.cpu_count()
    import subprocess
    try:
        nproc = int(subprocess.run(["nproc"], capture_output=True, text=True, check=True).stdout.strip())
    except (OSError, ValueError, subprocess.CalledProcessError):
        nproc = None
    return {"cpu_model": model, "sched_getaffinity": affinity, "nproc": nproc,
            "omp_num_threads": os.environ.get("OMP_NUM_THREADS")}


def oracle_step(f, A, B):
    """The oracle's whole step on operands A [ra, K] and B [rb, K] (K along rows): quantize both,
    the exact phase-binned GEMM, dequantize the activation codes.  Wall time of each phase."""
    import oracle
    t = {}
    t0 = time.perf_counter()
    ca, sa = oracle.quantize(A, f)
    t["quantize_a"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    cb, sb = oracle.quantize(B, f)
    t["quantize_b"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.gemm_exact(ca, sa, cb, sb, f)
    t["gemm"] = time.perf_counter() - t0
    t0 = time.perf_counter()
    oracle.dequantize(ca, sa, f)
    t["dequantize"] = time.perf_counter() - t0
    t["total"] = sum(t.values())
    return t


def gemm_operands_rows(w):
    """A and B of a workload with K along their rows (the layout the oracle quantizes)."""
    import numpy as np
    A, B = w.operand("a"), w.operand("b")
    A = A if w.a.axis == 1 else np.ascontiguousarray(A.T)
    B = B if w.b.axis == 1 else np.ascontiguousarray(B.T)
    return A, B


def sampled_rows(X, step: int):
    import numpy as np
    return np.ascontiguousarray(X[::step]) if step > 1 else X


def extrapolate(t, w, sa: int, sb: int):
    """Full-step time from a run on every sa-th row of A and every sb-th row of B: the quantize
    and dequantize phases scale with their operand's rows, the GEMM with the product count."""
    ra, rb = -(-w.M // sa), -(-w.N // sb)
    return (t["quantize_a"] * w.M / ra + t["quantize_b"] * w.N / rb + t["gemm"] * (w.M * w.N) / (ra * rb)
            + t["dequantize"] * w.M / ra)


def cpu_baseline(w, seconds: float):
    """The oracle, as it stands, on a bounded sample of the same step: every s-th row of A and of
    B (s a power of two, lowered until one run takes about `seconds`) -- quantize both, exact
    phase-binned GEMM, dequantize; value = the sampled GEMM's 2 ra rb K flop over the wall time."""
    import oracle

    f = oracle.get_format(w.fmt)
    A, B = gemm_operands_rows(w)
    nthreads = oracle.load_library().oracle_max_threads()
    step = 1
    while step < 4096 and (w.M // step) * (w.N // step) * w.K > 2.0e8:
        step *= 2
    while True:
        t = oracle_step(f, sampled_rows(A, step), sampled_rows(B, step))
        if t["total"] >= 0.4 * seconds or step == 1:
            break
        step //= 2
    ra, rb = -(-w.M // step), -(-w.N // step)
    flops = 2.0 * ra * rb * w.K
    out = {
        "value": flops / t["total"] / 1e12,
        "unit": "TFLOP/s",
        "cores": nthreads,
        "kind": "oracle",
        "sample": f"every {step}th row of A and of B of {w.name} ({ra} x {rb} of the {w.M} x {w.N} outputs, "
                  f"K={w.K}): oracle quantize of both samples, exact phase-binned GEMM, dequantize; "
                  f"{t['total']:.1f} s wall on {nthreads} threads; value = 2*{ra}*{rb}*{w.K} flop / wall",
        "seconds": t["total"],
        "phases_seconds": {k: v for k, v in t.items() if k != "total"},
        "full_step_seconds_extrapolated": extrapolate(t, w, step, step),
    }
    out.update(host_cpu())
    return out


def cpu_baseline_table():
    """The oracle's step timed on every configuration: full size for the tiny and inference cases;
    every 32nd row of A and of B for the rest (1/1024 of the products, 1/32 of each operand's
    quantize), with the full-size time extrapolated phase by phase."""
    import oracle
    from paper_2608_10010_amd import workloads as W

    nthreads = oracle.load_library().oracle_max_threads()
    rows = []
    for name in CONFIGS:
        w = W.get(name)
        f = oracle.get_format(w.fmt)
        A, B = gemm_operands_rows(w)
        step = 1 if name in ("tiny", "inference") else 32
        t = oracle_step(f, sampled_rows(A, step), sampled_rows(B, step))
        ra, rb = -(-w.M // step), -(-w.N // step)
        products = float(ra) * rb * w.K
        rows.append({"workload": w.name, "format": w.fmt, "M": w.M, "N": w.N, "K": w.K,
                     "row_step": step, "rows_a": ra, "rows_b": rb, "seconds": t["total"],
                     "phases_seconds": {k: v for k, v in t.items() if k != "total"},
                     "gemm_products_per_s": products / t["gemm"],
                     "seconds_full": t["total"] if step == 1 else None,
                     "seconds_full_extrapolated": extrapolate(t, w, step, step)})
        print(json.dumps(rows[-1]), flush=True)
    out = {"kind": "oracle", "threads": nthreads, "configs": rows}
    out.update(host_cpu())
    return out


_HOLD_CYCLES = None


def gpu_hold(stream, us: float = 300.0):
    """Enqueue a short spin kernel (torch's) on `stream`, so that the host has enqueued the timed
    call and its events before the GPU reaches them: the interval between the events is then the
    call's GPU time, without the host's time to marshal and launch it (which a caller from C or
    from a captured graph does not pay)."""
    import torch
    global _HOLD_CYCLES
    if _HOLD_CYCLES is None:
        n = 200000
        with torch.cuda.stream(stream):
            torch.cuda._sleep(1000)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            torch.cuda._sleep(n)
            e1.record(stream)
        torch.cuda.synchronize()
        us_per_cycle = max(e0.elapsed_time(e1) * 1e3 / n, 1e-5)
        _HOLD_CYCLES = int(min(max(us / us_per_cycle, 1e4), 1e8))
    with torch.cuda.stream(stream):
        torch.cuda._sleep(_HOLD_CYCLES)


def timed_median(fn, stream, reps: int = 20, warm: int = 3, before=None):
    """Median of `reps` individually timed calls: HIP events on the library's stream around each
    call, the GPU held back by gpu_hold until both events and the call are enqueued; `before`
    (e.g. a cache flush) runs ahead of the hold each time."""
    import numpy as np
    import torch
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    ts = []
    for _ in range(reps):
        if before is not None:
            before()
        gpu_hold(stream)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1) * 1e-3)
    return float(np.median(ts))


def copy_peak(dev, stream, nbytes: int = 1 << 30, reps: int = 20):
    """A plain 1 GiB device-to-device copy (read once, written once): the achievable HBM rate on
    this box, median of individually timed copies."""
    import torch
    x = torch.empty(nbytes, dtype=torch.uint8, device=dev)
    y = torch.empty_like(x)
    x.fill_(1)
    t = timed_median(lambda: y.copy_(x), stream, reps)
    del x, y
    return {"bytes_moved": 2 * nbytes, "us": t * 1e6, "gbps": 2 * nbytes / t / 1e9,
            "what": f"torch copy_ of a {nbytes >> 20} MiB device buffer (read + write), median of {reps}"}


def vendor_reference(w, dev, stream, gemm_tflops: float, reps: int = 20):
    """Context for the GEMM's roofline fraction: the vendor library's plain fp16 GEMM (torch.matmul,
    hipBLASLt) on M x N with 3K, the same matrix-core work as the CurveFP GEMM's three fp16
    products per useful product; median of `reps` individually timed calls."""
    import torch
    M, N, K = w.M, w.N, 3 * w.K
    a = torch.randn(M, K, device=dev, dtype=torch.float32).to(torch.float16).contiguous()
    b = torch.randn(K, N, device=dev, dtype=torch.float32).to(torch.float16).contiguous()
    c = torch.empty((M, N), device=dev, dtype=torch.float16)
    t = timed_median(lambda: torch.matmul(a, b, out=c), stream, reps)
    tf = 2.0 * M * N * K / t / 1e12
    del a, b, c
    torch.cuda.empty_cache()
    return {"what": f"torch.matmul fp16 {M}x{N}x{K} (hipBLASLt), median of {reps}", "us": t * 1e6,
            "tflops": tf, "frac": tf / F16_DENSE_PEAK_TFLOPS,
            "curvefp_gemm_matrix_core_tflops": 3.0 * gemm_tflops,
            "curvefp_vs_vendor": 3.0 * gemm_tflops / tf}


def config_sweep(cf, W, dev, stream, gemm_path: str, reps: int = 20):
    """Every configuration timed on its own: quantize of each operand (GB/s, algorithmic bytes)
    and the GEMM call (TFLOP/s, fraction of dense fp16 peak: curvefp_gemm_ws, expansion included,
    or curvefp_gemm); with prepared operands also each operand's curvefp_prepare, its
    curvefp_quantize_prepare (quantize and prepare in one launch, where the shape allows), the
    curvefp_gemm_prepared call alone, and the whole step (both operands quantized and prepared,
    then the prepared GEMM); medians of `reps` calls each."""
    import torch
    out = {}
    # written before each cold call: 512 MiB evicts the 256 MB MALL and the L2s
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    for name in CONFIGS:
        w = W.get(name)
        tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        ta = torch.from_numpy(w.operand("a")).to(tdt).to(dev)
        tb = torch.from_numpy(w.operand("b")).to(tdt).to(dev)
        ca, sa = cf.curvefp_quantize(ta, w.fmt, block_axis=w.a.axis)
        cb, sb = cf.curvefp_quantize(tb, w.fmt, block_axis=w.b.axis)
        C = torch.empty((w.M, w.N), dtype=torch.float32, device=dev)
        ws = cf.gemm_workspace(w.M, w.N, w.K, dev) if gemm_path in ("ws", "prepared") else None
        q_a = lambda: cf.curvefp_quantize(ta, w.fmt, block_axis=w.a.axis, codes=ca, scales=sa)
        q_b = lambda: cf.curvefp_quantize(tb, w.fmt, block_axis=w.b.axis, codes=cb, scales=sb)
        t_a, t_b = timed_median(q_a, stream, reps), timed_median(q_b, stream, reps)
        t_a_cold = timed_median(q_a, stream, reps, warm=0, before=flush.zero_)
        t_b_cold = timed_median(q_b, stream, reps, warm=0, before=flush.zero_)
        if gemm_path in ("ws", "prepared"):
            t_g = timed_median(lambda: cf.curvefp_gemm_ws(ca, sa, cb, sb, w.M, w.N, w.K, w.fmt, c=C, workspace=ws),
                               stream, reps)
        else:
            t_g = timed_median(lambda: cf.curvefp_gemm(ca, sa, cb, sb, w.M, w.N, w.K, w.fmt, c=C), stream, reps)
        bpe = quantize_bytes_per_elem(w.fmt, w.dtype)
        tf = w.flops() / t_g / 1e12
        out[name] = {
            "workload": w.name, "format": w.fmt, "M": w.M, "N": w.N, "K": w.K,
            "quantize_a": {"us": t_a * 1e6, "gbps": w.M * w.K * bpe / t_a / 1e9,
                           "us_cold": t_a_cold * 1e6, "gbps_cold": w.M * w.K * bpe / t_a_cold / 1e9,
                           "axis": w.a.axis},
            "quantize_b": {"us": t_b * 1e6, "gbps": w.N * w.K * bpe / t_b / 1e9,
                           "us_cold": t_b_cold * 1e6, "gbps_cold": w.N * w.K * bpe / t_b_cold / 1e9,
                           "axis": w.b.axis},
            "gemm": {"us": t_g * 1e6, "gflop": w.flops() / 1e9, "tflops": tf,
                     "frac": tf / F16_DENSE_PEAK_TFLOPS},
        }
        if gemm_path == "prepared":
            pa = cf.curvefp_prepare(ca, sa, w.M, w.K, w.fmt)
            pb = cf.curvefp_prepare(cb, sb, w.N, w.K, w.fmt)
            nws = cf.curvefp_gemm_prepared_workspace_bytes(w.M, w.N, w.K)
            gws = torch.empty(nws, dtype=torch.uint8, device=dev) if nws else None
            t_pa = timed_median(lambda: cf.curvefp_prepare(ca, sa, w.M, w.K, w.fmt, prepared=pa), stream, reps)
            t_pb = timed_median(lambda: cf.curvefp_prepare(cb, sb, w.N, w.K, w.fmt, prepared=pb), stream, reps)
            t_gp = timed_median(lambda: cf.curvefp_gemm_prepared(pa, w.fmt, pb, w.fmt, w.M, w.N, w.K, c=C,
                                                                 workspace=gws), stream, reps)
            tfp = w.flops() / t_gp / 1e12
            out[name].update({
                "prepare_a": {"us": t_pa * 1e6}, "prepare_b": {"us": t_pb * 1e6},
                "gemm_prepared": {"us": t_gp * 1e6, "tflops": tfp, "frac": tfp / F16_DENSE_PEAK_TFLOPS},
            })
            # one launch per operand where it applies (blocks along K)
            fused = w.a.axis == 1 and w.b.axis == 1
            if fused:
                t_qpa = timed_median(lambda: cf.curvefp_quantize_prepare(ta, w.fmt, codes=ca, scales=sa, prepared=pa),
                                     stream, reps)
                t_qpb = timed_median(lambda: cf.curvefp_quantize_prepare(tb, w.fmt, codes=cb, scales=sb, prepared=pb),
                                     stream, reps)
                out[name].update({"quantize_prepare_a": {"us": t_qpa * 1e6}, "quantize_prepare_b": {"us": t_qpb * 1e6}})

            # the whole step on this configuration, as the headline runs it: quantize and prepare
            # both operands (one pair launch; quantize-transposed operands: quantize and prepare
            # each), then the GEMM on the prepared operands; one stream, median of `reps` steps
            def step():
                if fused:
                    cf.curvefp_quantize_prepare_pair(ta, tb, w.fmt, out_a=(ca, sa, pa), out_b=(cb, sb, pb))
                else:
                    cf.curvefp_quantize(ta, w.fmt, block_axis=w.a.axis, codes=ca, scales=sa)
                    cf.curvefp_quantize(tb, w.fmt, block_axis=w.b.axis, codes=cb, scales=sb)
                    cf.curvefp_prepare(ca, sa, w.M, w.K, w.fmt, prepared=pa)
                    cf.curvefp_prepare(cb, sb, w.N, w.K, w.fmt, prepared=pb)
                cf.curvefp_gemm_prepared(pa, w.fmt, pb, w.fmt, w.M, w.N, w.K, c=C, workspace=gws)
            t_step = timed_median(step, stream, reps)
            tfs = w.flops() / t_step / 1e12
            out[name]["step"] = {"us": t_step * 1e6, "tflops": tfs, "what": "quantize_prepare_pair + gemm_prepared"
                                 if fused else "quantize x2 (transpose) + prepare x2 + gemm_prepared"}
            del pa, pb, gws
        del ta, tb, ca, sa, cb, sb, C, ws
        torch.cuda.empty_cache()
    out["timing"] = (f"median of {reps} individually timed calls each (HIP events), inputs resident in HBM; "
                     f"*_cold: each call after a 512 MiB write that evicts the MALL and the L2s")
    out["roofline"] = (f"quantize against {HBM_PEAK_GBS / 1000:.0f} TB/s (algorithmic bytes: source + codes + "
                       f"scales); GEMM against {F16_DENSE_PEAK_TFLOPS / 1000:.1f} PFLOP/s dense fp16 (2MNK flop)")
    return out


def backward_mixed(cf, W, dev, stream, reps: int = 20):
    """dX = Q_G(dY) Q_W(W) and dW = Q_G(dY)^T Q_A(X) of the 7B up-projection: dY quantized once
    in E5C2 along its rows, W and X as their forward E4C3 codes.  Each GEMM call (prep,
    expansions, MFMA GEMM) is timed with HIP events on the library's stream: median of `reps`
    individually timed calls after warm-up.  Operands are quantized before timing."""
    import numpy as np
    import torch

    out = {}
    src = {}
    for name in ("dgrad_mixed", "wgrad_mixed"):
        w = W.get(name)
        ops = []
        for which, op in (("a", w.a), ("b", w.b)):
            key = (op.seed, op.axis)
            if key not in src:
                x = torch.from_numpy(w.operand(which)).to(torch.bfloat16).to(dev)
                src[key] = cf.curvefp_quantize(x, w.fmt_of(which), block_axis=op.axis)
                del x
            ops.append(src[key])
        (ca, sa), (cb, sb) = ops
        C = torch.empty((w.M, w.N), dtype=torch.float32, device=dev)
        ws = cf.gemm_mixed_workspace(w.M, w.N, w.K, dev)

        def call():
            cf.curvefp_gemm_mixed(ca, sa, w.fmt_of("a"), w.a.trans, cb, sb, w.fmt_of("b"), w.b.trans,
                                  w.M, w.N, w.K, c=C, workspace=ws)

        t = timed_median(call, stream, reps)
        tf = w.flops() / t / 1e12
        # the same product on prepared operands (each expanded in its own layout), the GEMM alone
        fa, fb = w.fmt_of("a"), w.fmt_of("b")
        pa = cf.curvefp_prepare(ca, sa, w.M, w.K, fa, trans=w.a.trans)
        pb = cf.curvefp_prepare(cb, sb, w.N, w.K, fb, trans=w.b.trans)
        nws = cf.curvefp_gemm_prepared_workspace_bytes(w.M, w.N, w.K)
        gws = torch.empty(nws, dtype=torch.uint8, device=dev) if nws else None
        t_pa = timed_median(lambda: cf.curvefp_prepare(ca, sa, w.M, w.K, fa, trans=w.a.trans, prepared=pa), stream, reps)
        t_pb = timed_median(lambda: cf.curvefp_prepare(cb, sb, w.N, w.K, fb, trans=w.b.trans, prepared=pb), stream, reps)
        t_gp = timed_median(lambda: cf.curvefp_gemm_prepared(pa, fa, pb, fb, w.M, w.N, w.K, c=C, workspace=gws),
                            stream, reps)
        tfp = w.flops() / t_gp / 1e12
        out[name.split("_")[0]] = {
            "workload": w.name, "M": w.M, "N": w.N, "K": w.K,
            "formats": f"{fa} x {fb}", "trans": [w.a.trans, w.b.trans],
            "us": t * 1e6, "achieved": tf, "peak": F16_DENSE_PEAK_TFLOPS, "unit": "TFLOP/s",
            "frac": tf / F16_DENSE_PEAK_TFLOPS, "mfma_pipe_frac": 3.0 * tf / F16_DENSE_PEAK_TFLOPS,
            "timing": f"median of {reps} individually timed curvefp_gemm_mixed calls",
            "prepared": {"prepare_a_us": t_pa * 1e6, "prepare_b_us": t_pb * 1e6, "gemm_us": t_gp * 1e6,
                         "tflops": tfp, "frac": tfp / F16_DENSE_PEAK_TFLOPS,
                         "what": "curvefp_prepare of each operand in its layout, then curvefp_gemm_prepared "
                                 "(the GEMM kernel alone)"},
        }
        del C, ws, pa, pb, gws
    src.clear()
    torch.cuda.empty_cache()
    return out


def requant(cf, w, ca, sa, cb, sb, dev, stream, reps: int = 20):
    """The inference GEMM with its output requantized to E3C3 (the next layer's activation
    format): curvefp_gemm_requant (fused epilogue) against curvefp_gemm_ws followed by
    curvefp_quantize of the fp32 C; median of `reps` individually timed calls each."""
    import numpy as np
    import torch

    ofmt = "E3C3"
    ws = cf.gemm_workspace(w.M, w.N, w.K, dev)
    C = torch.empty((w.M, w.N), dtype=torch.float32, device=dev)
    out = {}
    exact = True
    # output blocks of 32, and of 64 (the activation block size of Sec. 4.2's G64 setting)
    for G in (32, 64):
        oc = torch.empty((w.M, w.N // 32, 28), dtype=torch.uint8, device=dev)
        os_ = torch.empty((w.M, w.N // G), dtype=torch.int8, device=dev)
        oc2, os2 = torch.empty_like(oc), torch.empty_like(os_)

        def fused():
            cf.curvefp_gemm_requant(ca, sa, cb, sb, w.M, w.N, w.K, w.fmt, ofmt, out_codes=oc, out_scales=os_,
                                    workspace=ws, out_block=G)

        def two_step():
            cf.curvefp_gemm_ws(ca, sa, cb, sb, w.M, w.N, w.K, w.fmt, c=C, workspace=ws)
            cf.curvefp_quantize(C, ofmt, block=G, codes=oc2, scales=os2)

        for name, fn in (("fused", fused), ("gemm_then_quantize", two_step)):
            t = timed_median(fn, stream, reps)
            key = name if G == 32 else f"{name}_G{G}"
            out[key] = {"us": t * 1e6, "tflops": w.flops() / t / 1e12}
        torch.cuda.synchronize()
        exact = exact and bool(torch.equal(oc, oc2) and torch.equal(os_, os2))
    out["bit_exact"] = exact
    out["workload"] = f"{w.name}, output requantized to {ofmt} in blocks of 32 (and of 64: *_G64) along its rows"
    out["timing"] = f"median of {reps} individually timed calls each"
    del ws, C
    return out


def static_scales(cf, w, tb, dev, stream, reps: int = 20):
    """The inference weight (4096 x 4096 bf16) quantized as a static operand: curvefp_quantize_mse
    with 4 candidate scales, against curvefp_quantize (ceil-absmax) on the same tensor; median of
    `reps` individually timed calls each, bytes as for quantize (source + codes + scales)."""
    import numpy as np
    import torch

    out = {}
    nbytes = w.N * w.K * quantize_bytes_per_elem(w.fmt, w.dtype)
    cm, sm = cf.curvefp_quantize_mse(tb, w.fmt, block_axis=w.b.axis, candidates=4)
    cc, sc = cf.curvefp_quantize(tb, w.fmt, block_axis=w.b.axis)
    calls = {"mse_search": lambda: cf.curvefp_quantize_mse(tb, w.fmt, block_axis=w.b.axis, candidates=4,
                                                          codes=cm, scales=sm),
             "ceil_absmax": lambda: cf.curvefp_quantize(tb, w.fmt, block_axis=w.b.axis, codes=cc, scales=sc)}
    for name, fn in calls.items():
        t = timed_median(fn, stream, reps)
        out[name] = {"us": t * 1e6, "gbps": nbytes / t / 1e9}
    out["scales_moved_frac"] = float((sm != sc).float().mean().item())
    # the same search over blocks of 64 (Sec. 4.2's PTQ setting), one thread per block of 64
    cm64, sm64 = cf.curvefp_quantize_mse(tb, w.fmt, block_axis=w.b.axis, candidates=4, block=64)
    fn64 = lambda: cf.curvefp_quantize_mse(tb, w.fmt, block_axis=w.b.axis, candidates=4, block=64,
                                           codes=cm64, scales=sm64)
    t = timed_median(fn64, stream, reps)
    nb64 = w.N * w.K * (quantize_bytes_per_elem(w.fmt, w.dtype) - 1.0 / 32.0 + 1.0 / 64.0)
    out["mse_search_G64"] = {"us": t * 1e6, "gbps": nb64 / t / 1e9}
    out["workload"] = f"{w.name} weight {w.N}x{w.K} {w.dtype} -> {w.fmt}, 4 candidate scales"
    out["timing"] = f"median of {reps} individually timed calls each"
    return out


def block_sizes(cf, w, ta, tb, dev, stream, reps: int = 20):
    """The inference workload with one scale per G elements (Eq. effective-rate; Sec. 4.2's G64
    and G512, and rowwise G = K): per G the median of `reps` individually timed calls of
    quantize(act), quantize(weight) and curvefp_gemm_ws.  Quantize bytes are the algorithmic
    source + codes + one scale byte per G elements; G = 4096 runs the scale pass first and reads
    the source twice."""
    import numpy as np
    import torch

    out = {}
    C = torch.empty((w.M, w.N), dtype=torch.float32, device=dev)
    ws = cf.gemm_workspace(w.M, w.N, w.K, dev)

    def timed(fn):
        return timed_median(fn, stream, reps)

    for G in (32, 64, 512, w.K):
        ca, sa = cf.curvefp_quantize(ta, w.fmt, block_axis=w.a.axis, block=G)
        cb, sb = cf.curvefp_quantize(tb, w.fmt, block_axis=w.b.axis, block=G)
        per_elem = quantize_bytes_per_elem(w.fmt, w.dtype) - 1.0 / 32.0 + 1.0 / G
        t_a = timed(lambda: cf.curvefp_quantize(ta, w.fmt, block_axis=w.a.axis, block=G, codes=ca, scales=sa))
        t_b = timed(lambda: cf.curvefp_quantize(tb, w.fmt, block_axis=w.b.axis, block=G, codes=cb, scales=sb))
        t_g = timed(lambda: cf.curvefp_gemm_ws(ca, sa, cb, sb, w.M, w.N, w.K, w.fmt, block=G, c=C, workspace=ws))
        out[f"G{G}"] = {"quantize_act_gbps": w.M * w.K * per_elem / t_a / 1e9,
                        "quantize_weight_gbps": w.N * w.K * per_elem / t_b / 1e9,
                        "gemm_us": t_g * 1e6, "gemm_tflops": w.flops() / t_g / 1e12,
                        "bits_per_value_int8_scales": (7.0 if w.fmt == "E3C3" else 8.0) + 8.0 / G}
    # S-bit scale exponents at G64 (Sec. 4.2: S = 5 for activations, 4 for weights), same codes
    # layout; bytes: source + codes + S/G bits of offset per element + one reference byte per row
    for which, t, rows, S in (("act", ta, w.M, 5), ("weight", tb, w.N, 4)):
        G = 64
        cc, rr, oo = cf.curvefp_quantize_compact(t, w.fmt, G, S)
        per_elem = quantize_bytes_per_elem(w.fmt, w.dtype) - 1.0 / 32.0 + S / 8.0 / G
        tq = timed(lambda: cf.curvefp_quantize_compact(t, w.fmt, G, S, codes=cc, row_ref=rr, offsets=oo))
        out[f"compact_G{G}_S{S}_{which}"] = {
            "quantize_gbps": (rows * w.K * per_elem + rows) / tq / 1e9, "us": tq * 1e6,
            "bits_per_value": (7.0 if w.fmt == "E3C3" else 8.0) + S / G}
    # tensorwise: one scale per tensor (a max pass over the source, then the quantize pass)
    for which, t, rows in (("act", ta, w.M), ("weight", tb, w.N)):
        cc, ss = cf.curvefp_quantize_tensorwise(t, w.fmt)
        wsw = torch.empty((1,), dtype=torch.int32, device=dev)
        per_elem = quantize_bytes_per_elem(w.fmt, w.dtype) - 1.0 / 32.0
        tq = timed(lambda: cf.curvefp_quantize_tensorwise(t, w.fmt, codes=cc, scales=ss, workspace=wsw))
        out[f"tensorwise_{which}"] = {"quantize_gbps": (rows * w.K * per_elem + rows) / tq / 1e9, "us": tq * 1e6}
    out["workload"] = (f"{w.name}: act {w.M}x{w.K}, weight {w.N}x{w.K} {w.dtype} -> {w.fmt}, G = 32, 64, 512, K; "
                       f"S-bit scales at G64 (S = 5 act, 4 weight); tensorwise")
    out["timing"] = f"median of {reps} individually timed calls each"
    return out


def radix_variants(cf, w, ta, tb, dev, stream, reps: int = 20):
    """The inference workload's operands quantized and multiplied in E4C3 with the radices of
    Tab. radix-frontier (r = 2: 8 phases; 2^(8/9): 9; 2^(3/4): 32): per format the median of
    `reps` individually timed calls of quantize(act), quantize(weight) and curvefp_gemm_ws."""
    import numpy as np
    import torch

    out = {}
    C = torch.empty((w.M, w.N), dtype=torch.float32, device=dev)
    ws = cf.gemm_workspace(w.M, w.N, w.K, dev)
    for fmt in ("E4C3", "E4C3_r8/9", "E4C3_r3/4"):
        ca, sa = cf.curvefp_quantize(ta, fmt, block_axis=w.a.axis)
        cb, sb = cf.curvefp_quantize(tb, fmt, block_axis=w.b.axis)
        calls = {
            "quantize_act": lambda: cf.curvefp_quantize(ta, fmt, block_axis=w.a.axis, codes=ca, scales=sa),
            "quantize_weight": lambda: cf.curvefp_quantize(tb, fmt, block_axis=w.b.axis, codes=cb, scales=sb),
            "gemm": lambda: cf.curvefp_gemm_ws(ca, sa, cb, sb, w.M, w.N, w.K, fmt, c=C, workspace=ws),
        }
        t = {}
        for name, fn in calls.items():
            t[name] = timed_median(fn, stream, reps)
        p, q = cf.curvefp_format_radix(fmt)
        H = cf.curvefp_format_info(fmt)[3]
        qa = w.M * w.K * quantize_bytes_per_elem(fmt, w.dtype)
        qb = w.N * w.K * quantize_bytes_per_elem(fmt, w.dtype)
        tf = w.flops() / t["gemm"] / 1e12
        out[fmt] = {
            "radix": f"2^({p}/{q})", "phases": H,
            "us": {k: v * 1e6 for k, v in t.items()},
            "quantize_gbps": {"act": qa / t["quantize_act"] / 1e9, "weight": qb / t["quantize_weight"] / 1e9},
            "gemm_tflops": tf, "gemm_frac": tf / F16_DENSE_PEAK_TFLOPS,
        }
    out["workload"] = f"{w.name} operands ({w.M}x{w.K} act, {w.N}x{w.K} weight, bf16), block 32"
    out["timing"] = f"median of {reps} individually timed calls each"
    del C, ws
    return out


def main():
    args = parse()
    if args.summarize_pmc:
        summarize_pmc(args)
        return
    if args.summarize_stream_pmc:
        summarize_stream_pmc(args)
        return
    if args.cpu_baseline_table:
        print(json.dumps(cpu_baseline_table()), flush=True)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only: the library has no multi-GPU path "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE={world}).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2608_10010_amd import curvefp as cf
    from paper_2608_10010_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = W.get(args.workload)
    A = w.operand("a")
    B = w.operand("b")
    ta = torch.from_numpy(A).to(torch.bfloat16 if w.dtype == "bf16" else torch.float32).to(dev)
    tb = torch.from_numpy(B).to(torch.bfloat16 if w.dtype == "bf16" else torch.float32).to(dev)
    outer_a = w.M
    ka = w.K
    stream = torch.cuda.current_stream()
    ca, sa = cf.curvefp_quantize(ta, w.fmt, block_axis=w.a.axis)
    cb, sb = cf.curvefp_quantize(tb, w.fmt, block_axis=w.b.axis)
    C = torch.empty((w.M, w.N), dtype=torch.float32, device=dev)
    D = torch.empty((outer_a, ka), dtype=torch.float32, device=dev)
    # workspaces and prepared buffers are allocated once, like C: the timed calls only use them
    prepared = args.gemm == "prepared"
    # one launch per operand (curvefp_quantize_prepare): both operands with blocks along K
    fused_step = prepared and not args.separate_step and not args.serial_step and w.a.axis == 1 and w.b.axis == 1
    ws = cf.gemm_workspace(w.M, w.N, w.K, dev) if args.gemm == "ws" else None
    pa = pb = gws = None
    if prepared:
        pa = torch.empty(cf.curvefp_prepared_bytes(w.M, w.K), dtype=torch.uint8, device=dev)
        pb = torch.empty(cf.curvefp_prepared_bytes(w.N, w.K), dtype=torch.uint8, device=dev)
        nws = cf.curvefp_gemm_prepared_workspace_bytes(w.M, w.N, w.K)
        gws = torch.empty(nws, dtype=torch.uint8, device=dev) if nws else None

    def prepare_a(s=None):
        cf.curvefp_prepare(ca, sa, w.M, w.K, w.fmt, prepared=pa, stream=s)

    def prepare_b(s=None):
        cf.curvefp_prepare(cb, sb, w.N, w.K, w.fmt, prepared=pb, stream=s)

    def gemm():
        if prepared:
            cf.curvefp_gemm_prepared(pa, w.fmt, pb, w.fmt, w.M, w.N, w.K, c=C, workspace=gws)
        elif args.gemm == "ws":
            cf.curvefp_gemm_ws(ca, sa, cb, sb, w.M, w.N, w.K, w.fmt, c=C, workspace=ws)
        else:
            cf.curvefp_gemm(ca, sa, cb, sb, w.M, w.N, w.K, w.fmt, c=C)

    # Default (prepared path): one curvefp_quantize_prepare_pair launch quantizes and expands both
    # operands (the activations also reconstructed), then the GEMM (MFMA-bound, every SIMD's
    # registers taken by its waves) runs alone; one stream.  Separate calls: on two streams (both
    # at the default priority) the activations are quantized, their codes reconstructed and
    # (prepared path) expanded on the main stream while the weights are quantized and expanded on
    # the side stream; the GEMM then runs on the main stream once both operands are there.
    side = torch.cuda.Stream(device=dev)

    def rec(ev, key, s):
        if ev is not None and key in ev:
            ev[key].record(s)

    def step_serial(ev=None):
        rec(ev, "qa0", stream)
        cf.curvefp_quantize(ta, w.fmt, block_axis=w.a.axis, codes=ca, scales=sa, stream=stream)
        rec(ev, "qa1", stream)
        rec(ev, "qb0", stream)
        cf.curvefp_quantize(tb, w.fmt, block_axis=w.b.axis, codes=cb, scales=sb, stream=stream)
        rec(ev, "qb1", stream)
        if prepared:
            rec(ev, "pa0", stream)
            prepare_a(stream)
            rec(ev, "pa1", stream)
            rec(ev, "pb0", stream)
            prepare_b(stream)
            rec(ev, "pb1", stream)
        rec(ev, "d0", stream)
        cf.curvefp_dequantize(ca, sa, w.fmt, outer_a, ka, dst=D, stream=stream)
        rec(ev, "d1", stream)
        rec(ev, "g0", stream)
        gemm()
        rec(ev, "g1", stream)

    def step_fused(ev=None):
        rec(ev, "qp0", stream)
        cf.curvefp_quantize_prepare_pair(ta, tb, w.fmt, out_a=(ca, sa, pa, D), out_b=(cb, sb, pb), stream=stream)
        rec(ev, "qp1", stream)
        rec(ev, "g0", stream)
        gemm()
        rec(ev, "g1", stream)

    def step(ev=None):
        if fused_step:
            step_fused(ev)
            return
        if args.serial_step:
            step_serial(ev)
            return
        side.wait_stream(stream)
        rec(ev, "qa0", stream)
        cf.curvefp_quantize(ta, w.fmt, block_axis=w.a.axis, codes=ca, scales=sa, stream=stream)
        rec(ev, "qa1", stream)
        rec(ev, "qb0", side)
        cf.curvefp_quantize(tb, w.fmt, block_axis=w.b.axis, codes=cb, scales=sb, stream=side)
        rec(ev, "qb1", side)
        if prepared:
            rec(ev, "pb0", side)
            prepare_b(side)
            rec(ev, "pb1", side)
        rec(ev, "d0", stream)
        cf.curvefp_dequantize(ca, sa, w.fmt, outer_a, ka, dst=D, stream=stream)
        rec(ev, "d1", stream)
        if prepared:
            # the activations' expansion after their reconstruction (measured the fastest order)
            rec(ev, "pa0", stream)
            prepare_a(stream)
            rec(ev, "pa1", stream)
        stream.wait_stream(side)
        rec(ev, "g0", stream)
        gemm()
        rec(ev, "g1", stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: exactly `steps` steps, synchronized on both sides; HIP events on the main
    # stream bracket the GEMM of every step (the roofline's kernel).  Events around the other
    # calls would add their own latency to the step (each record is a barrier packet: ~0.9% of
    # the step with events around all six calls), so those are timed in the steps after it.
    keys = ("qp", "g") if fused_step else ("qa", "qb", "g", "d") + (("pa", "pb") if prepared else ())
    evs = [{"g0": torch.cuda.Event(enable_timing=True), "g1": torch.cuda.Event(enable_timing=True)}
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = wall * 1e3 / args.steps
    ndiag = min(args.steps, 10)
    diag = [{k + e: torch.cuda.Event(enable_timing=True) for k in keys for e in "01"} for _ in range(ndiag)]
    for i in range(ndiag):
        step(diag[i])
    torch.cuda.synchronize()
    if fused_step:
        names = {"quantize_prepare_pair": "qp", "gemm": "g"}
    else:
        names = {"quantize_a": "qa", "quantize_b": "qb", "gemm": "g", "dequantize": "d"}
        if prepared:
            names.update({"prepare_a": "pa", "prepare_b": "pb"})
    per = {n: float(np.mean([diag[i][k + "0"].elapsed_time(diag[i][k + "1"]) for i in range(ndiag)]))
           for n, k in names.items()}
    per["gemm"] = float(np.mean([evs[i]["g0"].elapsed_time(evs[i]["g1"]) for i in range(args.steps)]))

    flops = w.flops()
    gemm_tflops = flops / (per["gemm"] * 1e-3) / 1e12
    qa_bytes = outer_a * ka * quantize_bytes_per_elem(w.fmt, w.dtype)
    qb_bytes = w.N * w.K * quantize_bytes_per_elem(w.fmt, w.dtype)
    dq_bytes = outer_a * ka * dequantize_bytes_per_elem(w.fmt)
    # a prepared operand's algorithmic bytes: its codes and scales read, its planes (4 bytes per
    # element of the rows padded to 256) and row maxima written
    pa_bytes = w.M * w.K * (quantize_bytes_per_elem(w.fmt, w.dtype) - (2.0 if w.dtype == "bf16" else 4.0)) + \
        cf.curvefp_prepared_bytes(w.M, w.K)
    pb_bytes = w.N * w.K * (quantize_bytes_per_elem(w.fmt, w.dtype) - (2.0 if w.dtype == "bf16" else 4.0)) + \
        cf.curvefp_prepared_bytes(w.N, w.K)
    # quantize-prepare: source read, codes + scales, planes + row maxima (and, for the activations,
    # the fp32 reconstruction) written
    qpa_bytes = qa_bytes + cf.curvefp_prepared_bytes(w.M, w.K) + 4.0 * w.M * w.K
    qpb_bytes = qb_bytes + cf.curvefp_prepared_bytes(w.N, w.K)

    result = {
        "metric": METRIC,
        "value": flops / (ms_per_step * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "format": w.fmt,
            "source_dtype": w.dtype,
            "M": w.M, "N": w.N, "K": w.K, "block": 32,
            "step": ("quantize_prepare_pair(act with its reconstruction, weight) -- quantize, dequantize and "
                     "prepare of both operands in one launch -- then gemm_prepared, one stream"
                     if fused_step else
                     "[quantize(act) -> dequantize(act codes) -> prepare(act)] || [quantize(weight) -> "
                     "prepare(weight)] on two streams, then gemm_prepared" if prepared else
                     "[quantize(act) -> dequantize(act codes)] || quantize(weight) on two streams, then gemm"),
            "gemm_arith": "fp16 hi/lo operand split, 3 MFMA f32_32x32x16_f16 per k-slice, fp32 accumulate",
            "gemm_path": {"prepared": "curvefp_prepare of each operand (its codes expanded once into fp16 "
                                      "hi/lo planes), then curvefp_gemm_prepared",
                          "ws": "curvefp_gemm_ws: codes expanded once into a workspace, then the GEMM",
                          "fused": "curvefp_gemm: expansion inside the GEMM kernel"}[args.gemm],
            "parallelism": "single GPU",
        },
        "roofline": {
            "bound": "mfma",
            "kernel": {"prepared": "gemm_ws_kernel (the curvefp_gemm_prepared call)",
                       "ws": "gemm call (prep_kernel, expand_kernel, gemm_ws_kernel)",
                       "fused": "gemm call (" + ", ".join(CALL_KERNELS["fused"]) + ")"}[args.gemm],
            "achieved": gemm_tflops,
            "peak": F16_DENSE_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": gemm_tflops / F16_DENSE_PEAK_TFLOPS,
            "traffic": measured_traffic(w.name, args.gemm),
            "mfma_pipe_frac": 3.0 * gemm_tflops / F16_DENSE_PEAK_TFLOPS,
        },
        "kernels_us": {n: per[n] * 1e3 for n in names},
        "kernels_us_note": ("each call between HIP events on the stream; gemm: mean over the timed steps; "
                            "quantize_prepare_pair: over 10 steps right after them with events around both calls"
                            if fused_step else
                            "each call between HIP events on the stream it runs on (quantize_a, dequantize, "
                            "prepare_a, gemm: main; quantize_b, prepare_b: side, alongside the main "
                            "stream's calls before the GEMM); gemm: mean over the timed steps; the "
                            "others: over 10 steps right after them with events around every call"
                            if prepared else
                            "each call between HIP events on the stream it runs on (quantize_a, dequantize, "
                            "gemm: main; quantize_b: side, alongside quantize_a and dequantize); gemm: "
                            "mean over the timed steps; the others: over 10 steps right after them"),
        "per_call_timing": "outside the step, every figure timed per call is the median of calls each "
                           "between HIP events on the library's stream, enqueued behind a ~0.3 ms spin "
                           "kernel so that the GPU reaches the first event only after the host has "
                           "enqueued the call: GPU time, without the Python binding's host time",
        "gemm_tflops": gemm_tflops,
    }
    if fused_step:
        result["quantize_prepare_gbps"] = {
            "pair": (qpa_bytes + qpb_bytes) / (per["quantize_prepare_pair"] * 1e-3) / 1e9,
            "bytes": "both sources read; codes, scales, planes and row maxima written, and the activations' "
                     "fp32 reconstruction"}
    else:
        result["quantize_gbps"] = {"act": qa_bytes / (per["quantize_a"] * 1e-3) / 1e9,
                                   "weight": qb_bytes / (per["quantize_b"] * 1e-3) / 1e9}
        result["dequantize_gbps"] = dq_bytes / (per["dequantize"] * 1e-3) / 1e9
    if prepared and not fused_step:
        result["prepare_gbps"] = {"act": pa_bytes / (per["prepare_a"] * 1e-3) / 1e9,
                                  "weight": pb_bytes / (per["prepare_b"] * 1e-3) / 1e9,
                                  "bytes": "codes + scales read, planes + row maxima written"}

    # The step above runs back to back on the same inputs, so sources that fit the 256 MB MALL
    # may be served from it.  Each call again on its own after a 512 MiB write that evicts the
    # MALL and the L2s (median of 20): the cold-cache figures, inputs from HBM.
    flush = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    cold_calls = {
        "quantize_a": lambda: cf.curvefp_quantize(ta, w.fmt, block_axis=w.a.axis, codes=ca, scales=sa),
        "quantize_b": lambda: cf.curvefp_quantize(tb, w.fmt, block_axis=w.b.axis, codes=cb, scales=sb),
        "gemm": gemm,
        "dequantize": lambda: cf.curvefp_dequantize(ca, sa, w.fmt, outer_a, ka, dst=D),
    }
    if prepared:
        cold_calls.update({"prepare_a": prepare_a, "prepare_b": prepare_b})
    # the whole step, its sources and operands read from HBM
    cold_calls["step"] = step
    if fused_step:
        cold_calls.update({
            "quantize_prepare_pair": lambda: cf.curvefp_quantize_prepare_pair(
                ta, tb, w.fmt, out_a=(ca, sa, pa, D), out_b=(cb, sb, pb)),
            "quantize_prepare_a": lambda: cf.curvefp_quantize_prepare(ta, w.fmt, codes=ca, scales=sa, prepared=pa,
                                                                      dst=D),
            "quantize_prepare_b": lambda: cf.curvefp_quantize_prepare(tb, w.fmt, codes=cb, scales=sb, prepared=pb)})
    cold = {}
    for n, fn in cold_calls.items():
        cold[n] = timed_median(fn, stream, 20, warm=0, before=flush.zero_) * 1e6
    del flush
    result["kernels_us_cold"] = cold
    result["cold_cache"] = {
        "step_tflops": flops / (cold["step"] * 1e-6) / 1e12,
        "gemm_tflops": flops / (cold["gemm"] * 1e-6) / 1e12,
        "quantize_gbps": {"act": qa_bytes / (cold["quantize_a"] * 1e-6) / 1e9,
                          "weight": qb_bytes / (cold["quantize_b"] * 1e-6) / 1e9},
        "dequantize_gbps": dq_bytes / (cold["dequantize"] * 1e-6) / 1e9,
        "protocol": "each call alone after a 512 MiB device write (MALL and L2 evicted), median of 20",
    }
    if prepared:
        result["cold_cache"]["prepare_gbps"] = {"act": pa_bytes / (cold["prepare_a"] * 1e-6) / 1e9,
                                                "weight": pb_bytes / (cold["prepare_b"] * 1e-6) / 1e9}
    if fused_step:
        result["cold_cache"]["quantize_prepare_gbps"] = {
            "pair": (qpa_bytes + qpb_bytes) / (cold["quantize_prepare_pair"] * 1e-6) / 1e9,
            "act": qpa_bytes / (cold["quantize_prepare_a"] * 1e-6) / 1e9,
            "weight": qpb_bytes / (cold["quantize_prepare_b"] * 1e-6) / 1e9}

    if args.copy_calibration:
        xc = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev)
        yc = torch.empty_like(xc)
        for _ in range(3):
            yc.copy_(xc)
        torch.cuda.synchronize()
        del xc, yc

    if not args.no_stream:
        # streaming quantize: 32768 x 16384 bf16 (1 GiB source) -> E4C3, larger than the MALL
        g = torch.Generator(device=dev)
        g.manual_seed(77)
        xs = torch.randn((32768, 16384), generator=g, device=dev, dtype=torch.float32).to(torch.bfloat16)
        cs, ss = cf.curvefp_quantize(xs, "E4C3")
        torch.cuda.synchronize()
        # median of >= 20 individually timed calls after warm-up (each call alone on the GPU,
        # enqueued behind a spin kernel); the mean of 10 back-to-back calls is reported too
        # (it runs hotter: on long back-to-back runs the per-call time rises by up to ~40%)
        t_q = timed_median(lambda: cf.curvefp_quantize(xs, "E4C3", codes=cs, scales=ss), stream, 20)
        reps = 10
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            cf.curvefp_quantize(xs, "E4C3", codes=cs, scales=ss)
        e1.record(stream)
        torch.cuda.synchronize()
        t_b2b = e0.elapsed_time(e1) / reps * 1e-3
        nbytes = xs.numel() * quantize_bytes_per_elem("E4C3", "bf16")
        gbs = nbytes / t_q / 1e9
        del xs, cs, ss
        torch.cuda.empty_cache()
        # (not in the counter runs: their calibration copies must be the largest copy dispatches)
        cp = None if args.copy_calibration else copy_peak(dev, stream)
        result["quantize_stream"] = {
            "shape": [32768, 16384], "format": "E4C3", "source_dtype": "bf16",
            "us": t_q * 1e6, "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": gbs / HBM_PEAK_GBS, "bytes_per_elem": quantize_bytes_per_elem("E4C3", "bf16"),
            "traffic": measured_stream_traffic(),
            "timing": "median of 20 individually timed calls",
            "us_back_to_back": t_b2b * 1e6, "achieved_back_to_back": nbytes / t_b2b / 1e9,
            "copy": cp, "frac_of_copy": gbs / cp["gbps"] if cp else None,
            "frac_of_copy_back_to_back": nbytes / t_b2b / 1e9 / cp["gbps"] if cp else None,
        }

    if not args.no_reference:
        result["vendor_fp16_gemm_reference"] = vendor_reference(w, dev, stream, gemm_tflops)

    # the headline's buffers are no longer needed
    del ta, tb, ca, sa, cb, sb, C, D, ws
    torch.cuda.empty_cache()

    if not args.no_configs:
        result["configs"] = config_sweep(cf, W, dev, stream, args.gemm)

    # the adjacent variants run on the inference workload (E3C3, 2048 x 4096 x 4096)
    if not (args.no_requant and args.no_static and args.no_radix and args.no_blocks):
        wi = W.get("inference")
        ti = torch.from_numpy(wi.operand("a")).to(torch.bfloat16).to(dev)
        tw = torch.from_numpy(wi.operand("b")).to(torch.bfloat16).to(dev)
        if not args.no_requant:
            cia, sia = cf.curvefp_quantize(ti, wi.fmt, block_axis=wi.a.axis)
            ciw, siw = cf.curvefp_quantize(tw, wi.fmt, block_axis=wi.b.axis)
            result["requant"] = requant(cf, wi, cia, sia, ciw, siw, dev, stream)
            del cia, sia, ciw, siw
        if not args.no_static:
            result["static_scales"] = static_scales(cf, wi, tw, dev, stream)
        if not args.no_radix:
            result["radix_variants"] = radix_variants(cf, wi, ti, tw, dev, stream)
        if not args.no_blocks:
            result["block_sizes"] = block_sizes(cf, wi, ti, tw, dev, stream)
        del ti, tw
        torch.cuda.empty_cache()

    if not args.no_backward:
        result["backward_mixed"] = backward_mixed(cf, W, dev, stream)

    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(w, args.cpu_seconds)

    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
