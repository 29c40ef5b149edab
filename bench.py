#!/usr/bin/env python3
"""Benchmark of the fused W4A4 + sparse-residual linear layer on one MI355X.

Workload (the layer the headline metric is quoted on): a LLaMA3-8B-shaped
attention projection, K = N = 4096, fp32 weights N(0, 0.02) with 0.5 % x20
outliers, base INT4 with group-128 fp16 scales, 10 % of the 128x128 blocks
(102) carrying an INT4 residual selected by Frobenius norm, fp16 activations
N(0,1) with 4 channels x30 -- swept over M = 1, 16, 256, 4096 tokens.

One step = the whole hot path at every M of the sweep: per-token activation
quantisation and the fused GEMM, called as one layer (mq_linear: a single
kernel at decode sizes, mq_quantize_act then mq_fused_gemm otherwise).  Inputs
are resident in HBM before timing; every call of a step reads its own copy of
the packed weights, rotating through more than 512 MB of copies so that the
256 MB last-level cache cannot serve weights from an earlier call.

value = effective TOPS of a step = sum_M 2*M*N*K / step time (the residual
MACs are extra work, not counted in "effective").  Per-M rows report
microseconds per layer call (us_call, mq_linear) and, separately, of the
fused GEMM alone on quantised input (us_gemm) and of the quantiser alone
(us_quant); effective TOPS, the fraction of the INT8 MFMA peak (algorithmic
ops including residual) and of HBM bandwidth (algorithmic bytes) of the GEMM;
and hipBLASLt W16A16 (torch.nn.functional.linear, fp16) timed the same way on
the same shapes with rotating weights, compared with us_call.

All timing replays HIP graphs (captured with torch.cuda.graph, which the
binding follows because it launches on torch's current stream), so host-side
launch overhead is outside the timed region; HIP events are recorded on the
replay stream.  roofline: the dominant kernel is the fused GEMM at M = 4096;
its average launch duration is the graph-replayed per-call time, its work the
algorithmic ops 2 M (N K + nnzb 128^2), its peak that of the fp6 matrix
instruction it runs on (the INT8 fraction is reported beside it); traffic is
the HBM bytes per launch from the FETCH_SIZE / WRITE_SIZE counter passes
(--traffic, --summarize-traffic) when they were taken on the current kernel
source.  cpu_baseline: the CPU oracle (C, OpenMP) repeating whole steps of
the same workload for about 10 s on the host cores.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_FP6_TOPS = 10100.0        # MI355X dense FP6 MFMA, TOP/s (the instruction the GEMM runs on)
PEAK_I8_TOPS = 5000.0          # MI355X dense INT8 MFMA, TOP/s (the target's reference peak)
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E, GB/s
ROTATE_BYTES = 600 << 20       # > 512 MB of distinct weight copies
TRAFFIC_CALLS = 8              # dispatches per kernel in a --traffic counter run
COPY_BYTES = 256 << 20         # size of the reference copy in a --traffic run
CPU_MIN_S = 10.0               # cpu_baseline repeats whole steps for at least this long
CPU_MAX_STEPS = 8
GEMM_SRC = os.path.join(ROOT, "paper_2606_15652_amd", "csrc", "fused_gemm.hip")
XCDS, SIMDS = 8, 1024          # MI355X: 8 XCDs, 256 CUs x 4 SIMDs


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--ms", type=str, default="1,16,256,4096")
    ap.add_argument("--reps", type=int, default=50, help="back-to-back calls per per-M timing")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-blas", action="store_true")
    ap.add_argument("--quick", action="store_true", help="short run for profilers")
    ap.add_argument("--summarize-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="fold the counter_collection.csv files of two --traffic runs (FETCH_SIZE, "
                         "WRITE_SIZE) into profiles/fused_gemm_traffic.json; needs no GPU")
    ap.add_argument("--families", action="store_true",
                    help="time the fused GEMM and the whole layer call on every layer of the other "
                         "workload families (one JSON line per layer and M; not the headline line)")
    ap.add_argument("--only", metavar="LAYERS", help="--families: comma-separated layer names (default: all)")
    ap.add_argument("--table5", action="store_true",
                    help="--families: the Qwen3-8B concatenated-output operators (qkv, o, gate_up, down) "
                         "at decode and prefill batch sizes instead of the workload families")
    ap.add_argument("--max-m", type=int, default=None, help="--families: skip token counts above this")
    ap.add_argument("--unfused", action="store_true",
                    help="--families: also time the three-kernel baseline (dense GEMM, residual GEMM, "
                         "reduce-add) and the dense-only GEMM on the same operands")
    ap.add_argument("--kernel-run", metavar="SPECS",
                    help="counter / trace run: comma-separated layer:M[:variant] specs; per spec, "
                         "--calls eager fused GEMM launches (rotating weight copies), then a "
                         "plain 256 MiB elementwise kernel as the byte-counter reference")
    ap.add_argument("--calls", type=int, default=8, help="GEMM launches per spec in --kernel-run")
    ap.add_argument("--summarize-counters", nargs="+", metavar=("OUT_MD", "CSV"),
                    help="fold the counter_collection.csv files of --kernel-run passes into a "
                         "markdown table OUT_MD (needs no GPU); SPECS from --kernel-run")
    ap.add_argument("--selection", action="store_true",
                    help="residual block selection study (Section 3 Eq. (5), Fig. 2b): output-distortion "
                         "reduction C(S) of Delta-Hessian, residual-norm, weight-magnitude and random "
                         "selection (and exact greedy selection on the smallest layer) over block budgets")
    ap.add_argument("--summarize-trace", nargs=2, metavar=("OUT_MD", "KERNEL_TRACE_CSV"),
                    help="fold the kernel_trace.csv of a rocprofv3 --kernel-trace run of --kernel-run into "
                         "per-spec launch durations (markdown, appended to OUT_MD; needs no GPU)")
    ap.add_argument("--summarize-families", nargs="+", metavar=("OUT_MD", "JSONL"),
                    help="format the JSON lines of --families runs as a markdown table (appended to OUT_MD; "
                         "needs no GPU)")
    ap.add_argument("--sweep", metavar="LAYERS",
                    help="time AUTO and every kernel family that applies over a range of M on these layers "
                         "(comma-separated names; one JSON line per layer and M)")
    ap.add_argument("--sweep-ms", type=str,
                    default="1,16,32,48,64,128,256,384,512,768,1024,1280,1536,2048,3072,4096,6144,8192")
    ap.add_argument("--summarize-sweep", nargs="+", metavar=("OUT_MD", "JSONL"),
                    help="append the markdown table of --sweep JSON lines to OUT_MD; needs no GPU")
    ap.add_argument("--traffic", action="store_true",
                    help="counter run: eager fused GEMM launches at the largest M, then a plain "
                         "256 MiB device copy as the scale reference for FETCH_SIZE / WRITE_SIZE")
    return ap.parse_args()


def src_hash(path):
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def algorithmic(M, N, K, nnzb):
    """Ops (int8 MACs x2, residual included) and bytes of one fused GEMM call."""
    ops = 2.0 * M * (N * K + nnzb * 128 * 128)
    byts = (N * K / 2 + N * K / 128 * 2           # Wq + s_w
            + nnzb * (128 * 64 + 128 * 2 + 4)     # Rq + s_r + kb
            + (N / 128 + 1) * 4                   # rowptr
            + M * K / 2 + M * 2                   # Xq + s_x
            + M * N * 2)                          # Y
    return ops, byts


def cpu_model():
    """The host CPU's model name (/proc/cpuinfo), or None."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def quant_bytes(M, K):
    return M * K * 2 + M * K / 2 + M * 2


def summarize_traffic(fetch_csv, write_csv, m):
    """HBM bytes per fused GEMM dispatch from two rocprofv3 --pmc runs of
    `bench.py --traffic`.  Each counter (KiB per dispatch) is scaled by
    known bytes / counter reading of the reference copy, the last
    TRAFFIC_CALLS dispatches of the run."""
    import csv
    import statistics

    def per_kernel(path, counter):
        rows = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        by_disp = {}
        for r in rows:       # one value per dispatch (summed over any per-XCD rows)
            d = int(r["Dispatch_Id"])
            name, v = by_disp.get(d, (r["Kernel_Name"], 0.0))
            by_disp[d] = (name, v + float(r["Counter_Value"]))
        disp = sorted(by_disp.items())
        gemm = [v for _, (name, v) in disp if "gemm_tiled_kernel" in name]
        copy = [v for _, (_, v) in disp[-TRAFFIC_CALLS:]]
        if not gemm or len(copy) < TRAFFIC_CALLS:
            raise SystemExit(f"{path}: no gemm_tiled_kernel or reference copy dispatches for {counter}")
        return statistics.median(gemm), statistics.median(copy)

    g_f, c_f = per_kernel(fetch_csv, "FETCH_SIZE")
    g_w, c_w = per_kernel(write_csv, "WRITE_SIZE")
    kib = COPY_BYTES / 1024.0
    f_scale, w_scale = kib / c_f, kib / c_w
    fetch_b = g_f * f_scale * 1024.0
    write_b = g_w * w_scale * 1024.0
    out = {"kernel": "gemm_tiled_kernel", "M": m, "src_hash": src_hash(GEMM_SRC),
           "fetch_kib_raw": g_f, "write_kib_raw": g_w,
           "copy_fetch_kib_raw": c_f, "copy_write_kib_raw": c_w, "copy_bytes": COPY_BYTES,
           "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
           "fetch_bytes": round(fetch_b), "write_bytes": round(write_b),
           "bytes_per_launch": round(fetch_b + write_b)}
    path = os.path.join(ROOT, "profiles", "fused_gemm_traffic.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out))


def parse_specs(text):
    out = []
    for item in text.split(","):
        f = item.strip().split(":")
        out.append((f[0], int(f[1]), f[2] if len(f) > 2 else "auto"))
    return out


def kernel_run(args):
    """Eager launches for rocprofv3 (--pmc or --kernel-trace): for each spec,
    the layer's weights prepared on the GPU and copied until the copies exceed
    ROTATE_BYTES, activations quantised, then args.calls fused GEMM launches,
    each on the next copy (so the weights come from HBM, not the last-level
    cache); finally TRAFFIC_CALLS elementwise kernels that read and write
    COPY_BYTES each, the reference that scales the byte counters."""
    import torch

    import paper_2606_15652_amd as mq
    import synth

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    mq.load()
    dev = torch.device("cuda:0")
    for name, m, variant in parse_specs(args.kernel_run):
        layer = synth.workload(name)
        K, N = layer.K, layer.N
        pw0 = mq.prepare_weight(torch.from_numpy(layer.weight()).to(dev), layer.nnzb)
        ncopy = max(2, -(-ROTATE_BYTES // pw0.nbytes))
        copies = [pw0] + [mq.PackedWeight(N, K, pw0.Wq.clone(), pw0.s_w.clone(), pw0.rowptr.clone(),
                                          pw0.kb.clone(), pw0.Rq.clone(), pw0.s_r.clone())
                          for _ in range(ncopy - 1)]
        Xq, sx = mq.quantize_act(torch.from_numpy(layer.act(m)).to(dev))
        Y = torch.empty((m, N), dtype=torch.float16, device=dev)
        ws = torch.empty(max(1, mq.load().mq_fused_gemm_workspace_size(m, N, K)), dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()
        for i in range(args.calls):
            mq.fused_gemm(Xq, sx, copies[(i + 1) % ncopy], out=Y, variant=variant, workspace=ws)
        torch.cuda.synchronize()
        print(json.dumps({"spec": f"{name}:{m}:{variant}", "K": K, "N": N, "M": m, "nnzb": layer.nnzb,
                          "calls": args.calls}), flush=True)
        del copies, pw0, Xq, sx, Y, ws
        torch.cuda.empty_cache()
    src = torch.ones(COPY_BYTES // 4, dtype=torch.int32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(TRAFFIC_CALLS):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"reference": "neg", "bytes_read": COPY_BYTES, "bytes_written": COPY_BYTES,
                      "calls": TRAFFIC_CALLS}), flush=True)


def summarize_trace(args):
    """Per spec of a --kernel-run: the kernel, grid and average / min / max
    duration of its GEMM launches (dispatches of gemm_* / reduce_* kernels in
    dispatch order, args.calls per spec) from a rocprofv3 kernel trace."""
    import csv
    import statistics

    out_md, path = args.summarize_trace
    specs = parse_specs(args.kernel_run)
    rows = sorted(csv.DictReader(open(path)), key=lambda r: int(r["Dispatch_Id"]))
    gemm = [r for r in rows if "gemm_" in r["Kernel_Name"] or "reduce_splits" in r["Kernel_Name"]]
    runs, last = [], None
    for r in gemm:
        d = int(r["Dispatch_Id"])
        if runs and last is not None and d == last + 1:
            runs[-1].append(r)
        else:
            runs.append([r])
        last = d
    runs = [r for r in runs if len(r) >= args.calls]
    if len(runs) != len(specs):
        raise SystemExit(f"{path}: {len(runs)} GEMM dispatch runs for {len(specs)} specs")
    lines = ["| spec | kernel | grid | launches | average µs | min µs | max µs | algorithmic ops / average |",
             "|---|---|---|---|---|---|---|---|"]
    for (name, m, variant), run in zip(specs, runs):
        import synth
        layer = synth.workload(name)
        ops, _ = algorithmic(m, layer.N, layer.K, layer.nnzb)
        per_launch = len(run) // args.calls
        durs = [sum(int(x["End_Timestamp"]) - int(x["Start_Timestamp"]) for x in run[j:j + per_launch]) / 1e3
                for j in range(0, per_launch * args.calls, per_launch)]
        avg = statistics.mean(durs)
        kname = run[0]["Kernel_Name"].split("(")[0].replace("void ", "")
        lines.append(f"| {name} M={m} ({variant}) | `{kname}` | {run[0].get('Grid_Size_X', run[0].get('Grid_Size', ''))} | {len(durs)} | "
                     f"{avg:.2f} | {min(durs):.2f} | {max(durs):.2f} | {ops / avg / 1e6:.0f} TOP/s |")
    with open(out_md, "a") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_families(args):
    """Markdown table of --families JSON lines (one row per layer and M)."""
    out_md, paths = args.summarize_families[0], args.summarize_families[1:]
    lines = ["| layer | K → N | M | ρ | nnzb | GEMM µs | layer call µs | eff. TOPS | int8 peak | HBM | "
             "unfused µs | fused speed-up | W16A16 µs | call speed-up |", "|" + "---|" * 14]
    for path in paths:
        for line in open(path):
            if not line.startswith("{"):
                continue
            d = json.loads(line)
            rho = f"{d['density_pct']} %" + (" (skewed)" if d.get("skewed") else "")
            unf = d.get("us_unfused")
            fsu = "-" if unf is None else f"{unf / d['us_gemm']:.2f}×"
            lines.append(
                f"| {d['layer']} | {d['K']} → {d['N']} | {d['M']} | {rho} | {d['nnzb']} | {d['us_gemm']:.1f} | "
                f"{d['us_call']:.1f} | {d['eff_tops']:.0f} | {100 * d['int8_peak_frac']:.1f} % | "
                f"{100 * d['hbm_frac']:.1f} % | {'-' if unf is None else f'{unf:.1f}'} | "
                f"{fsu} | {d['us_w16a16']:.1f} | "
                f"{d['speedup_vs_w16a16']:.2f}× |")
    with open(out_md, "a") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def summarize_counters(args):
    """Per spec of a --kernel-run: the median per dispatch of every counter
    over its GEMM launches (dispatches of kernels named gemm_* / reduce_*,
    grouped into consecutive runs, one run per spec), and derived figures:
    matrix-core ops from SQ_INSTS_VALU_MFMA_MOPS_F6F4 (x 512), MFMA busy
    fraction SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / XCDs x 1024 SIMDs),
    VALU instructions other than MFMA per MFMA, and HBM bytes from FETCH_SIZE,
    WRITE_SIZE and TCC_EA0_RDREQ_DRAM scaled by what the same counter reads
    for the reference kernel of known bytes."""
    import csv
    import statistics

    out_md, csvs = args.summarize_counters[0], args.summarize_counters[1:]
    specs = parse_specs(args.kernel_run)
    per = [dict() for _ in specs]       # spec index -> counter -> median per dispatch
    ref = {}
    for path in csvs:
        disp = {}
        for r in csv.DictReader(open(path)):
            d = int(r["Dispatch_Id"])
            e = disp.setdefault(d, {"name": r["Kernel_Name"], "grid": r.get("Grid_Size", ""), "c": {}})
            e["c"][r["Counter_Name"]] = e["c"].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        order = sorted(disp)
        gemm = [d for d in order if "gemm_" in disp[d]["name"] or "reduce_splits" in disp[d]["name"]]
        runs = []                           # maximal runs of consecutive GEMM dispatch ids
        for d in gemm:
            if runs and d == runs[-1][-1] + 1:
                runs[-1].append(d)
            else:
                runs.append([d])
        runs = [r for r in runs if len(r) >= args.calls]
        if len(runs) != len(specs):
            raise SystemExit(f"{path}: {len(runs)} GEMM dispatch runs for {len(specs)} specs")
        for i, run in enumerate(runs):
            per_launch = len(run) // args.calls          # 2 with a split-K reduction
            launches = [run[j:j + per_launch] for j in range(0, per_launch * args.calls, per_launch)]
            for cname in disp[run[0]]["c"]:
                per[i][cname] = statistics.median(sum(disp[d]["c"].get(cname, 0.0) for d in L)
                                                  for L in launches)
            per[i]["kernel"] = disp[run[0]]["name"].split("(")[0].replace("void ", "")
            per[i]["grid"] = disp[run[0]]["grid"]
        refd = order[-TRAFFIC_CALLS:]
        for cname in disp[refd[0]]["c"]:
            ref[cname] = statistics.median(disp[d]["c"][cname] for d in refd)
    lines = ["| spec | kernel | matrix ops / launch (counter) | algorithmic ops | MFMA busy | "
             "VALU beside MFMA | VALU per MFMA | wave cycles waiting | LDS bank-conflict cycles / LDS instr | "
             "FETCH bytes | WRITE bytes | DRAM read bytes | algorithmic bytes |", "|" + "---|" * 13]
    for (name, m, variant), c in zip(specs, per):
        import synth
        layer = synth.workload(name)
        ops, byts = algorithmic(m, layer.N, layer.K, layer.nnzb)
        f = lambda x: "-" if x is None else (f"{x:.3g}" if abs(x) < 1e4 else f"{x:.4g}")
        mops = c.get("SQ_INSTS_VALU_MFMA_MOPS_F6F4")
        busy = None
        if "SQ_VALU_MFMA_BUSY_CYCLES" in c and c.get("GRBM_GUI_ACTIVE"):
            busy = c["SQ_VALU_MFMA_BUSY_CYCLES"] / (c["GRBM_GUI_ACTIVE"] / XCDS * SIMDS)
        vpm = None
        if c.get("SQ_INSTS_MFMA"):
            vpm = (c.get("SQ_INSTS_VALU", 0.0) - c["SQ_INSTS_MFMA"]) / c["SQ_INSTS_MFMA"]
        lds = c["SQ_LDS_BANK_CONFLICT"] / c["SQ_INSTS_LDS"] if c.get("SQ_INSTS_LDS") else None
        coexec = (c["SQ_VALU_MFMA_COEXEC_CYCLES"] / c["SQ_VALU_MFMA_BUSY_CYCLES"]
                  if c.get("SQ_VALU_MFMA_BUSY_CYCLES") and "SQ_VALU_MFMA_COEXEC_CYCLES" in c else None)
        wait = c["SQ_WAIT_ANY"] / c["SQ_WAVE_CYCLES"] if c.get("SQ_WAVE_CYCLES") and "SQ_WAIT_ANY" in c else None
        pct = lambda x: "-" if x is None else f"{100 * x:.1f} %"

        def scaled(cn, ref_bytes):
            if cn in c and ref.get(cn):
                return c[cn] / ref[cn] * ref_bytes
            return None
        fetch = scaled("FETCH_SIZE", COPY_BYTES)
        write = scaled("WRITE_SIZE", COPY_BYTES)
        dram = scaled("TCC_EA0_RDREQ_DRAM_sum", COPY_BYTES) or scaled("TCC_EA0_RDREQ_DRAM", COPY_BYTES)
        lines.append(f"| {name} M={m} ({variant}) | `{c['kernel']}` grid {c['grid']} | "
                     f"{f(None if mops is None else mops * 512)} | {f(ops)} | "
                     f"{pct(busy)} | {pct(coexec)} | {f(vpm)} | {pct(wait)} | {f(lds)} | "
                     f"{f(fetch)} | {f(write)} | {f(dram)} | {f(byts)} |")
    raw = ["", "Raw medians per launch (counter: value; reference kernel in the last column):", "",
           "| counter | " + " | ".join(f"{n} M={m}" for n, m, _ in specs) + " | reference |",
           "|" + "---|" * (len(specs) + 2)]
    for cn in sorted(set().union(*[set(k for k in c if k not in ("kernel", "grid")) for c in per])):
        raw.append(f"| {cn} | " + " | ".join(f"{c.get(cn, float('nan')):.6g}" for c in per)
                   + f" | {ref.get(cn, float('nan')):.6g} |")
    with open(out_md, "a") as fh:
        fh.write("\n".join(lines + raw) + "\n")
    print("\n".join(lines + raw))


SELECTION_BUDGETS = (0.01, 0.02, 0.05, 0.10, 0.20, 0.30, 0.50)
SELECTION_LAYERS = ("c1_1024", "c2_4096", "c4_qo")
SELECTION_TOKENS = 512
GREEDY_MAX_BLOCKS = 64


def selection(args):
    """C(S) = (||X R||^2 - ||X (R - M_S . Q(R))||^2) / ||X R||^2 (Section 3,
    Eq. (5)) on the calibration activations X, for the block sets chosen by:
    Algorithm 1's Delta-Hessian score, the residual norm ||R_B||_F^2, the
    largest weight magnitude in the block, a random order and, where the layer
    has at most GREEDY_MAX_BLOCKS blocks, the exact greedy output-distortion
    selection (largest marginal gain first).  Scores, base and residual
    quantisation come from the library's weight preparation (GPU); the
    distortion sums are fp64 matrix products.  One JSON line per layer."""
    import numpy as np
    import torch
    import paper_2606_15652_amd as mq
    import synth

    dev = torch.device("cuda:0")
    names = args.only.split(",") if args.only else SELECTION_LAYERS
    for name in names:
        layer = synth.workload(name)
        N, K = layer.N, layer.K
        NB, KB = N // 128, K // 128
        W = torch.from_numpy(layer.weight()).to(dev)
        X = torch.from_numpy(layer.act(SELECTION_TOKENS)).to(dev)
        # every block's residual quantised: Q(R) of any selection is a mask of it
        pw = mq.prepare_weight(W, NB * KB)
        Wc, swc, Rc = mq.unpack_weights(pw)
        def codes(nib):
            lo = (nib & 0xF).to(torch.int16)
            hi = (nib >> 4).to(torch.int16)
            q = torch.stack((lo, hi), -1).reshape(*nib.shape[:-1], nib.shape[-1] * 2)
            return torch.where(q >= 8, q - 16, q).to(torch.float64)
        s_w = swc.to(torch.float64).repeat_interleave(128, dim=1)
        Qw = (codes(Wc).to(torch.float32) * s_w.to(torch.float32))      # exact: 3-bit code x fp16 scale
        R = (W - Qw).to(torch.float64)                                  # fp32 residual, as the library forms it
        QR = torch.zeros((N, K), dtype=torch.float64, device=dev)
        rowptr = pw.rowptr.cpu().numpy()
        kb = pw.kb.cpu().numpy()
        qr_blocks = codes(Rc) * pw.s_r.to(torch.float64)[:, :, None]
        for nb in range(NB):
            for p in range(rowptr[nb], rowptr[nb + 1]):
                QR[128 * nb:128 * nb + 128, 128 * kb[p]:128 * kb[p] + 128] = qr_blocks[p]
        Xd = X.to(torch.float64)
        XR = Xd @ R.T
        base = float((XR * XR).sum())
        # the effect of each block on X E^T: X_k (QR_B)^T for block (nb, kb)
        def dist(mask):
            E = R - QR * mask.repeat_interleave(128, 0).repeat_interleave(128, 1)
            XE = Xd @ E.T
            return float((XE * XE).sum())
        h = mq.hessian_diag(X)
        Wq_lib, s_w_lib, _ = mq.quantize_weight(W, with_score=False)
        scores = {
            "dhessian": mq.block_scores_dhessian(W, Wq_lib, s_w_lib, h),
            "resnorm": pw.score,
            "magnitude": W.abs().reshape(NB, 128, KB, 128).amax(dim=(1, 3)).to(torch.float64),
            "random": torch.from_numpy(np.random.default_rng(7).permutation(NB * KB).astype(np.float64))
                      .reshape(NB, KB).to(dev),
        }
        orders = {k: torch.argsort(v.reshape(-1), descending=True, stable=True) for k, v in scores.items()}
        if NB * KB <= GREEDY_MAX_BLOCKS:
            mask = torch.zeros(NB * KB, dtype=torch.float64, device=dev)
            order = []
            for _ in range(NB * KB):
                best, best_d = None, None
                for b in range(NB * KB):
                    if mask[b] > 0:
                        continue
                    mask[b] = 1
                    d = dist(mask.reshape(NB, KB))
                    mask[b] = 0
                    if best_d is None or d < best_d:
                        best, best_d = b, d
                mask[best] = 1
                order.append(best)
            orders["greedy_exact"] = torch.tensor(order, device=dev)
        rows = {}
        for crit, order in orders.items():
            curve = []
            for rho in SELECTION_BUDGETS:
                nsel = int(rho * NB * KB + 0.5)
                mask = torch.zeros(NB * KB, dtype=torch.float64, device=dev)
                mask[order[:nsel]] = 1
                curve.append(round(1.0 - dist(mask.reshape(NB, KB)) / base, 4))
            rows[crit] = curve
        print(json.dumps({"selection": name, "N": N, "K": K, "blocks": NB * KB, "tokens": SELECTION_TOKENS,
                          "budgets": list(SELECTION_BUDGETS), "C": rows}), flush=True)


def graph_of(torch, fn, calls):
    """Capture `calls` back-to-back invocations of fn in one HIP graph."""
    fn()                                   # warm the libraries outside capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(calls):
            fn()
    torch.cuda.synchronize()
    return g


def timed(torch, fn, reps):
    """Average microseconds per call of fn: reps calls replayed from a HIP
    graph (no host launch overhead in the timed region), HIP events on the
    replay stream."""
    g = graph_of(torch, fn, reps)
    g.replay()
    torch.cuda.synchronize()
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0.record()
    g.replay()
    t1.record()
    t1.synchronize()
    return t0.elapsed_time(t1) * 1e3 / reps


def families(args):
    """Per-layer timings of the workload families other than the headline
    layer: fused GEMM (AUTO variant), the whole layer call (mq_linear) and
    hipBLASLt W16A16 on the same shape, weights rotating through more than
    512 MB of copies (at least two).  One JSON line per layer and M."""
    import torch

    import paper_2606_15652_amd as mq
    import synth

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    mq.load()
    dev = torch.device("cuda:0")
    wcache = {}
    only = set(args.only.split(",")) if args.only else None
    for layer in (synth.table5_workloads() if args.table5 else synth.workloads()):
        if (only is None and layer.name == "c2_4096") or (only is not None and layer.name not in only):
            continue
        K, N, nnzb = layer.K, layer.N, layer.nnzb
        key = (K, N, layer.seed, layer.skewed)
        if key not in wcache:            # the density sweep shares one weight per shape
            wcache.clear()
            wcache[key] = torch.from_numpy(layer.weight()).to(dev)
        W = wcache[key]
        pw0 = mq.prepare_weight(W, nnzb)
        torch.cuda.synchronize()
        ncopy = max(2, -(-ROTATE_BYTES // pw0.nbytes))
        copies = [pw0] + [mq.PackedWeight(N, K, pw0.Wq.clone(), pw0.s_w.clone(), pw0.rowptr.clone(),
                                          pw0.kb.clone(), pw0.Rq.clone(), pw0.s_r.clone())
                          for _ in range(ncopy - 1)]
        rot = [0]

        def next_pw():
            rot[0] = (rot[0] + 1) % ncopy
            return copies[rot[0]]

        nb = max(2, -(-ROTATE_BYTES // (N * K * 2)))
        wbs = [W.to(torch.float16)] + [None] * (nb - 1)
        for i in range(1, nb):
            wbs[i] = wbs[0].clone()
        rb = [0]

        def next_wb():
            rb[0] = (rb[0] + 1) % nb
            return wbs[rb[0]]

        for m in layer.ms:
            if args.max_m is not None and m > args.max_m:
                continue
            X = torch.from_numpy(layer.act(m)).to(dev)
            Xq = torch.empty((m, mq.act_bytes(K)), dtype=torch.uint8, device=dev)
            sx = torch.empty((m,), dtype=torch.float16, device=dev)
            Y = torch.empty((m, N), dtype=torch.float16, device=dev)
            ws = torch.empty(max(1, mq.linear_workspace_bytes(m, N, K)), dtype=torch.uint8, device=dev)
            mq.quantize_act(X, out=(Xq, sx))
            reps = max(5, min(args.reps, int(2e5 // max(1.0, m * N * K / 1e9))))
            t_gemm = timed(torch, lambda: mq.fused_gemm(Xq, sx, next_pw(), out=Y), reps)
            t_call = timed(torch, lambda: mq.linear(X, next_pw(), out=Y, workspace=ws), reps)
            t_blas = None if args.no_blas else timed(torch, lambda: torch.nn.functional.linear(X, next_wb()), reps)
            ops, byts = algorithmic(m, N, K, nnzb)
            row = {"layer": layer.name, "K": K, "N": N, "M": m, "density_pct": layer.density_pct,
                   "nnzb": nnzb, "skewed": layer.skewed, "us_gemm": round(t_gemm, 3),
                   "us_call": round(t_call, 3),
                   "eff_tops": round(2.0 * m * N * K / (t_gemm * 1e-6) / 1e12, 2),
                   "int8_peak_frac": round(ops / (t_gemm * 1e-6) / 1e12 / PEAK_I8_TOPS, 4),
                   "hbm_frac": round(byts / (t_gemm * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
            if t_blas is not None:
                row["us_w16a16"] = round(t_blas, 3)
                row["speedup_vs_w16a16"] = round(t_blas / t_call, 3)
            if args.unfused:
                wsu = torch.empty(max(1, mq.load().mq_unfused_workspace_size(m, N, K)), dtype=torch.uint8,
                                  device=dev)
                dense = [mq.PackedWeight(N, K, c.Wq, c.s_w, c.rowptr.new_zeros(N // 128 + 1), c.kb[:0],
                                         c.Rq[:0], c.s_r[:0]) for c in copies]
                rd = [0]

                def next_dense():
                    rd[0] = (rd[0] + 1) % ncopy
                    return dense[rd[0]]
                t_unf = timed(torch, lambda: mq.unfused_gemm(Xq, sx, next_pw(), out=Y, workspace=wsu), reps)
                t_dense = timed(torch, lambda: mq.fused_gemm(Xq, sx, next_dense(), out=Y), reps)
                row["us_unfused"] = round(t_unf, 3)
                row["us_dense_only"] = round(t_dense, 3)
                row["fused_speedup_vs_unfused"] = round(t_unf / t_gemm, 3)
                row["residual_overhead_fused"] = round(t_gemm / t_dense - 1.0, 4)
                row["residual_overhead_unfused"] = round(t_unf / t_dense - 1.0, 4)
                del wsu, dense
            print(json.dumps(row), flush=True)
            del X, Xq, sx, Y, ws
        del copies, pw0, wbs
        torch.cuda.synchronize()
        torch.cuda.empty_cache()


def sweep(args):
    """Per layer and M: the fused GEMM under AUTO and under each kernel family
    that applies (decode up to M = 32, both tiled kernels, the medium tiles),
    weights rotating through more than 512 MB of copies, graph replays; with
    the family and K splits AUTO takes (mq_fused_gemm_plan)."""
    import torch

    import paper_2606_15652_amd as mq
    import synth

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    mq.load()
    dev = torch.device("cuda:0")
    for name in args.sweep.split(","):
        layer = synth.workload(name)
        K, N, nnzb = layer.K, layer.N, layer.nnzb
        pw0 = mq.prepare_weight(torch.from_numpy(layer.weight()).to(dev), nnzb)
        torch.cuda.synchronize()
        ncopy = max(2, -(-ROTATE_BYTES // pw0.nbytes))
        copies = [pw0] + [mq.PackedWeight(N, K, pw0.Wq.clone(), pw0.s_w.clone(), pw0.rowptr.clone(),
                                          pw0.kb.clone(), pw0.Rq.clone(), pw0.s_r.clone())
                          for _ in range(ncopy - 1)]
        rot = [0]

        def next_pw():
            rot[0] = (rot[0] + 1) % ncopy
            return copies[rot[0]]

        for m in (int(x) for x in args.sweep_ms.split(",")):
            X = torch.from_numpy(layer.act(m)).to(dev)
            Xq, sx = mq.quantize_act(X)
            Y = torch.empty((m, N), dtype=torch.float16, device=dev)
            ws = torch.empty(max(1, mq.load().mq_fused_gemm_workspace_size(m, N, K)), dtype=torch.uint8, device=dev)
            reps = max(5, min(args.reps, int(2e5 // max(1.0, m * N * K / 1e9))))
            variants = (["skinny"] if m <= 32 else []) + ["tiled"] + (["tiled_large"] if N % 256 == 0 else []) + \
                       ["medium", "auto"]
            # one untimed call of each first (buffers, code objects), then the
            # timings in the order above, AUTO last
            for v in variants:
                mq.fused_gemm(Xq, sx, next_pw(), out=Y, variant=v, workspace=ws)
            torch.cuda.synchronize()
            us = {v: round(timed(torch, lambda: mq.fused_gemm(Xq, sx, next_pw(), out=Y, variant=v, workspace=ws),
                                 reps), 3) for v in variants}
            fam, splits = mq.plan(m, N, K)
            print(json.dumps({"layer": name, "K": K, "N": N, "M": m, "auto_family": fam, "auto_splits": splits,
                              "us": us}), flush=True)
            del X, Xq, sx, Y, ws
        del copies, pw0
        torch.cuda.synchronize()
        torch.cuda.empty_cache()


def summarize_sweep(args):
    """Markdown table of --sweep JSON lines: per layer and M, AUTO's choice and
    time, every family's time, and AUTO's time over the fastest family's."""
    out_md, paths = args.summarize_sweep[0], args.summarize_sweep[1:]
    fams = ["skinny", "tiled", "tiled_large", "medium"]
    lines = ["| layer | K → N | M | AUTO takes | AUTO µs | " + " | ".join(f"{f} µs" for f in fams) +
             " | fastest | AUTO / fastest |", "|" + "---|" * (7 + len(fams))]
    for path in paths:
        for line in open(path):
            if not line.startswith("{"):
                continue
            d = json.loads(line)
            us = d["us"]
            best = min((us[f], f) for f in fams if f in us)
            take = d["auto_family"] + (f" ({d['auto_splits']} K splits)" if d["auto_splits"] > 1 else "")
            cells = " | ".join(f"{us[f]:.1f}" if f in us else "-" for f in fams)
            lines.append(f"| {d['layer']} | {d['K']} → {d['N']} | {d['M']} | {take} | {us['auto']:.1f} | {cells} | "
                         f"{best[1]} | {us['auto'] / best[0]:.2f} |")
    with open(out_md, "a") as fh:
        fh.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    args = parse()
    if args.summarize_sweep:
        summarize_sweep(args)
        return
    if args.summarize_counters:
        summarize_counters(args)
        return
    if args.summarize_trace:
        summarize_trace(args)
        return
    if args.summarize_families:
        summarize_families(args)
        return
    if args.summarize_traffic:
        summarize_traffic(*args.summarize_traffic, m=max(int(x) for x in args.ms.split(",")))
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if args.quick:
        args.steps, args.warmup, args.reps = 3, 1, 5
    if args.families:
        families(args)
        return
    if args.sweep:
        sweep(args)
        return
    if args.kernel_run:
        kernel_run(args)
        return
    if args.selection:
        selection(args)
        return

    import numpy as np
    import torch

    import paper_2606_15652_amd as mq
    import synth

    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    mq.load()
    dev = torch.device("cuda:0")
    layer = synth.workload("c2_4096")
    K, N, nnzb = layer.K, layer.N, layer.nnzb
    ms = [int(m) for m in args.ms.split(",")]

    # ---------------------------------------------------------------- setup
    W = torch.from_numpy(layer.weight()).to(dev)
    pw0 = mq.prepare_weight(W, nnzb)
    torch.cuda.synchronize()
    per_copy = pw0.nbytes
    ncopy = max(2, -(-ROTATE_BYTES // per_copy))
    copies = [pw0] + [mq.PackedWeight(N, K, pw0.Wq.clone(), pw0.s_w.clone(), pw0.rowptr.clone(),
                                      pw0.kb.clone(), pw0.Rq.clone(), pw0.s_r.clone())
                      for _ in range(ncopy - 1)]
    Xs = {m: torch.from_numpy(layer.act(m)).to(dev) for m in ms}
    Xqs = {m: torch.empty((m, mq.act_bytes(K)), dtype=torch.uint8, device=dev) for m in ms}
    sxs = {m: torch.empty((m,), dtype=torch.float16, device=dev) for m in ms}
    Ys = {m: torch.empty((m, N), dtype=torch.float16, device=dev) for m in ms}
    Ws = {m: torch.empty(max(1, mq.linear_workspace_bytes(m, N, K)), dtype=torch.uint8, device=dev) for m in ms}
    del W
    torch.cuda.synchronize()

    rot = [0]

    def next_pw():
        rot[0] = (rot[0] + 1) % ncopy
        return copies[rot[0]]

    def step():
        for m in ms:
            mq.linear(Xs[m], next_pw(), out=Ys[m], workspace=Ws[m])


    if args.traffic:
        # For rocprofv3 --pmc: TRAFFIC_CALLS GEMM dispatches at the largest M,
        # each on its own weight copy, then TRAFFIC_CALLS copies of 256 MiB.
        mdom = max(ms)
        mq.quantize_act(Xs[mdom], out=(Xqs[mdom], sxs[mdom]))     # the GEMM's own input
        for _ in range(TRAFFIC_CALLS):
            mq.fused_gemm(Xqs[mdom], sxs[mdom], next_pw(), out=Ys[mdom])
        # an elementwise kernel that reads and writes COPY_BYTES each (a
        # same-dtype copy_ could be served by a DMA engine, invisible to the counters)
        src = torch.ones(COPY_BYTES // 4, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(TRAFFIC_CALLS):
            torch.neg(src, out=dst)
        torch.cuda.synchronize()
        print(json.dumps({"traffic_run": True, "M": mdom, "calls": TRAFFIC_CALLS,
                          "copy_bytes": COPY_BYTES}), flush=True)
        return

    # ------------------------------------------------------------ timed steps
    # one graph replay = `steps` steps; warm-up replays of a separate graph
    warm = graph_of(torch, step, max(1, args.warmup))
    warm.replay()
    torch.cuda.synchronize()
    main_graph = graph_of(torch, step, args.steps)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    e0.record()
    main_graph.replay()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_per_step = e0.elapsed_time(e1) / args.steps

    eff_ops = sum(2.0 * m * N * K for m in ms)
    value = eff_ops / (ms_per_step * 1e-3) / 1e12

    # ------------------------------------------------------------ per-M rows
    rows = []
    for m in ms:
        ops, byts = algorithmic(m, N, K, nnzb)
        t_call = timed(torch, lambda: mq.linear(Xs[m], next_pw(), out=Ys[m], workspace=Ws[m]), args.reps)
        t_q = timed(torch, lambda: mq.quantize_act(Xs[m], out=(Xqs[m], sxs[m])), args.reps)
        t_gemm = timed(torch, lambda: mq.fused_gemm(Xqs[m], sxs[m], next_pw(), out=Ys[m]), args.reps)
        # the W4A8 variant (INT8 activations) on the same layer
        xq8 = torch.empty((m, 3 * K // 2), dtype=torch.uint8, device=dev)
        sx8 = torch.empty((m,), dtype=torch.float16, device=dev)
        t_q8 = timed(torch, lambda: mq.quantize_act8(Xs[m], out=(xq8, sx8)), args.reps)
        t_g8 = timed(torch, lambda: mq.fused_gemm_a8(xq8, sx8, next_pw(), out=Ys[m]), args.reps)
        del xq8, sx8
        row = {"M": m, "us_call": round(t_call, 3), "us_gemm": round(t_gemm, 3), "us_quant": round(t_q, 3),
               "us_gemm_w4a8": round(t_g8, 3), "us_quant_w4a8": round(t_q8, 3),
               "eff_tops": round(2.0 * m * N * K / (t_gemm * 1e-6) / 1e12, 2),
               "int8_peak_frac": round(ops / (t_gemm * 1e-6) / 1e12 / PEAK_I8_TOPS, 4),
               "hbm_frac": round(byts / (t_gemm * 1e-6) / 1e9 / PEAK_HBM_GBS, 4),
               "quant_hbm_frac": round(quant_bytes(m, K) / (t_q * 1e-6) / 1e9 / PEAK_HBM_GBS, 4)}
        rows.append(row)

    # hipBLASLt W16A16 on the same shapes, rotating fp16 weights
    if not args.no_blas:
        wb = torch.randn((N, K), dtype=torch.float16, device=dev) * 0.02
        nw = max(2, -(-ROTATE_BYTES // (N * K * 2)))
        wbs = [wb] + [wb.clone() for _ in range(nw - 1)]
        rb = [0]

        def next_wb():
            rb[0] = (rb[0] + 1) % nw
            return wbs[rb[0]]

        for row in rows:
            m = row["M"]
            x16 = Xs[m]
            t = timed(torch, lambda: torch.nn.functional.linear(x16, next_wb()), args.reps)
            row["us_w16a16"] = round(t, 3)
            row["w16a16_tops"] = round(2.0 * m * N * K / (t * 1e-6) / 1e12, 2)
            row["speedup_vs_w16a16"] = round(t / row["us_call"], 3)
        del wbs, wb

    # ------------------------------------------------------------ roofline
    mdom = max(ms)
    ops_dom, bytes_dom = algorithmic(mdom, N, K, nnzb)
    dom = next(r for r in rows if r["M"] == mdom)
    achieved = ops_dom / (dom["us_gemm"] * 1e-6) / 1e12
    traffic = None
    tpath = os.path.join(ROOT, "profiles", "fused_gemm_traffic.json")
    if os.path.exists(tpath):
        try:
            t = json.load(open(tpath))
            if t.get("src_hash") == src_hash(GEMM_SRC) and t.get("M") == mdom:
                traffic = t.get("bytes_per_launch")
        except (OSError, ValueError):
            traffic = None
    roofline = {"kernel": f"gemm_tiled_kernel M={mdom} N={N} K={K} nnzb={nnzb}",
                "bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_FP6_TOPS,
                "unit": "TOP/s", "frac": round(achieved / PEAK_FP6_TOPS, 4), "traffic": traffic,
                "int8_peak_frac": round(achieved / PEAK_I8_TOPS, 4),
                "algorithmic_ops": ops_dom, "algorithmic_bytes": bytes_dom}

    # ------------------------------------------------------------ CPU oracle
    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        oracle.build()
        Wn = layer.weight()
        ref = oracle.prepare_weight(Wn, nnzb)
        xs_np = {m: layer.act(m) for m in ms}
        oracle.linear(*oracle.quantize_act(xs_np[1]), ref)        # warm-up
        nsteps = 0
        c0 = time.perf_counter()
        while nsteps < CPU_MAX_STEPS and (nsteps == 0 or time.perf_counter() - c0 < CPU_MIN_S):
            for m in ms:
                xq, sx = oracle.quantize_act(xs_np[m])
                oracle.linear(xq, sx, ref)
            nsteps += 1
        cs = (time.perf_counter() - c0) / nsteps
        cpu = {"value": round(eff_ops / cs / 1e12, 6), "unit": "TOPS", "cores": oracle.num_threads(),
               "cpu_model": cpu_model(), "kind": "oracle", "seconds_per_step": round(cs, 3), "steps": nsteps,
               "sample": f"{nsteps} full step(s) of the same workload (M={','.join(map(str, ms))}: "
                         "activation quantisation + int64 GEMM + fp64 epilogue), weight "
                         "preparation excluded"}

    out = {
        "metric": "effective TOPS of fused W4A4+residual GEMM (with act quant) over M=1..4096",
        "value": round(value, 3), "unit": "TOPS", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "fp6_e2m3", "data": "synthetic",
        "config": {"workload": "LLaMA3-8B attention projection K=N=4096, 10% INT4 residual blocks, "
                               "M sweep", "K": K, "N": N, "ms": ms, "density": 0.10, "nnzb": nnzb,
                   "weight_copies": ncopy, "bytes_per_copy": per_copy},
        "per_m": rows, "roofline": roofline, "cpu_baseline": cpu,
        "wall_s_timed": round(wall, 3),
        "device": torch.cuda.get_device_name(0),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
