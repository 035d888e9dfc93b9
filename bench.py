"""Benchmark: SonicMoE layer forward+backward on one MI355X.

One step = the whole hot path on one batch: router GEMM + softmax/top-K +
routing metadata, token rounding (NR-f, M_tile = 128), forward (up-proj with
SwiGLU, down-proj, aggregation) and backward (dH with dS/A', dW2, dX~, dW1,
dX aggregation with the router gradient, dW_r).  Inputs are seeded synthetic
tensors already resident in HBM.  Prints one JSON line.

Model FLOPs per step are 18 * d * n * sum_e f_e over the rounded expert counts
(the paper's model-FLOP accounting); router FLOPs are not counted.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
FLUSH_BYTES = 512 << 20     # scratch written before each timed step: more than L2 (8 x 4 MB) + Infinity Cache (256 MB)
TRAFFIC_PROFILE = os.path.join(ROOT, "profiles", "l2_fabric_traffic_7b_tr128.md")

# kernel-name fragment -> kernel class (as in the library's timing classes)
KERNEL_CLASS_OF = [("OpUp<", "up_proj"), ("OpDown<", "down_proj"), ("OpDH<", "dH"), ("OpDW2<", "dW2"),
                   ("OpDXt<", "dXtilde"), ("OpDW1<", "dW1"), ("OpDWr<", "dWr"), ("OpRouter<", "router_gemm"),
                   ("OpRouterTopk<", "router_topk"),
                   ("agg_o_kernel", "aggregate_O"), ("agg_dx_kernel", "aggregate_dX"),
                   ("topk_lane_kernel", "topk"), ("topk_route_kernel", "topk"),
                   ("tr_local_kernel", "tr_local"), ("tr_reduce_kernel", "tr_reduce"), ("tr_merge_kernel", "tr_merge"),
                   ("token_count_kernel", "token_count"), ("token_place_kernel", "token_place")]


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def quantile(sorted_vals, q):
    """Linear-interpolation quantile of an ascending list."""
    if not sorted_vals:
        return float("nan")
    x = q * (len(sorted_vals) - 1)
    i = int(x)
    j = min(i + 1, len(sorted_vals) - 1)
    return sorted_vals[i] + (sorted_vals[j] - sorted_vals[i]) * (x - i)


def kernel_source_hash() -> str:
    """sha256 over the HIP/C++ sources of the library (sorted by file name), with comments and runs of
    whitespace removed, so that an edit of comments alone keeps a profile of unchanged kernels valid."""
    import hashlib
    import re
    h = hashlib.sha256()
    d = os.path.join(ROOT, "paper_2512_14080_amd", "csrc")
    for f in sorted(os.listdir(d)):
        if f.endswith((".hip", ".h", ".cpp")):
            h.update(f.encode())
            with open(os.path.join(d, f), encoding="utf-8") as fh:
                text = fh.read()
            text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
            text = re.sub(r"//[^\n]*", " ", text)
            h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def _pmc_per_dispatch(run_dir, counters):
    """Mean per dispatch of rocprofv3 counters, by kernel name: {kernel: {counter: value}}."""
    import csv
    import glob
    files = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {run_dir}")
    tot, disp = {}, {}
    for f in files:
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] not in counters:
                    continue
                k = r["Kernel_Name"]
                d = tot.setdefault(k, {})
                d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
                disp.setdefault(k, set()).add(r["Dispatch_Id"])
    return {k: {c: v / len(disp[k]) for c, v in d.items()} for k, d in tot.items()}


READ_COUNTERS = ["TCC_EA0_RDREQ", "TCC_EA0_RDREQ_32B", "TCC_EA0_RDREQ_64B", "TCC_EA0_RDREQ_128B"]
WRITE_COUNTERS = ["TCC_EA0_WRREQ", "TCC_EA0_WRREQ_64B"]


def _read_bytes(c):
    return 32.0 * c.get("TCC_EA0_RDREQ_32B", 0) + 64.0 * c.get("TCC_EA0_RDREQ_64B", 0) + \
        128.0 * c.get("TCC_EA0_RDREQ_128B", 0)


def _write_bytes(c):
    n, n64 = c.get("TCC_EA0_WRREQ", 0), c.get("TCC_EA0_WRREQ_64B", 0)
    return 64.0 * n64 + 32.0 * (n - n64)


def _stats_avg_s(stats_csv):
    """{kernel class: mean launch duration in s} from a rocprofv3 --stats kernel summary."""
    import csv
    tot = {}
    with open(stats_csv) as fh:
        for r in csv.DictReader(fh):
            cls = next((cl for frag, cl in KERNEL_CLASS_OF if frag in r["Name"]), None)
            if cls is None:
                continue
            t, n = tot.get(cls, (0.0, 0))
            tot[cls] = (t + float(r["TotalDurationNs"]) * 1e-9, n + int(r["Calls"]))
    return {c: t / n for c, (t, n) in tot.items() if n}


def traffic_report(read_dir, write_dir, copy_read_dir, copy_write_dir, copy_bytes, stats_csv=None):
    """Markdown summary of the bytes each kernel class moves between the L2 and the memory fabric per launch.

    Reads are the L2's read requests to the fabric by size (TCC_EA0_RDREQ_32B/_64B/_128B), writes its write
    requests (TCC_EA0_WRREQ, of which TCC_EA0_WRREQ_64B are 64-byte, the rest 32-byte).  These bytes include
    Infinity Cache (MALL) hits: the L2 counters cannot tell which requests reach DRAM.  A plain device copy of
    copy_bytes calibrates the sizes (it should read and write copy_bytes).  With stats_csv (a rocprofv3 --stats
    kernel summary of the same workload) the table adds each class's mean launch time and the bytes it moved
    per second."""
    cr = _pmc_per_dispatch(copy_read_dir, READ_COUNTERS)
    cw = _pmc_per_dispatch(copy_write_dir, WRITE_COUNTERS)
    ck = [k for k in cr if "copyBuffer" in k or "copy" in k.lower()]
    if not ck:
        raise RuntimeError("no copy kernel in the calibration run")
    rd = _pmc_per_dispatch(read_dir, READ_COUNTERS)
    wr = _pmc_per_dispatch(write_dir, WRITE_COUNTERS)
    copy_r, copy_w = _read_bytes(cr[ck[0]]), _write_bytes(cw[ck[0]])
    sized = sum(cr[ck[0]].get(c, 0) for c in READ_COUNTERS[1:])
    rows = []
    for frag, cls in KERNEL_CLASS_OF:
        ks = [k for k in rd if frag in k]
        if not ks:
            continue
        r = sum(_read_bytes(rd[k]) for k in ks) / len(ks)
        w = sum(_write_bytes(wr.get(k, {})) for k in ks) / len(ks)
        rows.append((cls, r, w))
    run = "python3 bench.py --steps 2 --warmup 1 --no-cpu-baseline"
    lines = [
        "# L2-to-fabric traffic per launch: 7B layer step (T=32768, d=1536, n=256, E=128, K=8), token rounding "
        "M_tile=128 nearest",
        "",
        "Commands (repository root, one MI355X; each counter set in a run of its own):",
        "",
        "```",
        f"rocprofv3 --pmc {' '.join(READ_COUNTERS)} --output-format csv -d {read_dir} -o run -- {run}",
        f"rocprofv3 --pmc {' '.join(WRITE_COUNTERS)} --output-format csv -d {write_dir} -o run -- {run}",
        f"rocprofv3 --pmc {' '.join(READ_COUNTERS)} --output-format csv -d {copy_read_dir} -o run -- "
        f"python3 bench.py --copy-calibration {copy_bytes}",
        f"rocprofv3 --pmc {' '.join(WRITE_COUNTERS)} --output-format csv -d {copy_write_dir} -o run -- "
        f"python3 bench.py --copy-calibration {copy_bytes}",
        f"python3 bench.py --traffic-report {read_dir} {write_dir} {copy_read_dir} {copy_write_dir} {copy_bytes}"
        + (f" {stats_csv}" if stats_csv else ""),
        "```",
        "",
        "Bytes are the L2's requests to the memory fabric, by request size: reads 32 B x RDREQ_32B + 64 B x "
        "RDREQ_64B + 128 B x RDREQ_128B, writes 64 B x WRREQ_64B + 32 B x the other WRREQ.  They include Infinity "
        "Cache (MALL) hits, which these counters cannot separate from DRAM accesses: this is L2-miss traffic, an "
        "upper bound on DRAM traffic.",
        "",
        f"Calibration: a device copy of {copy_bytes} bytes reads {copy_r:.0f} and writes {copy_w:.0f} bytes by "
        f"these counters (sized read requests {sized:.0f} of {cr[ck[0]].get('TCC_EA0_RDREQ', 0):.0f} total).",
        "",
    ]
    avg = _stats_avg_s(stats_csv) if stats_csv else None
    if avg is not None:
        lines += [f"Launch times: mean durations from `{stats_csv}` (a rocprofv3 --kernel-trace --stats run of the "
                  "same workload); GB/s = total bytes per launch / mean launch time.", ""]
        lines += ["| kernel class | read bytes/launch | write bytes/launch | total bytes/launch | avg us | GB/s |",
                  "|---|---|---|---|---|---|"]
    else:
        lines += ["| kernel class | read bytes/launch | write bytes/launch | total bytes/launch |", "|---|---|---|---|"]
    for cls, r, w in rows:
        if avg is not None and cls in avg:
            lines.append(f"| {cls} | {r:.0f} | {w:.0f} | {r + w:.0f} | {avg[cls] * 1e6:.1f} | "
                         f"{(r + w) / avg[cls] / 1e9:.0f} |")
        elif avg is not None:
            lines.append(f"| {cls} | {r:.0f} | {w:.0f} | {r + w:.0f} | | |")
        else:
            lines.append(f"| {cls} | {r:.0f} | {w:.0f} | {r + w:.0f} |")
    lines += ["", f"kernel sources sha256: {kernel_source_hash()}", ""]
    return "\n".join(lines)


MFMA_COUNTERS = ["SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_BUSY_CYCLES", "GRBM_GUI_ACTIVE"]
MI355X_SIMDS = 256 * 4      # compute units x SIMDs
MI355X_XCDS = 8             # GRBM_GUI_ACTIVE sums the busy cycles of the eight XCDs
FLOP_PER_MFMA_MOP = 512     # SQ_INSTS_VALU_MFMA_MOPS_* count in units of 512 FLOPs


def mfma_report(pmc_dir):
    """Markdown summary of the matrix-core work and utilisation of each GEMM class from one rocprofv3 --pmc
    run of MFMA_COUNTERS: bf16 MFMA FLOPs per launch (512 per counted MOP), the achieved rate over the
    dispatch's own timestamps against the 2.5 PFLOP/s dense peak, the clock the dispatch ran at (busy cycles
    per XCD over its duration) and the share of SIMD cycles the MFMA pipe was busy."""
    import csv
    import glob
    files = glob.glob(os.path.join(pmc_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {pmc_dir}")
    disp = {}  # dispatch id -> (kernel name, duration s, {counter: value})
    for f in files:
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] not in MFMA_COUNTERS:
                    continue
                k = (f, r["Dispatch_Id"])
                dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-9
                ent = disp.setdefault(k, (r["Kernel_Name"], dur, {}))
                ent[2][r["Counter_Name"]] = ent[2].get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    by_cls = {}
    for name, dur, c in disp.values():
        cls = next((cl for frag, cl in KERNEL_CLASS_OF if frag in name), None)
        if cls is not None and c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0) > 0:
            by_cls.setdefault(cls, []).append((dur, c))
    run = "python3 bench.py --steps 2 --warmup 1 --no-cpu-baseline"
    lines = [
        "# MFMA work and utilisation per GEMM launch: 7B layer step (T=32768, d=1536, n=256, E=128, K=8), token "
        "rounding M_tile=128 nearest",
        "",
        "Commands (repository root, one MI355X):",
        "",
        "```",
        f"rocprofv3 --pmc {' '.join(MFMA_COUNTERS)} --output-format csv -d {pmc_dir} -o run -- {run}",
        f"python3 bench.py --mfma-report {pmc_dir}",
        "```",
        "",
        f"Per launch, averaged over the dispatches of the run: bf16 MFMA FLOPs = {FLOP_PER_MFMA_MOP} x "
        "SQ_INSTS_VALU_MFMA_MOPS_BF16; time = the dispatch's end minus start timestamp; TFLOP/s = FLOPs / time, "
        "against the 2.5 PFLOP/s dense bf16 peak (1024 SIMDs x 1024 FLOP per cycle x 2.4 GHz); clock = "
        f"GRBM_GUI_ACTIVE / {MI355X_XCDS} XCDs / time; MFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / "
        f"{MI355X_XCDS} x {MI355X_SIMDS} SIMDs), the share of SIMD cycles at the clock the kernel ran at in which "
        "the matrix pipe was busy.  Under the power limit the clock falls below 2.4 GHz while the pipe is busy, "
        "so the fraction of peak is below the busy share.  For launches of a few tens of microseconds the "
        "counters' window is wider than the timestamps, which inflates their clock column.",
        "",
        "| kernel class | launches | MFMA GFLOP/launch | avg us | TFLOP/s | % of peak | clock GHz | MFMA busy |",
        "|---|---|---|---|---|---|---|---|",
    ]
    for _, cls in KERNEL_CLASS_OF:
        if cls not in by_cls:
            continue
        ent = by_cls.pop(cls)
        n = len(ent)
        t = sum(d for d, _ in ent) / n
        mean = {c: sum(e[1].get(c, 0.0) for e in ent) / n for c in MFMA_COUNTERS}
        flops = FLOP_PER_MFMA_MOP * mean["SQ_INSTS_VALU_MFMA_MOPS_BF16"]
        cyc = mean["GRBM_GUI_ACTIVE"] / MI355X_XCDS
        busy = mean["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * MI355X_SIMDS) if cyc else float("nan")
        clock = cyc / t / 1e9 if t else float("nan")
        rate = flops / t / 1e12 if t else float("nan")
        lines.append(f"| {cls} | {n} | {flops / 1e9:.1f} | {t * 1e6:.1f} | {rate:.0f} | "
                     f"{100 * rate / PEAK_BF16_TFLOPS:.1f} | {clock:.2f} | {100 * busy:.1f}% |")
    lines += ["", f"kernel sources sha256: {kernel_source_hash()}", ""]
    return "\n".join(lines)


def stats_report(stats_csv, title, command):
    """Markdown table of a rocprofv3 --stats kernel summary (kernel_stats.csv)."""
    import csv
    rows = list(csv.DictReader(open(stats_csv)))
    out = [f"# {title}", "", "Command (run from the repository root on one MI355X):", "", "```", command, "```", "",
           f"Table: `python3 bench.py --stats-report {stats_csv} TITLE COMMAND` (this file's title and command).", "",
           "| kernel | calls | avg us | min us | max us | % of GPU time |", "|---|---|---|---|---|---|"]
    for r in sorted(rows, key=lambda r: -float(r["TotalDurationNs"])):
        name = r["Name"].replace("smoe::", "").replace("|", "/")
        if len(name) > 80:
            name = name[:77] + "..."
        out.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                   f"{float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.2f} |")
    return "\n".join(out) + "\n"


def measured_traffic(kernel_class):
    """L2-to-fabric bytes per launch from the committed profile, if the kernels are unchanged since."""
    try:
        with open(TRAFFIC_PROFILE) as fh:
            text = fh.read()
    except OSError:
        return None
    if f"kernel sources sha256: {kernel_source_hash()}" not in text:
        return None
    for line in text.splitlines():
        cells = [c.strip() for c in line.strip().strip("|").split("|")]
        if len(cells) >= 4 and cells[0] == kernel_class:
            try:
                return float(cells[3])
            except ValueError:
                return None
    return None


def kernel_work(cls, cfg, P, T):
    """Algorithmic work of one launch of a kernel class: (amount, unit, bound).

    GEMMs count their FLOPs and their unique operand and result bytes (each tensor once; gathered rows counted
    as the tensor they are gathered from) and are bound by whichever takes longer at peak: MFMA or HBM."""
    d, n, E, K = cfg.d, cfg.n, cfg.E, cfg.K
    gemm = gemm_work(cfg, P, T)
    if cls in gemm:
        f, b = gemm[cls]
        if b / (PEAK_HBM_GBS * 1e9) > f / (PEAK_BF16_TFLOPS * 1e12):
            return b, "GB/s", "hbm"
        return f, "TFLOP/s", "mfma"
    hbm = {
        # read the P rows of Y (bf16) + weights/indices, write O
        "aggregate_O": 2.0 * P * d + 8.0 * P + 2.0 * T * d,
        "aggregate_dX": 2.0 * P * d + 12.0 * P + 2.0 * T * d + 2.0 * T * E,
        # read the logits, write the scores (token-major and transposed), the
        # top-K lists and the membership bitmap
        "topk": 12.0 * T * E + 8.0 * T * K + T * E / 8.0,
    }
    if cls in hbm:
        return hbm[cls], "GB/s", "hbm"
    return None, None, None


def gemm_work(cfg, P, T):
    """{GEMM kernel class: (FLOPs, unique operand and result bytes)} of one launch."""
    d, n, E = cfg.d, cfg.n, cfg.E
    return {  # FLOPs, bytes
        "up_proj": (2.0 * P * d * 2 * n, 2.0 * T * d + 2.0 * E * d * 2 * n + 2.0 * P * 2 * n + 2.0 * P * n),
        "down_proj": (2.0 * P * n * d, 2.0 * P * n + 2.0 * E * n * d + 2.0 * P * d),
        "dH": (2.0 * P * d * n, 2.0 * T * d + 2.0 * E * n * d + 2 * 2.0 * P * 2 * n + 2.0 * P * n + 4.0 * P),
        "dW2": (2.0 * P * n * d, 2.0 * P * n + 2.0 * T * d + 2.0 * E * n * d),
        "dXtilde": (2.0 * P * 2 * n * d, 2.0 * P * 2 * n + 2.0 * E * d * 2 * n + 2.0 * P * d),
        "dW1": (2.0 * P * d * 2 * n, 2.0 * T * d + 2.0 * P * 2 * n + 2.0 * E * d * 2 * n),
        "router_gemm": (2.0 * T * d * E, 2.0 * T * d + 2.0 * d * E + 4.0 * T * E),
        # X and W_r in; scores token- and expert-major (the rounded layer's
        # step writes both), the top-K lists and the membership bitmap out
        "router_topk": (2.0 * T * d * E, 2.0 * T * d + 2.0 * d * E + 8.0 * T * E + 8.0 * T * cfg.K + T * E / 8.0),
        "dWr": (2.0 * T * d * E, 2.0 * T * d + 2.0 * T * E + 4.0 * d * E),
    }


# the expert computation without router or routing (steps up-proj .. dX aggregation)
MOE_ONLY_CLASSES = ("up_proj", "down_proj", "aggregate_O", "dH", "dW2", "dXtilde", "dW1", "aggregate_dX")


def kernel_table(per, cfg, P):
    """Achieved rate of every kernel class with an algorithmic work model, against its own peak."""
    out = {}
    for c, t in per.items():
        work, unit, bound = kernel_work(c, cfg, P, cfg.T)
        if work is None or t <= 0:
            continue
        if unit == "TFLOP/s":
            a, peak = work / (t * 1e-3) / 1e12, PEAK_BF16_TFLOPS
        else:
            a, peak = work / (t * 1e-3) / 1e9, PEAK_HBM_GBS
        out[c] = {"ms": round(t, 5), "bound": bound, "achieved": round(a, 1), "unit": unit,
                  "frac": round(a / peak, 4)}
    return out


def padding_rows(layer):
    """Rows that 128-row MFMA blocks compute beyond the routed ones: sum_e (ceil(f_e / 128) * 128 - f_e)."""
    counts = layer.routing.arrays()["counts"].cpu().numpy().astype("int64")
    return int(((counts + 127) // 128 * 128 - counts).sum())


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(cfg, round_mode, inp, budget_s=8.0, repeats=3):
    """Time the CPU oracle (route + round + fwd + bwd, fp32) on a token sample of the workload.

    The sample is the first T' tokens of the same seeded inputs (full d, n, E, K), sized so one run takes
    about budget_s; the reported time is the median of `repeats` runs."""
    import statistics

    import numpy as np

    import oracle

    Xa, Wr, W1, W2, dOa = (inp.f32(k) for k in ("X", "Wr", "W1", "W2", "dO"))

    def run(T):
        X, dO = Xa[:T], dOa[:T]
        t0 = time.perf_counter()
        S, idx, R = oracle.route(X, Wr, cfg.K, bias=inp.bias, dtype=np.float32)
        if round_mode:
            member, _, _ = oracle.round_tokens(S, R.member, cfg.m_tile, mode=round_mode)
            R = oracle.routing_from_membership(member, S, np.float32)
        fw = oracle.forward(X, W1, W2, R)
        oracle.backward(dO, X, fw["H"], W1, W2, Wr, R)
        return time.perf_counter() - t0, R.P

    T = min(cfg.T, 1024)
    dt, P = run(T)
    if dt < budget_s / 3 and T < cfg.T:
        T = int(min(cfg.T, max(T, T * budget_s / max(dt, 1e-3) * 0.8)))
        T = max(64, T // 64 * 64)
    times = []
    for _ in range(repeats):
        dt, P = run(T)
        times.append(dt)
    dt = statistics.median(times)
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = os.cpu_count()
    tflops = cfg.model_flops(P) / dt / 1e12
    return {"value": round(tflops, 6), "unit": "TFLOPS", "cores": int(threads), "kind": "oracle",
            "host_cpus": os.cpu_count(), "blas_threads": int(threads), "cpu_model": cpu_model(),
            "runs_s": [round(t, 3) for t in times],
            "sample": f"{T} of {cfg.T} tokens of the {cfg.name} layer (full d, n, E, K), "
                      f"route+{'round+' if round_mode else ''}fwd+bwd in fp32 NumPy, median of {repeats} runs "
                      f"{dt:.2f} s, {T / dt:.1f} tokens/s"}


def measure(args, cfg, cpu):
    """One layer configuration: warm-up, per-kernel-class times, the timed steps; the JSON record."""
    import torch

    from paper_2512_14080_amd import binding as B
    from paper_2512_14080_amd import workloads as W
    from paper_2512_14080_amd.layer import DeviceLayer

    round_mode = None if args.round == "none" else args.round
    log(f"[bench] config {cfg}, rounding {round_mode}")
    inp = W.make_inputs(cfg, 0)
    # the logits feed nothing after the softmax: the step does not keep them
    layer = DeviceLayer(inp, round_mode=round_mode, keep_logits=False)
    stream = torch.cuda.current_stream()
    for _ in range(max(1, args.warmup)):
        layer.step()
    torch.cuda.synchronize()
    P = layer.rows()
    log(f"[bench] warmup done, rows P = {P}")

    # per-kernel-class times (HIP events on the launch stream), a short pass
    classes = B.KERNEL_CLASSES
    per = {}
    for c in classes:
        B.moe_prof_select(c)
        for _ in range(3 if args.breakdown else 2):
            layer.step()
        ms, nl = B.moe_prof_read()
        if nl:
            per[c] = ms / nl
    B.moe_prof_select(-1)
    B.moe_prof_read()
    cands = {c: t for c, t in per.items() if kernel_work(c, cfg, P, cfg.T)[0] is not None}
    dominant = max(cands, key=cands.get)
    log("[bench] per-launch ms: " + ", ".join(f"{c}={t:.4f}" for c, t in per.items()))

    # back-to-back steps without any timing hooks (the caches keep what the previous step left)
    torch.cuda.synchronize()
    eb0, eb1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    eb0.record(stream)
    for _ in range(args.steps):
        layer.step()
    eb1.record(stream)
    torch.cuda.synchronize()
    ms_b2b = eb0.elapsed_time(eb1) / args.steps

    # timed region: K steps, each after a write of FLUSH_BYTES of scratch (L2 and the Infinity Cache start
    # cold) and bracketed by its own events; the dominant kernel's launches are bracketed by the library's
    # events on the launch stream
    flush = torch.empty(FLUSH_BYTES // 4, dtype=torch.int32, device="cuda")
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    B.moe_prof_select(dominant)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        flush.fill_(i)
        evs[i][0].record(stream)
        layer.step()
        evs[i][1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    dom_ms, dom_n = B.moe_prof_read()
    B.moe_prof_select(-1)
    del flush
    step_ms = sorted(a.elapsed_time(b) for a, b in evs)
    ms_step = quantile(step_ms, 0.5)
    log(f"[bench] timed {args.steps} flushed steps: median {ms_step:.4f} ms/step, p10 {quantile(step_ms, 0.1):.4f}, "
        f"p90 {quantile(step_ms, 0.9):.4f} (wall incl. flushes {wall * 1e3 / args.steps:.4f} ms/step); "
        f"back-to-back without hooks {ms_b2b:.4f} ms/step")

    flops = cfg.model_flops(P)
    tflops = flops / (ms_step * 1e-3) / 1e12
    work, unit, bound = kernel_work(dominant, cfg, P, cfg.T)
    dom_avg = dom_ms / max(dom_n, 1)
    if unit == "TFLOP/s":
        achieved = work / (dom_avg * 1e-3) / 1e12
        peak = PEAK_BF16_TFLOPS
    else:
        achieved = work / (dom_avg * 1e-3) / 1e9
        peak = PEAK_HBM_GBS
    out = {
        "metric": "MoE layer fwd+bwd TFLOPS and tokens/s on 1 MI355X (% of bf16 MFMA peak)",
        "value": round(tflops, 3), "unit": "TFLOPS", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "step_ms": {"median": round(ms_step, 4), "mean": round(sum(step_ms) / len(step_ms), 4),
                    "p10": round(quantile(step_ms, 0.1), 4), "p90": round(quantile(step_ms, 0.9), 4),
                    "min": round(step_ms[0], 4), "max": round(step_ms[-1], 4),
                    "timing": f"each step after a {FLUSH_BYTES >> 20} MiB scratch write, own HIP events",
                    "back_to_back_mean": round(ms_b2b, 4)},
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: T={cfg.T} d={cfg.d} n={cfg.n} E={cfg.E} K={cfg.K} "
                               f"{'token rounding ' + round_mode + ' M_tile=' + str(cfg.m_tile) if round_mode else 'token choice'}",
                   "T": cfg.T, "d": cfg.d, "n": cfg.n, "E": cfg.E, "K": cfg.K,
                   "m_tile": cfg.m_tile if round_mode else None, "rows": P},
        "tokens_per_s": round(cfg.T / (ms_step * 1e-3), 1),
        "pct_bf16_peak": round(100.0 * tflops / PEAK_BF16_TFLOPS, 2),
        "roofline": {"kernel": dominant, "bound": bound, "achieved": round(achieved, 2), "peak": peak,
                     "unit": unit, "frac": round(achieved / peak, 4), "traffic": measured_traffic(dominant),
                     "traffic_note": "bytes per launch between L2 and the memory fabric from the TCC request "
                                     "counters by size (includes Infinity Cache hits; an upper bound on DRAM bytes)",
                     "launch_ms": round(dom_avg, 5), "launches": dom_n},
        "kernel_ms": {c: round(t, 5) for c, t in per.items()},
        "kernels": kernel_table(per, cfg, P),
        "moe_only_ms": round(sum(per.get(c, 0.0) for c in MOE_ONLY_CLASSES), 4),
        "padding_rows": padding_rows(layer),
    }
    if cpu:
        log("[bench] timing the CPU oracle on a sample ...")
        out["cpu_baseline"] = cpu_baseline(cfg, round_mode, inp)
    return out


def ablation(args):
    """Evidence for three design choices at the layer's shape (one JSON line each, not the benchmark record):
    gather-and-sum aggregation against a scatter-fused store + contiguous sum and fp32 atomics, the fused top-K
    router kernel against softmax + top-K in torch on the same logits, and the gathered inputs
    of up-proj, dH and dW1 against the same GEMMs on inputs already laid out per expert (a token-per-row layer
    with K = 1 whose tokens come sorted by expert, so every gather index is the identity)."""
    import numpy as np
    import torch

    from paper_2512_14080_amd import binding as B
    from paper_2512_14080_amd import workloads as W
    from paper_2512_14080_amd.layer import DeviceLayer

    cfg = W.CONFIGS[args.config]

    def class_ms(layer, classes, reps=5):
        out = {}
        for c in classes:
            B.moe_prof_select(c)
            for _ in range(reps):
                layer.step()
            ms, nl = B.moe_prof_read()
            out[c] = round(ms / nl, 5) if nl else None
        B.moe_prof_select(-1)
        return out

    layer = DeviceLayer(W.make_inputs(cfg, 0), round_mode="nearest", keep_logits=False)
    for _ in range(3):
        layer.step()
    P = layer.rows()
    gathered = class_ms(layer, ["router_topk", "up_proj", "dH", "dW1"])
    # the same routing as two launches (router GEMM, then softmax/top-K on the logits)
    fused_flags = layer.route_flags
    layer.route_flags = fused_flags | B.MOE_ROUTE_SEPARATE_TOPK
    gathered.update(class_ms(layer, ["router_gemm", "topk"]))
    layer.route_flags = fused_flags

    # expert-aggregation strategies: down-projection epilogue + aggregation kernel(s) per forward
    from paper_2512_14080_amd.layer import _aligned_empty
    ws = _aligned_empty(B.moe_workspace_bytes(layer.D, layer.routing.capacity, B.MOE_WS_FWD_AGG_ABLATION))
    O = torch.empty_like(layer.O)
    agg = {}
    for name in B.AGG_STRATEGIES:
        def fwd():
            B.moe_fwd_aggregation_ablation(layer.D, layer.X, layer.W1, layer.W2, layer.routing, layer.H, O, name, ws)
        for _ in range(3):
            fwd()
        t = {}
        for c in ("down_proj", "aggregate_O"):
            B.moe_prof_select(c)
            for _ in range(10):
                fwd()
            ms, nl = B.moe_prof_read()
            t[c] = ms / nl
        B.moe_prof_select(-1)
        agg[name] = {"down_ms": round(t["down_proj"], 5), "aggregation_ms": round(t["aggregate_O"], 5),
                     "total_ms": round(t["down_proj"] + t["aggregate_O"], 5)}
    print(json.dumps({"ablation": "expert aggregation", "workload": f"{cfg.name}: P={P} rows, d={cfg.d}",
                      "strategies": agg,
                      "note": "down_ms of scatter_sum includes the slot-map launch, of atomic_f32 the fp32 fill; "
                              "aggregation_ms of atomic_f32 is the fp32 -> bf16 conversion"}), flush=True)
    del ws, O, layer
    torch.cuda.empty_cache()

    g = torch.Generator(device="cuda").manual_seed(0)
    logits = torch.randn(cfg.T, cfg.E, device="cuda", generator=g)

    def torch_route():
        s = torch.softmax(logits, dim=1)
        v, i = torch.topk(s, cfg.K, dim=1)
        return s, v / v.sum(dim=1, keepdim=True), i

    for _ in range(3):
        torch_route()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(20):
        torch_route()
    e1.record()
    torch.cuda.synchronize()
    t_torch = e0.elapsed_time(e1) / 20
    rd = cfg.T * cfg.E * 4 / 1e9
    print(json.dumps({"ablation": "top-K router", "workload": f"T={cfg.T} E={cfg.E} K={cfg.K} fp32 logits",
                      "fused_kernel_ms": gathered["topk"], "torch_softmax_topk_ms": round(t_torch, 5),
                      "fused_logit_read_GBps": round(rd / (gathered["topk"] * 1e-3), 1),
                      "torch_logit_read_GBps": round(rd / (t_torch * 1e-3), 1),
                      "note": "the fused kernel also writes the transposed scores and the membership bitmap"}),
          flush=True)
    if gathered.get("router_topk") is not None:
        two = gathered["router_gemm"] + gathered["topk"]
        print(json.dumps({"ablation": "router GEMM with softmax/top-K in its epilogue",
                          "workload": f"T={cfg.T} d={cfg.d} E={cfg.E} K={cfg.K}",
                          "one_launch_ms": gathered["router_topk"], "router_gemm_ms": gathered["router_gemm"],
                          "topk_ms": gathered["topk"], "two_launches_ms": round(two, 5)}), flush=True)
    del logits
    torch.cuda.empty_cache()

    # the same GEMM work on inputs laid out per expert: P tokens, one expert each, sorted by expert
    per_e = max(cfg.m_tile, round(P / cfg.E / cfg.m_tile) * cfg.m_tile)
    cc = W.MoEConfig("contiguous", T=per_e * cfg.E, d=cfg.d, n=cfg.n, E=cfg.E, K=1, m_tile=cfg.m_tile)
    S = np.zeros((cc.T, cc.E), dtype=np.float32)
    S[np.arange(cc.T), np.arange(cc.T) // per_e] = 1.0
    layer = DeviceLayer(W.make_inputs(cc, 0), round_mode=None, scores_in=S)
    for _ in range(3):
        layer.step()
    contiguous = class_ms(layer, ["up_proj", "dH", "dW1"])
    print(json.dumps({"ablation": "gathered vs contiguous inputs", "workload": f"{cfg.name}: P={P} rows "
                      f"(contiguous: {cc.T} tokens, K=1, {per_e} per expert)",
                      "gathered_ms": {c: gathered[c] for c in contiguous}, "contiguous_ms": contiguous}),
          flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="7b")
    ap.add_argument("--round", default="nearest", help="rounding mode, or 'none' for token-choice routing")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--breakdown", action="store_true", help="also time every kernel class")
    ap.add_argument("--ablation", action="store_true",
                    help="fused top-K vs torch, gathered vs contiguous GEMM inputs (JSON lines, not the record)")
    ap.add_argument("--sweep", default=None,
                    help="measure every layer of a named sweep (e.g. 'paper': the paper's benchmark shapes), "
                         "one JSON line each, no CPU baseline")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run one plain device copy of BYTES (HBM counter calibration) and exit")
    ap.add_argument("--traffic-report", nargs="+", metavar="ARG",
                    help="READ_DIR WRITE_DIR COPY_READ_DIR COPY_WRITE_DIR COPY_BYTES [KERNEL_STATS_CSV]: print the "
                         "L2-to-fabric traffic markdown summary from rocprofv3 counter runs and exit")
    ap.add_argument("--stats-report", nargs=3, metavar=("KERNEL_STATS_CSV", "TITLE", "COMMAND"),
                    help="print a rocprofv3 --stats kernel summary as markdown and exit")
    ap.add_argument("--mfma-report", metavar="PMC_DIR",
                    help="print the MFMA work and utilisation of a rocprofv3 --pmc run of MFMA_COUNTERS and exit")
    args = ap.parse_args()
    if args.traffic_report:
        if len(args.traffic_report) not in (5, 6):
            ap.error("--traffic-report takes 5 or 6 arguments")
        fd, wd, cfd, cwd, nb = args.traffic_report[:5]
        stats = args.traffic_report[5] if len(args.traffic_report) == 6 else None
        print(traffic_report(fd, wd, cfd, cwd, int(nb), stats))
        return
    if args.stats_report:
        print(stats_report(*args.stats_report), end="")
        return
    if args.mfma_report:
        print(mfma_report(args.mfma_report), end="")
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}): the layer is built and measured on a "
              f"single MI355X; how the layer would shard over GPUs is described, not implemented.", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_calibration:
        a = torch.ones(args.copy_calibration, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        torch.cuda.synchronize()
        b.copy_(a)
        torch.cuda.synchronize()
        log(f"[bench] copied {args.copy_calibration} bytes once")
        return

    from paper_2512_14080_amd import binding as B
    from paper_2512_14080_amd import workloads as W

    B.lib()  # fail loudly if the library is missing
    if args.ablation:
        ablation(args)
        return
    if args.sweep:
        for name in W.SWEEPS[args.sweep]:
            out = measure(args, W.CONFIGS[name], cpu=False)
            print(json.dumps(out), flush=True)
            log(f"[sweep] {name}: {out['ms_per_step']:.3f} ms/step, {out['value']:.1f} TFLOPS "
                f"({out['pct_bf16_peak']:.1f}% of peak), MoE only {out['moe_only_ms']:.3f} ms")
        return
    out = measure(args, W.CONFIGS[args.config], cpu=not args.no_cpu_baseline)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
