"""Host-side logic of bench.py (no GPU): quantiles, the per-launch work model,
the rocprofv3 summaries it writes into profiles/, the source hash that keeps a
traffic profile tied to the kernels it measured, and the one-GPU rule."""
import csv
import math
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2512_14080_amd import workloads as W  # noqa: E402


def test_quantile_matches_numpy_linear():
    rng = np.random.default_rng(3)
    for n in (1, 2, 5, 20):
        v = sorted(rng.random(n).tolist())
        for q in (0.0, 0.1, 0.5, 0.9, 1.0):
            assert bench.quantile(v, q) == pytest.approx(float(np.quantile(v, q)), rel=1e-12, abs=1e-15)
    assert math.isnan(bench.quantile([], 0.5))


def test_expert_gemm_flops_sum_to_the_model_flops():
    """The six expert GEMMs' FLOPs per step add up to the model-FLOP count the
    headline metric divides by (18 d n per routed row), written separately in
    the workload module."""
    for name in ("tiny", "1b", "7b", "sparse", "coarse"):
        cfg = W.CONFIGS[name]
        P, T = cfg.T * cfg.K - 123, cfg.T
        work = bench.gemm_work(cfg, P, T)
        total = sum(work[c][0] for c in ("up_proj", "down_proj", "dH", "dW2", "dXtilde", "dW1"))
        assert total == pytest.approx(cfg.model_flops(P), rel=1e-12)
        # the bound kernel_work reports is the slower of the two at peak
        for cls, (f, b) in work.items():
            amount, unit, bound = bench.kernel_work(cls, cfg, P, T)
            assert (amount, unit) == ((b, "GB/s") if bound == "hbm" else (f, "TFLOP/s"))
            assert (bound == "hbm") == (b / 8e12 > f / 2.5e15)


def test_operand_bytes_are_the_tensor_sizes():
    """Algorithmic bytes and the bound of the forward GEMMs and the
    aggregation, against the sizes of the seeded tensors themselves (tiny
    layer, P routed rows)."""
    cfg = W.CONFIGS["tiny"]
    inp = W.make_inputs(cfg, 0)
    T, P, n, d = cfg.T, cfg.T * cfg.K, cfg.n, cfg.d
    bf16 = 2
    X, W1, W2 = inp.f32("X"), inp.f32("W1"), inp.f32("W2")
    expect = {
        # X and W1 in; H [P, 2n] and A [P, n] out
        "up_proj": (2.0 * P * d * 2 * n, (X.size + W1.size + P * 2 * n + P * n) * bf16),
        # A and W2 in; Y [P, d] out
        "down_proj": (2.0 * P * n * d, (P * n + W2.size + P * d) * bf16),
    }
    for cls, (flops, nbytes) in expect.items():
        hbm = nbytes / (bench.PEAK_HBM_GBS * 1e9) > flops / (bench.PEAK_BF16_TFLOPS * 1e12)
        want = (nbytes, "GB/s", "hbm") if hbm else (flops, "TFLOP/s", "mfma")
        assert bench.kernel_work(cls, cfg, P, T) == want, cls
    # Y rows and (row, weight) pairs in; O out
    assert bench.kernel_work("aggregate_O", cfg, P, T) == (P * d * bf16 + P * 8 + T * d * bf16, "GB/s", "hbm")
    assert bench.kernel_work("no-such-class", cfg, P, T) == (None, None, None)


def _write_counters(path, rows):
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "run_counter_collection.csv"), "w", newline="") as fh:
        w = csv.DictWriter(fh, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        w.writeheader()
        for r in rows:
            w.writerow(dict(zip(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"], r)))


def test_traffic_report_sizes_requests_and_averages_dispatches(tmp_path):
    gemm = "void smoe::grouped_gemm_kernel<OpDXt<GemmCfg<256, 256, 4, 2, 2, 64, 1> > >(...)"
    copy = "__amd_rocclr_copyBuffer"
    # two dispatches of the GEMM: per dispatch 10 x 32 B + 20 x 64 B + 30 x 128 B read, then 40 x 128 B
    _write_counters(tmp_path / "rd", [
        (1, gemm, "TCC_EA0_RDREQ", 60), (1, gemm, "TCC_EA0_RDREQ_32B", 10), (1, gemm, "TCC_EA0_RDREQ_64B", 20),
        (1, gemm, "TCC_EA0_RDREQ_128B", 30),
        (2, gemm, "TCC_EA0_RDREQ", 40), (2, gemm, "TCC_EA0_RDREQ_32B", 0), (2, gemm, "TCC_EA0_RDREQ_64B", 0),
        (2, gemm, "TCC_EA0_RDREQ_128B", 40),
    ])
    # writes: 8 requests of which 6 are 64-byte, per dispatch
    _write_counters(tmp_path / "wr", [
        (1, gemm, "TCC_EA0_WRREQ", 8), (1, gemm, "TCC_EA0_WRREQ_64B", 6),
        (2, gemm, "TCC_EA0_WRREQ", 8), (2, gemm, "TCC_EA0_WRREQ_64B", 6),
    ])
    _write_counters(tmp_path / "crd", [(7, copy, "TCC_EA0_RDREQ", 8), (7, copy, "TCC_EA0_RDREQ_128B", 8)])
    _write_counters(tmp_path / "cwr", [(7, copy, "TCC_EA0_WRREQ", 16), (7, copy, "TCC_EA0_WRREQ_64B", 16)])
    rep = bench.traffic_report(str(tmp_path / "rd"), str(tmp_path / "wr"), str(tmp_path / "crd"),
                               str(tmp_path / "cwr"), 1024)
    read = ((10 * 32 + 20 * 64 + 30 * 128) + (40 * 128)) / 2
    write = 6 * 64 + 2 * 32
    assert f"| dXtilde | {read:.0f} | {write:.0f} | {read + write:.0f} |" in rep
    assert "reads 1024 and writes 1024 bytes" in rep
    assert f"kernel sources sha256: {bench.kernel_source_hash()}" in rep
    # with a kernel summary: mean launch time of the class and bytes per second
    stats = tmp_path / "kernel_stats.csv"
    with open(stats, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs"])
        w.writerow([gemm, 4, 2000, 500, 100.0, 400, 600])
    rep = bench.traffic_report(str(tmp_path / "rd"), str(tmp_path / "wr"), str(tmp_path / "crd"),
                               str(tmp_path / "cwr"), 1024, str(stats))
    total = read + write
    assert f"| dXtilde | {read:.0f} | {write:.0f} | {total:.0f} | 0.5 | {total / 500e-9 / 1e9:.0f} |" in rep


def test_stats_report_orders_by_total_time(tmp_path):
    p = tmp_path / "kernel_stats.csv"
    with open(p, "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs", "MaxNs"])
        w.writerow(["small_kernel(int)", 10, 1000, 100, 10.0, 90, 110])
        w.writerow(["smoe::big_kernel(float const*)", 2, 9000, 4500, 90.0, 4400, 4600])
    out = bench.stats_report(str(p), "T", "cmd")
    rows = [l for l in out.splitlines() if l.startswith("| `")]
    assert rows[0] == "| `big_kernel(float const*)` | 2 | 4.50 | 4.40 | 4.60 | 90.00 |"
    assert rows[1] == "| `small_kernel(int)` | 10 | 0.10 | 0.09 | 0.11 | 10.00 |"


def test_measured_traffic_only_for_the_profiled_sources(tmp_path, monkeypatch):
    prof = tmp_path / "traffic.md"
    table = "| kernel class | read bytes/launch | write bytes/launch | total bytes/launch |\n|---|---|---|---|\n" \
            "| dXtilde | 100 | 20 | 120 |\n"
    prof.write_text(table + f"\nkernel sources sha256: {bench.kernel_source_hash()}\n")
    monkeypatch.setattr(bench, "TRAFFIC_PROFILE", str(prof))
    assert bench.measured_traffic("dXtilde") == 120.0
    assert bench.measured_traffic("up_proj") is None
    prof.write_text(table + "\nkernel sources sha256: " + "0" * 64 + "\n")
    assert bench.measured_traffic("dXtilde") is None


def test_source_hash_ignores_comments_only(tmp_path, monkeypatch):
    """A comment edit keeps a profile of unchanged kernels valid; a code edit
    (or a new source file) invalidates it."""
    src = tmp_path / "paper_2512_14080_amd" / "csrc"
    src.mkdir(parents=True)
    (src / "k.hip").write_text("int a = 1; // note\n/* block\n comment */ int   b=2;\n")
    (src / "notes.txt").write_text("not a source")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h0 = bench.kernel_source_hash()
    (src / "k.hip").write_text("int a = 1;\n// another note\nint b=2;   /* x */\n")
    assert bench.kernel_source_hash() == h0
    (src / "notes.txt").write_text("changed, still not a source")
    assert bench.kernel_source_hash() == h0
    (src / "k.hip").write_text("int a = 1; int b=3;\n")
    assert bench.kernel_source_hash() != h0
    (src / "k.hip").write_text("int a = 1; int b=2;\n")
    assert bench.kernel_source_hash() == h0
    (src / "extra.h").write_text("int c;\n")
    assert bench.kernel_source_hash() != h0


def test_more_than_one_gpu_is_refused_before_any_device_use():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU only" in r.stderr
    assert r.stdout == ""


def test_mfma_report_from_counters(tmp_path):
    """The MFMA report's arithmetic on a synthetic counter CSV: FLOPs from MOPs,
    the rate over the dispatch timestamps, the clock per XCD and the busy share
    of SIMD cycles, averaged over the dispatches of a class."""
    run = tmp_path / "pmc"
    run.mkdir()
    gemm = "void smoe::grouped_gemm_kernel<OpUp<GemmCfg<256, 256, 4, 2, 2, 64, 1> > >(...)"
    agg = "void smoe::agg_o_kernel<3, false>(...)"
    fields = ["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value", "Start_Timestamp", "End_Timestamp"]
    rows = []
    # two up-proj dispatches of 400 us at 2.0 GHz per XCD, 1e9 MOPs (512 GFLOP), pipe busy 25% of SIMD cycles
    for did, t0 in ((1, 1_000_000), (2, 5_000_000)):
        t1 = t0 + 400_000
        cyc = 2.0e9 * 400e-6
        for name, val in (("GRBM_GUI_ACTIVE", 8 * cyc), ("SQ_INSTS_VALU_MFMA_MOPS_BF16", 1e9),
                          ("SQ_VALU_MFMA_BUSY_CYCLES", 0.25 * cyc * 1024), ("SQ_BUSY_CYCLES", 4 * cyc)):
            rows.append((did, gemm, name, val, t0, t1))
    rows.append((3, agg, "SQ_INSTS_VALU_MFMA_MOPS_BF16", 0, 9_000_000, 9_100_000))
    with open(run / "run_counter_collection.csv", "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(fields)
        w.writerows(rows)
    rep = bench.mfma_report(str(run))
    rate = 512e9 / 400e-6 / 1e12
    assert f"| up_proj | 2 | 512.0 | 400.0 | {rate:.0f} | {100 * rate / 2500:.1f} | 2.00 | 25.0% |" in rep
    assert "aggregate_O" not in rep  # no MFMA work: not a GEMM row
    assert f"kernel sources sha256: {bench.kernel_source_hash()}" in rep
