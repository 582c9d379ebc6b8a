"""rocprofv3 summaries of the benchmark's dominant kernel.

    python -m paper_2609_30656_amd.profiling --mode forward --config c5 [--index-law zipf]

runs, one after another (each under its own time limit):
  1. a kernel trace of `bench.py` (--kernel-trace --stats): per-launch duration;
  2. three counter passes of `bench.py --copy-calibration`, one counter set
     each: FETCH_SIZE, WRITE_SIZE, and TCC_HIT_sum + TCC_MISS_sum.  The three
     1 GiB device-to-device copies at the end of each run (the run's last
     copies) read the same counters, which scales counter KiB to bytes (gfx950
     issues 128-byte read requests that FETCH_SIZE counts as 64 bytes).  The counts are L2<->fabric traffic, so
     Infinity Cache hits are included: an upper bound on HBM traffic;
and writes profiles/<kernel>_<config>_<law>_{kernel_trace,pmc}.txt, each with
the commands that made it and the hash of the kernel's sources, which
bench.py checks before it reports the counter traffic.
"""
from __future__ import annotations

import argparse
import collections
import csv
import hashlib
import json
import os
import re
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
PROFILES = os.path.join(ROOT, "profiles")

# the dominant kernel of each benchmark mode and the sources it is built from
KERNELS = {
    "forward": ("eb_pool_kernel", ("eb_device.h", "eb_forward.hip")),
    "fm": ("eb_fm_kernel", ("eb_device.h", "eb_fm.hip")),
    "seq": ("eb_seq_kernel", ("eb_device.h", "eb_seq.hip")),
    "backward": ("eb_bwd_tiles_kernel", ("eb_device.h", "eb_backward.hip")),
}


def _code_only(text: str) -> str:
    """Source text without comments and blank lines (comment edits leave the
    kernel, and so its counter summary, valid)."""
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    lines = (re.sub(r"//.*", "", ln).rstrip() for ln in text.splitlines())
    return "\n".join(ln for ln in lines if ln.strip())


def kernel_source_hash(mode: str) -> str:
    h = hashlib.sha256()
    for f in KERNELS[mode][1]:
        with open(os.path.join(CSRC, f)) as fh:
            h.update(_code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def summary_path(mode: str, config: str, law: str, kind: str) -> str:
    return os.path.join(PROFILES, f"{KERNELS[mode][0]}_{config}_{law}_{kind}.txt")


def read_summary(path: str) -> dict:
    vals = {}
    with open(path) as f:
        for line in f:
            if "=" in line and not line.startswith("#"):
                k, v = line.split("=", 1)
                vals[k.strip()] = v.split("(")[0].strip()
    return vals


def counter_traffic(config: str, law: str, mode: str):
    """Fabric bytes per launch of the mode's kernel from the committed counter
    summary, if it was taken on the current kernel source; else None."""
    path = summary_path(mode, config, law, "pmc")
    if not os.path.exists(path):
        return None
    vals = read_summary(path)
    if vals.get("kernel_source_sha256_16") != kernel_source_hash(mode):
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _bench_args(mode, config, law, steps, warmup, calib):
    """bench.py's arguments for one profiled run of workload `config` (a
    config name, or config-layout for int8 tables in a layout other than the
    config's own); only the main loop's kernel runs (no uniform control)."""
    cfg, _, layout = config.partition("-")
    a = [sys.executable, os.path.join(ROOT, "bench.py"), "--mode", mode, "--config", cfg, "--index-law", law,
         "--steps", str(steps), "--warmup", str(warmup), "--cpu-budget", "0", "--uniform-steps", "0"]
    if layout:
        a += ["--int8-layout", layout]
    return a + (["--copy-calibration"] if calib else [])


def _run(cmd, log, limit):
    print("[profiling] " + " ".join(cmd), flush=True)
    with open(log, "w") as f:
        r = subprocess.run(["timeout", "-s", "KILL", str(limit), *cmd], stdout=f, stderr=subprocess.STDOUT)
    if r.returncode != 0:
        with open(log) as f:
            sys.stdout.write(f.read()[-3000:])
        raise SystemExit(f"[profiling] step failed with status {r.returncode}")


def read_counters(path, kernel):
    """Counter values of a rocprofv3 --pmc CSV: {counter: [value per launch of
    `kernel`]} and {"copy:" + counter: [value per calibration copy]}.  The
    calibration copies are the process's last CALIBRATION_COPIES device copies
    (workload set-up may copy too: c5 builds its tables by copies)."""
    acc = collections.defaultdict(list)
    copies = collections.defaultdict(list)
    with open(path) as f:
        for r in csv.DictReader(f):
            v = float(r["Counter_Value"])
            if _match(r["Kernel_Name"], kernel):
                acc[r["Counter_Name"]].append(v)
            elif r["Kernel_Name"] == "__amd_rocclr_copyBuffer":
                copies[r["Counter_Name"]].append((int(r["Dispatch_Id"]), v))
    for name, lst in copies.items():
        acc["copy:" + name] = [v for _, v in sorted(lst)[-CALIBRATION_COPIES:]]
    return dict(acc)


def _bench_line(log):
    with open(log) as f:
        for line in f:
            if line.startswith("{") and '"metric"' in line:
                return json.loads(line)
    raise SystemExit(f"[profiling] no bench line in {log}")


CALIBRATION_COPIES = 3  # bench.py --copy-calibration: three copies of 1 GiB, after everything else


def _match(name, kernel):
    return kernel in name


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--mode", default="forward", choices=sorted(KERNELS))
    ap.add_argument("--config", default="c5",
                    help="workload (c1 c2 c3a c3b c4 c5), or c5-packed / c5-split for an int8 layout")
    ap.add_argument("--index-law", default="zipf", choices=["zipf", "uniform"])
    ap.add_argument("--work", default="/tmp/eb_profiling", help="scratch directory for rocprofv3 output")
    ap.add_argument("--limit", type=int, default=300, help="seconds allowed per rocprofv3 run")
    args = ap.parse_args(argv)

    mode, cfg, law = args.mode, args.config, args.index_law
    kernel = KERNELS[mode][0]
    work = os.path.join(args.work, f"{mode}_{cfg}_{law}")
    os.makedirs(work, exist_ok=True)
    src_hash = kernel_source_hash(mode)
    me = f"python -m paper_2609_30656_amd.profiling --mode {mode} --config {cfg} --index-law {law}"

    # 1. kernel trace
    kt_dir = os.path.join(work, "kt")
    kt_cmd = ["rocprofv3", "--kernel-trace", "--stats", "--output-format", "csv", "-d", kt_dir, "-o", "kt", "--",
              *_bench_args(mode, cfg, law, 50, 5, False)]
    _run(kt_cmd, os.path.join(work, "kt.log"), args.limit)
    line = _bench_line(os.path.join(work, "kt.log"))
    # bytes one launch of the kernel must move: the whole step's for the
    # lookup; the pooled output read plus the term written for the FM pass
    algo = float(line["fm_pass"]["pass_bytes"] if mode == "fm" else line["config"]["algorithmic_bytes_per_step"])
    rows = list(csv.DictReader(open(os.path.join(kt_dir, "kt_kernel_stats.csv"))))
    shown = " ".join(kt_cmd[:kt_cmd.index("--")]) + " -- python3 bench.py " + " ".join(
        _bench_args(mode, cfg, law, 50, 5, False)[2:])
    lines = [f"# rocprofv3 kernel-trace summary: {kernel}, workload {cfg} ({law} indices), bench mode {mode}",
             f"# made by: {me}",
             f"# command: {shown}",
             f"kernel_source_sha256_16 = {src_hash}"]
    for r in rows:
        if _match(r["Name"], kernel):
            avg = float(r["AverageNs"])
            lines += [f"kernel = {r['Name']}", f"calls = {r['Calls']}", f"average_ns = {avg:.1f}",
                      f"min_ns = {r['MinNs']}", f"max_ns = {r['MaxNs']}", f"stddev_ns = {float(r['StdDev']):.1f}",
                      f"percent_of_gpu_time = {r['Percentage']}"]
            if mode != "backward":
                lines += [f"algorithmic_bytes_per_launch = {algo:.0f}",
                          f"algorithmic_GBps_at_average = {algo / avg:.1f}"]
    lines.append("# kernels of the profiled process by total time (workload generation included):")
    top = sorted(rows, key=lambda r: -float(r["TotalDurationNs"]))
    for r in top[:8]:
        lines.append(f"#   {r['Calls']:>5} calls  avg {float(r['AverageNs']) / 1e3:10.2f} us  {r['Name'][:100]}")
    rest = [r for r in top[8:] if "eb::" in r["Name"]]
    if rest:
        lines.append("# the library's other kernels in the same process:")
        for r in rest:
            lines.append(f"#   {r['Calls']:>5} calls  avg {float(r['AverageNs']) / 1e3:10.2f} us  {r['Name'][:100]}")
    os.makedirs(PROFILES, exist_ok=True)
    with open(summary_path(mode, cfg, law, "kernel_trace"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines), flush=True)

    # 2. counters, one set per run
    passes = [("FETCH_SIZE",), ("WRITE_SIZE",), ("TCC_HIT_sum", "TCC_MISS_sum")]
    vals, cmds = {}, []
    for counters in passes:
        d = os.path.join(work, "pmc_" + counters[0])
        cmd = ["rocprofv3", "--pmc", *counters, "--output-format", "csv", "-d", d, "-o", "pmc", "--",
               *_bench_args(mode, cfg, law, 10, 2, True)]
        cmds.append(" ".join(cmd[:cmd.index("--")]) + " -- python3 bench.py " +
                    " ".join(_bench_args(mode, cfg, law, 10, 2, True)[2:]))
        _run(cmd, os.path.join(work, f"pmc_{counters[0]}.log"), args.limit)
        acc = read_counters(os.path.join(d, "pmc_counter_collection.csv"), kernel)
        vals.update({k: (sum(v) / len(v), len(v)) for k, v in acc.items()})

    GiB = 1 << 30
    fe, nfe = vals["FETCH_SIZE"]
    we, nwe = vals["WRITE_SIZE"]
    fc, nfc = vals["copy:FETCH_SIZE"]
    wc, nwc = vals["copy:WRITE_SIZE"]
    ff, wf = GiB / (fc * 1024), GiB / (wc * 1024)
    rd, wr = fe * 1024 * ff, we * 1024 * wf
    lines = [f"# rocprofv3 counter summary: {kernel}, workload {cfg} ({law} indices), bench mode {mode}",
             f"# made by: {me}"]
    lines += [f"# pass {i + 1}: {c}" for i, c in enumerate(cmds)]
    lines += ["# Calibration: --copy-calibration copies 1 GiB device-to-device (__amd_rocclr_copyBuffer);",
              "# the same counters read for it scale counter KiB to bytes.  Counts are L2<->fabric traffic,",
              "# so Infinity Cache (MALL) hits are included: an upper bound on HBM traffic.",
              f"kernel_source_sha256_16 = {src_hash}",
              f"fetch_size_kib_per_launch = {fe:.1f}   (mean of {nfe} launches)",
              f"write_size_kib_per_launch = {we:.1f}   (mean of {nwe} launches)",
              f"copy_1GiB_fetch_size_kib = {fc:.1f}   (mean of {nfc})",
              f"copy_1GiB_write_size_kib = {wc:.1f}   (mean of {nwc})",
              f"fetch_scale = {ff:.4f}",
              f"write_scale = {wf:.4f}",
              f"hbm_read_bytes_per_launch = {rd:.0f}",
              f"hbm_write_bytes_per_launch = {wr:.0f}",
              f"hbm_bytes_per_launch = {rd + wr:.0f}"]
    if mode != "backward":
        lines += [f"algorithmic_bytes_per_launch = {algo:.0f}",
                  f"traffic_over_algorithmic = {(rd + wr) / algo:.4f}"]
    if "TCC_HIT_sum" in vals and "TCC_MISS_sum" in vals:
        hit, miss = vals["TCC_HIT_sum"][0], vals["TCC_MISS_sum"][0]
        lines += [f"TCC_HIT_sum_per_launch = {hit:.0f}", f"TCC_MISS_sum_per_launch = {miss:.0f}",
                  f"l2_hit_rate = {hit / (hit + miss):.4f}"]
    with open(summary_path(mode, cfg, law, "pmc"), "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines), flush=True)


if __name__ == "__main__":
    main()
