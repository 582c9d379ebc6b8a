#!/usr/bin/env python3
"""Benchmark: pooled EmbeddingBag forward on one MI355X.

One step = one eb_forward over one batch of the workload (all tables, all
bags).  Other modes: --mode fm, one eb_forward_fm (the lookup, then the FM
cross term over its output); --mode seq, one eb_forward_seq (the un-pooled
lookup); --mode backward, one eb_backward_update with row-wise Adagrad.  Three
independently seeded index batches over the same tables are rotated so
consecutive steps do not replay identical lookups.  Tables, indices and
offsets are resident in HBM before the timed region starts.

Prints one JSON line:
  value            algorithmic GB/s over the K timed steps (wall clock): the
                   bytes the operation must move, duplicates counted, over
                   the time.  Zipf rows repeat within a batch and are served
                   from L2 and the Infinity Cache, so this rate is not an HBM
                   rate and can exceed the HBM peak; the fabric's own rate
                   (rocprofv3 byte counters) and a uniform-index control are
                   reported beside it
  lookups_per_s    pooled lookups per second over the same steps
  roofline         eb_pool_kernel's algorithmic bytes per launch / its mean
                   launch time: the K timed steps between one pair of HIP
                   events on the library's stream, divided by K; against
                   8 TB/s HBM3E; traffic from rocprofv3 counters;
                   p10/median/p90 of single launches (a second pass with an
                   event pair around every 7th launch, which also times the
                   events and the launch's dispatch); and `cold`: calls each
                   preceded (outside their events) by a 1 GiB read that
                   evicts L2 and the Infinity Cache
  uniform_control  the same tables with uniformly drawn indices (no reuse
                   between lookups): the kernel's rate when every row comes
                   from HBM
  cpu_baseline     the CPU oracle on a bounded sample of the same workload

The default workload is c5, the largest that fits one GPU (64 int8 row-wise
tables of 6 M rows: one GPU's share of a table-wise sharded model).

Algorithmic bytes per step = gathered row bytes (every lookup, duplicates
counted) + index bytes + offset bytes + weight bytes + output bytes.
"""
import argparse
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
METRIC = "EmbeddingBag fwd achieved HBM GB/s (% of peak) + pooled lookups/sec, 1 GPU"
METRIC_BACKWARD = ("EmbeddingBag bwd + fused row-wise Adagrad update achieved HBM GB/s (% of peak) + "
                   "lookups/sec, 1 GPU")
METRIC_FM = ("EmbeddingBag fwd + fused FM cross term achieved HBM GB/s (% of peak) + pooled lookups/sec, 1 GPU")
METRIC_SEQ = "Un-pooled (sequence) embedding lookup achieved HBM GB/s (% of peak) + lookups/sec, 1 GPU"
SAMPLE = 7


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_cores() -> int:
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def run_cpu_baseline_seq(w, budget_s: float, host_bytes_cap: float = 3e9, threads: int = 0):
    """Time the oracle's un-pooled lookup (as it stands) on the positions of
    the first tables of `w` whose rows fit in `host_bytes_cap` bytes, repeated
    until `budget_s` seconds have passed.  Returns (reps, seconds, threads,
    lookups per rep, algorithmic bytes per rep, tables used)."""
    import oracle

    if threads <= 0:
        threads = min(cpu_cores(), int(os.environ.get("OMP_NUM_THREADS", cpu_cores())))
    use, acc = 0, 0
    for t in w.tables:
        nbytes = t.rows.numel() * t.rows.element_size()
        if use and acc + nbytes > host_bytes_cap:
            break
        acc += nbytes
        use += 1
    B = w.batch
    off = w.offsets[:use * B + 1].cpu().numpy()
    idx = w.indices[:int(off[-1])].cpu().numpy()
    tabs = [oracle.OracleTable.of(t) for t in w.tables[:use]]
    esz = w.indices.element_size()
    look = int(off[-1])
    nbytes = (use + 1) * esz + sum(int(off[(t + 1) * B] - off[t * B]) * (w.tables[t].row_bytes + esz + 4 * w.tables[t].dim)
                                   for t in range(use))
    reps, t0 = 0, time.perf_counter()
    while True:
        oracle.ebo_forward_seq(tabs, idx, off, num_threads=threads)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    return reps, el, threads, look, nbytes, use


def run_cpu_baseline(w, budget_s: float, host_bytes_cap: float = 3e9, fm: bool = False, threads: int = 0):
    """Time the oracle (as it stands) on the bags of the first tables of `w`
    whose rows fit in `host_bytes_cap` bytes of host memory (all tables for the
    smaller workloads), repeated until `budget_s` seconds have passed.  With
    fm, each pass also runs the oracle's FM cross term over those tables'
    pooled fields.
    Returns (reps, seconds, threads, lookups per rep, algorithmic bytes per rep,
    tables used)."""
    import numpy as np

    import oracle

    if threads <= 0:
        threads = min(cpu_cores(), int(os.environ.get("OMP_NUM_THREADS", cpu_cores())))
    use, acc = 0, 0
    for t in w.tables:
        nbytes = t.rows.numel() * t.rows.element_size()
        if use and acc + nbytes > host_bytes_cap:
            break
        acc += nbytes
        use += 1
    tabs = [oracle.OracleTable.of(t, with_rows=i < use) for i, t in enumerate(w.tables)]
    idx = w.indices.cpu().numpy()
    off = w.offsets.cpu().numpy()
    wt = None if w.weights is None else w.weights.cpu().numpy()
    B = w.batch
    bags = None if use == w.num_tables else np.arange(use * B, dtype=np.int64)
    lens = w.lengths.view(w.num_tables, B).sum(dim=1).cpu().tolist()
    look = int(sum(lens[:use]))
    esz = w.indices.element_size()
    nbytes = sum(int(lens[t]) * w.tables[t].row_bytes + B * w.tables[t].dim * 4 for t in range(use))
    nbytes += look * (esz + (4 if wt is not None else 0)) + (use * B + 1) * esz
    if fm:
        nbytes += 4 * B
    D = w.tables[0].dim
    reps, t0 = 0, time.perf_counter()
    while True:
        out = oracle.ebo_forward(tabs, idx, off, wt, w.pooling, bags=bags, num_threads=threads)
        if fm:
            if bags is not None:  # bag k = (table k // B, example k % B): fields side by side per example
                out = out[:, :D].reshape(use, B, D).transpose(1, 0, 2).reshape(B, use * D)
            oracle.ebo_fm(out, use, D, num_threads=threads)
        reps += 1
        el = time.perf_counter() - t0
        if el >= budget_s:
            break
    return reps, el, threads, look, nbytes, use


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="c5", help="workload: c1 c2 c3a c3b c4 c5")
    ap.add_argument("--index-law", default="zipf", choices=["zipf", "uniform"],
                    help="uniform = no-reuse control at the same shapes")
    ap.add_argument("--cpu-budget", type=float, default=10.0, help="seconds of oracle timing (0 = skip)")
    ap.add_argument("--cold-reps", type=int, default=15,
                    help="after the timed loop, time this many calls each preceded (outside the events) by a "
                         "1 GiB read that evicts L2 and the Infinity Cache (0 = skip)")
    ap.add_argument("--int8-layout", default=None, choices=["packed", "split"],
                    help="layout of int8 row-wise tables (default: the workload's)")
    ap.add_argument("--uniform-steps", type=int, default=-1,
                    help="forward mode with Zipf indices: time this many steps over the same tables with uniform "
                         "indices (the no-reuse control; -1: min(steps, 20); 0 = skip)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a 1 GiB device copy (to scale rocprofv3 byte counters)")
    ap.add_argument("--mode", default="forward", choices=["forward", "fm", "seq", "backward"],
                    help="fm: eb_forward_fm (the lookup, then the FM cross term); seq: eb_forward_seq "
                         "(un-pooled lookup); backward: eb_backward_update with row-wise Adagrad")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py: measures one GPU only; --gpus {args.gpus} is not supported "
              "(the pooled lookup on one GPU is the per-GPU share of a table-wise sharded job)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_30656_amd import eb
    from paper_2609_30656_amd.profiling import KERNELS, counter_traffic
    from paper_2609_30656_amd.workload import CONFIGS, make_workload

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    lib = eb.load_library()
    law = None if args.index_law == "zipf" else "uniform"
    # the workload's name in profile summaries: the config, plus the int8
    # layout when it is not the config's own
    cfg_key = args.config if args.int8_layout in (None, CONFIGS[args.config].int8_layout) else \
        f"{args.config}-{args.int8_layout}"

    print(f"[bench] generating {args.config} ({CONFIGS[args.config].summary})", file=sys.stderr, flush=True)
    batches = [make_workload(args.config, dev, batch_seed=0, index_law=law, int8_layout=args.int8_layout)]
    for s in (1, 2):
        batches.append(make_workload(args.config, dev, batch_seed=s, index_law=law, tables=batches[0].tables))
    w0 = batches[0]
    if args.mode == "seq":
        # every position's row; sized for the largest of the three batches
        out = torch.empty(max(b.seq_output_numel() for b in batches), dtype=torch.float32, device=dev)
    else:
        out = torch.empty((w0.batch, w0.sum_dim), dtype=torch.float32, device=dev)
    if args.mode == "forward":
        algo = [b.algorithmic_bytes() for b in batches]
    elif args.mode == "fm":
        algo = [b.algorithmic_bytes() + 4 * b.batch for b in batches]
    elif args.mode == "seq":
        algo = [b.seq_algorithmic_bytes() for b in batches]
    else:
        algo = [b.backward_algorithmic_bytes() for b in batches]
    nlook = [b.num_indices for b in batches]
    # the lookup's long-bag pass runs for batches of at least 2^23 lookups or
    # of 64 lookups per bag on average, unless EB_LONG_BAG says otherwise
    # (its launch is part of every timed step then, whether or not a bag is
    # long)
    lb = os.environ.get("EB_LONG_BAG")
    m = re.match(r"\s*([+-]?\d+)", lb or "")
    lb_val = int(m.group(1)) if m else 0  # read as the library reads it
    long_len = 1024 if lb is None or lb_val < 0 else lb_val
    long_pass = long_len > 0 and (lb is not None or min(nlook) >= 1 << 23 or
                                  min(n / b.num_bags for n, b in zip(nlook, batches)) >= 64)
    also_in_step = []
    if long_pass and args.mode in ("forward", "fm"):
        longest = max(int(b.lengths.max()) for b in batches)
        also_in_step = [f"eb_long_pass_kernel ({'pools the bags of more than %d lookups' % long_len if longest > long_len else 'no bag is longer than %d lookups: it finds its queue empty' % long_len})"]
    torch.cuda.synchronize()

    stream = torch.cuda.Stream(device=dev)  # default priority
    h = eb.eb_create_tables(w0.tables, stream)
    # marshal once; the loop only calls into the library
    calls = [(eb._as_tensor(b.indices), eb._as_tensor(b.offsets), eb._as_tensor(b.weights),
              eb.POOLING[b.pooling]) for b in batches]
    o = eb._as_tensor(out)

    def forward_step(k):
        i, f, wt, mode = calls[k % 3]
        st = lib.eb_forward(h.ptr, i, f, wt, mode, o)
        if st != eb.EB_OK:
            raise eb.EBError(st, "eb_forward")

    if args.mode == "forward":
        step = forward_step
    elif args.mode == "seq":
        seq_outs = [eb._as_tensor(out[:b.seq_output_numel()]) for b in batches]

        def step(k):
            i, f, _, _ = calls[k % 3]
            st = lib.eb_forward_seq(h.ptr, i, f, seq_outs[k % 3])
            if st != eb.EB_OK:
                raise eb.EBError(st, "eb_forward_seq")
    elif args.mode == "fm":
        fm_out = torch.empty(w0.batch, dtype=torch.float32, device=dev)
        fm_t = eb._as_tensor(fm_out)

        def step(k):
            i, f, wt, mode = calls[k % 3]
            st = lib.eb_forward_fm(h.ptr, i, f, wt, mode, o, fm_t)
            if st != eb.EB_OK:
                raise eb.EBError(st, "eb_forward_fm")
    else:
        gen = torch.Generator(device=dev)
        gen.manual_seed(5)
        grad = torch.randn((w0.batch, w0.sum_dim), generator=gen, device=dev, dtype=torch.float32)
        state = torch.zeros(sum(t.num_rows for t in w0.tables), dtype=torch.float32, device=dev)
        ws_bytes = max(eb.eb_backward_workspace_size(h, b.num_indices) for b in batches)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
        g_t, s_t = eb._as_tensor(grad), eb._as_tensor(state)

        def step(k):
            i, f, wt, mode = calls[k % 3]
            st = lib.eb_backward_update(h.ptr, i, f, wt, mode, g_t, eb.EB_OPT_ROWWISE_ADAGRAD, 1e-3, 1e-8, s_t,
                                        ws.data_ptr(), ws_bytes)
            if st != eb.EB_OK:
                raise eb.EBError(st, "eb_backward_update")

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()

    # The timed loop: K back-to-back steps between one pair of HIP events on
    # the library's stream (so the kernels' GPU time per step, with no event
    # packets between them) and the host clock (`value`).
    def timed_region(fn):
        r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        r0.record(stream)
        for k in range(args.steps):
            fn(k)
        r1.record(stream)
        torch.cuda.synchronize()
        return time.perf_counter() - t0, r0.elapsed_time(r1) / 1e3

    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    wall, region_s = timed_region(step)
    kern_avg_s = region_s / args.steps
    kern_bytes = sum(algo[k % 3] for k in range(args.steps)) / args.steps

    # Then the spread of single launches: a second pass with an event pair
    # around every SAMPLE-th step (7 is coprime with the 3 rotating batches,
    # so all three are sampled).  Each such pair also times its own event
    # packets and the launch's dispatch, so these read a little longer than
    # the steady-state average above.
    sample = [k for k in range(args.steps) if k % SAMPLE == 0]
    starts = {k: torch.cuda.Event(enable_timing=True) for k in sample}
    ends = {k: torch.cuda.Event(enable_timing=True) for k in sample}
    for k in range(args.steps):
        if k in starts:
            starts[k].record(stream)
            step(k)
            ends[k].record(stream)
        else:
            step(k)
    torch.cuda.synchronize()
    kern_ms = [starts[k].elapsed_time(ends[k]) for k in sample]

    def quantiles(xs):
        xs = sorted(xs)
        pick = lambda f: xs[min(len(xs) - 1, int(f * (len(xs) - 1) + 0.5))]
        return pick(0.1), pick(0.5), pick(0.9)

    cold = None
    if args.cold_reps > 0:
        # every call starts with nothing of its inputs in L2 or the Infinity
        # Cache: a 1 GiB read on the same stream, outside the events, first (a
        # read, so no dirty lines are still being written back when it starts)
        print(f"[bench] {args.cold_reps} cold calls", file=sys.stderr, flush=True)
        scratch = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        sink = torch.empty((), dtype=torch.float32, device=dev)
        torch.cuda.synchronize()
        cold_ms, cold_bytes = [], 0
        for k in range(args.cold_reps):
            with torch.cuda.stream(stream):
                torch.sum(scratch, dim=0, out=sink)
            a_ev, b_ev = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a_ev.record(stream)
            step(k)
            b_ev.record(stream)
            b_ev.synchronize()
            cold_ms.append(a_ev.elapsed_time(b_ev))
            cold_bytes += algo[k % 3]
        del scratch, sink
        c10, c50, c90 = quantiles(cold_ms)
        cold = {"reps": args.cold_reps, "kernel_ms_p10": round(c10, 5), "kernel_ms_median": round(c50, 5),
                "kernel_ms_p90": round(c90, 5),
                "achieved": round(cold_bytes / args.cold_reps / (c50 * 1e-3) / 1e9, 2)}
    w10, w50, w90 = quantiles(kern_ms)

    uniform = None
    n_uni = min(args.steps, 20) if args.uniform_steps < 0 else args.uniform_steps
    if args.mode == "forward" and args.index_law == "zipf" and n_uni > 0:
        # the no-reuse control: one batch of the same shape over the same
        # tables with uniformly drawn rows, timed like the main loop
        print(f"[bench] uniform-index control, {n_uni} steps", file=sys.stderr, flush=True)
        wu = make_workload(args.config, dev, batch_seed=0, index_law="uniform", tables=w0.tables)
        cu = (eb._as_tensor(wu.indices), eb._as_tensor(wu.offsets), eb._as_tensor(wu.weights),
              eb.POOLING[wu.pooling])

        def uniform_step(k):
            st = lib.eb_forward(h.ptr, *cu[:3], cu[3], o)
            if st != eb.EB_OK:
                raise eb.EBError(st, "eb_forward")

        for k in range(min(3, n_uni)):
            uniform_step(k)
        r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        r0.record(stream)
        for k in range(n_uni):
            uniform_step(k)
        r1.record(stream)
        torch.cuda.synchronize()
        u_ms = r0.elapsed_time(r1) / n_uni
        u_bytes = wu.algorithmic_bytes()
        u_traffic = counter_traffic(cfg_key, "uniform", "forward")
        uniform = {"index_law": "uniform", "steps": n_uni, "kernel_ms_avg": round(u_ms, 5),
                   "lookups": wu.num_indices, "algorithmic_bytes": u_bytes,
                   "achieved": round(u_bytes / (u_ms * 1e-3) / 1e9, 2),
                   "frac": round(u_bytes / (u_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4),
                   "lookups_per_s": round(wu.num_indices / (u_ms * 1e-3), 1),
                   "traffic": None if u_traffic is None else round(u_traffic),
                   "traffic_frac": None if u_traffic is None else
                   round(u_traffic / (u_ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}
        del wu, cu

    bytes_total = sum(algo[k % 3] for k in range(args.steps))
    look_total = sum(nlook[k % 3] for k in range(args.steps))
    value = bytes_total / wall / 1e9
    achieved = kern_bytes / kern_avg_s / 1e9
    traffic = counter_traffic(cfg_key, args.index_law, args.mode) if args.mode in ("forward", "seq") else None

    fm_pass = None
    if args.mode == "fm":
        # the plain lookup on the same batches, timed the same way: the step's
        # extra time is the FM pass over the pooled output
        for k in range(args.warmup):
            forward_step(k)
        _, fwd_region_s = timed_region(forward_step)
        fwd_ms = fwd_region_s / args.steps * 1e3
        pass_bytes = w0.batch * w0.sum_dim * 4 + w0.batch * 4
        pass_ms = kern_avg_s * 1e3 - fwd_ms
        fm_pass = {
            "step_kernels_ms": round(kern_avg_s * 1e3, 5),
            "forward_only_ms": round(fwd_ms, 5),
            "pass_ms_by_difference": round(pass_ms, 5),
            "pass_bytes": pass_bytes,
            "pass_GBps": round(pass_bytes / (pass_ms * 1e-3) / 1e9, 1) if pass_ms > 0 else None,
        }

    if args.copy_calibration:
        n = 1 << 28  # 1 GiB of fp32
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    eb.eb_destroy(h)

    cpu = None
    if args.cpu_budget > 0 and args.mode in ("forward", "fm", "seq"):
        print(f"[bench] CPU oracle baseline ({args.cpu_budget:.0f} s budget)", file=sys.stderr, flush=True)
        fm = args.mode == "fm"
        if args.mode == "seq":
            reps, el, threads, look, nbytes, use = run_cpu_baseline_seq(w0, args.cpu_budget)
        else:
            reps, el, threads, look, nbytes, use = run_cpu_baseline(w0, args.cpu_budget, fm=fm)
        what = "the whole batch" if use == w0.num_tables else f"the bags of tables 0..{use - 1} of {w0.num_tables}"
        if fm:
            what += " plus the FM cross term over those fields"
        cpu = {
            "value": round(nbytes * reps / el / 1e9, 4),
            "unit": "GB/s",
            "lookups_per_s": round(look * reps / el, 1),
            "cores": threads,
            "kind": "oracle",
            "sample": f"{reps} pass(es) of the oracle over {what} of batch 0 of {args.config} "
                      f"({look} lookups per pass) on the host, {el:.1f} s",
            "cpu_model": cpu_model(),
        }
        if threads > 1:
            # the same sample on one thread, for a fifth of the budget (at least one pass)
            b1 = args.cpu_budget / 5
            if args.mode == "seq":
                r1, e1, _, look1, nb1, _ = run_cpu_baseline_seq(w0, b1, threads=1)
            else:
                r1, e1, _, look1, nb1, _ = run_cpu_baseline(w0, b1, fm=fm, threads=1)
            cpu["one_thread"] = {"value": round(nb1 * r1 / e1 / 1e9, 4), "unit": "GB/s",
                                 "lookups_per_s": round(look1 * r1 / e1, 1), "seconds": round(e1, 1)}

    dtypes = sorted({t.dtype for t in w0.tables})
    # what the path computes in: the stored values (u8 codes with fp16 scale
    # and bias, fp16 or fp32) widened or dequantised to fp32, summed in fp32
    path_dtype = "+".join(sorted({{"f32": "f32", "f16": "f16->f32"}.get(d, "u8->f32") for d in dtypes}))
    fabric_gbs = None if traffic is None else traffic / kern_avg_s / 1e9
    line = {
        "metric": {"forward": METRIC, "fm": METRIC_FM, "seq": METRIC_SEQ, "backward": METRIC_BACKWARD}[args.mode],
        "value": round(value, 2),
        "unit": "GB/s",
        "value_basis": "algorithmic bytes (rows gathered with duplicates counted, indices, offsets, weights, "
                       "outputs) / wall time of the timed steps; not an HBM rate when rows repeat",
        "algorithmic_pct_of_peak": round(100.0 * value / PEAK_HBM_GBS, 2),
        "fabric_pct_of_peak": None if fabric_gbs is None else round(100.0 * fabric_gbs / PEAK_HBM_GBS, 2),
        "lookups_per_s": round(look_total / wall, 1),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": path_dtype,
        "accumulate": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{args.config}: {CONFIGS[args.config].summary}",
            "index_law": args.index_law,
            "tables": w0.num_tables,
            "batch": w0.batch,
            "bags": w0.num_bags,
            "lookups_per_step": round(sum(nlook) / 3),
            "algorithmic_bytes_per_step": round(sum(algo) / 3),
            "index_dtype": str(w0.indices.dtype).replace("torch.", ""),
            "table_storage": dtypes,
            "int8_layout": ({"int8_rowwise": "packed (codes, scale, bias in each row)",
                             "int8_rowwise_split": "split (codes in the rows, scale/bias block after them)"}
                            .get(dtypes[0]) if len(dtypes) == 1 else None),
            "row_stride_bytes": sorted({t.row_stride_bytes for t in w0.tables}),
        },
        "mode": args.mode,
        "roofline": {
            "bound": "hbm",
            "kernel": {"forward": KERNELS["forward"][0], "fm": "eb_forward_fm (eb_pool_kernel, then eb_fm_kernel)",
                       "seq": KERNELS["seq"][0], "backward": "eb_backward_update (all its kernels)"}[args.mode],
            "achieved": round(achieved, 2),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4),
            "traffic": None if traffic is None else round(traffic),
            # the counter traffic per launch over the mean launch time: the
            # fabric's actual rate, which Zipf reuse in L2 keeps below the
            # algorithmic one
            "traffic_gbs": None if traffic is None else round(traffic / kern_avg_s / 1e9, 1),
            "traffic_frac": None if traffic is None else round(traffic / kern_avg_s / 1e9 / PEAK_HBM_GBS, 4),
            "kernel_ms_avg": round(kern_avg_s * 1e3, 5),
            # what one timed step enqueues besides the named kernel
            "also_in_step": also_in_step,
            "timed_launches": args.steps,
            "kernel_ms_p10": round(w10, 5),
            "kernel_ms_median": round(w50, 5),
            "kernel_ms_p90": round(w90, 5),
            "sampled_launches": len(sample),
            "cold": cold,
        },
        "uniform_control": uniform,
        "cpu_baseline": cpu,
    }
    if fm_pass is not None:
        line["fm_pass"] = fm_pass
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
