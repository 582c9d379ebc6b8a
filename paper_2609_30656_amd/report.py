"""Per-component report of the embedding path, in the columns of the paper's
result table (Sec. IV-A.1): component, latency, model size, TFLOP/s, MFU and
estimated average bandwidth with its utilisation.

    python -m paper_2609_30656_amd.report [--configs c2 c3a ...] [--json out.json]

Each component is one call of this library on a seeded workload, timed with
HIP events on its stream (median of --reps calls after --warmup calls):

  sparse_arch.lookup      eb_forward: the pooled lookup
  sparse_arch.lookup_seq  eb_forward_seq: the un-pooled (sequence) lookup
  inter_arch.fm           eb_fm_cross: the FM cross term over the pooled output
                          (workloads whose tables share one width)
  sparse_arch.backward    eb_backward_update with row-wise Adagrad
                          (workloads whose tables can train: fp32/fp16, D <= 256)

Bandwidth is the algorithmic bytes of the call (what it must read and write
at least, every lookup counted) over its latency, against 8 TB/s of HBM3E;
MFU is its algorithmic fp32 operations per second against the 157.3 TFLOP/s
vector fp32 peak (there is no matrix work on this path).
"""
from __future__ import annotations

import argparse
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_GBS = 8000.0
PEAK_FP32_TFLOPS = 157.3


def _flops_per_element(tb, weighted):
    if tb.dtype.startswith("int8_rowwise"):
        return 4 if weighted else 2  # dequantising fma (+ the weight's fma)
    return 2 if weighted else 1


def lookup_flops(w):
    off = w.offsets.cpu()
    B = w.batch
    total = 0
    for t, tb in enumerate(w.tables):
        n = int(off[(t + 1) * B] - off[t * B])
        total += n * tb.dim * _flops_per_element(tb, w.weights is not None)
        if w.pooling == "mean":
            total += B * tb.dim
    return total


def seq_flops(w):
    off = w.offsets.cpu()
    B = w.batch
    return sum(int(off[(t + 1) * B] - off[t * B]) * tb.dim * 2
               for t, tb in enumerate(w.tables) if tb.dtype.startswith("int8_rowwise"))


def fm_bytes_flops(w):
    T, D, B = w.num_tables, w.tables[0].dim, w.batch
    return B * T * D * 4 + 4 * B, B * (3 * T * D + 2 * D)


def backward_flops(w):
    """c_i * g into the row's sum (an fma per element and lookup), then the
    row-wise Adagrad step per touched row (squares, sum, scale: ~4 per element)."""
    import torch

    off = w.offsets.cpu()
    B = w.batch
    total = 0
    for t, tb in enumerate(w.tables):
        lo, hi = int(off[t * B]), int(off[(t + 1) * B])
        u = int(torch.unique(w.indices[lo:hi]).numel()) if hi > lo else 0
        total += (hi - lo) * tb.dim * 2 + u * tb.dim * 4
    return total


def _time(fn, stream, warmup, reps):
    import torch

    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ms = []
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        fn()
        b.record(stream)
        b.synchronize()
        ms.append(a.elapsed_time(b))
    ms.sort()
    return ms[len(ms) // 2]


def report(configs, warmup=5, reps=21, log=print):
    import torch

    from paper_2609_30656_amd import eb
    from paper_2609_30656_amd.workload import make_workload

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    lib = eb.load_library()
    rows = []
    for cfg in configs:
        log(f"[report] {cfg}: generating")
        w = make_workload(cfg, dev)
        table_mb = sum(t.rows.numel() * t.rows.element_size() for t in w.tables) / 2**20
        stream = torch.cuda.Stream(device=dev)
        h = eb.eb_create_tables(w.tables, stream)
        I, O, Wt = eb._as_tensor(w.indices), eb._as_tensor(w.offsets), eb._as_tensor(w.weights)
        mode = eb.POOLING[w.pooling]
        out = torch.empty((w.batch, w.sum_dim), dtype=torch.float32, device=dev)
        o = eb._as_tensor(out)

        def add(name, ms, nbytes, flops, model_mb):
            tfl = flops / (ms * 1e-3) / 1e12
            gbs = nbytes / (ms * 1e-3) / 1e9
            rows.append({"component": name, "workload": cfg, "latency_ms": round(ms, 5), "model_size_mb": round(model_mb, 1),
                         "tflops": round(tfl, 3), "mfu_pct": round(100 * tfl / PEAK_FP32_TFLOPS, 3),
                         "est_avg_bw_gbs": round(gbs, 1), "bw_util_pct": round(100 * gbs / PEAK_GBS, 1),
                         "algorithmic_bytes": int(nbytes), "flops": int(flops)})
            log(f"[report] {cfg} {name}: {ms:.4f} ms, {gbs:.0f} GB/s")

        def check(st, what):
            if st != eb.EB_OK:
                raise eb.EBError(st, what)

        ms = _time(lambda: check(lib.eb_forward(h.ptr, I, O, Wt, mode, o), "eb_forward"), stream, warmup, reps)
        add("sparse_arch.lookup", ms, w.algorithmic_bytes(), lookup_flops(w), table_mb)

        seq_out = torch.empty(w.seq_output_numel(), dtype=torch.float32, device=dev)
        so = eb._as_tensor(seq_out)
        ms = _time(lambda: check(lib.eb_forward_seq(h.ptr, I, O, so), "eb_forward_seq"), stream, warmup, reps)
        add("sparse_arch.lookup_seq", ms, w.seq_algorithmic_bytes(), seq_flops(w), table_mb)
        del seq_out

        if len({t.dim for t in w.tables}) == 1:
            fm = torch.empty(w.batch, dtype=torch.float32, device=dev)
            fo = eb._as_tensor(fm)
            ms = _time(lambda: check(lib.eb_fm_cross(h.ptr, o, fo), "eb_fm_cross"), stream, warmup, reps)
            nb, fl = fm_bytes_flops(w)
            add("inter_arch.fm", ms, nb, fl, 0.0)

        if all(t.dtype in ("f32", "f16") and t.dim <= 256 for t in w.tables):
            gen = torch.Generator(device=dev)
            gen.manual_seed(5)
            grad = torch.randn((w.batch, w.sum_dim), generator=gen, device=dev)
            state = torch.zeros(sum(t.num_rows for t in w.tables), dtype=torch.float32, device=dev)
            ws = torch.empty(max(eb.eb_backward_workspace_size(h, w.num_indices), 1), dtype=torch.uint8, device=dev)
            g_t, s_t = eb._as_tensor(grad), eb._as_tensor(state)
            ms = _time(lambda: check(lib.eb_backward_update(h.ptr, I, O, Wt, mode, g_t, eb.EB_OPT_ROWWISE_ADAGRAD, 1e-3,
                                                            1e-8, s_t, ws.data_ptr(), ws.numel()), "eb_backward_update"),
                       stream, warmup, reps)
            add("sparse_arch.backward", ms, w.backward_algorithmic_bytes(), backward_flops(w),
                table_mb + state.numel() * 4 / 2**20)
            del grad, state, ws
        eb.eb_destroy(h)
        del h, w, out
        torch.cuda.empty_cache()
    return rows


def markdown(rows):
    head = ("| Component | Workload | Latency (ms) | Model size (MB) | TFLOP/s | MFU % | Est. avg BW (GB/s) | "
            "BW util % |\n|---|---|---|---|---|---|---|---|")
    lines = [head]
    for r in rows:
        lines.append(f"| {r['component']} | {r['workload']} | {r['latency_ms']:.4f} | {r['model_size_mb']:.0f} | "
                     f"{r['tflops']:.3f} | {r['mfu_pct']:.3f} | {r['est_avg_bw_gbs']:.0f} | {r['bw_util_pct']:.1f} |")
    return "\n".join(lines)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--configs", nargs="+", default=["c2", "c3a", "c3b", "c4", "c5"])
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--reps", type=int, default=21)
    ap.add_argument("--json", default=None, help="also write the rows as JSON to this path")
    args = ap.parse_args(argv)
    rows = report(args.configs, args.warmup, args.reps, log=lambda m: print(m, file=sys.stderr, flush=True))
    print(markdown(rows), flush=True)
    if args.json:
        with open(args.json, "w") as f:
            json.dump(rows, f, indent=1)


if __name__ == "__main__":
    main()
