"""Throughput of the DynSparse forward pass on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload wan720p]

A step is one call of ``dynsparse_attn_fwd`` (recall target 0.95) over a whole
Wan-2.2-14B-like 720p attention layer (B=1, H=40, N=75600 = 21x45x80 latent tokens,
d=128, bf16), with the inputs already resident in HBM.  ``value`` is the effective
(dense-equivalent) throughput 4*B*H*N^2*d / time; the same run times the library's own
``dense_attn_fwd`` for the speedup, reports the kernel's bf16 MFMA roofline fraction on
the work it actually issues, and times the fp64 CPU oracle on a bounded sample of the
same layer as a reference point.  One JSON line is printed.

``--sweep`` instead prints one JSON line per rule/threshold on the given workload;
``--reorder-sweep`` prints, per rule/threshold, the row-major run next to the same run over
the spatio-temporally blocked token order (``dsattn_attn_fwd_reordered``, gathers and the
output scatter included in its time), plus the HBM rate of the row gather kernel;
``--reuse-sweep`` times a DynSparse call that writes its skip mask, then the mask-reuse call
(DSATTN_RULE_MASK) that applies that mask, per threshold and decision unit;
``--q8-sweep`` times the MX-FP8 quantisation of Q and K (and the key mean and shifted
quantisation of key smoothing), then per rule/threshold the bf16 call next to the call with
MX-FP8 Q and K (DSATTN_QK_MXFP8), with plain and with smoothed keys.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "effective TFLOP/s (dense-equiv) + speedup vs own dense FA at matched recall"
PEAK_BF16_TFLOPS = 2500.0    # MI355X dense bf16 MFMA
PEAK_FP8_TFLOPS = 5000.0     # MI355X dense fp8 MFMA
HBM_PEAK_GBS = 8000.0
TILE_Q, TILE_K, D = 128, 64, 128


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="wan720p")
    ap.add_argument("--recall", type=float, default=None, help="recall target (default: workload's)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate CPU budget of the oracle baseline (0 = skip)")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense timing (profiling)")
    ap.add_argument("--sweep", action="store_true", help="one line per rule/threshold")
    ap.add_argument("--reorder-sweep", action="store_true",
                    help="row-major vs blocked token order, one line per rule/threshold")
    ap.add_argument("--reuse-sweep", action="store_true",
                    help="rule call writing its mask, then mask reuse, one line per threshold")
    ap.add_argument("--q8-sweep", action="store_true",
                    help="bf16 vs MX-FP8 Q K^T, one line per rule/threshold")
    ap.add_argument("--q-block", default="2,8,8", help="query block (t,y,x) for --reorder-sweep")
    ap.add_argument("--kv-block", default="1,8,8", help="key/value block for --reorder-sweep")
    ap.add_argument("--calib-copy", action="store_true",
                    help="also run a plain 1 GiB -> 1 GiB copy kernel (HBM counter calibration)")
    ap.add_argument("--no-gemm-ref", action="store_true",
                    help="skip the hipBLASLt bf16 GEMM reference rate")
    ap.add_argument("--trace-summary", default=None, metavar="DIR",
                    help="summarise a rocprofv3 --kernel-trace --stats csv output dir and exit")
    ap.add_argument("--traffic-summary", nargs=2, default=None, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="turn two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of "
                         "`bench.py --calib-copy` into profiles/hbm_traffic_<workload>.json")
    ap.add_argument("--command", default="", help="command line recorded in summaries")
    return ap.parse_args()


def upload(bits):
    import numpy as np
    import torch

    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def time_calls(fn, steps, warmup):
    """Average milliseconds per call, measured with events on the launch stream."""
    import torch

    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    start = torch.cuda.Event(enable_timing=True)
    end = torch.cuda.Event(enable_timing=True)
    start.record(stream)
    for _ in range(steps):
        fn()
    end.record(stream)
    torch.cuda.synchronize()
    return start.elapsed_time(end) / steps


def algorithmic_flops(stats, d=D, reuse=False):
    """QK^T on every pair plus P.V on kept pairs: 2*d per valid element each.  A reused
    mask skips QK^T of the skipped pairs too (reuse=True)."""
    elems = int(stats[:, 2].sum())
    skipped = int(stats[:, 3].sum())
    return 2 * d * (elems - skipped if reuse else elems) + 2 * d * (elems - skipped)


def kernel_source_digest():
    """sha256 of the kernel source: HBM counters are only valid for the code they measured."""
    import hashlib

    src = os.path.join(ROOT, "paper_2606_16317_amd", "csrc", "fa_fwd_kernel.hip")
    return hashlib.sha256(open(src, "rb").read()).hexdigest()


def measured_traffic(workload):
    """HBM bytes per launch of the DynSparse kernel from the committed rocprofv3 counter
    summary, or None when there is none or the kernel source changed since."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel_sha256") != kernel_source_digest():
        return None
    return rec.get("bytes_per_launch")


def gemm_reference(n=8192, steps=10):
    """bf16 GEMM rate of the vendor library on this GPU (context for the MFMA peak)."""
    import torch

    a = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    b = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
    ms = time_calls(lambda: torch.matmul(a, b), steps, 3)
    del a, b
    return 2.0 * n ** 3 / (ms * 1e-3) / 1e12


def cpu_baseline(q, k, v, scale, lam, budget_s):
    """Time the fp64 oracle on Q tiles of head (0, 0) for about budget_s seconds."""
    import numpy as np
    import oracle

    try:
        from threadpoolctl import threadpool_info

        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = 1
    N = q.shape[2]
    n_qt = -(-N // TILE_Q)
    t0 = time.perf_counter()
    oracle.rule_attention(q, k, v, scale, "dynsparse", lam, TILE_Q, TILE_K, tiles=[(0, 0, 0)])
    per_tile = time.perf_counter() - t0
    n = int(max(1, min(n_qt, budget_s / max(per_tile, 1e-3))))
    picks = sorted(set(np.linspace(0, n_qt - 1, n).astype(int).tolist()))
    tiles = [(0, 0, i) for i in picks]
    t0 = time.perf_counter()
    oracle.rule_attention(q, k, v, scale, "dynsparse", lam, TILE_Q, TILE_K, tiles=tiles)
    dt = time.perf_counter() - t0
    rows = sum(min(N, (i + 1) * TILE_Q) - i * TILE_Q for i in picks)
    eff = 4.0 * rows * N * D / dt / 1e12
    return {"value": eff, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{len(tiles)} of {n_qt} query tiles of head (0,0), all {-(-N // TILE_K)} "
                      f"key tiles each, {dt:.1f} s; dense-equivalent FLOP of the sample / time"}


def _find_csv(d, suffix):
    for root, _, files in os.walk(d):
        for f in files:
            if f.endswith(suffix):
                return os.path.join(root, f)
    raise FileNotFoundError(f"no *{suffix} under {d}")


def trace_summary(d, command):
    """Text summary of rocprofv3 kernel statistics (kernel_stats.csv)."""
    import csv

    rows = list(csv.DictReader(open(_find_csv(d, "kernel_stats.csv"))))
    lines = [f"# rocprofv3 --kernel-trace --stats summary", f"# command: {command}",
             f"{'calls':>6} {'avg_ms':>10} {'total_ms':>10} {'pct':>6}  kernel"]
    for r in rows:
        name = r["Name"]
        short = name if len(name) < 90 else name[:87] + "..."
        lines.append(f"{int(r['Calls']):>6} {float(r['AverageNs']) / 1e6:>10.3f} "
                     f"{float(r['TotalDurationNs']) / 1e6:>10.3f} {float(r['Percentage']):>6.2f}  {short}")
    return "\n".join(lines)


def traffic_summary(fetch_dir, write_dir, workload, command):
    """HBM bytes per launch of the DynSparse kernel from FETCH_SIZE / WRITE_SIZE (KiB per
    dispatch), each scaled by what the same counter reads for a 1 GiB copy."""
    import csv
    import statistics

    def per_kernel(d, counter):
        vals = {"main": [], "copy": []}
        for r in csv.DictReader(open(_find_csv(d, "counter_collection.csv"))):
            if r["Counter_Name"] != counter:
                continue
            kib = float(r["Counter_Value"])
            # DynSparse rule, 128-row units, ascending order, bf16 Q and K
            if re.search(r"fa_fwd_kernel<2, 128, 0, false(, 64)?>", r["Kernel_Name"]):
                vals["main"].append(kib)
            elif "AUnaryFunctor" in r["Kernel_Name"] or "MulFunctor" in r["Kernel_Name"]:
                vals["copy"].append(kib)
        return vals

    f = per_kernel(fetch_dir, "FETCH_SIZE")
    w = per_kernel(write_dir, "WRITE_SIZE")
    gib_kib = float(1 << 20)
    f_scale = statistics.median(f["copy"]) / gib_kib
    w_scale = statistics.median(w["copy"]) / gib_kib
    fetch = statistics.median(f["main"]) * 1024 / f_scale
    write = statistics.median(w["main"]) * 1024 / w_scale
    rec = {"workload": workload, "kernel": "fa_fwd_kernel<DynSparse>",
           "bytes_per_launch": fetch + write, "fetch_bytes": fetch, "write_bytes": write,
           "fetch_counter_per_copy_byte": f_scale, "write_counter_per_copy_byte": w_scale,
           "dispatches": [len(f["main"]), len(w["main"])], "command": command,
           "kernel_sha256": kernel_source_digest()}
    return rec


def main():
    args = parse()
    if args.trace_summary:
        print(trace_summary(args.trace_summary, args.command))
        return
    if args.traffic_summary:
        rec = traffic_summary(*args.traffic_summary, args.workload, args.command)
        path = os.path.join(ROOT, "profiles", f"hbm_traffic_{args.workload}.json")
        with open(path, "w") as fh:
            json.dump(rec, fh, indent=1)
        print(json.dumps(rec))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(--gpus must be 1)", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2606_16317_amd as dsa
    from synth import WORKLOADS, workload_inputs

    w = WORKLOADS[args.workload]
    recall = w.recall if args.recall is None else args.recall
    B, H, N = w.B, w.H, w.N
    scale = 1.0 / math.sqrt(D)
    print(f"[bench] generating {w.describe()}", file=sys.stderr, flush=True)
    q, k, v, meta = workload_inputs(w)
    qd, kd, vd = upload(q), upload(k), upload(v)
    o = torch.empty_like(qd)
    od = torch.empty_like(qd)
    stats = torch.zeros(B * H * 4, dtype=torch.int64, device="cuda")
    dense_stats = torch.zeros(B * H * 4, dtype=torch.int64, device="cuda")
    dense_flop = 4.0 * B * H * N * N * D
    lam = dsa.dsattn_lambda_from_recall(recall, N)

    if args.sweep:
        return sweep(args, dsa, w, qd, kd, vd, o, od, stats, scale, dense_flop)
    if args.reorder_sweep:
        return reorder_sweep(args, dsa, w, qd, kd, vd, o, od, stats, scale, dense_flop)
    if args.reuse_sweep:
        return reuse_sweep(args, dsa, w, qd, kd, vd, o, od, stats, scale, dense_flop)
    if args.q8_sweep:
        return q8_sweep(args, dsa, w, qd, kd, vd, o, od, stats, scale, dense_flop)

    def step():
        dsa.dynsparse_attn_fwd(qd, kd, vd, o, scale=scale, recall_target=recall, stats_out=stats)

    print(f"[bench] dynsparse recall={recall} lambda={lam:.3f}: {args.warmup} warmup + "
          f"{args.steps} timed steps", file=sys.stderr, flush=True)
    ms = time_calls(step, args.steps, args.warmup)
    st = stats.cpu().numpy().reshape(B * H, 4)
    flop_alg = algorithmic_flops(st)
    sp_tiles = float(st[:, 1].sum() / st[:, 0].sum())
    sp_elems = float(st[:, 3].sum() / st[:, 2].sum())

    dense_ms = None
    rel_l2 = None
    if not args.no_dense:
        print("[bench] dense reference timing", file=sys.stderr, flush=True)

        def dstep():
            dsa.dense_attn_fwd(qd, kd, vd, od, scale=scale, stats_out=dense_stats)

        dense_ms = time_calls(dstep, args.steps, args.warmup)
        diff = (o.float() - od.float()).pow(2).sum().sqrt()
        rel_l2 = float(diff / od.float().pow(2).sum().sqrt())

    achieved = flop_alg / (ms * 1e-3) / 1e12
    traffic = measured_traffic(w.name)
    if args.calib_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
    gemm = None
    if not args.no_gemm_ref:
        gemm = gemm_reference()
    cpu = None
    if args.cpu_seconds > 0:
        print("[bench] cpu oracle baseline", file=sys.stderr, flush=True)
        cpu = cpu_baseline(q, k, v, scale, lam, args.cpu_seconds)

    out = {
        "metric": METRIC,
        "value": dense_flop / (ms * 1e-3) / 1e12,
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{w.name}: Wan-2.2-14B-like 720p attention layer, "
                               f"B={B} H={H} N={N} ({'x'.join(map(str, w.grid))}) d={D}, "
                               f"bf16 in / fp32 accumulate, tile {TILE_Q}x{TILE_K}",
                   "rule": "dynsparse", "recall_target": recall, "lambda": lam,
                   "seed": w.seed},
        "speedup_vs_dense": (dense_ms / ms) if dense_ms else None,
        "dense_ms_per_step": dense_ms,
        "dense_effective_tflops": (dense_flop / (dense_ms * 1e-3) / 1e12) if dense_ms else None,
        "actual_tflops": achieved,
        "sparsity_tiles": sp_tiles,
        "sparsity_elems": sp_elems,
        "rel_l2_vs_dense": rel_l2,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                     "traffic": traffic},
        "cpu_baseline": cpu,
        "context": {"hipblaslt_bf16_gemm_tflops": gemm,
                    "note": "torch.matmul 8192^3 bf16 on the same GPU: the dense MFMA rate a "
                            "tuned library sustains here, next to the 2500 TFLOP/s headline"},
    }
    print(json.dumps(out), flush=True)


def sweep(args, dsa, w, qd, kd, vd, o, od, stats, scale, dense_flop):
    import torch

    B, H, N = w.B, w.H, w.N
    # 128-row decisions in ascending key order (the default); then every wave's 32 rows
    # deciding on their own (tile_q = 32); then the diagonal-first key order.
    # 128-key decisions (tile_k = 128, both orders) and 32-key decisions close the list.
    asc, diag = dsa.ORDER_ASCENDING, dsa.ORDER_DIAGONAL
    points = [("dense", 0.0, TILE_Q, asc)] + \
             [("dynsparse_recall", r, TILE_Q, asc) for r in (0.90, 0.95, 0.98, 0.99)] + \
             [("dynsparse_lambda", l, TILE_Q, asc) for l in (-6.0, -8.0, -10.0)] + \
             [("blasst", t, TILE_Q, asc) for t in (1e-2, 1e-3, 1e-4)] + \
             [("dynsparse_recall", 0.95, 32, asc), ("dynsparse_lambda", -6.0, 32, asc),
              ("dynsparse_lambda", -8.0, 32, asc), ("dynsparse_lambda", -10.0, 32, asc),
              ("blasst", 1e-2, 32, asc)] + \
             [("dynsparse_recall", 0.95, TILE_Q, diag), ("dynsparse_lambda", -6.0, TILE_Q, diag),
              ("dynsparse_lambda", -8.0, TILE_Q, diag), ("dynsparse_lambda", -10.0, TILE_Q, diag),
              ("blasst", 1e-2, TILE_Q, diag), ("dynsparse_lambda", -8.0, 32, diag)]
    points = [pt + (TILE_K,) for pt in points] + \
             [("dense", 0.0, TILE_Q, asc, 128), ("dynsparse_recall", 0.95, TILE_Q, asc, 128),
              ("dynsparse_lambda", -6.0, TILE_Q, asc, 128),
              ("dynsparse_lambda", -8.0, TILE_Q, asc, 128),
              ("dynsparse_lambda", -10.0, TILE_Q, asc, 128), ("blasst", 1e-2, TILE_Q, asc, 128),
              ("dynsparse_lambda", -6.0, 32, asc, 128),
              ("dynsparse_recall", 0.95, TILE_Q, diag, 128),
              ("dynsparse_lambda", -6.0, TILE_Q, diag, 128),
              ("dynsparse_lambda", -8.0, TILE_Q, diag, 128),
              ("dense", 0.0, TILE_Q, asc, 32), ("dynsparse_recall", 0.95, TILE_Q, asc, 32),
              ("dynsparse_lambda", -6.0, TILE_Q, asc, 32),
              ("dynsparse_lambda", -8.0, TILE_Q, asc, 32),
              ("dynsparse_lambda", -10.0, TILE_Q, asc, 32), ("blasst", 1e-2, TILE_Q, asc, 32),
              ("dynsparse_lambda", -6.0, 32, asc, 32)]
    rule_ids = {"dense": dsa.RULE_DENSE, "dynsparse_recall": dsa.RULE_DYNSPARSE_RECALL,
                "dynsparse_lambda": dsa.RULE_DYNSPARSE_LAMBDA, "blasst": dsa.RULE_BLASST}
    dense_ms = None
    for rule, p, tq, order, tk in points:
        out = od if (rule == "dense" and tk == TILE_K) else o
        fn = lambda: dsa.dsattn_attn_fwd_ex(rule_ids[rule], p, qd, kd, vd, out, scale=scale,
                                            tile_q=tq, tile_k=tk, stats_out=stats,
                                            key_order=order)
        print(f"[sweep] {rule} {p} tile_q={tq} tile_k={tk} order={order}", file=sys.stderr,
              flush=True)
        ms = time_calls(fn, args.steps, args.warmup)
        st = stats.cpu().numpy().reshape(B * H, 4)
        if rule == "dense" and tk == TILE_K:
            dense_ms = ms
            rel = 0.0
        else:
            rel = float((o.float() - od.float()).pow(2).sum().sqrt() /
                        od.float().pow(2).sum().sqrt())
        rec = {"workload": w.name, "rule": rule, "param": p, "tile_q": tq, "tile_k": tk,
               "key_order": "diagonal" if order == diag else "ascending", "ms": ms,
               "effective_tflops": dense_flop / (ms * 1e-3) / 1e12,
               "actual_tflops": algorithmic_flops(st) / (ms * 1e-3) / 1e12,
               "sparsity_tiles": float(st[:, 1].sum() / st[:, 0].sum()),
               "speedup_vs_dense": dense_ms / ms, "rel_l2_vs_dense": rel}
        print(json.dumps(rec), flush=True)


def reorder_sweep(args, dsa, w, qd, kd, vd, o, od, stats, scale, dense_flop):
    import torch

    B, H, N = w.B, w.H, w.N
    qb = tuple(int(x) for x in args.q_block.split(","))
    kb = tuple(int(x) for x in args.kv_block.split(","))
    q_idx = torch.from_numpy(dsa.dsattn_block_order(w.grid, qb)).cuda()
    kv_idx = torch.from_numpy(dsa.dsattn_block_order(w.grid, kb)).cuda()
    ws = torch.empty(dsa.dsattn_reordered_workspace_bytes(B, H, N, D), dtype=torch.uint8,
                     device="cuda")

    # row gather kernel alone: one [B,H,N,128] bf16 tensor, read once and written once
    g = torch.empty_like(qd)
    ms = time_calls(lambda: dsa.dsattn_gather_rows(qd, q_idx, g), args.steps, args.warmup)
    moved = 2 * B * H * N * D * 2 + N * 4
    del g
    print(json.dumps({"workload": w.name, "kernel": "gather_rows", "ms": ms,
                      "roofline": {"bound": "hbm", "achieved": moved / (ms * 1e-3) / 1e9,
                                   "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                   "frac": moved / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}}),
          flush=True)

    rules = {"dense": dsa.RULE_DENSE, "dynsparse_recall": dsa.RULE_DYNSPARSE_RECALL,
             "dynsparse_lambda": dsa.RULE_DYNSPARSE_LAMBDA, "blasst": dsa.RULE_BLASST}
    points = [("dense", 0.0), ("dynsparse_recall", 0.95), ("dynsparse_lambda", -10.0),
              ("dynsparse_lambda", -8.0), ("dynsparse_lambda", -6.0), ("blasst", 1e-2)]
    dense_ms = None
    for rule, p in points:
        rec = {"workload": w.name, "rule": rule, "param": p, "q_block": qb, "kv_block": kb}
        for order in ("row_major", "blocked"):
            if order == "row_major":
                fn = lambda: dsa.dsattn_attn_fwd_ex(rules[rule], p, qd, kd, vd, o, scale=scale,
                                                    stats_out=stats)
            else:
                fn = lambda: dsa.dsattn_attn_fwd_reordered(rules[rule], p, qd, kd, vd, q_idx,
                                                           kv_idx, o, scale=scale,
                                                           stats_out=stats, workspace=ws)
            print(f"[reorder-sweep] {rule} {p} {order}", file=sys.stderr, flush=True)
            ms = time_calls(fn, args.steps, args.warmup)
            st = stats.cpu().numpy().reshape(B * H, 4)
            if rule == "dense" and order == "row_major":
                dense_ms = ms
                od.copy_(o)
            rel = float((o.float() - od.float()).pow(2).sum().sqrt() /
                        od.float().pow(2).sum().sqrt())
            rec[order] = {"ms": ms, "effective_tflops": dense_flop / (ms * 1e-3) / 1e12,
                          "sparsity_tiles": float(st[:, 1].sum() / st[:, 0].sum()),
                          "speedup_vs_dense": dense_ms / ms, "rel_l2_vs_dense": rel}
        print(json.dumps(rec), flush=True)


def reuse_sweep(args, dsa, w, qd, kd, vd, o, od, stats, scale, dense_flop):
    import torch

    B, H, N = w.B, w.H, w.N
    dense_ms = time_calls(lambda: dsa.dense_attn_fwd(qd, kd, vd, od, scale=scale),
                          args.steps, args.warmup)
    for tq in (TILE_Q, 32):
        n_qu, n_kt = -(-N // tq), -(-N // TILE_K)
        for lam in (-6.0, -8.0, -10.0):
            mask = torch.zeros(B * H * n_qu * n_kt, dtype=torch.uint8, device="cuda")
            print(f"[reuse-sweep] lambda={lam} tile_q={tq}", file=sys.stderr, flush=True)
            rule_ms = time_calls(lambda: dsa.dsattn_attn_fwd_ex(
                dsa.RULE_DYNSPARSE_LAMBDA, lam, qd, kd, vd, o, scale=scale, tile_q=tq,
                mask_out=mask), args.steps, args.warmup)
            sp = float(mask.float().mean())
            reuse_ms = time_calls(lambda: dsa.dsattn_attn_fwd_ex(
                dsa.RULE_MASK, 0.0, qd, kd, vd, o, scale=scale, tile_q=tq, mask_in=mask,
                stats_out=stats), args.steps, args.warmup)
            st = stats.cpu().numpy().reshape(B * H, 4)
            rel = float((o.float() - od.float()).pow(2).sum().sqrt() /
                        od.float().pow(2).sum().sqrt())
            print(json.dumps({"workload": w.name, "lambda": lam, "tile_q": tq,
                              "sparsity_tiles": sp, "dense_ms": dense_ms, "rule_ms": rule_ms,
                              "reuse_ms": reuse_ms,
                              "reuse_effective_tflops": dense_flop / (reuse_ms * 1e-3) / 1e12,
                              "reuse_actual_tflops": algorithmic_flops(st, reuse=True) /
                              (reuse_ms * 1e-3) / 1e12,
                              "reuse_speedup_vs_dense": dense_ms / reuse_ms,
                              "rel_l2_vs_dense": rel}), flush=True)


def q8_sweep(args, dsa, w, qd, kd, vd, o, od, stats, scale, dense_flop):
    import torch

    B, H, N = w.B, w.H, w.N
    qc = torch.empty(qd.shape, dtype=torch.uint8, device="cuda")
    qs = torch.empty((B, H, N, D // 32), dtype=torch.uint8, device="cuda")
    kc, ks = torch.empty_like(qc), torch.empty_like(qs)
    ms = time_calls(lambda: dsa.dsattn_quantize_mxfp8(qd, qc, qs), args.steps, args.warmup)
    moved = B * H * N * (2 * D + D + D // 32)           # bf16 in, codes and exponents out
    print(json.dumps({"workload": w.name, "kernel": "quantize_mxfp8", "ms": ms,
                      "roofline": {"bound": "hbm", "achieved": moved / (ms * 1e-3) / 1e9,
                                   "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                   "frac": moved / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}}),
          flush=True)
    dsa.dsattn_quantize_mxfp8(kd, kc, ks)
    # key smoothing: the per-head mean key, then K - mean quantised
    mean = torch.empty((B, H, D), dtype=torch.float32, device="cuda")
    ms = time_calls(lambda: dsa.dsattn_key_mean(kd, mean), args.steps, args.warmup)
    moved = B * H * N * D * 2 + B * H * D * 4
    print(json.dumps({"workload": w.name, "kernel": "key_mean", "ms": ms,
                      "roofline": {"bound": "hbm", "achieved": moved / (ms * 1e-3) / 1e9,
                                   "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                   "frac": moved / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}}),
          flush=True)
    kcs, kss = torch.empty_like(kc), torch.empty_like(ks)
    ms = time_calls(lambda: dsa.dsattn_quantize_mxfp8(kd, kcs, kss, shift=mean), args.steps,
                    args.warmup)
    moved = B * H * N * (2 * D + D + D // 32) + B * H * D * 4
    print(json.dumps({"workload": w.name, "kernel": "quantize_mxfp8_shift", "ms": ms,
                      "roofline": {"bound": "hbm", "achieved": moved / (ms * 1e-3) / 1e9,
                                   "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                   "frac": moved / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS}}),
          flush=True)
    rules = {"dense": dsa.RULE_DENSE, "dynsparse_recall": dsa.RULE_DYNSPARSE_RECALL,
             "dynsparse_lambda": dsa.RULE_DYNSPARSE_LAMBDA, "blasst": dsa.RULE_BLASST}
    points = [("dense", 0.0), ("dynsparse_recall", 0.95), ("dynsparse_lambda", -10.0),
              ("dynsparse_lambda", -8.0), ("dynsparse_lambda", -6.0), ("blasst", 1e-2)]
    dense_ms = None
    for rule, p in points:
        rec = {"workload": w.name, "rule": rule, "param": p}
        for fmt in ("bf16", "mxfp8", "mxfp8_smooth"):
            out = od if (rule == "dense" and fmt == "bf16") else o
            if fmt == "bf16":
                fn = lambda: dsa.dsattn_attn_fwd_ex(rules[rule], p, qd, kd, vd, out, scale=scale,
                                                    stats_out=stats)
            else:
                kk, kks = (kc, ks) if fmt == "mxfp8" else (kcs, kss)
                fn = lambda: dsa.dsattn_attn_fwd_mxfp8(rules[rule], p, qc, qs, kk, kks, vd, out,
                                                       scale=scale, stats_out=stats)
            print(f"[q8-sweep] {rule} {p} {fmt}", file=sys.stderr, flush=True)
            ms = time_calls(fn, args.steps, args.warmup)
            st = stats.cpu().numpy().reshape(B * H, 4)
            if dense_ms is None:
                dense_ms = ms
            rel = float((out.float() - od.float()).pow(2).sum().sqrt() /
                        od.float().pow(2).sum().sqrt())
            elems, skipped = int(st[:, 2].sum()), int(st[:, 3].sum())
            qk, pv = 2 * D * elems, 2 * D * (elems - skipped)
            # time the issued MFMA work needs at peak: Q K^T at the fp8 (or bf16) rate, P V
            # at the bf16 rate
            t_min = qk / ((PEAK_BF16_TFLOPS if fmt == "bf16" else PEAK_FP8_TFLOPS) * 1e12) + \
                pv / (PEAK_BF16_TFLOPS * 1e12)
            rec[fmt] = {"ms": ms, "effective_tflops": dense_flop / (ms * 1e-3) / 1e12,
                        "sparsity_tiles": float(st[:, 1].sum() / st[:, 0].sum()),
                        "speedup_vs_bf16_dense": dense_ms / ms, "rel_l2_vs_bf16_dense": rel,
                        "mfma_roofline_frac": t_min / (ms * 1e-3)}
        print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
