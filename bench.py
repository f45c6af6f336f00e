"""Throughput of the DynSparse forward pass on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload wan720p]

A step is one call of ``dynsparse_attn_fwd`` (recall target 0.95) over one synthetic
video attention layer -- by default the Wan-2.2-14B-like 720p layer (B=1, H=40,
N=75600 = 21x45x80 latent tokens, d=128, bf16) -- with the inputs already resident in
HBM.  ``value`` is the effective (dense-equivalent) throughput 4*B*H*N^2*d / time; the
same run times the library's own ``dense_attn_fwd`` for the speedup, reports the
kernel's bf16 MFMA roofline fraction on the work it actually issues and the achieved
per-row recall (from the kernels' own LSE outputs), and times the fp64 CPU oracle on a
bounded sample of the same layer, teacher-forced on the GPU's skip mask (which also gives
the sampled-tile decision mismatch count).  One JSON line is printed.

``--all-configs`` prints one JSON line per workload and rule instead: the tiny, 480p and
720p layers at their recall target (720p also at the paper's lambda = -6 and at -8),
every point of the threshold sweep plus lambda = -6 on its draw, and the stress layer
(recall target and lambda = -6), each with throughput,
roofline fraction, speedup over dense, sparsity, relative L2 against dense, achieved
recall and the oracle mismatch count on sampled query tiles.

``--lam L`` times DynSparse at a fixed threshold instead of the recall target (the sparse
path, for profiling); ``--tag`` names the traffic record that line reads.

``--trace-summary``, ``--counter-summary`` and ``--traffic-summary`` turn rocprofv3 output
(kernel trace with stats; SQ/GRBM counter passes; FETCH_SIZE and WRITE_SIZE passes of a
``--calib-copy`` run) into the summaries kept under ``profiles/``; each summary records the
command that produced its input.

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
import multiprocessing
import os
import re
import shutil
import sys
import tempfile
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "effective TFLOP/s (dense-equiv) + speedup vs own dense FA at matched recall"
PEAK_BF16_TFLOPS = 2500.0    # MI355X dense bf16 MFMA
PEAK_FP8_TFLOPS = 5000.0     # MI355X dense fp8 MFMA
HBM_PEAK_GBS = 8000.0
TILE_Q, TILE_K, D = 128, 64, 128
CPU_SHARE = 16               # host cores that go with one GPU on the GPU machines


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="wan720p")
    ap.add_argument("--recall", type=float, default=None, help="recall target (default: workload's)")
    ap.add_argument("--lam", type=float, default=None,
                    help="time DynSparse at this fixed lambda instead of a recall target "
                         "(profiling of the sparse path)")
    ap.add_argument("--tag", default="",
                    help="suffix of the traffic record read or written "
                         "(profiles/hbm_traffic_<workload>[_<tag>].json)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="approximate wall-clock budget of the oracle baseline (0 = skip)")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense timing (profiling)")
    ap.add_argument("--all-configs", action="store_true",
                    help="one line per workload and rule (throughput, sparsity, error, recall)")
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
    ap.add_argument("--counter-summary", nargs="+", default=None, metavar="DIR",
                    help="summarise rocprofv3 --pmc csv output dirs (SQ / GRBM counters of "
                         "the attention kernels) and exit")
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


def traffic_path(workload, tag=""):
    return os.path.join(ROOT, "profiles",
                        f"hbm_traffic_{workload}{'_' + tag if tag else ''}.json")


def measured_traffic(workload, tag=""):
    """HBM bytes per launch of the DynSparse kernel from the committed rocprofv3 counter
    summary, or None when there is none or the kernel source changed since."""
    path = traffic_path(workload, tag)
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


# ---------------------------------------------------------------------------------------
# CPU leg: the fp64 oracle on the host's cores, one worker process per core with one BLAS
# thread each.  The pool is started before anything touches the GPU and its workers
# never do; they read the sampled heads from .npy files (memory-mapped) and run the
# oracle on their query tiles, teacher-forced on the GPU's skip decisions.

_HEADS = {}


_ONE_THREAD = {"OMP_NUM_THREADS": "1", "OPENBLAS_NUM_THREADS": "1", "MKL_NUM_THREADS": "1",
               "BLIS_NUM_THREADS": "1"}


def _worker_init():
    # one BLAS thread per worker: set before numpy (and its BLAS) is first imported here,
    # then enforced on whatever BLAS got loaded
    os.environ.update(_ONE_THREAD)
    import numpy  # noqa: F401

    try:
        from threadpoolctl import threadpool_limits

        threadpool_limits(1)
    except Exception:
        pass


def _oracle_task(task):
    """Run the oracle on one query tile; returns timing and the comparison with the GPU."""
    import numpy as np
    import oracle

    path, hi, qi, rule, thr, forced, o_gpu = task
    if path not in _HEADS:
        _HEADS.clear()
        _HEADS[path] = tuple(np.load(os.path.join(path, f"{x}.npy"), mmap_mode="r")
                             for x in ("q", "k", "v"))
    q, k, v = _HEADS[path]
    t0 = time.perf_counter()
    run = oracle.rule_attention(q[hi:hi + 1][None], k[hi:hi + 1][None], v[hi:hi + 1][None],
                                1.0 / math.sqrt(D), rule, thr, TILE_Q, TILE_K,
                                tiles=[(0, 0, qi)], forced_mask=forced)
    dt = time.perf_counter() - t0
    res = run.results[0]
    r0, r1 = run.row_ranges[0]
    own = res.margin < 0
    bad = own != res.skip
    worst = float(np.abs(res.margin[bad]).max()) if bad.any() else 0.0
    err = 0.0
    if o_gpu is not None:
        err = float(np.abs(oracle.bf16_to_f64(o_gpu) - res.o_sparse).max())
    return {"seconds": dt, "rows": r1 - r0, "mismatches": int(bad.sum()), "worst": worst,
            "near": int((np.abs(res.margin) < 1e-3).sum()), "o_max_abs": err}


def host_cpu():
    """CPU model, visible logical CPUs and the physical cores behind them."""
    cpus = sorted(os.sched_getaffinity(0))
    model, phys = "unknown", set()
    try:
        cur = {}
        for line in open("/proc/cpuinfo"):
            if not line.strip():
                if cur.get("processor") is not None and int(cur["processor"]) in cpus:
                    phys.add((cur.get("physical id"), cur.get("core id")))
                    model = cur.get("model name", model)
                cur = {}
                continue
            key, _, val = line.partition(":")
            cur[key.strip()] = val.strip()
    except OSError:
        pass
    return {"cpu_model": model, "logical_cpus_visible": len(cpus),
            "physical_cores_visible": len(phys) or None}


class OracleLeg:
    """Spawned worker pool for the oracle; created before the first GPU call."""

    def __init__(self):
        self.info = host_cpu()
        self.workers = max(1, min(self.info["logical_cpus_visible"],
                                  int(os.environ.get("OMP_NUM_THREADS", CPU_SHARE)), CPU_SHARE))
        ctx = multiprocessing.get_context("spawn")
        saved = {k: os.environ.get(k) for k in _ONE_THREAD}
        os.environ.update(_ONE_THREAD)          # inherited by the spawned workers
        try:
            self.pool = ctx.Pool(self.workers, initializer=_worker_init)
        finally:
            for k, val in saved.items():
                if val is None:
                    os.environ.pop(k, None)
                else:
                    os.environ[k] = val
        self.dir = tempfile.mkdtemp(prefix="dsattn_oracle_")
        self.paths = {}

    def stage(self, name, q, k, v, heads):
        """Write the sampled heads (list of flat b*H + h indices) of one workload."""
        import numpy as np

        path = os.path.join(self.dir, name)
        os.makedirs(path, exist_ok=True)
        B, H = q.shape[:2]
        for x, arr in (("q", q), ("k", k), ("v", v)):
            np.save(os.path.join(path, f"{x}.npy"), arr.reshape(B * H, *arr.shape[2:])[heads])
        self.paths[name] = (path, list(heads))

    def run(self, name, rule, thr, tiles, mask=None, o=None, budget_s=None):
        """Oracle over ``tiles`` = [(flat head, query tile)], teacher-forced on ``mask``
        ([BH][n_qt][n_kt] numpy, or None).  With budget_s the sample is cut to what the
        pool does in about that long (from the time of a first round of one tile per
        worker)."""
        path, heads = self.paths[name]
        pos = {h: i for i, h in enumerate(heads)}

        def task(t):
            bh, qi = t
            f = None if mask is None else mask[bh][None, None]
            og = None if o is None else o[bh, qi * TILE_Q:(qi + 1) * TILE_Q]
            return (path, pos[bh], qi, rule, thr, f, og)

        tiles = list(tiles)
        t0 = time.perf_counter()
        # generous deadlines: a worker that cannot start must not hang the bench
        first = self.pool.map_async(_oracle_task, [task(t) for t in tiles[:self.workers]]
                                    ).get(timeout=600)
        done = list(first)
        rest = tiles[self.workers:]
        if budget_s is not None and rest:
            per_round = time.perf_counter() - t0
            rounds = max(0, int(budget_s / max(per_round, 1e-3)) - 1)
            rest = rest[:rounds * self.workers]
        if rest:
            done += self.pool.map_async(_oracle_task, [task(t) for t in rest], chunksize=1
                                        ).get(timeout=600 + 4 * (budget_s or 600))
        wall = time.perf_counter() - t0
        n = len(done)
        return {"tiles": n, "wall_s": wall, "rows": sum(r["rows"] for r in done),
                "mismatches": sum(r["mismatches"] for r in done),
                "max_mismatch_margin": max([r["worst"] for r in done] or [0.0]),
                "within_band": sum(r["near"] for r in done),
                "o_max_abs_vs_gpu": max([r["o_max_abs"] for r in done] or [0.0]),
                "sampled": tiles[:n]}

    def close(self):
        self.pool.close()
        self.pool.join()
        shutil.rmtree(self.dir, ignore_errors=True)


def spread_tiles(heads, n_qt, per_head):
    """Query tiles spread evenly over each head (always the first and the last)."""
    import numpy as np

    picks = sorted(set(np.linspace(0, n_qt - 1, max(2, per_head)).round().astype(int).tolist()))
    # interleave heads so that a cut sample still covers every head
    return [(h, qi) for qi in picks for h in heads]


def cpu_baseline_record(res, N, workers, info, name, forced=True):
    eff = 4.0 * res["rows"] * N * D / res["wall_s"] / 1e12
    how = "teacher-forced on the GPU mask" if forced else "own decisions"
    return {"value": eff, "unit": "TFLOP/s", "cores": workers, "kind": "oracle",
            "sample": f"{res['tiles']} query tiles of {name} spread over sampled heads, every "
                      f"key tile of each, {how}; "
                      f"{res['wall_s']:.1f} s wall on {workers} worker processes with one "
                      f"BLAS thread each; dense-equivalent FLOP of the sample / wall time",
            "cpu_model": info["cpu_model"], "physical_cores_visible": info["physical_cores_visible"],
            "logical_cpus_visible": info["logical_cpus_visible"], "blas_threads_per_worker": 1}


# ---------------------------------------------------------------------------------------
# GPU measurement of one rule on one workload

def rule_ids(dsa):
    return {"dense": dsa.RULE_DENSE, "dynsparse_recall": dsa.RULE_DYNSPARSE_RECALL,
            "dynsparse_lambda": dsa.RULE_DYNSPARSE_LAMBDA, "blasst": dsa.RULE_BLASST}


def oracle_threshold(rule, p, N):
    if rule == "dense":
        return "dense", 0.0
    if rule == "blasst":
        return "blasst", math.log(p) if p > 0 else -math.inf
    if rule == "dynsparse_recall":
        return "dynsparse", math.log((1.0 - p) / N) if p < 1 else -math.inf
    return "dynsparse", p


class Layer:
    """Device copies of one workload plus its dense reference (time, output, LSE)."""

    def __init__(self, dsa, w, q, k, v, steps, warmup, dense=True):
        import torch

        self.dsa, self.w = dsa, w
        self.B, self.H, self.N = w.B, w.H, w.N
        self.qd, self.kd, self.vd = upload(q), upload(k), upload(v)
        self.o = torch.empty_like(self.qd)
        self.od = torch.empty_like(self.qd)
        self.stats = torch.zeros(self.B * self.H * 4, dtype=torch.int64, device="cuda")
        self.lse = torch.empty(self.B * self.H * self.N, dtype=torch.float32, device="cuda")
        self.lse_d = torch.empty_like(self.lse)
        self.dense_flop = 4.0 * self.B * self.H * self.N * self.N * D
        self.steps, self.warmup = steps, warmup
        self.dense_ms = None
        if dense:
            self.dense_ms = time_calls(lambda: dsa.dense_attn_fwd(self.qd, self.kd, self.vd,
                                                                  self.od, scale=self.scale),
                                       steps, warmup)
            dsa.dsattn_attn_fwd_ex(dsa.RULE_DENSE, 0.0, self.qd, self.kd, self.vd, self.od,
                                   scale=self.scale, lse_out=self.lse_d)

    @property
    def scale(self):
        return 1.0 / math.sqrt(D)

    def measure(self, rule, p, tile_q=TILE_Q, tile_k=TILE_K, mask=None, time_it=True):
        """Time the rule (unless time_it is False), then, outside the timed region, one call
        with its LSE and mask for recall, relative L2 against dense, and the decisions."""
        import torch

        dsa = self.dsa
        rid = rule_ids(dsa)[rule]
        fn = lambda: dsa.dsattn_attn_fwd_ex(rid, p, self.qd, self.kd, self.vd, self.o,
                                            scale=self.scale, tile_q=tile_q, tile_k=tile_k,
                                            stats_out=self.stats)
        rec = {}
        if time_it:
            ms = time_calls(fn, self.steps, self.warmup)
            st = self.stats.cpu().numpy().reshape(self.B * self.H, 4)
            flop = algorithmic_flops(st)
            rec = {"ms": ms, "effective_tflops": self.dense_flop / (ms * 1e-3) / 1e12,
                   "actual_tflops": flop / (ms * 1e-3) / 1e12,
                   "roofline_frac": flop / (ms * 1e-3) / 1e12 / PEAK_BF16_TFLOPS,
                   "sparsity_tiles": float(st[:, 1].sum() / st[:, 0].sum()),
                   "sparsity_elems": float(st[:, 3].sum() / st[:, 2].sum())}
        dsa.dsattn_attn_fwd_ex(rid, p, self.qd, self.kd, self.vd, self.o, scale=self.scale,
                               tile_q=tile_q, tile_k=tile_k, lse_out=self.lse, mask_out=mask)
        torch.cuda.synchronize()
        if time_it and self.dense_ms is not None:
            rec["dense_ms"] = self.dense_ms
            rec["speedup_vs_dense"] = self.dense_ms / ms
        if self.dense_ms is not None:
            od, o = self.od.float(), self.o.float()
            rec["rel_l2_vs_dense"] = float((o - od).pow(2).sum().sqrt() / od.pow(2).sum().sqrt())
            # per-row recall: dense softmax mass of the kept keys, exp(LSE_kept - LSE_all)
            r = torch.exp(self.lse.double() - self.lse_d.double())
            rec["recall_min"] = float(r.min())
            rec["recall_mean"] = float(r.mean())
        return rec


def layer_inputs(w):
    from synth import workload_inputs

    return workload_inputs(w)


def sample_heads(w, n):
    import numpy as np

    BH = w.B * w.H
    return sorted(set(np.linspace(0, BH - 1, min(n, BH)).round().astype(int).tolist()))


def main():
    args = parse()
    if args.trace_summary:
        print(trace_summary(args.trace_summary, args.command))
        return
    if args.counter_summary:
        print(counter_summary(args.counter_summary, args.command))
        return
    if args.traffic_summary:
        rec = traffic_summary(*args.traffic_summary, args.workload, args.command)
        path = traffic_path(args.workload, args.tag)
        with open(path, "w") as fh:
            json.dump(rec, fh, indent=1)
        print(json.dumps(rec))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(--gpus must be 1)", file=sys.stderr)
        sys.exit(2)

    from synth import WORKLOADS

    sweeps = args.sweep or args.reorder_sweep or args.reuse_sweep or args.q8_sweep
    # The oracle's worker pool starts before the first GPU call.
    leg = OracleLeg() if (args.cpu_seconds > 0 and not sweeps) else None
    try:
        if args.all_configs:
            return all_configs(args, leg)
        w = WORKLOADS[args.workload]
        print(f"[bench] generating {w.describe()}", file=sys.stderr, flush=True)
        q, k, v, meta = layer_inputs(w)
        if leg is not None:
            leg.stage(w.name, q, k, v, sample_heads(w, 8))
        import torch  # noqa: F401  (first GPU use below)

        import paper_2606_16317_amd as dsa

        if sweeps:
            return legacy_sweeps(args, dsa, w, q, k, v)
        return headline(args, dsa, w, q, k, v, leg)
    finally:
        if leg is not None:
            leg.close()


def headline(args, dsa, w, q, k, v, leg):
    import torch

    B, H, N = w.B, w.H, w.N
    fixed = args.lam is not None
    recall = None if fixed else (w.recall if args.recall is None else args.recall)
    lam = args.lam if fixed else dsa.dsattn_lambda_from_recall(recall, N)
    rule, param = ("dynsparse_lambda", lam) if fixed else ("dynsparse_recall", recall)
    L = Layer(dsa, w, q, k, v, args.steps, args.warmup, dense=not args.no_dense)
    n_qt, n_kt = -(-N // TILE_Q), -(-N // TILE_K)
    mask = torch.empty(B * H * n_qt * n_kt, dtype=torch.uint8, device="cuda")
    print(f"[bench] dynsparse recall={recall} lambda={lam:.3f}: {args.warmup} warmup + "
          f"{args.steps} timed steps", file=sys.stderr, flush=True)

    # the timed step: dynsparse_attn_fwd (named entry point) with stats, or its fixed-lambda
    # variant
    def step():
        if fixed:
            dsa.dynsparse_attn_fwd_lambda(L.qd, L.kd, L.vd, L.o, scale=L.scale, lam=lam,
                                          stats_out=L.stats)
        else:
            dsa.dynsparse_attn_fwd(L.qd, L.kd, L.vd, L.o, scale=L.scale, recall_target=recall,
                                   stats_out=L.stats)

    ms = time_calls(step, args.steps, args.warmup)
    st = L.stats.cpu().numpy().reshape(B * H, 4)
    flop_alg = algorithmic_flops(st)
    achieved = flop_alg / (ms * 1e-3) / 1e12
    # outside the timed region: LSE, mask and output of the same rule for recall, error
    # and the oracle comparison
    rec = L.measure(rule, param, mask=mask, time_it=False)

    traffic = measured_traffic(w.name, args.tag)
    if args.calib_copy:
        src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)
        torch.cuda.synchronize()
        del src, dst
    gemm = None if args.no_gemm_ref else gemm_reference()
    cpu, oracle_cmp = None, None
    if leg is not None:
        print("[bench] cpu oracle baseline (teacher-forced on the GPU mask)", file=sys.stderr,
              flush=True)
        m = mask.cpu().numpy().reshape(B * H, n_qt, n_kt)
        o_np = L.o.view(torch.int16).cpu().numpy().view("uint16").reshape(B * H, N, D)
        _, heads = leg.paths[w.name]
        name, thr = oracle_threshold(rule, param, N)
        res = leg.run(w.name, name, thr, spread_tiles(heads, n_qt, 64), mask=m, o=o_np,
                      budget_s=args.cpu_seconds)
        cpu = cpu_baseline_record(res, N, leg.workers, leg.info, w.name)
        oracle_cmp = {k_: res[k_] for k_ in ("tiles", "mismatches", "max_mismatch_margin",
                                            "within_band", "o_max_abs_vs_gpu")}

    dense_ms = L.dense_ms
    out = {
        "metric": METRIC,
        "value": L.dense_flop / (ms * 1e-3) / 1e12,
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
        "config": {"workload": f"{w.describe()}; bf16 in / fp32 accumulate, "
                               f"tile {TILE_Q}x{TILE_K}",
                   "rule": "dynsparse", "recall_target": recall, "lambda": lam,
                   "seed": w.seed},
        "speedup_vs_dense": (dense_ms / ms) if dense_ms else None,
        "dense_ms_per_step": dense_ms,
        "dense_effective_tflops": (L.dense_flop / (dense_ms * 1e-3) / 1e12) if dense_ms else None,
        "actual_tflops": achieved,
        "sparsity_tiles": float(st[:, 1].sum() / st[:, 0].sum()),
        "sparsity_elems": float(st[:, 3].sum() / st[:, 2].sum()),
        "rel_l2_vs_dense": rec.get("rel_l2_vs_dense"),
        "recall_min": rec.get("recall_min"),
        "recall_mean": rec.get("recall_mean"),
        "oracle_comparison": oracle_cmp,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                     "traffic": traffic},
        "cpu_baseline": cpu,
        "context": {"hipblaslt_bf16_gemm_tflops": gemm,
                    "note": "torch.matmul 8192^3 bf16 on the same GPU: the dense MFMA rate a "
                            "tuned library sustains here, next to the 2500 TFLOP/s headline"},
    }
    print(json.dumps(out), flush=True)


# the per-config record: (workload, rule, parameter) in the order printed
ALL_CONFIGS = [("tiny", "dynsparse_recall", 0.95),
               ("wan480p", "dynsparse_recall", 0.95),
               ("wan720p", "dynsparse_recall", 0.95),
               ("wan720p", "dynsparse_lambda", -8.0),
               ("wan720p", "dynsparse_lambda", -6.0),
               ("wan720p_sweep", "dynsparse_recall", 0.90),
               ("wan720p_sweep", "dynsparse_recall", 0.95),
               ("wan720p_sweep", "dynsparse_recall", 0.98),
               ("wan720p_sweep", "dynsparse_recall", 0.99),
               ("wan720p_sweep", "blasst", 1e-2),
               ("wan720p_sweep", "blasst", 1e-3),
               ("wan720p_sweep", "blasst", 1e-4),
               ("wan720p_sweep", "dynsparse_lambda", -6.0),
               ("wan720p_sweep", "dense", 0.0),
               ("stress", "dynsparse_recall", 0.95),
               ("stress", "dynsparse_lambda", -6.0)]


def all_configs(args, leg):
    import torch

    from synth import WORKLOADS

    current = None
    for name, rule, p in ALL_CONFIGS:
        w = WORKLOADS[name]
        if current is None or current[0] != name:
            current = None
            print(f"[all-configs] generating {w.describe()}", file=sys.stderr, flush=True)
            q, k, v, meta = layer_inputs(w)
            if leg is not None:
                leg.stage(name, q, k, v, sample_heads(w, 4))
            import paper_2606_16317_amd as dsa

            # tiny layers need more calls per timing to rise above launch overhead
            steps = args.steps * (20 if w.N < 8192 else 1)
            current = (name, Layer(dsa, w, q, k, v, steps, args.warmup))
            del q, k, v
        L = current[1]
        n_qt, n_kt = -(-w.N // TILE_Q), -(-w.N // TILE_K)
        mask = torch.empty(w.B * w.H * n_qt * n_kt, dtype=torch.uint8, device="cuda")
        print(f"[all-configs] {name} {rule} {p}", file=sys.stderr, flush=True)
        rec = L.measure(rule, p, mask=mask)
        name_o, thr = oracle_threshold(rule, p, w.N)
        out = {"workload": w.describe(), "rule": rule, "param": p,
               "threshold_natural_log": thr if rule != "dense" else None,
               "tile_q": TILE_Q, "tile_k": TILE_K, **rec}
        if leg is not None:
            m = mask.cpu().numpy().reshape(w.B * w.H, n_qt, n_kt)
            o_np = L.o.view(torch.int16).cpu().numpy().view("uint16").reshape(w.B * w.H, w.N, D)
            _, heads = leg.paths[name]
            res = leg.run(name, name_o, thr, spread_tiles(heads, n_qt, 4), mask=m, o=o_np)
            out["oracle_sampled"] = {k_: res[k_] for k_ in ("tiles", "mismatches",
                                                           "max_mismatch_margin", "within_band",
                                                           "o_max_abs_vs_gpu", "wall_s")}
        print(json.dumps(out), flush=True)
    current = None


def legacy_sweeps(args, dsa, w, q, k, v):
    import torch

    B, H, N = w.B, w.H, w.N
    scale = 1.0 / math.sqrt(D)
    qd, kd, vd = upload(q), upload(k), upload(v)
    o = torch.empty_like(qd)
    od = torch.empty_like(qd)
    stats = torch.zeros(B * H * 4, dtype=torch.int64, device="cuda")
    dense_flop = 4.0 * B * H * N * N * D
    if args.sweep:
        return sweep(args, dsa, w, qd, kd, vd, o, od, stats, scale, dense_flop)
    if args.reorder_sweep:
        return reorder_sweep(args, dsa, w, qd, kd, vd, o, od, stats, scale, dense_flop)
    if args.reuse_sweep:
        return reuse_sweep(args, dsa, w, qd, kd, vd, o, od, stats, scale, dense_flop)
    return q8_sweep(args, dsa, w, qd, kd, vd, o, od, stats, scale, dense_flop)


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
    # The attention kernels per run of consecutive dispatches with one launch shape (in
    # issue order: each timed configuration is such a run), from the dispatch list
    try:
        trace = _find_csv(d, "kernel_trace.csv")
    except FileNotFoundError:
        return "\n".join(lines)
    disp = []
    for r in csv.DictReader(open(trace)):
        m = re.search(r"(fa_fwd_(?:mask_)?kernel<[^>]*>)", r["Kernel_Name"])
        if not m:
            continue
        disp.append((int(r["Start_Timestamp"]), m.group(1),
                     f"{int(r['Grid_Size_X']) // max(1, int(r['Workgroup_Size_X']))}x"
                     f"{r['Grid_Size_Y']}", r["Scratch_Size"], r["LDS_Block_Size"],
                     int(r["End_Timestamp"]) - int(r["Start_Timestamp"])))
    disp.sort()
    runs = []
    for _, name, grid, scr, lds, ns in disp:
        # a new run where the shape changes, or where the time moves more than 4 % from
        # the run's mean (another threshold on the same kernel)
        if runs and runs[-1][0] == (name, grid, scr, lds) and \
                abs(ns - sum(runs[-1][1]) / len(runs[-1][1])) <= 0.04 * sum(runs[-1][1]) / len(runs[-1][1]):
            runs[-1][1].append(ns)
        else:
            runs.append(((name, grid, scr, lds), [ns]))
    lines += ["", "# attention kernels, runs of consecutive dispatches in issue order, split "
                  "where the shape changes or the time moves by more than 4 % (grid in "
                  "workgroups; scratch and LDS bytes per workgroup)",
              f"{'run':>4} {'calls':>6} {'avg_ms':>10} {'min_ms':>10}  {'grid':>10} "
              f"{'scratch':>7} {'lds':>6}  kernel"]
    for n, ((name, grid, scr, lds), ns) in enumerate(runs):
        lines.append(f"{n:>4} {len(ns):>6} {sum(ns) / len(ns) / 1e6:>10.3f} "
                     f"{min(ns) / 1e6:>10.3f}  {grid:>10} {scr:>7} {lds:>6}  {name}")
    return "\n".join(lines)


# gfx950: 8 accelerator dies (GRBM_GUI_ACTIVE is summed over them), 256 CUs x 4 SIMDs
XCDS, SIMDS = 8, 1024
KERNEL_RULES = {"0": "dense", "1": "blasst", "2": "dynsparse"}


def counter_summary(dirs, command):
    """Text summary of rocprofv3 --pmc passes (one dir per pass) over the attention kernels
    (128-row units, ascending order, bf16, 64-key tiles): the last dispatch's value of each
    counter, then per-SIMD and per-wave-cycle ratios.  SQ_*_CYCLES / SQ_WAIT_* /
    SQ_ACTIVE_INST_* count per wave (in the same unit as SQ_WAVE_CYCLES), summed over the
    chip; SQ_VALU_MFMA_BUSY_CYCLES counts per SIMD."""
    import csv

    vals = {}
    for d in dirs:
        for r in csv.DictReader(open(_find_csv(d, "counter_collection.csv"))):
            m = re.search(r"fa_fwd_kernel<(\d), 128, 0, false, 64>", r["Kernel_Name"])
            if not m:
                continue
            kern = KERNEL_RULES[m.group(1)]
            vals.setdefault(kern, {}).setdefault(r["Counter_Name"], []).append(
                float(r["Counter_Value"]))
    lines = ["# rocprofv3 --pmc summary: SQ / GRBM counters of the attention kernels",
             f"# command: {command}",
             "# values: last dispatch of each kernel (counts summed over the chip)"]
    for kern, cs in vals.items():
        last = {c: v[-1] for c, v in cs.items()}
        lines.append(f"kernel fa_fwd_kernel<{kern}>  dispatches per pass: "
                     f"{min(len(v) for v in cs.values())}")
        for c in sorted(last):
            lines.append(f"  {c:<30} {last[c]:.5g}")
        cyc = last.get("GRBM_GUI_ACTIVE", 0.0) / XCDS
        if cyc and "SQ_VALU_MFMA_BUSY_CYCLES" in last:
            lines.append(f"  = MFMA busy per SIMD per cycle        "
                         f"{last['SQ_VALU_MFMA_BUSY_CYCLES'] / SIMDS / cyc:.3f}")
        wave = last.get("SQ_WAVE_CYCLES")
        if wave:
            for c in ("SQ_ACTIVE_INST_ANY", "SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_LDS",
                      "SQ_ACTIVE_INST_SCA", "SQ_ACTIVE_INST_MISC", "SQ_ACTIVE_INST_VMEM",
                      "SQ_WAIT_INST_ANY", "SQ_WAIT_INST_LDS", "SQ_WAIT_ANY", "SQ_BUSY_CYCLES"):
                if c in last:
                    lines.append(f"  = {c:<30} per wave cycle {last[c] / wave:.3f}")
        mfma = last.get("SQ_INSTS_MFMA")
        if mfma:
            for c in ("SQ_INSTS_VALU", "SQ_INSTS_VALU_TRANS_F32", "SQ_INSTS_LDS",
                      "SQ_INSTS_SALU", "SQ_INSTS_BRANCH"):
                if c in last:
                    lines.append(f"  = {c:<30} per MFMA {last[c] / mfma:.3f}")
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
