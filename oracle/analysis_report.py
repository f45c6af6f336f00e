"""Report of the oracle-side analysis on the synthetic video layers (CPU only).

TEST INFRASTRUCTURE: calls only ``oracle`` and the seeded input generator.

    python -m oracle.analysis_report [--workload wan480p] [--heads 4] [--masks DIR]

1. DynSparse's gap to the sorted selection of Section 3 at equal error variance, per
   threshold, averaged over sampled rows.
2. Table 3's kurtosis statistics over attention rows of the synthetic heads at several
   concentrations (MAE at recall ~0.8, recall at MAE ~0.05, by excess-kurtosis bin).
3. Optionally, PGM pictures of full skip masks of one head (row-major and blocked token
   order, ascending and diagonal-first key order).
"""

from __future__ import annotations

import argparse
import math
import os

import numpy as np

from oracle import bf16_to_f64, lambda_from_recall, rule_attention
from oracle.analysis import dynsparse_gap, kurtosis_table, mask_pgm, softmax_row
from oracle.reorder import block_order, gather_rows
from synth import WORKLOADS, make_video_qkv


def gap_report(w, heads, rng):
    q, k, v, meta = make_video_qkv(1, heads, w.grid, w.a_lo, w.a_hi, True, w.seed)
    N = q.shape[2]
    scale = 1 / math.sqrt(128)
    n_qt = -(-N // 128)
    lines = ["| lambda | DynSparse token sparsity | optimal at equal error | recall (DynSparse / optimal) |",
             "|---|---|---|---|"]
    for lam in (lambda_from_recall(0.95, N), -10.0, -8.0, -6.0):
        acc = []
        for h in range(heads):
            for qi in rng.choice(n_qt, 2, replace=False):
                run = rule_attention(q, k, v, scale, "dynsparse", lam, 128, 64,
                                     tiles=[(0, h, int(qi))])
                res = run.results[0]
                r0, r1 = run.row_ranges[0]
                s = scale * (bf16_to_f64(q[0, h, r0:r1]) @ bf16_to_f64(k[0, h]).T)
                for r in rng.choice(r1 - r0, 4, replace=False):
                    acc.append(dynsparse_gap(s[r], res.kept_cols))
        mean = lambda key: float(np.mean([a[key] for a in acc]))
        lines.append(f"| {lam:.2f} | {mean('dynsparse_sparsity'):.3f} | "
                     f"{mean('optimal_sparsity'):.3f} | {mean('dynsparse_recall'):.4f} / "
                     f"{mean('optimal_recall'):.4f} |")
    return "\n".join(lines)


def kurtosis_report(w, rng, rows_per_a=12):
    lines = ["| excess kurtosis | rows | MAE at recall ~0.8 (mean +- std) | recall at MAE ~0.05 (mean (var)) |",
             "|---|---|---|---|"]
    rows, vals = [], None
    grid = (2, 16, 32)
    for a in (0.5, 1.0, 2.0, 3.0, 4.0, 6.0, 8.0):
        q, k, v, _ = make_video_qkv(1, 1, grid, a, a, False, 100 + int(10 * a))
        scale = 1 / math.sqrt(128)
        kk = bf16_to_f64(k[0, 0])
        vals = bf16_to_f64(v[0, 0])
        for r in rng.choice(q.shape[2], rows_per_a, replace=False):
            rows.append(softmax_row(scale * (bf16_to_f64(q[0, 0, r]) @ kk.T)))
    for t in kurtosis_table(rows, vals):
        lo, hi = t["bin"]
        mae = ("-" if t["mae_at_recall_mean"] is None
               else f"{t['mae_at_recall_mean']:.4f} +- {t['mae_at_recall_std']:.4f}")
        rec = ("-" if t["recall_at_mae_mean"] is None
               else f"{t['recall_at_mae_mean']:.3f} ({t['recall_at_mae_var']:.4f})")
        lines.append(f"| ({lo:g}, {hi:g}] | {t['rows']} | {mae} | {rec} |")
    return "\n".join(lines)


def write_masks(w, out_dir):
    os.makedirs(out_dir, exist_ok=True)
    q, k, v, _ = make_video_qkv(1, 1, w.grid, 2.5, 2.5, False, w.seed)
    scale = 1 / math.sqrt(128)
    qp, kp = block_order(w.grid, (2, 8, 8)), block_order(w.grid, (1, 8, 8))
    variants = {"rowmajor_asc": (q, k, v, "ascending"),
                "rowmajor_diag": (q, k, v, "diagonal"),
                "blocked_asc": (gather_rows(q, qp), gather_rows(k, kp), gather_rows(v, kp),
                                "ascending")}
    for name, (qq, kk, vv, order) in variants.items():
        run = rule_attention(qq, kk, vv, scale, "dynsparse", -8.0, 128, 64, key_order=order)
        mask = np.stack([r.skip for r in run.results])
        path = os.path.join(out_dir, f"mask_{w.name}_{name}_lam-8.pgm")
        with open(path, "wb") as fh:
            fh.write(mask_pgm(mask))
        print(f"wrote {path}: sparsity {mask.mean():.3f}")


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawTextHelpFormatter)
    ap.add_argument("--workload", default="wan480p")
    ap.add_argument("--heads", type=int, default=4)
    ap.add_argument("--masks", default=None, help="write PGM skip masks into this directory")
    args = ap.parse_args(argv)
    w = WORKLOADS[args.workload]
    rng = np.random.default_rng(0)
    print(f"## DynSparse vs the sorted selection at equal error ({w.describe()}, "
          f"{args.heads} heads, 8 rows of 2 query tiles each)\n")
    print(gap_report(w, args.heads, rng))
    print("\n## Table 3 statistics on synthetic rows (one 2x16x32 head per concentration)\n")
    print(kurtosis_report(w, rng))
    if args.masks:
        print()
        write_masks(w, args.masks)


if __name__ == "__main__":
    main()
