"""Oracle-side analysis of the sparsity/accuracy trade-off (CPU, float64).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: these functions analyse softmax
rows and skip masks produced by the oracle; no GPU path calls them.

What they compute, in the paper's notation (one attention row ``p`` summing to 1, a
discarded set S and the kept set K = complement of S):

* ``error_variance`` -- Section 2.1.1 (Eq. 1) and Section 2.2 (Eq. 2, Eq. 3): with
  i.i.d. values of variance sigma^2, the error of the renormalised sparse output is
  E = sum_S p_j v_j - S_1 / (1 - S_1) * sum_K p_j v_j with S_1 = sum_S p_j, whose variance
  divided by sigma^2 is  sum_S p_j^2 + (S_1 / (1 - S_1))^2 sum_K p_j^2.
* ``optimal_discard`` -- the selection procedure at the opening of Section 3: sort p
  ascending, move the smallest entries into S one at a time, and stop before the variance
  metric of Eq. 3 exceeds the tolerance Theta.
* ``epsilon_upper_bound`` -- Eq. 4: eps_ub solves ||P_S||^2 + eps_ub^2 ||P_K||^2 = Theta.
* ``dynsparse_gap`` -- for the kept set DynSparse chose for a row, the variance metric it
  reaches and the sparsity the sorted selection reaches at that same metric: how far the
  online rule is from the distribution-aware optimum (Section 2.2 argues a fixed eps
  cannot be optimal).
* ``excess_kurtosis`` / ``topk_mae_recall`` / ``kurtosis_table`` -- the study behind
  Table 3 (Appendix, accuracy vs recall; the ablation of Section 4.4): rows are binned by
  the excess kurtosis of their probabilities; in each bin, Top-K selections give the MAE
  at recall ~0.8 and the recall at MAE ~0.05.
* ``mask_pgm`` -- a skip mask as a portable graymap image (the mask pictures of Section
  4.3 for synthetic inputs).

Parity status: pinned by ``tests/test_oracle_analysis.py`` (Monte Carlo simulation of the
error from its definition, the uniform-row closed form of the optimal discard, brute force
over subsets on tiny rows, closed-form kurtosis of two-point and large Gaussian/exponential
samples, Top-K limits).
"""

from __future__ import annotations

import math

import numpy as np


def error_variance(p: np.ndarray, discard: np.ndarray) -> float:
    """Var(E) / sigma^2 of Eq. 3 for a probability row ``p`` and a boolean discard mask."""
    p = np.asarray(p, dtype=np.float64)
    discard = np.asarray(discard, dtype=bool)
    s1 = float(p[discard].sum())
    if s1 >= 1.0:
        return math.inf
    ratio = s1 / (1.0 - s1)
    return float((p[discard] ** 2).sum() + ratio * ratio * (p[~discard] ** 2).sum())


def optimal_discard(p: np.ndarray, theta: float):
    """Sorted selection of Section 3: discard the smallest entries while Eq. 3's metric
    stays within ``theta``.  Returns (discard mask, S_1, metric)."""
    p = np.asarray(p, dtype=np.float64)
    order = np.argsort(p, kind="stable")
    discard = np.zeros(p.size, dtype=bool)
    best_metric = 0.0
    for idx in order[:-1]:                 # the largest entry is always kept
        discard[idx] = True
        m = error_variance(p, discard)
        if m > theta:
            discard[idx] = False
            break
        best_metric = m
    return discard, float(p[discard].sum()), best_metric


def epsilon_upper_bound(p: np.ndarray, discard: np.ndarray, theta: float) -> float:
    """eps_ub of Eq. 4 for a discard set: sqrt((Theta - ||P_S||^2) / ||P_K||^2), or nan
    when ||P_S||^2 alone already exceeds Theta."""
    p = np.asarray(p, dtype=np.float64)
    discard = np.asarray(discard, dtype=bool)
    ps = float((p[discard] ** 2).sum())
    pk = float((p[~discard] ** 2).sum())
    if ps > theta or pk == 0.0:
        return math.nan
    return math.sqrt((theta - ps) / pk)


def softmax_row(s: np.ndarray) -> np.ndarray:
    s = np.asarray(s, dtype=np.float64)
    e = np.exp(s - s.max())
    return e / e.sum()


def dynsparse_gap(s_row: np.ndarray, kept_cols: np.ndarray) -> dict:
    """Compare a row's DynSparse kept set with the sorted selection at equal error.

    ``s_row``: the row's logits over all keys; ``kept_cols``: key indices DynSparse kept.
    Returns token sparsities of both, the shared variance metric and the kept mass.
    """
    p = softmax_row(s_row)
    discard = np.ones(p.size, dtype=bool)
    discard[np.asarray(kept_cols, dtype=np.int64)] = False
    metric = error_variance(p, discard)
    opt, opt_s1, opt_metric = optimal_discard(p, metric)
    return {"dynsparse_sparsity": float(discard.mean()),
            "optimal_sparsity": float(opt.mean()),
            "metric": metric, "optimal_metric": opt_metric,
            "dynsparse_recall": float(1.0 - p[discard].sum()),
            "optimal_recall": float(1.0 - opt_s1)}


def excess_kurtosis(x: np.ndarray) -> float:
    """Population excess kurtosis m4 / m2^2 - 3 of the values ``x``."""
    x = np.asarray(x, dtype=np.float64)
    d = x - x.mean()
    m2 = float((d * d).mean())
    m4 = float((d ** 4).mean())
    return m4 / (m2 * m2) - 3.0


def topk_mae_recall(p: np.ndarray, v: np.ndarray, ks) -> list:
    """For each K in ``ks``: keep the K largest probabilities, renormalise, and return
    (K, recall = kept mass, MAE = mean |O - O'| over the head dimension)."""
    p = np.asarray(p, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    order = np.argsort(-p, kind="stable")
    o_dense = p @ v
    out = []
    for k in ks:
        keep = order[:k]
        mass = float(p[keep].sum())
        o_sparse = (p[keep] @ v[keep]) / mass
        out.append((int(k), mass, float(np.abs(o_dense - o_sparse).mean())))
    return out


DEFAULT_BINS = (-math.inf, 0.0, 1.0, 3.0, 10.0, 30.0, 100.0, 300.0, 1000.0, 3000.0, 10000.0,
                math.inf)


def kurtosis_table(rows, v, bins=DEFAULT_BINS, recall_target=0.8, recall_tol=0.01,
                   mae_target=0.05, mae_tol=0.005):
    """Table 3's statistics over probability rows ``rows`` (each sums to 1) sharing the
    value matrix ``v``: per excess-kurtosis bin, MAE at recall ~recall_target (mean, std)
    and recall at MAE ~mae_target (mean, variance), from Top-K selections of every K."""
    per_bin = {i: {"mae_at_recall": [], "recall_at_mae": [], "rows": 0}
               for i in range(len(bins) - 1)}
    for p in rows:
        kurt = excess_kurtosis(p)
        b = next(i for i in range(len(bins) - 1) if bins[i] < kurt <= bins[i + 1]) \
            if kurt > bins[0] else 0
        per_bin[b]["rows"] += 1
        sweep = topk_mae_recall(p, v, range(1, p.size + 1))
        for _, rec, mae in sweep:
            if abs(rec - recall_target) <= recall_tol:
                per_bin[b]["mae_at_recall"].append(mae)
            if abs(mae - mae_target) <= mae_tol:
                per_bin[b]["recall_at_mae"].append(rec)
    table = []
    for i in range(len(bins) - 1):
        d = per_bin[i]
        mae = np.array(d["mae_at_recall"])
        rec = np.array(d["recall_at_mae"])
        table.append({"bin": (bins[i], bins[i + 1]), "rows": d["rows"],
                      "mae_at_recall_mean": float(mae.mean()) if mae.size else None,
                      "mae_at_recall_std": float(mae.std()) if mae.size else None,
                      "recall_at_mae_mean": float(rec.mean()) if rec.size else None,
                      "recall_at_mae_var": float(rec.var()) if rec.size else None})
    return table


def mask_pgm(mask: np.ndarray) -> bytes:
    """A 2-D skip mask (1 = skipped) as a binary PGM image: kept pairs white, skipped
    black, one pixel per (query tile, key tile) pair."""
    m = np.asarray(mask).astype(bool)
    if m.ndim != 2:
        raise ValueError("mask must be 2-D")
    h, w = m.shape
    pix = np.where(m, 0, 255).astype(np.uint8)
    return f"P5\n{w} {h}\n255\n".encode() + pix.tobytes()
