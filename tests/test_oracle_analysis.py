"""Pins of the oracle-side analysis tools (``oracle.analysis``), CPU only.

* The error-variance metric of Eq. 2/3 is checked against a Monte Carlo simulation of
  the error of the renormalised sparse output, computed from its definition (dense output
  minus sparse output) with Gaussian values -- not by retyping the formula.
* The sorted selection of Section 3 is checked against the closed form for a uniform row
  and against brute force over every subset of tiny rows (it finds the largest discard
  set that meets the tolerance).
* eps_ub of Eq. 4 is checked on a hand-worked row.
* Excess kurtosis is checked on distributions with known values (two-point: -2; large
  Gaussian sample: 0; large exponential sample: 6).
* Top-K limits: K = L keeps everything (recall 1, MAE 0); recall grows with K.
"""

import itertools
import math

import numpy as np
import pytest

from oracle import rule_attention
from oracle.analysis import (dynsparse_gap, epsilon_upper_bound, error_variance,
                             excess_kurtosis, kurtosis_table, mask_pgm, optimal_discard,
                             softmax_row, topk_mae_recall)
from synth import make_video_qkv


@pytest.mark.parametrize("seed,L,n_discard", [(0, 12, 5), (1, 40, 20), (2, 7, 1)])
def test_error_variance_matches_simulation(seed, L, n_discard):
    rng = np.random.default_rng(seed)
    p = softmax_row(rng.normal(0.0, 1.5, L))
    discard = np.zeros(L, dtype=bool)
    discard[np.argsort(p)[:n_discard]] = True
    sigma = 1.7
    v = rng.normal(0.0, sigma, size=(200_000, L))         # i.i.d. values, many draws
    dense = v @ p
    kept = ~discard
    sparse = (v[:, kept] @ p[kept]) / p[kept].sum()
    emp = float((dense - sparse).var())
    assert emp / sigma ** 2 == pytest.approx(error_variance(p, discard), rel=0.02)
    assert abs(float((dense - sparse).mean())) < 5 * math.sqrt(emp / 200_000)  # unbiased


@pytest.mark.parametrize("L,theta", [(100, 1e-3), (1000, 1e-4), (500, 0.01), (64, 1e-6)])
def test_optimal_discard_uniform_closed_form(L, theta):
    """p = 1/L: discarding k entries gives k / (L (L - k)), so the largest admissible k is
    floor(Theta L^2 / (1 + Theta L))."""
    p = np.full(L, 1.0 / L)
    discard, s1, metric = optimal_discard(p, theta)
    k = math.floor(theta * L * L / (1 + theta * L) + 1e-12)
    k = min(k, L - 1)
    assert int(discard.sum()) == k
    assert s1 == pytest.approx(k / L)
    assert metric == pytest.approx(k / (L * (L - k)) if k else 0.0)


def test_optimal_discard_is_the_largest_admissible_set_on_tiny_rows():
    rng = np.random.default_rng(7)
    for _ in range(150):
        L = int(rng.integers(3, 8))
        p = softmax_row(rng.normal(0, rng.uniform(0.2, 3), L))
        theta = float(rng.uniform(1e-4, 0.05))
        discard, _, metric = optimal_discard(p, theta)
        assert metric <= theta
        best = max(r for r in range(L)
                   for S in itertools.combinations(range(L), r)
                   if error_variance(p, np.isin(np.arange(L), S)) <= theta)
        assert int(discard.sum()) == best


def test_epsilon_upper_bound_hand_worked():
    p = np.array([0.5, 0.3, 0.15, 0.05])
    discard = np.array([False, False, False, True])
    # ||P_S||^2 = 0.0025, ||P_K||^2 = 0.25 + 0.09 + 0.0225 = 0.3625
    theta = 0.0025 + 0.3625 * 0.04 ** 2
    assert epsilon_upper_bound(p, discard, theta) == pytest.approx(0.04)
    assert math.isnan(epsilon_upper_bound(p, discard, 0.001))


def test_excess_kurtosis_known_values():
    assert excess_kurtosis(np.array([1.0, -1.0] * 50)) == pytest.approx(-2.0)
    rng = np.random.default_rng(3)
    assert excess_kurtosis(rng.normal(size=400_000)) == pytest.approx(0.0, abs=0.05)
    assert excess_kurtosis(rng.exponential(size=400_000)) == pytest.approx(6.0, abs=0.3)


def test_topk_limits_and_monotone_recall():
    rng = np.random.default_rng(4)
    p = softmax_row(rng.normal(0, 2, 50))
    v = rng.normal(size=(50, 16))
    sweep = topk_mae_recall(p, v, range(1, 51))
    recalls = [r for _, r, _ in sweep]
    assert recalls == sorted(recalls)
    assert sweep[-1][1] == pytest.approx(1.0)
    assert sweep[-1][2] == pytest.approx(0.0, abs=1e-14)


def test_kurtosis_table_separates_flat_and_peaked_rows():
    """Flat rows (low kurtosis) tolerate a low recall; peaked rows do not (the trend of
    Table 3): the MAE at recall ~0.8 grows from the flattest to the peakiest bin."""
    rng = np.random.default_rng(5)
    L, d = 512, 32
    v = rng.normal(size=(L, d))
    rows = [softmax_row(rng.normal(0, a, L)) for a in np.linspace(0.2, 4.0, 60)]
    table = kurtosis_table(rows, v)
    filled = [t for t in table if t["mae_at_recall_mean"] is not None]
    assert len(filled) >= 3
    assert filled[-1]["mae_at_recall_mean"] > filled[0]["mae_at_recall_mean"]
    assert sum(t["rows"] for t in table) == len(rows)


def test_dynsparse_gap_on_video_rows():
    """DynSparse's kept set meets some error variance; the sorted selection at that same
    variance discards at least as many tokens (it is the optimum of Section 3)."""
    q, k, v, _ = make_video_qkv(1, 1, (2, 16, 32), 5.0, 5.0, True, 8)
    scale = 1 / math.sqrt(128)
    run = rule_attention(q, k, v, scale, "dynsparse", -6.0, 128, 64, tiles=[(0, 0, 3)])
    res = run.results[0]
    from oracle import bf16_to_f64
    s = scale * (bf16_to_f64(q[0, 0, 384:512]) @ bf16_to_f64(k[0, 0]).T)
    for r in range(0, 128, 17):
        g = dynsparse_gap(s[r], res.kept_cols)
        assert g["optimal_metric"] <= g["metric"] + 1e-15
        assert g["optimal_sparsity"] >= g["dynsparse_sparsity"]
        assert g["dynsparse_recall"] == pytest.approx(float(res.recall[r]), rel=1e-9)


def test_mask_pgm_header_and_pixels():
    img = mask_pgm(np.array([[0, 1, 0], [1, 1, 0]]))
    assert img.startswith(b"P5\n3 2\n255\n")
    assert list(img[-6:]) == [255, 0, 255, 0, 0, 255]
