"""Pins of the oracle's key-tile visit order (ascending and diagonal-first), CPU only.

The DynSparse decision of a tile depends on the tiles kept *before* it (Eq. 5 reads the
LSE of the kept tiles so far), so the visit order is part of the rule.  These tests pin
the diagonal-first order by orders worked out by hand, and the rule under any order by a
from-scratch brute force that rebuilds the reference from the full logits and the kept set
in visit order, by the uniform closed form (the first tiles *in visit order* are kept), by
the recall theorem of Section 3.1 (which holds for any order) and by the dense case (order
does not change softmax attention).
"""

import math

import numpy as np
import pytest

import oracle
from oracle import diagonal_first_order, filter_q_tile, lambda_from_recall, rule_attention
from synth import make_random_qkv, make_video_qkv


def f64(bits):
    return oracle.bf16_to_f64(bits)


@pytest.mark.parametrize("n_kt,start,expect", [
    (4, 2, [2, 3, 1, 0]),
    (7, 2, [2, 3, 1, 4, 0, 5, 6]),      # the left side runs out first
    (7, 5, [5, 6, 4, 3, 2, 1, 0]),      # the right side runs out first
    (6, 0, [0, 1, 2, 3, 4, 5]),         # start at the first tile: ascending
    (5, 4, [4, 3, 2, 1, 0]),            # start at the last tile: descending
    (1, 0, [0]),
])
def test_diagonal_order_hand_worked(n_kt, start, expect):
    assert diagonal_first_order(n_kt, start) == expect


@pytest.mark.parametrize("n_kt", [1, 2, 3, 10, 37])
def test_diagonal_order_is_a_permutation_by_distance(n_kt):
    for start in range(n_kt):
        order = diagonal_first_order(n_kt, start)
        assert sorted(order) == list(range(n_kt))
        dist = [abs(t - start) for t in order]
        assert dist == sorted(dist)            # never moves away and back
        assert order[0] == start


def brute_force_in_order(s, rule, thr, tile_k, order):
    """Every decision recomputed from the full logits and the set kept so far, visiting
    key tiles in ``order`` (plain Python floats)."""
    rows, n = len(s), len(s[0])
    kept_cols, skip = [], {}
    for j in order:
        cols = range(j * tile_k, min(n, (j + 1) * tile_k))
        keep = False
        for r in range(rows):
            m_hat = max(s[r][c] for c in cols)
            if not kept_cols:
                ref = -math.inf
            elif rule == "dynsparse":
                ref = math.log(math.fsum(math.exp(s[r][c]) for c in kept_cols))
            else:
                ref = max(s[r][c] for c in kept_cols)
            if not (m_hat - ref < thr):
                keep = True
        skip[j] = not keep
        if keep:
            kept_cols.extend(cols)
    return np.array([skip[j] for j in range(len(order))]), sorted(kept_cols)


@pytest.mark.parametrize("rule,thr", [("dynsparse", -1.5), ("dynsparse", -3.0),
                                      ("blasst", math.log(0.2))])
@pytest.mark.parametrize("seed", range(5))
def test_rule_in_diagonal_order_equals_brute_force(rule, thr, seed):
    q, k, v = make_random_qkv(1, 1, 37, 6, 3000 + seed, q_std=2.5, k_std=2.5)
    run = rule_attention(q, k, v, 0.7, rule, thr, 4, 3, key_order="diagonal", order_rows=8)
    n_kt = -(-37 // 3)
    skipped = 0
    for res, (r0, r1) in zip(run.results, run.row_ranges):
        s = 0.7 * (f64(q[0, 0, r0:r1]) @ f64(k[0, 0]).T)
        order = diagonal_first_order(n_kt, (r0 // 8) * 8 // 3)
        skip, kept = brute_force_in_order(s.tolist(), rule, thr, 3, order)
        assert np.array_equal(res.skip, skip)
        assert sorted(res.kept_cols.tolist()) == kept
        assert not res.skip[order[0]]            # the first visited tile is always kept
        skipped += int(skip.sum())
    assert skipped > 0


def test_query_tiles_of_one_block_share_the_order():
    """With 32-row query tiles and 128-row order blocks, the four tiles of a block start
    at the same key tile (the block's first row): with a threshold nothing passes, each
    tile keeps exactly its first visited tile."""
    q, k, v = make_random_qkv(1, 1, 300, 8, 7)
    run = rule_attention(q, k, v, 0.3, "dynsparse", 50.0, 32, 64, key_order="diagonal")
    for (_, _, qi), res in zip(run.tiles, run.results):
        assert np.nonzero(~res.skip)[0].tolist() == [(qi // 4) * 2]


def test_uniform_closed_form_in_visit_order():
    """Uniform logits: DynSparse keeps the first floor(e^-lambda / B_c) + 1 tiles of the
    visit order and skips the rest (the LSE grows as ln(kept keys))."""
    n, tk, lam = 2048, 64, -6.0
    s = np.zeros((3, n))
    v = np.ones((n, 2))
    order = diagonal_first_order(n // tk, 13)
    res = filter_q_tile(s, v, "dynsparse", lam, tk, order=order)
    n_keep = math.floor(math.exp(-lam) / tk) + 1
    assert sorted(np.nonzero(~res.skip)[0].tolist()) == sorted(order[:n_keep])


@pytest.mark.parametrize("recall", [0.9, 0.99])
def test_recall_bound_holds_in_diagonal_order(recall):
    q, k, v, _ = make_video_qkv(1, 2, (2, 16, 32), 6.0, 6.0, True, 5)
    N = q.shape[2]
    run = rule_attention(q, k, v, 1 / math.sqrt(128), "dynsparse",
                         lambda_from_recall(recall, N), 128, 64, key_order="diagonal")
    assert min(float(r.recall.min()) for r in run.results) >= recall
    assert np.mean([r.skip.mean() for r in run.results]) > 0.1


def test_order_does_not_change_dense_attention():
    q, k, v = make_random_qkv(1, 1, 500, 16, 9)
    a = rule_attention(q, k, v, 0.25, "dense", 0.0, 128, 64)
    b = rule_attention(q, k, v, 0.25, "dense", 0.0, 128, 64, key_order="diagonal")
    for ra, rb in zip(a.results, b.results):
        np.testing.assert_allclose(ra.o_sparse, rb.o_sparse, rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(ra.lse_kept, rb.lse_kept, rtol=1e-13)


def test_order_changes_decisions_on_video_inputs():
    """Not vacuous: on video-shaped inputs the diagonal order skips differently (the
    tiles near a query's own position come first and raise its LSE early)."""
    q, k, v, _ = make_video_qkv(1, 2, (2, 16, 32), 4.0, 4.0, True, 6)
    a = rule_attention(q, k, v, 1 / math.sqrt(128), "dynsparse", -8.0, 128, 64)
    b = rule_attention(q, k, v, 1 / math.sqrt(128), "dynsparse", -8.0, 128, 64,
                       key_order="diagonal")
    sa = np.mean([r.skip.mean() for r in a.results])
    sb = np.mean([r.skip.mean() for r in b.results])
    assert sb > sa              # 0.0625 against 0.039 for this seed


def test_bad_orders_are_rejected():
    s = np.zeros((2, 10))
    v = np.ones((10, 2))
    with pytest.raises(ValueError):
        filter_q_tile(s, v, "dynsparse", -1.0, 4, order=[0, 1, 1])
    with pytest.raises(ValueError):
        diagonal_first_order(3, 3)
    with pytest.raises(ValueError):
        rule_attention(np.zeros((1, 1, 4, 8), np.uint16), np.zeros((1, 1, 4, 8), np.uint16),
                       np.zeros((1, 1, 4, 8), np.uint16), 1.0, "dense", 0.0, 4, 2,
                       key_order="backwards")
