"""Pins of the fp64 oracle to what the paper and plain mathematics fix (CPU only).

Each test checks the oracle against something other than itself: a naive triple loop, a
from-scratch brute force of the tile rule, closed forms of constructed inputs, the
recall theorem of Section 3.1, torch's own attention and the error figures printed in
Section 2.3.
"""

import json
import math
import os

import numpy as np
import pytest

import oracle
from oracle import filter_q_tile, lambda_from_recall, log_threshold_blasst, rule_attention
from synth import bf16_bits, make_random_qkv, make_video_qkv

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------------------------------
# helpers written independently of the oracle (plain Python floats)

def naive_attention(q, k, v, scale):
    """Triple-loop softmax attention with math.fsum; q, k, v are lists of float rows."""
    out = []
    for qi in q:
        s = [scale * math.fsum(a * b for a, b in zip(qi, kj)) for kj in k]
        mx = max(s)
        w = [math.exp(x - mx) for x in s]
        z = math.fsum(w)
        out.append([math.fsum(w[j] * v[j][c] for j in range(len(k))) / z
                    for c in range(len(v[0]))])
    return np.array(out)


def brute_force_rule(s, rule, thr, tile_k):
    """Recompute every tile decision from scratch: the LSE (or max) of the kept keys
    before the tile is rebuilt from the full logit matrix and the kept set each time."""
    rows, n = len(s), len(s[0])
    n_kt = -(-n // tile_k)
    kept_cols, skip = [], []
    for j in range(n_kt):
        cols = range(j * tile_k, min(n, (j + 1) * tile_k))
        decide_keep = False
        for r in range(rows):
            m_hat = max(s[r][c] for c in cols)
            if not kept_cols:
                ref = -math.inf
            elif rule == "dynsparse":
                ref = math.log(math.fsum(math.exp(s[r][c]) for c in kept_cols))
            else:
                ref = max(s[r][c] for c in kept_cols)
            t = m_hat - ref
            if rule == "dense" or not (t < thr):
                decide_keep = True
        skip.append(not decide_keep)
        if decide_keep:
            kept_cols.extend(cols)
    return np.array(skip), kept_cols


def sparse_output_from_scratch(s, v, kept_cols):
    """O[r] = sum_{c kept} softmax-over-kept(S[r])[c] V[c] with plain Python sums."""
    out = []
    for r in range(s.shape[0]):
        w = [math.exp(s[r][c]) for c in kept_cols]
        z = math.fsum(w)
        out.append([math.fsum(w[i] * v[c][d] for i, c in enumerate(kept_cols)) / z
                    for d in range(v.shape[1])])
    return np.array(out)


def f64(bits):
    return oracle.bf16_to_f64(bits)


# ---------------------------------------------------------------------------------------
# P1: the dense special case is textbook softmax attention

@pytest.mark.parametrize("n,d,seed", [(1, 4, 0), (7, 8, 1), (33, 16, 2), (64, 8, 3)])
def test_dense_matches_triple_loop(n, d, seed):
    q, k, v = make_random_qkv(1, 1, n, d, seed)
    q, k, v = f64(q[0, 0]), f64(k[0, 0]), f64(v[0, 0])
    scale = 1.0 / math.sqrt(d)
    ref = naive_attention(q.tolist(), k.tolist(), v.tolist(), scale)
    np.testing.assert_allclose(oracle.dense_attention(q, k, v, scale), ref, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("rule,param", [("dense", 0.0), ("dynsparse", -math.inf),
                                        ("blasst", -math.inf)])
def test_rules_at_infinite_threshold_are_dense(rule, param):
    q, k, v = make_random_qkv(2, 2, 45, 16, 7, q_std=3.0, k_std=3.0)
    run = rule_attention(q, k, v, 0.25, rule, param, 8, 4)
    for (b, h, qi), res, (r0, r1) in zip(run.tiles, run.results, run.row_ranges):
        assert not res.skip.any()
        ref = naive_attention(f64(q[b, h, r0:r1]).tolist(), f64(k[b, h]).tolist(),
                              f64(v[b, h]).tolist(), 0.25)
        np.testing.assert_allclose(res.o_sparse, ref, rtol=1e-11, atol=1e-12)
        np.testing.assert_allclose(res.o_dense, ref, rtol=1e-11, atol=1e-12)
        np.testing.assert_allclose(res.recall, 1.0, rtol=0, atol=1e-12)


def test_dense_matches_torch_sdpa_fp64():
    torch = pytest.importorskip("torch")
    q, k, v = make_random_qkv(1, 3, 200, 128, 11, q_std=2.0, k_std=2.0)
    scale = 1.0 / math.sqrt(128)
    run = rule_attention(q, k, v, scale, "dense", 0.0, 128, 64)
    tq = torch.from_numpy(f64(q))
    tk = torch.from_numpy(f64(k))
    tv = torch.from_numpy(f64(v))
    ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, scale=scale).numpy()
    for (b, h, qi), res, (r0, r1) in zip(run.tiles, run.results, run.row_ranges):
        np.testing.assert_allclose(res.o_dense, ref[b, h, r0:r1], rtol=1e-10, atol=1e-12)
        np.testing.assert_allclose(res.o_sparse, ref[b, h, r0:r1], rtol=1e-10, atol=1e-12)


def test_bf16_upcast_matches_torch():
    torch = pytest.importorskip("torch")
    bits = np.arange(0, 65536, dtype=np.uint32).astype(np.uint16)
    ours = oracle.bf16_to_f64(bits)
    ref = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).double().numpy()
    same = (ours == ref) | (np.isnan(ours) & np.isnan(ref))
    assert same.all()


# ---------------------------------------------------------------------------------------
# P2: brute force on tiny inputs (decisions rebuilt from scratch at every tile)

@pytest.mark.parametrize("rule", ["dynsparse", "blasst"])
@pytest.mark.parametrize("tile_q,tile_k", [(4, 2), (8, 4), (3, 5)])
@pytest.mark.parametrize("seed", range(6))
def test_streaming_rule_equals_brute_force(rule, tile_q, tile_k, seed):
    rng = np.random.default_rng(100 + seed)
    n = int(rng.integers(9, 41))
    d = 6
    # spread of logits wide enough that tiles do get skipped
    q, k, v = make_random_qkv(1, 1, n, d, 1000 + seed, q_std=2.5, k_std=2.5)
    thr = {"dynsparse": [-1.0, -2.5, -4.0], "blasst": [math.log(0.3), math.log(0.05)]}[rule]
    for th in thr:
        run = rule_attention(q, k, v, 0.7, rule, th, tile_q, tile_k)
        for res, (r0, r1) in zip(run.results, run.row_ranges):
            s = 0.7 * (f64(q[0, 0, r0:r1]) @ f64(k[0, 0]).T)
            skip, kept = brute_force_rule(s.tolist(), rule, th, tile_k)
            # brute force uses exp() of raw logits: fine for |S| here (< 40)
            assert np.array_equal(res.skip, skip), (rule, th, res.skip, skip)
            assert list(res.kept_cols) == kept
            ref = sparse_output_from_scratch(s, f64(v[0, 0]), kept)
            np.testing.assert_allclose(res.o_sparse, ref, rtol=1e-11, atol=1e-12)
            # margins are well defined: skip iff margin < 0
            assert np.array_equal(res.skip, res.margin < 0)


def test_brute_force_actually_skips():
    """The brute-force comparison above is not vacuous: many tiles are skipped."""
    skipped = total = 0
    for seed in range(6):
        q, k, v = make_random_qkv(1, 1, 40, 6, 1000 + seed, q_std=2.5, k_std=2.5)
        run = rule_attention(q, k, v, 0.7, "dynsparse", -2.5, 4, 2)
        for res in run.results:
            skipped += int(res.skip.sum())
            total += res.skip.size
    assert skipped > 0.1 * total


# ---------------------------------------------------------------------------------------
# P2b: exact ties.  Section 3.1 skips a tile only when its metric is strictly below the
# threshold, so t == threshold keeps it.  Every case below is built from values that are
# exact in binary floating point (logits 0, -0.5, -0.75; a single zero logit has LSE 0;
# the running max of zero logits is 0), so the tie is exact and a "<=" comparison would
# give a different answer in each one.

def _next_up(x):
    return float(np.nextafter(x, math.inf))


def _next_down(x):
    return float(np.nextafter(x, -math.inf))


def test_tie_keeps_tile_dynsparse_single_keys():
    """Single-key tiles, two rows.  After tile 0 (logit 0) the LSE of both rows is 0, so
    tile 1 has t = (-0.5, -0.75) and the unit's metric is max_r t = -0.5."""
    s = np.array([[0.0, -0.5], [0.0, -0.75]])
    v = np.array([[1.0, 0.0], [0.0, 1.0]])
    at = filter_q_tile(s, v, "dynsparse", -0.5, 1)
    assert list(at.skip) == [False, False]           # t == lambda: kept
    assert at.margin[1] == 0.0
    assert list(filter_q_tile(s, v, "dynsparse", _next_up(-0.5), 1).skip) == [False, True]
    assert list(filter_q_tile(s, v, "dynsparse", _next_down(-0.5), 1).skip) == [False, False]
    # the kept tile enters the LSE: row 0 keeps e^0 + e^-0.5 of its mass
    np.testing.assert_allclose(at.lse_kept[0], math.log(1.0 + math.exp(-0.5)), rtol=1e-15)


def test_tie_keeps_tile_blasst_single_keys():
    """BLASST on the same logits: the running max after tile 0 is 0, so tile 1 has
    t = (-0.5, -0.75); ln(tau) = -0.5 is a tie and keeps it."""
    s = np.array([[0.0, -0.5], [0.0, -0.75]])
    v = np.eye(2)
    assert list(filter_q_tile(s, v, "blasst", -0.5, 1).skip) == [False, False]
    assert list(filter_q_tile(s, v, "blasst", _next_up(-0.5), 1).skip) == [False, True]


def test_tie_keeps_tile_uniform_dynsparse_full_pipeline():
    """Q = 0 from bf16 inputs, single-key tiles, lambda = 0: tile 1 has t = 0 - ln(1) = 0,
    a tie, and is kept; from tile 2 on t = -ln 2 < 0.  So exactly tiles 0 and 1 are kept
    (a strict "<" is the only comparison that keeps two), the recall is 2/N and the output
    is the mean of the first two value rows."""
    n = 8
    q = np.zeros((1, 1, n, 4), np.uint16)          # bf16 +0
    k = bf16_bits(np.arange(n * 4, dtype=np.float32).reshape(1, 1, n, 4) / 7)
    v = bf16_bits(np.random.default_rng(3).standard_normal((1, 1, n, 4)).astype(np.float32))
    run = rule_attention(q, k, v, 1.0, "dynsparse", 0.0, n, 1)
    res = run.results[0]
    assert list(np.nonzero(~res.skip)[0]) == [0, 1]
    assert res.margin[1] == 0.0
    np.testing.assert_allclose(res.recall, 2.0 / n, rtol=1e-15)
    vv = f64(v[0, 0])
    np.testing.assert_allclose(res.o_sparse, np.tile((vv[0] + vv[1]) / 2, (n, 1)), rtol=1e-15)


def test_tie_keeps_every_tile_blasst_tau_one_full_pipeline():
    """Uniform logits under BLASST with tau = 1: every tile has t = 0 - 0 = ln(1), a tie,
    so nothing is skipped and the output is dense attention (the mean of V)."""
    n = 96
    q = np.zeros((1, 1, n, 8), np.uint16)
    k = bf16_bits(np.random.default_rng(4).standard_normal((1, 1, n, 8)).astype(np.float32))
    v = bf16_bits(np.random.default_rng(5).standard_normal((1, 1, n, 8)).astype(np.float32))
    run = rule_attention(q, k, v, 0.5, "blasst", log_threshold_blasst(1.0), 32, 16)
    assert all(not r.skip.any() for r in run.results)
    for r in run.results:
        assert r.margin[0] == math.inf and (r.margin[1:] == 0.0).all()
    mean = f64(v[0, 0]).mean(axis=0)
    for r in run.results:
        np.testing.assert_allclose(r.o_sparse, np.tile(mean, (r.o_sparse.shape[0], 1)),
                                   rtol=1e-13, atol=1e-15)


@pytest.mark.parametrize("seed", range(4))
def test_blasst_integer_logit_ties_match_brute_force(seed):
    """Integer logits and integer thresholds: BLASST's metric m_hat - m is an integer, so
    exact ties occur throughout; the streaming oracle equals the from-scratch brute force
    (which keeps a tile unless t < threshold) and ties do occur."""
    rng = np.random.default_rng(200 + seed)
    s = rng.integers(-4, 1, size=(3, 24)).astype(np.float64)
    v = rng.standard_normal((24, 3))
    ties = 0
    for thr in (-1.0, -2.0, -3.0):
        for tk in (1, 2, 3):
            res = filter_q_tile(s, v, "blasst", thr, tk)
            skip, kept = brute_force_rule(s.tolist(), "blasst", thr, tk)
            assert np.array_equal(res.skip, skip)
            assert list(res.kept_cols) == kept
            ties += int((res.margin == 0.0).sum())
    assert ties > 0


# ---------------------------------------------------------------------------------------
# P3/P4: the recall theorem of Section 3.1

def _concentrated_inputs(a, seed, grid=(2, 16, 32)):
    return make_video_qkv(1, 2, grid, a, a, True, seed)


@pytest.mark.parametrize("a,seed", [(6.0, 0), (8.0, 1)])
@pytest.mark.parametrize("recall", [0.9, 0.95, 0.99])
def test_recall_bound_holds_per_row(a, seed, recall):
    q, k, v, _ = _concentrated_inputs(a, seed)
    N = q.shape[2]
    lam = lambda_from_recall(recall, N)
    run = rule_attention(q, k, v, 1 / math.sqrt(128), "dynsparse", lam, 128, 64)
    n_skipped = 0
    for res in run.results:
        rows = res.o_sparse.shape[0]
        nsk_tok = sum(min(N, (j + 1) * 64) - j * 64 for j in np.nonzero(res.skip)[0])
        n_skipped += int(res.skip.sum())
        lost = 1.0 - res.recall
        assert (res.recall >= recall - 1e-12).all()
        assert (lost <= nsk_tok * math.exp(lam) + 1e-12).all()
        assert rows > 0
    assert n_skipped > 0, "inputs too flat: the bound was not exercised"


@pytest.mark.parametrize("lam", [-3.0, -6.0, -9.0])
def test_pointwise_bound_on_skipped_tokens(lam):
    """Every skipped token's dense probability is at most e^t of its row (and < e^lambda)."""
    q, k, v, _ = _concentrated_inputs(6.0, 5)
    scale = 1 / math.sqrt(128)
    run = rule_attention(q, k, v, scale, "dynsparse", lam, 128, 64, tiles=[(0, 0, 3), (0, 1, 7)])
    checked = 0
    for (b, h, qi), res, (r0, r1) in zip(run.tiles, run.results, run.row_ranges):
        s = scale * (f64(q[b, h, r0:r1]) @ f64(k[b, h]).T)
        p = np.exp(s - res.lse_all[:, None])
        for j in np.nonzero(res.skip)[0]:
            blk = p[:, j * 64:(j + 1) * 64]
            bound = np.exp(res.tmetric[:, j])[:, None]
            assert (blk <= bound * (1 + 1e-12)).all()
            assert (blk < math.exp(lam)).all()
            checked += 1
    assert checked > 0


# ---------------------------------------------------------------------------------------
# P5: tile 0 is never skipped

@pytest.mark.parametrize("rule,thr", [("dynsparse", 5.0), ("dynsparse", -1.0), ("blasst", 0.0),
                                      ("blasst", -0.5)])
def test_first_tile_always_kept(rule, thr):
    q, k, v = make_random_qkv(1, 2, 100, 8, 3, q_std=3.0, k_std=3.0)
    run = rule_attention(q, k, v, 1.0, rule, thr, 16, 8)
    for res in run.results:
        assert not res.skip[0]


# ---------------------------------------------------------------------------------------
# P6: monotonicity

def test_blasst_skip_set_monotone_in_tau():
    q, k, v, _ = _concentrated_inputs(2.5, 9)
    scale = 1 / math.sqrt(128)
    prev = None
    for tau in [1e-4, 1e-3, 1e-2, 1e-1, 0.5]:
        run = rule_attention(q, k, v, scale, "blasst", log_threshold_blasst(tau), 128, 64)
        cur = np.stack([r.skip for r in run.results])
        if prev is not None:
            assert (cur | ~prev).all() and (cur >= prev).all()
        prev = cur
    assert prev.any()


def test_dynsparse_not_set_monotone_counterexample():
    """Single-key tiles with logits (0, -0.15, 0): lambda=-0.2 skips the third tile,
    lambda=-0.1 skips the second; neither skip set contains the other."""
    s = np.array([[0.0, -0.15, 0.0]])
    v = np.eye(3)
    a = filter_q_tile(s, v, "dynsparse", -0.2, 1)
    b = filter_q_tile(s, v, "dynsparse", -0.1, 1)
    assert list(a.skip) == [False, False, True]
    assert list(b.skip) == [False, True, False]


def test_dynsparse_sparsity_monotone_on_sweep():
    q, k, v, _ = _concentrated_inputs(2.5, 12)
    scale = 1 / math.sqrt(128)
    prev = -1.0
    for lam in [-12.0, -10.0, -8.0, -6.0, -4.0, -2.0]:
        run = rule_attention(q, k, v, scale, "dynsparse", lam, 128, 64)
        sp = np.mean([r.skip.mean() for r in run.results])
        assert sp >= prev
        prev = sp
    assert prev > 0.3


# ---------------------------------------------------------------------------------------
# P7: invariances

def test_row_permutation_and_value_scaling_invariance():
    q, k, v, _ = _concentrated_inputs(3.0, 21)
    scale = 1 / math.sqrt(128)
    base = rule_attention(q, k, v, scale, "dynsparse", -6.0, 128, 64, tiles=[(0, 1, 5)])
    perm = np.random.default_rng(0).permutation(128)
    qp = q.copy()
    qp[0, 1, 640:768] = q[0, 1, 640:768][perm]
    permd = rule_attention(qp, k, v, scale, "dynsparse", -6.0, 128, 64, tiles=[(0, 1, 5)])
    assert np.array_equal(base.results[0].skip, permd.results[0].skip)
    np.testing.assert_allclose(permd.results[0].o_sparse, base.results[0].o_sparse[perm],
                               rtol=1e-12, atol=1e-14)
    # V * 2 is exact in bf16: outputs double, decisions unchanged
    v2 = bf16_bits(2.0 * oracle.bf16_to_f64(v).astype(np.float32))
    sc = rule_attention(q, k, v2, scale, "dynsparse", -6.0, 128, 64, tiles=[(0, 1, 5)])
    assert np.array_equal(base.results[0].skip, sc.results[0].skip)
    np.testing.assert_allclose(sc.results[0].o_sparse, 2 * base.results[0].o_sparse,
                               rtol=1e-12, atol=1e-14)


def test_key_permutation_inside_tiles_invariance():
    q, k, v, _ = _concentrated_inputs(3.0, 22)
    scale = 1 / math.sqrt(128)
    N = q.shape[2]
    perm = np.arange(N)
    rng = np.random.default_rng(1)
    for j in range(N // 64):
        perm[j * 64:(j + 1) * 64] = j * 64 + rng.permutation(64)
    base = rule_attention(q, k, v, scale, "dynsparse", -7.0, 128, 64, tiles=[(0, 0, 2)])
    pk = rule_attention(q, k[:, :, perm], v[:, :, perm], scale, "dynsparse", -7.0, 128, 64,
                        tiles=[(0, 0, 2)])
    assert np.array_equal(base.results[0].skip, pk.results[0].skip)
    np.testing.assert_allclose(pk.results[0].o_sparse, base.results[0].o_sparse, rtol=1e-10,
                               atol=1e-13)


# ---------------------------------------------------------------------------------------
# P8: uniform attention closed form

@pytest.mark.parametrize("lam,tile_k,n", [(-6.0, 64, 2048), (-4.0, 16, 1000), (-8.5, 64, 4000)])
def test_uniform_closed_form(lam, tile_k, n):
    s = np.zeros((5, n))
    v = oracle.bf16_to_f64(make_random_qkv(1, 1, n, 8, 4)[2][0, 0])
    res = filter_q_tile(s, v, "dynsparse", lam, tile_k)
    n_kt = -(-n // tile_k)
    # tile j is kept iff ln(j * tile_k) <= -lambda, i.e. floor(e^-lambda / tile_k) + 1 tiles
    n_keep = min(n_kt, math.floor(math.exp(-lam) / tile_k) + 1)
    assert list(np.nonzero(~res.skip)[0]) == list(range(n_keep))
    kept_keys = min(n, n_keep * tile_k)
    np.testing.assert_allclose(res.recall, kept_keys / n, rtol=1e-12)
    np.testing.assert_allclose(res.o_sparse, np.tile(v[:kept_keys].mean(axis=0), (5, 1)),
                               rtol=1e-10, atol=1e-13)
    blasst = filter_q_tile(s, v, "blasst", math.log(0.999), tile_k)
    assert not blasst.skip.any()


def test_uniform_under_recall_mapping_skips_nothing():
    n = 3000
    s = np.zeros((2, n))
    v = np.ones((n, 2))
    res = filter_q_tile(s, v, "dynsparse", lambda_from_recall(0.95, n), 64)
    assert not res.skip.any()


# ---------------------------------------------------------------------------------------
# P9: winner closed form (order dependence)

@pytest.mark.parametrize("w_tile,expect_kept", [(1, [0, 1]), (31, [0, 1, 2, 3, 4, 5, 6, 31])])
def test_winner_closed_form(w_tile, expect_kept):
    n, tk, sw, lam = 2048, 64, 20.0, -6.0
    s = np.zeros((3, n))
    w = w_tile * tk + 17
    s[:, w] = sw
    v = oracle.bf16_to_f64(make_random_qkv(1, 1, n, 4, 8)[2][0, 0])
    res = filter_q_tile(s, v, "dynsparse", lam, tk)
    assert list(np.nonzero(~res.skip)[0]) == expect_kept
    kept = np.concatenate([np.arange(j * tk, (j + 1) * tk) for j in expect_kept])
    z_kept = math.exp(sw) + len(kept) - 1
    np.testing.assert_allclose(res.lse_kept, math.log(z_kept), rtol=1e-13)
    np.testing.assert_allclose(res.recall, z_kept / (math.exp(sw) + n - 1), rtol=1e-12)
    wts = np.ones(len(kept))
    wts[kept == w] = math.exp(sw)
    np.testing.assert_allclose(res.o_sparse[0], (wts @ v[kept]) / z_kept, rtol=1e-10)
    # BLASST on the early winner: the running max jumps to s_w, later tiles have t = -s_w
    bl = filter_q_tile(s, v, "blasst", math.log(1e-2), tk)
    if w_tile == 1:
        assert list(np.nonzero(~bl.skip)[0]) == [0, 1]
    else:
        assert not bl.skip.any()


# ---------------------------------------------------------------------------------------
# P10: uniform-attention error figures printed in Section 2.3

def _std_closed_form(n, k):
    return (1.0 / math.sqrt(k)) * math.sqrt((n - k) / (n - 1))


def test_paper_uniform_std_figures():
    g = json.load(open(os.path.join(GOLDEN, "uniform_std_error.json")))
    assert math.ceil(g["N_tokens"] / g["block"]) == g["N_units"]
    for case in g["cases"]:
        k = case["kept_fraction"] * g["N_units"]
        pct = 100 * _std_closed_form(g["N_units"], k)
        assert round(pct, 1) == case["std_over_delta_percent"]


@pytest.mark.parametrize("kept_fraction", [0.8, 0.95])
def test_oracle_uniform_error_matches_paper_std(kept_fraction):
    """Uniform logits, single-key tiles: choose lambda so DynSparse keeps K of the 214
    units; the spread of (sparse - dense) over many independent V draws matches the
    closed form of Section 2.3 (unit-variance V)."""
    g = json.load(open(os.path.join(GOLDEN, "uniform_std_error.json")))
    n = g["N_units"]
    k_keep = round(kept_fraction * n)
    lam = -math.log(k_keep - 0.5)  # keeps tiles 0..k_keep-1, skips the rest
    rng = np.random.default_rng(77)
    errs = []
    s = np.zeros((1, n))
    for _ in range(96):
        v = rng.standard_normal((n, 128))
        res = filter_q_tile(s, v, "dynsparse", lam, 1)
        assert int((~res.skip).sum()) == k_keep
        errs.append(res.o_sparse[0] - res.o_dense[0])
    e = np.concatenate(errs)
    expect = math.sqrt(1.0 / k_keep - 1.0 / n)     # iid unit-variance V
    assert abs(e.std() / expect - 1) < 0.05
    assert abs(_std_closed_form(n, k_keep) / expect - 1) < 0.01


# ---------------------------------------------------------------------------------------
# lambda mapping and statistics bookkeeping

def test_lambda_mapping():
    assert lambda_from_recall(1.0, 10) == -math.inf
    assert lambda_from_recall(0.95, 2048) == pytest.approx(math.log(0.05) - math.log(2048))
    assert lambda_from_recall(0.95, 75600) == pytest.approx(-14.2290, abs=1e-4)
    with pytest.raises(ValueError):
        lambda_from_recall(0.0, 10)
    with pytest.raises(ValueError):
        lambda_from_recall(1.01, 10)
    assert log_threshold_blasst(0.0) == -math.inf
    assert log_threshold_blasst(1e-2) == pytest.approx(-4.60517, abs=1e-5)


def test_stats_counts_ragged():
    q, k, v = make_random_qkv(1, 2, 150, 8, 5, q_std=3, k_std=3)
    run = rule_attention(q, k, v, 1.0, "dynsparse", -2.0, 64, 32)
    st = run.stats(1, 2)
    n_qt, n_kt = 3, 5
    assert (st[0, :, 0] == n_qt * n_kt).all()
    assert (st[0, :, 2] == 150 * 150).all()
    for h in range(2):
        sk = [r for (b, hh, _), r in zip(run.tiles, run.results) if hh == h]
        assert st[0, h, 1] == sum(int(r.skip.sum()) for r in sk)
    assert (st[0, :, 3] <= st[0, :, 2]).all()


def test_forced_mask_follows_given_decisions():
    q, k, v = make_random_qkv(1, 1, 96, 8, 6, q_std=3, k_std=3)
    own = rule_attention(q, k, v, 1.0, "dynsparse", -3.0, 32, 16)
    forced = np.zeros((1, 1, 3, 6), dtype=np.uint8)
    forced[0, 0, :, 3] = 1
    run = rule_attention(q, k, v, 1.0, "dynsparse", -3.0, 32, 16, forced_mask=forced)
    for res, o in zip(run.results, own.results):
        assert list(res.skip) == [False, False, False, True, False, False]
        # margins are the oracle's own up to the first divergence
        first = np.argmax(res.skip != o.skip) if (res.skip != o.skip).any() else 6
        np.testing.assert_array_equal(res.margin[:first + 1], o.margin[:first + 1])
