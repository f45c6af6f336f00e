"""GPU parity of per-wave skip decisions (tile_q = 32): every 32-row slice of a query tile
decides on its own key tiles, against the oracle run with 32-row query tiles.

The rule is the same (Eq. 5 / Eq. 6, every valid row of the decision unit below the
threshold); only the unit shrinks, so the oracle needs no change: ``rule_attention`` with
``tile_q = 32``.  Decisions are compared teacher-forced as in ``test_gpu_parity.py``.
"""

import math
import sys

import numpy as np
import pytest

import oracle
from synth import WORKLOADS, make_random_qkv, make_video_qkv, workload_inputs

from _parity import (assert_parity, compare, expected_stats_from_mask, run_gpu,
                     sample_tiles, to_device)

pytestmark = pytest.mark.gpu

SCALE = 1.0 / math.sqrt(128)
UNIT = 32


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_16317_amd as dsa

    dsa.lib()
    return torch


def announce(msg):
    print(f"\n[case] {msg}", flush=True)
    sys.stdout.flush()


def upload(q, k, v):
    return to_device(q), to_device(k), to_device(v)


@pytest.fixture(scope="module")
def tiny():
    q, k, v, _ = workload_inputs("tiny")
    return (q, k, v), upload(q, k, v)


@pytest.mark.parametrize("rule,param", [("dense", 0.0), ("dynsparse_recall", 0.95),
                                        ("dynsparse_lambda", -4.0), ("dynsparse_lambda", -6.0),
                                        ("dynsparse_lambda", -8.0), ("blasst", 1e-1),
                                        ("blasst", 1e-2)])
def test_tiny_workload_every_unit(tiny, rule, param):
    (q, k, v), dev = tiny
    announce(f"tiny tile_q=32 rule={rule} param={param}")
    g = run_gpu(*dev, rule, param, SCALE, tile_q=UNIT)
    rep = compare(q, k, v, g, rule, param, SCALE, tile_q=UNIT)
    print(rep, flush=True)
    assert_parity(rep)
    assert (g.stats == expected_stats_from_mask(g.mask, q.shape[2], UNIT)).all()
    assert (g.mask[..., 0] == 0).all()


@pytest.mark.parametrize("B,H,N", [(1, 1, 1), (1, 1, 33), (1, 1, 65), (1, 2, 100),
                                   (2, 3, 129), (2, 1, 777), (1, 1, 2047)])
@pytest.mark.parametrize("rule,param", [("dense", 0.0), ("dynsparse_lambda", -3.0),
                                        ("blasst", 0.05)])
def test_ragged_shapes(B, H, N, rule, param):
    """Partial query tiles leave whole waves without valid rows: they have no mask row and
    no counters, and their neighbours still decide correctly."""
    q, k, v = make_random_qkv(B, H, N, 128, 7000 + 1000 * B + 10 * H + N, q_std=1.5,
                              k_std=1.5)
    announce(f"ragged tile_q=32 B={B} H={H} N={N} rule={rule} param={param}")
    g = run_gpu(*upload(q, k, v), rule, param, SCALE, tile_q=UNIT)
    assert_parity(compare(q, k, v, g, rule, param, SCALE, tile_q=UNIT))
    assert (g.stats == expected_stats_from_mask(g.mask, N, UNIT)).all()
    assert not np.isnan(g.lse).any()


@pytest.fixture(scope="module")
def peaked():
    q, k, v, _ = make_video_qkv(1, 4, (2, 16, 32), 6.0, 6.0, True, 31)
    return (q, k, v), upload(q, k, v)


@pytest.mark.parametrize("rule,param,oracle_sparsity", [
    ("dynsparse_recall", 0.95, 0.4722), ("dynsparse_lambda", -6.0, 0.5171),
    ("dynsparse_lambda", -8.0, 0.4937), ("blasst", 1e-2, 0.5366)])
def test_concentrated_heads(peaked, rule, param, oracle_sparsity):
    """Per-wave units skip more than 128-row tiles on these heads (the oracle's figures:
    0.38 / 0.42 / 0.41 / 0.42 at 128 rows against the values given here at 32 rows)."""
    (q, k, v), dev = peaked
    announce(f"peaked tile_q=32 rule={rule} param={param}")
    g = run_gpu(*dev, rule, param, SCALE, tile_q=UNIT)
    rep = compare(q, k, v, g, rule, param, SCALE, tile_q=UNIT)
    print(rep, flush=True)
    assert_parity(rep)
    assert abs(rep.sparsity - oracle_sparsity) < 0.01
    if rule == "dynsparse_recall":
        # the recall bound of Section 3.1 holds for every row at any decision unit
        for h in range(q.shape[1]):
            s = SCALE * (oracle.bf16_to_f64(q[0, h]) @ oracle.bf16_to_f64(k[0, h]).T)
            mx = s.max(axis=1)
            lse_all = mx + np.log(np.exp(s - mx[:, None]).sum(axis=1))
            assert np.exp(g.lse[0, h].astype(np.float64) - lse_all).min() >= param - 1e-3


def test_dense_output_does_not_depend_on_the_unit(tiny):
    (q, k, v), dev = tiny
    announce("dense tile_q=32 vs tile_q=128")
    a = run_gpu(*dev, "dense", 0.0, SCALE, tile_q=UNIT)
    b = run_gpu(*dev, "dense", 0.0, SCALE)
    assert np.array_equal(a.o, b.o)
    assert np.array_equal(a.lse.view(np.uint32), b.lse.view(np.uint32))
    assert (a.stats[..., 0] == 4 * b.stats[..., 0]).all()
    assert (a.stats[..., 2] == b.stats[..., 2]).all()
    assert not a.mask.any()


@pytest.mark.slow
def test_wan720p_sampled_units():
    w = WORKLOADS["wan720p"]
    announce(f"generate {w.describe()}")
    q, k, v, _ = workload_inputs("wan720p")
    dev = upload(q, k, v)
    tiles = sample_tiles(w.B, w.H, w.N, per_head=3, heads=[(0, 5), (0, 22), (0, 37)], seed=5,
                         tile_q=UNIT)
    for rule, param in (("dynsparse_recall", 0.95), ("dynsparse_lambda", -8.0)):
        announce(f"wan720p tile_q=32 rule={rule} param={param} units={len(tiles)}")
        g = run_gpu(*dev, rule, param, SCALE, tile_q=UNIT)
        rep = compare(q, k, v, g, rule, param, SCALE, tiles=tiles, tile_q=UNIT)
        print(rep, f"full-run unit sparsity={float(g.mask.mean()):.4f}", flush=True)
        assert_parity(rep)
        assert (g.stats == expected_stats_from_mask(g.mask, w.N, UNIT)).all()
