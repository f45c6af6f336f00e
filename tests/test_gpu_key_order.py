"""GPU parity of the diagonal-first key-tile order against the oracle run in the same
order (``rule_attention(..., key_order="diagonal")``), teacher-forced on the GPU's mask.

The kernel maps loop steps to key tiles by a closed form; the oracle sorts tiles by their
distance from the start tile.  Both must visit the same tiles in the same order, which the
decisions (order dependent through the LSE of Eq. 5) and the outputs check.
"""

import math
import sys

import numpy as np
import pytest

from synth import WORKLOADS, make_random_qkv, make_video_qkv, workload_inputs

from _parity import (DeviceRun, RULE_NAMES, TILE_K, assert_parity, expected_stats_from_mask,
                     from_device_bf16, oracle_rule, sample_tiles, to_device)

import oracle

pytestmark = pytest.mark.gpu

SCALE = 1.0 / math.sqrt(128)


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


def run_diag(qd, kd, vd, rule, param, tile_q=128, key_order=1):
    import torch
    import paper_2606_16317_amd as dsa

    B, H, N, d = qd.shape
    n_qt, n_kt = -(-N // tile_q), -(-N // TILE_K)
    o = torch.empty_like(qd)
    stats = torch.full((B * H * 4,), -7, dtype=torch.int64, device="cuda")
    mask = torch.full((B * H * n_qt * n_kt,), 7, dtype=torch.uint8, device="cuda")
    lse = torch.full((B * H * N,), float("nan"), dtype=torch.float32, device="cuda")
    dsa.dsattn_attn_fwd_ex(RULE_NAMES[rule], param, qd, kd, vd, o, scale=SCALE, tile_q=tile_q,
                           stats_out=stats, mask_out=mask, lse_out=lse, key_order=key_order)
    torch.cuda.synchronize()
    return DeviceRun(from_device_bf16(o), mask.cpu().numpy().reshape(B, H, n_qt, n_kt),
                  lse.cpu().numpy().reshape(B, H, N), stats.cpu().numpy().reshape(B, H, 4))


def compare_diag(q, k, v, g, rule, param, tile_q=128, tiles=None):
    """Teacher-forced comparison with the oracle in diagonal-first order; returns
    (mismatches, worst mismatch margin, max abs err, rel-L2, max LSE err, sparsity)."""
    N = q.shape[2]
    name, thr = oracle_rule(rule, param, N)
    run = oracle.rule_attention(q, k, v, SCALE, name, thr, tile_q, TILE_K, tiles=tiles,
                                forced_mask=g.mask, key_order="diagonal")
    mism, worst, max_abs, lse_err, num, den = 0, 0.0, 0.0, 0.0, 0.0, 0.0
    for (b, h, qi), res, (r0, r1) in zip(run.tiles, run.results, run.row_ranges):
        bad = (res.margin < 0) != res.skip
        mism += int(bad.sum())
        if bad.any():
            worst = max(worst, float(np.abs(res.margin[bad]).max()))
        go = oracle.bf16_to_f64(g.o[b, h, r0:r1])
        max_abs = max(max_abs, float(np.abs(go - res.o_sparse).max()))
        num += float(((go - res.o_sparse) ** 2).sum())
        den += float((res.o_sparse ** 2).sum())
        lse_err = max(lse_err, float(np.abs(g.lse[b, h, r0:r1] - res.lse_kept).max()))
        # the first visited tile (the block's own position) is always kept
        start = (r0 // 128) * 128 // TILE_K
        assert not res.skip[start]
    sp = float(np.mean([r.skip.mean() for r in run.results]))
    return mism, worst, max_abs, math.sqrt(num / den), lse_err, sp


def check(rep):
    mism, worst, max_abs, rel, lse_err, _ = rep
    assert mism == 0 or worst < 1e-3, rep
    assert max_abs <= 2e-2 and rel <= 1e-2 and lse_err <= 2e-3, rep


def upload(q, k, v):
    return to_device(q), to_device(k), to_device(v)


@pytest.fixture(scope="module")
def peaked():
    q, k, v, _ = make_video_qkv(1, 4, (2, 16, 32), 6.0, 6.0, True, 31)
    return (q, k, v), upload(q, k, v)


@pytest.mark.parametrize("tile_q", [128, 32])
@pytest.mark.parametrize("rule,param", [("dense", 0.0), ("dynsparse_recall", 0.95),
                                        ("dynsparse_lambda", -6.0), ("dynsparse_lambda", -9.0),
                                        ("blasst", 1e-2)])
def test_peaked_heads_every_tile(peaked, rule, param, tile_q):
    (q, k, v), dev = peaked
    announce(f"diagonal order peaked tile_q={tile_q} rule={rule} param={param}")
    g = run_diag(*dev, rule, param, tile_q)
    rep = compare_diag(q, k, v, g, rule, param, tile_q)
    print(rep, flush=True)
    check(rep)
    assert (g.stats == expected_stats_from_mask(g.mask, q.shape[2], tile_q)).all()
    if rule != "dense":
        assert rep[5] > 0.1


@pytest.mark.parametrize("B,H,N", [(1, 1, 1), (1, 1, 65), (1, 2, 200), (2, 1, 777),
                                   (1, 1, 2047)])
@pytest.mark.parametrize("rule,param", [("dynsparse_lambda", -3.0), ("blasst", 0.05)])
def test_ragged_shapes(B, H, N, rule, param):
    """Ragged key tiles sit in the middle of the visit order here, not at its end."""
    q, k, v = make_random_qkv(B, H, N, 128, 9000 + N + B, q_std=1.5, k_std=1.5)
    announce(f"diagonal order ragged B={B} H={H} N={N} rule={rule} param={param}")
    g = run_diag(*upload(q, k, v), rule, param)
    check(compare_diag(q, k, v, g, rule, param))
    assert (g.stats == expected_stats_from_mask(g.mask, N)).all()


def test_dense_is_the_same_attention_in_either_order(peaked):
    (q, k, v), dev = peaked
    a = run_diag(*dev, "dense", 0.0, key_order=0)
    b = run_diag(*dev, "dense", 0.0, key_order=1)
    oa = oracle.bf16_to_f64(a.o)
    ob = oracle.bf16_to_f64(b.o)
    assert np.abs(oa - ob).max() < 2e-2
    assert np.abs(a.lse - b.lse).max() < 1e-4


def test_ascending_order_is_the_default_path(peaked):
    """key_order = 0 through _ex is bit-identical to the named entry point."""
    import torch
    import paper_2606_16317_amd as dsa

    (q, k, v), dev = peaked
    a = run_diag(*dev, "dynsparse_lambda", -6.0, key_order=0)
    o = dsa.dynsparse_attn_fwd_lambda(*dev, scale=SCALE, lam=-6.0)
    torch.cuda.synchronize()
    assert np.array_equal(a.o, from_device_bf16(o))


@pytest.mark.slow
def test_wan720p_sampled_diagonal():
    w = WORKLOADS["wan720p"]
    announce(f"generate {w.describe()}")
    q, k, v, _ = workload_inputs("wan720p")
    dev = upload(q, k, v)
    tiles = sample_tiles(w.B, w.H, w.N, per_head=3, heads=[(0, 3), (0, 29)], seed=8)
    for rule, param in (("dynsparse_recall", 0.95), ("dynsparse_lambda", -8.0)):
        announce(f"wan720p diagonal order rule={rule} param={param}")
        g = run_diag(*dev, rule, param)
        rep = compare_diag(q, k, v, g, rule, param, tiles=tiles)
        print(rep, f"full-run sparsity={float(g.mask.mean()):.4f}", flush=True)
        check(rep)
        assert (g.stats == expected_stats_from_mask(g.mask, w.N)).all()

