"""GPU tests of mask reuse (DSATTN_RULE_MASK): an earlier call's skip mask applied as
given, visiting only the key tiles some row of the workgroup keeps.

* Reusing the mask a rule call wrote must reproduce that call bit for bit (output, LSE,
  counters): both visit the same kept tiles in the same order with the same arithmetic.
* Arbitrary masks (units that keep nothing, masks that skip the first tile) are compared
  with the oracle's output for that kept set (``rule_attention`` with ``forced_mask``,
  whose decisions then do not matter).
"""

import math
import sys

import numpy as np
import pytest

import oracle
from synth import WORKLOADS, make_random_qkv, make_video_qkv, workload_inputs

from _parity import (DeviceRun, RULE_NAMES, TILE_K, expected_stats_from_mask, from_device_bf16,
                     run_gpu, to_device)

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


def upload(q, k, v):
    return to_device(q), to_device(k), to_device(v)


def run_reuse(qd, kd, vd, mask, tile_q, tile_k=TILE_K):
    import torch
    import paper_2606_16317_amd as dsa

    B, H, N, d = qd.shape
    n_qu, n_kt = -(-N // tile_q), -(-N // tile_k)
    o = torch.empty_like(qd)
    stats = torch.full((B * H * 4,), -7, dtype=torch.int64, device="cuda")
    mask_out = torch.full((B * H * n_qu * n_kt,), 7, dtype=torch.uint8, device="cuda")
    lse = torch.full((B * H * N,), float("nan"), dtype=torch.float32, device="cuda")
    mask_in = torch.from_numpy(np.ascontiguousarray(mask, dtype=np.uint8).reshape(-1)).cuda()
    dsa.dsattn_attn_fwd_ex(dsa.RULE_MASK, 0.0, qd, kd, vd, o, scale=SCALE, tile_q=tile_q,
                           tile_k=tile_k, stats_out=stats, mask_out=mask_out, lse_out=lse,
                           mask_in=mask_in)
    torch.cuda.synchronize()
    return DeviceRun(from_device_bf16(o), mask_out.cpu().numpy().reshape(B, H, n_qu, n_kt),
                  lse.cpu().numpy().reshape(B, H, N), stats.cpu().numpy().reshape(B, H, 4))


@pytest.fixture(scope="module")
def peaked():
    q, k, v, _ = make_video_qkv(1, 4, (2, 16, 32), 6.0, 6.0, True, 31)
    return (q, k, v), upload(q, k, v)


@pytest.mark.parametrize("tile_q", [128, 32])
@pytest.mark.parametrize("rule,param", [("dynsparse_lambda", -6.0), ("dynsparse_recall", 0.95),
                                        ("blasst", 1e-2), ("dense", 0.0)])
def test_reusing_a_rule_mask_is_bit_identical(peaked, rule, param, tile_q):
    (q, k, v), dev = peaked
    announce(f"mask reuse of {rule}={param} tile_q={tile_q}")
    ref = run_gpu(*dev, rule, param, SCALE, tile_q=tile_q)
    got = run_reuse(*dev, ref.mask, tile_q)
    assert np.array_equal(got.o, ref.o)
    assert np.array_equal(got.lse.view(np.uint32), ref.lse.view(np.uint32))
    assert np.array_equal(got.stats, ref.stats)
    assert np.array_equal(got.mask, ref.mask)
    if rule != "dense":
        assert ref.mask.mean() > 0.1


def compare_forced(q, k, v, g, tile_q, tile_k=TILE_K):
    """Output and LSE of a reuse run against the oracle's for the same kept set."""
    B, H, N, d = q.shape
    run = oracle.rule_attention(q, k, v, SCALE, "dense", 0.0, tile_q, tile_k,
                                forced_mask=g.mask)
    max_abs, num, den, lse_err = 0.0, 0.0, 0.0, 0.0
    for (b, h, _), res, (r0, r1) in zip(run.tiles, run.results, run.row_ranges):
        go = oracle.bf16_to_f64(g.o[b, h, r0:r1])
        max_abs = max(max_abs, float(np.abs(go - res.o_sparse).max()))
        num += float(((go - res.o_sparse) ** 2).sum())
        den += float((res.o_sparse ** 2).sum())
        gl, ol = g.lse[b, h, r0:r1].astype(np.float64), res.lse_kept
        assert np.array_equal(np.isinf(gl), np.isinf(ol))          # units that keep nothing
        fin = ~np.isinf(ol)
        if fin.any():
            lse_err = max(lse_err, float(np.abs(gl[fin] - ol[fin]).max()))
    assert max_abs <= 2e-2 and lse_err <= 2e-3
    assert den == 0.0 or math.sqrt(num / den) <= 1e-2


@pytest.mark.parametrize("B,H,N,tile_q", [(1, 2, 2048, 128), (1, 2, 2048, 32), (2, 1, 777, 128),
                                          (1, 3, 1000, 32), (1, 1, 65, 32), (1, 1, 1, 128)])
@pytest.mark.parametrize("density", [0.1, 0.5, 0.95])
def test_arbitrary_masks_match_the_oracle(B, H, N, tile_q, density):
    q, k, v = make_random_qkv(B, H, N, 128, 500 + N + tile_q, q_std=1.5, k_std=1.5)
    announce(f"mask reuse random B={B} H={H} N={N} tile_q={tile_q} kept={density}")
    n_qu, n_kt = -(-N // tile_q), -(-N // TILE_K)
    rng = np.random.default_rng(N + int(density * 100))
    mask = (rng.random((B, H, n_qu, n_kt)) >= density).astype(np.uint8)
    mask[0, 0, 0, :] = 1                     # one unit keeps nothing
    if n_kt > 1:
        mask[-1, -1, -1, 0] = 1              # the first key tile skipped, others kept
        mask[-1, -1, -1, 1:] = 0
    g = run_reuse(*upload(q, k, v), mask, tile_q)
    assert np.array_equal(g.mask, mask)
    compare_forced(q, k, v, g, tile_q)
    assert (g.stats == expected_stats_from_mask(mask, N, tile_q)).all()
    assert not g.o[0, 0, :min(N, tile_q)].any()               # zeros for the empty unit


@pytest.mark.parametrize("tile_q", [128, 32])
@pytest.mark.parametrize("rule,param", [("dynsparse_lambda", -6.0), ("blasst", 1e-2)])
def test_reusing_a_128_key_rule_mask(peaked, rule, param, tile_q):
    """A mask of 128-key decisions keeps or skips both 64-key tiles of each decision: the
    reuse run matches the oracle for that kept set, carries the mask and counters over,
    and agrees with the rule call that wrote the mask to the parity tolerance (the two
    raise the softmax reference at different points, so they are not bit-identical)."""
    (q, k, v), dev = peaked
    announce(f"mask reuse of 128-key {rule}={param} tile_q={tile_q}")
    ref = run_gpu(*dev, rule, param, SCALE, tile_q=tile_q, tile_k=128)
    got = run_reuse(*dev, ref.mask, tile_q, tile_k=128)
    assert np.array_equal(got.mask, ref.mask)
    assert np.array_equal(got.stats, ref.stats)
    assert ref.mask.mean() > 0.1
    compare_forced(q, k, v, got, tile_q, tile_k=128)
    diff = oracle.bf16_to_f64(got.o) - oracle.bf16_to_f64(ref.o)
    assert np.abs(diff).max() <= 2e-2
    assert np.abs(got.lse - ref.lse).max() <= 2e-3


@pytest.mark.parametrize("B,H,N,tile_q", [(1, 2, 2048, 128), (1, 3, 1000, 32), (1, 1, 65, 128),
                                          (2, 1, 191, 32)])
@pytest.mark.parametrize("density", [0.2, 0.8])
def test_arbitrary_128_key_masks_match_the_oracle(B, H, N, tile_q, density):
    q, k, v = make_random_qkv(B, H, N, 128, 900 + N + tile_q, q_std=1.5, k_std=1.5)
    announce(f"mask reuse 128-key random B={B} H={H} N={N} tile_q={tile_q} kept={density}")
    n_qu, n_kd = -(-N // tile_q), -(-N // 128)
    rng = np.random.default_rng(7 * N + int(density * 100))
    mask = (rng.random((B, H, n_qu, n_kd)) >= density).astype(np.uint8)
    mask[0, 0, 0, :] = 1                     # one unit keeps nothing
    g = run_reuse(*upload(q, k, v), mask, tile_q, tile_k=128)
    assert np.array_equal(g.mask, mask)
    compare_forced(q, k, v, g, tile_q, tile_k=128)
    assert (g.stats == expected_stats_from_mask(mask, N, tile_q, 128)).all()
    assert not g.o[0, 0, :min(N, tile_q)].any()


@pytest.mark.slow
def test_wan720p_reuse_of_lambda_mask():
    w = WORKLOADS["wan720p"]
    announce(f"generate {w.describe()}")
    q, k, v, _ = workload_inputs("wan720p")
    dev = upload(q, k, v)
    ref = run_gpu(*dev, "dynsparse_lambda", -6.0, SCALE)
    got = run_reuse(*dev, ref.mask, 128)
    print(f"[case] reuse of a {ref.mask.mean():.3f}-sparse mask", flush=True)
    assert np.array_equal(got.o, ref.o)
    assert np.array_equal(got.lse.view(np.uint32), ref.lse.view(np.uint32))
    assert np.array_equal(got.stats, ref.stats)
