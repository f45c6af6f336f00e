"""GPU skip decisions on inputs whose masks are known in closed form.

``synth.vote_pattern_inputs`` gives every 32-row group of query rows its own peaks in a
seeded set of key tiles (about 20 natural-log units above everything else).  With
lambda = -10 (or BLASST at tau = 1e-4) a 128-row unit skips a key tile exactly when none
of its groups peaks there, and a 32-row unit skips exactly its group's other tiles.
Across key tiles every group's vote flips in both vote buffers, and tiles kept by 0-4
groups all occur, so each way a workgroup combines its waves' votes is exercised: in
particular a wave whose vote is unchanged writes nothing, and a wave that keeps a tile
does not read the others' votes.  Checked: the mask equals the closed form bit for bit,
the counters follow from it, and the outputs and LSE agree with the oracle
(teacher-forced); MX-FP8 Q and K give the same mask.
"""

import math
import sys

import numpy as np
import pytest

from synth import expected_skip, vote_pattern_inputs

from _parity import (assert_parity, compare, expected_stats_from_mask, run_gpu, to_device)

pytestmark = pytest.mark.gpu

SCALE = 1.0 / math.sqrt(128)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_16317_amd as dsa

    dsa.lib()               # raises if the HIP library is not built


def announce(msg):
    print(f"\n[case] {msg}", flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("N", [2560, 2348])
@pytest.mark.parametrize("tile_q", [128, 32])
@pytest.mark.parametrize("rule,param", [("dynsparse_lambda", -10.0), ("blasst", 1e-4)])
def test_mask_matches_closed_form(N, tile_q, rule, param):
    q, k, v, pattern = vote_pattern_inputs(N, 2, seed=50 + N % 7)
    announce(f"vote patterns N={N} tile_q={tile_q} rule={rule} param={param}")
    g = run_gpu(to_device(q), to_device(k), to_device(v), rule, param, SCALE, tile_q=tile_q)
    assert np.array_equal(g.mask, expected_skip(pattern, N, tile_q))
    assert (g.stats == expected_stats_from_mask(g.mask, N, tile_q)).all()
    rep = compare(q, k, v, g, rule, param, SCALE, tile_q=tile_q)
    print(rep, flush=True)
    assert_parity(rep)
    assert rep.mismatches == 0


@pytest.mark.parametrize("tile_q", [128, 32])
def test_mask_matches_closed_form_mxfp8(tile_q):
    import torch
    import paper_2606_16317_amd as dsa

    N = 2348
    q, k, v, pattern = vote_pattern_inputs(N, 2, seed=57)
    announce(f"vote patterns MX-FP8 N={N} tile_q={tile_q}")
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    qc, qs = dsa.dsattn_quantize_mxfp8(qd)
    kc, ks = dsa.dsattn_quantize_mxfp8(kd)
    n_units = -(-N // tile_q)
    mask = torch.full((2 * n_units * (-(-N // 64)),), 7, dtype=torch.uint8, device="cuda")
    dsa.dsattn_attn_fwd_mxfp8(dsa.RULE_DYNSPARSE_LAMBDA, -10.0, qc, qs, kc, ks, vd,
                              scale=SCALE, tile_q=tile_q, mask_out=mask)
    torch.cuda.synchronize()
    got = mask.cpu().numpy().reshape(1, 2, n_units, -1)
    assert np.array_equal(got, expected_skip(pattern, N, tile_q))


@pytest.mark.parametrize("tile_k,key_order", [(32, 0), (128, 0), (64, 1), (128, 1)])
@pytest.mark.parametrize("tile_q", [128, 32])
@pytest.mark.parametrize("rule,param", [("dynsparse_lambda", -10.0), ("blasst", 1e-4)])
def test_mask_closed_form_key_tiles(tile_k, key_order, tile_q, rule, param):
    """32-key pattern tiles: 32-key decisions (two halves of each 64-key tile, the second
    voted after the first), 128-key pair decisions and diagonal-first order all give the
    closed-form mask."""
    N = 2348
    q, k, v, pattern = vote_pattern_inputs(N, 2, seed=58, p_bit=0.12, pattern_tile=32)
    order = "diagonal" if key_order else "ascending"
    announce(f"vote patterns N={N} tile_q={tile_q} tile_k={tile_k} order={order} rule={rule}")
    g = run_gpu(to_device(q), to_device(k), to_device(v), rule, param, SCALE, tile_q=tile_q,
                tile_k=tile_k, key_order=key_order)
    assert np.array_equal(g.mask, expected_skip(pattern, N, tile_q, tile_k=tile_k,
                                                pattern_tile=32))
    assert (g.stats == expected_stats_from_mask(g.mask, N, tile_q, tile_k)).all()
    rep = compare(q, k, v, g, rule, param, SCALE, tile_q=tile_q, tile_k=tile_k,
                  key_order=order)
    print(rep, flush=True)
    assert_parity(rep)
    assert rep.mismatches == 0
