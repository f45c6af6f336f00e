"""The oracle against closed-form skip masks (CPU).

The inputs of ``synth.vote_pattern_inputs`` give every 32-row group of query rows peaks in
a chosen set of key tiles, far above everything else (about 20 in natural-log units), so
Eq. 5 with lambda = -10 keeps exactly a group's peak tiles and skips the rest; BLASST
with tau = 1e-4 does the same (every non-peak row max lies about 20 below the running
max).  A tile decision over several groups therefore follows from the patterns alone:
skipped when no group with valid rows keeps it (the all-rows aggregation of the tile
rule), or per group with 32-row units.  This pins the oracle's aggregation, its running
LSE / max over kept tiles only, and its handling of ragged query and key tiles.
"""

import math

import numpy as np
import pytest

import oracle
from synth import expected_skip, vote_pattern_inputs

SCALE = 1.0 / math.sqrt(128)


@pytest.mark.parametrize("N", [2560, 2348])
@pytest.mark.parametrize("unit", [128, 32])
@pytest.mark.parametrize("rule,thr", [("dynsparse", -10.0), ("blasst", math.log(1e-4))])
def test_oracle_mask_is_closed_form(N, unit, rule, thr):
    q, k, v, pattern = vote_pattern_inputs(N, 1, seed=40 + N % 7)
    run = oracle.rule_attention(q, k, v, SCALE, rule, thr, unit, 64)
    want = expected_skip(pattern, N, unit)
    got = np.stack([r.skip for r in run.results]).astype(np.uint8)
    assert np.array_equal(got, want[0, 0])
    margins = np.concatenate([r.margin[1:] for r in run.results])
    assert np.abs(margins).min() > 3.0          # no decision is anywhere near a tie
    assert 0.1 < want.mean() < 0.9              # both kinds of decision occur


def test_patterns_cover_every_vote_transition():
    """With 128-row units each group's vote flips between keep and skip in both parities
    of the key-tile index, and tiles kept by one, two, three and four groups all occur."""
    q, k, v, pattern = vote_pattern_inputs(2560, 2, seed=41)
    bits = np.stack([(pattern >> w) & 1 for w in range(4)], axis=-1)[:, :, 1:]
    flips = bits[:, :, 2:] != bits[:, :, :-2]          # same vote buffer, two steps apart
    assert flips.any(axis=(0, 1, 2)).all()
    counts = np.unique(bits.sum(axis=-1))
    assert set(counts.tolist()) >= {0, 1, 2, 3, 4}


@pytest.mark.parametrize("tile_k,key_order", [(32, "ascending"), (64, "ascending"),
                                              (128, "ascending"), (64, "diagonal"),
                                              (128, "diagonal")])
@pytest.mark.parametrize("unit", [128, 32])
@pytest.mark.parametrize("rule,thr", [("dynsparse", -10.0), ("blasst", math.log(1e-4))])
def test_oracle_mask_closed_form_key_tiles(tile_k, key_order, unit, rule, thr):
    """32-key pattern tiles: B_c = 32 decides each pattern tile, 64 and 128 the OR of two
    and four; the same mask in ascending and diagonal-first order."""
    N = 2348
    q, k, v, pattern = vote_pattern_inputs(N, 1, seed=43, p_bit=0.12, pattern_tile=32)
    run = oracle.rule_attention(q, k, v, SCALE, rule, thr, unit, tile_k, key_order=key_order)
    want = expected_skip(pattern, N, unit, tile_k=tile_k, pattern_tile=32)
    got = np.stack([r.skip for r in run.results]).astype(np.uint8)
    assert np.array_equal(got, want[0, 0])
    margins = np.concatenate([np.delete(r.margin, np.argmax(r.margin)) for r in run.results])
    assert np.abs(margins).min() > 3.0
    assert 0.05 < want.mean() < 0.95
