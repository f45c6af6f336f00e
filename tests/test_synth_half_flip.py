"""The 32-key "flip" inputs (``synth.half_flip``) against the oracle (CPU).

The GPU test of 32-key decisions compares the kernel's mask with the mask these inputs
are designed to produce; here the oracle (Section 3.1's loop over 32-key blocks, Eq. 5 /
the BLASST rule) must take exactly those decisions, each by a margin of at least 1.2, so
that the designed mask is the rule's and not a guess.
"""

import math

import numpy as np
import pytest

import oracle
from synth import half_flip_inputs
from synth.half_flip import KINDS


@pytest.mark.parametrize("rule,thr", [("dynsparse", -6.0), ("dynsparse", -12.0),
                                      ("blasst", math.log(1e-2)), ("blasst", math.log(1e-3))])
@pytest.mark.parametrize("T,n_tail", [(24, 0), (20, 20)])
def test_oracle_takes_the_designed_decisions(rule, thr, T, n_tail):
    H = 3
    q, k, v, kinds, skip, scale = half_flip_inputs(T, H, rule, thr, seed=T + n_tail,
                                                   n_tail=n_tail)
    N = q.shape[2]
    assert skip.shape == (H, -(-N // 32))
    run = oracle.rule_attention(q, k, v, scale, rule, thr, 128, 32,
                                tiles=[(0, h, 0) for h in range(H)])
    for h, res in enumerate(run.results):
        assert set(kinds[h, 1:]) == set(KINDS)          # every kind on every head
        assert (res.skip.astype(np.uint8) == skip[h]).all()
        assert np.isinf(res.margin[0])                  # the first block has no reference
        assert np.abs(res.margin[1:]).min() >= 1.2
        # a "flip" tile: h0 kept, h1 skipped although it passes against the state before
        flips = [j for j in range(1, T) if kinds[h, j] == "flip"]
        assert flips and all(skip[h, 2 * j] == 0 and skip[h, 2 * j + 1] == 1 for j in flips)


def test_every_row_sees_the_same_scores():
    q, k, v, kinds, skip, scale = half_flip_inputs(6, 1, "dynsparse", -8.0, seed=1)
    s = scale * (oracle.bf16_to_f64(q[0, 0]) @ oracle.bf16_to_f64(k[0, 0]).T)
    assert (s == s[:1]).all()
    assert (s[0, :64] == 0).all()


def test_rejects_unusable_arguments():
    with pytest.raises(ValueError):
        half_flip_inputs(8, 1, "dense", -8.0, 0)
    with pytest.raises(ValueError):
        half_flip_inputs(8, 1, "dynsparse", -3.0, 0)
    with pytest.raises(ValueError):
        half_flip_inputs(8, 1, "dynsparse", -8.0, 0, n_tail=30)
