"""Near-threshold inputs (``synth.margin_band``): the scores are exact, and the oracle's
margins on them follow closed forms, so the GPU test built on the same inputs really
does exercise decisions within the 1e-3 tolerance band (CPU only)."""

import math

import numpy as np
import pytest

import oracle
from oracle import log_threshold_blasst, rule_attention
from synth.margin_band import KEY_TILE, LOW, PEAK_POS, margin_band_inputs, three_part_bf16


def f64(bits):
    return oracle.bf16_to_f64(bits)


def peak_scores(k, h, T):
    """Designed peak score of every tile j >= 1 (the sum of its three bf16 parts)."""
    kk = f64(k[0, h])
    return np.array([math.fsum(kk[KEY_TILE * j + PEAK_POS, 0:3]) for j in range(1, T)])


def test_three_part_split_is_close():
    for x in (-9.84, -16.0 + 4.1588, -4.605170185988091 + 3e-3, 1e-7 - 12.0):
        a, b, c = three_part_bf16(x)
        assert abs((a + b + c) - x) <= abs(x) * 2.0 ** -22


@pytest.mark.parametrize("n_tail", [0, 20])
def test_scores_are_exact(n_tail):
    T = 12
    q, k, v, deltas, scale = margin_band_inputs(T, 2, "dynsparse", -16.0, 1, n_tail=n_tail)
    N = q.shape[2]
    for h in range(2):
        s = scale * (f64(q[0, h]) @ f64(k[0, h]).T)
        peaks = peak_scores(k, h, T)
        rows7 = np.arange(N) % 32 == 7
        assert (s[:, :KEY_TILE] == 0.0).all()
        for j in range(1, T):
            cols = np.arange(KEY_TILE * j, min(N, KEY_TILE * (j + 1)))
            pk = KEY_TILE * j + PEAK_POS
            assert (s[rows7, pk] == peaks[j - 1]).all()
            assert (s[~rows7, pk] == peaks[j - 1] - 1.0).all()
            rest = cols[cols != pk]
            assert (s[:, rest] == LOW).all()


@pytest.mark.parametrize("tau", [1e-3, 1e-2])
def test_blasst_margins_closed_form(tau):
    """The running max stays at tile 0's 0 (every peak is negative), so the margin of
    tile j is exactly its peak score minus ln(tau)."""
    T, H = 30, 2
    thr = log_threshold_blasst(tau)
    q, k, v, deltas, scale = margin_band_inputs(T, H, "blasst", thr, 3)
    run = rule_attention(q, k, v, scale, "blasst", thr, 128, 64,
                         tiles=[(0, h, 0) for h in range(H)])
    for h, res in enumerate(run.results):
        expect = peak_scores(k, h, T) - thr
        assert np.array_equal(res.margin[1:], expect)
        assert np.array_equal(res.skip[1:], expect < 0)
        # the designed offsets are met to within the three-part rounding
        assert np.abs(expect - deltas[h, 1:]).max() < 1e-6


@pytest.mark.parametrize("lam", [-16.0, -12.0])
def test_dynsparse_margins_closed_form(lam):
    """Row 7 of each group has the largest metric; its LSE before tile j is
    ln(64 + sum over kept tiles i < j of (e^{p_i} + 63 e^{-40})), computed here with
    math.fsum over the exact scores."""
    T, H = 30, 2
    q, k, v, deltas, scale = margin_band_inputs(T, H, "dynsparse", lam, 5)
    run = rule_attention(q, k, v, scale, "dynsparse", lam, 128, 64,
                         tiles=[(0, h, 0) for h in range(H)])
    for h, res in enumerate(run.results):
        peaks = peak_scores(k, h, T)
        terms = [1.0] * KEY_TILE
        for j in range(1, T):
            margin = peaks[j - 1] - math.log(math.fsum(terms)) - lam
            assert res.margin[j] == pytest.approx(margin, abs=1e-12)
            assert res.skip[j] == (margin < 0)
            if not res.skip[j]:
                terms += [math.exp(peaks[j - 1])] + [math.exp(LOW)] * (KEY_TILE - 1)


@pytest.mark.parametrize("rule,thr,tiny", [("dynsparse", -16.0, 2e-6), ("dynsparse", -12.0, 1e-4),
                                           ("blasst", math.log(1e-3), 2e-6),
                                           ("blasst", math.log(1e-2), 2e-6)])
def test_band_is_populated(rule, thr, tiny):
    """On the GPU test's inputs (four heads of 48 tiles) the oracle puts many decisions
    within the tolerance band, on both sides of the threshold, and some within ``tiny``
    of it (down to 2e-6 where kept peaks barely move the reference: e^-16 per kept tile;
    at lambda = -12 each kept tile moves it by about 6e-6)."""
    T, H = 48, 4
    q, k, v, deltas, scale = margin_band_inputs(T, H, rule, thr, 11)
    run = rule_attention(q, k, v, scale, rule, thr, 128, 64,
                         tiles=[(0, h, 0) for h in range(H)])
    m = np.concatenate([r.margin[1:] for r in run.results])
    band = np.abs(m) < 1e-3
    assert band.sum() >= 40
    assert (m[band] > 0).sum() >= 10 and (m[band] < 0).sum() >= 10
    assert (np.abs(m) < tiny).sum() >= 4
    assert (np.abs(m) > 1.0).sum() >= 10           # clear decisions too
