"""Pins of the MX-FP8 quantisation oracle (``oracle.mxfp8``), CPU only.

They check the E4M3 code table against the format's definition at landmark codes, the
nearest-value search against brute force over every code (ties to even, saturation), and
the block quantisation on hand-worked blocks (scale choice, exact round trips, zero
blocks, subnormal elements).
"""

import math

import numpy as np
import pytest

from oracle.mxfp8 import (dequantize_mxfp8, e4m3_decode, e4m3_round, e4m3_value,
                          quantize_mxfp8)


def test_e4m3_landmarks():
    assert e4m3_value(0x00) == 0.0
    assert e4m3_value(0x38) == 1.0                 # exponent 7 = bias
    assert e4m3_value(0x7E) == 448.0               # largest finite
    assert e4m3_value(0x08) == 2.0 ** -6           # smallest normal
    assert e4m3_value(0x01) == 2.0 ** -9           # smallest subnormal
    assert e4m3_value(0x07) == 7 * 2.0 ** -9       # largest subnormal
    assert e4m3_value(0xB8) == -1.0
    assert math.isnan(e4m3_value(0x7F)) and math.isnan(e4m3_value(0xFF))


def test_round_matches_brute_force():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.normal(0, 30, 3000), rng.normal(0, 0.01, 1000),
                        rng.uniform(-600, 600, 500)])
    got = e4m3_round(x)
    finite = [c for c in range(256) if not math.isnan(e4m3_value(c))]
    vals = np.array([e4m3_value(c) for c in finite])
    for xi, ci in zip(x, got):
        a = min(abs(xi), 448.0) * (1 if xi >= 0 else -1)
        d = np.abs(vals - a)
        best = d.min()
        cands = [finite[i] for i in np.nonzero(d == best)[0]]
        # among equally near codes the even one (mantissa lsb 0); +-0 are the same value
        cands_even = [c for c in cands if c % 2 == 0] or cands
        assert e4m3_value(ci) in [e4m3_value(c) for c in cands_even]


def test_ties_go_to_even():
    # 1.0625 lies halfway between 1.0 (0x38, even) and 1.125 (0x39): even wins
    assert e4m3_round(np.array([1.0625]))[0] == 0x38
    # 1.1875 lies halfway between 1.125 (0x39) and 1.25 (0x3a, even)
    assert e4m3_round(np.array([1.1875]))[0] == 0x3A
    # subnormal tie: 1.5 * 2^-9 between 2^-9 (0x01) and 2 * 2^-9 (0x02, even)
    assert e4m3_round(np.array([1.5 * 2.0 ** -9]))[0] == 0x02


def test_saturation_and_sign():
    c = e4m3_round(np.array([500.0, -1e9, 447.0, -448.0, 0.0, -0.0]))
    assert list(e4m3_decode(c)) == [448.0, -448.0, 448.0, -448.0, 0.0, 0.0]


def test_block_scale_is_floor_log2_amax_minus_8():
    x = np.zeros(64)
    x[3] = 3.0          # block 0: amax 3 -> floor(log2 3) = 1 -> E = -7 -> code 120
    x[40] = -1000.0     # block 1: amax 1000 -> floor(log2) = 9 -> E = 1 -> code 128
    codes, scales = quantize_mxfp8(x)
    assert scales.tolist() == [120, 128]
    # 3 / 2^-7 = 384 = 1.5 * 2^8 -> exactly representable (0x74)
    assert e4m3_value(codes[3]) == 384.0
    # 1000 / 2 = 500 -> saturates to 448 (0xfe with the sign)
    assert codes[40] == 0xFE
    np.testing.assert_array_equal(dequantize_mxfp8(codes, scales)[[3, 40]], [3.0, -896.0])


def test_exact_round_trip_for_representable_blocks():
    rng = np.random.default_rng(1)
    base = np.array([e4m3_value(c) for c in range(0x7F)])
    for _ in range(20):
        e = int(rng.integers(-20, 20))
        vals = rng.choice(base, 32) * rng.choice([-1, 1], 32)
        vals[0] = 448.0                          # pins the block maximum: scale 2^e
        x = vals * 2.0 ** e
        codes, scales = quantize_mxfp8(x)
        assert scales[0] == e + 127
        np.testing.assert_array_equal(dequantize_mxfp8(codes, scales), x)


def test_zero_and_tiny_blocks():
    codes, scales = quantize_mxfp8(np.zeros(32))
    assert scales[0] == 0 and not codes.any()
    # a block whose small entries fall into the subnormal range of the scaled values
    x = np.zeros(32)
    x[0] = 256.0                      # E = 0
    x[1] = 3 * 2.0 ** -9              # scaled value 3 * 2^-9: subnormal code 0x03
    codes, scales = quantize_mxfp8(x)
    assert scales[0] == 127 and codes[1] == 0x03


def test_quantisation_error_bound():
    """Relative error of an element whose scaled value is normal and below 448 is at most
    2^-4 (3 mantissa bits); scaled values in (448, 512) saturate to 448 (the block maximum
    scales into [256, 512)), an error below 1 - 448/512."""
    rng = np.random.default_rng(2)
    x = rng.normal(0, 1, (50, 128))
    codes, scales = quantize_mxfp8(x)
    deq = dequantize_mxfp8(codes, scales)
    scaled = np.abs(x) / np.repeat(np.ldexp(1.0, scales.astype(np.int64) - 127), 32, axis=-1)
    rel = np.abs(deq - x) / np.abs(x)
    normal = (scaled >= 2.0 ** -6) & (scaled <= 448.0)
    assert rel[normal].max() <= 2.0 ** -4 + 1e-12
    sat = scaled > 448.0
    assert sat.any() and rel[sat].max() < 1 - 448 / 512
    assert (scaled.reshape(50, 4, 32).max(axis=-1) >= 256).all()


def test_rule_attention_accepts_dequantised_inputs():
    """Float q/k inputs are used as given: bf16 values passed as floats give the same run."""
    import oracle
    from synth import make_random_qkv

    q, k, v = make_random_qkv(1, 1, 200, 128, 3, q_std=2.0, k_std=2.0)
    a = oracle.rule_attention(q, k, v, 0.1, "dynsparse", -4.0, 128, 64)
    b = oracle.rule_attention(oracle.bf16_to_f64(q), oracle.bf16_to_f64(k), v, 0.1,
                              "dynsparse", -4.0, 128, 64)
    for ra, rb in zip(a.results, b.results):
        assert np.array_equal(ra.skip, rb.skip)
        np.testing.assert_array_equal(ra.o_sparse, rb.o_sparse)


def test_key_mean_closed_forms():
    from oracle.mxfp8 import key_mean

    k = np.zeros((2, 3, 100, 8))
    k[0, 1] = 2.5                                   # constant keys: the constant
    k[1, 2, :, 3] = np.arange(100)                  # 0..99: mean 49.5
    k[1, 0, :, 0] = np.where(np.arange(100) % 2, 1.0, -3.0)   # alternating: -1
    m = key_mean(k)
    assert m.shape == (2, 3, 8)
    assert (m[0, 1] == 2.5).all() and (m[0, 0] == 0).all()
    assert m[1, 2, 3] == 49.5 and m[1, 0, 0] == -1.0


def test_smooth_keys_rounds_each_difference_to_float32():
    from oracle.mxfp8 import smooth_keys

    k = np.array([[[1.5, 1.0, 3.0e38]]])
    sh = np.array([[0.25, 2.0 ** -30, -1.0]])
    out = smooth_keys(k, sh)
    assert out.dtype == np.float32
    assert out[0, 0, 0] == 1.25                     # exact
    assert out[0, 0, 1] == np.float32(1.0)          # 1 - 2^-30 rounds back to 1 in float32
    assert out[0, 0, 2] == np.float32(3.0e38)       # 3e38 + 1 rounds to 3e38


def test_smoothing_leaves_output_and_decisions_unchanged():
    """Subtracting the mean key shifts every score of a row by one constant: in exact
    arithmetic the output and the rule's decisions do not move.  In float64 the outputs
    agree to rounding and every decision with a margin above rounding is the same."""
    import oracle
    from oracle.mxfp8 import key_mean, smooth_keys
    from synth import make_video_qkv

    q, k, v, _ = make_video_qkv(1, 2, (2, 8, 32), 4.0, 4.0, True, 12)
    kf = oracle.bf16_to_f64(k)
    ks = smooth_keys(kf, key_mean(kf)).astype(np.float64)
    assert np.abs(key_mean(ks)).max() < 1e-3 * np.abs(kf).max()   # common part removed
    a = oracle.rule_attention(q, kf, v, 0.088, "dynsparse", -6.0, 128, 64)
    b = oracle.rule_attention(q, ks, v, 0.088, "dynsparse", -6.0, 128, 64)
    skipped = 0
    for ra, rb in zip(a.results, b.results):
        sure = np.abs(ra.margin) > 1e-9
        assert np.array_equal(ra.skip[sure], rb.skip[sure])
        skipped += int(ra.skip.sum())
        if np.array_equal(ra.skip, rb.skip):
            np.testing.assert_allclose(rb.o_sparse, ra.o_sparse, rtol=0, atol=1e-6)
    assert skipped > 0


def test_smoothing_reduces_the_quantisation_error_of_a_common_key_component():
    """Keys with a large shared component quantise with a large error relative to their
    spread; after smoothing the error on the scores is several times smaller."""
    from oracle.mxfp8 import key_mean, smooth_keys

    rng = np.random.default_rng(9)
    k = 8.0 + rng.normal(0, 1, (1, 1, 512, 128))      # common part 8, spread 1
    q = rng.normal(0, 1, (64, 128))
    s = q @ k[0, 0].T
    m = key_mean(k)
    s_plain = q @ dequantize_mxfp8(*quantize_mxfp8(k))[0, 0].T
    ks = smooth_keys(k, m).astype(np.float64)
    s_smooth = q @ dequantize_mxfp8(*quantize_mxfp8(ks))[0, 0].T + (q @ m[0, 0].astype(np.float32))[:, None]
    err = lambda x: np.sqrt(((x - s) ** 2).mean())
    assert err(s_smooth) * 4 < err(s_plain)
