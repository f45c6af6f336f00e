"""CPU oracle of the MX-FP8 quantisation used for a quantised Q K^T (CPU, exact).

TEST INFRASTRUCTURE ONLY (same rule as the rest of ``oracle/``).

The Conclusion (Section 5) lists quantisation among the methods DynSparse combines with.  The
quantised variant here stores Q and K in the OCP Microscaling (MX) FP8 format: every run of
32 consecutive values of a row (a block along the head dimension) shares one power-of-two
scale stored as an E8M0 exponent, and each value is an FP8 E4M3 number (1 sign bit, 4
exponent bits with bias 7, 3 mantissa bits; no infinities; largest finite magnitude
448 = 1.75 * 2^8; subnormals m * 2^-9).

Quantisation of one block x[0..31] (as in the MX specification):
* amax = max |x|; if amax == 0 the scale code is 0 and every element is +0;
* shared exponent E = floor(log2(amax)) - 8 (8 = largest E4M3 exponent), stored as the
  E8M0 code E + 127 (clamped to 0..254);
* each element is x / 2^E rounded to the nearest E4M3 value, ties to the even code,
  magnitudes above 448 saturating to 448.

Key smoothing (optional, before quantising K): subtracting one vector m from every key of
a head adds the same constant -q.m to every score of a query row, which the softmax
removes, so the attention output and every skip decision of the rule (which compares
score differences only) are unchanged in exact arithmetic, while the keys lose their
common component and quantise with a smaller relative error.  The natural choice of m is
the mean key of the head; the subtraction is done in float32 (x - m rounded to nearest
float32) and the result quantised as above.  The LSE of the smoothed scores is that of
the original ones minus scale * q.m.

This module finds the nearest E4M3 value by searching the table of all codes, which is a
different route from the bit manipulation of the HIP kernel.  Parity status: pinned by
``tests/test_oracle_mxfp8.py`` (hand-worked blocks, exactly representable round trips,
ties, saturation, subnormals, zero blocks, the decoded code table; the key mean on
constant and arithmetic-progression keys, the float32 rounding of the subtraction, and the
invariance of the attention output and of the rule's decisions under smoothing).
"""

from __future__ import annotations

import math

import numpy as np

BLOCK = 32
E4M3_MAX = 448.0
E4M3_EMAX = 8


def e4m3_value(code: int) -> float:
    """Value of an E4M3 code (0x7f / 0xff are NaN)."""
    code = int(code) & 0xFF
    sign = -1.0 if code & 0x80 else 1.0
    e = (code >> 3) & 0xF
    m = code & 0x7
    if e == 0xF and m == 0x7:
        return math.nan
    if e == 0:
        return sign * m * 2.0 ** -9
    return sign * (1.0 + m / 8.0) * 2.0 ** (e - 7)


# positive finite codes 0x00..0x7e and their values, ascending
_POS_CODES = np.arange(0x7F, dtype=np.int64)
_POS_VALUES = np.array([e4m3_value(c) for c in _POS_CODES])


def e4m3_round(x: np.ndarray) -> np.ndarray:
    """Nearest E4M3 code (uint8) of each finite value, ties to the even code, saturating."""
    x = np.asarray(x, dtype=np.float64)
    a = np.minimum(np.abs(x), E4M3_MAX)
    idx = np.searchsorted(_POS_VALUES, a)          # first value >= a
    hi = np.clip(idx, 0, len(_POS_VALUES) - 1)
    lo = np.clip(idx - 1, 0, len(_POS_VALUES) - 1)
    d_hi = _POS_VALUES[hi] - a
    d_lo = a - _POS_VALUES[lo]
    pick_lo = (d_lo < d_hi) | ((d_lo == d_hi) & (_POS_CODES[lo] % 2 == 0))
    code = np.where(pick_lo, _POS_CODES[lo], _POS_CODES[hi])
    neg = (x < 0) & (code != 0)
    return (code | np.where(neg, 0x80, 0)).astype(np.uint8)


def e4m3_decode(codes: np.ndarray) -> np.ndarray:
    codes = np.asarray(codes, dtype=np.int64) & 0xFF
    table = np.array([e4m3_value(c) for c in range(256)])
    return table[codes]


def quantize_mxfp8(x: np.ndarray):
    """Quantise the last axis of ``x`` (a multiple of 32) block by block.

    Returns (codes uint8 like x, scale codes uint8 [..., n / 32]).
    """
    x = np.asarray(x, dtype=np.float64)
    n = x.shape[-1]
    if n % BLOCK:
        raise ValueError("last axis must be a multiple of 32")
    blocks = x.reshape(*x.shape[:-1], n // BLOCK, BLOCK)
    amax = np.abs(blocks).max(axis=-1)
    exp = np.zeros(amax.shape, dtype=np.int64)
    nz = amax > 0
    # floor(log2(amax)) exactly, from the binary exponent
    mant, e2 = np.frexp(amax[nz])               # amax = mant * 2^e2, mant in [0.5, 1)
    exp[nz] = e2 - 1 - E4M3_EMAX
    scale_code = np.where(nz, np.clip(exp + 127, 0, 254), 0).astype(np.uint8)
    scale = np.where(nz, np.ldexp(1.0, scale_code.astype(np.int64) - 127), 1.0)
    codes = e4m3_round(blocks / scale[..., None])
    codes = np.where(nz[..., None], codes, 0).astype(np.uint8)
    return codes.reshape(x.shape), scale_code


def dequantize_mxfp8(codes: np.ndarray, scale_codes: np.ndarray) -> np.ndarray:
    """float64 values of MX-FP8 data (inverse of ``quantize_mxfp8`` up to rounding)."""
    codes = np.asarray(codes)
    n = codes.shape[-1]
    vals = e4m3_decode(codes).reshape(*codes.shape[:-1], n // BLOCK, BLOCK)
    scale = np.ldexp(1.0, np.asarray(scale_codes, dtype=np.int64) - 127)
    return (vals * scale[..., None]).reshape(codes.shape)


def key_mean(k: np.ndarray) -> np.ndarray:
    """Mean key of every head: float64 [..., d] of k [..., N, d] (float values)."""
    return np.asarray(k, dtype=np.float64).mean(axis=-2)


def smooth_keys(k: np.ndarray, shift: np.ndarray) -> np.ndarray:
    """float32 k - shift for every key of a head: k [..., N, d] (values exactly
    representable in float32, e.g. bf16), shift [..., d] rounded to float32 first; each
    difference is rounded to nearest float32, as the quantiser does."""
    k32 = np.asarray(k, dtype=np.float64).astype(np.float32)
    s32 = np.asarray(shift, dtype=np.float64).astype(np.float32)
    return (k32 - s32[..., None, :]).astype(np.float32)
