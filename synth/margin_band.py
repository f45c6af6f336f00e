"""Inputs whose skip decisions sit right at the threshold, for exercising the tolerance on
decisions whose margin is tiny.

Every score is exact in binary floating point on both sides of a parity check: with the
softmax scale 1/8, query rows carry 8 in dimensions 0-2 (and 8 * rho in dimension 3),
so a key's score is k0 + k1 + k2 + rho * k3, a sum of at most four bf16 numbers whose
binary exponents span less than 24 bits: float32 accumulation adds them without
rounding, in any order.

Layout of one head (N = 64 * T keys, key tiles of 64):

* key tile 0: 64 keys of score 0;
* key tile j >= 1: one "peak" key (position 64 j + 5) of score p_j, the other 63 keys at
  -40; the peak also has k3 = 1;
* query rows: rho = 0 for row 7 of every 32-row group, rho = -1 for all other rows, so
  in every group one row sees the peaks at p_j and the others one unit lower (the unit's
  decision follows its highest row);
* peaks p_j = base + thr + delta_j, where thr is the rule's threshold in natural-log
  units and base is the reference the rule compares with right after tile 0: ln 64 (the
  log-sum-exp of 64 zero scores) for DynSparse, 0 (their maximum) for BLASST.  delta_j is
  drawn from +-{1e-7, 1e-6, 1e-5, 3e-5, 1e-4, 3e-4, 1e-3, 3e-3, 5e-3} with seeded signs,
  and every fifth tile gets +-3 (a clear keep or skip).  p_j is rounded to the nearest
  sum of three bf16 numbers (relative error below 2^-24).

Each kept peak raises the DynSparse reference by about e^thr (1e-7 at thr = -16), so the
actual margins drift slightly from delta_j as tiles are kept; the oracle computes them
exactly from the bf16 inputs.  V is standard normal.

No attention arithmetic lives here: this only places numbers.
"""

from __future__ import annotations

import math

import numpy as np

from .video_qkv import bf16_bits

KEY_TILE = 64
PEAK_POS = 5
SCALE = 0.125                      # exact power of two
LOW = -40.0                        # score of the non-peak keys of tiles >= 1
BAND = (1e-7, 1e-6, 1e-5, 3e-5, 1e-4, 3e-4, 1e-3, 3e-3, 5e-3)


def _bf16_value(x: float) -> float:
    """Value of the bf16 number nearest to x (round to nearest even)."""
    bits = bf16_bits(np.array([x], dtype=np.float32))
    return float((bits.astype(np.uint32) << np.uint32(16)).view(np.float32)[0])


def three_part_bf16(x: float) -> tuple:
    """Greedy split of x into three bf16 numbers whose sum approximates x to ~2^-24."""
    a = _bf16_value(x)
    b = _bf16_value(x - a)
    c = _bf16_value(x - a - b)
    return a, b, c


def margin_band_inputs(T: int, H: int, rule: str, thr: float, seed: int, d: int = 128,
                       n_tail: int = 0):
    """Return (q, k, v, deltas, scale): bf16 bit arrays [1][H][N][d] with N = 64 T - n_tail,
    the designed offsets deltas [H][T] (NaN for tile 0) and the softmax scale to use.
    ``rule`` is "dynsparse" or "blasst", ``thr`` the threshold in natural-log units."""
    if rule not in ("dynsparse", "blasst"):
        raise ValueError("rule is dynsparse or blasst")
    if not 0 <= n_tail < KEY_TILE - PEAK_POS:
        raise ValueError("the last tile must still hold its peak key")
    if d < 4:
        raise ValueError("need four head dimensions")
    N = KEY_TILE * T - n_tail
    base = math.log(KEY_TILE) if rule == "dynsparse" else 0.0
    rng = np.random.default_rng(seed)
    q = np.zeros((1, H, N, d), np.float32)
    rows = np.arange(N)
    q[0, :, :, 0:3] = 8.0
    q[0, :, :, 3] = np.where(rows % 32 == 7, 0.0, -8.0)
    k = np.zeros((1, H, N, d), np.float32)
    deltas = np.full((H, T), np.nan)
    for h in range(H):
        for j in range(1, T):
            if j % 5 == 0:
                delta = 3.0 * rng.choice([-1.0, 1.0])
            else:
                delta = rng.choice(BAND) * rng.choice([-1.0, 1.0])
            deltas[h, j] = delta
            t0 = KEY_TILE * j
            k[0, h, t0:min(N, t0 + KEY_TILE), 0] = LOW
            peak = t0 + PEAK_POS
            k[0, h, peak, 0:3] = three_part_bf16(base + thr + delta)
            k[0, h, peak, 3] = 1.0
    v = rng.standard_normal((1, H, N, d)).astype(np.float32)
    return bf16_bits(q), bf16_bits(k), bf16_bits(v), deltas, SCALE
