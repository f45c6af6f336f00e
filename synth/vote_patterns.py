"""Inputs whose skip decisions are known in closed form, for checking how the decisions of
several query rows are combined.

Query rows are grouped like the kernels' decision units: row r belongs to query tile
i = r // 128 and to its 32-row group w = (r % 128) // 32.  Every group (i, w) gets its own
direction e_(4i + w) of R^128: its query rows are A * e plus small noise.  Key tile t
(64 keys) holds one "peak" key at position 64 t + 3 carrying A * e for every group whose
bit is set in pattern[i, t] (4 bits per query tile and key tile); all other keys are
noise.  So a group's rows score about A^2 * scale on the peak keys of its own tiles and
about zero elsewhere.  Key tile 0 carries every group's peak.  V is standard normal.

With A^2 * scale ~ 20 (natural-log units) and a threshold like lambda = -10, each group's
rows keep exactly the tiles of its own pattern bits: a peak tile's margin is -ln(number
of peak tiles so far) > -3.7 for up to 40 key tiles, every other tile's about -20.
"""

from __future__ import annotations

import numpy as np

from .video_qkv import bf16_bits

GROUP_ROWS = 32
TILE_ROWS = 128
KEY_TILE = 64
PEAK_OFFSET = 3


def vote_pattern_inputs(N: int, H: int, seed: int, p_bit: float = 0.35, amp: float = 15.0,
                        d: int = 128):
    """Return (q, k, v, pattern) for B = 1: bf16 bit arrays [1][H][N][d] and the uint8
    pattern [H][n_qt][n_kt] of 4-bit group masks (bit w = group w peaks in key tile t)."""
    n_qt = -(-N // TILE_ROWS)
    n_kt = -(-N // KEY_TILE)
    if 4 * n_qt > d:
        raise ValueError("at most d / 4 query tiles: one direction per 32-row group")
    rng = np.random.default_rng(seed)
    q = np.empty((1, H, N, d), np.uint16)
    k = np.empty_like(q)
    v = np.empty_like(q)
    pattern = np.empty((H, n_qt, n_kt), np.uint8)
    rows = np.arange(N)
    direction = 4 * (rows // TILE_ROWS) + (rows % TILE_ROWS) // GROUP_ROWS
    for h in range(H):
        bits = (rng.random((n_qt, n_kt, 4)) < p_bit).astype(np.uint8)
        pat = bits[..., 0] | (bits[..., 1] << 1) | (bits[..., 2] << 2) | (bits[..., 3] << 3)
        pat[:, 0] = 0xF
        pattern[h] = pat
        qf = 0.02 * rng.standard_normal((N, d))
        qf[rows, direction] += amp
        kf = 0.3 * rng.standard_normal((N, d))
        for t in range(n_kt):
            key = KEY_TILE * t + PEAK_OFFSET
            if key >= N:
                continue
            for i in range(n_qt):
                for w in range(4):
                    if pat[i, t] >> w & 1:
                        kf[key, 4 * i + w] += amp
        q[0, h] = bf16_bits(qf.astype(np.float32))
        k[0, h] = bf16_bits(kf.astype(np.float32))
        v[0, h] = bf16_bits(rng.standard_normal((N, d)).astype(np.float32))
    return q, k, v, pattern


def expected_skip(pattern: np.ndarray, N: int, unit_rows: int) -> np.ndarray:
    """Closed-form skip mask [1][H][n_units][n_kt] (1 = skipped) for 128-row units (a tile is
    skipped when no group with valid rows peaks in it) or 32-row units (each group keeps
    its own peak tiles).  Groups without valid rows do not vote."""
    H, n_qt, n_kt = pattern.shape
    valid = np.zeros((n_qt, 4), bool)
    for i in range(n_qt):
        for w in range(4):
            valid[i, w] = TILE_ROWS * i + GROUP_ROWS * w < N
    bits = np.stack([(pattern >> w) & 1 for w in range(4)], axis=-1).astype(bool)  # H,qt,kt,4
    if unit_rows == TILE_ROWS:
        keep = (bits & valid[None, :, None, :]).any(axis=-1)
        return (~keep).astype(np.uint8)[None]
    n_units = -(-N // GROUP_ROWS)
    keep = bits.transpose(0, 1, 3, 2).reshape(H, 4 * n_qt, n_kt)[:, :n_units]
    return (~keep).astype(np.uint8)[None]
