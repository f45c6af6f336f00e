"""Inputs whose skip decisions are known in closed form, for checking how the decisions of
several query rows are combined.

Query rows are grouped like the kernels' decision units: row r belongs to query tile
i = r // 128 and to its 32-row group w = (r % 128) // 32.  Every group (i, w) gets its own
direction e_(4i + w) of R^128: its query rows are A * e plus small noise.  Pattern tile t
(64 keys by default) holds one "peak" key at its position 3 carrying A * e for every group
whose bit is set in pattern[i, t] (4 bits per query tile and pattern tile); all other
keys are noise.  So a group's rows score about A^2 * scale on the peak keys of its own tiles and
about zero elsewhere.  Key tile 0 carries every group's peak.  V is standard normal.

With A^2 * scale ~ 20 (natural-log units) and a threshold like lambda = -10, each group's
rows keep exactly the tiles of its own pattern bits: a peak tile's margin is -ln(number
of peak tiles so far) > -5 for up to 140 pattern tiles, every other tile's about -20.

Pattern tiles may be 32 keys instead of 64 (peak at 32 t + 3); a decision tile of B_c
keys is then kept by a group when any of its pattern tiles is.  Pattern tile 0 and the
pattern tile holding key 128 i (query tile i's own position, where diagonal-first order
starts) carry every group's peak, so the decisions are the same in ascending and in
diagonal-first order.
"""

from __future__ import annotations

import numpy as np

from .video_qkv import bf16_bits

GROUP_ROWS = 32
TILE_ROWS = 128
KEY_TILE = 64
PEAK_OFFSET = 3


def vote_pattern_inputs(N: int, H: int, seed: int, p_bit: float = 0.35, amp: float = 15.0,
                        d: int = 128, pattern_tile: int = KEY_TILE):
    """Return (q, k, v, pattern) for B = 1: bf16 bit arrays [1][H][N][d] and the uint8
    pattern [H][n_qt][n_pt] of 4-bit group masks (bit w = group w peaks in pattern tile
    t of ``pattern_tile`` keys, 32 or 64)."""
    if pattern_tile not in (32, 64):
        raise ValueError("pattern tiles are 32 or 64 keys")
    n_qt = -(-N // TILE_ROWS)
    n_kt = -(-N // pattern_tile)
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
        for i in range(n_qt):                 # where diagonal-first order starts
            pat[i, (TILE_ROWS * i) // pattern_tile] = 0xF
        pattern[h] = pat
        qf = 0.02 * rng.standard_normal((N, d))
        qf[rows, direction] += amp
        kf = 0.3 * rng.standard_normal((N, d))
        for t in range(n_kt):
            key = pattern_tile * t + PEAK_OFFSET
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


def expected_skip(pattern: np.ndarray, N: int, unit_rows: int, tile_k: int = KEY_TILE,
                  pattern_tile: int = KEY_TILE) -> np.ndarray:
    """Closed-form skip mask [1][H][n_units][ceil(N / tile_k)] (1 = skipped) for 128-row
    units (a tile is skipped when no group with valid rows peaks in it) or 32-row units
    (each group keeps its own peak tiles); a decision tile of tile_k keys keeps a group
    when any of its pattern tiles does.  Groups without valid rows do not vote."""
    if tile_k % pattern_tile:
        raise ValueError("decision tiles must be whole pattern tiles")
    H, n_qt, n_pt = pattern.shape
    per = tile_k // pattern_tile
    n_dt = -(-N // tile_k)
    pad = np.zeros((H, n_qt, n_dt * per), np.uint8)
    pad[:, :, :n_pt] = pattern
    pat = np.bitwise_or.reduce(pad.reshape(H, n_qt, n_dt, per), axis=-1)
    valid = np.zeros((n_qt, 4), bool)
    for i in range(n_qt):
        for w in range(4):
            valid[i, w] = TILE_ROWS * i + GROUP_ROWS * w < N
    bits = np.stack([(pat >> w) & 1 for w in range(4)], axis=-1).astype(bool)  # H,qt,dt,4
    if unit_rows == TILE_ROWS:
        keep = (bits & valid[None, :, None, :]).any(axis=-1)
        return (~keep).astype(np.uint8)[None]
    n_units = -(-N // GROUP_ROWS)
    keep = bits.transpose(0, 1, 3, 2).reshape(H, 4 * n_qt, n_dt)[:, :n_units]
    return (~keep).astype(np.uint8)[None]
