"""Inputs for 32-key skip decisions (B_c = 32) whose outcome depends on the order of the
two halves of a 64-key tile.

With 32-key decisions the second half h1 of a tile is decided against the state that
includes the first half h0 when h0 is kept.  A kernel may take that decision early when
it is certain; these inputs make the difference visible: on a "flip" tile h1 passes the
threshold against the state before the tile and fails it once h0 is counted, both by a
wide margin, so taking h1's decision early, or against the wrong state, keeps a block
that must be skipped.

Every query row is alike (dimensions 0-2 hold 8, the rest 0; with the softmax scale 1/8
a key's score is k0 + k1 + k2, an exact sum of three bf16 numbers), so every decision unit
decides the same way.  Key tile 0 holds 64 keys of score 0.  Every later tile holds one
peak in h0 (position 5) and one in h1 (position 41); its other keys score -40.  Peaks sit
at designed offsets from a reference level that follows the rule's reference: the
log-sum-exp of the peaks laid down so far for DynSparse (ln 64 after tile 0), their
maximum for BLASST (0 after tile 0).  Tile kinds, drawn with a seeded generator, and the
blocks the rule then skips (threshold thr in natural-log units):

  kind     DynSparse h0 / h1 offsets      BLASST h0 / h1 offsets     skipped
  flip     ln 15 / thr + 1.4              3 / thr + 1.5              h1
  sure     ln 15 / thr + 8.5              3 / 3 + thr + 1.5          none
  late     ln 15 / thr + 4.2              3 / 3 + thr + 1.5          none
  h1only   thr - 1.5 / thr + 1.5          thr - 1.5 / thr + 1.5      h0
  none     thr - 2 / thr - 1.5            thr - 2 / thr - 1.5        both

(An h0 peak at ln 15 above the level multiplies the kept mass by 16: h1's margin then
drops by ln 16 = 2.77.  "sure" leaves h1 kept however the state after h0 is bounded,
"late" only against the exact state.)  Every designed margin is at least 1.2 in absolute
value.  V is standard normal.  Only numbers are placed here; the oracle computes the
decisions.
"""

from __future__ import annotations

import math

import numpy as np

from .margin_band import three_part_bf16
from .video_qkv import bf16_bits

KEY_TILE = 64
H0_PEAK, H1_PEAK = 5, 41
SCALE = 0.125
LOW = -40.0
KINDS = ("flip", "sure", "late", "h1only", "none")
# skipped (h0, h1) 32-key blocks of each kind
EXPECTED_SKIP = {"flip": (0, 1), "sure": (0, 0), "late": (0, 0), "h1only": (1, 0),
                 "none": (1, 1)}
_DYN = {"flip": (math.log(15.0), 1.4), "sure": (math.log(15.0), 8.5),
        "late": (math.log(15.0), 4.2), "h1only": (None, 1.5), "none": (None, -1.5)}


def _offsets(kind: str, rule: str, thr: float):
    """(h0, h1) peak offsets from the reference level."""
    if rule == "dynsparse":
        a, b = _DYN[kind]
        if a is None:
            a = thr - (1.5 if kind == "h1only" else 2.0)
        return a, thr + b
    if kind == "flip":
        return 3.0, thr + 1.5
    if kind in ("sure", "late"):
        return 3.0, 3.0 + thr + 1.5
    if kind == "h1only":
        return thr - 1.5, thr + 1.5
    return thr - 2.0, thr - 1.5


def half_flip_inputs(T: int, H: int, rule: str, thr: float, seed: int, d: int = 128,
                     n_tail: int = 0):
    """Return (q, k, v, kinds, skip, scale): bf16 bit arrays [1][H][N][d] with
    N = 64 T - n_tail, the tile kinds [H][T] (tile 0 is "start"), the designed skip mask of
    32-key blocks [H][ceil(N / 32)] (1 = skipped) and the softmax scale.  ``rule`` is
    "dynsparse" or "blasst"; ``thr`` is lambda or ln(tau), at most -4 (tile 0's second
    half must be kept)."""
    if rule not in ("dynsparse", "blasst"):
        raise ValueError("rule is dynsparse or blasst")
    if thr > -4.0:
        raise ValueError("thresholds above -4 would skip part of tile 0")
    if not 0 <= n_tail < KEY_TILE - H1_PEAK:
        raise ValueError("the last tile must still hold its h1 peak")
    if T < 2 or d < 3:
        raise ValueError("need two tiles and three head dimensions")
    N = KEY_TILE * T - n_tail
    rng = np.random.default_rng(seed)
    q = np.zeros((1, H, N, d), np.float32)
    q[0, :, :, 0:3] = 8.0
    k = np.zeros((1, H, N, d), np.float32)
    kinds = np.empty((H, T), dtype=object)
    n_blk = -(-N // 32)
    skip = np.zeros((H, n_blk), np.uint8)
    for h in range(H):
        kinds[h, 0] = "start"
        # every kind at least once per head (a "flip" first), the rest drawn
        order = ["flip"] + list(rng.permutation(KINDS))
        order += list(rng.choice(KINDS, size=max(0, T - 1 - len(order))))
        level = math.log(KEY_TILE) if rule == "dynsparse" else 0.0
        for j in range(1, T):
            kind = order[j - 1]
            kinds[h, j] = kind
            a, b = _offsets(kind, rule, thr)
            t0 = KEY_TILE * j
            k[0, h, t0:min(N, t0 + KEY_TILE), 0] = LOW
            k[0, h, t0 + H0_PEAK, 0:3] = three_part_bf16(level + a)
            k[0, h, t0 + H1_PEAK, 0:3] = three_part_bf16(level + b)
            s0, s1 = EXPECTED_SKIP[kind]
            skip[h, 2 * j], skip[h, 2 * j + 1] = s0, s1
            # follow the reference over the peaks that are kept (both placed from the
            # level before the tile)
            kept = [0.0] + ([a] if not s0 else []) + ([b] if not s1 else [])
            if rule == "dynsparse":
                level = level + float(np.logaddexp.reduce(kept))
            else:
                level = level + max(kept)
    v = rng.standard_normal((1, H, N, d)).astype(np.float32)
    return bf16_bits(q), bf16_bits(k), bf16_bits(v), kinds, skip, SCALE
