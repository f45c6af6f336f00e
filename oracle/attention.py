"""CPU fp64 oracle for the tile-filtered FlashAttention forward pass.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this module.  It shares no code with the
HIP path (no kernels, headers, helpers or constants); both sides only share the seeded
bf16 inputs drawn by ``synth``.

What it computes, in the paper's notation (natural logarithms throughout):

* Attention logits ``S = scale * Q K^T`` of one query tile (``B_r`` rows) against the
  whole key sequence, from bf16 inputs upcast exactly to float64.
* A FlashAttention-2 loop over key tiles ``j = 1..T_c`` of ``B_c`` columns in ascending
  order (Section 1: tile-based attention over (Q_i, K_j) pairs).  For each tile it forms
  the tile's row maximum ``m_hat`` and evaluates one of three rules:

  - DynSparse (Section 3.1, Eq. 5 and Eq. 6): ``t = m_hat - LSE^(j-1)``, where
    ``LSE^(j-1)`` is the log-sum-exp of the logits of all key tiles *kept* before tile j;
    the tile is skipped when ``t < lambda``.
  - BLASST (Section 1 and Section 2.1, item 4): ``t = m_hat - m^(j-1)``, the tile maximum
    minus the running maximum of the kept tiles; skipped when ``t < ln(tau)``.
  - dense: never skips.

  The per-row metric is turned into one decision per (Q-tile, K-tile) pair by requiring
  *every* valid row of the Q tile to be below the threshold (the reading that keeps the
  per-row recall bound of Section 3.1).  Ties (``t == threshold``) keep the tile.
* A skipped tile contributes nothing: no exponentials, no row-sum, no P.V, and it does
  not change the running maximum or the LSE.
* The output is renormalised over the kept keys only (Eq. 1: the sparse output divides by
  the kept mass), ``O[r] = sum_{c kept} exp(S[r,c] - LSE_kept[r]) V[c]``.
* The recall of a row is the dense softmax mass of its kept keys,
  ``exp(LSE_kept - LSE_all)`` (Section 3.1: the lost recall is the lost probability mass).

Parity status: every function here is pinned by ``tests/test_oracle_pins.py`` against
closed forms, brute force on tiny inputs, the recall theorem of Section 3.1 and the
uniform-attention error figures printed in Section 2.3 (``tests/golden/``).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

RULES = ("dense", "blasst", "dynsparse")


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact upcast of bf16 bit patterns (uint16) to float64."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32).astype(np.float64)


def lambda_from_recall(recall: float, n_keys: int) -> float:
    """Threshold lambda that guarantees a kept-mass (recall) of at least ``recall``.

    Section 3.1 (recall bound): a skipped token's dense softmax probability is at most
    ``e^t < e^lambda``; with ``lambda = ln(eps / L)`` for ``L`` keys the total lost mass
    stays below ``eps``.  Here ``eps = 1 - recall``; ``recall == 1`` gives ``-inf`` (dense).
    """
    if not (0.0 < recall <= 1.0):
        raise ValueError("recall must lie in (0, 1]")
    if n_keys <= 0:
        raise ValueError("n_keys must be positive")
    if recall == 1.0:
        return -math.inf
    return math.log((1.0 - recall) / n_keys)


def log_threshold_blasst(tau: float) -> float:
    """BLASST compares tile max minus running max with ``ln(tau)``; ``tau == 0`` never skips."""
    if not (0.0 <= tau <= 1.0):
        raise ValueError("tau must lie in [0, 1]")
    return -math.inf if tau == 0.0 else math.log(tau)


def _logsumexp_rows(x: np.ndarray) -> np.ndarray:
    """Row-wise ln(sum(exp(x))) computed as max + ln(sum(exp(x - max)))."""
    mx = x.max(axis=1)
    return mx + np.log(np.exp(x - mx[:, None]).sum(axis=1))


def dense_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float) -> np.ndarray:
    """Textbook softmax attention ``softmax(scale Q K^T) V`` for one head, float64."""
    s = scale * (q @ k.T)
    p = np.exp(s - s.max(axis=1, keepdims=True))
    return (p / p.sum(axis=1, keepdims=True)) @ v


@dataclass
class QTileResult:
    """Everything the oracle records for one query tile."""

    skip: np.ndarray          # bool [T_c]: decision per key tile
    margin: np.ndarray        # float64 [T_c]: max over rows of (t - threshold); skip iff < 0
    tmetric: np.ndarray       # float64 [rows, T_c]: per-row metric t at decision time
    lse_kept: np.ndarray      # float64 [rows]: LSE over kept keys
    lse_all: np.ndarray       # float64 [rows]: LSE over all keys
    o_sparse: np.ndarray      # float64 [rows, d]: output renormalised over kept keys
    o_dense: np.ndarray       # float64 [rows, d]: dense softmax attention output
    kept_cols: np.ndarray = field(default=None)  # int64 indices of kept keys

    @property
    def recall(self) -> np.ndarray:
        return np.exp(self.lse_kept - self.lse_all)


def filter_q_tile(s: np.ndarray, v: np.ndarray, rule: str, threshold: float, tile_k: int,
                  forced_skip=None, order=None) -> QTileResult:
    """Run the tile loop for one query tile.

    ``s``: float64 [rows, N] scaled logits of the tile's valid rows; ``v``: float64 [N, d].
    ``threshold``: lambda (DynSparse) or ln(tau) (BLASST), natural-log units; ignored for
    dense.  ``forced_skip`` (bool [T_c]) makes the loop take those decisions instead of its
    own while still recording its own margins (used to compare against another run's
    decisions without letting one near-tie change every later decision).  ``order``: the
    sequence in which key tiles are visited (default ascending); the running LSE and max
    cover the tiles kept earlier in that sequence.  Results are indexed by key tile.
    """
    if rule not in RULES:
        raise ValueError(f"unknown rule {rule!r}")
    rows, n = s.shape
    n_kt = -(-n // tile_k)
    order = list(range(n_kt)) if order is None else [int(j) for j in order]
    if sorted(order) != list(range(n_kt)):
        raise ValueError("order must visit every key tile exactly once")
    lse = np.full(rows, -np.inf)      # LSE over kept tiles so far (Eq. 6)
    m_run = np.full(rows, -np.inf)    # running max over kept tiles
    skip = np.zeros(n_kt, dtype=bool)
    margin = np.zeros(n_kt)
    tmetric = np.zeros((rows, n_kt))
    kept = []
    for j in order:
        cols = slice(j * tile_k, min(n, (j + 1) * tile_k))
        blk = s[:, cols]
        m_hat = blk.max(axis=1)
        if rule == "dynsparse":
            t = m_hat - lse                      # Eq. 5
        elif rule == "blasst":
            t = m_hat - m_run
        else:
            t = np.full(rows, np.inf)
        tmetric[:, j] = t
        if rule == "dense":
            margin[j] = np.inf
        else:
            margin[j] = np.max(t) - threshold
        decided = bool(margin[j] < 0)
        skip[j] = decided if forced_skip is None else bool(forced_skip[j])
        if not skip[j]:
            lse = np.logaddexp(lse, _logsumexp_rows(blk))
            m_run = np.maximum(m_run, m_hat)
            kept.append(np.arange(cols.start, cols.stop))
    kept_cols = np.concatenate(kept) if kept else np.zeros(0, dtype=np.int64)
    o_sparse = np.exp(s[:, kept_cols] - lse[:, None]) @ v[kept_cols]
    lse_all = _logsumexp_rows(s)
    o_dense = np.exp(s - lse_all[:, None]) @ v
    return QTileResult(skip, margin, tmetric, lse, lse_all, o_sparse, o_dense, kept_cols)


@dataclass
class RuleRun:
    """Oracle results over a set of (b, h, Q-tile) triples."""

    tiles: list                  # list of (b, h, qi)
    results: list                # list of QTileResult, same order
    row_ranges: list             # list of (row_start, row_stop)
    tile_q: int
    tile_k: int
    N: int

    def stats(self, B, H):
        """Per-(b, h) counters {tiles_total, tiles_skipped, elems_total, elems_skipped}
        over the covered Q tiles (all tiles if the run covered every tile)."""
        out = np.zeros((B, H, 4), dtype=np.int64)
        for (b, h, _), res, (r0, r1) in zip(self.tiles, self.results, self.row_ranges):
            nrows = r1 - r0
            widths = np.array([min(self.N, (j + 1) * self.tile_k) - j * self.tile_k
                               for j in range(len(res.skip))])
            out[b, h, 0] += len(res.skip)
            out[b, h, 1] += int(res.skip.sum())
            out[b, h, 2] += int(nrows * widths.sum())
            out[b, h, 3] += int(nrows * widths[res.skip].sum())
        return out


def diagonal_first_order(n_kt: int, start: int) -> list:
    """Key tiles ranked by their distance from ``start``: the start tile, then the tile
    after it, the tile before it, two after, two before, and so on; once one side runs out
    the other continues in order.  (A reading of the "diagonal-first" key order: for
    self-attention the tiles around a query tile's own position come first.)"""
    if not 0 <= start < n_kt:
        raise ValueError("start must be a key tile")

    def rank(t):
        if t == start:
            return 0
        return 2 * (t - start) - 1 if t > start else 2 * (start - t)

    return sorted(range(n_kt), key=rank)


def _as_f64(x: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) upcast exactly, or values already given as floats."""
    return bf16_to_f64(x) if x.dtype == np.uint16 else np.asarray(x, dtype=np.float64)


def rule_attention(q_bits, k_bits, v_bits, scale, rule, threshold, tile_q, tile_k,
                   tiles=None, forced_mask=None, key_order="ascending",
                   order_rows=128) -> RuleRun:
    """Run the oracle on bf16 inputs ``[B][H][N][d]`` (uint16 bit patterns; q and k may
    instead be float arrays, e.g. dequantised MX-FP8 values).

    ``tiles``: iterable of (b, h, qi) to evaluate (default: every query tile of every
    head).  ``forced_mask``: optional uint8/bool array [B][H][T_r][T_c] of decisions to
    follow (see ``filter_q_tile``).  ``key_order``: "ascending" or "diagonal"; the
    diagonal order of a query tile starts at the key tile holding the first row of the
    ``order_rows``-row block that contains the query tile (so query tiles smaller than
    that block share one order).
    """
    if key_order not in ("ascending", "diagonal"):
        raise ValueError(f"unknown key order {key_order!r}")
    B, H, N, d = q_bits.shape
    n_qt = -(-N // tile_q)
    if tiles is None:
        tiles = [(b, h, i) for b in range(B) for h in range(H) for i in range(n_qt)]
    tiles = list(tiles)
    results, ranges = [], []
    cache_bh, k64, v64 = None, None, None
    for (b, h, qi) in tiles:
        if cache_bh != (b, h):
            k64 = _as_f64(k_bits[b, h])
            v64 = _as_f64(v_bits[b, h])
            cache_bh = (b, h)
        r0, r1 = qi * tile_q, min(N, (qi + 1) * tile_q)
        q64 = _as_f64(q_bits[b, h, r0:r1])
        s = scale * (q64 @ k64.T)
        forced = None if forced_mask is None else np.asarray(forced_mask[b, h, qi]).astype(bool)
        order = None
        if key_order == "diagonal":
            block_row0 = (r0 // order_rows) * order_rows
            order = diagonal_first_order(-(-N // tile_k), block_row0 // tile_k)
        results.append(filter_q_tile(s, v64, rule, threshold, tile_k, forced, order))
        ranges.append((r0, r1))
    return RuleRun(tiles, results, ranges, tile_q, tile_k, N)
