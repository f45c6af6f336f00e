"""CPU oracle of the spatio-temporal token reordering that precedes the attention loop.

TEST INFRASTRUCTURE ONLY (same rule as ``oracle.attention``: imported by ``tests/``,
``__graft_entry__.smoke()`` and ``bench.py``'s CPU baseline leg only).

Section 3.1 (end of the hyperparameter-selection paragraph) notes that mapping the
flattened token sequence back to its spatio-temporal layout before the attention raises
the correlation inside a tile; Section 1 (related work) describes the same grouping of tokens
that are close in time and space into one block.  The paper fixes no block shape, so the
order is parameterised by one: the T x Y x X latent grid (tokens row-major, x fastest) is
cut into blocks of bt x by x bx grid points (the last block along an axis may be
shorter), blocks are visited in row-major block order, and the tokens of a block in
row-major order inside the block.

``block_order`` returns the gather map ``perm``: position ``i`` of the reordered sequence
holds original token ``perm[i]``.  Attention over reordered queries and keys gives, for
reordered query ``i``, the output of original query ``perm[i]``; scattering rows back
(``out[perm[i]] = out_reordered[i]``) restores the original order.

Parity status: pinned by ``tests/test_oracle_reorder.py`` (hand-worked small orders,
closed forms for degenerate block shapes, bijectivity, block locality).
"""

from __future__ import annotations

import numpy as np


def block_order(grid, block) -> np.ndarray:
    """Gather map of the blocked order of a row-major T x Y x X token grid (int64 [N])."""
    T, Y, X = (int(g) for g in grid)
    bt, by, bx = (int(b) for b in block)
    if min(T, Y, X) <= 0 or min(bt, by, bx) <= 0:
        raise ValueError("grid and block extents must be positive")
    out = []
    for t0 in range(0, T, bt):
        for y0 in range(0, Y, by):
            for x0 in range(0, X, bx):
                for t in range(t0, min(T, t0 + bt)):
                    for y in range(y0, min(Y, y0 + by)):
                        for x in range(x0, min(X, x0 + bx)):
                            out.append((t * Y + y) * X + x)
    return np.asarray(out, dtype=np.int64)


def inverse_permutation(perm: np.ndarray) -> np.ndarray:
    """``inv`` with ``inv[perm[i]] = i``."""
    perm = np.asarray(perm, dtype=np.int64)
    inv = np.empty_like(perm)
    inv[perm] = np.arange(perm.size, dtype=np.int64)
    return inv


def gather_rows(x: np.ndarray, index: np.ndarray) -> np.ndarray:
    """``out[..., i, :] = x[..., index[i], :]`` over the sequence axis (axis -2)."""
    return np.ascontiguousarray(np.take(x, np.asarray(index, dtype=np.int64), axis=-2))


def scatter_rows(x: np.ndarray, index: np.ndarray) -> np.ndarray:
    """``out[..., index[i], :] = x[..., i, :]``: undoes ``gather_rows`` with the same map."""
    out = np.empty_like(x)
    out[..., np.asarray(index, dtype=np.int64), :] = x
    return out
