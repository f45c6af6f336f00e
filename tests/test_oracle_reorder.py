"""Pins of the oracle's spatio-temporal token order (``oracle.reorder``).

The blocked order is pinned by orders worked out by hand, by closed forms that hold for
degenerate block shapes (a block as large as the grid, single-point blocks, whole-frame
blocks, single-column blocks = a transpose of the grid), and by structural invariants:
the map is a permutation, every complete block occupies a contiguous run of positions
inside its own box, and gather/scatter undo each other.
"""

import itertools

import numpy as np
import pytest

from oracle.reorder import block_order, gather_rows, inverse_permutation, scatter_rows


def test_hand_worked_3x3_grid_2x2_blocks():
    # Grid (1, 3, 3), tokens numbered y*3 + x:
    #   0 1 2
    #   3 4 5
    #   6 7 8
    # Blocks of 2x2 in row-major block order: {0,1,3,4}, {2,5}, {6,7}, {8}.
    assert block_order((1, 3, 3), (1, 2, 2)).tolist() == [0, 1, 3, 4, 2, 5, 6, 7, 8]


def test_hand_worked_time_blocks():
    # Grid (3, 1, 2), tokens t*2 + x; blocks 2 x 1 x 1: (t 0-1, x 0), (t 0-1, x 1), then the
    # clipped last slab (t 2, x 0), (t 2, x 1).
    assert block_order((3, 1, 2), (2, 1, 1)).tolist() == [0, 2, 1, 3, 4, 5]


@pytest.mark.parametrize("grid", [(2, 3, 5), (4, 4, 4), (1, 7, 3)])
def test_identity_for_degenerate_blocks(grid):
    n = int(np.prod(grid))
    T, Y, X = grid
    ident = list(range(n))
    assert block_order(grid, grid).tolist() == ident              # one block = whole grid
    assert block_order(grid, (1, 1, 1)).tolist() == ident         # single-point blocks
    assert block_order(grid, (1, Y, X)).tolist() == ident         # one frame per block
    assert block_order(grid, (1, 1, X)).tolist() == ident         # one x-row per block
    assert block_order(grid, (T + 3, Y + 1, X + 5)).tolist() == ident  # oversized block


@pytest.mark.parametrize("grid", [(2, 3, 5), (3, 2, 2), (5, 1, 4)])
def test_single_column_blocks_transpose_the_grid(grid):
    # Blocks T x 1 x 1: the order visits (y, x) row-major and, inside, every t: the grid
    # transposed to (Y, X, T).
    T, Y, X = grid
    expect = np.arange(T * Y * X).reshape(T, Y, X).transpose(1, 2, 0).ravel()
    assert np.array_equal(block_order(grid, (T, 1, 1)), expect)


@pytest.mark.parametrize("grid,block", [((21, 45, 80), (2, 8, 8)), ((21, 45, 80), (1, 8, 8)),
                                        ((3, 5, 7), (2, 3, 4)), ((2, 32, 32), (1, 8, 16))])
def test_is_a_permutation_with_inverse(grid, block):
    perm = block_order(grid, block)
    n = int(np.prod(grid))
    assert perm.shape == (n,)
    assert np.array_equal(np.sort(perm), np.arange(n))
    inv = inverse_permutation(perm)
    assert np.array_equal(perm[inv], np.arange(n))
    assert np.array_equal(inv[perm], np.arange(n))


@pytest.mark.parametrize("grid,block", [((4, 6, 10), (2, 3, 4)), ((3, 5, 7), (2, 2, 3))])
def test_blocks_are_contiguous_boxes(grid, block):
    """Each block's tokens fill one contiguous run of the order, in row-major order, and lie
    inside that block's box; runs follow row-major block order."""
    T, Y, X = grid
    bt, by, bx = block
    perm = block_order(grid, block)
    pos = 0
    for t0, y0, x0 in itertools.product(range(0, T, bt), range(0, Y, by), range(0, X, bx)):
        box = [(t * Y + y) * X + x
               for t in range(t0, min(T, t0 + bt))
               for y in range(y0, min(Y, y0 + by))
               for x in range(x0, min(X, x0 + bx))]
        run = perm[pos:pos + len(box)].tolist()
        assert run == box
        pos += len(box)
    assert pos == T * Y * X


def test_gather_scatter_roundtrip():
    rng = np.random.default_rng(3)
    x = rng.integers(0, 65535, size=(2, 3, 60, 5)).astype(np.uint16)
    perm = block_order((3, 4, 5), (2, 2, 2))
    g = gather_rows(x, perm)
    assert np.array_equal(g[:, :, 7], x[:, :, perm[7]])
    assert np.array_equal(scatter_rows(g, perm), x)
    assert np.array_equal(gather_rows(x, inverse_permutation(perm)), scatter_rows(x, perm))


def test_rejects_bad_extents():
    with pytest.raises(ValueError):
        block_order((0, 2, 2), (1, 1, 1))
    with pytest.raises(ValueError):
        block_order((2, 2, 2), (1, 0, 1))
