"""GPU 32-key decisions on inputs where the second half of a tile passes the threshold
against the state before the tile and fails it once the first half is counted
(``synth.half_flip``).

Section 3.1 decides each 32-key block against the state that includes every block kept
before it, so such an h1 must be skipped.  The kernel may settle h1 before the tile when
it is certain whatever h0 adds (BLASST exactly, DynSparse through a bound on the LSE) and
otherwise decides it mid-step; the tile kinds exercise both ways, a skipped h0 with a kept
h1, and a skipped tile.  Every designed margin is at least 1.2, so the kernel's mask must
equal the designed one exactly, for both decision units, exact and ragged lengths, and
the teacher-forced parity with the oracle must hold.
"""

import math
import sys

import numpy as np
import pytest

from synth import half_flip_inputs

from _parity import assert_parity, compare, expected_stats_from_mask, run_gpu, to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_16317_amd as dsa

    dsa.lib()               # raises if the HIP library is not built


def announce(msg):
    print(f"\n[case] {msg}", flush=True)
    sys.stdout.flush()


CASES = [("dynsparse_lambda", -6.0, "dynsparse", -6.0),
         ("dynsparse_lambda", -12.0, "dynsparse", -12.0),
         ("blasst", 1e-2, "blasst", math.log(1e-2)),
         ("blasst", 1e-3, "blasst", math.log(1e-3))]


@pytest.mark.parametrize("T,n_tail", [(24, 0), (20, 20)])
@pytest.mark.parametrize("tile_q", [128, 32])
@pytest.mark.parametrize("rule,param,oname,thr", CASES)
def test_half_flip_decisions(T, n_tail, tile_q, rule, param, oname, thr):
    H = 4
    q, k, v, kinds, skip, scale = half_flip_inputs(T, H, oname, thr, seed=7 + T,
                                                   n_tail=n_tail)
    N = q.shape[2]
    announce(f"half flip N={N} tile_q={tile_q} rule={rule} param={param}")
    g = run_gpu(to_device(q), to_device(k), to_device(v), rule, param, scale, tile_q=tile_q,
                tile_k=32)
    assert (g.stats == expected_stats_from_mask(g.mask, N, tile_q, 32)).all()
    for h in range(H):
        assert (g.mask[0, h] == skip[h][None, :]).all(), (h, g.mask[0, h, 0], skip[h])
    rep = compare(q, k, v, g, rule, param, scale, tile_q=tile_q, tile_k=32)
    print(rep, flush=True)
    assert rep.mismatches == 0
    assert_parity(rep)
