"""Host-side argument checks that need real device pointers: outputs that overlap an input
or another output are rejected before anything is enqueued; buffers that merely touch
(one ends where the next begins, inside one allocation) are accepted and computed."""

import ctypes
import math
import sys

import numpy as np
import pytest

from synth import make_random_qkv

from _parity import to_device

pytestmark = pytest.mark.gpu

SCALE = 1.0 / math.sqrt(128)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_16317_amd as dsa

    dsa.lib()
    return torch


def args_for(dsa, q, k, v, o, N, **kw):
    a = dsa.DsAttnArgs(dsa.RULE_DYNSPARSE_LAMBDA, -6.0, q, k, v, o, 1, 2, N, 128, SCALE, 128,
                       64, None, None, None, None, 0, None, 0, None, None)
    for key, val in kw.items():
        setattr(a, key, val)
    return a


def call(dsa, a):
    return dsa.lib().dsattn_attn_fwd_ex(ctypes.byref(a)), dsa.last_error()


def test_overlapping_outputs_are_rejected():
    import torch
    import paper_2606_16317_amd as dsa

    print("\n[case] overlap checks", flush=True)
    N = 256
    elems = 2 * N * 128                               # one [1, 2, N, 128] bf16 tensor
    pool = torch.zeros(6 * elems, dtype=torch.bfloat16, device="cuda")
    base = pool.data_ptr()
    t = lambda i: base + i * elems * 2                 # byte address of tensor slot i
    q, k, v, o = t(0), t(1), t(2), t(3)
    # o starting half-way into v
    rc, err = call(dsa, args_for(dsa, q, k, v, v + elems, N))
    assert rc == -1 and "o must not overlap v" in err
    # lse_out inside o
    rc, err = call(dsa, args_for(dsa, q, k, v, o, N, lse_out=o + 1024))
    assert rc == -1 and "lse_out must not overlap o" in err
    # stats_out inside q
    rc, err = call(dsa, args_for(dsa, q, k, v, o, N, stats_out=q + 4096))
    assert rc == -1 and "stats_out must not overlap q" in err
    # mask_out over mask_in (mask reuse)
    m = t(4)
    rc, err = call(dsa, args_for(dsa, q, k, v, o, N, rule=dsa.RULE_MASK, mask_in=m,
                                 mask_out=m + 2))
    assert rc == -1 and "mask_out must not overlap mask_in" in err
    # mask_out over lse_out
    rc, err = call(dsa, args_for(dsa, q, k, v, o, N, lse_out=t(4), mask_out=t(4) + 64))
    assert rc == -1 and "must not overlap" in err
    torch.cuda.synchronize()


def test_touching_buffers_are_accepted():
    import torch
    import paper_2606_16317_amd as dsa

    print("\n[case] adjacent buffers in one allocation", flush=True)
    N = 256
    q, k, v = make_random_qkv(1, 2, N, 128, 3)
    elems = 2 * N * 128
    pool = torch.zeros(4 * elems + 2 * N * 2, dtype=torch.bfloat16, device="cuda")
    for i, x in enumerate((q, k, v)):
        pool[i * elems:(i + 1) * elems].copy_(to_device(x).reshape(-1))
    base = pool.data_ptr()
    lse = base + 4 * elems * 2                         # right after o
    rc, err = call(dsa, args_for(dsa, base, base + elems * 2, base + 2 * elems * 2,
                                 base + 3 * elems * 2, N, lse_out=lse))
    torch.cuda.synchronize()
    assert rc == 0, err
    ref = dsa.dsattn_attn_fwd_ex(dsa.RULE_DYNSPARSE_LAMBDA, -6.0, to_device(q), to_device(k),
                                 to_device(v), scale=SCALE)
    torch.cuda.synchronize()
    assert torch.equal(pool[3 * elems:4 * elems], ref.reshape(-1))
