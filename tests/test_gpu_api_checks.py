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


def test_reordered_workspace_and_index_overlaps_are_rejected():
    """The reordered entry point gathers into its workspace, runs the kernel over it and
    scatters back: a workspace that aliases any other argument buffer, or an index array
    that aliases an output, is rejected on the host before anything is enqueued."""
    import torch
    import paper_2606_16317_amd as dsa

    print("\n[case] reordered overlap checks", flush=True)
    N, BH = 256, 2
    elems = BH * N * 128
    pool = torch.zeros(8 * elems, dtype=torch.bfloat16, device="cuda")
    base = pool.data_ptr()
    t = lambda i: base + i * elems * 2
    q, k, v, o = t(0), t(1), t(2), t(3)
    need = dsa.dsattn_reordered_workspace_bytes(1, BH, N, 128, with_lse=True)
    ws = torch.empty(need + 4096, dtype=torch.uint8, device="cuda")
    w0 = ws.data_ptr()
    idx = torch.arange(N, dtype=torch.int32, device="cuda")
    extra = torch.zeros(64 * 1024, dtype=torch.uint8, device="cuda")
    e0 = extra.data_ptr()

    def run(q_index=idx.data_ptr(), kv_index=idx.data_ptr(), workspace=w0, **kw):
        a = args_for(dsa, q, k, v, o, N, **kw)
        rc = dsa.lib().dsattn_attn_fwd_reordered(ctypes.byref(a), ctypes.c_void_p(q_index),
                                                 ctypes.c_void_p(kv_index),
                                                 ctypes.c_void_p(workspace),
                                                 ctypes.c_size_t(need))
        return rc, dsa.last_error()

    cases = [
        (dict(lse_out=w0 + 256), "workspace must not overlap lse_out"),
        (dict(mask_out=w0 + 512), "workspace must not overlap mask_out"),
        (dict(stats_out=w0 + 1024), "workspace must not overlap stats_out"),
        (dict(rule=dsa.RULE_MASK, mask_in=w0 + 2048), "workspace must not overlap mask_in"),
        (dict(q_index=w0 + 4096), "workspace must not overlap q_index"),
        (dict(kv_index=w0 + 8192), "workspace must not overlap kv_index"),
        (dict(workspace=o + 256), "workspace must not overlap o"),
        (dict(q_index=e0, lse_out=e0), "lse_out must not overlap q_index"),
        (dict(kv_index=e0 + 8, mask_out=e0), "mask_out must not overlap kv_index"),
        (dict(q_index=e0 + 16, stats_out=e0), "stats_out must not overlap q_index"),
        (dict(q_index=o + 128), "o must not overlap q_index"),
    ]
    for kw, msg in cases:
        rc, err = run(**kw)
        assert rc == -1 and msg in err, (kw, rc, err)
    # disjoint buffers are accepted
    rc, err = run(lse_out=e0, stats_out=e0 + 32 * 1024)
    torch.cuda.synchronize()
    assert rc == 0, err
