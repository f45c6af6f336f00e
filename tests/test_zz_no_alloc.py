"""The allocation-free reordered entry point (``dsattn_attn_fwd_reordered_noalloc``): its
workspace is the library's static per-GPU scratch.  Called through the C ABI, it must give
the same bits as ``dsattn_attn_fwd_reordered`` with a caller-owned workspace (output, LSE,
skip mask, counters) on two calls in a row, the second smaller than the first; a problem
whose workspace exceeds the static maximum is rejected on the host with nothing enqueued.
"""

import ctypes
import math
import os
import re
import sys

import numpy as np
import pytest

from synth import make_random_qkv, make_video_qkv

from _parity import to_device

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SCALE = 1.0 / math.sqrt(128)


@pytest.fixture(scope="module", autouse=True)
def gpu():
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2606_16317_amd as dsa

    dsa.lib()
    return torch


def announce(msg):
    print(f"\n[case] {msg}", flush=True)
    sys.stdout.flush()


def _run(dsa, fn, q, k, v, qi, ki, rule, param, **extra):
    import torch

    B, H, N, d = q.shape
    n_qt, n_kt = -(-N // 128), -(-N // 64)
    o = torch.full_like(q, float("nan"))
    lse = torch.full((B * H * N,), float("nan"), dtype=torch.float32, device="cuda")
    mask = torch.full((B * H * n_qt * n_kt,), 7, dtype=torch.uint8, device="cuda")
    stats = torch.full((B * H * 4,), -1, dtype=torch.int64, device="cuda")
    fn(rule, param, q, k, v, qi, ki, o, scale=SCALE, stats_out=stats, mask_out=mask,
       lse_out=lse, **extra)
    torch.cuda.synchronize()
    return o, lse, mask, stats


def _same(a, b):
    import torch

    for x, y in zip(a, b):
        if x.dtype == torch.bfloat16:
            x, y = x.view(torch.int16), y.view(torch.int16)
        assert torch.equal(x, y)


def test_header_limit_matches_binding():
    import paper_2606_16317_amd as dsa

    text = open(os.path.join(ROOT, "include", "dsattn.h")).read()
    m = re.search(r"#define DSATTN_STATIC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == dsa.STATIC_SCRATCH_BYTES


def test_noalloc_matches_caller_workspace_twice():
    import torch
    import paper_2606_16317_amd as dsa

    # first call: four peaked video heads (real skips), blocked order, lambda = -6
    grid = (4, 24, 32)
    q, k, v, _ = make_video_qkv(1, 4, grid, 3.0, 6.0, True, 91)
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    qi = torch.from_numpy(dsa.dsattn_block_order(grid, (2, 8, 8))).cuda()
    ki = torch.from_numpy(dsa.dsattn_block_order(grid, (1, 8, 8))).cuda()
    need = dsa.dsattn_reordered_workspace_bytes(1, 4, qd.shape[2], 128, True)
    assert need <= dsa.STATIC_SCRATCH_BYTES
    announce(f"noalloc call 1: N={qd.shape[2]} H=4 workspace={need}")
    ref = _run(dsa, dsa.dsattn_attn_fwd_reordered, qd, kd, vd, qi, ki,
               dsa.RULE_DYNSPARSE_LAMBDA, -6.0)
    got = _run(dsa, dsa.dsattn_attn_fwd_reordered_noalloc, qd, kd, vd, qi, ki,
               dsa.RULE_DYNSPARSE_LAMBDA, -6.0)
    _same(ref, got)
    assert 0.05 < float(got[2].float().mean()) < 0.95          # some tiles skipped
    assert not torch.isnan(got[1]).any()

    # second call, smaller and ragged (N = 1000, random order), another rule
    q, k, v = make_random_qkv(1, 2, 1000, 128, 92, q_std=1.5, k_std=1.5)
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    g = torch.Generator().manual_seed(5)
    qi = torch.randperm(1000, generator=g).to(torch.int32).cuda()
    ki = torch.randperm(1000, generator=g).to(torch.int32).cuda()
    announce("noalloc call 2: N=1000 H=2 random order, BLASST 0.05")
    ref = _run(dsa, dsa.dsattn_attn_fwd_reordered, qd, kd, vd, qi, ki, dsa.RULE_BLASST, 0.05)
    got = _run(dsa, dsa.dsattn_attn_fwd_reordered_noalloc, qd, kd, vd, qi, ki,
               dsa.RULE_BLASST, 0.05)
    _same(ref, got)
    assert not torch.isnan(got[1]).any()


def test_noalloc_rejects_problems_beyond_the_scratch():
    import torch
    import paper_2606_16317_amd as dsa

    N = 100_000      # 4 x 25.6 MB of reordered copies: more than the 96 MiB scratch
    need = dsa.dsattn_reordered_workspace_bytes(1, 1, N, 128, False)
    assert need > dsa.STATIC_SCRATCH_BYTES
    announce(f"noalloc too large: N={N} workspace={need}")
    q, k, v, o = (torch.zeros((1, 1, N, 128), dtype=torch.bfloat16, device="cuda")
                  for _ in range(4))
    idx = torch.arange(N, dtype=torch.int32, device="cuda")
    a = dsa.DsAttnArgs(dsa.RULE_DENSE, 0.0, q.data_ptr(), k.data_ptr(), v.data_ptr(),
                       o.data_ptr(), 1, 1, N, 128, SCALE, 128, 64, None, None, None, None, 0,
                       None, 0, None, None)
    o.fill_(1.0)
    torch.cuda.synchronize()
    rc = dsa.lib().dsattn_attn_fwd_reordered_noalloc(ctypes.byref(a), idx.data_ptr(),
                                                     idx.data_ptr())
    torch.cuda.synchronize()
    assert rc == -1 and "static scratch" in dsa.last_error()
    assert bool((o == 1.0).all())                  # nothing was launched
