"""HIP graph capture of the C-ABI calls (torch.cuda.CUDAGraph over the library's kernels).

The library clears stats_out with a fill kernel rather than a memset node, and allocates
nothing, so a call can be captured and replayed.  Each graph is replayed several times
with the program's own eager work and synchronisations in between and with new inputs
copied into the captured buffers; every replay must equal an eager call on the same
inputs bit for bit (the kernels are deterministic).
"""

import math
import sys

import numpy as np
import pytest

from synth import make_random_qkv, make_video_qkv

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


def announce(msg):
    print(f"\n[case] {msg}", flush=True)
    sys.stdout.flush()


def buffers(B, H, N, tile_q=128, tile_k=64):
    import torch

    n_qt, n_kt = -(-N // tile_q), -(-N // tile_k)
    return (torch.empty((B, H, N, 128), dtype=torch.bfloat16, device="cuda"),
            torch.zeros(B * H * 4, dtype=torch.int64, device="cuda"),
            torch.zeros(B * H * n_qt * n_kt, dtype=torch.uint8, device="cuda"),
            torch.zeros(B * H * N, dtype=torch.float32, device="cuda"))


@pytest.mark.parametrize("rule,param,tile_q,tile_k", [(3, -6.0, 128, 64), (1, 1e-2, 32, 64),
                                                      (0, 0.0, 128, 64), (3, -6.0, 128, 128),
                                                      (2, 0.9, 128, 32)])
def test_attention_call_replays_match_eager(rule, param, tile_q, tile_k):
    import torch
    import paper_2606_16317_amd as dsa

    announce(f"graph rule={rule} param={param} tile_q={tile_q} tile_k={tile_k}")
    B, H, N = 1, 3, 1000
    inputs = [make_video_qkv(B, H, (2, 10, 50), 4.0, 4.0, True, s)[:3] for s in (1, 2, 3)]
    qd, kd, vd = (to_device(x) for x in inputs[0])
    o, st, mk, ls = buffers(B, H, N, tile_q, tile_k)

    def call(q, k, v, o, st, mk, ls):
        dsa.dsattn_attn_fwd_ex(rule, param, q, k, v, o, scale=SCALE, tile_q=tile_q,
                               tile_k=tile_k, stats_out=st, mask_out=mk, lse_out=ls)

    call(qd, kd, vd, o, st, mk, ls)                      # warm-up outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(qd, kd, vd, o, st, mk, ls)
    for rep in range(4):
        q, k, v = inputs[rep % 3]
        qd.copy_(to_device(q)); kd.copy_(to_device(k)); vd.copy_(to_device(v))
        st.fill_(-1); mk.fill_(9); o.zero_()
        g.replay()
        ref = buffers(B, H, N, tile_q, tile_k)
        call(to_device(q), to_device(k), to_device(v), *ref)   # eager, other buffers
        torch.cuda.synchronize()
        for got, want in zip((o, st, mk, ls), ref):
            assert torch.equal(got, want), rep


def test_quantise_and_q8_attention_replays_match_eager():
    import torch
    import paper_2606_16317_amd as dsa

    announce("graph quantise + mxfp8 attention")
    B, H, N = 1, 2, 777
    q, k, v = make_random_qkv(B, H, N, 128, 11, q_std=2.0, k_std=2.0)
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    qc = torch.empty((B, H, N, 128), dtype=torch.uint8, device="cuda")
    kc = torch.empty_like(qc)
    qs = torch.empty((B, H, N, 4), dtype=torch.uint8, device="cuda")
    ks = torch.empty_like(qs)
    mean = torch.empty((B, H, 128), dtype=torch.float32, device="cuda")
    o, st, mk, ls = buffers(B, H, N)

    def pipeline(o, st, mk, ls):
        dsa.dsattn_quantize_mxfp8(qd, qc, qs)
        dsa.dsattn_key_mean(kd, mean)
        dsa.dsattn_quantize_mxfp8(kd, kc, ks, shift=mean)
        dsa.dsattn_attn_fwd_mxfp8(3, -4.0, qc, qs, kc, ks, vd, o, scale=SCALE, stats_out=st,
                                  mask_out=mk, lse_out=ls)

    pipeline(o, st, mk, ls)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pipeline(o, st, mk, ls)
    for rep in range(3):
        kd.mul_(1.5 if rep % 2 else 0.75)                 # new keys each replay
        g.replay()
        torch.cuda.synchronize()
        got = [t.clone() for t in (o, st, mk, ls)]
        pipeline(o, st, mk, ls)                           # eager on the same inputs
        torch.cuda.synchronize()
        for a, b in zip(got, (o, st, mk, ls)):
            assert torch.equal(a, b), rep


def test_diagonal_rule_then_mask_reuse_replays_match_eager():
    """One graph holding a DynSparse call in diagonal-first order that writes its mask and
    a mask-reuse call that consumes it: every replay (new inputs each time) equals the
    same two calls run eagerly."""
    import torch
    import paper_2606_16317_amd as dsa

    announce("graph: diagonal-order rule call, then mask reuse")
    B, H, N = 1, 3, 1000
    inputs = [make_video_qkv(B, H, (2, 10, 50), 5.0, 5.0, True, s)[:3] for s in (4, 5, 6)]
    qd, kd, vd = (to_device(x) for x in inputs[0])

    def bufs():
        return (buffers(B, H, N), buffers(B, H, N))

    def pipeline(q, k, v, first, second):
        o1, st1, mk1, ls1 = first
        o2, st2, mk2, ls2 = second
        dsa.dsattn_attn_fwd_ex(dsa.RULE_DYNSPARSE_LAMBDA, -6.0, q, k, v, o1, scale=SCALE,
                               stats_out=st1, mask_out=mk1, lse_out=ls1,
                               key_order=dsa.ORDER_DIAGONAL)
        dsa.dsattn_attn_fwd_ex(dsa.RULE_MASK, 0.0, q, k, v, o2, scale=SCALE, stats_out=st2,
                               mask_out=mk2, lse_out=ls2, mask_in=mk1)

    first, second = bufs()
    pipeline(qd, kd, vd, first, second)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pipeline(qd, kd, vd, first, second)
    for rep in range(4):
        q, k, v = inputs[rep % 3]
        qd.copy_(to_device(q)); kd.copy_(to_device(k)); vd.copy_(to_device(v))
        for t in first + second:
            t.zero_()
        g.replay()
        ref_first, ref_second = bufs()
        pipeline(to_device(q), to_device(k), to_device(v), ref_first, ref_second)
        torch.cuda.synchronize()
        for got, want in zip(first + second, ref_first + ref_second):
            assert torch.equal(got, want), rep
        assert float(first[2].float().mean()) > 0.05           # the first call skipped


def test_reordered_attention_replays_match_eager():
    """The reordered entry point (row gathers, the rule, the output scatter) captured with
    a caller-provided workspace: replays equal eager calls."""
    import torch
    import paper_2606_16317_amd as dsa

    announce("graph: reordered attention")
    B, H, N, grid = 1, 2, 1000, (2, 10, 50)
    inputs = [make_video_qkv(B, H, grid, 5.0, 5.0, True, s)[:3] for s in (7, 8, 9)]
    qd, kd, vd = (to_device(x) for x in inputs[0])
    qi = torch.from_numpy(dsa.dsattn_block_order(grid, (2, 8, 8))).cuda()
    ki = torch.from_numpy(dsa.dsattn_block_order(grid, (1, 8, 8))).cuda()
    ws = torch.empty(dsa.dsattn_reordered_workspace_bytes(B, H, N, 128, True),
                     dtype=torch.uint8, device="cuda")
    ws_ref = torch.empty_like(ws)

    def call(q, k, v, out, work):
        o, st, mk, ls = out
        dsa.dsattn_attn_fwd_reordered(dsa.RULE_DYNSPARSE_LAMBDA, -6.0, q, k, v, qi, ki, o,
                                      scale=SCALE, stats_out=st, mask_out=mk, lse_out=ls,
                                      workspace=work)

    out = buffers(B, H, N)
    call(qd, kd, vd, out, ws)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(qd, kd, vd, out, ws)
    for rep in range(4):
        q, k, v = inputs[rep % 3]
        qd.copy_(to_device(q)); kd.copy_(to_device(k)); vd.copy_(to_device(v))
        for t in out:
            t.zero_()
        g.replay()
        ref = buffers(B, H, N)
        call(to_device(q), to_device(k), to_device(v), ref, ws_ref)
        torch.cuda.synchronize()
        for got, want in zip(out, ref):
            assert torch.equal(got, want), rep


def test_calls_on_two_streams_match_serial_calls():
    """Two different problems enqueued on two streams at once (default priority) give the
    same bits as the same calls run one after the other: the library keeps no state
    between calls besides the caller's buffers."""
    import torch
    import paper_2606_16317_amd as dsa

    announce("two streams")
    B, H, N = 1, 3, 1000
    a = [to_device(x) for x in make_video_qkv(B, H, (2, 10, 50), 5.0, 5.0, True, 11)[:3]]
    b = [to_device(x) for x in make_video_qkv(B, H, (2, 10, 50), 3.0, 3.0, True, 12)[:3]]
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    out_a, out_b = buffers(B, H, N), buffers(B, H, N, tile_q=32)
    torch.cuda.synchronize()
    for _ in range(3):
        with torch.cuda.stream(s1):
            o, st, mk, ls = out_a
            dsa.dsattn_attn_fwd_ex(dsa.RULE_DYNSPARSE_LAMBDA, -6.0, *a, o, scale=SCALE,
                                   stats_out=st, mask_out=mk, lse_out=ls,
                                   stream=s1)
        with torch.cuda.stream(s2):
            o, st, mk, ls = out_b
            dsa.dsattn_attn_fwd_ex(dsa.RULE_BLASST, 1e-2, *b, o, scale=SCALE, tile_q=32,
                                   stats_out=st, mask_out=mk, lse_out=ls,
                                   stream=s2)
    torch.cuda.synchronize()
    ref_a, ref_b = buffers(B, H, N), buffers(B, H, N, tile_q=32)
    o, st, mk, ls = ref_a
    dsa.dsattn_attn_fwd_ex(dsa.RULE_DYNSPARSE_LAMBDA, -6.0, *a, o, scale=SCALE, stats_out=st,
                           mask_out=mk, lse_out=ls)
    o, st, mk, ls = ref_b
    dsa.dsattn_attn_fwd_ex(dsa.RULE_BLASST, 1e-2, *b, o, scale=SCALE, tile_q=32, stats_out=st,
                           mask_out=mk, lse_out=ls)
    torch.cuda.synchronize()
    for got, want in zip(out_a + out_b, ref_a + ref_b):
        assert torch.equal(got, want)
