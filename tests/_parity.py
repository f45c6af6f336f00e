"""Shared helpers of the GPU parity tests: run a rule through the C ABI and compare it with
the oracle, teacher-forced on the GPU's own skip decisions."""

from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

import oracle

TILE_Q, TILE_K = 128, 64
MARGIN_TOL = 1e-3       # decisions may differ only where |oracle margin| < this
O_MAX_ABS = 2e-2        # output tolerances against the oracle's sparse output
O_REL_L2 = 1e-2
LSE_ABS = 2e-3


def to_device(bits: np.ndarray):
    import torch

    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).cuda()


def from_device_bf16(t) -> np.ndarray:
    import torch

    return t.view(torch.int16).cpu().numpy().view(np.uint16)


RULE_NAMES = {"dense": 0, "blasst": 1, "dynsparse_recall": 2, "dynsparse_lambda": 3}


@dataclass
class DeviceRun:
    o: np.ndarray        # uint16 [B,H,N,d]
    mask: np.ndarray     # uint8 [B,H,n_qt,n_kt]
    lse: np.ndarray      # float32 [B,H,N]
    stats: np.ndarray    # int64 [B,H,4]


def run_gpu(qd, kd, vd, rule: str, param: float, scale: float, tile_q: int = TILE_Q,
            tile_k: int = TILE_K, key_order: int = 0) -> DeviceRun:
    import torch
    import paper_2606_16317_amd as dsa

    B, H, N, d = qd.shape
    n_qt, n_kt = -(-N // tile_q), -(-N // tile_k)
    o = torch.empty_like(qd)
    stats = torch.full((B * H * 4,), -7, dtype=torch.int64, device=qd.device)
    mask = torch.full((B * H * n_qt * n_kt,), 7, dtype=torch.uint8, device=qd.device)
    lse = torch.full((B * H * N,), float("nan"), dtype=torch.float32, device=qd.device)
    dsa.dsattn_attn_fwd_ex(RULE_NAMES[rule], param, qd, kd, vd, o, scale=scale, tile_q=tile_q,
                           tile_k=tile_k, stats_out=stats, mask_out=mask, lse_out=lse,
                           key_order=key_order)
    torch.cuda.synchronize()
    return DeviceRun(from_device_bf16(o), mask.cpu().numpy().reshape(B, H, n_qt, n_kt),
                  lse.cpu().numpy().reshape(B, H, N), stats.cpu().numpy().reshape(B, H, 4))


def oracle_rule(rule: str, param: float, N: int):
    """(oracle rule name, natural-log threshold) for a C-ABI rule and parameter."""
    if rule == "dense":
        return "dense", 0.0
    if rule == "blasst":
        return "blasst", oracle.log_threshold_blasst(param)
    if rule == "dynsparse_recall":
        return "dynsparse", oracle.lambda_from_recall(param, N)
    return "dynsparse", param


def expected_stats_from_mask(mask: np.ndarray, N: int, tile_q: int = TILE_Q,
                             tile_k: int = TILE_K) -> np.ndarray:
    """Counters implied by a full skip mask [B,H,n_qt,n_kt]."""
    B, H, n_qt, n_kt = mask.shape
    rows = np.array([min(N, (i + 1) * tile_q) - i * tile_q for i in range(n_qt)], dtype=np.int64)
    cols = np.array([min(N, (j + 1) * tile_k) - j * tile_k for j in range(n_kt)], dtype=np.int64)
    area = rows[:, None] * cols[None, :]
    m = mask.astype(bool)
    out = np.zeros((B, H, 4), dtype=np.int64)
    out[..., 0] = n_qt * n_kt
    out[..., 1] = m.sum(axis=(2, 3))
    out[..., 2] = N * N
    out[..., 3] = (m * area).sum(axis=(2, 3))
    return out


@dataclass
class Report:
    tiles: int
    pairs: int
    mismatches: int
    max_mismatch_margin: float
    max_abs: float
    rel_l2: float
    rel_l2_vs_dense: float
    sparsity: float
    lse_max_err: float
    near: int = 0          # pairs whose oracle margin lies within the tolerance band


def compare(q, k, v, g: DeviceRun, rule: str, param: float, scale: float, tiles=None,
            tile_q: int = TILE_Q, key_order: str = "ascending", tile_k: int = TILE_K) -> Report:
    """Teacher-forced comparison of a GPU run with the oracle over ``tiles`` (b, h, qi),
    where qi counts query tiles of ``tile_q`` rows (the decision unit)."""
    B, H, N, d = q.shape
    name, thr = oracle_rule(rule, param, N)
    run = oracle.rule_attention(q, k, v, scale, name, thr, tile_q, tile_k, tiles=tiles,
                                forced_mask=g.mask, key_order=key_order)
    mism, worst, near = 0, 0.0, 0
    num = den = dnum = 0.0
    max_abs = lse_err = 0.0
    pairs = 0
    for (b, h, qi), res, (r0, r1) in zip(run.tiles, run.results, run.row_ranges):
        own = res.margin < 0
        bad = own != res.skip
        mism += int(bad.sum())
        near += int((np.abs(res.margin) < MARGIN_TOL).sum())
        if bad.any():
            worst = max(worst, float(np.abs(res.margin[bad]).max()))
        pairs += res.skip.size
        go = oracle.bf16_to_f64(g.o[b, h, r0:r1])
        diff = go - res.o_sparse
        max_abs = max(max_abs, float(np.abs(diff).max()))
        num += float((diff ** 2).sum())
        den += float((res.o_sparse ** 2).sum())
        dnum += float(((go - res.o_dense) ** 2).sum())
        lse_err = max(lse_err, float(np.abs(g.lse[b, h, r0:r1] - res.lse_kept).max()))
    dden = sum(float((r.o_dense ** 2).sum()) for r in run.results)
    return Report(len(run.tiles), pairs, mism, worst, max_abs, math.sqrt(num / den),
                  math.sqrt(dnum / dden), float(np.mean([r.skip.mean() for r in run.results])),
                  lse_err, near)


def assert_parity(rep: Report):
    assert rep.mismatches == 0 or rep.max_mismatch_margin < MARGIN_TOL, rep
    assert rep.max_abs <= O_MAX_ABS, rep
    assert rep.rel_l2 <= O_REL_L2, rep
    assert rep.lse_max_err <= LSE_ABS, rep


def sample_tiles(B, H, N, per_head=3, heads=None, seed=0, tile_q=TILE_Q):
    """First, last and random Q tiles of a few heads."""
    n_qt = -(-N // tile_q)
    rng = np.random.default_rng(seed)
    heads = heads or [(b, h) for b in range(B) for h in range(H)]
    out = []
    for (b, h) in heads:
        picks = {0, n_qt - 1}
        while len(picks) < min(n_qt, per_head):
            picks.add(int(rng.integers(0, n_qt)))
        out += [(b, h, i) for i in sorted(picks)]
    return out
