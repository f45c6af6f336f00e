"""Video-shaped Q/K/V generator (bf16 bit patterns, [B][H][N][d] row-major).

The paper evaluates on attention layers of Wan 2.2 video diffusion transformers
(Section 4.1); neither the model weights nor the VBench prompts are available here, so
these seeded inputs stand in for them.  Tokens are laid out row-major over a
T x Y x X latent video grid, as a video DiT flattens them, and queries/keys carry a
shared positional signal so that attention concentrates on spatio-temporal neighbours.

Recipe (d = 128):

* token i <-> integer grid point p = (t, y, x), row-major (x fastest);
* u(p) in R^128: for each axis in (t, y, x), 21 frequency pairs
  [sin(w_k * coord), cos(w_k * coord)] with w_k = 10000^(-k/21), k = 0..20
  (axis-major: t features in u[0:42], y in u[42:84], x in u[84:126]),
  then two zero pads u[126:128];
* per head a concentration a and a head type: "spatial" heads zero the t block of u,
  "temporal" heads keep the full u;
* Q = a*u + 0.5*e, K = a*u + 0.5*e', V = n with e, e', n ~ N(0, 1) i.i.d.;
* every value is formed in float32 and rounded to bf16 with round-to-nearest-even.

Randomness: ``np.random.SeedSequence(seed).spawn(1 + B*H)``.  Child 0 draws the per-head
concentrations (U[a_lo, a_hi]) and a permutation that makes exactly half the heads
spatial (``perm[h] < H//2``); heads are shared across the batch.  Child 1 + b*H + h
draws e, e', n for head (b, h), in that order, as float32 standard normals.

No attention arithmetic lives here.
"""

from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np

D_MODEL_HEAD = 128
N_FREQ = 21


@dataclass(frozen=True)
class Workload:
    """One synthetic attention layer: shape, grid, concentration law and seed."""

    name: str
    B: int
    H: int
    grid: tuple  # (T, Y, X)
    a_lo: float
    a_hi: float
    mixed_heads: bool  # False: every head uses the full u (t, y, x)
    seed: int
    recall: float = 0.95
    d: int = D_MODEL_HEAD

    @property
    def N(self) -> int:
        t, y, x = self.grid
        return t * y * x

    def describe(self) -> str:
        t, y, x = self.grid
        return (f"{self.name}: B={self.B} H={self.H} N={self.N} ({t}x{y}x{x}) d={self.d} "
                f"a~U[{self.a_lo},{self.a_hi}] seed={self.seed}")


# The five layer shapes: a tiny single head, Wan-2.2-14B-like 480p and 720p layers, a
# 720p threshold-sweep draw and a long low-concentration stress layer.
WORKLOADS = {
    "tiny": Workload("tiny", 1, 1, (2, 32, 32), 2.0, 2.0, False, 0),
    "wan480p": Workload("wan480p", 1, 40, (21, 30, 52), 1.0, 3.0, True, 1),
    "wan720p": Workload("wan720p", 1, 40, (21, 45, 80), 1.0, 3.0, True, 2),
    "wan720p_sweep": Workload("wan720p_sweep", 1, 40, (21, 45, 80), 1.0, 3.0, True, 3),
    "stress": Workload("stress", 2, 8, (32, 64, 64), 0.25, 3.0, True, 4),
}


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bf16 (nearest, ties to even); return the uint16 bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32)
    r = b + (np.uint32(0x7FFF) + ((b >> np.uint32(16)) & np.uint32(1)))
    return (r >> np.uint32(16)).astype(np.uint16)


def position_features(grid, d: int = D_MODEL_HEAD) -> tuple:
    """Return (u_full, u_spatial), float32 [N][d]: sinusoidal features of each grid point."""
    if d < 6 * N_FREQ:
        raise ValueError(f"d={d} too small for {6 * N_FREQ} positional features")
    T, Y, X = grid
    t, y, x = np.meshgrid(np.arange(T), np.arange(Y), np.arange(X), indexing="ij")
    coords = [c.reshape(-1).astype(np.float64) for c in (t, y, x)]
    w = 10000.0 ** (-np.arange(N_FREQ, dtype=np.float64) / N_FREQ)
    n = T * Y * X
    u = np.zeros((n, d), dtype=np.float64)
    for ax, c in enumerate(coords):
        ang = c[:, None] * w[None, :]
        blk = np.empty((n, 2 * N_FREQ))
        blk[:, 0::2] = np.sin(ang)
        blk[:, 1::2] = np.cos(ang)
        u[:, ax * 2 * N_FREQ:(ax + 1) * 2 * N_FREQ] = blk
    u_full = u.astype(np.float32)
    u_spatial = u_full.copy()
    u_spatial[:, 0:2 * N_FREQ] = 0.0
    return u_full, u_spatial


def _head_params(ss_child0, H, a_lo, a_hi, mixed):
    rng = np.random.default_rng(ss_child0)
    a = rng.uniform(a_lo, a_hi, size=H) if a_hi > a_lo else np.full(H, float(a_lo))
    if mixed:
        perm = rng.permutation(H)
        spatial = perm < (H // 2)
    else:
        spatial = np.zeros(H, dtype=bool)
    return a, spatial


def make_video_qkv(B, H, grid, a_lo, a_hi, mixed_heads, seed, d=D_MODEL_HEAD,
                   threads=None):
    """Draw video-shaped bf16 Q, K, V of shape [B][H][N][d] (uint16 bit patterns).

    Returns (q, k, v, meta) where meta holds the per-head concentration ``a`` and the
    boolean ``spatial`` head-type vector.
    """
    N = int(np.prod(grid))
    children = np.random.SeedSequence(seed).spawn(1 + B * H)
    a, spatial = _head_params(children[0], H, a_lo, a_hi, mixed_heads)
    u_full, u_spat = position_features(grid, d)
    q = np.empty((B, H, N, d), dtype=np.uint16)
    k = np.empty_like(q)
    v = np.empty_like(q)
    half = np.float32(0.5)

    def one(bh):
        b, h = divmod(bh, H)
        rng = np.random.default_rng(children[1 + bh])
        u = u_spat if spatial[h] else u_full
        ah = np.float32(a[h])
        e = rng.standard_normal((N, d), dtype=np.float32)
        q[b, h] = bf16_bits(u * ah + half * e)
        e = rng.standard_normal((N, d), dtype=np.float32)
        k[b, h] = bf16_bits(u * ah + half * e)
        e = rng.standard_normal((N, d), dtype=np.float32)
        v[b, h] = bf16_bits(e)

    nthr = threads or min(8, os.cpu_count() or 1, B * H)
    if nthr > 1:
        with ThreadPoolExecutor(nthr) as ex:
            list(ex.map(one, range(B * H)))
    else:
        for bh in range(B * H):
            one(bh)
    meta = {"a": a, "spatial": spatial, "grid": tuple(grid), "seed": seed}
    return q, k, v, meta


def workload_inputs(name_or_workload, threads=None):
    """Inputs for one of the named workloads (see ``WORKLOADS``)."""
    w = WORKLOADS[name_or_workload] if isinstance(name_or_workload, str) else name_or_workload
    return make_video_qkv(w.B, w.H, w.grid, w.a_lo, w.a_hi, w.mixed_heads, w.seed, w.d,
                          threads=threads)


def make_random_qkv(B, H, N, d, seed, q_std=1.0, k_std=1.0, v_std=1.0):
    """Plain Gaussian bf16 Q, K, V of shape [B][H][N][d] (uint16 bit patterns)."""
    rng = np.random.default_rng(seed)
    q = bf16_bits(np.float32(q_std) * rng.standard_normal((B, H, N, d), dtype=np.float32))
    k = bf16_bits(np.float32(k_std) * rng.standard_normal((B, H, N, d), dtype=np.float32))
    v = bf16_bits(np.float32(v_std) * rng.standard_normal((B, H, N, d), dtype=np.float32))
    return q, k, v
