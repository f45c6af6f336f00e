"""GPU parity of the MX-FP8 path, called through the C ABI, against the CPU oracle.

* Quantisation (``dsattn_quantize_mxfp8``) against ``oracle.mxfp8``: codes and block
  exponents must match bit for bit.  The inputs mix Gaussian rows of several scales,
  all-zero blocks, bf16 subnormals, the largest bf16 magnitudes, values exactly halfway
  between two E4M3 codes after scaling, and blocks whose scaled maximum rounds up to the
  saturation limit.
* Key smoothing: the per-head key mean (``dsattn_key_mean``) against the float64 mean
  within the float32 summation bound of its fixed order, and the shifted quantiser
  (``dsattn_quantize_mxfp8_shift``) bit for bit against ``oracle.mxfp8.smooth_keys`` +
  ``quantize_mxfp8`` with the same float32 shift.
* Attention with MX-FP8 Q and K (DSATTN_QK_MXFP8) against the oracle run on the
  dequantised Q and K (exact float64 values of the codes): the same teacher-forced
  comparison and tolerances as the bf16 path, since S differs from the oracle's only by
  the fp32 rounding of the MFMA sums.
"""

import math
import sys

import numpy as np
import pytest

from oracle import bf16_to_f64
from oracle.mxfp8 import dequantize_mxfp8, key_mean, quantize_mxfp8, smooth_keys
from synth import bf16_bits, make_random_qkv

from _parity import (DeviceRun, RULE_NAMES, assert_parity, compare, expected_stats_from_mask,
                     from_device_bf16, sample_tiles, to_device)

pytestmark = pytest.mark.gpu


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


def edge_rows():
    rows = np.zeros((8, 128))
    rows[1, :32] = 3.0 * 2.0 ** -130                  # bf16 subnormals
    rows[1, 32:64] = np.linspace(-2.0 ** 127, 2.0 ** 127, 32)
    rows[2, :32] = 1.0 + np.arange(32) / 128.0        # mantissas between E4M3 codes
    rows[2, 0] = 256.0                                # scale 2^0: values land on ties
    rows[2, 32:64] = 1.0625                           # tie between 1.0 and 1.125 after scale
    rows[2, 32] = 256.0
    rows[3, :32] = np.arange(32) * (464.0 / 31.0)     # block maximum 464 -> saturates
    rows[3, 32:64] = -rows[3, :32]
    rows[4, :] = 2.0 ** -20 * np.arange(128)          # small magnitudes, subnormal codes
    rows[5, :] = -0.0
    rows[6, ::2] = 1e30
    rows[6, 1::2] = -1e-30
    rows[7, :] = np.tile([448.0, 0.5, -7.0, 2.0 ** -9], 32)
    return bf16_bits(rows.astype(np.float32))


def run(bits):
    import torch
    import paper_2606_16317_amd as dsa

    x = to_device(bits)
    codes, scales = dsa.dsattn_quantize_mxfp8(x)
    torch.cuda.synchronize()
    return codes.cpu().numpy(), scales.cpu().numpy()


def test_quantize_edge_rows_bit_exact():
    announce("mxfp8 edge rows")
    bits = edge_rows()
    codes, scales = run(bits)
    want_c, want_s = quantize_mxfp8(bf16_to_f64(bits))
    np.testing.assert_array_equal(scales, want_s)
    np.testing.assert_array_equal(codes, want_c)


@pytest.mark.parametrize("N,std,seed", [(200, 1.0, 0), (1000, 40.0, 1), (77, 1e-3, 2),
                                        (4096, 3.0, 3)])
def test_quantize_random_qk_bit_exact(N, std, seed):
    announce(f"mxfp8 random N={N} std={std} seed={seed}")
    q, k, _ = make_random_qkv(1, 2, N, 128, seed, q_std=std, k_std=std)
    for bits in (q, k):
        codes, scales = run(bits)
        want_c, want_s = quantize_mxfp8(bf16_to_f64(bits))
        np.testing.assert_array_equal(scales, want_s)
        np.testing.assert_array_equal(codes, want_c)


def test_quantize_empty_and_row_len_32():
    import torch
    import paper_2606_16317_amd as dsa

    announce("mxfp8 empty and 32-wide rows")
    x = torch.empty((0, 128), dtype=torch.bfloat16, device="cuda")
    c, s = dsa.dsattn_quantize_mxfp8(x)
    assert c.shape == (0, 128) and s.shape == (0, 4)
    bits = make_random_qkv(1, 1, 333, 32, 5)[0]
    codes, scales = run(bits)
    want_c, want_s = quantize_mxfp8(bf16_to_f64(bits))
    np.testing.assert_array_equal(scales, want_s)
    np.testing.assert_array_equal(codes, want_c)


# ---- attention with MX-FP8 Q and K --------------------------------------------------------

SCALE = 1.0 / math.sqrt(128)


def quantised(q, k):
    """Oracle quantisation of bf16 q, k: (codes, exponents) of each and the dequantised
    float64 values the oracle attends with."""
    qc, qs = quantize_mxfp8(bf16_to_f64(q))
    kc, ks = quantize_mxfp8(bf16_to_f64(k))
    return (qc, qs, kc, ks), (dequantize_mxfp8(qc, qs), dequantize_mxfp8(kc, ks))


def run_gpu_q8(qc, qs, kc, ks, vd, rule, param, scale=SCALE, tile_q=128, key_order=0,
               tile_k=64):
    import torch
    import paper_2606_16317_amd as dsa

    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
    B, H, N, d = vd.shape
    n_qt, n_kt = -(-N // tile_q), -(-N // tile_k)
    o = torch.empty_like(vd)
    stats = torch.full((B * H * 4,), -7, dtype=torch.int64, device=vd.device)
    mask = torch.full((B * H * n_qt * n_kt,), 7, dtype=torch.uint8, device=vd.device)
    lse = torch.full((B * H * N,), float("nan"), dtype=torch.float32, device=vd.device)
    args = [dev(a) if isinstance(a, np.ndarray) else a for a in (qc, qs, kc, ks)]
    dsa.dsattn_attn_fwd_mxfp8(RULE_NAMES[rule], param, *args, vd, o, scale=scale,
                              tile_q=tile_q, stats_out=stats, mask_out=mask, lse_out=lse,
                              key_order=key_order, tile_k=tile_k)
    torch.cuda.synchronize()
    return DeviceRun(from_device_bf16(o), mask.cpu().numpy().reshape(B, H, n_qt, n_kt),
                  lse.cpu().numpy().reshape(B, H, N), stats.cpu().numpy().reshape(B, H, 4))


Q8_RULES = [("dense", 0.0), ("dynsparse_lambda", -3.0), ("dynsparse_lambda", -6.0),
            ("dynsparse_recall", 0.95), ("blasst", 0.05)]


@pytest.mark.parametrize("B,H,N", [(1, 1, 1), (1, 1, 64), (1, 1, 65), (2, 3, 129),
                                   (1, 2, 1000), (1, 1, 2047)])
@pytest.mark.parametrize("rule,param", Q8_RULES)
def test_q8_attention_ragged(B, H, N, rule, param):
    q, k, v = make_random_qkv(B, H, N, 128, 7000 + 100 * B + 10 * H + N, q_std=1.5, k_std=1.5)
    announce(f"q8 attention B={B} H={H} N={N} rule={rule} param={param}")
    codes, (qf, kf) = quantised(q, k)
    g = run_gpu_q8(*codes, to_device(v), rule, param)
    rep = compare(qf, kf, v, g, rule, param, SCALE)
    print(rep, flush=True)
    assert_parity(rep)
    assert (g.stats == expected_stats_from_mask(g.mask, N)).all()
    assert not np.isnan(g.lse).any()


@pytest.fixture(scope="module")
def peaked_q8():
    from synth import make_video_qkv

    q, k, v, _ = make_video_qkv(1, 4, (2, 16, 32), 6.0, 6.0, True, 31)
    codes, deq = quantised(q, k)
    return (q, k, v), codes, deq, to_device(v)


@pytest.mark.parametrize("rule,param", [("dynsparse_lambda", -6.0), ("dynsparse_recall", 0.9),
                                        ("blasst", 1e-2)])
def test_q8_attention_concentrated_heads_skip(peaked_q8, rule, param):
    (q, k, v), codes, (qf, kf), vd = peaked_q8
    announce(f"q8 peaked a=6 rule={rule} param={param}")
    g = run_gpu_q8(*codes, vd, rule, param)
    rep = compare(qf, kf, v, g, rule, param, SCALE,
                  tiles=sample_tiles(1, 4, q.shape[2], per_head=4, seed=3))
    print(rep, flush=True)
    assert_parity(rep)
    assert rep.sparsity > 0.1
    assert (g.stats == expected_stats_from_mask(g.mask, q.shape[2])).all()


@pytest.mark.parametrize("tile_q,order", [(32, "ascending"), (128, "diagonal"),
                                           (32, "diagonal")])
@pytest.mark.parametrize("rule,param", [("dynsparse_lambda", -6.0), ("dynsparse_recall", 0.9),
                                        ("blasst", 1e-2), ("dense", 0.0)])
def test_q8_attention_decision_units_and_orders(peaked_q8, tile_q, order, rule, param):
    """The quantised path at 32-row decision units and in diagonal-first key order: the
    oracle runs the same unit and order on the dequantised inputs."""
    (q, k, v), codes, (qf, kf), vd = peaked_q8
    announce(f"q8 peaked tile_q={tile_q} order={order} rule={rule} param={param}")
    g = run_gpu_q8(*codes, vd, rule, param, tile_q=tile_q,
                   key_order=1 if order == "diagonal" else 0)
    N = q.shape[2]
    rep = compare(qf, kf, v, g, rule, param, SCALE, tile_q=tile_q, key_order=order,
                  tiles=sample_tiles(1, 4, N, per_head=5, seed=7, tile_q=tile_q))
    print(rep, flush=True)
    assert_parity(rep)
    assert (g.stats == expected_stats_from_mask(g.mask, N, tile_q)).all()
    if rule != "dense":
        assert rep.sparsity > 0.1


@pytest.mark.parametrize("N", [65, 1000])
def test_q8_attention_ragged_units_and_orders(N):
    q, k, v = make_random_qkv(2, 2, N, 128, 9100 + N, q_std=1.5, k_std=1.5)
    codes, (qf, kf) = quantised(q, k)
    vd = to_device(v)
    for tile_q, order in ((32, 0), (128, 1), (32, 1)):
        announce(f"q8 ragged N={N} tile_q={tile_q} order={order}")
        g = run_gpu_q8(*codes, vd, "dynsparse_lambda", -3.0, tile_q=tile_q, key_order=order)
        rep = compare(qf, kf, v, g, "dynsparse_lambda", -3.0, SCALE, tile_q=tile_q,
                      key_order="diagonal" if order else "ascending")
        assert_parity(rep)
        assert (g.stats == expected_stats_from_mask(g.mask, N, tile_q)).all()


def test_q8_attention_from_gpu_quantisation_is_identical():
    """Quantising on the GPU and attending gives the same bits as attending with the
    oracle's codes (the quantiser is bit-exact), and a second run repeats them."""
    import paper_2606_16317_amd as dsa

    announce("q8 pipeline N=1000 H=2 lambda=-4")
    q, k, v = make_random_qkv(1, 2, 1000, 128, 77, q_std=2.0, k_std=2.0)
    codes, _ = quantised(q, k)
    vd = to_device(v)
    a = run_gpu_q8(*codes, vd, "dynsparse_lambda", -4.0)
    qc, qs = dsa.dsattn_quantize_mxfp8(to_device(q))
    kc, ks = dsa.dsattn_quantize_mxfp8(to_device(k))
    b = run_gpu_q8(qc, qs, kc, ks, vd, "dynsparse_lambda", -4.0)
    c = run_gpu_q8(qc, qs, kc, ks, vd, "dynsparse_lambda", -4.0)
    for x in (b, c):
        np.testing.assert_array_equal(x.o, a.o)
        np.testing.assert_array_equal(x.mask, a.mask)
        np.testing.assert_array_equal(x.lse, a.lse)


def test_q8_attention_close_to_bf16_attention():
    """The difference between the dense outputs of the MX-FP8 and bf16 paths is the
    quantisation error the oracle predicts (fp64 attention on dequantised vs bf16 Q, K):
    the GPU's relative L2 difference lies within 10 % of the oracle's."""
    import paper_2606_16317_amd as dsa

    announce("q8 vs bf16 dense N=1024 H=2")
    q, k, v = make_random_qkv(1, 2, 1024, 128, 78)
    codes, (qf, kf) = quantised(q, k)
    vd = to_device(v)
    a = bf16_to_f64(run_gpu_q8(*codes, vd, "dense", 0.0).o)
    b = bf16_to_f64(from_device_bf16(dsa.dense_attn_fwd(to_device(q), to_device(k), vd)))

    def attend(qq, kk, vv):
        s = SCALE * (qq @ kk.T)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        return (p / p.sum(axis=1, keepdims=True)) @ vv

    for h in range(2):
        vv = bf16_to_f64(v[0, h])
        exact = attend(bf16_to_f64(q[0, h]), bf16_to_f64(k[0, h]), vv)
        quant = attend(qf[0, h], kf[0, h], vv)
        want = np.linalg.norm(quant - exact) / np.linalg.norm(exact)
        got = np.linalg.norm(a[0, h] - b[0, h]) / np.linalg.norm(b[0, h])
        assert abs(got - want) < 0.1 * want, (h, got, want)


# ---- key smoothing --------------------------------------------------------------------

@pytest.mark.parametrize("B,H,N,d,seed", [(1, 2, 1, 128, 0), (2, 3, 777, 128, 1),
                                          (1, 4, 10000, 128, 2), (1, 1, 333, 32, 3),
                                          (1, 2, 4100, 256, 4), (1, 1, 64, 8, 5)])
def test_key_mean_within_summation_bound(B, H, N, d, seed):
    import torch
    import paper_2606_16317_amd as dsa

    announce(f"key mean B={B} H={H} N={N} d={d}")
    _, k, _ = make_random_qkv(B, H, N, d, seed, k_std=3.0)
    k = (bf16_to_f64(k) + 5.0).astype(np.float32)          # a common component
    bits = bf16_bits(k)
    kd = to_device(bits)
    m1 = dsa.dsattn_key_mean(kd).cpu().numpy()
    m2 = dsa.dsattn_key_mean(kd).cpu().numpy()
    np.testing.assert_array_equal(m1, m2)                  # fixed summation order
    exact = key_mean(bf16_to_f64(bits))
    par = 256 // (min(d, 32) // 8)                         # rows summed in parallel
    terms = -(-N // par) + par + 2
    bound = terms * 2.0 ** -24 * np.abs(bf16_to_f64(bits)).mean(axis=-2) + 1e-30
    assert (np.abs(m1 - exact) <= bound).all(), float((np.abs(m1 - exact) / bound).max())


@pytest.mark.parametrize("N,seed", [(200, 0), (1000, 1), (4097, 2)])
def test_shifted_quantize_bit_exact(N, seed):
    import torch
    import paper_2606_16317_amd as dsa

    announce(f"shifted quantize N={N}")
    _, k, _ = make_random_qkv(2, 3, N, 128, 40 + seed, k_std=2.0)
    kf = bf16_to_f64(k)
    shift = key_mean(kf).astype(np.float32) + np.float32(0.37)   # any float32 vector
    codes, scales = dsa.dsattn_quantize_mxfp8(to_device(k),
                                              shift=torch.from_numpy(shift).cuda())
    want_c, want_s = quantize_mxfp8(smooth_keys(kf, shift).astype(np.float64))
    np.testing.assert_array_equal(scales.cpu().numpy(), want_s)
    np.testing.assert_array_equal(codes.cpu().numpy(), want_c)


def smoothed_codes(k):
    """Key mean on the CPU (rounded to float32), the oracle's smoothed codes, and the
    dequantised smoothed keys the oracle attends with."""
    kf = bf16_to_f64(k)
    shift = key_mean(kf).astype(np.float32)
    kc, ks = quantize_mxfp8(smooth_keys(kf, shift).astype(np.float64))
    return shift, kc, ks, dequantize_mxfp8(kc, ks)


@pytest.mark.parametrize("rule,param", [("dense", 0.0), ("dynsparse_lambda", -6.0),
                                        ("blasst", 1e-2)])
def test_q8_attention_smoothed_keys(peaked_q8, rule, param):
    """Parity on smoothed keys (the oracle attends with the dequantised smoothed keys),
    and smoothing brings the output closer to the bf16 path's."""
    import paper_2606_16317_amd as dsa

    (q, k, v), codes, _, vd = peaked_q8
    announce(f"q8 smoothed keys a=6 rule={rule} param={param}")
    qc, qs = codes[0], codes[1]
    shift, kc, ks, kf = smoothed_codes(k)
    g = run_gpu_q8(qc, qs, kc, ks, vd, rule, param)
    qf = dequantize_mxfp8(qc, qs)
    rep = compare(qf, kf, v, g, rule, param, SCALE,
                  tiles=sample_tiles(1, 4, q.shape[2], per_head=4, seed=5))
    print(rep, flush=True)
    assert_parity(rep)
    if rule == "dense":
        plain = run_gpu_q8(*codes, vd, rule, param)
        ref = bf16_to_f64(from_device_bf16(dsa.dense_attn_fwd(to_device(q), to_device(k), vd)))
        err = lambda x: np.linalg.norm(bf16_to_f64(x.o) - ref) / np.linalg.norm(ref)
        assert err(g) < 0.8 * err(plain), (err(g), err(plain))


@pytest.mark.slow
def test_q8_wan720p_sampled():
    """The 720p layer with MX-FP8 Q and K quantised on the GPU (bit-exact with the oracle's
    quantiser, as the tests above show): sampled query tiles of three heads against the
    oracle on the dequantised values."""
    import torch
    import paper_2606_16317_amd as dsa
    from synth import WORKLOADS, workload_inputs

    from _parity import sample_tiles

    w = WORKLOADS["wan720p"]
    announce(f"generate {w.describe()}")
    q, k, v, _ = workload_inputs("wan720p")
    qd, kd, vd = to_device(q), to_device(k), to_device(v)
    qc, qs = dsa.dsattn_quantize_mxfp8(qd)
    kc, ks = dsa.dsattn_quantize_mxfp8(kd)
    del qd, kd
    heads = [(0, 1), (0, 20), (0, 33)]
    tiles = sample_tiles(w.B, w.H, w.N, per_head=3, heads=heads, seed=6)
    qf = np.zeros(q.shape, np.float64)
    kf = np.zeros(k.shape, np.float64)
    for (b, h) in heads:                       # dequantise the sampled heads only
        qf[b, h] = dequantize_mxfp8(qc[b, h].cpu().numpy(), qs[b, h].cpu().numpy())
        kf[b, h] = dequantize_mxfp8(kc[b, h].cpu().numpy(), ks[b, h].cpu().numpy())
    for rule, param, tk in [("dynsparse_lambda", -6.0, 64), ("dynsparse_recall", 0.95, 64),
                            ("dynsparse_lambda", -6.0, 32)]:
        announce(f"q8 wan720p rule={rule} param={param} tile_k={tk} tiles={len(tiles)}")
        g = run_gpu_q8(qc, qs, kc, ks, vd, rule, param, tile_k=tk)
        rep = compare(qf, kf, v, g, rule, param, SCALE, tiles=tiles, tile_k=tk)
        print(rep, f"full-run tile sparsity={float(g.mask.mean()):.4f}", flush=True)
        assert_parity(rep)
        assert (g.stats == expected_stats_from_mask(g.mask, w.N, 128, tk)).all()
