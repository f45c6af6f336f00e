"""GPU parity of the MX-FP8 quantisation kernel, called through the C ABI, against the
CPU oracle (``oracle.mxfp8``): codes and block exponents must match bit for bit.

The inputs mix Gaussian rows of several scales, all-zero blocks, bf16 subnormals, the
largest bf16 magnitudes, values exactly halfway between two E4M3 codes after scaling,
and blocks whose scaled maximum rounds up to the saturation limit.
"""

import sys

import numpy as np
import pytest

from oracle import bf16_to_f64
from oracle.mxfp8 import quantize_mxfp8
from synth import bf16_bits, make_random_qkv

from _parity import to_device

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
