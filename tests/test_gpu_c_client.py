"""The C ABI from a plain C program on the GPU: ``tests/c_client/dsattn_gpu_client.c``
includes only ``include/dsattn.h`` and the HIP runtime header, takes device buffers from
hipMalloc, runs the DynSparse rule through ``dsattn_attn_fwd_ex`` and
``dynsparse_attn_fwd_lambda`` on the default stream and writes the results to files.
They must match the oracle (teacher-forced on the program's own mask), the counters must
follow from the mask, and the two entry points must give the same output bits."""

import math
import os
import shutil
import subprocess
import sys

import numpy as np
import pytest

from synth import make_video_qkv

from _parity import DeviceRun, assert_parity, compare, expected_stats_from_mask

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2606_16317_amd")
SCALE = 1.0 / math.sqrt(128)


@pytest.fixture(scope="module")
def client(tmp_path_factory):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    if not os.path.exists(os.path.join(PKG, "libdsattn.so")):
        pytest.fail("libdsattn.so is not built")
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path_factory.mktemp("gpu_client") / "dsattn_gpu_client")
    cmd = ["gcc", "-std=c99", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I" + os.path.join(ROOT, "include"), "-I/opt/rocm/include",
           os.path.join(ROOT, "tests", "c_client", "dsattn_gpu_client.c"), "-L" + PKG,
           "-ldsattn", "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath," + PKG,
           "-Wl,-rpath,/opt/rocm/lib", "-o", exe]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return exe


# peaked video-shaped heads (concentration a) so that the threshold really skips; the
# second and third grids give ragged query and key tiles
@pytest.mark.parametrize("B,H,grid,a,lam,tile_q", [(1, 2, (2, 16, 32), 6.0, -8.0, 128),
                                                   (2, 1, (1, 13, 27), 6.0, -6.0, 32),
                                                   (1, 1, (3, 11, 31), 5.0, -8.0, 128)])
def test_c_program_matches_oracle(client, tmp_path, B, H, grid, a, lam, tile_q):
    q, k, v, _ = make_video_qkv(B, H, grid, a, a, True, 77)
    N = q.shape[2]
    print(f"\n[case] C client B={B} H={H} N={N} lambda={lam} tile_q={tile_q}", flush=True)
    for name, arr in (("q", q), ("k", k), ("v", v)):
        np.ascontiguousarray(arr).tofile(str(tmp_path / f"{name}.bin"))
    res = subprocess.run([client, str(tmp_path), str(B), str(H), str(N), repr(lam),
                          str(tile_q)], capture_output=True, text=True, timeout=120)
    assert res.returncode == 0, res.stderr
    n_qt, n_kt = -(-N // tile_q), -(-N // 64)
    o = np.fromfile(str(tmp_path / "o.bin"), dtype=np.uint16).reshape(B, H, N, 128)
    o_named = np.fromfile(str(tmp_path / "o_named.bin"), dtype=np.uint16).reshape(B, H, N, 128)
    mask = np.fromfile(str(tmp_path / "mask.bin"), dtype=np.uint8).reshape(B, H, n_qt, n_kt)
    lse = np.fromfile(str(tmp_path / "lse.bin"), dtype=np.float32).reshape(B, H, N)
    stats = np.fromfile(str(tmp_path / "stats.bin"), dtype=np.uint64).astype(np.int64)
    run = DeviceRun(o, mask, lse, stats.reshape(B, H, 4))
    assert np.array_equal(o, o_named)
    assert (run.stats == expected_stats_from_mask(mask, N, tile_q)).all()
    rep = compare(q, k, v, run, "dynsparse_lambda", lam, SCALE, tile_q=tile_q)
    print(rep, flush=True)
    assert_parity(rep)
    assert 0.0 < float(mask.mean()) < 1.0
