"""C-ABI checks that need no GPU: the library loads, exports every declared symbol, maps
recall to lambda like the oracle, and rejects bad arguments on the host."""

import ctypes
import math
import os
import re

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dsattn.h")


def _lib():
    import paper_2606_16317_amd as pkg

    if not os.path.exists(pkg.LIB_PATH):
        pytest.skip("libdsattn.so not built")
    return pkg


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\s*\*?\s*([a-z_][a-z0-9_]*)\s*\(",
                       text, flags=re.M)
    return sorted(set(names))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for n in ("dynsparse_attn_fwd", "dynsparse_attn_fwd_lambda", "blasst_attn_fwd",
              "dense_attn_fwd", "dsattn_attn_fwd_ex", "dsattn_lambda_from_recall",
              "dsattn_last_error", "dsattn_version", "dsattn_block_order",
              "dsattn_gather_rows", "dsattn_scatter_rows", "dsattn_reordered_workspace_bytes",
              "dsattn_attn_fwd_reordered"):
        assert n in names


def test_library_exports_every_declared_symbol():
    pkg = _lib()
    raw = ctypes.CDLL(pkg.LIB_PATH)
    for name in declared_functions():
        assert hasattr(raw, name), name


def test_struct_mirror_matches_header_field_order():
    pkg = _lib()
    text = open(HEADER).read()
    body = re.search(r"typedef struct dsattn_args \{(.*?)\} dsattn_args;", text, re.S).group(1)
    body = re.sub(r"/\*.*?\*/", "", body, flags=re.S)
    fields = []
    for decl in body.split(";"):
        decl = decl.strip()
        if not decl:
            continue
        if "," in decl:
            fields += [p.strip().replace("*", "").split()[-1] for p in decl.split(",")]
        else:
            fields.append(decl.replace("*", " ").split()[-1])
    assert fields == [f[0] for f in pkg.DsAttnArgs._fields_]


@pytest.mark.parametrize("r,n", [(0.95, 2048), (0.95, 32760), (0.95, 75600), (0.9, 75600),
                                 (0.99, 131072), (0.5, 7)])
def test_lambda_mapping_matches_oracle(r, n):
    pkg = _lib()
    got = pkg.dsattn_lambda_from_recall(r, n)
    ref = oracle.lambda_from_recall(float(ctypes.c_float(r).value), n)
    assert got == pytest.approx(ref, rel=1e-6)


def test_lambda_mapping_edges():
    pkg = _lib()
    assert pkg.dsattn_lambda_from_recall(1.0, 10) == -math.inf
    assert math.isnan(pkg.dsattn_lambda_from_recall(0.0, 10))
    assert math.isnan(pkg.dsattn_lambda_from_recall(1.5, 10))
    assert math.isnan(pkg.dsattn_lambda_from_recall(0.9, 0))


def _call_raw(name, *args):
    pkg = _lib()
    L = pkg.lib()
    return getattr(L, name)(*args), pkg.last_error()


def _fwd(name, param, B=1, H=1, N=128, d=128, scale=0.1, tq=128, tk=64, ptr=None):
    p = ptr
    return _call_raw(name, p, p, p, p, B, H, N, d, scale, param, tq, tk, None, None)


@pytest.mark.parametrize("name,param,kw,code,msg", [
    ("dynsparse_attn_fwd", 0.95, {}, -1, "non-null"),
    ("dynsparse_attn_fwd", 0.0, {}, -1, "recall"),
    ("dynsparse_attn_fwd", 1.5, {}, -1, "recall"),
    ("dynsparse_attn_fwd", float("nan"), {}, -1, "recall"),
    ("dynsparse_attn_fwd_lambda", float("nan"), {}, -1, "lambda"),
    ("dynsparse_attn_fwd_lambda", float("inf"), {}, -1, "lambda"),
    ("blasst_attn_fwd", -0.1, {}, -1, "tau"),
    ("blasst_attn_fwd", 1.1, {}, -1, "tau"),
    ("dynsparse_attn_fwd", 0.95, {"d": 64}, -2, "head dimension"),
    ("dynsparse_attn_fwd", 0.95, {"tq": 64}, -2, "tile"),
    ("dynsparse_attn_fwd", 0.95, {"tq": 32, "tk": 32}, -1, "non-null"),  # 32-key decisions pass
    ("dynsparse_attn_fwd", 0.95, {"tq": 32, "tk": 16}, -2, "tile"),
    ("dynsparse_attn_fwd", 0.95, {"tq": 32}, -1, "non-null"),   # 32 x 64 passes the shape check
    ("dynsparse_attn_fwd", 0.95, {"tk": 128}, -1, "non-null"),  # 128-key decisions pass
    ("dynsparse_attn_fwd", 0.95, {"tk": 96}, -2, "tile"),
    ("dynsparse_attn_fwd", 0.95, {"N": -1}, -1, ">= 0"),
    ("dynsparse_attn_fwd", 0.95, {"N": 8388608}, -1, "N must be <= 8388607"),
    ("dynsparse_attn_fwd", 0.95, {"N": 8388607}, -1, "non-null"),   # the largest N passes
    ("dynsparse_attn_fwd", 0.95, {"B": -2}, -1, ">= 0"),
    ("dynsparse_attn_fwd", 0.95, {"scale": 0.0}, -1, "scale"),
    ("dynsparse_attn_fwd", 0.95, {"scale": float("inf")}, -1, "scale"),
    ("dynsparse_attn_fwd", 0.95, {"B": 300, "H": 300}, -1, "65535"),
])
def test_argument_errors_are_reported_on_host(name, param, kw, code, msg):
    rc, err = _fwd(name, param, **kw)
    assert rc == code
    assert msg in err


def test_dense_entry_rejects_null_and_bad_tiles():
    rc, err = _call_raw("dense_attn_fwd", None, None, None, None, 1, 1, 16, 128, 0.1, 128, 64,
                        None, None)
    assert rc == -1 and "non-null" in err
    rc, err = _call_raw("dense_attn_fwd", None, None, None, None, 1, 1, 16, 128, 0.1, 64, 64,
                        None, None)
    assert rc == -2


def test_host_pointer_is_rejected():
    """A host buffer passed as q must be refused before any launch."""
    buf = (ctypes.c_uint16 * (128 * 128))()
    p = ctypes.addressof(buf)
    rc, err = _call_raw("dense_attn_fwd", p, p + 2, p + 4, p + 6, 1, 1, 32, 128, 0.1, 128, 64,
                        None, None)
    assert rc == -1 and "device pointer" in err


def test_ex_rejects_unknown_rule_and_null_args():
    pkg = _lib()
    L = pkg.lib()
    assert L.dsattn_attn_fwd_ex(None) == -1
    a = pkg.DsAttnArgs(9, 0.0, None, None, None, None, 1, 1, 16, 128, 0.1, 128, 64,
                       None, None, None, None)
    assert L.dsattn_attn_fwd_ex(ctypes.byref(a)) == -1
    assert "unknown rule" in pkg.last_error()


def test_ex_rejects_unknown_key_order():
    pkg = _lib()
    L = pkg.lib()
    a = pkg.DsAttnArgs(pkg.RULE_DENSE, 0.0, None, None, None, None, 1, 1, 16, 128, 0.1, 128,
                       64, None, None, None, None, 7)
    assert L.dsattn_attn_fwd_ex(ctypes.byref(a)) == -1
    assert "key order" in pkg.last_error()
    a.key_order = pkg.ORDER_DIAGONAL
    assert L.dsattn_attn_fwd_ex(ctypes.byref(a)) == -1
    assert "non-null" in pkg.last_error()     # a valid order passes to the pointer checks


def test_mask_reuse_argument_checks():
    pkg = _lib()
    L = pkg.lib()
    a = pkg.DsAttnArgs(pkg.RULE_MASK, 0.0, None, None, None, None, 1, 1, 300, 128, 0.1, 128,
                       64, None, None, None, None, pkg.ORDER_DIAGONAL, None)
    assert L.dsattn_attn_fwd_ex(ctypes.byref(a)) == -2
    assert "ascending" in pkg.last_error()
    a.key_order = pkg.ORDER_ASCENDING
    a.N = 262144 + 64
    assert L.dsattn_attn_fwd_ex(ctypes.byref(a)) == -2
    assert "262144" in pkg.last_error()
    a.N = 262144                     # at the limit: passes on to the pointer checks
    assert L.dsattn_attn_fwd_ex(ctypes.byref(a)) == -1
    assert "non-null" in pkg.last_error()


def test_empty_problem_is_a_no_op():
    rc, err = _fwd("dynsparse_attn_fwd", 0.95, N=0)
    assert rc == 0 and err == ""
    rc, err = _fwd("dynsparse_attn_fwd", 0.95, B=0)
    assert rc == 0


def test_version_string():
    pkg = _lib()
    assert b"gfx950" in pkg.lib().dsattn_version()


# ---- token reordering (host side) ---------------------------------------------------------

@pytest.mark.parametrize("grid,block", [((1, 3, 3), (1, 2, 2)), ((21, 45, 80), (2, 8, 8)),
                                        ((21, 45, 80), (1, 8, 8)), ((3, 5, 7), (2, 3, 4)),
                                        ((32, 64, 64), (1, 8, 8)), ((2, 32, 32), (5, 7, 9))])
def test_block_order_matches_oracle(grid, block):
    """The library's closed-form block order equals the oracle's enumeration, bit for bit."""
    import numpy as np
    from oracle.reorder import block_order

    pkg = _lib()
    got = pkg.dsattn_block_order(grid, block)
    assert got.dtype == np.int32
    assert np.array_equal(got.astype(np.int64), block_order(grid, block))


@pytest.mark.parametrize("args,msg", [
    ((0, 2, 2, 1, 1, 1), "positive"),
    ((2, 2, 2, 1, -1, 1), "positive"),
    ((2048, 2048, 1024, 1, 1, 1), "2^31"),
])
def test_block_order_rejects_bad_extents(args, msg):
    import numpy as np

    pkg = _lib()
    buf = np.zeros(16, dtype=np.int32)
    rc = pkg.lib().dsattn_block_order(*args, buf.ctypes.data)
    assert rc == -1 and msg in pkg.last_error()
    assert pkg.lib().dsattn_block_order(2, 2, 2, 1, 1, 1, None) == -1


@pytest.mark.parametrize("name", ["dsattn_gather_rows", "dsattn_scatter_rows"])
@pytest.mark.parametrize("bh,n,row,msg", [
    (1, 4, 6, "multiple of 4"), (1, 4, 0, "multiple of 4"), (-1, 4, 16, ">= 0"),
    (70000, 4, 16, "65535"), (1, 1 << 30, 64, "too large"), (1, 4, 16, "non-null"),
])
def test_row_moves_reject_bad_arguments(name, bh, n, row, msg):
    rc, err = _call_raw(name, None, None, None, bh, n, row, None)
    assert rc == -1 and msg in err


@pytest.mark.parametrize("name", ["dsattn_gather_rows", "dsattn_scatter_rows"])
def test_row_moves_reject_host_pointers_and_accept_empty(name):
    buf = (ctypes.c_uint32 * 64)()
    p = ctypes.addressof(buf)
    rc, err = _call_raw(name, p, p + 128, p, 1, 4, 16, None)
    assert rc == -1 and "device pointer" in err
    rc, err = _call_raw(name, None, None, None, 0, 4, 16, None)
    assert rc == 0 and err == ""


def test_reordered_workspace_size():
    pkg = _lib()
    L = pkg.lib()
    tensor = 1 * 40 * 75600 * 128 * 2
    slice_ = -(-tensor // 256) * 256
    assert L.dsattn_reordered_workspace_bytes(1, 40, 75600, 128, 0) == 4 * slice_
    lse = -(-(40 * 75600 * 4) // 256) * 256
    assert L.dsattn_reordered_workspace_bytes(1, 40, 75600, 128, 1) == 4 * slice_ + lse
    assert L.dsattn_reordered_workspace_bytes(0, 40, 75600, 128, 1) == 0
    assert L.dsattn_reordered_workspace_bytes(1, 3, 100, 128, 0) == 4 * (-(-(3 * 100 * 256) // 256) * 256)


def test_reordered_rejects_bad_arguments():
    pkg = _lib()
    L = pkg.lib()
    assert L.dsattn_attn_fwd_reordered(None, None, None, None, 0) == -1
    a = pkg.DsAttnArgs(pkg.RULE_DYNSPARSE_LAMBDA, float("nan"), None, None, None, None, 1, 1,
                       16, 128, 0.1, 128, 64, None, None, None, None)
    assert L.dsattn_attn_fwd_reordered(ctypes.byref(a), None, None, None, 0) == -1
    assert "lambda" in pkg.last_error()
    a.param = -6.0
    assert L.dsattn_attn_fwd_reordered(ctypes.byref(a), None, None, None, 0) == -1
    assert "non-null" in pkg.last_error()
    a.tile_q = 64
    assert L.dsattn_attn_fwd_reordered(ctypes.byref(a), None, None, None, 0) == -2
    a.tile_q, a.N = 128, 0
    assert L.dsattn_attn_fwd_reordered(ctypes.byref(a), None, None, None, 0) == 0


@pytest.mark.parametrize("rows,row_len,msg", [
    (4, 48, "multiple of 32"), (4, 0, "multiple of 32"), (-1, 128, ">= 0"),
    (1 << 40, 128, "too large"), (1 << 35, 128, "too large"), (4, 128, "non-null"),
])
def test_quantize_rejects_bad_arguments(rows, row_len, msg):
    rc, err = _call_raw("dsattn_quantize_mxfp8", None, None, None, rows, row_len, None)
    assert rc == -1 and msg in err


def test_quantize_rejects_host_pointers_and_accepts_empty():
    buf = (ctypes.c_uint32 * 64)()
    p = ctypes.addressof(buf)
    rc, err = _call_raw("dsattn_quantize_mxfp8", p, p, p, 1, 32, None)
    assert rc == -1 and "device pointer" in err
    rc, err = _call_raw("dsattn_quantize_mxfp8", None, None, None, 0, 128, None)
    assert rc == 0 and err == ""


def test_qk_format_argument_checks():
    pkg = _lib()
    L = pkg.lib()

    def call(**kw):
        a = pkg.DsAttnArgs(pkg.RULE_DYNSPARSE_LAMBDA, -6.0, None, None, None, None, 1, 1, 256,
                           128, 0.1, 128, 64, None, None, None, None, 0, None, pkg.QK_MXFP8,
                           None, None)
        for key, val in kw.items():
            setattr(a, key, val)
        return L.dsattn_attn_fwd_ex(ctypes.byref(a)), pkg.last_error()

    assert call(qk_format=7) == (-1, "unknown qk format 7")
    rc, err = call(tile_q=64)
    assert rc == -2 and "tile shape" in err
    rc, err = call(tile_q=32, key_order=pkg.ORDER_DIAGONAL)
    assert rc == -1 and "non-null" in err           # supported: fails only on the pointers
    rc, err = call(rule=pkg.RULE_MASK)
    assert rc == -2 and "bf16" in err
    rc, err = call()
    assert rc == -1 and "non-null" in err
    assert call(N=0) == (0, "")
    a = pkg.DsAttnArgs(pkg.RULE_DENSE, 0.0, None, None, None, None, 1, 1, 256, 128, 0.1, 128,
                       64, None, None, None, None, 0, None, pkg.QK_MXFP8, None, None)
    ws = (ctypes.c_uint8 * 256)()
    assert L.dsattn_attn_fwd_reordered(ctypes.byref(a), None, None, ws, 256) == -2
    assert "bf16" in pkg.last_error()


@pytest.mark.parametrize("bh,n,d,msg", [
    (-1, 4, 128, ">= 0"), (70000, 4, 128, "65535"), (1, 4, 96, "power of two"),
    (1, 4, 4, "power of two"), (1, 4, 2048, "power of two"), (1, 0, 128, "zero keys"),
    (1, 1 << 30, 128, "too large"), (1, 4, 128, "non-null"),
])
def test_key_mean_rejects_bad_arguments(bh, n, d, msg):
    rc, err = _call_raw("dsattn_key_mean", None, None, bh, n, d, None)
    assert rc == -1 and msg in err


def test_key_mean_and_shifted_quantize_host_checks():
    buf = (ctypes.c_uint32 * 64)()
    p = ctypes.addressof(buf)
    rc, err = _call_raw("dsattn_key_mean", p, p, 1, 4, 128, None)
    assert rc == -1 and "device pointers" in err
    assert _call_raw("dsattn_key_mean", None, None, 0, 4, 128, None) == (0, "")
    rc, err = _call_raw("dsattn_quantize_mxfp8_shift", None, None, None, None, 4, 128, 4, None)
    assert rc == -1 and "shift must be non-null" in err
    rc, err = _call_raw("dsattn_quantize_mxfp8_shift", None, p, None, None, 4, 128, 0, None)
    assert rc == -1 and "group_rows" in err
    rc, err = _call_raw("dsattn_quantize_mxfp8_shift", None, p, None, None, 4, 100, 4, None)
    assert rc == -1 and "multiple of 32" in err
    rc, err = _call_raw("dsattn_quantize_mxfp8_shift", None, p, None, None, 0, 128, 4, None)
    assert rc == 0 and err == ""


def test_key_tile_restrictions():
    pkg = _lib()
    L = pkg.lib()
    a = pkg.DsAttnArgs(pkg.RULE_DYNSPARSE_LAMBDA, -6.0, None, None, None, None, 1, 1, 256,
                       128, 0.1, 128, 128, None, None, None, None, pkg.ORDER_DIAGONAL, None, 0,
                       None, None)
    assert L.dsattn_attn_fwd_ex(ctypes.byref(a)) == -1      # 128 in diagonal order: supported
    assert "non-null" in pkg.last_error()
    a.key_order, a.rule = pkg.ORDER_ASCENDING, pkg.RULE_MASK
    assert L.dsattn_attn_fwd_ex(ctypes.byref(a)) == -1      # 128-key masks are reusable
    assert "mask_in" in pkg.last_error() or "non-null" in pkg.last_error()
    a.tile_k = 32
    assert L.dsattn_attn_fwd_ex(ctypes.byref(a)) == -2
    assert "tile_k = 64 or 128" in pkg.last_error()
    a.tile_k = 128
    a.rule = pkg.RULE_BLASST
    a.param = 0.01
    assert L.dsattn_attn_fwd_ex(ctypes.byref(a)) == -1
    assert "non-null" in pkg.last_error()
    a.tile_k, a.qk_format = 32, pkg.QK_MXFP8
    assert L.dsattn_attn_fwd_ex(ctypes.byref(a)) == -1     # supported: fails on the pointers
    assert "non-null" in pkg.last_error()
    a.qk_format, a.key_order = 0, pkg.ORDER_DIAGONAL
    assert L.dsattn_attn_fwd_ex(ctypes.byref(a)) == -2
    assert "ascending" in pkg.last_error()


def test_last_error_is_per_thread():
    """dsattn_last_error belongs to the calling thread: threads that fail with different
    arguments each read their own message, and a thread whose call succeeds reads ""."""
    import threading

    pkg = _lib()
    L = pkg.lib()
    results = {}
    barrier = threading.Barrier(3)

    def worker(name, call):
        barrier.wait()
        out = []
        for _ in range(200):
            rc = call()
            out.append((rc, pkg.last_error()))
        results[name] = out

    calls = {
        "recall": lambda: _fwd("dynsparse_attn_fwd", 1.5)[0],            # bad recall
        "head": lambda: L.dsattn_key_mean(None, None, 1, 4, 12, None),  # bad d
        "ok": lambda: L.dsattn_key_mean(None, None, 0, 4, 128, None),   # empty: success
    }
    threads = [threading.Thread(target=worker, args=(n, c)) for n, c in calls.items()]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert all(rc == -1 and "recall" in msg for rc, msg in results["recall"])
    assert all(rc == -1 and "power of two" in msg for rc, msg in results["head"])
    assert all(rc == 0 and msg == "" for rc, msg in results["ok"])
