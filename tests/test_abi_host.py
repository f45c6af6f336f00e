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
              "dsattn_last_error", "dsattn_version"):
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
        toks = decl.replace("*", " ").split()
        if "," in decl:
            first = toks[-1] if "," not in toks[-1] else None
            parts = [p.strip().replace("*", "").split()[-1] for p in decl.split(",")]
            fields += parts
        else:
            fields.append(toks[-1])
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
    ("dynsparse_attn_fwd", 0.95, {"tk": 128}, -2, "tile"),
    ("dynsparse_attn_fwd", 0.95, {"N": -1}, -1, ">= 0"),
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
    rc, err = _call_raw("dense_attn_fwd", None, None, None, None, 1, 1, 16, 128, 0.1, 32, 64,
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


def test_empty_problem_is_a_no_op():
    rc, err = _fwd("dynsparse_attn_fwd", 0.95, N=0)
    assert rc == 0 and err == ""
    rc, err = _fwd("dynsparse_attn_fwd", 0.95, B=0)
    assert rc == 0


def test_version_string():
    pkg = _lib()
    assert b"gfx950" in pkg.lib().dsattn_version()
