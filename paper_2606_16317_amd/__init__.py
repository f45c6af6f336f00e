"""Python binding of libdsattn.so (argument marshalling only).

Every function here takes torch tensors that live on the GPU, checks dtype/shape/device,
and calls the C entry point of the same name with raw device pointers and the current
torch stream.  All arithmetic runs in the HIP kernels of the library; there is no
fallback: if the library is missing or a call fails, a RuntimeError is raised.

Tensor conventions: q, k, v, o are contiguous bf16 tensors of shape [B, H, N, 128];
``stats_out`` is an int64 tensor of B*H*4 elements (uint64 counters
{tiles_total, tiles_skipped, elems_total, elems_skipped} per head); ``mask_out`` is a
uint8 tensor of B*H*ceil(N/tile_q)*ceil(N/64) elements (tile_q = 128, or 32 for per-wave
decisions); ``lse_out`` a float32 tensor of
B*H*N elements.
"""

from __future__ import annotations

import ctypes
import math
import os

LIB_NAME = "libdsattn.so"
# DSATTN_LIB selects another build of the same library (for instance the host-sanitizer
# build, libdsattn_san.so); by default the in-tree libdsattn.so is loaded.
LIB_PATH = os.environ.get("DSATTN_LIB") or os.path.join(
    os.path.dirname(os.path.abspath(__file__)), LIB_NAME)

TILE_Q = 128
TILE_K = 64
HEAD_DIM = 128

RULE_DENSE = 0
RULE_BLASST = 1
RULE_DYNSPARSE_RECALL = 2
RULE_DYNSPARSE_LAMBDA = 3
RULE_MASK = 4

ORDER_ASCENDING = 0
ORDER_DIAGONAL = 1

QK_BF16 = 0
QK_MXFP8 = 1

_lib = None


class DsAttnArgs(ctypes.Structure):
    """Mirror of ``dsattn_args`` in include/dsattn.h."""

    _fields_ = [
        ("rule", ctypes.c_int),
        ("param", ctypes.c_float),
        ("q", ctypes.c_void_p),
        ("k", ctypes.c_void_p),
        ("v", ctypes.c_void_p),
        ("o", ctypes.c_void_p),
        ("B", ctypes.c_int),
        ("H", ctypes.c_int),
        ("N", ctypes.c_int),
        ("d", ctypes.c_int),
        ("scale", ctypes.c_float),
        ("tile_q", ctypes.c_int),
        ("tile_k", ctypes.c_int),
        ("stream", ctypes.c_void_p),
        ("stats_out", ctypes.c_void_p),
        ("mask_out", ctypes.c_void_p),
        ("lse_out", ctypes.c_void_p),
        ("key_order", ctypes.c_int),
        ("mask_in", ctypes.c_void_p),
        ("qk_format", ctypes.c_int),
        ("q_scales", ctypes.c_void_p),
        ("k_scales", ctypes.c_void_p),
    ]


_FWD_ARGS = [ctypes.c_void_p] * 4 + [ctypes.c_int] * 4 + [ctypes.c_float, ctypes.c_float,
                                                           ctypes.c_int, ctypes.c_int,
                                                           ctypes.c_void_p, ctypes.c_void_p]
_DENSE_ARGS = [ctypes.c_void_p] * 4 + [ctypes.c_int] * 4 + [ctypes.c_float, ctypes.c_int,
                                                            ctypes.c_int, ctypes.c_void_p,
                                                            ctypes.c_void_p]


def lib():
    """Load libdsattn.so once (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is not built; run `python -m paper_2606_16317_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name in ("dynsparse_attn_fwd", "dynsparse_attn_fwd_lambda", "blasst_attn_fwd"):
            getattr(L, name).argtypes = _FWD_ARGS
            getattr(L, name).restype = ctypes.c_int
        L.dense_attn_fwd.argtypes = _DENSE_ARGS
        L.dense_attn_fwd.restype = ctypes.c_int
        L.dsattn_attn_fwd_ex.argtypes = [ctypes.POINTER(DsAttnArgs)]
        L.dsattn_attn_fwd_ex.restype = ctypes.c_int
        L.dsattn_lambda_from_recall.argtypes = [ctypes.c_float, ctypes.c_int]
        L.dsattn_lambda_from_recall.restype = ctypes.c_float
        L.dsattn_block_order.argtypes = [ctypes.c_int] * 6 + [ctypes.c_void_p]
        L.dsattn_block_order.restype = ctypes.c_int
        for name in ("dsattn_gather_rows", "dsattn_scatter_rows"):
            getattr(L, name).argtypes = [ctypes.c_void_p] * 3 + [ctypes.c_int] * 3 + [
                ctypes.c_void_p]
            getattr(L, name).restype = ctypes.c_int
        L.dsattn_reordered_workspace_bytes.argtypes = [ctypes.c_int] * 5
        L.dsattn_reordered_workspace_bytes.restype = ctypes.c_size_t
        L.dsattn_attn_fwd_reordered.argtypes = [ctypes.POINTER(DsAttnArgs), ctypes.c_void_p,
                                                ctypes.c_void_p, ctypes.c_void_p,
                                                ctypes.c_size_t]
        L.dsattn_attn_fwd_reordered.restype = ctypes.c_int
        L.dsattn_attn_fwd_reordered_noalloc.argtypes = [ctypes.POINTER(DsAttnArgs),
                                                        ctypes.c_void_p, ctypes.c_void_p]
        L.dsattn_attn_fwd_reordered_noalloc.restype = ctypes.c_int
        L.dsattn_quantize_mxfp8.argtypes = [ctypes.c_void_p] * 3 + [ctypes.c_longlong,
                                                                      ctypes.c_int,
                                                                      ctypes.c_void_p]
        L.dsattn_quantize_mxfp8.restype = ctypes.c_int
        L.dsattn_quantize_mxfp8_shift.argtypes = [ctypes.c_void_p] * 4 + [
            ctypes.c_longlong, ctypes.c_int, ctypes.c_longlong, ctypes.c_void_p]
        L.dsattn_quantize_mxfp8_shift.restype = ctypes.c_int
        L.dsattn_key_mean.argtypes = [ctypes.c_void_p, ctypes.c_void_p] + [ctypes.c_int] * 3 + [
            ctypes.c_void_p]
        L.dsattn_key_mean.restype = ctypes.c_int
        L.dsattn_last_error.argtypes = []
        L.dsattn_last_error.restype = ctypes.c_char_p
        L.dsattn_version.argtypes = []
        L.dsattn_version.restype = ctypes.c_char_p
        _lib = L
    return _lib


def last_error() -> str:
    return lib().dsattn_last_error().decode()


def dsattn_lambda_from_recall(recall_target: float, N: int) -> float:
    return float(lib().dsattn_lambda_from_recall(recall_target, N))


def _check(rc: int, name: str):
    if rc != 0:
        raise RuntimeError(f"{name} failed ({rc}): {last_error()}")


def _shape(q, k, v, o):
    import torch

    for name, t in (("q", q), ("k", k), ("v", v), ("o", o)):
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"{name} must be a torch.Tensor")
        if t.dtype != torch.bfloat16:
            raise TypeError(f"{name} must be bfloat16 (got {t.dtype})")
        if not t.is_cuda:
            raise ValueError(f"{name} must be on the GPU")
        if not t.is_contiguous():
            raise ValueError(f"{name} must be contiguous")
        if t.dim() != 4:
            raise ValueError(f"{name} must have shape [B, H, N, d]")
    if not (q.shape == k.shape == v.shape == o.shape):
        raise ValueError("q, k, v and o must have the same shape")
    return tuple(int(x) for x in q.shape)


def _ptr(t, numel=None, dtype=None, name="buffer"):
    if t is None:
        return None
    if dtype is not None and t.dtype not in dtype:
        raise TypeError(f"{name} has dtype {t.dtype}")
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous GPU tensor")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} needs at least {numel} elements (got {t.numel()})")
    return t.data_ptr()


def _stream(stream):
    import torch

    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _out(q, o):
    import torch

    return torch.empty_like(q) if o is None else o


def _buffers(B, H, N, stats_out, mask_out=None, lse_out=None, tile_q=TILE_Q, tile_k=TILE_K):
    import torch

    n_qt = -(-N // max(1, tile_q))
    n_kt = -(-N // max(1, tile_k))
    return (_ptr(stats_out, B * H * 4, (torch.int64, torch.uint64), "stats_out"),
            _ptr(mask_out, B * H * n_qt * n_kt, (torch.uint8,), "mask_out"),
            _ptr(lse_out, B * H * N, (torch.float32,), "lse_out"))


def dynsparse_attn_fwd(q, k, v, o=None, scale=None, recall_target=0.95, tile_q=TILE_Q,
                       tile_k=TILE_K, stats_out=None, stream=None):
    """DynSparse forward with lambda = ln((1 - recall_target) / N); returns o."""
    o = _out(q, o)
    B, H, N, d = _shape(q, k, v, o)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    st, _, _ = _buffers(B, H, N, stats_out)
    rc = lib().dynsparse_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                  B, H, N, d, scale, recall_target, tile_q, tile_k,
                                  _stream(stream), st)
    _check(rc, "dynsparse_attn_fwd")
    return o


def dynsparse_attn_fwd_lambda(q, k, v, o=None, scale=None, lam=-6.0, tile_q=TILE_Q,
                              tile_k=TILE_K, stats_out=None, stream=None):
    """DynSparse forward with an explicit threshold lambda (natural log); returns o."""
    o = _out(q, o)
    B, H, N, d = _shape(q, k, v, o)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    st, _, _ = _buffers(B, H, N, stats_out)
    rc = lib().dynsparse_attn_fwd_lambda(q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                         o.data_ptr(), B, H, N, d, scale, lam, tile_q, tile_k,
                                         _stream(stream), st)
    _check(rc, "dynsparse_attn_fwd_lambda")
    return o


def blasst_attn_fwd(q, k, v, o=None, scale=None, threshold=1e-3, tile_q=TILE_Q,
                    tile_k=TILE_K, stats_out=None, stream=None):
    """BLASST-style forward (skip when tile max - running max < ln threshold); returns o."""
    o = _out(q, o)
    B, H, N, d = _shape(q, k, v, o)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    st, _, _ = _buffers(B, H, N, stats_out)
    rc = lib().blasst_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                               B, H, N, d, scale, threshold, tile_q, tile_k, _stream(stream),
                               st)
    _check(rc, "blasst_attn_fwd")
    return o


def dense_attn_fwd(q, k, v, o=None, scale=None, tile_q=TILE_Q, tile_k=TILE_K,
                   stats_out=None, stream=None):
    """Dense forward of the same kernel family; returns o."""
    o = _out(q, o)
    B, H, N, d = _shape(q, k, v, o)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    st, _, _ = _buffers(B, H, N, stats_out)
    rc = lib().dense_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                              B, H, N, d, scale, tile_q, tile_k, _stream(stream), st)
    _check(rc, "dense_attn_fwd")
    return o


def dsattn_attn_fwd_ex(rule, param, q, k, v, o=None, scale=None, tile_q=TILE_Q,
                       tile_k=TILE_K, stats_out=None, mask_out=None, lse_out=None,
                       stream=None, key_order=ORDER_ASCENDING, mask_in=None):
    """Any rule (RULE_* constants) with optional stats, skip mask and LSE outputs, and
    the key-tile visit order (ORDER_* constants).  RULE_MASK reuses ``mask_in`` (a uint8
    GPU tensor laid out like ``mask_out``)."""
    import torch

    o = _out(q, o)
    B, H, N, d = _shape(q, k, v, o)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    st, mk, ls = _buffers(B, H, N, stats_out, mask_out, lse_out, tile_q, tile_k)
    mi = None
    if mask_in is not None:
        n_qu = -(-N // max(1, tile_q))
        mi = _ptr(mask_in, B * H * n_qu * (-(-N // max(1, tile_k))), (torch.uint8,), "mask_in")
    a = DsAttnArgs(rule, param, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                   B, H, N, d, scale, tile_q, tile_k, _stream(stream), st, mk, ls, key_order,
                   mi)
    _check(lib().dsattn_attn_fwd_ex(ctypes.byref(a)), "dsattn_attn_fwd_ex")
    return o


def dsattn_attn_fwd_mxfp8(rule, param, q8, q_scales, k8, k_scales, v, o=None, scale=None,
                          tile_q=TILE_Q, stats_out=None, mask_out=None, lse_out=None,
                          stream=None, key_order=ORDER_ASCENDING, tile_k=TILE_K):
    """A rule with MX-FP8 Q and K (``dsattn_qk_format`` DSATTN_QK_MXFP8): q8 / k8 are uint8
    E4M3 codes [B, H, N, 128] and q_scales / k_scales their uint8 E8M0 exponents
    [B, H, N, 4], as returned by ``dsattn_quantize_mxfp8``; v is bf16."""
    import torch

    o = torch.empty_like(v) if o is None else o
    B, H, N, d = _shape(v, v, v, o)
    for name, t, n in (("q8", q8, d), ("k8", k8, d), ("q_scales", q_scales, d // 32),
                       ("k_scales", k_scales, d // 32)):
        if not isinstance(t, torch.Tensor) or t.dtype != torch.uint8:
            raise TypeError(f"{name} must be a uint8 tensor")
        if not t.is_cuda or not t.is_contiguous() or tuple(t.shape) != (B, H, N, n):
            raise ValueError(f"{name} must be a contiguous GPU tensor of shape {(B, H, N, n)}")
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    st, mk, ls = _buffers(B, H, N, stats_out, mask_out, lse_out, tile_q, tile_k)
    a = DsAttnArgs(rule, param, q8.data_ptr(), k8.data_ptr(), v.data_ptr(), o.data_ptr(),
                   B, H, N, d, scale, tile_q, tile_k, _stream(stream), st, mk, ls,
                   key_order, None, QK_MXFP8, q_scales.data_ptr(), k_scales.data_ptr())
    _check(lib().dsattn_attn_fwd_ex(ctypes.byref(a)), "dsattn_attn_fwd_ex")
    return o


def dsattn_block_order(grid, block):
    """Gather map (numpy int32 [T*Y*X]) of the blocked token order, computed by the
    library's host code: position i of the reordered sequence holds token perm[i]."""
    import numpy as np

    T, Y, X = (int(g) for g in grid)
    bt, by, bx = (int(b) for b in block)
    n = max(T, 0) * max(Y, 0) * max(X, 0)
    perm = np.empty(max(n, 1), dtype=np.int32)
    rc = lib().dsattn_block_order(T, Y, X, bt, by, bx, perm.ctypes.data)
    _check(rc, "dsattn_block_order")
    return perm[:n]


def _rows(src, index, dst):
    import torch

    if not isinstance(src, torch.Tensor) or not src.is_cuda or not src.is_contiguous():
        raise ValueError("src must be a contiguous GPU tensor")
    if src.dim() < 2:
        raise ValueError("src must have shape [..., N, row]")
    if index.dtype != torch.int32 or not index.is_cuda or not index.is_contiguous():
        raise ValueError("index must be a contiguous int32 GPU tensor")
    N = int(src.shape[-2])
    if index.numel() != N:
        raise ValueError(f"index must have N={N} entries (got {index.numel()})")
    row_bytes = int(src.shape[-1]) * src.element_size()
    bh = src.numel() // max(1, N * int(src.shape[-1]))
    dst = torch.empty_like(src) if dst is None else dst
    if dst.shape != src.shape or dst.dtype != src.dtype or not dst.is_contiguous():
        raise ValueError("dst must be a contiguous tensor like src")
    return dst, bh, N, row_bytes


def dsattn_gather_rows(src, index, dst=None, stream=None):
    """dst[..., i, :] = src[..., index[i], :] on the GPU; returns dst."""
    dst, bh, N, row_bytes = _rows(src, index, dst)
    rc = lib().dsattn_gather_rows(src.data_ptr(), dst.data_ptr(), index.data_ptr(), bh, N,
                                  row_bytes, _stream(stream))
    _check(rc, "dsattn_gather_rows")
    return dst


def dsattn_scatter_rows(src, index, dst=None, stream=None):
    """dst[..., index[i], :] = src[..., i, :] on the GPU; returns dst."""
    dst, bh, N, row_bytes = _rows(src, index, dst)
    rc = lib().dsattn_scatter_rows(src.data_ptr(), dst.data_ptr(), index.data_ptr(), bh, N,
                                   row_bytes, _stream(stream))
    _check(rc, "dsattn_scatter_rows")
    return dst


def dsattn_quantize_mxfp8(x, codes=None, scales=None, shift=None, stream=None):
    """MX-FP8 codes (uint8, like x) and E8M0 block scales (uint8 [..., n / 32]) of a
    contiguous bf16 GPU tensor whose last axis is a multiple of 32.  With ``shift`` (float32
    [B, H, n] for x [B, H, N, n], e.g. from ``dsattn_key_mean``) every row first has its
    head's vector subtracted (key smoothing)."""
    import torch

    if x.dtype != torch.bfloat16 or not x.is_cuda or not x.is_contiguous():
        raise ValueError("x must be a contiguous bf16 GPU tensor")
    n = int(x.shape[-1])
    rows = x.numel() // max(1, n)
    codes = torch.empty(x.shape, dtype=torch.uint8, device=x.device) if codes is None else codes
    if scales is None:
        scales = torch.empty((*x.shape[:-1], n // 32), dtype=torch.uint8, device=x.device)
    if shift is None:
        rc = lib().dsattn_quantize_mxfp8(x.data_ptr(), codes.data_ptr(), scales.data_ptr(), rows,
                                         n, _stream(stream))
        _check(rc, "dsattn_quantize_mxfp8")
        return codes, scales
    if x.dim() != 4 or tuple(shift.shape) != (x.shape[0], x.shape[1], n) or \
            shift.dtype != torch.float32 or not shift.is_cuda or not shift.is_contiguous():
        raise ValueError("shift must be a contiguous float32 GPU tensor [B, H, n] for x [B, H, N, n]")
    rc = lib().dsattn_quantize_mxfp8_shift(x.data_ptr(), shift.data_ptr(), codes.data_ptr(),
                                           scales.data_ptr(), rows, n, int(x.shape[2]),
                                           _stream(stream))
    _check(rc, "dsattn_quantize_mxfp8_shift")
    return codes, scales


def dsattn_key_mean(k, out=None, stream=None):
    """Mean key of every head: float32 [B, H, d] of a contiguous bf16 GPU tensor
    [B, H, N, d] (fixed summation order)."""
    import torch

    if k.dtype != torch.bfloat16 or not k.is_cuda or not k.is_contiguous() or k.dim() != 4:
        raise ValueError("k must be a contiguous bf16 GPU tensor [B, H, N, d]")
    B, H, N, d = (int(x) for x in k.shape)
    out = torch.empty((B, H, d), dtype=torch.float32, device=k.device) if out is None else out
    rc = lib().dsattn_key_mean(k.data_ptr(), out.data_ptr(), B * H, N, d, _stream(stream))
    _check(rc, "dsattn_key_mean")
    return out


def dsattn_reordered_workspace_bytes(B, H, N, d=HEAD_DIM, with_lse=False):
    return int(lib().dsattn_reordered_workspace_bytes(B, H, N, d, int(bool(with_lse))))


def dsattn_attn_fwd_reordered(rule, param, q, k, v, q_index, kv_index, o=None, scale=None,
                              tile_q=TILE_Q, tile_k=TILE_K, stats_out=None, mask_out=None,
                              lse_out=None, workspace=None, stream=None,
                              key_order=ORDER_ASCENDING):
    """``dsattn_attn_fwd_ex`` over queries taken in ``q_index`` order and keys/values in
    ``kv_index`` order (int32 GPU tensors); o and lse_out come back in the original query
    order, mask_out and stats_out describe the reordered tiles.  ``workspace`` (a uint8
    GPU tensor) is allocated here when not given."""
    import torch

    o = _out(q, o)
    B, H, N, d = _shape(q, k, v, o)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    st, mk, ls = _buffers(B, H, N, stats_out, mask_out, lse_out, tile_q, tile_k)
    for name, t in (("q_index", q_index), ("kv_index", kv_index)):
        if t.dtype != torch.int32 or not t.is_cuda or not t.is_contiguous() or t.numel() != N:
            raise ValueError(f"{name} must be a contiguous int32 GPU tensor of N={N} entries")
    need = dsattn_reordered_workspace_bytes(B, H, N, d, lse_out is not None)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    a = DsAttnArgs(rule, param, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                   B, H, N, d, scale, tile_q, tile_k, _stream(stream), st, mk, ls, key_order)
    rc = lib().dsattn_attn_fwd_reordered(ctypes.byref(a), q_index.data_ptr(),
                                         kv_index.data_ptr(), workspace.data_ptr(),
                                         workspace.numel() * workspace.element_size())
    _check(rc, "dsattn_attn_fwd_reordered")
    return o


STATIC_SCRATCH_BYTES = 96 << 20    # DSATTN_STATIC_SCRATCH_BYTES of include/dsattn.h


def dsattn_attn_fwd_reordered_noalloc(rule, param, q, k, v, q_index, kv_index, o=None,
                                      scale=None, tile_q=TILE_Q, tile_k=TILE_K, stats_out=None,
                                      mask_out=None, lse_out=None, stream=None,
                                      key_order=ORDER_ASCENDING):
    """``dsattn_attn_fwd_reordered`` with the workspace taken from the library's static
    per-GPU scratch (at most STATIC_SCRATCH_BYTES): the C call allocates nothing.  Pass
    ``o`` (and any optional outputs) to keep this wrapper from allocating either."""
    import torch

    o = _out(q, o)
    B, H, N, d = _shape(q, k, v, o)
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    st, mk, ls = _buffers(B, H, N, stats_out, mask_out, lse_out, tile_q, tile_k)
    for name, t in (("q_index", q_index), ("kv_index", kv_index)):
        if t.dtype != torch.int32 or not t.is_cuda or not t.is_contiguous() or t.numel() != N:
            raise ValueError(f"{name} must be a contiguous int32 GPU tensor of N={N} entries")
    a = DsAttnArgs(rule, param, q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                   B, H, N, d, scale, tile_q, tile_k, _stream(stream), st, mk, ls, key_order)
    rc = lib().dsattn_attn_fwd_reordered_noalloc(ctypes.byref(a), q_index.data_ptr(),
                                                 kv_index.data_ptr())
    _check(rc, "dsattn_attn_fwd_reordered_noalloc")
    return o


__all__ = [
    "HEAD_DIM", "TILE_Q", "TILE_K", "ORDER_ASCENDING", "ORDER_DIAGONAL", "RULE_DENSE", "RULE_BLASST", "RULE_DYNSPARSE_RECALL",
    "RULE_DYNSPARSE_LAMBDA", "RULE_MASK", "DsAttnArgs", "lib", "last_error", "dsattn_lambda_from_recall",
    "dynsparse_attn_fwd", "dynsparse_attn_fwd_lambda", "blasst_attn_fwd", "dense_attn_fwd",
    "dsattn_attn_fwd_ex", "dsattn_block_order", "dsattn_gather_rows", "dsattn_scatter_rows",
    "dsattn_reordered_workspace_bytes", "dsattn_attn_fwd_reordered",
    "dsattn_attn_fwd_reordered_noalloc", "STATIC_SCRATCH_BYTES", "dsattn_quantize_mxfp8",
    "dsattn_attn_fwd_mxfp8", "dsattn_key_mean", "QK_BF16", "QK_MXFP8",
]
