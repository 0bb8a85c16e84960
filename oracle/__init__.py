"""fp64 CPU oracle for SD attention -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never does, and
this package imports nothing from the product.

It binds ``liboracle.so`` (built from ``oracle.c``; see that file for the
passages of the paper each function follows):

* :func:`attention` -- Eq. 3 in three passes per row (max, exp-sum,
  normalise times V), returning O and Eq. 4's L and S.
* :func:`softmax_rows` -- Eq. 4's reduction (L, S) on a given matrix and the
  element-wise step p = exp(a - L) / S.
* :func:`logits` and :func:`softmax_pv` -- the first and last steps of the
  partially fused softmax (Sec. 3.2.1): A = scale Q K^T, and
  O = exp(A - L) / S times V.
* :func:`linear` and :func:`attention_block` -- the projections around the
  attention in SD's transformer blocks and the whole multi-head block.
* :func:`group_norm`, :func:`gelu` and :func:`geglu` -- the specialised
  kernels of Sec. 3.1: group normalisation (Eq. 1) and GELU (Eq. 2) with its
  split and multiply.
* :func:`conv3x3` -- the 3x3 convolution (stride 1, zero padding 1) that
  Sec. 3.3 computes with Winograd's algorithm, by its definition.

Inputs are numpy arrays: float16, float32, float64, or bfloat16 passed as a
uint16 bit-pattern array with ``dtype="bf16"``.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_F16, _BF16, _F32, _F64 = 0, 1, 2, 3
_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB) or (
                os.path.getmtime(_build.LIB) < os.path.getmtime(_build.SRC)):
            _build.build()
        lib = ctypes.CDLL(_build.LIB)
        vp, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_float
        lib.oracle_attention_f64.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, i32,
                                             f32, vp, i64, i32, vp, vp, vp, vp]
        lib.oracle_attention_f64.restype = i32
        lib.oracle_softmax_rows_f64.argtypes = [vp, i32, i64, i64, f32, i32, vp, vp]
        lib.oracle_softmax_rows_f64.restype = i32
        lib.oracle_logits_f64.argtypes = [vp, vp, i32, i32, i32, i32, i32, i32, f32, vp, i64,
                                          i32, vp]
        lib.oracle_logits_f64.restype = i32
        lib.oracle_softmax_pv_f64.argtypes = [vp, i32, vp, vp, i32, i32, i32, i32, i32, i32,
                                              vp, i64, i32, vp]
        lib.oracle_softmax_pv_f64.restype = i32
        lib.oracle_linear_f64.argtypes = [vp, i32, vp, i32, vp, i64, i32, i32, i32, vp]
        lib.oracle_linear_f64.restype = i32
        lib.oracle_attention_block_f64.argtypes = [vp, vp, vp, vp, vp, vp, vp, i32, i32, i32, i32,
                                                   i32, i32, i32, f32, vp, i64, i32, vp]
        lib.oracle_attention_block_f64.restype = i32
        f64 = ctypes.c_double
        lib.oracle_group_norm_f64.argtypes = [vp, i32, vp, vp, i32, i32, i64, i32, f64, i32, vp,
                                              vp, vp]
        lib.oracle_group_norm_f64.restype = i32
        lib.oracle_gelu_f64.argtypes = [vp, i32, i64, vp]
        lib.oracle_gelu_f64.restype = i32
        lib.oracle_geglu_f64.argtypes = [vp, i32, i64, i32, i32, vp]
        lib.oracle_geglu_f64.restype = i32
        lib.oracle_conv3x3_f64.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, vp]
        lib.oracle_conv3x3_f64.restype = i32
        lib.oracle_widen.argtypes = [vp, i32, i64, vp]
        lib.oracle_widen.restype = i32
        lib.oracle_num_threads.argtypes = [i32]
        lib.oracle_num_threads.restype = i32
        _lib = lib
    return _lib


def _code(arr, dtype):
    if dtype == "bf16":
        if arr.dtype != np.uint16:
            raise TypeError("bf16 inputs are passed as uint16 bit patterns")
        return _BF16
    if dtype is not None and dtype != "auto":
        raise ValueError(f"unknown dtype tag {dtype!r}")
    return {np.dtype(np.float16): _F16, np.dtype(np.float32): _F32,
            np.dtype(np.float64): _F64}[arr.dtype]


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def num_threads(requested: int = 0) -> int:
    """Threads the oracle's OpenMP regions use for ``requested`` (0 = default)."""
    return _load().oracle_num_threads(int(requested))


def widen(x, dtype=None):
    """Exact widening of a float16 / bfloat16 (uint16) / float32 array to float64."""
    x = np.ascontiguousarray(x)
    code = _code(x, dtype)
    out = np.empty(x.shape, dtype=np.float64)
    if _load().oracle_widen(_ptr(x), code, x.size, _ptr(out)) != 0:
        raise ValueError("oracle_widen rejected its arguments")
    return out


def attention(q, k, v, scale, rows=None, dtype=None, nthreads=0, want_dev=False):
    """Eq. 3 in fp64.  q: [B,H,Lq,D], k, v: [B,H,Lk,D], same element type.

    rows: optional 1-D array of flat query-row indices (b*H + h)*Lq + i; the
    outputs then hold only those rows, in that order.
    Returns (O, L, S): O is [B,H,Lq,D] (or [len(rows), D]); L and S are
    Eq. 4's row maximum and shifted exponential sum, shaped like O[..., 0].
    With want_dev, also DEV shaped like O: dev_id = sum_j p_ij |v_jd - o_id|,
    the weighted mean absolute deviation of each value column (what a
    relative rounding of the weights can move o_id by, to first order).
    """
    q, k, v = (np.ascontiguousarray(t) for t in (q, k, v))
    if q.ndim != 4 or k.shape != v.shape or q.shape[:2] != k.shape[:2] or q.shape[3] != k.shape[3]:
        raise ValueError("expected q [B,H,Lq,D] and k, v [B,H,Lk,D]")
    if not (q.dtype == k.dtype == v.dtype):
        raise TypeError("q, k and v must share one element type")
    B, H, Lq, D = q.shape
    Lk = k.shape[2]
    code = _code(q, dtype)
    if rows is None:
        n, rp, shape = B * H * Lq, None, (B, H, Lq)
    else:
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        n, rp, shape = rows.size, _ptr(rows), (rows.size,)
    out = np.empty(shape + (D,), dtype=np.float64)
    L = np.empty(shape, dtype=np.float64)
    S = np.empty(shape, dtype=np.float64)
    dev = np.empty(shape + (D,), dtype=np.float64) if want_dev else None
    rc = _load().oracle_attention_f64(_ptr(q), _ptr(k), _ptr(v), code, B, H, Lq, Lk, D,
                                      float(np.float32(scale)), rp, n, int(nthreads),
                                      _ptr(out), _ptr(L), _ptr(S), _ptr(dev) if want_dev else None)
    if rc != 0:
        raise ValueError("oracle_attention_f64 rejected its arguments")
    return (out, L, S, dev) if want_dev else (out, L, S)


def softmax_rows(a, scale=1.0, want_p=False, dtype=None, nthreads=0):
    """Eq. 4 on a [rows, cols] matrix with a_ij = scale * A_ij.

    Returns (L, S) and, if want_p, also p = exp(a - L) / S (all fp64).
    """
    a = np.ascontiguousarray(a)
    if a.ndim != 2:
        raise ValueError("expected a 2-D matrix")
    code = _code(a, dtype)
    rows, cols = a.shape
    ls = np.empty((rows, 2), dtype=np.float64)
    p = np.empty((rows, cols), dtype=np.float64) if want_p else None
    rc = _load().oracle_softmax_rows_f64(_ptr(a), code, rows, cols, float(np.float32(scale)),
                                         int(nthreads), _ptr(ls), _ptr(p) if want_p else None)
    if rc != 0:
        raise ValueError("oracle_softmax_rows_f64 rejected its arguments")
    if want_p:
        return ls[:, 0], ls[:, 1], p
    return ls[:, 0], ls[:, 1]


def _rows_arg(rows, total):
    if rows is None:
        return total, None, None
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    return rows.size, rows, _ptr(rows)


def logits(q, k, scale, rows=None, dtype=None, nthreads=0):
    """A = scale * Q K^T in fp64 for q [B,H,Lq,D], k [B,H,Lk,D].

    Returns [B,H,Lq,Lk] (or [len(rows), Lk] for the flat query rows listed).
    """
    q, k = np.ascontiguousarray(q), np.ascontiguousarray(k)
    if q.ndim != 4 or k.ndim != 4 or q.shape[:2] != k.shape[:2] or q.shape[3] != k.shape[3]:
        raise ValueError("expected q [B,H,Lq,D] and k [B,H,Lk,D]")
    if q.dtype != k.dtype:
        raise TypeError("q and k must share one element type")
    B, H, Lq, D = q.shape
    Lk = k.shape[2]
    n, rows, rp = _rows_arg(rows, B * H * Lq)
    out = np.empty((n, Lk), dtype=np.float64)
    rc = _load().oracle_logits_f64(_ptr(q), _ptr(k), _code(q, dtype), B, H, Lq, Lk, D,
                                   float(np.float32(scale)), rp, n, int(nthreads), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_logits_f64 rejected its arguments")
    return out.reshape(B, H, Lq, Lk) if rows is None else out


def softmax_pv(a, v, ls=None, rows=None, a_dtype=None, v_dtype=None, nthreads=0):
    """O = exp(A - L) / S times V in fp64, for a [B,H,Lq,Lk] (scale applied) and v [B,H,Lk,D].

    ls: optional [B,H,Lq,2] (L, S) to use; None computes Eq. 4 from A.
    Returns [B,H,Lq,D] (or [len(rows), D]).
    """
    a, v = np.ascontiguousarray(a), np.ascontiguousarray(v)
    if a.ndim != 4 or v.ndim != 4 or a.shape[:2] != v.shape[:2] or a.shape[3] != v.shape[2]:
        raise ValueError("expected a [B,H,Lq,Lk] and v [B,H,Lk,D]")
    B, H, Lq, Lk = a.shape
    D = v.shape[3]
    lsp = None
    if ls is not None:
        ls = np.ascontiguousarray(ls, dtype=np.float64)
        if ls.size != B * H * Lq * 2:
            raise ValueError("ls must hold (L, S) for every row")
        lsp = _ptr(ls)
    n, rows, rp = _rows_arg(rows, B * H * Lq)
    out = np.empty((n, D), dtype=np.float64)
    rc = _load().oracle_softmax_pv_f64(_ptr(a), _code(a, a_dtype), lsp, _ptr(v), _code(v, v_dtype),
                                       B, H, Lq, Lk, D, rp, n, int(nthreads), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_softmax_pv_f64 rejected its arguments")
    return out.reshape(B, H, Lq, D) if rows is None else out


def linear(x, w, bias=None, dtype=None, nthreads=0):
    """y = x w^T + bias in fp64: x [..., K], w [N, K] (out, in), bias [N] like w.

    Returns [..., N].
    """
    x, w = np.ascontiguousarray(x), np.ascontiguousarray(w)
    K = x.shape[-1]
    if w.ndim != 2 or w.shape[1] != K:
        raise ValueError("expected x [..., K] and w [N, K]")
    N = w.shape[0]
    M = x.size // K
    bp = None
    if bias is not None:
        bias = np.ascontiguousarray(bias)
        if bias.shape != (N,) or bias.dtype != w.dtype:
            raise ValueError("bias must be [N] of w's type")
        bp = _ptr(bias)
    y = np.empty((M, N), dtype=np.float64)
    rc = _load().oracle_linear_f64(_ptr(x), _code(x, dtype), _ptr(w), _code(w, dtype), bp, M, K, N,
                                   int(nthreads), _ptr(y))
    if rc != 0:
        raise ValueError("oracle_linear_f64 rejected its arguments")
    return y.reshape(x.shape[:-1] + (N,))


def attention_block(x, ctx, wq, wk, wv, wo, bo, heads, scale, rows=None, dtype=None, nthreads=0):
    """SD's multi-head attention block in fp64 (see oracle.c): x [B,Lq,C], ctx [B,Lk,Cc],
    weights [out, in], bo [C] (or None).  Returns [B,Lq,C] (or [len(rows), C] for the
    flat rows b*Lq + i listed)."""
    arrs = [np.ascontiguousarray(t) for t in (x, ctx, wq, wk, wv, wo)]
    x, ctx, wq, wk, wv, wo = arrs
    if len({a.dtype for a in arrs}) != 1:
        raise TypeError("all tensors must share one element type")
    B, Lq, C = x.shape
    Lk, Cc = ctx.shape[1], ctx.shape[2]
    if wq.shape != (C, C) or wk.shape != (C, Cc) or wv.shape != (C, Cc) or wo.shape != (C, C):
        raise ValueError("weight shapes do not match x and ctx")
    bp = None
    if bo is not None:
        bo = np.ascontiguousarray(bo)
        bp = _ptr(bo)
    n, rows, rp = _rows_arg(rows, B * Lq)
    out = np.empty((n, C), dtype=np.float64)
    rc = _load().oracle_attention_block_f64(_ptr(x), _ptr(ctx), _ptr(wq), _ptr(wk), _ptr(wv),
                                            _ptr(wo), bp, _code(x, dtype), B, Lq, Lk, C, Cc,
                                            int(heads), float(np.float32(scale)), rp, n,
                                            int(nthreads), _ptr(out))
    if rc != 0:
        raise ValueError("oracle_attention_block_f64 rejected its arguments")
    return out.reshape(B, Lq, C) if rows is None else out


def group_norm(x, groups, gamma=None, beta=None, eps=1e-5, dtype=None, nthreads=0):
    """Group normalisation (Eq. 1 with eps and the per-channel affine terms) in
    fp64 of x [B, C, ...] (channel-major; the trailing axes are the pixels).

    eps is rounded to fp32 first (the value the GPU receives).
    Returns (y, mean, rstd): y like x, mean and rstd [B, groups].
    """
    x = np.ascontiguousarray(x)
    B, C = x.shape[:2]
    HW = int(np.prod(x.shape[2:])) if x.ndim > 2 else 1
    code = _code(x, dtype)
    gp = bp = None
    for t in (gamma, beta):
        if t is not None and (t.shape != (C,) or t.dtype != x.dtype):
            raise ValueError("gamma and beta must be [C] of x's type")
    if gamma is not None:
        gamma = np.ascontiguousarray(gamma)
        gp = _ptr(gamma)
    if beta is not None:
        beta = np.ascontiguousarray(beta)
        bp = _ptr(beta)
    y = np.empty(x.shape, dtype=np.float64)
    mean = np.empty((B, groups), dtype=np.float64)
    rstd = np.empty((B, groups), dtype=np.float64)
    rc = _load().oracle_group_norm_f64(_ptr(x), code, gp, bp, B, C, HW, groups,
                                       float(np.float32(eps)), int(nthreads), _ptr(y), _ptr(mean),
                                       _ptr(rstd))
    if rc != 0:
        raise ValueError("oracle_group_norm_f64 rejected its arguments")
    return y, mean, rstd


def gelu(x, dtype=None):
    """GELU of Eq. 2 element-wise in fp64 (erf form)."""
    x = np.ascontiguousarray(x)
    out = np.empty(x.shape, dtype=np.float64)
    if _load().oracle_gelu_f64(_ptr(x), _code(x, dtype), x.size, _ptr(out)) != 0:
        raise ValueError("oracle_gelu_f64 rejected its arguments")
    return out


def geglu(h, dtype=None, nthreads=0):
    """h [..., 2F] -> h[..., :F] * GELU(h[..., F:]) in fp64."""
    h = np.ascontiguousarray(h)
    if h.shape[-1] % 2:
        raise ValueError("the last axis must have an even length")
    F = h.shape[-1] // 2
    M = h.size // (2 * F)
    out = np.empty(h.shape[:-1] + (F,), dtype=np.float64)
    if _load().oracle_geglu_f64(_ptr(h), _code(h, dtype), M, F, int(nthreads), _ptr(out)) != 0:
        raise ValueError("oracle_geglu_f64 rejected its arguments")
    return out


def conv3x3(x, w, bias=None, dtype=None, nthreads=0):
    """3x3 convolution, stride 1, zero padding 1, in fp64: x [B, Ci, H, W],
    w [Co, Ci, 3, 3], bias [Co] (x's type).  Returns [B, Co, H, W]."""
    x, w = np.ascontiguousarray(x), np.ascontiguousarray(w)
    if x.ndim != 4 or w.ndim != 4 or w.shape[1] != x.shape[1] or w.shape[2:] != (3, 3):
        raise ValueError("expected x [B, Ci, H, W] and w [Co, Ci, 3, 3]")
    if x.dtype != w.dtype:
        raise TypeError("x and w must share one element type")
    B, Ci, H, W = x.shape
    Co = w.shape[0]
    bp = None
    if bias is not None:
        bias = np.ascontiguousarray(bias)
        if bias.shape != (Co,) or bias.dtype != x.dtype:
            raise ValueError("bias must be [Co] of x's type")
        bp = _ptr(bias)
    y = np.empty((B, Co, H, W), dtype=np.float64)
    rc = _load().oracle_conv3x3_f64(_ptr(x), _ptr(w), bp, _code(x, dtype), B, Ci, Co, H, W,
                                    int(nthreads), _ptr(y))
    if rc != 0:
        raise ValueError("oracle_conv3x3_f64 rejected its arguments")
    return y
