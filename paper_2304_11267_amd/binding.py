"""ctypes binding of libsdattn.so (argument marshalling only).

Every function takes torch tensors that already live on the GPU, passes their
device pointers, sizes and the current HIP stream to the C entry point of the
same name, and raises :class:`SdattnError` on a nonzero status.  No
arithmetic of the attention happens here.  The library is loaded from the
package directory on first use; a missing library raises, there is no other
code path.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_NAME = "libsdattn.so"

STATUS_OK = 0
STATUS_INVALID_ARG = 1
STATUS_UNSUPPORTED = 2
STATUS_MISALIGNED = 3
STATUS_HIP = 4
STATUS_SCRATCH = 5

DTYPE_F16 = 0
DTYPE_BF16 = 1
DTYPE_F32 = 2

# every symbol include/sdattn.h declares
EXPORTS = ("sdattn_forward", "sdattn_forward_ex", "sdattn_softmax_rows", "sdattn_logits",
           "sdattn_softmax_pv", "sdattn_linear", "sdattn_attention_block_workspace",
           "sdattn_attention_block", "sdattn_attention_block_static", "sdattn_project_kv",
           "sdattn_attention_block_kv",
           "sdattn_group_norm", "sdattn_geglu", "sdattn_winograd_weights_elems",
           "sdattn_winograd_weights", "sdattn_conv3x3_workspace", "sdattn_conv3x3",
           "sdattn_status_str", "sdattn_last_hip_error", "sdattn_version")

LAYOUT_ROWS = 0
LAYOUT_HEADS = 1

_lib = None


class SdattnError(RuntimeError):
    def __init__(self, fn: str, status: int, hip_error: int, text: str):
        super().__init__(f"{fn} failed: status {status} ({text}), hip error {hip_error}")
        self.status = status
        self.hip_error = hip_error


def library_path() -> str:
    return os.environ.get("SDATTN_LIBRARY", os.path.join(HERE, LIB_NAME))


def load_library():
    """Load libsdattn.so and declare its signatures (raises if it is missing)."""
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build() "
                           "(the HIP library is the only implementation)")
    lib = ctypes.CDLL(path)
    vp, i32, i64, f32 = ctypes.c_void_p, ctypes.c_int, ctypes.c_longlong, ctypes.c_float
    lib.sdattn_forward.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, f32, vp]
    lib.sdattn_forward.restype = i32
    lib.sdattn_forward_ex.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, f32, i32, vp]
    lib.sdattn_forward_ex.restype = i32
    lib.sdattn_softmax_rows.argtypes = [vp, vp, vp, i64, i64, f32, i32, vp]
    lib.sdattn_softmax_rows.restype = i32
    lib.sdattn_logits.argtypes = [vp, vp, vp, i32, i32, i32, i32, i32, f32, i32, i32, vp]
    lib.sdattn_logits.restype = i32
    lib.sdattn_softmax_pv.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, vp]
    lib.sdattn_softmax_pv.restype = i32
    lib.sdattn_linear.argtypes = [vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, i32, i32, vp]
    lib.sdattn_linear.restype = i32
    lib.sdattn_attention_block_workspace.argtypes = [i32, i32, i32, i32]
    lib.sdattn_attention_block_workspace.restype = i64
    lib.sdattn_attention_block.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp, i64, i32, i32, i32,
                                           i32, i32, i32, f32, i32, vp]
    lib.sdattn_attention_block.restype = i32
    lib.sdattn_attention_block_static.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i32, i32, i32, i32,
                                                  i32, i32, f32, i32, vp]
    lib.sdattn_attention_block_static.restype = i32
    lib.sdattn_project_kv.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, vp]
    lib.sdattn_project_kv.restype = i32
    lib.sdattn_attention_block_kv.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, i64, i32, i32, i32,
                                              i32, i32, f32, i32, vp]
    lib.sdattn_attention_block_kv.restype = i32
    lib.sdattn_group_norm.argtypes = [vp, vp, vp, vp, i32, i32, i64, i32, f32, i32, vp]
    lib.sdattn_group_norm.restype = i32
    lib.sdattn_geglu.argtypes = [vp, vp, i64, i32, i32, vp]
    lib.sdattn_geglu.restype = i32
    lib.sdattn_winograd_weights_elems.argtypes = [i32, i32]
    lib.sdattn_winograd_weights_elems.restype = i64
    lib.sdattn_winograd_weights.argtypes = [vp, vp, i32, i32, i32, vp]
    lib.sdattn_winograd_weights.restype = i32
    lib.sdattn_conv3x3_workspace.argtypes = [i32, i32, i32, i32, i32]
    lib.sdattn_conv3x3_workspace.restype = i64
    lib.sdattn_conv3x3.argtypes = [vp, vp, vp, vp, vp, i64, i32, i32, i32, i32, i32, i32, vp]
    lib.sdattn_conv3x3.restype = i32
    lib.sdattn_status_str.argtypes = [i32]
    lib.sdattn_status_str.restype = ctypes.c_char_p
    lib.sdattn_last_hip_error.argtypes = []
    lib.sdattn_last_hip_error.restype = i32
    lib.sdattn_version.argtypes = []
    lib.sdattn_version.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _check(fn: str, status: int):
    if status != STATUS_OK:
        lib = load_library()
        raise SdattnError(fn, status, lib.sdattn_last_hip_error(),
                          lib.sdattn_status_str(status).decode())


def _dtype_code(t):
    import torch
    if t.dtype == torch.float16:
        return DTYPE_F16
    if t.dtype == torch.bfloat16:
        return DTYPE_BF16
    if t.dtype == torch.float32:
        return DTYPE_F32
    raise TypeError(f"unsupported element type {t.dtype}")


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dev(t, name):
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _expect(t, shape, like, name):
    """Raise unless tensor t has exactly `shape` and the element type of `like`:
    the C entry points see only pointers and sizes, so a tensor smaller than
    the sizes say would be read or written past its end."""
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if like is not None and t.dtype != like.dtype:
        raise TypeError(f"{name} is {t.dtype}, expected {like.dtype}")


def forward(q, k, v, out, scale: float, stream=None):
    """out = softmax(scale * q k^T) v for q/out [B,H,Lq,D], k/v [B,H,Lk,D], fp16."""
    B, H, Lq, D = q.shape
    Lk = k.shape[2]
    _expect(k, (B, H, Lk, D), q, "k")
    _expect(v, (B, H, Lk, D), q, "v")
    _expect(out, q.shape, q, "out")
    status = load_library().sdattn_forward(
        _dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out"),
        B, H, Lq, Lk, D, ctypes.c_float(scale), _stream(stream))
    _check("sdattn_forward", status)
    return out


def forward_ex(q, k, v, out, scale: float, ls=None, stream=None):
    """forward for fp16 or bf16, optionally writing fp32 (L, S) per row to ls [B,H,Lq,2]."""
    B, H, Lq, D = q.shape
    Lk = k.shape[2]
    _expect(k, (B, H, Lk, D), q, "k")
    _expect(v, (B, H, Lk, D), q, "v")
    _expect(out, q.shape, q, "out")
    if ls is not None:
        _expect(ls, (B, H, Lq, 2), None, "ls")
        if ls.element_size() != 4:
            raise TypeError("ls must hold float32")
    ls_ptr = _dev(ls, "ls") if ls is not None else None
    status = load_library().sdattn_forward_ex(
        _dev(q, "q"), _dev(k, "k"), _dev(v, "v"), _dev(out, "out"), ls_ptr,
        B, H, Lq, Lk, D, ctypes.c_float(scale), _dtype_code(q), _stream(stream))
    _check("sdattn_forward_ex", status)
    return out


def softmax_rows(a, ls, p=None, scale: float = 1.0, stream=None):
    """Eq. 4 on a [rows, cols]: ls[r] = (L_r, S_r) fp32; p (optional) = exp(scale*a - L)/S."""
    rows, cols = a.shape
    if ls.numel() != 2 * rows or ls.element_size() != 4:
        raise ValueError("ls must hold 2 float32 values per row")
    if p is not None:
        _expect(p, a.shape, a, "p")
    p_ptr = _dev(p, "p") if p is not None else None
    status = load_library().sdattn_softmax_rows(
        _dev(a, "a"), _dev(ls, "ls"), p_ptr, rows, cols, ctypes.c_float(scale),
        _dtype_code(a), _stream(stream))
    _check("sdattn_softmax_rows", status)
    return ls


def logits(q, k, a, scale: float, stream=None):
    """a = scale * q k^T: q [B,H,Lq,D], k [B,H,Lk,D] (fp16/bf16), a [B,H,Lq,Lk] (fp16/bf16/fp32)."""
    B, H, Lq, D = q.shape
    Lk = k.shape[2]
    _expect(k, (B, H, Lk, D), q, "k")
    _expect(a, (B, H, Lq, Lk), None, "a")
    status = load_library().sdattn_logits(
        _dev(q, "q"), _dev(k, "k"), _dev(a, "a"), B, H, Lq, Lk, D, ctypes.c_float(scale),
        _dtype_code(q), _dtype_code(a), _stream(stream))
    _check("sdattn_logits", status)
    return a


def softmax_pv(a, ls, v, out, stream=None):
    """out = exp(a - L) / S times v, with (L, S) = ls [B,H,Lq,2] fp32 of a's rows."""
    B, H, Lq, Lk = a.shape
    D = v.shape[3]
    _expect(v, (B, H, Lk, D), None, "v")
    _expect(out, (B, H, Lq, D), v, "out")
    if ls.numel() != 2 * B * H * Lq or ls.element_size() != 4:
        raise ValueError("ls must hold 2 float32 values per row")
    status = load_library().sdattn_softmax_pv(
        _dev(a, "a"), _dev(ls, "ls"), _dev(v, "v"), _dev(out, "out"), B, H, Lq, Lk, D,
        _dtype_code(a), _dtype_code(v), _stream(stream))
    _check("sdattn_softmax_pv", status)
    return out


def linear(x, w, y, bias=None, heads=1, x_layout=LAYOUT_ROWS, y_layout=LAYOUT_ROWS, stream=None):
    """y = x w^T + bias over token rows.  Rows layout tensors are [B, L, C], heads layout
    [B, H, L, C/H]; w is [N, K] (out, in)."""
    if x_layout == LAYOUT_HEADS:
        B, H, L, hw = x.shape
        K = H * hw
    else:
        B, L, K = x.shape
    N = w.shape[0]
    _expect(w, (N, K), x, "w")
    if bias is not None:
        _expect(bias, (N,), x, "bias")
    if y_layout == LAYOUT_HEADS:
        if heads < 1 or N % heads:
            raise ValueError("heads must divide the output channels")
        _expect(y, (B, heads, L, N // heads), x, "y")
    else:
        _expect(y, (B, L, N), x, "y")
    if x_layout == LAYOUT_HEADS and H != heads:
        raise ValueError("x's head count differs from heads")
    status = load_library().sdattn_linear(
        _dev(x, "x"), _dev(w, "w"), _dev(bias, "bias") if bias is not None else None, _dev(y, "y"),
        B, L, K, N, heads, x_layout, y_layout, _dtype_code(x), _stream(stream))
    _check("sdattn_linear", status)
    return y


def attention_block_workspace(B, Lq, Lk, C):
    """Bytes of workspace sdattn_attention_block needs."""
    return int(load_library().sdattn_attention_block_workspace(B, Lq, Lk, C))


def attention_block(x, ctx, wq, wk, wv, wo, bo, out, workspace, heads, scale, stream=None):
    """SD's attention block: out = MHA(x, ctx) with weights [out, in]; workspace is a device
    tensor of at least attention_block_workspace(...) bytes."""
    B, Lq, C = x.shape
    Lk, Cc = ctx.shape[1], ctx.shape[2]
    _expect(ctx, (B, Lk, Cc), x, "ctx")
    for t, shape, name in ((wq, (C, C), "wq"), (wk, (C, Cc), "wk"), (wv, (C, Cc), "wv"),
                           (wo, (C, C), "wo"), (out, (B, Lq, C), "out")):
        _expect(t, shape, x, name)
    if bo is not None:
        _expect(bo, (C,), x, "bo")
    status = load_library().sdattn_attention_block(
        _dev(x, "x"), _dev(ctx, "ctx"), _dev(wq, "wq"), _dev(wk, "wk"), _dev(wv, "wv"),
        _dev(wo, "wo"), _dev(bo, "bo") if bo is not None else None, _dev(out, "out"),
        _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
        B, Lq, Lk, C, Cc, heads, ctypes.c_float(scale), _dtype_code(x), _stream(stream))
    _check("sdattn_attention_block", status)
    return out


def attention_block_static(x, ctx, wq, wk, wv, wo, bo, out, heads, scale, stream=None):
    """attention_block through the library's static scratch (no workspace argument)."""
    B, Lq, C = x.shape
    Lk, Cc = ctx.shape[1], ctx.shape[2]
    _expect(ctx, (B, Lk, Cc), x, "ctx")
    for t, shape, name in ((wq, (C, C), "wq"), (wk, (C, Cc), "wk"), (wv, (C, Cc), "wv"),
                           (wo, (C, C), "wo"), (out, (B, Lq, C), "out")):
        _expect(t, shape, x, name)
    if bo is not None:
        _expect(bo, (C,), x, "bo")
    status = load_library().sdattn_attention_block_static(
        _dev(x, "x"), _dev(ctx, "ctx"), _dev(wq, "wq"), _dev(wk, "wk"), _dev(wv, "wv"),
        _dev(wo, "wo"), _dev(bo, "bo") if bo is not None else None, _dev(out, "out"),
        B, Lq, Lk, C, Cc, heads, ctypes.c_float(scale), _dtype_code(x), _stream(stream))
    _check("sdattn_attention_block_static", status)
    return out


def project_kv(ctx, wk, wv, k, v, heads, stream=None):
    """K = ctx wk^T, V = ctx wv^T split into heads: ctx [B, Lk, Cc], k, v [B, H, Lk, C/H]."""
    B, Lk, Cc = ctx.shape
    C = wk.shape[0]
    _expect(wk, (C, Cc), ctx, "wk")
    _expect(wv, (C, Cc), ctx, "wv")
    if heads < 1 or C % heads:
        raise ValueError("heads must divide the channels")
    _expect(k, (B, heads, Lk, C // heads), ctx, "k")
    _expect(v, (B, heads, Lk, C // heads), ctx, "v")
    status = load_library().sdattn_project_kv(
        _dev(ctx, "ctx"), _dev(wk, "wk"), _dev(wv, "wv"), _dev(k, "k"), _dev(v, "v"),
        B, Lk, Cc, C, heads, _dtype_code(ctx), _stream(stream))
    _check("sdattn_project_kv", status)
    return k, v


def attention_block_kv(x, wq, k, v, wo, bo, out, workspace, scale, stream=None):
    """The attention block with K and V given in heads layout [B, H, Lk, C/H];
    workspace of at least attention_block_workspace(B, Lq, 0, C) bytes."""
    B, Lq, C = x.shape
    H, Lk = k.shape[1], k.shape[2]
    _expect(k, (B, H, Lk, C // H), x, "k")
    _expect(v, k.shape, x, "v")
    for t, shape, name in ((wq, (C, C), "wq"), (wo, (C, C), "wo"), (out, (B, Lq, C), "out")):
        _expect(t, shape, x, name)
    if bo is not None:
        _expect(bo, (C,), x, "bo")
    status = load_library().sdattn_attention_block_kv(
        _dev(x, "x"), _dev(wq, "wq"), _dev(k, "k"), _dev(v, "v"), _dev(wo, "wo"),
        _dev(bo, "bo") if bo is not None else None, _dev(out, "out"), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), B, Lq, Lk, C, H, ctypes.c_float(scale),
        _dtype_code(x), _stream(stream))
    _check("sdattn_attention_block_kv", status)
    return out


def group_norm(x, groups, y, gamma=None, beta=None, eps=1e-5, stream=None):
    """Group normalisation of channel-major feature maps x [B, C, ...] into y
    (same shape; y may be x); gamma, beta [C] or None."""
    B, C = x.shape[:2]
    HW = 1
    for d in x.shape[2:]:
        HW *= d
    _expect(y, x.shape, x, "y")
    for t, name in ((gamma, "gamma"), (beta, "beta")):
        if t is not None:
            _expect(t, (C,), x, name)
    status = load_library().sdattn_group_norm(
        _dev(x, "x"), _dev(gamma, "gamma") if gamma is not None else None,
        _dev(beta, "beta") if beta is not None else None, _dev(y, "y"), B, C, HW, groups,
        ctypes.c_float(eps), _dtype_code(x), _stream(stream))
    _check("sdattn_group_norm", status)
    return y


def geglu(h, out, stream=None):
    """out[..., f] = h[..., f] * GELU(h[..., F + f]) for h [..., 2F], out [..., F]."""
    F2 = h.shape[-1]
    if F2 % 2:
        raise ValueError("h's last axis must have an even length")
    F = F2 // 2
    _expect(out, tuple(h.shape[:-1]) + (F,), h, "out")
    M = h.numel() // F2
    status = load_library().sdattn_geglu(_dev(h, "h"), _dev(out, "out"), M, F, _dtype_code(h),
                                         _stream(stream))
    _check("sdattn_geglu", status)
    return out


def winograd_weights(w, u, stream=None):
    """u [36, Co, Ci] = the F(4x4, 3x3) transform of the kernels w [Co, Ci, 3, 3]."""
    Co, Ci = w.shape[:2]
    _expect(w, (Co, Ci, 3, 3), None, "w")
    _expect(u, (36, Co, Ci), w, "u")
    status = load_library().sdattn_winograd_weights(_dev(w, "w"), _dev(u, "u"), Co, Ci,
                                                     _dtype_code(w), _stream(stream))
    _check("sdattn_winograd_weights", status)
    return u


def conv3x3_workspace(B, Ci, Co, H, W):
    """Bytes of workspace sdattn_conv3x3 needs."""
    return int(load_library().sdattn_conv3x3_workspace(B, Ci, Co, H, W))


def conv3x3(x, u, y, workspace, bias=None, stream=None):
    """y [B, Co, H, W] = 3x3 convolution (stride 1, zero padding 1) of x [B, Ci, H, W]
    with the transformed kernels u [36, Co, Ci] (from winograd_weights) + bias [Co]."""
    B, Ci, H, W = x.shape
    Co = u.shape[1]
    _expect(u, (36, Co, Ci), x, "u")
    _expect(y, (B, Co, H, W), x, "y")
    if bias is not None:
        _expect(bias, (Co,), x, "bias")
    status = load_library().sdattn_conv3x3(
        _dev(x, "x"), _dev(u, "u"), _dev(bias, "bias") if bias is not None else None, _dev(y, "y"),
        _dev(workspace, "workspace"), workspace.numel() * workspace.element_size(),
        B, Ci, Co, H, W, _dtype_code(x), _stream(stream))
    _check("sdattn_conv3x3", status)
    return y
