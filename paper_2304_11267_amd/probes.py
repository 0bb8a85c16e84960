"""ctypes binding of libsdattn_probes.so (include/sdattn_probes.h): the
measurement kernels behind the sustained rates the benchmark reports beside
the datasheet peaks.  Argument marshalling only; a missing library raises.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_NAME = "libsdattn_probes.so"

# every symbol include/sdattn_probes.h declares
EXPORTS = ("sdattn_probe_mix", "sdattn_probe_tile", "sdattn_probe_copy", "sdattn_probe_read",
           "sdattn_probe_strip_copy")

MIX_MFMA, MIX_FMA, MIX_EXP = 0, 1, 2
MIX_MFMA_FMA, MIX_MFMA_EXP = 3, 4
MIX_MFMA_HALF, MIX_FMA_HALF, MIX_EXP_HALF = 5, 6, 7
MIX_MFMA_NOISE = 8
MFMA_FLOPS_PER_ITER = 4 * 2 * 32 * 32 * 16     # four 32x32x16 MFMAs per wave and iteration
VALU_OPS_PER_ITER = 16

_lib = None


def library_path() -> str:
    return os.path.join(HERE, LIB_NAME)


def load_library():
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build()")
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_longlong
    lib.sdattn_probe_mix.argtypes = [i32, i32, i32, i32, vp, vp, vp]
    lib.sdattn_probe_tile.argtypes = [i32, i32, i32, i32, vp, vp, vp]
    lib.sdattn_probe_copy.argtypes = [vp, vp, i64, i32, vp]
    lib.sdattn_probe_read.argtypes = [vp, i64, vp, i32, vp]
    lib.sdattn_probe_strip_copy.argtypes = [vp, vp, vp, vp, vp, i32, i32, i32, i32, i32, i32, vp]
    for name in EXPORTS:
        getattr(lib, name).restype = i32
    _lib = lib
    return lib


def _check(name, rc):
    if rc != 0:
        raise RuntimeError(f"{name} failed: hip error {rc}")


def _stream(stream):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def mix(mode, blocks, it_m, it_v, out, clk=None, stream=None):
    _check("sdattn_probe_mix", load_library().sdattn_probe_mix(
        mode, blocks, it_m, it_v, ctypes.c_void_p(out.data_ptr()),
        ctypes.c_void_p(clk.data_ptr()) if clk is not None else None, _stream(stream)))


def tile(blocks, iters, exps, out, noise=False, clk=None, stream=None, stagger=0):
    _check("sdattn_probe_tile", load_library().sdattn_probe_tile(
        blocks, iters, (1 if exps else 0) | (2 if noise else 0), stagger, ctypes.c_void_p(out.data_ptr()),
        ctypes.c_void_p(clk.data_ptr()) if clk is not None else None, _stream(stream)))


def copy(src, dst, nbytes, blocks, stream=None):
    _check("sdattn_probe_copy", load_library().sdattn_probe_copy(
        ctypes.c_void_p(src.data_ptr()), ctypes.c_void_p(dst.data_ptr()), nbytes, blocks, _stream(stream)))


def read(src, nbytes, sink, blocks, stream=None):
    _check("sdattn_probe_read", load_library().sdattn_probe_read(
        ctypes.c_void_p(src.data_ptr()), nbytes, ctypes.c_void_p(sink.data_ptr()), blocks, _stream(stream)))


def strip_copy(q, k, v, o, sink, waves=8, stream=None):
    B, H, Lq, D = q.shape
    Lk = k.shape[2]
    _check("sdattn_probe_strip_copy", load_library().sdattn_probe_strip_copy(
        *(ctypes.c_void_p(t.data_ptr()) for t in (q, k, v, o, sink)), B, H, Lq, Lk, D, waves, _stream(stream)))
