"""The C ABI on the host: the library loads, exports what include/sdattn.h
declares, and rejects bad arguments with the documented status before any
HIP call (so these run without a GPU; the pointers are never dereferenced).
"""
import ctypes
import os
import re

import pytest

from paper_2304_11267_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sdattn.h")

OK, INVALID, UNSUPPORTED, MISALIGNED, HIPERR = 0, 1, 2, 3, 4
F16, BF16, F32 = 0, 1, 2

# fake, well-aligned, non-overlapping device addresses (never touched)
QA, KA, VA, OA, LA = (ctypes.c_void_p(x) for x in (0x10000000, 0x20000000, 0x30000000,
                                                   0x40000000, 0x50000000))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(binding.library_path()):
        pytest.skip("libsdattn.so not built")
    return binding.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sdattn_\w+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(binding.EXPORTS)


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_status_strings(lib):
    for code in (OK, INVALID, UNSUPPORTED, MISALIGNED, HIPERR, 99, -1):
        s = lib.sdattn_status_str(code)
        assert isinstance(s, bytes) and len(s) > 0
    assert lib.sdattn_status_str(OK) == b"ok"
    assert lib.sdattn_status_str(99) == b"unknown status"
    assert lib.sdattn_last_hip_error() == 0
    assert b"gfx950" in lib.sdattn_version()


def fwd(lib, q=QA, k=KA, v=VA, o=OA, B=2, H=8, Lq=64, Lk=77, D=40, scale=0.158):
    return lib.sdattn_forward(q, k, v, o, B, H, Lq, Lk, D, ctypes.c_float(scale), None)


def fwd_ex(lib, ls=None, dtype=F16, **kw):
    a = dict(q=QA, k=KA, v=VA, o=OA, B=2, H=8, Lq=64, Lk=77, D=40, scale=0.158)
    a.update(kw)
    return lib.sdattn_forward_ex(a["q"], a["k"], a["v"], a["o"], ls, a["B"], a["H"], a["Lq"],
                                 a["Lk"], a["D"], ctypes.c_float(a["scale"]), dtype, None)


@pytest.mark.parametrize("field", ["q", "k", "v", "o"])
def test_null_pointer_is_invalid(lib, field):
    assert fwd(lib, **{field: None}) == INVALID


@pytest.mark.parametrize("field", ["B", "H", "Lq", "Lk", "D"])
@pytest.mark.parametrize("value", [0, -3])
def test_nonpositive_sizes_are_invalid(lib, field, value):
    assert fwd(lib, **{field: value}) == INVALID


@pytest.mark.parametrize("scale", [float("inf"), float("-inf"), float("nan")])
def test_nonfinite_scale_is_invalid(lib, scale):
    assert fwd(lib, scale=scale) == INVALID


@pytest.mark.parametrize("D", [4, 12, 41, 264, 512])
def test_unsupported_head_width(lib, D):
    assert fwd(lib, D=D) == UNSUPPORTED


def test_oversized_problem_is_unsupported(lib):
    assert fwd(lib, B=1 << 20, H=1 << 20, Lq=1 << 20, D=8) == UNSUPPORTED


@pytest.mark.parametrize("field", ["q", "k", "v", "o"])
def test_misaligned_pointer(lib, field):
    base = {"q": 0x10000000, "k": 0x20000000, "v": 0x30000000, "o": 0x40000000}[field]
    assert fwd(lib, **{field: ctypes.c_void_p(base + 8)}) == MISALIGNED


def test_output_overlapping_an_input_is_invalid(lib):
    # q spans 2*8*64*40*2 bytes from QA; put out inside it
    assert fwd(lib, o=ctypes.c_void_p(0x10000000 + 4096)) == INVALID
    assert fwd(lib, o=KA) == INVALID
    assert fwd(lib, o=ctypes.c_void_p(0x30000000 - 16)) == INVALID   # out's tail runs into v


def test_forward_ex_checks(lib):
    assert fwd_ex(lib, dtype=F32) == UNSUPPORTED
    assert fwd_ex(lib, dtype=7) == INVALID
    assert fwd_ex(lib, ls=ctypes.c_void_p(0x50000004)) == MISALIGNED
    assert fwd_ex(lib, ls=ctypes.c_void_p(0x40000000 + 64)) == INVALID   # ls inside out
    assert fwd_ex(lib, dtype=BF16, D=44) == UNSUPPORTED


def sm(lib, a=QA, ls=LA, p=None, rows=16, cols=4096, scale=1.0, dtype=F16):
    return lib.sdattn_softmax_rows(a, ls, p, rows, cols, ctypes.c_float(scale), dtype, None)


def test_softmax_rows_checks(lib):
    assert sm(lib, a=None) == INVALID
    assert sm(lib, ls=None) == INVALID
    assert sm(lib, rows=0) == INVALID
    assert sm(lib, cols=-1) == INVALID
    assert sm(lib, scale=float("nan")) == INVALID
    assert sm(lib, dtype=9) == INVALID
    assert sm(lib, rows=1 << 40, cols=1 << 30) == UNSUPPORTED
    assert sm(lib, a=ctypes.c_void_p(0x10000002)) == MISALIGNED
    assert sm(lib, p=ctypes.c_void_p(0x30000008)) == MISALIGNED
    assert sm(lib, ls=ctypes.c_void_p(0x50000004)) == MISALIGNED
    assert sm(lib, ls=ctypes.c_void_p(0x10000000 + 1024)) == INVALID    # ls inside a
    assert sm(lib, p=ctypes.c_void_p(0x10000000 + 4096)) == INVALID     # p overlaps a
    assert sm(lib, p=ctypes.c_void_p(0x50000000 - 64)) == INVALID       # p overlaps ls


def test_rejected_calls_leave_no_hip_error(lib):
    fwd(lib, q=None)
    sm(lib, a=None)
    assert lib.sdattn_last_hip_error() == 0


def test_binding_raises_when_library_missing(monkeypatch, tmp_path):
    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setenv("SDATTN_LIBRARY", str(tmp_path / "absent.so"))
    with pytest.raises(RuntimeError, match="not built"):
        binding.load_library()


def lg(lib, q=QA, k=KA, a=OA, B=2, H=8, Lq=64, Lk=77, D=40, scale=0.158, dtype=F16, a_dtype=F16):
    return lib.sdattn_logits(q, k, a, B, H, Lq, Lk, D, ctypes.c_float(scale), dtype, a_dtype, None)


def pv(lib, a=QA, ls=LA, v=VA, o=OA, B=2, H=8, Lq=64, Lk=77, D=40, a_dtype=F16, dtype=F16):
    return lib.sdattn_softmax_pv(a, ls, v, o, B, H, Lq, Lk, D, a_dtype, dtype, None)


def test_logits_checks(lib):
    for field in ("q", "k", "a"):
        assert lg(lib, **{field: None}) == INVALID
    for field in ("B", "H", "Lq", "Lk", "D"):
        assert lg(lib, **{field: 0}) == INVALID
    assert lg(lib, scale=float("nan")) == INVALID
    assert lg(lib, dtype=F32) == UNSUPPORTED
    assert lg(lib, a_dtype=9) == INVALID
    assert lg(lib, D=44) == UNSUPPORTED
    assert lg(lib, B=1 << 20, H=1 << 20, Lq=1 << 12, Lk=1 << 12) == UNSUPPORTED
    assert lg(lib, a=ctypes.c_void_p(0x40000000 + 8)) == MISALIGNED
    assert lg(lib, a=ctypes.c_void_p(0x20000000 - 64)) == INVALID        # a's tail runs into k
    assert lg(lib, a=ctypes.c_void_p(0x10000000 + 4096), a_dtype=F32) == INVALID   # inside q


def test_softmax_pv_checks(lib):
    for field in ("a", "ls", "v", "o"):
        assert pv(lib, **{field: None}) == INVALID
    for field in ("B", "H", "Lq", "Lk", "D"):
        assert pv(lib, **{field: -1}) == INVALID
    assert pv(lib, dtype=F32) == UNSUPPORTED
    assert pv(lib, a_dtype=5) == INVALID
    assert pv(lib, D=300) == UNSUPPORTED
    assert pv(lib, ls=ctypes.c_void_p(0x50000004)) == MISALIGNED
    assert pv(lib, v=ctypes.c_void_p(0x30000008)) == MISALIGNED
    assert pv(lib, o=ctypes.c_void_p(0x10000000 + 1024)) == INVALID      # out inside a
    assert pv(lib, o=ctypes.c_void_p(0x50000000 - 64)) == INVALID        # out's tail runs into ls


ROWS, HEADS_L = 0, 1


def lin(lib, x=QA, w=KA, b=None, y=OA, B=2, L=64, K=320, N=320, H=8, xl=ROWS, yl=HEADS_L, dtype=F16):
    return lib.sdattn_linear(x, w, b, y, B, L, K, N, H, xl, yl, dtype, None)


def test_linear_checks(lib):
    for field in ("x", "w", "y"):
        assert lin(lib, **{field: None}) == INVALID
    for field in ("B", "L", "K", "N"):
        assert lin(lib, **{field: 0}) == INVALID
    assert lin(lib, H=0) == INVALID
    assert lin(lib, xl=2) == INVALID
    assert lin(lib, dtype=F32) == UNSUPPORTED
    assert lin(lib, K=324) == UNSUPPORTED               # K % 8
    assert lin(lib, K=65544) == UNSUPPORTED             # K above 65536
    assert lin(lib, N=320, H=3) == UNSUPPORTED          # heads do not divide N
    assert lin(lib, N=96, H=8) == UNSUPPORTED           # head width 12 % 8
    assert lin(lib, y=ctypes.c_void_p(0x40000000 + 4)) == MISALIGNED
    assert lin(lib, y=ctypes.c_void_p(0x10000000 + 1024)) == INVALID   # y inside x
    assert lin(lib, b=ctypes.c_void_p(0x40000000 + 64)) == INVALID    # bias inside y


def blk(lib, ws=ctypes.c_void_p(0x60000000), wsb=1 << 26, **kw):
    a = dict(x=QA, ctx=KA, wq=ctypes.c_void_p(0x70000000), wk=ctypes.c_void_p(0x71000000),
             wv=ctypes.c_void_p(0x72000000), wo=ctypes.c_void_p(0x73000000),
             bo=ctypes.c_void_p(0x74000000), out=OA, B=2, Lq=64, Lk=77, C=320, Cc=768, H=8,
             scale=0.158, dtype=F16)
    a.update(kw)
    return lib.sdattn_attention_block(a["x"], a["ctx"], a["wq"], a["wk"], a["wv"], a["wo"], a["bo"],
                                      a["out"], ws, wsb, a["B"], a["Lq"], a["Lk"], a["C"], a["Cc"],
                                      a["H"], ctypes.c_float(a["scale"]), a["dtype"], None)


def test_attention_block_checks(lib):
    need = lib.sdattn_attention_block_workspace(2, 64, 77, 320)
    assert need >= 2 * 2 * (2 * 64 * 320 + 2 * 77 * 320)
    assert blk(lib, wsb=need - 1) == INVALID
    assert blk(lib, ws=None) == INVALID
    assert blk(lib, ws=ctypes.c_void_p(0x60000008)) == MISALIGNED
    assert blk(lib, C=321, H=8) == INVALID              # heads do not divide C
    assert blk(lib, C=96, H=8) == UNSUPPORTED           # head width 12
    assert blk(lib, Cc=770) == UNSUPPORTED              # context channels % 8
    assert blk(lib, scale=float("inf")) == INVALID
    assert blk(lib, out=ctypes.c_void_p(0x60000000 + 4096)) == INVALID   # out inside the workspace
    assert blk(lib, x=ctypes.c_void_p(0x60000000 + 1024)) == INVALID     # x inside the workspace


def test_attention_block_static_refuses_before_any_hip_call(lib):
    # the sizes and pointers it can check without the scratch's device address
    def bst(**kw):
        a = dict(x=QA, ctx=KA, wq=ctypes.c_void_p(0x70000000), wk=ctypes.c_void_p(0x71000000),
                 wv=ctypes.c_void_p(0x72000000), wo=ctypes.c_void_p(0x73000000),
                 bo=ctypes.c_void_p(0x74000000), out=OA, B=2, Lq=64, Lk=77, C=320, Cc=768, H=8,
                 scale=0.158, dtype=F16)
        a.update(kw)
        return lib.sdattn_attention_block_static(a["x"], a["ctx"], a["wq"], a["wk"], a["wv"], a["wo"],
                                                 a["bo"], a["out"], a["B"], a["Lq"], a["Lk"], a["C"],
                                                 a["Cc"], a["H"], ctypes.c_float(a["scale"]), a["dtype"],
                                                 None)
    SCRATCH = 5
    for field in ("x", "ctx", "wq", "wk", "wv", "wo", "out"):
        assert bst(**{field: None}) == INVALID
    assert bst(B=0) == INVALID
    assert bst(C=321) == INVALID                        # heads do not divide C
    # 32 MiB of scratch: the 64x64-level self block at B = 2 needs 21 MB, at B = 4 42 MB
    assert lib.sdattn_attention_block_workspace(2, 4096, 4096, 320) <= 32 << 20
    assert lib.sdattn_attention_block_workspace(4, 4096, 4096, 320) > 32 << 20
    assert bst(B=4, Lq=4096, Lk=4096, C=320, Cc=320) == SCRATCH
    assert lib.sdattn_status_str(SCRATCH) == b"needs more than the static scratch holds"
    assert lib.sdattn_last_hip_error() == 0


def test_project_kv_checks(lib):
    W1, W2 = ctypes.c_void_p(0x71000000), ctypes.c_void_p(0x72000000)

    def pkv(ctx=KA, wk=W1, wv=W2, k=QA, v=VA, B=2, Lk=77, Cc=768, C=320, H=8, dtype=F16):
        return lib.sdattn_project_kv(ctx, wk, wv, k, v, B, Lk, Cc, C, H, dtype, None)
    for field in ("ctx", "wk", "wv", "k", "v"):
        assert pkv(**{field: None}) == INVALID
    assert pkv(H=0) == INVALID
    assert pkv(C=321) == INVALID                        # heads do not divide C
    assert pkv(C=96) == UNSUPPORTED                     # head width 12
    assert pkv(Cc=770) == UNSUPPORTED                   # context channels % 8
    assert pkv(v=ctypes.c_void_p(0x10000000 + 4096)) == INVALID   # v overlaps k
    assert pkv(k=ctypes.c_void_p(0x10000008)) == MISALIGNED


def test_attention_block_kv_checks(lib):
    def bkv(ws=ctypes.c_void_p(0x60000000), wsb=1 << 26, **kw):
        a = dict(x=QA, wq=ctypes.c_void_p(0x70000000), k=KA, v=VA, wo=ctypes.c_void_p(0x73000000),
                 bo=ctypes.c_void_p(0x74000000), out=OA, B=2, Lq=64, Lk=77, C=320, H=8,
                 scale=0.158, dtype=F16)
        a.update(kw)
        return lib.sdattn_attention_block_kv(a["x"], a["wq"], a["k"], a["v"], a["wo"], a["bo"],
                                             a["out"], ws, wsb, a["B"], a["Lq"], a["Lk"], a["C"],
                                             a["H"], ctypes.c_float(a["scale"]), a["dtype"], None)
    need = lib.sdattn_attention_block_workspace(2, 64, 0, 320)
    assert need == 2 * ((2 * 2 * 64 * 320 + 255) // 256 * 256)
    assert bkv(wsb=need - 1) == INVALID
    for field in ("x", "wq", "k", "v", "wo", "out"):
        assert bkv(**{field: None}) == INVALID
    assert bkv(ws=None) == INVALID
    assert bkv(C=321) == INVALID
    assert bkv(C=96) == UNSUPPORTED
    assert bkv(scale=float("nan")) == INVALID
    assert bkv(k=ctypes.c_void_p(0x60000000 + 512)) == INVALID   # k inside the workspace


def test_group_norm_checks(lib):
    def gn(x=QA, gamma=KA, beta=VA, y=OA, B=2, C=320, HW=4096, G=32, eps=1e-5, dtype=F16):
        return lib.sdattn_group_norm(x, gamma, beta, y, B, C, HW, G, ctypes.c_float(eps), dtype, None)
    for field in ("x", "y"):
        assert gn(**{field: None}) == INVALID
    for field in ("B", "C", "HW", "G"):
        assert gn(**{field: 0}) == INVALID
    assert gn(G=33) == INVALID                          # groups do not divide C
    assert gn(eps=-1e-5) == INVALID
    assert gn(eps=float("inf")) == INVALID
    assert gn(dtype=F32) == UNSUPPORTED
    assert gn(dtype=7) == INVALID
    assert gn(x=ctypes.c_void_p(0x10000008)) == MISALIGNED
    assert gn(gamma=ctypes.c_void_p(0x20000001)) == MISALIGNED
    assert gn(y=ctypes.c_void_p(0x10000000 + 4096)) == INVALID     # partial overlap with x
    assert gn(gamma=ctypes.c_void_p(0x40000000 + 64)) == INVALID   # gamma inside y


def test_geglu_checks(lib):
    def ge(h=QA, out=OA, M=8192, F=1280, dtype=F16):
        return lib.sdattn_geglu(h, out, M, F, dtype, None)
    for field in ("h", "out"):
        assert ge(**{field: None}) == INVALID
    assert ge(M=0) == INVALID
    assert ge(F=0) == INVALID
    assert ge(F=1284) == UNSUPPORTED                    # F % 8
    assert ge(dtype=F32) == UNSUPPORTED
    assert ge(out=ctypes.c_void_p(0x40000004)) == MISALIGNED
    assert ge(out=ctypes.c_void_p(0x10000000 + 2 * 1280 * 2)) == INVALID   # out inside h


def test_winograd_checks_and_table2_factors(lib):
    import os
    # Table 2, 4x4 tile: weights grow 4x, the transformed input 2.25x
    path = os.path.join(os.path.dirname(__file__), "golden", "winograd_table2.txt")
    row = [list(map(float, l.split())) for l in open(path) if l.strip() and not l.startswith("#")][1]
    assert row[0] == 4
    assert lib.sdattn_winograd_weights_elems(320, 640) == row[3] * 9 * 320 * 640
    B, Ci, Co, H, W = 2, 320, 640, 64, 64
    part = lambda e: (2 * e + 255) // 256 * 256
    T = B * (H // 4) * (W // 4)
    ws = lib.sdattn_conv3x3_workspace(B, Ci, Co, H, W)
    assert ws == part(36 * T * Ci) + part(36 * T * Co)
    assert 36 * T * Ci == row[2] * B * Ci * H * W
    assert lib.sdattn_conv3x3_workspace(0, Ci, Co, H, W) == -1

    U = ctypes.c_void_p(0x60000000)

    def wt(w=KA, u=U, Co=64, Ci=32, dtype=F16):
        return lib.sdattn_winograd_weights(w, u, Co, Ci, dtype, None)
    assert wt(w=None) == INVALID and wt(u=None) == INVALID and wt(Co=0) == INVALID
    assert wt(dtype=F32) == UNSUPPORTED
    assert wt(u=ctypes.c_void_p(0x60000008)) == MISALIGNED
    assert wt(u=ctypes.c_void_p(0x20000000 + 64)) == INVALID     # u overlaps w

    def cv(x=QA, u=U, bias=VA, y=OA, ws=ctypes.c_void_p(0x50000000), wsb=1 << 24, B=1, Ci=32,
           Co=64, H=16, W=16, dtype=F16):
        return lib.sdattn_conv3x3(x, u, bias, y, ws, wsb, B, Ci, Co, H, W, dtype, None)
    for field in ("x", "u", "y", "ws"):
        assert cv(**{field: None}) == INVALID
    for field in ("B", "Ci", "Co", "H", "W"):
        assert cv(**{field: 0}) == INVALID
    assert cv(Ci=36) == UNSUPPORTED                     # Ci % 8
    assert cv(Co=20) == UNSUPPORTED                     # Co % 8
    assert cv(dtype=F32) == UNSUPPORTED
    assert cv(wsb=lib.sdattn_conv3x3_workspace(1, 32, 64, 16, 16) - 1) == INVALID
    assert cv(x=ctypes.c_void_p(0x10000008)) == MISALIGNED
    assert cv(y=ctypes.c_void_p(0x10000000 + 256)) == INVALID      # y overlaps x
    assert cv(ws=ctypes.c_void_p(0x60000000 + 512)) == INVALID     # workspace overlaps u


# ------------------------------------------------ the measurement kernels

def test_probe_library_exports_every_declared_symbol():
    from paper_2304_11267_amd import probes
    if not os.path.exists(probes.library_path()):
        pytest.skip("libsdattn_probes.so not built")
    text = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "sdattn_probes.h")).read(), flags=re.S)
    declared = sorted(set(re.findall(r"\b(sdattn_probe_\w+)\s*\(", text)))
    assert declared == sorted(probes.EXPORTS)
    plib = probes.load_library()
    for name in declared:
        assert hasattr(plib, name), name
    # out-of-range arguments are refused before any launch (hipErrorInvalidValue = 1)
    assert plib.sdattn_probe_mix(9, 1, 1, 1, QA, None, None) == 1
    assert plib.sdattn_probe_mix(-1, 1, 1, 1, QA, None, None) == 1
    assert plib.sdattn_probe_tile(1, 0, 1, 0, QA, None, None) == 1
    assert plib.sdattn_probe_tile(1, 1, 4, 0, QA, None, None) == 1
    assert plib.sdattn_probe_tile(1, 1, 1, 65, QA, None, None) == 1
    assert plib.sdattn_probe_copy(QA, KA, 15, 1, None) == 1
    assert plib.sdattn_probe_copy(QA, ctypes.c_void_p(0x10000010), 4096, 1, None) == 1   # overlap
    assert plib.sdattn_probe_read(QA, 0, KA, 1, None) == 1
    assert plib.sdattn_probe_strip_copy(QA, KA, VA, OA, LA, 2, 8, 4096, 77, 12, 8, None) == 1
    assert plib.sdattn_probe_strip_copy(QA, KA, VA, OA, LA, 2, 8, 4096, 129, 40, 8, None) == 1
    assert plib.sdattn_probe_strip_copy(QA, KA, VA, OA, LA, 2, 8, 4096, 77, 40, 3, None) == 1
