"""GPU parity of the partially fused softmax (Sec. 3.2.1) as separate steps:
sdattn_logits -> sdattn_softmax_rows -> sdattn_softmax_pv, against the fp64
oracle's logits, softmax_pv and attention on the same seeded inputs.

Bounds are derived from the arithmetic the kernels perform:
* logits accumulate exact fp16/bf16 products in fp32 and apply the fp32
  scale, so |g - r| <= (D + 2) 2^-22 |scale| sum_d |q_d k_d| (a wide margin
  over the 2^-24 unit roundoff), plus half an output ulp when A is stored in
  fp16 or bf16;
* the attention outputs use the forward tolerance (parity_util.TOL).
With A stored in fp16 the method computes attention of the fp16-rounded
logits; its reference is the oracle evaluated on the oracle's own logits
rounded to fp16 (numpy's correctly rounded conversion).
"""
import numpy as np
import pytest

import oracle
import paper_2304_11267_amd as sd
from paper_2304_11267_amd import workloads as wl

from parity_util import TOL, assert_close, to_device, to_host64, ulp

pytestmark = pytest.mark.gpu

A_TYPES = {"f16": None, "bf16": None, "f32": None}


@pytest.fixture(scope="module", autouse=True)
def _needs_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    sd.load_library()
    A_TYPES.update(f16=torch.float16, bf16=torch.bfloat16, f32=torch.float32)


def gpu_logits(q, k, scale, a_type, dtype="f16"):
    import torch
    qd, kd = to_device(q, dtype), to_device(k, dtype)
    B, H, Lq, _ = q.shape
    a = torch.empty(B, H, Lq, k.shape[2], dtype=A_TYPES[a_type], device="cuda")
    sd.logits(qd, kd, a, scale)
    torch.cuda.synchronize()
    return a


def gpu_chain(q, k, v, scale, a_type, dtype="f16"):
    """logits -> softmax_rows -> softmax_pv on the GPU; returns (O, A) device tensors."""
    import torch
    a = gpu_logits(q, k, scale, a_type, dtype)
    B, H, Lq, Lk = a.shape
    ls = torch.empty(B, H, Lq, 2, dtype=torch.float32, device="cuda")
    sd.softmax_rows(a.view(B * H * Lq, Lk), ls.view(B * H * Lq, 2), None, scale=1.0)
    vd = to_device(v, dtype)
    out = torch.empty(B, H, Lq, v.shape[3], dtype=vd.dtype, device="cuda")
    sd.softmax_pv(a, ls, vd, out)
    torch.cuda.synchronize()
    return out, a


def logits_bound(q, k, scale, dtype=None):
    qa = np.abs(oracle.widen(q, dtype=dtype))
    ka = np.abs(oracle.widen(k, dtype=dtype))
    D = q.shape[3]
    return (D + 2) * 2.0 ** -22 * abs(scale) * np.matmul(qa, np.swapaxes(ka, 2, 3))


LOGIT_SHAPES = [
    # (B, H, Lq, Lk, D): ragged query and key tiles, unaligned rows (Lk % 8 != 0)
    (1, 2, 130, 256, 40),
    (2, 1, 97, 77, 80),
    (1, 1, 33, 129, 160),
    (1, 2, 64, 200, 24),
    (1, 1, 40, 64, 256),
]


@pytest.mark.parametrize("a_type", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("shape", LOGIT_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_logits_match_oracle(shape, a_type):
    B, H, Lq, Lk, D = shape
    q, k, _ = wl.make_qkv(B, H, Lq, Lk, D, 5000 + Lq + Lk + D)
    scale = float(np.float32(1 / np.sqrt(D)))
    g = to_host64(gpu_logits(q, k, scale, a_type))
    r = oracle.logits(q, k, scale)
    bound = logits_bound(q, k, scale)
    if a_type == "f16":
        bound = bound + 0.5 * ulp(r, "f16")
    elif a_type == "bf16":
        bound = bound + 0.5 * ulp(r, "bf16")
    assert np.all(np.abs(g - r) <= bound), np.max(np.abs(g - r) - bound)


def test_logits_bf16_inputs_and_negative_scale():
    q, k, _ = wl.make_qkv(1, 2, 70, 136, 64, 5100, dtype="bf16")
    g = to_host64(gpu_logits(q, k, -0.3, "f32", dtype="bf16"))
    r = oracle.logits(q, k, -0.3, dtype="bf16")
    assert np.all(np.abs(g - r) <= logits_bound(q, k, -0.3, dtype="bf16"))


@pytest.mark.parametrize("a_type", ["f32", "f16"])
@pytest.mark.parametrize("Lk", [64, 77, 200, 1024])
def test_softmax_pv_on_given_logits(Lk, a_type):
    """O from a seeded synthetic A, with (L, S) from the GPU's softmax_rows."""
    import torch
    B, H, Lq, D = 1, 2, 150, 40
    rng = np.random.default_rng(5200 + Lk)
    a = (rng.standard_normal((B, H, Lq, Lk), dtype=np.float32) * np.float32(2.5))
    a = a.astype(np.float16) if a_type == "f16" else a
    _, _, v = wl.make_qkv(B, H, 1, Lk, D, 5300 + Lk)
    ad = torch.from_numpy(a).cuda()
    ls = torch.empty(B, H, Lq, 2, dtype=torch.float32, device="cuda")
    sd.softmax_rows(ad.view(B * H * Lq, Lk), ls.view(B * H * Lq, 2), None, scale=1.0)
    vd = to_device(v)
    out = torch.empty(B, H, Lq, D, dtype=torch.float16, device="cuda")
    sd.softmax_pv(ad, ls, vd, out)
    torch.cuda.synchronize()
    r = oracle.softmax_pv(a, v)
    assert_close(to_host64(out), r, what=f"Lk={Lk} A={a_type}")


@pytest.mark.parametrize("name", ["mid8_self", "l16_self", "l16_self_peaked", "mid8_cross",
                                  "l32_cross"])
def test_chain_with_fp32_logits_is_attention(name):
    case = wl.CASES[name]
    q, k, v = wl.case_inputs(case)
    out, _ = gpu_chain(q, k, v, case.scale, "f32")
    r, _, _ = oracle.attention(q, k, v, case.scale)
    assert_close(to_host64(out), r, what=name)


@pytest.mark.parametrize("name,per_head", [("l32_self", 24), ("l64_self", 12)])
def test_chain_at_full_size_sampled_rows(name, per_head):
    case = wl.CASES[name]
    q, k, v = wl.case_inputs(case)
    out, _ = gpu_chain(q, k, v, case.scale, "f32")
    rows = wl.sample_rows(case.B, case.H, case.Lq, per_head, seed=case.seed)
    r, _, _ = oracle.attention(q, k, v, case.scale, rows=rows)
    assert_close(to_host64(out).reshape(-1, case.D)[rows], r, what=name)


def _rounded_logit_reference(q, k, v, scale, rows_by_head):
    """Oracle attention of the fp16-rounded oracle logits for the listed rows of
    each head, and the most the GPU's output may differ from it because a
    logit computed in fp32 can round to the neighbouring fp16 value: only
    logits whose exact value lies within the fp32 error bound of a rounding
    midpoint can flip, each by the gap to its neighbour, which moves o_i by
    p_ij * gap * (v_j - o_i) to first order (x1.1 for the second order)."""
    B, H, Lq, D = q.shape
    ref, extra = {}, {}
    for (b, h), idx in rows_by_head.items():
        flat = (b * H + h) * Lq + np.asarray(idx)
        a64 = oracle.logits(q, k, scale, rows=flat)
        a16 = a64.astype(np.float16)
        vb = v[b:b + 1, h:h + 1]
        o = oracle.softmax_pv(a16.reshape(1, 1, len(idx), -1), vb).reshape(len(idx), D)
        _, _, p = oracle.softmax_rows(a16.astype(np.float64), want_p=True)
        eps = logits_bound(q[b:b + 1, h:h + 1, idx], k[b:b + 1, h:h + 1], scale).reshape(a64.shape)
        lo = np.nextafter(a16, np.float16(-np.inf)).astype(np.float64)
        hi = np.nextafter(a16, np.float16(np.inf)).astype(np.float64)
        c = a16.astype(np.float64)
        near_lo = np.abs(a64 - (lo + c) / 2) <= eps
        near_hi = np.abs(a64 - (c + hi) / 2) <= eps
        gap = np.where(near_lo, c - lo, 0.0) + np.where(near_hi, hi - c, 0.0)
        vf = oracle.widen(vb).reshape(-1, D)
        dev = np.abs(vf[None, :, :] - o[:, None, :])             # |v_j - o_i|, [rows, Lk, D]
        extra[(b, h)] = 1.1 * np.einsum("ij,ijd->id", p * gap, dev)
        ref[(b, h)] = o
    return ref, extra


@pytest.mark.parametrize("name,per_head", [("l16_self", 256), ("l16_self_peaked", 256),
                                           ("l64_self", 8)])
def test_chain_with_fp16_logits(name, per_head):
    case = wl.CASES[name]
    q, k, v = wl.case_inputs(case)
    out, a = gpu_chain(q, k, v, case.scale, "f16")
    g = to_host64(out)
    rng = np.random.default_rng(case.seed + 7)
    rows_by_head = {(b, h): np.sort(rng.choice(case.Lq, size=min(per_head, case.Lq), replace=False))
                    for b in range(case.B) for h in range(case.H)}
    ref, extra = _rounded_logit_reference(q, k, v, case.scale, rows_by_head)
    got = np.concatenate([g[b, h, idx] for (b, h), idx in rows_by_head.items()])
    exp = np.concatenate([ref[key] for key in rows_by_head])
    ext = np.concatenate([extra[key] for key in rows_by_head])
    atol, rtol = TOL["f16"]
    diff = np.abs(got - exp)
    ratio = diff / (np.maximum(atol, ulp(exp)) + ext)
    assert np.all(np.isfinite(got)) and ratio.max() <= 1.0, (name, float(diff.max()), float(ratio.max()))
    rms = float(np.sqrt(np.mean(exp * exp)))
    assert (np.maximum(diff - ext, 0.0) / np.maximum(np.abs(exp), rms)).max() <= rtol
    # the flip term is a small correction, not a blanket allowance
    assert float(np.mean(ext)) < atol


def test_chain_bf16():
    q, k, v = wl.make_qkv(1, 2, 200, 136, 80, 5400, dtype="bf16")
    scale = float(np.float32(1 / np.sqrt(80)))
    out, _ = gpu_chain(q, k, v, scale, "f32", dtype="bf16")
    r, _, _ = oracle.attention(q, k, v, scale, dtype="bf16")
    assert_close(to_host64(out), r, "bf16", what="bf16 chain")


@pytest.mark.parametrize("Lk", [8, 64, 72, 136, 264])
def test_softmax_pv_uneven_key_halves_after_nan_lds(Lk):
    """Key counts whose tiles split unevenly between the two wave halves (or
    leave the second half none), run right after a kernel that left NaN in LDS:
    a half must not multiply p = 0 by a V buffer it never filled."""
    import torch
    nan = np.full((2, 8, 512, 64), np.nan, dtype=np.float16)
    nd = torch.from_numpy(nan).cuda()
    sd.forward(nd, nd, nd, torch.empty_like(nd), 0.125)   # K/V tiles of NaN in LDS
    B, H, Lq, D = 2, 4, 300, 40
    rng = np.random.default_rng(5500 + Lk)
    a = (rng.standard_normal((B, H, Lq, Lk), dtype=np.float32) * np.float32(2.0)).astype(np.float16)
    _, _, v = wl.make_qkv(B, H, 1, Lk, D, 5600 + Lk)
    ad = torch.from_numpy(a).cuda()
    ls = torch.empty(B, H, Lq, 2, dtype=torch.float32, device="cuda")
    sd.softmax_rows(ad.view(-1, Lk), ls.view(-1, 2), None, scale=1.0)
    out = torch.empty(B, H, Lq, D, dtype=torch.float16, device="cuda")
    sd.softmax_pv(ad, ls, to_device(v), out)
    torch.cuda.synchronize()
    assert_close(to_host64(out), oracle.softmax_pv(a, v), what=f"Lk={Lk}")
