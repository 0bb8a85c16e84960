"""GPU parity of the specialised kernels of Sec. 3.1 against the fp64 oracle:
group normalisation (Eq. 1 with eps and the affine terms) and GELU (Eq. 2)
with its split and multiply.

Bounds derived from the arithmetic:
* group norm: the mean and the mean square deviation are fp32 sums of up to
  49152 terms (per-thread runs of at most 96, then a tree of 512), so each is
  within about 1e-5 of its size; y = (x - mu) rstd gamma + beta then carries
  |g - r| <= 1e-4 (|r - beta| + |gamma| rstd mean|x_g - 0|) (ten times that
  estimate) plus one output ulp for the final rounding;
* GEGLU: erf to within 3e-7 (the 1.5e-7 of the approximation plus the fp32
  reciprocal and exponential), so GELU(g) is within 0.5 |g| 3e-7 + 2^-21
  |GELU(g)| and out within |a| times that, plus one output ulp.
"""
import numpy as np
import pytest

import oracle
import paper_2304_11267_amd as sd
from paper_2304_11267_amd import workloads as wl

from parity_util import to_device, to_host64, ulp

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _needs_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    sd.load_library()


def gn_bound(x64, gamma64, beta64, r, mean, rstd, G, dtype):
    B, C = x64.shape[:2]
    xg = np.abs(x64.reshape(B, G, -1)).mean(axis=2)                     # mean |x| per group
    per_c = lambda v: np.repeat(v, C // G, axis=1)[:, :, None]           # [B, G] -> [B, C, 1]
    ga = np.abs(gamma64)[None, :, None] if gamma64 is not None else 1.0
    be = beta64[None, :, None] if beta64 is not None else 0.0
    r3 = r.reshape(B, C, -1)
    bound = 1e-4 * (np.abs(r3 - be) + ga * per_c(rstd) * per_c(xg)) + ulp(r3, dtype)
    return bound.reshape(r.shape)


def run_gn(x, gamma, beta, G, eps, dtype="f16", in_place=False):
    import torch
    xd = to_device(x, dtype)
    gd = to_device(gamma, dtype) if gamma is not None else None
    bd = to_device(beta, dtype) if beta is not None else None
    y = xd if in_place else torch.empty_like(xd)
    sd.group_norm(xd, G, y, gd, bd, eps)
    torch.cuda.synchronize()
    return to_host64(y)


def check_gn(x, gamma, beta, G, eps, dtype="f16", in_place=False):
    g = run_gn(x, gamma, beta, G, eps, dtype, in_place)
    r, mean, rstd = oracle.group_norm(x, G, gamma, beta, eps, dtype=dtype if dtype == "bf16" else None)
    w = lambda t: None if t is None else oracle.widen(t, dtype="bf16" if dtype == "bf16" else None)
    bound = gn_bound(w(x), w(gamma), w(beta), r, mean, rstd, G, dtype)
    assert np.all(np.isfinite(g))
    excess = np.abs(g - r) / bound
    assert excess.max() <= 1.0, (float(excess.max()), float(np.abs(g - r).max()))


@pytest.mark.parametrize("name", list(wl.NORM_CASES))
def test_group_norm_unet_levels(name):
    case = wl.NORM_CASES[name]
    x, gamma, beta = wl.norm_inputs(case)
    check_gn(x, gamma, beta, wl.GN_GROUPS, wl.GN_EPS)


@pytest.mark.parametrize("shape", [
    (1, 64, 4096, 2),      # 131072 values per group: the kernel that reads the run three times
    (2, 12, 30, 4),        # HW % 8 != 0: element-wise path
    (3, 32, 8, 32),        # one channel per group, 8 pixels
    (1, 96, 520, 3),       # 16640 values per group, ragged last chunk row
    (2, 8, 1, 8),          # one value per group: y = beta
], ids=lambda s: "x".join(map(str, s)))
def test_group_norm_shapes(shape):
    B, C, HW, G = shape
    x, gamma, beta = wl.make_norm(B, C, HW, 8000 + C + HW)
    check_gn(x, gamma, beta, G, 1e-5)


def test_group_norm_without_affine_and_eps_matters():
    # tiny-variance groups: eps = 1e-5 against var ~ 1e-6 changes y by ~3x
    rng = np.random.default_rng(8100)
    x = (5.0 + 1e-3 * rng.standard_normal((2, 64, 256))).astype(np.float16)
    check_gn(x, None, None, 32, 1e-5)
    check_gn(x, None, None, 32, 0.0)
    g1 = run_gn(x, None, None, 32, 1e-5)
    g0 = run_gn(x, None, None, 32, 0.0)
    assert np.abs(g0).max() > 2 * np.abs(g1).max()


def test_group_norm_in_place_and_bf16():
    x, gamma, beta = wl.make_norm(2, 320, 1024, 8200)
    check_gn(x, gamma, beta, 32, 1e-5, in_place=True)
    xb, gb, bb = wl.make_norm(2, 320, 1024, 8201, dtype="bf16")
    check_gn(xb, gb, bb, 32, 1e-5, dtype="bf16")
    x2, g2, b2 = wl.make_norm(1, 64, 4096, 8202)
    check_gn(x2, g2, b2, 2, 1e-5, in_place=True)   # three-read kernel in place


def geglu_bound(h64, r, dtype):
    F = h64.shape[-1] // 2
    a, gt = h64[..., :F], h64[..., F:]
    gl = oracle.gelu(gt)
    return np.abs(a) * (0.5 * np.abs(gt) * 3e-7 + 2.0 ** -21 * np.abs(gl)) + ulp(r, dtype)


def run_geglu(h, dtype="f16"):
    import torch
    hd = to_device(h, dtype)
    out = torch.empty(hd.shape[:-1] + (hd.shape[-1] // 2,), dtype=hd.dtype, device="cuda")
    sd.geglu(hd, out)
    torch.cuda.synchronize()
    return to_host64(out)


@pytest.mark.parametrize("name", list(wl.GEGLU_CASES))
def test_geglu_unet_levels(name):
    case = wl.GEGLU_CASES[name]
    h = wl.geglu_inputs(case)
    g = run_geglu(h)
    r = oracle.geglu(h)
    assert np.all(np.abs(g - r) <= geglu_bound(h.astype(np.float64), r, "f16"))


def test_geglu_edges_and_bf16():
    # gate values across the whole fp16 range that matters: deep negative tails
    # (GELU -> -0), zero, the erf knee, large positive (GELU -> x)
    F = 64
    gates = np.concatenate([np.linspace(-12, 12, F - 8), [0.0, -0.0, 30.0, -30.0, 1e-4, -1e-4, 40000.0, -40000.0]])
    h = np.concatenate([np.full((3, F), 1.5), np.tile(gates, (3, 1))], axis=1).astype(np.float16)
    g = run_geglu(h)
    r = oracle.geglu(h)
    assert np.all(np.abs(g - r) <= geglu_bound(h.astype(np.float64), r, "f16"))
    hb = wl.make_geglu(100, 320, 8300, dtype="bf16")
    gb = run_geglu(hb, "bf16")
    rb = oracle.geglu(hb, dtype="bf16")
    assert np.all(np.abs(gb - rb) <= geglu_bound(oracle.widen(hb, dtype="bf16"), rb, "bf16"))
    # ragged row count and one row
    for M in (1, 3, 777):
        h3 = wl.make_geglu(M, 40, 8400 + M)
        assert np.all(np.abs(run_geglu(h3) - oracle.geglu(h3)) <= geglu_bound(h3.astype(np.float64), oracle.geglu(h3), "f16"))
