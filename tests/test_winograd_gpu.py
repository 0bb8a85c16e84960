"""GPU parity of the Winograd F(4x4, 3x3) convolution (Sec. 3.3) against the
oracle's direct fp64 convolution.

Error bound derived from the arithmetic (the transforms here are re-derived
from the interpolation points 0, 1, -1, 1/2, -2 and infinity, independently of
the kernels' tables, and used only to size the bound):
  U = G g G^T and V = B^T d B are rounded to the input type (relative error
  u = 2^-11 for fp16, 2^-8 for bf16) and multiplied and summed over Ci in
  fp32 ((Ci + 2) 2^-24 relative to the sum of magnitudes); the sum M is
  rounded again (u |M|); the output transform (fp32) and the final rounding
  add 2^-22 sum |A^T M A| and one output ulp.  Per output pixel p of tile t
  and channel o:
    |y - r| <= sum_xi |A_xi,p| [ S_xi (2u + (Ci + 2) 2^-24) + u |M_xi| ] + ...
  with S_xi = sum_c |U_xi,o,c| |V_xi,t,c|.
A second, tighter check models each rounding as an independent relative
error uniform in [-u, u]: the output's standard deviation is
  sigma^2 = sum_xi A_xi,p^2 (2 sum_c (U V)^2 + M_xi^2) u^2 / 3,
and every output must lie within 7 sigma + one ulp of the oracle.
"""
import numpy as np
import pytest

import oracle
import paper_2304_11267_amd as sd

from parity_util import to_device, to_host64, ulp

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _needs_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    sd.load_library()


def transforms():
    """A^T (4x6), G (6x3), B^T (6x6) of F(4, 3) from Lagrange interpolation at
    0, 1, -1, 1/2, -2 and the point at infinity; B^T solved from the 1-D identity."""
    p = [0, 1, -1, 0.5, -2]
    m, r, n = 4, 3, 6
    AT, G = np.zeros((m, n)), np.zeros((n, r))
    for i, pi in enumerate(p):
        AT[:, i] = [pi ** k for k in range(m)]
        N = np.prod([pi - pl for l, pl in enumerate(p) if l != i])
        G[i] = [pi ** j / N for j in range(r)]
    AT[m - 1, n - 1] = 1
    G[n - 1, r - 1] = 1
    rows, rhs = [], []
    for k in range(m):
        for t in range(r):
            for s in range(n):
                c = np.zeros((n, n))
                c[:, s] = AT[k] * G[:, t]
                rows.append(c.ravel())
                rhs.append(1.0 if s == k + t else 0.0)
    BT = np.linalg.lstsq(np.array(rows), np.array(rhs), rcond=None)[0].reshape(n, n)
    return AT, G, np.round(BT, 12)


def winograd_bound(x64, w64, r, dtype):
    AT, G, BT = transforms()
    u = 2.0 ** -11 if dtype == "f16" else 2.0 ** -8
    B, Ci, H, W = x64.shape
    Co = w64.shape[0]
    th, tw = (H + 3) // 4, (W + 3) // 4
    xp = np.zeros((B, Ci, 4 * th + 2, 4 * tw + 2))
    xp[:, :, 1:H + 1, 1:W + 1] = x64
    # patches [B, th, tw, Ci, 6, 6]
    idx_r = 4 * np.arange(th)[:, None] + np.arange(6)[None, :]
    idx_c = 4 * np.arange(tw)[:, None] + np.arange(6)[None, :]
    d = xp[:, :, idx_r[:, None, :, None], idx_c[None, :, None, :]]          # [B, Ci, th, tw, 6, 6]
    V = np.einsum("ik,bcyxkl,jl->bcyxij", BT, d, BT).reshape(B, Ci, th * tw, 36)
    U = np.einsum("ik,ockl,jl->ocij", G, w64, G).reshape(Co, Ci, 36)
    Vt = V.transpose(3, 0, 2, 1).reshape(36, B * th * tw, Ci)               # [xi, T, Ci]
    Ut = U.transpose(2, 1, 0)                                               # [xi, Ci, Co]
    S = np.abs(Vt) @ np.abs(Ut)                                             # [xi, T, Co]
    M = Vt @ Ut
    dM = S * (2 * u + (Ci + 2) * 2.0 ** -24) + u * np.abs(M)
    A2 = np.abs(np.einsum("pi,qj->pqij", AT, AT)).reshape(16, 36)           # |A_xi,p|
    dY = np.einsum("xto,px->top", dM, A2) + 2.0 ** -22 * np.einsum("xto,px->top", np.abs(M), A2)
    # rounding-error model: each stored U, V and M value carries an independent
    # relative error uniform in [-u, u] (variance u^2 / 3)
    S2 = (Vt * Vt) @ (Ut * Ut)
    var = np.einsum("xto,px->top", (2 * S2 + M * M) * (u * u / 3), A2 * A2)
    tile = lambda a: a.reshape(B, th, tw, Co, 4, 4).transpose(0, 3, 1, 4, 2, 5).reshape(
        B, Co, 4 * th, 4 * tw)[:, :, :H, :W]
    return tile(dY) + ulp(r, dtype), tile(np.sqrt(var))


def run_conv(x, w, bias, dtype="f16"):
    import torch
    xd, wd = to_device(x, dtype), to_device(w, dtype)
    bd = to_device(bias, dtype) if bias is not None else None
    B, Ci, H, W = x.shape
    Co = w.shape[0]
    u = torch.empty(36, Co, Ci, dtype=xd.dtype, device="cuda")
    sd.winograd_weights(wd, u)
    ws = torch.empty(sd.conv3x3_workspace(B, Ci, Co, H, W), dtype=torch.uint8, device="cuda")
    y = torch.empty(B, Co, H, W, dtype=xd.dtype, device="cuda")
    sd.conv3x3(xd, u, y, ws, bd)
    torch.cuda.synchronize()
    return to_host64(y)


def make(B, Ci, Co, H, W, seed, dtype="f16"):
    from paper_2304_11267_amd import workloads as wl
    return wl.make_conv(B, Ci, Co, H, W, seed, dtype)


def check(x, w, bias, dtype="f16", co=None):
    g = run_conv(x, w, bias, dtype)
    ws = w if co is None else w[co]
    bs = None if bias is None else (bias if co is None else bias[co])
    odt = "bf16" if dtype == "bf16" else None
    r = oracle.conv3x3(x, ws, bs, dtype=odt)
    wid = lambda t: oracle.widen(t, dtype=odt)
    bound, sigma = winograd_bound(wid(x), wid(ws), r, dtype)
    gg = g if co is None else g[:, co]
    assert np.all(np.isfinite(gg))
    err = np.abs(gg - r)
    # the worst case, every rounding adding up
    excess = err / bound
    assert excess.max() <= 1.0, (float(excess.max()), float(err.max()))
    # and the statistical size: 7 standard deviations of the rounding model
    # (a Gaussian exceeds that with probability 3e-12 per output) plus one ulp
    z = err / (7 * sigma + ulp(r, dtype))
    assert z.max() <= 1.0, (float(z.max()), float(err.max()))
    return float(err.max())


@pytest.mark.parametrize("shape", [
    (1, 8, 16, 8, 8),        # one segment, whole tiles
    (2, 16, 8, 13, 10),      # ragged tiles at the bottom and right, W % 4 != 0
    (1, 32, 24, 5, 100),     # several 16-tile segments, partial last one
    (3, 8, 8, 4, 4),         # one tile per image
    (1, 40, 48, 1, 7),       # one row
    (2, 64, 64, 20, 36),     # channel blocks of 32, W % 4 == 0
], ids=lambda s: "x".join(map(str, s)))
def test_conv3x3_small(shape):
    B, Ci, Co, H, W = shape
    x, w, b = make(B, Ci, Co, H, W, 9000 + Ci + H + W)
    check(x, w, b)


def test_conv3x3_without_bias_and_bf16():
    x, w, b = make(1, 16, 32, 12, 12, 9100)
    check(x, w, None)
    xb, wb, bb = make(1, 16, 32, 12, 12, 9101, dtype="bf16")
    check(xb, wb, bb, dtype="bf16")


@pytest.mark.parametrize("level", [(320, 64), (640, 32), (1280, 16), (1280, 8)])
def test_conv3x3_unet_levels_sampled_channels(level):
    C, L = level
    x, w, b = make(2, C, C, L, L, 9200 + C + L)
    co = np.sort(np.random.default_rng(C + L).choice(C, size=8, replace=False))
    check(x, w, b, co=co)
