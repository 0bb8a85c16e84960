"""Helpers shared by the GPU parity tests: device transfer and the tolerance.

Tolerance for fp16 in / fp32 accumulate (applied per call, r = fp64 oracle):
    abs:  |g - r| <= max(2e-3, ulp(r))      for every element
    rel:  |g - r| / max(|r|, rms(r)) <= 1e-2
with rms over the whole output of that call.  A bare |r| denominator would be
meaningless: outputs average many N(0,1) values and some sit near zero.

ulp(r) is the spacing of the output format at |r|.  The output is stored in
fp16, whose spacing at |r| >= 4 is 3.9e-3: there even the exact result,
rounded to fp16, can be 1.95e-3 away, so a flat 2e-3 would demand correct
rounding of a value computed in fp32.  Below |r| = 4 the bound is exactly
2e-3.  bfloat16 keeps 8 significant bits instead of 11: its bounds are 1e-2
(or one bf16 ulp) and 3e-2.
"""
import numpy as np

TOL = {"f16": (2e-3, 1e-2), "bf16": (1e-2, 3e-2)}


def torch_mod():
    import torch
    return torch


def to_device(arr, dtype="f16"):
    torch = torch_mod()
    if dtype == "bf16":
        t = torch.from_numpy(np.ascontiguousarray(arr).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(arr))
    return t.cuda()


def empty_like_out(q_dev):
    return q_dev.new_empty(q_dev.shape)


def to_host64(t):
    return t.float().cpu().numpy().astype(np.float64)


def ulp(r, dtype="f16"):
    """Spacing of the fp16 / bf16 grid at |r| (normal range)."""
    mant = 10 if dtype == "f16" else 7
    a = np.maximum(np.abs(np.asarray(r, dtype=np.float64)), 2.0 ** -14)
    return 2.0 ** (np.floor(np.log2(a)) - mant)


def errors(g, r):
    g = np.asarray(g, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    diff = np.abs(g - r)
    rms = float(np.sqrt(np.mean(r * r)))
    denom = np.maximum(np.abs(r), rms)
    return float(diff.max()), float((diff / denom).max()), float(np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-300))


def assert_close(g, r, dtype="f16", what=""):
    atol, rtol = TOL[dtype]
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    max_abs, max_rel, l2 = errors(g, r)
    bound = np.maximum(atol, ulp(r, dtype))
    excess = float((np.abs(np.asarray(g, np.float64) - r) / bound).max())
    assert excess <= 1.0 and max_rel <= rtol, (
        f"{what}: max_abs={max_abs:.3e} (bound max({atol}, ulp), worst ratio {excess:.3f}) "
        f"max_rel={max_rel:.3e} (<= {rtol}) l2={l2:.3e}")
    return max_abs, max_rel, l2
