"""Helpers shared by the GPU parity tests: device transfer and the tolerance.

Tolerance for fp16 in / fp32 accumulate (applied per call, r = fp64 oracle):

    abs:  |g - r| <= max(2e-3, ulp(g, r) / 2 + 2^-11 (1 + 2^-3) dev + 2^-16 (dev + |r|))
    rel:  |g - r| / max(|r|, rms(r)) <= 1e-2

with rms over the whole output of that call.  A bare |r| denominator would be
meaningless: outputs average many N(0,1) values and some sit near zero.

The absolute bound is the flat 2e-3 wherever an fp16 result can meet it.  It
grows only where the arithmetic the precision reading fixes cannot: the GPU
rounds every weight p to fp16 before the P V product (relative error 2^-11,
with an eighth more for the fp32 exponent argument), and then rounds O to
fp16 (half a spacing of the output grid, ulp(max(|g|, |r|)) / 2 -- 1.95e-3
at |r| >= 4).  dev is the oracle's dev_id = sum_j p_ij |v_jd - o_id|: a
relative rounding e of every weight moves o_id by at most e dev_id (pinned in
the oracle's tests).  The last term covers fp32 accumulation: each MFMA
adds 16 keys' products to an fp32 accumulator, so n keys take n / 16 steps
that may each lose half an ulp of it -- 2^-16 relative for the 4096 keys of
the UNet's longest sequences, n 2^-28 beyond (tests of longer sequences pass
n_keys).  Without dev (a reference that is not a softmax of the oracle), the
bound is max(2e-3, ulp / 2).

bfloat16 keeps 8 significant bits instead of 11: its bounds are
max(1e-2, ulp / 2 + 2^-8 (1 + 2^-3) dev + 2^-16 (dev + |r|)) and 3e-2.

Every call records max |g - r|, the number of elements above the flat 2e-3
(1e-2 for bf16) and the worst ratio to the bound; with SDATTN_PARITY_REPORT
set, the test session writes them to that file as JSON lines.
"""
import json
import os

import numpy as np

TOL = {"f16": (2e-3, 1e-2), "bf16": (1e-2, 3e-2)}
P_ROUND = {"f16": 2.0 ** -11, "bf16": 2.0 ** -8}   # relative rounding of a weight p
RECORDS = []


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


def accumulation_allowance(n_keys=None):
    """Relative fp32 accumulation error for n_keys keys (16 per MFMA step)."""
    return 2.0 ** -16 if n_keys is None else max(2.0 ** -16, n_keys * 2.0 ** -28)


def abs_bound(g, r, dtype="f16", dev=None, n_keys=None):
    """Per-element absolute bound (see the module docstring)."""
    atol = TOL[dtype][0]
    g = np.asarray(g, dtype=np.float64)
    r = np.asarray(r, dtype=np.float64)
    half_ulp = ulp(np.maximum(np.abs(g), np.abs(r)), dtype) / 2
    if dev is None:
        return np.maximum(atol, half_ulp)
    dev = np.asarray(dev, dtype=np.float64)
    return np.maximum(atol, half_ulp + P_ROUND[dtype] * (1 + 2.0 ** -3) * dev
                      + accumulation_allowance(n_keys) * (dev + np.abs(r)))


def assert_close(g, r, dtype="f16", what="", dev=None, n_keys=None):
    atol, rtol = TOL[dtype]
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    max_abs, max_rel, l2 = errors(g, r)
    diff = np.abs(np.asarray(g, np.float64) - np.asarray(r, np.float64))
    bound = abs_bound(g, r, dtype, dev, n_keys)
    ratio = diff / bound
    worst = int(np.argmax(ratio))
    over = diff > atol
    rec = {"what": what, "dtype": dtype, "n": int(diff.size), "max_abs": max_abs,
           "over_flat": int(over.sum()), "max_rel": max_rel, "l2": l2,
           "worst_ratio": float(ratio.flat[worst]),
           "abs_r_at_worst": float(abs(np.asarray(r, np.float64).flat[worst])),
           "min_abs_r_over_flat": float(np.abs(np.asarray(r, np.float64))[over].min()) if over.any() else None}
    RECORDS.append(rec)
    assert rec["worst_ratio"] <= 1.0 and max_rel <= rtol, (
        f"{what}: max_abs={max_abs:.3e} ({rec['over_flat']} of {rec['n']} above {atol}; worst "
        f"ratio to the bound {rec['worst_ratio']:.3f} at |r|={rec['abs_r_at_worst']:.3f}) "
        f"max_rel={max_rel:.3e} (<= {rtol}) l2={l2:.3e}")
    return max_abs, max_rel, l2


def write_report():
    path = os.environ.get("SDATTN_PARITY_REPORT")
    if path and RECORDS:
        os.makedirs(os.path.dirname(os.path.abspath(path)), exist_ok=True)
        with open(path, "a") as f:
            for rec in RECORDS:
                f.write(json.dumps(rec) + "\n")
        RECORDS.clear()
