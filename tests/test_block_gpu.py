"""GPU parity of the projections around Eq. 3 (sdattn_linear, with the head
split / merge layouts) and of SD's attention block (sdattn_attention_block)
against the fp64 oracle on seeded inputs.

Bounds derived from the arithmetic:
* linear: fp16/bf16 products are exact in fp32 and summed in fp32, so
  |g - r| <= (K + 2) 2^-22 sum_k |x_k w_nk| plus half an output ulp;
* block: the GPU stores Q, K, V and O in the input type between the five
  launches, so the reference is the oracle's steps with the same roundings
  (oracle.linear -> fp16 -> oracle.attention -> fp16 -> oracle.linear) at the
  forward tolerance; the fp64 block without those roundings is checked at the
  propagated size of one input-type rounding.
"""
import numpy as np
import pytest

import oracle
import paper_2304_11267_amd as sd
from paper_2304_11267_amd import workloads as wl

from parity_util import TOL, assert_close, to_device, to_host64, ulp

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _needs_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    sd.load_library()


def heads_of(t, H):
    """[B, L, C] -> [B, H, L, C/H] (numpy layout change only)."""
    B, L, C = t.shape
    return np.ascontiguousarray(t.reshape(B, L, H, C // H).transpose(0, 2, 1, 3))


def rows_of(t):
    """[B, H, L, D] -> [B, L, H*D]."""
    B, H, L, D = t.shape
    return np.ascontiguousarray(t.transpose(0, 2, 1, 3).reshape(B, L, H * D))


def lin_bound(xa, wa, r, dtype="f16"):
    """fp32 accumulation error of the K-term dot products plus one output ulp
    (half an ulp for the rounding, doubled in case it lands in the next binade)."""
    K = wa.shape[1]
    return (K + 2) * 2.0 ** -22 * (np.abs(xa) @ np.abs(wa).T) + ulp(r, dtype)


LIN_SHAPES = [
    # (B, L, K, N, H): ragged token tiles, channel tails of the 64-wide loop, N past 64-multiples
    (2, 100, 320, 320, 8),
    (1, 300, 768, 320, 8),
    (2, 77, 768, 640, 8),
    (1, 129, 40, 1280, 8),
    (1, 33, 1280, 1280, 8),
    (3, 10, 24, 16, 2),
    # one 64-channel slice with sequences shorter than a 32-row store pass,
    # three slices with head widths 48 / 40, the 64x64 level's 8192 token rows,
    # and Q, K and V's 960 outputs in one product
    (3, 10, 64, 80, 2),
    (2, 300, 192, 160, 4),
    (2, 4096, 320, 320, 8),
    (1, 1000, 320, 960, 8),
]


@pytest.mark.parametrize("shape", LIN_SHAPES, ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("mode", ["rows_rows_bias", "rows_heads", "heads_rows_bias"])
def test_linear_matches_oracle(shape, mode):
    import torch
    B, L, K, N, H = shape
    rng = np.random.default_rng(7000 + B + L + K + N)
    x = rng.standard_normal((B, L, K), dtype=np.float32).astype(np.float16)
    w = (rng.standard_normal((N, K), dtype=np.float32) / np.float32(np.sqrt(K))).astype(np.float16)
    bias = (rng.standard_normal(N, dtype=np.float32) * np.float32(0.5)).astype(np.float16)
    use_bias = mode.endswith("bias")
    x_heads = mode.startswith("heads")
    y_heads = mode == "rows_heads"
    xd = to_device(heads_of(x, H) if x_heads else x)
    wd, bd = to_device(w), to_device(bias)
    y = torch.empty((B, H, L, N // H) if y_heads else (B, L, N), dtype=torch.float16, device="cuda")
    if (x_heads and (K % H or (K // H) % 8)) or (y_heads and (N % H or (N // H) % 8)):
        # a head width that is not a multiple of 8 is refused before any launch,
        # and y is left as it was
        y.fill_(7.0)
        with pytest.raises(sd.SdattnError) as e:
            sd.linear(xd, wd, y, bias=bd if use_bias else None, heads=H,
                      x_layout=sd.LAYOUT_HEADS if x_heads else sd.LAYOUT_ROWS,
                      y_layout=sd.LAYOUT_HEADS if y_heads else sd.LAYOUT_ROWS)
        assert e.value.status == sd.STATUS_UNSUPPORTED
        torch.cuda.synchronize()
        assert bool((y == 7.0).all())
        return
    sd.linear(xd, wd, y, bias=bd if use_bias else None, heads=H,
              x_layout=sd.LAYOUT_HEADS if x_heads else sd.LAYOUT_ROWS,
              y_layout=sd.LAYOUT_HEADS if y_heads else sd.LAYOUT_ROWS)
    torch.cuda.synchronize()
    g = to_host64(y)
    g = rows_of(g) if y_heads else g
    r = oracle.linear(x, w, bias if use_bias else None)
    bound = lin_bound(x.astype(np.float64), w.astype(np.float64), r)
    assert np.all(np.abs(g - r) <= bound), float(np.max(np.abs(g - r) / bound))


def test_linear_bf16():
    import torch
    rng = np.random.default_rng(7100)
    x = wl.to_bf16_bits(rng.standard_normal((2, 70, 320), dtype=np.float32))
    w = wl.to_bf16_bits(rng.standard_normal((640, 320), dtype=np.float32) / np.float32(18.0))
    y = torch.empty(2, 70, 640, dtype=torch.bfloat16, device="cuda")
    sd.linear(to_device(x, "bf16"), to_device(w, "bf16"), y)
    torch.cuda.synchronize()
    r = oracle.linear(x, w, dtype="bf16")
    bound = lin_bound(oracle.widen(x, dtype="bf16"), oracle.widen(w, dtype="bf16"), r, "bf16")
    assert np.all(np.abs(to_host64(y) - r) <= bound)


def gpu_block(inputs, H, scale):
    import torch
    x, ctx, wq, wk, wv, wo, bo = (to_device(t) for t in inputs)
    B, Lq, C = inputs[0].shape
    Lk = inputs[1].shape[1]
    ws = torch.empty(sd.attention_block_workspace(B, Lq, Lk, C), dtype=torch.uint8, device="cuda")
    out = torch.empty(B, Lq, C, dtype=torch.float16, device="cuda")
    sd.attention_block(x, ctx, wq, wk, wv, wo, bo, out, ws, H, scale)
    torch.cuda.synchronize()
    return to_host64(out)


def rounded_chain(inputs, H, scale, rows=None):
    """The block's steps in the oracle with Q, K, V, O stored in fp16 between them."""
    x, ctx, wq, wk, wv, wo, bo = inputs
    q = heads_of(oracle.linear(x, wq).astype(np.float16), H)
    k = heads_of(oracle.linear(ctx, wk).astype(np.float16), H)
    v = heads_of(oracle.linear(ctx, wv).astype(np.float16), H)
    if rows is None:
        o, _, _ = oracle.attention(q, k, v, scale)
        return oracle.linear(rows_of(o.astype(np.float16)), wo, bo)
    # selected token rows r = b*Lq + i: every head's output row, then the projection
    B, _, Lq, D = q.shape
    b, i = rows // Lq, rows % Lq
    flat = ((b[:, None] * H + np.arange(H)[None, :]) * Lq + i[:, None]).reshape(-1)
    o, _, _ = oracle.attention(q, k, v, scale, rows=flat)
    o16 = o.astype(np.float16).reshape(len(rows), H * D)
    return oracle.linear(o16, wo, bo)


# (B, Lq, Lk, C, Cc, H, self): short-key kernel (Lk = 77, 64), tiled kernel (Lk = 200),
# the general kernel (head width 16 with 150 keys; 256 with 120 keys)
@pytest.mark.parametrize("shape", [(2, 37, 77, 320, 768, 8, False), (1, 200, 200, 320, 320, 8, True),
                                   (2, 64, 64, 1280, 1280, 8, True), (1, 130, 77, 640, 768, 8, False),
                                   (1, 150, 150, 128, 128, 8, True), (1, 100, 120, 2048, 2048, 8, True)],
                         ids=lambda s: "x".join(map(str, s)))
def test_block_small_full(shape):
    B, Lq, Lk, C, Cc, H, self_attn = shape
    inputs = wl.make_block(B, Lq, Lk, C, Cc, 7200 + Lq + C, self_attn)
    scale = float(np.float32(1 / np.sqrt(C // H)))
    g = gpu_block(inputs, H, scale)
    assert_close(g, rounded_chain(inputs, H, scale), what=f"{shape} rounded chain")
    # against the fp64 block: one fp16 rounding of Q/K/V/O moves the output by
    # at most a few 2^-11 of its size; allow 1 % of the output's rms plus 2e-3
    r64 = oracle.attention_block(*inputs, H, scale)
    rms = float(np.sqrt(np.mean(r64 * r64)))
    assert np.max(np.abs(g - r64)) <= 2e-3 + 1e-2 * rms


@pytest.mark.parametrize("name,per_b", [("blk64_self", 24), ("blk64_cross", 64), ("blk32_self", 48),
                                        ("blk16_cross", 128)])
def test_block_unet_sampled_rows(name, per_b):
    case = wl.BLOCK_CASES[name]
    inputs = wl.block_inputs(case)
    g = gpu_block(inputs, case.H, case.scale).reshape(-1, case.C)
    rng = np.random.default_rng(case.seed + 5)
    rows = np.sort(np.concatenate([b * case.Lq + rng.choice(case.Lq, size=per_b, replace=False)
                                   for b in range(case.B)]))
    assert_close(g[rows], rounded_chain(inputs, case.H, case.scale, rows=rows), what=name)


@pytest.mark.parametrize("name", ["blk64_cross", "blk16_cross"])
def test_cached_context_block(name):
    """K and V of the text context computed once (project_kv), then the per-step
    block with them: K and V match the oracle's projections, the output matches
    the oracle chain, and both equal the one-call block bit for bit."""
    import torch
    case = wl.BLOCK_CASES[name]
    inputs = wl.block_inputs(case)
    x, ctx, wq, wk, wv, wo, bo = (to_device(t) for t in inputs)
    D = case.C // case.H
    k = torch.empty(case.B, case.H, case.Lk, D, dtype=torch.float16, device="cuda")
    v = torch.empty_like(k)
    sd.project_kv(ctx, wk, wv, k, v, case.H)
    ws = torch.empty(sd.attention_block_workspace(case.B, case.Lq, 0, case.C), dtype=torch.uint8,
                     device="cuda")
    out = torch.empty(case.B, case.Lq, case.C, dtype=torch.float16, device="cuda")
    sd.attention_block_kv(x, wq, k, v, wo, bo, out, ws, case.scale)
    torch.cuda.synchronize()
    for t, w in ((k, inputs[3]), (v, inputs[4])):
        r = oracle.linear(inputs[1], w)
        bound = lin_bound(inputs[1].astype(np.float64), w.astype(np.float64), r)
        assert np.all(np.abs(rows_of(to_host64(t)) - r) <= bound)
    g = to_host64(out).reshape(-1, case.C)
    rng = np.random.default_rng(case.seed + 9)
    rows = np.sort(np.concatenate([b * case.Lq + rng.choice(case.Lq, size=64, replace=False)
                                   for b in range(case.B)]))
    assert_close(g[rows], rounded_chain(inputs, case.H, case.scale, rows=rows), what=name)
    full = gpu_block(inputs, case.H, case.scale).reshape(-1, case.C)
    assert np.array_equal(full, g)
