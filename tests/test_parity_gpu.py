"""GPU parity of the HIP attention path against the fp64 oracle.

Every call goes through the C ABI (libsdattn.so) via the thin binding; the
reference is the oracle on the same seeded inputs.  Sizes span several
128-row query tiles and 64-key tiles with ragged tails; the UNet shapes run
at full size (sampled rows where the oracle would be slow), in the launch
configuration the benchmark times.
"""
import numpy as np
import pytest

import oracle
import paper_2304_11267_amd as sd
from paper_2304_11267_amd import workloads as wl

from parity_util import accumulation_allowance, assert_close, to_device, to_host64

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _needs_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    sd.load_library()


def run_forward(q, k, v, scale, dtype="f16", want_ls=False):
    import torch
    qd, kd, vd = (to_device(t, dtype) for t in (q, k, v))
    out = torch.empty_like(qd)
    ls = None
    if want_ls:
        ls = torch.empty(qd.shape[:3] + (2,), dtype=torch.float32, device=qd.device)
    if dtype == "f16" and not want_ls:
        sd.forward(qd, kd, vd, out, scale)
    else:
        sd.forward_ex(qd, kd, vd, out, scale, ls=ls)
    torch.cuda.synchronize()
    o = to_host64(out)
    return (o, ls.cpu().numpy().astype(np.float64)) if want_ls else o


def check_case(q, k, v, scale, dtype="f16", rows=None, what="", literal=False):
    """Both launches against the oracle: the plain one (the configuration the
    benchmark times) and the one that also returns Eq. 4's statistics.
    literal: also hold fp16 results to the flat max-abs 2e-3 / max-rel 1e-2
    stated for the UNet configurations, without the rounding allowance."""
    g_plain = run_forward(q, k, v, scale, dtype)
    g, ls = run_forward(q, k, v, scale, dtype, want_ls=True)
    r, L, S, dev = oracle.attention(q, k, v, scale, rows=rows, dtype="bf16" if dtype == "bf16" else None,
                                    want_dev=True)
    D = q.shape[3]
    if rows is not None:
        g = g.reshape(-1, D)[rows]
        g_plain = g_plain.reshape(-1, D)[rows]
        ls = ls.reshape(-1, 2)[rows]
    else:
        ls = ls.reshape(L.shape + (2,))
    for out, tag in ((g_plain, " (plain)"), (g, " (with statistics)")):
        max_abs, max_rel, _ = assert_close(out, r, dtype, what + tag, dev=dev)
        if literal and dtype == "f16":
            assert max_abs <= 2e-3 and max_rel <= 1e-2, f"{what}{tag}: {max_abs:.3e} / {max_rel:.3e}"
    # Eq. 4's statistics: L to fp32 rounding of the logits, S to the rounding of p
    assert np.max(np.abs(ls[..., 0] - L) / np.maximum(1.0, np.abs(L))) <= 1e-5, what
    srel = 2e-3 if dtype == "f16" else 1e-2
    assert np.max(np.abs(ls[..., 1] - S) / S) <= srel, what


@pytest.mark.parametrize("name", ["mid8_self", "mid8_cross", "l16_self", "l16_self_peaked",
                                  "l16_cross", "l32_cross", "l64_cross"])
def test_unet_case_full(name):
    case = wl.CASES[name]
    q, k, v = wl.case_inputs(case)
    check_case(q, k, v, case.scale, what=name, literal=True)


@pytest.mark.parametrize("name,per_head", [("l32_self", 96), ("l64_self", 48)])
def test_unet_case_sampled_rows(name, per_head):
    case = wl.CASES[name]
    q, k, v = wl.case_inputs(case)
    rows = wl.sample_rows(case.B, case.H, case.Lq, per_head, seed=case.seed + 5)
    check_case(q, k, v, case.scale, rows=rows, what=name, literal=True)


@pytest.mark.parametrize("name", ["mid8_self", "l16_self_peaked", "l32_cross"])
def test_unet_case_bf16(name):
    case = wl.CASES[name]
    q, k, v = wl.case_inputs(case, dtype="bf16")
    check_case(q, k, v, case.scale, dtype="bf16", what=name + "/bf16")


@pytest.mark.parametrize("name,per_head", [("l32_self", 48), ("l64_self", 24)])
def test_unet_case_bf16_sampled_rows(name, per_head):
    """The 32x32 self-attention (64-row workgroups, keys split four ways) and
    the 64x64 one (256-row workgroups, 128-key tiles) in bf16."""
    case = wl.CASES[name]
    q, k, v = wl.case_inputs(case, dtype="bf16")
    rows = wl.sample_rows(case.B, case.H, case.Lq, per_head, seed=case.seed + 7)
    check_case(q, k, v, case.scale, dtype="bf16", rows=rows, what=name + "/bf16")


RAGGED = [
    # (B, H, Lq, Lk, D)
    (1, 1, 1, 1, 40),
    (1, 2, 5, 3, 8),
    (2, 1, 100, 65, 16),
    (1, 3, 129, 63, 24),
    (2, 2, 130, 129, 32),
    (1, 1, 257, 200, 48),
    (1, 2, 64, 77, 64),
    (2, 1, 200, 300, 80),
    (1, 1, 131, 127, 96),
    (1, 1, 70, 191, 128),
    (1, 1, 33, 77, 160),
    (1, 1, 40, 70, 200),
    (1, 1, 40, 65, 256),
]


@pytest.mark.parametrize("shape", RAGGED, ids=lambda s: "x".join(map(str, s)))
def test_ragged_shapes(shape):
    B, H, Lq, Lk, D = shape
    seed = 77 + Lq * 3 + Lk * 5 + D
    q, k, v = wl.make_qkv(B, H, Lq, Lk, D, seed)
    check_case(q, k, v, float(np.float32(1 / np.sqrt(D))), what=str(shape))


# Short key sequences (the text context, Lk <= 128): every count of 32-key
# sub-tiles, Lk on, just past and just short of each 16- and 32-key boundary,
# and Lq = 97 so a workgroup holds one full 32-row strip, one partial strip
# and two strips wholly past Lq.
SHORT_LK = [1, 2, 15, 16, 17, 31, 32, 33, 48, 49, 63, 64, 65, 77, 80, 95, 96, 97, 112, 113,
            127, 128]
SHORT_D = [32, 40, 56, 80, 96, 160]


@pytest.mark.parametrize("D", SHORT_D)
@pytest.mark.parametrize("Lk", SHORT_LK)
def test_short_key_sequences(Lk, D):
    q, k, v = wl.make_qkv(1, 2, 97, Lk, D, 3000 + 7 * Lk + D)
    check_case(q, k, v, float(np.float32(1 / np.sqrt(D))), what=f"Lk={Lk} D={D}")


@pytest.mark.parametrize("Lk,D", [(33, 40), (77, 80), (128, 160), (49, 96)])
def test_short_key_sequences_bf16(Lk, D):
    q, k, v = wl.make_qkv(2, 1, 161, Lk, D, 3500 + Lk + D, dtype="bf16")
    check_case(q, k, v, float(np.float32(1 / np.sqrt(D))), dtype="bf16", what=f"Lk={Lk} D={D}")


@pytest.mark.parametrize("Lk,D", [(77, 40), (77, 160), (20, 80)])
def test_statistics_output_does_not_change_o(Lk, D):
    q, k, v = wl.make_qkv(2, 2, 300, Lk, D, 3600 + Lk + D)
    scale = float(np.float32(1 / np.sqrt(D)))
    o_plain = run_forward(q, k, v, scale)
    o_stats, _ = run_forward(q, k, v, scale, want_ls=True)
    assert np.array_equal(o_plain, o_stats)


# Grids of at least 256 workgroups of 256 query rows take the largest
# geometry (eight waves, 128-key tiles) for D <= 64: a partial last query
# block, a ragged last key tile in either half, every head width it covers.
@pytest.mark.parametrize("Lk,D,dtype", [(1000, 40, "f16"), (1100, 32, "f16"), (900, 48, "f16"),
                                        (1000, 64, "f16"), (4095, 40, "f16"), (1000, 40, "bf16")])
def test_large_grid_ragged(Lk, D, dtype):
    q, k, v = wl.make_qkv(2, 8, 4000, Lk, D, 3700 + Lk + D, dtype=dtype)
    rows = wl.sample_rows(2, 8, 4000, 16, seed=Lk + D)
    rows = np.unique(np.concatenate([rows, [4000 * 16 - 1, 3999, 3840]]))
    check_case(q, k, v, float(np.float32(1 / np.sqrt(D))), dtype=dtype, rows=rows,
               what=f"Lq=4000 Lk={Lk} D={D} {dtype}")


@pytest.mark.parametrize("scale", [0.0, -0.2, 1.0])
def test_scale_values(scale):
    q, k, v = wl.make_qkv(1, 2, 70, 90, 40, 901)
    check_case(q, k, v, scale, what=f"scale={scale}")


@pytest.mark.parametrize("scale", [0.0, -0.2, 1.0])
@pytest.mark.parametrize("Lk,D", [(600, 80), (2100, 40)])
def test_scale_values_long_keys(scale, Lk, D):
    """Zero, negative and large scales through the tiled kernel's key loop
    (64 query rows with the keys split four ways)."""
    q, k, v = wl.make_qkv(1, 2, 100, Lk, D, 905 + Lk)
    check_case(q, k, v, scale, what=f"scale={scale} Lk={Lk} D={D}")


def test_constant_keys_give_mean_of_values():
    q, k, v = wl.make_qkv(1, 2, 130, 100, 40, 902)
    k[:] = k[:, :, :1]
    g = run_forward(q, k, v, 0.158)
    ref = np.broadcast_to(v.astype(np.float64).mean(axis=2, keepdims=True), g.shape)
    assert_close(g, ref, what="constant K")


def test_single_key_returns_value():
    q, k, v = wl.make_qkv(2, 2, 100, 1, 80, 903)
    g = run_forward(q, k, v, 0.11)
    assert np.array_equal(g, np.broadcast_to(v.astype(np.float64), g.shape))


def test_one_hot_dominant_logit():
    B, H, Lq, Lk, D = 1, 1, 64, 77, 40
    q = np.zeros((B, H, Lq, D), np.float16)
    k = (np.random.default_rng(904).standard_normal((B, H, Lk, D)) * 0.05).astype(np.float16)
    v = np.random.default_rng(905).standard_normal((B, H, Lk, D)).astype(np.float16)
    star = np.arange(Lq) % Lk
    # query i points at key star[i] through its own coordinate d = i % D
    for i in range(Lq):
        q[0, 0, i, i % D] = 8.0
    for j in range(Lk):
        k[0, 0, j, j % D] = 8.0
    # logits: 64*scale for the matching key(s) vs < 1 otherwise; several keys share i % D
    g = run_forward(q, k, v, 1.0)
    r, _, _, dev = oracle.attention(q, k, v, 1.0, want_dev=True)
    assert_close(g, r, what="one-hot", dev=dev)
    lone = [i for i in range(Lq) if sum(1 for j in range(Lk) if j % D == i % D) == 1]
    for i in lone:
        assert np.max(np.abs(g[0, 0, i] - v[0, 0, i % D].astype(np.float64))) <= 2e-3


def _long_keys_case(Lq, Lk, seed, planted):
    """q, k, v ~ N(0, 1) fp16 drawn on the GPU (torch's generator, seeded), with
    key j of each (row r, key j) in `planted` set to 4 q_r (exact in fp16):
    its logit, 4 |q_r|^2 / sqrt(D), stands far above the rest, so row r's
    output is led by v_j and a key read from the wrong place shows at once."""
    import torch
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    D = 40
    q = torch.randn(1, 1, Lq, D, dtype=torch.float16, device="cuda", generator=g)
    k = torch.randn(1, 1, Lk, D, dtype=torch.float16, device="cuda", generator=g)
    v = torch.randn(1, 1, Lk, D, dtype=torch.float16, device="cuda", generator=g)
    for r, j in planted:
        k[0, 0, j] = q[0, 0, r] * 4
    return q, k, v


def _check_long(q, k, v, rows, what):
    # fp32 accumulation over Lk keys: the allowance of the tolerance grows as
    # Lk 2^-28 past 4096 keys (parity_util)
    import torch
    scale = 1.0 / q.shape[3] ** 0.5
    out = torch.empty_like(q)
    sd.forward(q, k, v, out, scale)
    out2 = torch.empty_like(q)
    ls = torch.empty(q.shape[:3] + (2,), dtype=torch.float32, device="cuda")
    sd.forward_ex(q, k, v, out2, scale, ls=ls)
    torch.cuda.synchronize()
    qh, kh, vh = (t.cpu().numpy() for t in (q, k, v))
    r, L, S, dev = oracle.attention(qh, kh, vh, scale, rows=rows, want_dev=True)
    D = q.shape[3]
    Lk = k.shape[2]
    for o, tag in ((out, " (plain)"), (out2, " (with statistics)")):
        assert_close(to_host64(o).reshape(-1, D)[rows], r, what=what + tag, dev=dev, n_keys=Lk)
    lsr = ls.cpu().numpy().astype(np.float64).reshape(-1, 2)[rows]
    assert np.max(np.abs(lsr[:, 0] - L) / np.maximum(1.0, np.abs(L))) <= 1e-5
    assert np.max(np.abs(lsr[:, 1] - S) / S) <= 2e-3 + accumulation_allowance(Lk)


def test_a_million_keys_in_the_tiled_kernel():
    # 1 000 003 keys (a ragged last tile) through the tiled kernel's 64-row
    # workgroups; the planted keys sit in the last tile, mid-sequence and in
    # the first sub-tile, so rows 0 and 1 also take the exact fallback
    Lk = 1_000_003
    q, k, v = _long_keys_case(256, Lk, 9301, [(0, Lk - 1), (1, Lk // 2), (2, 5)])
    _check_long(q, k, v, np.array([0, 1, 2, 100, 255]), "1M keys")


def test_key_byte_offsets_past_32_bits():
    # 26 843 648 keys of D = 40: a head's K (and V) spans 2 147 491 840 bytes,
    # past what 32-bit offsets address, so the call takes the general kernel
    # (64-bit addressing).  Every key is zero (logit 0, value 0) except three
    # planted ones, one past the 2 GiB mark: then Eq. 3 reduces to a sum over
    # the planted keys plus (Lk - 3) e^-M in the denominator, evaluated here
    # in fp64.  Each planted key k_j = a_r q_r (rounded to fp16; the reference
    # takes the rounded values) has logit ln(Lk) + 14: it carries all but
    # e^-14 of its row's weight, so its row's output is its value row, read
    # from where it lies.
    import torch
    Lk, D, Lq = 26_843_648, 40, 64
    assert Lk * D * 2 > 2 ** 31
    scale = float(np.float32(1.0 / D ** 0.5))
    rng = np.random.default_rng(9302)
    q = rng.standard_normal((1, 1, Lq, D)).astype(np.float16)
    planted = [(0, Lk - 1), (1, 20_000_000), (2, 3)]
    kp, vp = [], []
    for r, j in planted:
        q64 = q[0, 0, r].astype(np.float64)
        a = (np.log(Lk) + 14.0) / (scale * (q64 @ q64))
        kp.append((q64 * a).astype(np.float16))
        vp.append(rng.standard_normal(D).astype(np.float16))
    qd = to_device(q)
    k = torch.zeros(1, 1, Lk, D, dtype=torch.float16, device="cuda")
    v = torch.zeros_like(k)
    for (r, j), kj, vj in zip(planted, kp, vp):
        k[0, 0, j] = torch.from_numpy(kj).cuda()
        v[0, 0, j] = torch.from_numpy(vj).cuda()
    out = torch.empty_like(qd)
    sd.forward(qd, k, v, out, scale)
    ls = torch.empty(1, 1, Lq, 2, dtype=torch.float32, device="cuda")
    out2 = torch.empty_like(qd)
    sd.forward_ex(qd, k, v, out2, scale, ls=ls)
    torch.cuda.synchronize()
    # Eq. 3 for this input: planted logits s_j, Lk - 3 logits of 0 with value 0
    Kp = np.array(kp, np.float64)
    Vp = np.array(vp, np.float64)
    s = scale * (q[0, 0].astype(np.float64) @ Kp.T)                  # [Lq, 3]
    M = np.maximum(0.0, s.max(axis=1))
    e = np.exp(s - M[:, None])
    Ssum = e.sum(axis=1) + (Lk - len(planted)) * np.exp(-M)
    ref = (e @ Vp) / Ssum[:, None]
    dev = (e[:, :, None] * np.abs(Vp[None] - ref[:, None])).sum(axis=1) / Ssum[:, None] \
        + ((Lk - len(planted)) * np.exp(-M) / Ssum)[:, None] * np.abs(ref)
    for o, tag in ((out, " (plain)"), (out2, " (with statistics)")):
        assert_close(to_host64(o)[0, 0], ref, what="2 GiB of keys" + tag, dev=dev, n_keys=Lk)
    lsr = ls.cpu().numpy().astype(np.float64)[0, 0]
    assert np.max(np.abs(lsr[:, 0] - M) / np.maximum(1.0, M)) <= 1e-5
    assert np.max(np.abs(lsr[:, 1] - Ssum) / Ssum) <= 2e-3 + accumulation_allowance(Lk)
    # the planted rows are their value rows, to the fp16 rounding of the output
    for r, _ in planted:
        assert e[r].max() / Ssum[r] > 1 - 1e-6
        assert np.max(np.abs(to_host64(out)[0, 0, r] - Vp[r]) / np.maximum(1.0, np.abs(Vp[r]))) <= 2e-3


def test_joint_permutation_invariance_on_gpu():
    q, k, v = wl.make_qkv(1, 2, 128, 77, 40, 906)
    perm = np.random.default_rng(907).permutation(77)
    g1 = run_forward(q, k, v, 0.158)
    g2 = run_forward(q, k[:, :, perm].copy(), v[:, :, perm].copy(), 0.158)
    assert np.max(np.abs(g1 - g2)) <= 2e-3


def test_bitwise_deterministic():
    q, k, v = wl.make_qkv(2, 8, 1024, 1024, 40, 908)
    outs = [run_forward(q, k, v, 0.158) for _ in range(3)]
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


def test_inputs_may_alias():
    import torch
    q, _, _ = wl.make_qkv(1, 2, 96, 96, 40, 909)
    qd = to_device(q)
    out = torch.empty_like(qd)
    sd.forward(qd, qd, qd, out, 0.158)
    torch.cuda.synchronize()
    r, _, _, dev = oracle.attention(q, q, q, 0.158, want_dev=True)
    assert_close(to_host64(out), r, what="q=k=v", dev=dev)


def test_bad_arguments_raise():
    import torch
    q = torch.zeros(1, 1, 8, 12, dtype=torch.float16, device="cuda")
    with pytest.raises(sd.SdattnError) as e:
        sd.forward(q, q, q, torch.empty_like(q), 1.0)
    assert e.value.status == sd.STATUS_UNSUPPORTED


@pytest.mark.parametrize("step", range(20))
def test_sweep_step_sampled(step):
    """One UNet evaluation (16 blocks, self then cross) at each of the 20
    denoising steps, with that step's own seeds: 8 sampled rows per head plus
    every head's first and last row."""
    for case in wl.sweep_cases(step):
        q, k, v = wl.case_inputs(case)
        rows = wl.sample_rows(case.B, case.H, case.Lq, 8, seed=case.seed)
        check_case(q, k, v, case.scale, rows=rows, what=case.name, literal=True)


# ------------------------------------------------------------ softmax_rows

def run_softmax_rows(a, scale, dtype, want_p):
    import torch
    ad = to_device(a, "bf16" if dtype == "bf16" else None)
    rows, cols = a.shape
    ls = torch.empty(rows, 2, dtype=torch.float32, device="cuda")
    p = torch.empty_like(ad) if want_p else None
    sd.softmax_rows(ad, ls, p, scale=scale)
    torch.cuda.synchronize()
    return ls.cpu().numpy().astype(np.float64), (to_host64(p) if want_p else None)


@pytest.mark.parametrize("rows,cols,dtype", [
    (64, 4096, "f16"), (7, 77, "f16"), (33, 1000, "f32"), (5, 13, "f32"),
    (16, 20000, "f16"), (3, 50001, "f32"), (100, 256, "bf16"), (1, 1, "f16"),
])
def test_softmax_rows_matches_oracle(rows, cols, dtype):
    a = wl.make_matrix(rows, cols, seed=rows * 7 + cols, dtype=dtype, sigma=4.0)
    scale = 0.7
    ls, p = run_softmax_rows(a, scale, dtype, want_p=True)
    L, S, P = oracle.softmax_rows(a, scale=scale, want_p=True, dtype="bf16" if dtype == "bf16" else None)
    assert np.max(np.abs(ls[:, 0] - L) / np.maximum(1.0, np.abs(L))) <= 1e-6
    assert np.max(np.abs(ls[:, 1] - S) / S) <= 1e-4
    # fp32: the exponent argument a - L (up to ~25 in log2 units here) carries
    # fp32 rounding of ~25 * 2^-23, i.e. ~2.5e-6 relative in p; fp16 / bf16 add
    # the rounding of p itself (2^-11 / 2^-8), measured above fp16's subnormal range.
    ptol = {"f32": 1e-5, "f16": 1e-3, "bf16": 8e-3}[dtype]
    prel = float(np.max(np.abs(p - P) / np.maximum(P, 1e-30 if dtype == "f32" else 6e-5)))
    assert prel <= ptol, f"p relative error {prel:.3e} > {ptol}"
    psum = float(np.max(np.abs(p.sum(axis=1) - 1.0)))
    assert psum <= {"f32": 1e-5, "f16": 2e-3, "bf16": 1.6e-2}[dtype], f"rows of p sum to 1 +- {psum:.3e}"


def test_softmax_rows_without_p_and_negative_scale():
    a = wl.make_matrix(40, 4096, seed=11, dtype="f16")
    ls, _ = run_softmax_rows(a, -1.5, "f16", want_p=False)
    L, S = oracle.softmax_rows(a, scale=-1.5)
    assert np.max(np.abs(ls[:, 0] - L) / np.maximum(1.0, np.abs(L))) <= 1e-6
    assert np.max(np.abs(ls[:, 1] - S) / S) <= 1e-4


def test_softmax_rows_on_attention_logits_matches_forward_stats():
    """softmax_rows on A = Q K^T reproduces the (L, S) the fused forward reports."""
    import torch
    q, k, v = wl.make_qkv(1, 2, 256, 256, 40, 910)
    scale = 0.158
    a = np.einsum("bhid,bhjd->bhij", q.astype(np.float64), k.astype(np.float64)).reshape(-1, 256)
    ls_rows, _ = run_softmax_rows(a.astype(np.float32), scale, "f32", want_p=False)
    _, ls_fwd = run_forward(q, k, v, scale, want_ls=True)
    ls_fwd = ls_fwd.reshape(-1, 2)
    assert np.max(np.abs(ls_rows[:, 0] - ls_fwd[:, 0])) <= 1e-5 * np.abs(ls_rows[:, 0]).max()
    assert np.max(np.abs(ls_rows[:, 1] - ls_fwd[:, 1]) / ls_rows[:, 1]) <= 2e-3


# ------------------------------------ the fixed-maximum path and its fallback

@pytest.mark.parametrize("Lk,D", [(300, 40), (1024, 80), (4096, 40), (520, 64)])
def test_late_dominant_keys_overflow_fast_path_and_fall_back(Lk, D):
    """Keys far larger than the first 32 of each key half: with the reference
    maximum fixed at the first sub-tile, p overflows, and the kernel must fall
    back to the running-maximum path and still match the oracle."""
    rng = np.random.default_rng(Lk + D)
    B, H, Lq = 1, 2, 160
    q = np.zeros((B, H, Lq, D), np.float16)
    q[..., 0] = 8.0
    q[..., 1:] = (rng.standard_normal((B, H, Lq, D - 1)) * 0.1).astype(np.float16)
    k = (rng.standard_normal((B, H, Lk, D)) * 0.1).astype(np.float16)
    v = rng.standard_normal((B, H, Lk, D)).astype(np.float16)
    ntiles = (Lk + 63) // 64
    nh = (ntiles + 1) // 2
    for j in (40, 77, nh * 64 + 40, Lk - 1):      # past the first sub-tile of each half
        if j < Lk:
            k[..., j, 0] = 8.0                    # logit 64 vs ~0 elsewhere (scale 1)
    check_case(q, k, v, 1.0, what=f"late dominant keys Lk={Lk} D={D}")


@pytest.mark.parametrize("Lk,D", [(2048, 40), (700, 80)])
def test_key_norms_growing_along_the_sequence(Lk, D):
    rng = np.random.default_rng(7 * Lk + D)
    q = rng.standard_normal((2, 2, 256, D)).astype(np.float16)
    grow = (1.0 + 3.0 * np.arange(Lk) / Lk)[None, None, :, None]
    k = (rng.standard_normal((2, 2, Lk, D)) * grow).astype(np.float16)
    v = rng.standard_normal((2, 2, Lk, D)).astype(np.float16)
    for scale in (float(np.float32(1 / np.sqrt(D))), 1.0):
        check_case(q, k, v, scale, what=f"growing norms Lk={Lk} D={D} scale={scale}")


# ------------------- the workgroup geometries the UNet levels launch, with the
# fixed-maximum fast path and its exact fallback.  B = 2, H = 8 at Lq = 4096
# (D <= 64) fills the chip with 256-row workgroups of eight waves and 128-key
# tiles (the 64x64 level); Lq = 2048 takes 128-row workgroups; the launch with
# statistics always takes 128-row workgroups.  The overflow vote and the
# online rerun run per workgroup, so only the heads whose keys are planted
# take the fallback while the others stay on the fast path.

def _late_dominant_inputs(B, H, Lq, Lk, D, tile_keys, seed, dtype):
    """q.k = 64 for a few keys past the first 32-key sub-tile of each key half
    (about 0 elsewhere) in the even heads: with scale 1 the rounded p of those
    keys overflows under a maximum fixed at the first sub-tile."""
    rng = np.random.default_rng(seed)
    q = np.zeros((B, H, Lq, D), np.float32)
    q[..., 0] = 8.0
    q[..., 1:] = rng.standard_normal((B, H, Lq, D - 1), dtype=np.float32) * 0.1
    k = rng.standard_normal((B, H, Lk, D), dtype=np.float32) * 0.1
    v = rng.standard_normal((B, H, Lk, D), dtype=np.float32)
    ntiles = (Lk + tile_keys - 1) // tile_keys
    nh = (ntiles + 1) // 2
    for j in (40, 77, nh * tile_keys + 40, Lk - 1):
        if j < Lk:
            k[:, ::2, j, 0] = 8.0
    if dtype == "bf16":
        return tuple(wl.to_bf16_bits(t) for t in (q, k, v))
    return tuple(t.astype(np.float16) for t in (q, k, v))


def _rows_with_edges(B, H, Lq, per_head, seed):
    rows = wl.sample_rows(B, H, Lq, per_head, seed=seed)
    return np.unique(np.concatenate([rows, [Lq - 1, Lq, 2 * Lq - 1, B * H * Lq - 1]]))


@pytest.mark.parametrize("Lk,dtype", [(4096, "f16"), (4096, "bf16"), (700, "f16"), (350, "f16")])
def test_big_geometry_late_dominant_keys_fall_back(Lk, dtype):
    """256-row workgroups (plain launch) and 128-row ones (with statistics):
    the eight-wave vote and the online rerun over 128-key tiles, including a
    ragged last tile of key half 1 left pending in buffer 0 (Lk = 700 for
    128-key tiles, Lk = 350 for 64-key tiles)."""
    B, H, Lq, D = 2, 8, 4096, 40
    q, k, v = _late_dominant_inputs(B, H, Lq, Lk, D, 128, 5100 + Lk, dtype)
    rows = _rows_with_edges(B, H, Lq, 24, seed=Lk)
    check_case(q, k, v, 1.0, dtype=dtype, rows=rows, what=f"big late-dominant Lk={Lk} {dtype}")
    if Lk == 350:   # the 64-key tiles of the statistics launch: plant per its tiling too
        q, k, v = _late_dominant_inputs(B, H, Lq, Lk, D, 64, 5200 + Lk, dtype)
        check_case(q, k, v, 1.0, dtype=dtype, rows=rows, what=f"late-dominant 64-key tiles Lk={Lk}")


@pytest.mark.parametrize("dtype", ["f16", "bf16"])
def test_big_geometry_growing_key_norms(dtype):
    """Key norms growing along the sequence at scale 1: later tiles dominate,
    so the fixed maximum overflows in every workgroup."""
    B, H, Lq, Lk, D = 2, 8, 4096, 4096, 40
    rng = np.random.default_rng(5300)
    q = rng.standard_normal((B, H, Lq, D), dtype=np.float32)
    grow = (1.0 + 3.0 * np.arange(Lk) / Lk).astype(np.float32)[None, None, :, None]
    k = rng.standard_normal((B, H, Lk, D), dtype=np.float32) * grow
    v = rng.standard_normal((B, H, Lk, D), dtype=np.float32)
    if dtype == "bf16":
        q, k, v = (wl.to_bf16_bits(t) for t in (q, k, v))
    else:
        q, k, v = (t.astype(np.float16) for t in (q, k, v))
    rows = _rows_with_edges(B, H, Lq, 24, seed=7)
    for scale in (float(np.float32(1 / np.sqrt(D))), 1.0):
        check_case(q, k, v, scale, dtype=dtype, rows=rows, what=f"big growing norms scale={scale} {dtype}")


@pytest.mark.parametrize("D", [40, 80])
@pytest.mark.parametrize("variant", ["normal", "late_dominant"])
def test_128_row_geometry_plain_launch(D, variant):
    """B2 H8 Lq 2048: 256 workgroups of 128 rows, the plain launch's middle
    geometry (two 32-row blocks per wave at D = 40, one at D = 80)."""
    B, H, Lq, Lk = 2, 8, 2048, 2048
    if variant == "normal":
        q, k, v = wl.make_qkv(B, H, Lq, Lk, D, 5400 + D)
        scale = float(np.float32(1 / np.sqrt(D)))
    else:
        q, k, v = _late_dominant_inputs(B, H, Lq, Lk, D, 64, 5500 + D, "f16")
        scale = 1.0
    rows = _rows_with_edges(B, H, Lq, 24, seed=D)
    check_case(q, k, v, scale, rows=rows, what=f"128-row Lq=2048 D={D} {variant}")


def test_bitwise_deterministic_at_the_64x64_level():
    case = wl.CASES["l64_self"]
    q, k, v = wl.case_inputs(case)
    outs = [run_forward(q, k, v, case.scale) for _ in range(3)]
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])


# ------------- 64-row workgroups with the keys split four ways (eight waves):
# the plain launch's geometry for grids of fewer than 256 128-row blocks once
# Lk >= 512 and D <= 80 (the 32x32 level).  Split s takes tiles s*nh ..
# s*nh + nh - 1 (nh = ceil(ntiles / 4)); the last splits may be short or
# empty.  These tiles carry no constant block, so the row sum comes from
# v_dot2 and the padded d rows read V columns that are never stored.

QUARTER = [
    # (B, H, Lq, Lk, D, dtype)
    (1, 2, 200, 700, 80, "f16"),    # 11 tiles: 3 + 3 + 3 + 2, ragged last tile
    (1, 2, 130, 513, 40, "f16"),    # 9 tiles: 3 + 3 + 3 + 0, last tile one key
    (2, 1, 100, 1000, 56, "f16"),
    (1, 3, 64, 600, 72, "f16"),
    (1, 1, 97, 2048, 32, "f16"),
    (1, 1, 33, 4100, 64, "f16"),    # 65 tiles: 17 + 17 + 17 + 14
    (1, 2, 160, 777, 48, "bf16"),
    (1, 2, 96, 1024, 80, "bf16"),
]


@pytest.mark.parametrize("shape", QUARTER, ids=lambda s: "x".join(map(str, s)))
def test_quarter_key_split_geometry(shape):
    B, H, Lq, Lk, D, dtype = shape
    q, k, v = wl.make_qkv(B, H, Lq, Lk, D, 6100 + Lq + 3 * Lk + D, dtype=dtype)
    check_case(q, k, v, float(np.float32(1 / np.sqrt(D))), dtype=dtype, what=f"quarter {shape}")


@pytest.mark.parametrize("Lk,D,dtype", [(700, 80, "f16"), (1024, 40, "f16"), (513, 64, "f16"),
                                        (1500, 80, "bf16")])
def test_quarter_geometry_late_dominant_keys_fall_back(Lk, D, dtype):
    """Keys past the first 32-key sub-tile of every one of the four splits
    dominate in the even heads: the eight-wave vote sends the workgroup
    through the online rerun and the four-way merge."""
    B, H, Lq = 1, 4, 150
    rng = np.random.default_rng(6200 + Lk + D)
    q = np.zeros((B, H, Lq, D), np.float32)
    q[..., 0] = 8.0
    q[..., 1:] = rng.standard_normal((B, H, Lq, D - 1), dtype=np.float32) * 0.1
    k = rng.standard_normal((B, H, Lk, D), dtype=np.float32) * 0.1
    v = rng.standard_normal((B, H, Lk, D), dtype=np.float32)
    nh = ((Lk + 63) // 64 + 3) // 4
    for s in range(4):
        j = s * nh * 64 + 40
        if j < Lk:
            k[:, ::2, j, 0] = 8.0
    k[:, ::2, Lk - 1, 0] = 8.0
    if dtype == "bf16":
        q, k, v = (wl.to_bf16_bits(t) for t in (q, k, v))
    else:
        q, k, v = (t.astype(np.float16) for t in (q, k, v))
    check_case(q, k, v, 1.0, dtype=dtype, what=f"quarter late-dominant Lk={Lk} D={D} {dtype}")


def test_quarter_geometry_bitwise_deterministic():
    case = wl.CASES["l32_self"]
    q, k, v = wl.case_inputs(case)
    outs = [run_forward(q, k, v, case.scale) for _ in range(3)]
    assert np.array_equal(outs[0], outs[1]) and np.array_equal(outs[0], outs[2])
