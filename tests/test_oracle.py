"""Pins of the fp64 oracle against facts it must reproduce (CPU only).

Each pin is something other than the oracle's own formula: exact decoding
against numpy's float16 routine, a 50-digit brute force of Eq. 3 written
without the max subtraction, closed forms (constant keys, zero scale, one key,
constant value columns, identity values), invariants (joint key/value
permutation, linearity in V, shift invariance of Eq. 4), the block-merge rule
of the multi-stage reduction (Sec. 3.2.1), and torch's fp64 CPU attention and
softmax as independent library routines.  A dropped term, a wrong sign, a
wrong scale, a transposed operand or a wrong row index fails at least one.
"""
import numpy as np
import pytest

import oracle
from paper_2304_11267_amd import workloads as wl

mpmath = pytest.importorskip("mpmath")


def _rand16(rng, shape, mult=1.0):
    return (rng.standard_normal(shape, dtype=np.float32) * np.float32(mult)).astype(np.float16)


# ----------------------------------------------------------------- decoding

def test_widen_binary16_every_bit_pattern():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    h = bits.view(np.float16)
    got = oracle.widen(h)
    ref = h.astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])
    # signed zeros keep their sign
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def test_widen_bfloat16_matches_float32_upper_half():
    rng = np.random.default_rng(7)
    bits = rng.integers(0, 65536, size=20000, dtype=np.uint32).astype(np.uint16)
    got = oracle.widen(bits, dtype="bf16")
    with np.errstate(invalid="ignore"):
        ref = (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


# ------------------------------------------------------ brute force, Eq. 3

def _brute_force(q, k, v, scale):
    """Eq. 3 at 50 digits, direct form sum_j e^{s_j} v_j / sum_j e^{s_j}."""
    mp = mpmath.mp
    mp.dps = 50
    B, H, Lq, D = q.shape
    Lk = k.shape[2]
    qf, kf, vf = (t.astype(np.float64) for t in (q, k, v))
    sc = mpmath.mpf(float(np.float32(scale)))
    out = np.zeros((B, H, Lq, D))
    devs = np.zeros((B, H, Lq, D))
    Ls = np.zeros((B, H, Lq))
    Ss = np.zeros((B, H, Lq))
    for b in range(B):
        for h in range(H):
            for i in range(Lq):
                s = [sc * mpmath.fsum(mpmath.mpf(float(qf[b, h, i, d])) * mpmath.mpf(float(kf[b, h, j, d]))
                                      for d in range(D)) for j in range(Lk)]
                w = [mpmath.exp(x) for x in s]
                tot = mpmath.fsum(w)
                for d in range(D):
                    od = mpmath.fsum(w[j] * mpmath.mpf(float(vf[b, h, j, d])) for j in range(Lk)) / tot
                    out[b, h, i, d] = float(od)
                    devs[b, h, i, d] = float(mpmath.fsum(
                        w[j] * abs(mpmath.mpf(float(vf[b, h, j, d])) - od) for j in range(Lk)) / tot)
                L = max(s)
                Ls[b, h, i] = float(L)
                Ss[b, h, i] = float(mpmath.fsum(mpmath.exp(x - L) for x in s))
    _brute_force.dev = devs
    return out, Ls, Ss


BRUTE_SHAPES = [
    # (B, H, Lq, Lk, D, q_mult, scale or None for 1/sqrt(D))
    (1, 1, 1, 1, 8, 1.0, None),
    (1, 1, 3, 5, 8, 1.0, None),
    (2, 2, 4, 7, 16, 1.0, None),
    (1, 2, 8, 8, 40, 1.0, None),
    (1, 1, 5, 3, 24, 1.0, None),
    (1, 1, 6, 8, 16, 8.0, 1.0),     # logits in the hundreds: needs the max shift
    (1, 1, 4, 6, 8, 4.0, -0.75),    # negative scale
]


@pytest.mark.parametrize("shape", BRUTE_SHAPES)
def test_brute_force_small(shape):
    B, H, Lq, Lk, D, mult, scale = shape
    rng = np.random.default_rng(1000 + Lq * 31 + Lk * 7 + D)
    q = _rand16(rng, (B, H, Lq, D), mult)
    k = _rand16(rng, (B, H, Lk, D))
    v = _rand16(rng, (B, H, Lk, D))
    if scale is None:
        scale = float(np.float32(1 / np.sqrt(D)))
    o, L, S, dev = oracle.attention(q, k, v, scale, want_dev=True)
    ro, rL, rS = _brute_force(q, k, v, scale)
    vmax = np.abs(v.astype(np.float64)).max()
    assert np.max(np.abs(o - ro)) <= 1e-12 * vmax
    assert np.max(np.abs(L - rL) / np.maximum(1.0, np.abs(rL))) <= 1e-12
    assert np.max(np.abs(S - rS) / rS) <= 1e-12
    # the weighted mean absolute deviation of the value columns (the parity
    # tests' sensitivity of O to a relative rounding of the weights)
    assert np.max(np.abs(dev - _brute_force.dev)) <= 1e-12 * vmax
    o2, L2, S2 = oracle.attention(q, k, v, scale)
    assert np.array_equal(o, o2) and np.array_equal(L, L2) and np.array_equal(S, S2)


def test_value_deviation_closed_forms():
    """dev_id = sum_j p_ij |v_jd - o_id|: zero for one key or constant value
    columns; |v_0 - v_1| / 2 for two keys of equal logit; bounded by the
    largest |v_jd - o_id|; and, being first order in the weights, the change
    of o_id when every weight is rounded by a relative 2^-11."""
    rng = np.random.default_rng(12)
    q = _rand16(rng, (1, 2, 9, 16), 2.0)
    k = _rand16(rng, (1, 2, 1, 16))
    v = _rand16(rng, (1, 2, 1, 16))
    _, _, _, dev = oracle.attention(q, k, v, 0.3, want_dev=True)
    assert np.all(dev == 0.0)
    k = _rand16(rng, (1, 2, 13, 16))
    v = np.broadcast_to(_rand16(rng, (1, 2, 1, 16)), (1, 2, 13, 16)).copy()
    _, _, _, dev = oracle.attention(q, k, v, 0.3, want_dev=True)
    assert np.max(np.abs(dev)) <= 1e-15
    # two identical keys: equal weights
    k = np.broadcast_to(_rand16(rng, (1, 2, 1, 16)), (1, 2, 2, 16)).copy()
    v = _rand16(rng, (1, 2, 2, 16))
    _, _, _, dev = oracle.attention(q, k, v, 0.3, want_dev=True)
    vf = v.astype(np.float64)
    half = np.abs(vf[:, :, 0] - vf[:, :, 1])[:, :, None, :] / 2
    assert np.max(np.abs(dev - np.broadcast_to(half, dev.shape))) <= 1e-15
    # bound and first-order sensitivity on random inputs
    q = _rand16(rng, (1, 1, 7, 16), 2.0)
    k = _rand16(rng, (1, 1, 50, 16))
    v = _rand16(rng, (1, 1, 50, 16))
    o, L, S, dev = oracle.attention(q, k, v, 0.4, want_dev=True)
    vf = v.astype(np.float64)[0, 0]
    assert np.all(dev[0, 0] <= np.abs(vf[None, :, :] - o[0, 0][:, None, :]).max(axis=1) + 1e-15)
    a = oracle.logits(q, k, 0.4)[0, 0]
    p = np.exp(a - L[0, 0][:, None]) / S[0, 0][:, None]
    worst = 0.0
    for trial in range(200):
        delta = rng.choice([-1.0, 1.0], size=p.shape) * 2.0 ** -11
        pt = p * (1 + delta)
        ot = (pt @ vf) / pt.sum(axis=1, keepdims=True)
        worst = max(worst, float(np.max(np.abs(ot - o[0, 0]) / (2.0 ** -11 * dev[0, 0] * (1 + 2.0 ** -10)
                                                                   + 1e-300))))
    assert worst <= 1.0


# --------------------------------------------------------------- structure

def test_row_subset_and_thread_count_do_not_change_results():
    rng = np.random.default_rng(3)
    q = _rand16(rng, (2, 3, 37, 24))
    k = _rand16(rng, (2, 3, 29, 24))
    v = _rand16(rng, (2, 3, 29, 24))
    full, L, S = oracle.attention(q, k, v, 0.2, nthreads=1)
    full8, L8, S8 = oracle.attention(q, k, v, 0.2, nthreads=8)
    assert np.array_equal(full, full8) and np.array_equal(L, L8) and np.array_equal(S, S8)
    rows = np.array([0, 5, 36, 37, 100, 221, 2 * 3 * 37 - 1])
    sub, Ls, Ss = oracle.attention(q, k, v, 0.2, rows=rows)
    flat = full.reshape(-1, 24)
    assert np.array_equal(sub, flat[rows])
    assert np.array_equal(Ls, L.reshape(-1)[rows])
    assert np.array_equal(Ss, S.reshape(-1)[rows])


def test_constant_keys_give_mean_of_values():
    rng = np.random.default_rng(4)
    q = _rand16(rng, (2, 2, 9, 40))
    k = np.broadcast_to(_rand16(rng, (2, 2, 1, 40)), (2, 2, 13, 40)).copy()
    v = _rand16(rng, (2, 2, 13, 40))
    o, _, S = oracle.attention(q, k, v, 0.3)
    ref = v.astype(np.float64).mean(axis=2, keepdims=True)
    assert np.max(np.abs(o - ref)) <= 1e-14
    assert np.allclose(S, 13.0, rtol=0, atol=1e-12)


def test_zero_scale_gives_mean_of_values():
    rng = np.random.default_rng(5)
    q, k, v = (_rand16(rng, (1, 2, n, 16)) for n in (5, 11, 11))
    o, L, S = oracle.attention(q, k, v, 0.0)
    assert np.max(np.abs(o - v.astype(np.float64).mean(axis=2, keepdims=True))) <= 1e-14
    assert np.all(L == 0.0) and np.all(S == 11.0)


def test_single_key_returns_its_value_exactly():
    rng = np.random.default_rng(6)
    q = _rand16(rng, (2, 2, 7, 32), 3.0)
    k = _rand16(rng, (2, 2, 1, 32))
    v = _rand16(rng, (2, 2, 1, 32))
    o, _, S = oracle.attention(q, k, v, 0.5)
    assert np.array_equal(o, np.broadcast_to(v.astype(np.float64), o.shape))
    assert np.all(S == 1.0)


def test_constant_value_columns_give_the_constant():
    rng = np.random.default_rng(8)
    q = _rand16(rng, (1, 2, 6, 16), 2.0)
    k = _rand16(rng, (1, 2, 19, 16))
    cols = _rand16(rng, (1, 2, 1, 16))
    v = np.broadcast_to(cols, (1, 2, 19, 16)).copy()
    o, _, _ = oracle.attention(q, k, v, 0.25)
    ref = np.broadcast_to(cols.astype(np.float64), o.shape)
    assert np.max(np.abs(o - ref) / np.maximum(np.abs(ref), 1e-300)) <= 1e-14


def test_identity_values_reproduce_softmax_rows():
    """V = I with Lk = D gives O = P, the element-wise step of Eq. 4."""
    rng = np.random.default_rng(9)
    D = 16
    q = _rand16(rng, (1, 1, 10, D), 2.0)
    k = _rand16(rng, (1, 1, D, D))
    v = np.eye(D, dtype=np.float16)[None, None]
    scale = 0.35
    o, L, S = oracle.attention(q, k, v, scale)
    a = q[0, 0].astype(np.float64) @ k[0, 0].astype(np.float64).T   # library matmul
    Lr, Sr, P = oracle.softmax_rows(a, scale=scale, want_p=True)
    assert np.max(np.abs(o[0, 0] - P)) <= 1e-14
    assert np.max(np.abs(L[0, 0] - Lr)) <= 1e-13
    assert np.max(np.abs(S[0, 0] - Sr) / Sr) <= 1e-13


def test_joint_key_value_permutation_invariance():
    rng = np.random.default_rng(10)
    q = _rand16(rng, (2, 2, 8, 40), 2.0)
    k = _rand16(rng, (2, 2, 77, 40))
    v = _rand16(rng, (2, 2, 77, 40))
    perm = rng.permutation(77)
    o1, L1, S1 = oracle.attention(q, k, v, 0.158)
    o2, L2, S2 = oracle.attention(q, k[:, :, perm].copy(), v[:, :, perm].copy(), 0.158)
    assert np.max(np.abs(o1 - o2)) <= 1e-13
    assert np.array_equal(L1, L2)
    assert np.max(np.abs(S1 - S2) / S1) <= 1e-13
    # permuting keys alone does change the output (the pairing matters)
    o3, _, _ = oracle.attention(q, k[:, :, perm].copy(), v, 0.158)
    assert np.max(np.abs(o1 - o3)) > 1e-2


def test_linear_in_values():
    rng = np.random.default_rng(11)
    q = rng.standard_normal((1, 2, 5, 8))
    k = rng.standard_normal((1, 2, 9, 8))
    v1 = rng.standard_normal((1, 2, 9, 8))
    v2 = rng.standard_normal((1, 2, 9, 8))
    o1, _, _ = oracle.attention(q, k, v1, 0.4)
    o2, _, _ = oracle.attention(q, k, v2, 0.4)
    o12, _, _ = oracle.attention(q, k, 2.0 * v1 - 3.0 * v2, 0.4)
    assert np.max(np.abs(o12 - (2.0 * o1 - 3.0 * o2))) <= 1e-13


def test_one_hot_dominant_logit_selects_its_value_row():
    rng = np.random.default_rng(12)
    Lk, D = 20, 8
    k = rng.standard_normal((1, 1, Lk, D)) * 0.1
    v = rng.standard_normal((1, 1, Lk, D))
    star = 13
    k[0, 0, star, 0] = 10.0
    q = np.zeros((1, 1, 3, D))
    q[0, 0, :, 0] = 6.0        # logit gap >= 6*(10 - 0.5) = 57 > 40
    o, L, S = oracle.attention(q, k, v, 1.0)
    assert np.max(np.abs(o[0, 0] - v[0, 0, star])) <= 1e-15 * 1e3
    assert np.allclose(L, 60.0) and np.all(np.abs(S - 1.0) < 1e-16 * 1e3)


# ------------------------------------------------------ Eq. 4 and its merge

def test_softmax_rows_probabilities_sum_to_one():
    a = wl.make_matrix(33, 517, seed=13, dtype="f16", sigma=3.0)
    L, S, P = oracle.softmax_rows(a, scale=0.7, want_p=True)
    assert np.max(np.abs(P.sum(axis=1) - 1.0)) <= 1e-13
    assert np.all(P >= 0) and np.all(P <= 1.0)
    # the max element has weight exactly 1/S
    am = float(np.float32(0.7)) * a.astype(np.float64)   # the scale the GPU receives is fp32
    assert np.array_equal(L, am.max(axis=1))
    assert np.allclose(P[np.arange(33), am.argmax(axis=1)], 1.0 / S, rtol=1e-15)


def test_softmax_rows_shift_invariance():
    rng = np.random.default_rng(14)
    a = rng.standard_normal((12, 64))
    c = rng.integers(-50, 50, size=(12, 1)).astype(np.float64)
    L1, S1, P1 = oracle.softmax_rows(a, want_p=True)
    L2, S2, P2 = oracle.softmax_rows(a + c, want_p=True)
    assert np.max(np.abs(L2 - (L1 + c[:, 0]))) <= 1e-13
    assert np.max(np.abs(S2 - S1) / S1) <= 1e-12
    assert np.max(np.abs(P2 - P1)) <= 1e-12


def _merge(m1, s1, m2, s2):
    """Combine two blocks' (max, shifted sum) pairs: the multi-stage reduction."""
    M = np.maximum(m1, m2)
    return M, s1 * np.exp(m1 - M) + s2 * np.exp(m2 - M)


def test_block_merge_rule_reproduces_whole_row_statistics():
    rng = np.random.default_rng(15)
    a = rng.standard_normal((40, 300)) * 4.0
    L, S = oracle.softmax_rows(a)
    for _ in range(5):
        cut = int(rng.integers(1, 299))
        L1, S1 = oracle.softmax_rows(np.ascontiguousarray(a[:, :cut]))
        L2, S2 = oracle.softmax_rows(np.ascontiguousarray(a[:, cut:]))
        M, T = _merge(L1, S1, L2, S2)
        assert np.array_equal(M, L)
        assert np.max(np.abs(T - S) / S) <= 1e-13
    # four-way, merged in two different orders
    parts = np.array_split(np.arange(300), 4)
    st = [oracle.softmax_rows(np.ascontiguousarray(a[:, p])) for p in parts]
    left = _merge(*_merge(*st[0], *st[1]), *_merge(*st[2], *st[3]))
    right = _merge(*st[0], *_merge(*st[1], *_merge(*st[2], *st[3])))
    for m, s in (left, right):
        assert np.array_equal(m, L)
        assert np.max(np.abs(s - S) / S) <= 1e-13


def test_softmax_rows_matches_torch_logsumexp():
    torch = pytest.importorskip("torch")
    a = wl.make_matrix(20, 1000, seed=16, dtype="f32", sigma=5.0)
    L, S, P = oracle.softmax_rows(a, scale=0.5, want_p=True)
    t = torch.from_numpy(a.astype(np.float64)) * float(np.float32(0.5))
    assert np.array_equal(L, t.max(dim=1).values.numpy())
    lse = torch.logsumexp(t, dim=1).numpy()
    assert np.max(np.abs(np.log(S) + L - lse)) <= 1e-12
    assert np.max(np.abs(P - torch.softmax(t, dim=1).numpy())) <= 1e-15


# ----------------------------------- independent library at workload shapes

def _torch_sdpa_rows(q, k, v, scale, rows):
    torch = pytest.importorskip("torch")
    B, H, Lq, D = q.shape
    qq = torch.from_numpy(q.astype(np.float64)).reshape(B * H, Lq, D)
    kk = torch.from_numpy(k.astype(np.float64)).reshape(B * H, -1, D)
    vv = torch.from_numpy(v.astype(np.float64)).reshape(B * H, -1, D)
    out = np.empty((rows.size, D))
    bh = rows // Lq
    for g in np.unique(bh):
        sel = np.nonzero(bh == g)[0]
        qi = qq[g, rows[sel] % Lq][None]
        o = torch.nn.functional.scaled_dot_product_attention(qi, kk[g][None], vv[g][None],
                                                             scale=float(np.float32(scale)))
        out[sel] = o[0].numpy()
    return out


@pytest.mark.parametrize("name", ["mid8_self", "mid8_cross", "l16_self_peaked", "l16_cross",
                                  "l32_self", "l32_cross", "l64_self", "l64_cross"])
def test_matches_torch_fp64_sdpa_at_unet_shapes(name):
    case = wl.CASES[name]
    q, k, v = wl.case_inputs(case)
    per_head = case.Lq if case.Lq <= 256 else 8
    rows = wl.sample_rows(case.B, case.H, case.Lq, per_head, seed=case.seed)
    o, _, _ = oracle.attention(q, k, v, case.scale, rows=rows)
    ref = _torch_sdpa_rows(q, k, v, case.scale, rows)
    assert np.max(np.abs(o - ref)) <= 1e-12


def test_rejects_bad_arguments():
    q = np.zeros((1, 1, 2, 8), np.float16)
    with pytest.raises(ValueError):
        oracle.attention(q, np.zeros((1, 1, 3, 8), np.float16), np.zeros((1, 1, 4, 8), np.float16), 1.0)
    with pytest.raises(ValueError):
        oracle.attention(q, q, q, 1.0, rows=np.array([2]))
    with pytest.raises(ValueError):
        oracle.softmax_rows(np.zeros((0, 4), np.float32))


# ------------------------------------------------------ the input generator

def test_generator_is_seeded_and_shaped():
    c = wl.CASES["l32_cross"]
    q1, k1, v1 = wl.case_inputs(c)
    q2, k2, v2 = wl.case_inputs(c)
    assert q1.shape == (2, 8, 1024, 80) and k1.shape == (2, 8, 77, 80) and v1.shape == k1.shape
    assert q1.dtype == np.float16
    assert np.array_equal(q1, q2) and np.array_equal(k1, k2) and np.array_equal(v1, v2)
    assert abs(float(q1.astype(np.float64).std()) - 1.0) < 0.01
    peaked = wl.case_inputs(wl.CASES["l16_self_peaked"])[0]
    plain = wl.case_inputs(wl.CASES["l16_self"])[0]
    assert np.array_equal(peaked.astype(np.float64), 4.0 * plain.astype(np.float64))


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(17)
    x = rng.standard_normal(50000, dtype=np.float32) * 3
    ours = wl.to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)


def test_sweep_has_sixteen_blocks_of_self_and_cross():
    cases = wl.sweep_cases(0)
    assert len(cases) == 32
    sides = [c.Lq for c in cases[::2]]
    assert sides == [4096] * 2 + [1024] * 2 + [256] * 2 + [64] + [256] * 3 + [1024] * 3 + [4096] * 3
    assert all(c.Lk == 77 for c in cases[1::2])
    assert len({c.seed for s in range(20) for c in wl.sweep_cases(s)}) == 640


# ------------------------------------------- partially fused softmax steps
# (Sec. 3.2.1: logits A = scale Q K^T, Eq. 4's reduction, then exp(A - L)/S
# times V.)  Pins: numpy's fp64 matmul for the logits, a 50-digit brute force
# of the last step on a given A, the composition identity with the pinned
# attention, closed forms, and the roles of L and S when they are passed in.

def test_logits_match_numpy_fp64_matmul():
    rng = np.random.default_rng(40)
    q = _rand16(rng, (2, 3, 17, 40))
    k = _rand16(rng, (2, 3, 29, 40))
    a = oracle.logits(q, k, 0.375)
    ref = 0.375 * np.matmul(q.astype(np.float64), np.swapaxes(k.astype(np.float64), 2, 3))
    assert a.shape == (2, 3, 17, 29)
    assert np.max(np.abs(a - ref)) <= 1e-13 * np.abs(ref).max()
    # a transposed operand or a swapped head would not match
    assert np.max(np.abs(a[0, 1] - a[0, 2])) > 1.0


def test_logits_rows_subset_and_bf16():
    rng = np.random.default_rng(41)
    q, k, _ = wl.make_qkv(1, 2, 9, 11, 16, 42, dtype="bf16")
    a = oracle.logits(q, k, 0.25, dtype="bf16")
    qf, kf = oracle.widen(q, dtype="bf16"), oracle.widen(k, dtype="bf16")
    ref = 0.25 * np.matmul(qf, np.swapaxes(kf, 2, 3))
    assert np.max(np.abs(a - ref)) <= 1e-13 * np.abs(ref).max()
    rows = np.array([0, 8, 9, 17])
    sub = oracle.logits(q, k, 0.25, rows=rows, dtype="bf16")
    assert np.array_equal(sub, a.reshape(-1, 11)[rows])


def _brute_force_pv(a, v):
    """sum_j e^{a_j} v_j / sum_j e^{a_j} at 50 digits, no max shift."""
    mp = mpmath.mp
    mp.dps = 50
    B, H, Lq, Lk = a.shape
    D = v.shape[3]
    out = np.zeros((B, H, Lq, D))
    for b in range(B):
        for h in range(H):
            for i in range(Lq):
                w = [mpmath.exp(mpmath.mpf(float(x))) for x in a[b, h, i]]
                tot = mpmath.fsum(w)
                for d in range(D):
                    out[b, h, i, d] = float(mpmath.fsum(w[j] * mpmath.mpf(float(v[b, h, j, d]))
                                                        for j in range(Lk)) / tot)
    return out


@pytest.mark.parametrize("a_scale", [1.0, 40.0])
def test_softmax_pv_brute_force_small(a_scale):
    rng = np.random.default_rng(43)
    a = (rng.standard_normal((1, 2, 4, 9)) * a_scale).astype(np.float32)   # logits up to ~100
    v = _rand16(rng, (1, 2, 9, 8))
    o = oracle.softmax_pv(a, v)
    ref = _brute_force_pv(a, v)
    assert np.max(np.abs(o - ref)) <= 1e-12 * np.abs(v.astype(np.float64)).max()


def test_logits_then_softmax_pv_is_attention():
    q, k, v = wl.make_qkv(2, 2, 33, 47, 24, 44)
    scale = float(np.float32(1 / np.sqrt(24)))
    a = oracle.logits(q, k, scale)
    o = oracle.softmax_pv(a, v)
    r, _, _ = oracle.attention(q, k, v, scale)
    assert np.max(np.abs(o - r)) <= 1e-13
    # with Eq. 4's statistics taken from softmax_rows on the same A
    L, S = oracle.softmax_rows(a.reshape(-1, 47))
    o2 = oracle.softmax_pv(a, v, ls=np.stack([L, S], axis=1))
    assert np.max(np.abs(o2 - r)) <= 1e-13


def test_softmax_pv_closed_forms():
    rng = np.random.default_rng(45)
    v = _rand16(rng, (1, 2, 13, 16))
    vf = v.astype(np.float64)
    # constant rows of A: uniform weights, the mean of V
    a = np.broadcast_to(rng.standard_normal((1, 2, 6, 1)), (1, 2, 6, 13)).copy()
    o = oracle.softmax_pv(a, v)
    assert np.max(np.abs(o - vf.mean(axis=2, keepdims=True))) <= 1e-14
    # one logit 60 above the rest (other weights < 1e-25): that value row
    a = rng.standard_normal((1, 2, 6, 13))
    star = rng.integers(0, 13, size=(2, 6))
    for h in range(2):
        for i in range(6):
            a[0, h, i, star[h, i]] = 60.0
    o = oracle.softmax_pv(a, v)
    for h in range(2):
        for i in range(6):
            assert np.max(np.abs(o[0, h, i] - vf[0, h, star[h, i]])) <= 1e-15


def test_softmax_pv_uses_the_given_l_and_s():
    rng = np.random.default_rng(46)
    a = rng.standard_normal((1, 1, 5, 12))
    v = _rand16(rng, (1, 1, 12, 8))
    L, S = oracle.softmax_rows(a.reshape(-1, 12))
    base = oracle.softmax_pv(a, v, ls=np.stack([L, S], axis=1))
    # (L + c, S e^{-c}) is the same normalisation: the result does not move
    c = 3.5
    same = oracle.softmax_pv(a, v, ls=np.stack([L + c, S * np.exp(-c)], axis=1))
    assert np.max(np.abs(same - base)) <= 1e-14
    # doubling S halves O; lowering L by 1 scales O by e
    half = oracle.softmax_pv(a, v, ls=np.stack([L, 2 * S], axis=1))
    assert np.max(np.abs(half - base / 2)) <= 1e-15
    up = oracle.softmax_pv(a, v, ls=np.stack([L - 1, S], axis=1))
    assert np.max(np.abs(up - base * np.e)) <= 1e-14


# ------------------------------------------------- projections and the block
# Pins: numpy's fp64 matmul for the linear layer; torch's fp64 CPU
# scaled_dot_product_attention composed with torch matmuls (an independent
# library) for the multi-head block; closed forms (zero value or output
# weights leave the bias; one head is the single-head attention of the
# projections); row subsets.

def _blk_inputs(seed, B=2, Lq=9, Lk=7, C=32, Cc=24, dtype=np.float16):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((B, Lq, C)).astype(dtype)
    ctx = rng.standard_normal((B, Lk, Cc)).astype(dtype)
    ws = [(rng.standard_normal(s) / np.sqrt(s[1])).astype(dtype)
          for s in ((C, C), (C, Cc), (C, Cc), (C, C))]
    bo = (rng.standard_normal(C) * 0.5).astype(dtype)
    return x, ctx, ws, bo


def test_linear_matches_numpy_matmul():
    rng = np.random.default_rng(60)
    x = _rand16(rng, (3, 5, 40))
    w = _rand16(rng, (24, 40))
    b = _rand16(rng, (24,))
    y = oracle.linear(x, w, b)
    ref = x.astype(np.float64) @ w.astype(np.float64).T + b.astype(np.float64)
    assert y.shape == (3, 5, 24)
    assert np.max(np.abs(y - ref)) <= 1e-13 * np.abs(ref).max()
    assert np.max(np.abs(oracle.linear(x, w) - (ref - b.astype(np.float64)))) <= 1e-13 * np.abs(ref).max()


def test_linear_closed_forms():
    rng = np.random.default_rng(64)
    x = _rand16(rng, (2, 3, 16))
    eye = np.eye(16, dtype=np.float16)
    assert np.array_equal(oracle.linear(x, eye), x.astype(np.float64))
    # w picks and scales single input channels: y[..., n] = 2 x[..., 15 - n]
    sel = np.zeros((16, 16), dtype=np.float16)
    sel[np.arange(16), 15 - np.arange(16)] = 2.0
    assert np.array_equal(oracle.linear(x, sel), 2.0 * x.astype(np.float64)[..., ::-1])
    b = _rand16(rng, (8,))
    w = _rand16(rng, (8, 16))
    assert np.array_equal(oracle.linear(np.zeros_like(x), w, b)[1, 2], b.astype(np.float64))


def test_attention_block_matches_torch_fp64():
    torch = pytest.importorskip("torch")
    x, ctx, (wq, wk, wv, wo), bo = _blk_inputs(61)
    H, scale = 4, float(np.float32(0.3))   # the oracle takes the scale as fp32
    out = oracle.attention_block(x, ctx, wq, wk, wv, wo, bo, H, scale)
    t = lambda a: torch.from_numpy(a.astype(np.float64))
    B, Lq, C = x.shape
    Lk = ctx.shape[1]
    q = (t(x) @ t(wq).T).view(B, Lq, H, C // H).transpose(1, 2)
    k = (t(ctx) @ t(wk).T).view(B, Lk, H, C // H).transpose(1, 2)
    v = (t(ctx) @ t(wv).T).view(B, Lk, H, C // H).transpose(1, 2)
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, scale=scale)
    ref = (o.transpose(1, 2).reshape(B, Lq, C) @ t(wo).T + t(bo)).numpy()
    assert np.max(np.abs(out - ref)) <= 1e-12 * max(1.0, np.abs(ref).max())


def test_attention_block_closed_forms():
    x, ctx, (wq, wk, wv, wo), bo = _blk_inputs(62)
    z = np.zeros_like(wo)
    bf = bo.astype(np.float64)
    assert np.max(np.abs(oracle.attention_block(x, ctx, wq, wk, wv, z, bo, 4, 0.3) - bf)) == 0.0
    assert np.max(np.abs(oracle.attention_block(x, ctx, wq, wk, np.zeros_like(wv), wo, bo, 4, 0.3)
                         - bf)) <= 1e-15
    # one head: the single-head attention of the fp64 projections, then wo
    out1 = oracle.attention_block(x, ctx, wq, wk, wv, wo, None, 1, 0.3)
    q, k, v = (oracle.linear(a, w)[:, None] for a, w in ((x, wq), (ctx, wk), (ctx, wv)))
    o, _, _ = oracle.attention(q, k, v, 0.3)
    ref = oracle.linear(o[:, 0], wo)
    assert np.max(np.abs(out1 - ref)) <= 1e-13


def test_attention_block_rows_subset():
    x, ctx, (wq, wk, wv, wo), bo = _blk_inputs(63)
    full = oracle.attention_block(x, ctx, wq, wk, wv, wo, bo, 2, 0.25)
    rows = np.array([0, 3, 8, 9, 17])
    sub = oracle.attention_block(x, ctx, wq, wk, wv, wo, bo, 2, 0.25, rows=rows)
    assert np.array_equal(sub, full.reshape(-1, full.shape[-1])[rows])


# ---- the specialised kernels of Sec. 3.1: group normalisation (Eq. 1) and GELU
# (Eq. 2) with its split and multiply.  Pinned against torch's fp64 group_norm
# and exact gelu (independent implementations), closed forms and invariants.

def test_group_norm_matches_torch_fp64():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(70)
    for (B, C, H, W, G, eps) in ((2, 32, 5, 7, 8, 1e-5), (1, 12, 4, 4, 3, 1e-6), (3, 6, 1, 1, 6, 1e-5),
                                 (2, 10, 9, 2, 1, 0.0), (1, 64, 3, 3, 32, 1e-5)):
        x = (rng.standard_normal((B, C, H, W)) * 2 + 0.5).astype(np.float16)
        gamma = (1 + 0.3 * rng.standard_normal(C)).astype(np.float16)
        beta = (0.2 * rng.standard_normal(C)).astype(np.float16)
        y, mean, rstd = oracle.group_norm(x, G, gamma, beta, eps)
        e32 = float(np.float32(eps))
        ref = torch.nn.functional.group_norm(torch.from_numpy(x.astype(np.float64)), G,
                                             torch.from_numpy(gamma.astype(np.float64)),
                                             torch.from_numpy(beta.astype(np.float64)), e32).numpy()
        assert np.max(np.abs(y - ref)) <= 1e-12 * max(1.0, np.abs(ref).max()), (B, C, G)
        xg = x.astype(np.float64).reshape(B, G, -1)
        assert np.allclose(mean, xg.mean(axis=2), rtol=0, atol=1e-13)
        assert np.allclose(rstd, 1 / np.sqrt(xg.var(axis=2) + e32), rtol=1e-12, atol=0)


def test_group_norm_closed_forms():
    B, C, HW, G = 2, 8, 6, 4
    # a constant group normalises to zero: the output is beta
    x = np.full((B, C, HW), 3.5, dtype=np.float16)
    beta = np.arange(C, dtype=np.float16) / 4
    y, _, _ = oracle.group_norm(x, G, None, beta, 1e-5)
    assert np.array_equal(y, np.broadcast_to(beta.astype(np.float64)[None, :, None], y.shape))
    # a group of +a and -a in equal numbers: mean 0, variance a^2, so the output
    # is +-a / sqrt(a^2 + eps) (+-1 for eps = 0); a small a makes eps visible
    s = np.where(np.arange(2 * HW) % 2 == 0, 1.0, -1.0).reshape(2, HW)
    for a, eps in ((0.5, 0.0), (2.0 ** -10, 1e-6), (2.0 ** -8, 1e-5)):
        x = np.tile((a * s)[None], (B, G, 1)).astype(np.float16)   # [B, C, HW], 2 channels per group
        y, mean, _ = oracle.group_norm(x, G, None, None, eps)
        e32 = float(np.float32(eps))
        want = a * s / np.sqrt(a * a + e32)
        assert np.allclose(y, np.tile(want[None], (B, G, 1)), rtol=1e-14, atol=0)
        assert np.array_equal(mean, np.zeros((B, G)))


def test_group_norm_invariants():
    rng = np.random.default_rng(71)
    B, C, HW, G = 2, 12, 50, 4
    x = rng.standard_normal((B, C, HW)).astype(np.float16)
    y, _, rstd = oracle.group_norm(x, G, None, None, 1e-5)
    yg = y.reshape(B, G, -1)
    # zero mean and variance var / (var + eps) per group
    var = 1 / rstd ** 2 - float(np.float32(1e-5))
    assert np.max(np.abs(yg.mean(axis=2))) <= 1e-14
    assert np.allclose(yg.var(axis=2), var / (var + float(np.float32(1e-5))), rtol=1e-12)
    # the affine terms act per channel after the normalisation
    gamma = (1 + rng.standard_normal(C)).astype(np.float16)
    beta = rng.standard_normal(C).astype(np.float16)
    ya, _, _ = oracle.group_norm(x, G, gamma, beta, 1e-5)
    want = y * gamma.astype(np.float64)[None, :, None] + beta.astype(np.float64)[None, :, None]
    assert np.max(np.abs(ya - want)) <= 1e-14
    # the groups are consecutive channel blocks: moving one value inside a group
    # changes only that group's outputs
    x2 = x.copy()
    x2[1, 5, 7] += np.float16(3)
    y2, _, _ = oracle.group_norm(x2, G, None, None, 1e-5)
    changed = np.any(y2 != y, axis=2)
    assert changed[1, 3:6].all() and changed.sum() == 3


def test_gelu_known_values_and_identities():
    torch = pytest.importorskip("torch")
    # the standard normal CDF at 1 is 0.841344746068542948... (tables)
    assert abs(oracle.gelu(np.array([1.0]))[0] - 0.8413447460685429) <= 1e-15
    x = np.linspace(-12, 12, 2001)
    g = oracle.gelu(x)
    assert g[1000] == 0.0
    # GELU(x) - GELU(-x) = x
    assert np.max(np.abs(g - g[::-1] - x)) <= 1e-14
    # tails: x for large x, 0 for large -x
    assert abs(g[-1] - 12.0) <= 1e-30 and abs(g[0]) <= 1e-30
    # slope 1/2 at 0
    h = 1e-6
    d = (oracle.gelu(np.array([h]))[0] - oracle.gelu(np.array([-h]))[0]) / (2 * h)
    assert abs(d - 0.5) <= 1e-9
    ref = torch.nn.functional.gelu(torch.from_numpy(x), approximate="none").numpy()
    assert np.max(np.abs(g - ref)) <= 1e-15
    # fp16 and bf16 inputs are widened exactly
    x16 = np.array([-3.5, -0.25, 0.0, 1.0, 6.0], dtype=np.float16)
    assert np.array_equal(oracle.gelu(x16), oracle.gelu(x16.astype(np.float64)))


def test_geglu_split_and_product():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(72)
    h = (rng.standard_normal((3, 5, 2 * 24)) * 2).astype(np.float16)
    out = oracle.geglu(h)
    ht = torch.from_numpy(h.astype(np.float64))
    a, gate = ht.chunk(2, dim=-1)
    ref = (a * torch.nn.functional.gelu(gate, approximate="none")).numpy()
    assert out.shape == (3, 5, 24)
    assert np.max(np.abs(out - ref)) <= 1e-14 * max(1.0, np.abs(ref).max())
    # the first half is the value, the second the gate
    v = np.concatenate([np.ones((4, 6)), rng.standard_normal((4, 6))], axis=1)
    assert np.array_equal(oracle.geglu(v), oracle.gelu(v[:, 6:]))
    big = np.concatenate([rng.standard_normal((4, 6)), np.full((4, 6), 40.0)], axis=1)
    assert np.array_equal(oracle.geglu(big), big[:, :6] * 40.0)   # GELU(40) = 40 in fp64


# ---- the 3x3 convolution of Sec. 3.3 (the oracle is its definition): pinned
# against torch's fp64 conv2d, kernels with a known effect (a centred delta is
# the identity, a corner delta shifts, which fails for a flipped kernel), the
# zero padding (all-ones kernel on a constant map), and linearity.

def test_conv3x3_matches_torch_fp64():
    torch = pytest.importorskip("torch")
    rng = np.random.default_rng(80)
    for (B, Ci, Co, H, W) in ((2, 3, 4, 7, 9), (1, 1, 1, 1, 1), (1, 5, 2, 1, 6), (2, 8, 8, 4, 4)):
        x = rng.standard_normal((B, Ci, H, W)).astype(np.float16)
        w = (rng.standard_normal((Co, Ci, 3, 3)) / 3).astype(np.float16)
        b = rng.standard_normal(Co).astype(np.float16)
        y = oracle.conv3x3(x, w, b)
        t = lambda a: torch.from_numpy(a.astype(np.float64))
        ref = torch.nn.functional.conv2d(t(x), t(w), t(b), padding=1).numpy()
        assert np.max(np.abs(y - ref)) <= 1e-13 * max(1.0, np.abs(ref).max()), (B, Ci, Co, H, W)


def test_conv3x3_known_kernels():
    rng = np.random.default_rng(81)
    x = rng.standard_normal((2, 1, 5, 6)).astype(np.float16)
    xd = x.astype(np.float64)
    delta = np.zeros((1, 1, 3, 3), dtype=np.float16)
    delta[0, 0, 1, 1] = 1
    assert np.array_equal(oracle.conv3x3(x, delta), xd)
    # w[.., 0, 0] = 1 reads the input one row up and one column left
    corner = np.zeros((1, 1, 3, 3), dtype=np.float16)
    corner[0, 0, 0, 0] = 1
    want = np.zeros_like(xd)
    want[..., 1:, 1:] = xd[..., :-1, :-1]
    assert np.array_equal(oracle.conv3x3(x, corner), want)
    # all-ones kernel on a constant map: 9c inside, 6c on the edges, 4c in the corners
    c = np.full((1, 1, 4, 5), 2.0, dtype=np.float16)
    y = oracle.conv3x3(c, np.ones((1, 1, 3, 3), dtype=np.float16))[0, 0]
    assert np.array_equal(y[1:-1, 1:-1], np.full((2, 3), 18.0))
    assert y[0, 0] == y[0, -1] == y[-1, 0] == y[-1, -1] == 8.0
    assert np.array_equal(y[0, 1:-1], np.full(3, 12.0)) and np.array_equal(y[1:-1, 0], np.full(2, 12.0))


def test_conv3x3_linearity_over_channels():
    rng = np.random.default_rng(82)
    x = rng.standard_normal((1, 2, 6, 5))
    w = rng.standard_normal((3, 2, 3, 3))
    both = oracle.conv3x3(x, w)
    parts = oracle.conv3x3(x[:, :1], w[:, :1]) + oracle.conv3x3(x[:, 1:], w[:, 1:])
    assert np.max(np.abs(both - parts)) <= 1e-13
    assert np.max(np.abs(oracle.conv3x3(2.5 * x, w) - 2.5 * both)) <= 1e-12


def test_winograd_table2_closed_forms():
    """Table 2's figures follow from F(m x m, 3 x 3): an m x m output tile costs
    (m + 2)^2 products instead of 9 m^2, the transformed input tile holds
    (m + 2)^2 values for m^2 outputs, and a transformed 3x3 kernel (m + 2)^2
    values for 9.  The paper prints them to two decimals (rounding up twice)."""
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "winograd_table2.txt")
    rows = [list(map(float, l.split())) for l in open(path) if l.strip() and not l.startswith("#")]
    assert [int(r[0]) for r in rows] == [2, 4, 6, 8]
    for m, saving, tensor, weight in rows:
        t = (m + 2) ** 2
        assert abs(9 * m * m / t - saving) <= 0.005, m
        assert abs(t / (m * m) - tensor) <= 0.025, m
        assert abs(t / 9 - weight) <= 0.015, m
