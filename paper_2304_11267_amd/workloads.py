"""Seeded synthetic inputs at the shapes of SD1.4's UNet attention.

This module builds inputs only; it holds none of the attention arithmetic, so
both the HIP path's tests and the fp64 oracle can draw from it.

The paper's workload is the UNet of Stable Diffusion 1.4 generating a 512x512
image (Sec. 4), i.e. a 64x64 latent (Sec. 3, image decoder).  Its attention
runs over the latent grid (self-attention, Lq = Lk = h*w tokens) and over the
text embedding tau_theta(y) (cross-attention, Sec. 3, denoising network).
Trained weights and CLIP embeddings are not available, so N(0, 1) tensors of
the same shapes stand in for the projected Q, K and V: batch 2 (classifier-free
guidance: conditional and unconditional), 8 heads, head width 40/80/160/160 at
the 64/32/16/8 latent levels, and a 77-token text context.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

SEED0 = 230411267
BATCH = 2
HEADS = 8
TEXT_TOKENS = 77

# latent side -> (tokens, head width) of SD1.4's transformer blocks
LEVELS = {64: (4096, 40), 32: (1024, 80), 16: (256, 160), 8: (64, 160)}

# the 16 transformer blocks of one UNet evaluation, in execution order
UNET_BLOCKS = ([("down", 64)] * 2 + [("down", 32)] * 2 + [("down", 16)] * 2 +
               [("mid", 8)] + [("up", 16)] * 3 + [("up", 32)] * 3 + [("up", 64)] * 3)
DENOISE_STEPS = 20


@dataclass(frozen=True)
class Case:
    name: str
    B: int
    H: int
    Lq: int
    Lk: int
    D: int
    seed: int
    q_mult: float = 1.0  # the peaked variant multiplies Q by 4 (exact in fp16)

    @property
    def scale(self) -> float:
        """1/sqrt(d) with the true head width d, rounded to fp32."""
        return float(np.float32(1.0 / np.sqrt(self.D)))

    @property
    def flops(self) -> int:
        """Useful flops: 2*Lk*D for Q K^T plus 2*Lk*D for P V, per query row."""
        return 4 * self.B * self.H * self.Lq * self.Lk * self.D

    @property
    def bytes(self) -> int:
        """Algorithmic HBM bytes: Q, K, V read once and O written once (2-byte elements)."""
        return 2 * self.B * self.H * self.D * 2 * (self.Lq + self.Lk)


# The parity and benchmark cases (batch 2 for classifier-free guidance, 8 heads).
CASES = {
    "mid8_self": Case("mid8_self", BATCH, HEADS, 64, 64, 160, SEED0 + 1),
    "mid8_cross": Case("mid8_cross", BATCH, HEADS, 64, TEXT_TOKENS, 160, SEED0 + 11),
    "l16_self": Case("l16_self", BATCH, HEADS, 256, 256, 160, SEED0 + 2),
    "l16_self_peaked": Case("l16_self_peaked", BATCH, HEADS, 256, 256, 160, SEED0 + 2, 4.0),
    "l16_cross": Case("l16_cross", BATCH, HEADS, 256, TEXT_TOKENS, 160, SEED0 + 12),
    "l32_self": Case("l32_self", BATCH, HEADS, 1024, 1024, 80, SEED0 + 3),
    "l32_cross": Case("l32_cross", BATCH, HEADS, 1024, TEXT_TOKENS, 80, SEED0 + 13),
    "l64_self": Case("l64_self", BATCH, HEADS, 4096, 4096, 40, SEED0 + 4),
    "l64_cross": Case("l64_cross", BATCH, HEADS, 4096, TEXT_TOKENS, 40, SEED0 + 14),
}


def sweep_cases(step: int):
    """The 32 attention calls of one UNet evaluation at denoising step `step`.

    Block b does self-attention (seed S0 + 1000*(step+1) + 10*b) and then
    cross-attention over the text context (same seed + 1).
    """
    out = []
    for b, (where, side) in enumerate(UNET_BLOCKS):
        L, D = LEVELS[side]
        base = SEED0 + 1000 * (step + 1) + 10 * b
        out.append(Case(f"s{step}_b{b}_{where}{side}_self", BATCH, HEADS, L, L, D, base))
        out.append(Case(f"s{step}_b{b}_{where}{side}_cross", BATCH, HEADS, L, TEXT_TOKENS, D, base + 1))
    return out


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (nearest, ties to even); uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def make_qkv(B, H, Lq, Lk, D, seed, dtype="f16", q_mult=1.0):
    """Draw Q, then K, then V ~ N(0, 1) in float32 from numpy's default_rng(seed).

    dtype "f16": float16 arrays (round to nearest even).
    dtype "bf16": uint16 arrays holding bfloat16 bit patterns.
    q_mult multiplies Q after rounding (use a power of two to stay exact).
    """
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((B, H, Lq, D), dtype=np.float32)
    k = rng.standard_normal((B, H, Lk, D), dtype=np.float32)
    v = rng.standard_normal((B, H, Lk, D), dtype=np.float32)
    if dtype == "f16":
        q, k, v = (t.astype(np.float16) for t in (q, k, v))
        if q_mult != 1.0:
            q = (q.astype(np.float32) * np.float32(q_mult)).astype(np.float16)
        return q, k, v
    if dtype == "bf16":
        if q_mult != 1.0:
            q = q * np.float32(q_mult)
        return to_bf16_bits(q), to_bf16_bits(k), to_bf16_bits(v)
    raise ValueError(f"unknown dtype {dtype!r}")


def case_inputs(case: Case, dtype="f16"):
    return make_qkv(case.B, case.H, case.Lq, case.Lk, case.D, case.seed, dtype, case.q_mult)


def make_matrix(rows, cols, seed, dtype="f16", sigma=1.0):
    """A [rows, cols] matrix ~ N(0, sigma^2) standing in for A = Q K^T."""
    rng = np.random.default_rng(seed)
    a = rng.standard_normal((rows, cols), dtype=np.float32) * np.float32(sigma)
    if dtype == "f16":
        return a.astype(np.float16)
    if dtype == "f32":
        return a
    if dtype == "bf16":
        return to_bf16_bits(a)
    raise ValueError(f"unknown dtype {dtype!r}")


def sample_rows(B, H, Lq, per_head, seed):
    """Flat query-row indices: `per_head` distinct random rows of every (b, h),
    always including the first and last row of each head."""
    rng = np.random.default_rng(seed)
    out = []
    for bh in range(B * H):
        k = min(per_head, Lq)
        pick = set(rng.choice(Lq, size=k, replace=False).tolist())
        pick.update({0, Lq - 1})
        out.extend(bh * Lq + i for i in sorted(pick))
    return np.asarray(out, dtype=np.int64)


# SD1.4's attention blocks around Eq. 3: channels C = H * D per level, the
# text context of CLIP ViT-L/14 (77 tokens x 768 channels) for cross-attention.
CONTEXT_CHANNELS = 768


@dataclass(frozen=True)
class BlockCase:
    name: str
    B: int
    Lq: int
    Lk: int
    C: int          # latent channels (H heads of D)
    Cc: int         # context channels (C for self-attention)
    H: int
    seed: int
    self_attn: bool

    @property
    def D(self) -> int:
        return self.C // self.H

    @property
    def scale(self) -> float:
        return float(np.float32(1.0 / np.sqrt(self.D)))

    @property
    def flops(self) -> int:
        """Algorithmic flops: four projections (2 per multiply-add) and Eq. 3."""
        proj = 2 * self.B * (self.Lq * self.C * self.C * 2 + self.Lk * self.Cc * self.C * 2)
        return proj + 4 * self.B * self.H * self.Lq * self.Lk * self.D


def _block(name, level, self_attn, seed):
    L, D = LEVELS[level]
    C = HEADS * D
    return BlockCase(name, BATCH, L, L if self_attn else TEXT_TOKENS, C,
                     C if self_attn else CONTEXT_CHANNELS, HEADS, seed, self_attn)


BLOCK_CASES = {
    "blk64_self": _block("blk64_self", 64, True, SEED0 + 21),
    "blk64_cross": _block("blk64_cross", 64, False, SEED0 + 22),
    "blk32_self": _block("blk32_self", 32, True, SEED0 + 23),
    "blk16_cross": _block("blk16_cross", 16, False, SEED0 + 24),
}


def make_block(B, Lq, Lk, C, Cc, seed, self_attn=False, dtype="f16"):
    """Draw x [B,Lq,C], ctx [B,Lk,Cc] (x itself for self-attention), then wq, wk,
    wv, wo (weights [out, in]) and bo, in that order, from default_rng(seed) in
    float32: tokens ~ N(0, 1), weights ~ N(0, 1/fan_in), bias ~ N(0, 0.01).
    Returns (x, ctx, wq, wk, wv, wo, bo) as float16 (or bf16 bit patterns)."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((B, Lq, C), dtype=np.float32)
    ctx = x if self_attn else rng.standard_normal((B, Lk, Cc), dtype=np.float32)
    ws = [rng.standard_normal((C, fan), dtype=np.float32) / np.float32(np.sqrt(fan))
          for fan in (C, Cc, Cc, C)]
    bo = rng.standard_normal(C, dtype=np.float32) * np.float32(0.1)
    out = [x, ctx, *ws, bo]
    if dtype == "f16":
        return tuple(t.astype(np.float16) for t in out)
    if dtype == "bf16":
        return tuple(to_bf16_bits(t) for t in out)
    raise ValueError(f"unknown dtype {dtype!r}")


def block_inputs(case: BlockCase, dtype="f16"):
    return make_block(case.B, case.Lq, case.Lk, case.C, case.Cc, case.seed, case.self_attn, dtype)


# Group normalisation and the gated feed-forward around the transformer
# blocks (Sec. 3.1): SD1.4's feature maps per level (channels x pixels), 32
# groups; the feed-forward's inner width is 4C, so GEGLU's input has 8C columns.
GN_GROUPS = 32
GN_EPS = 1e-5


@dataclass(frozen=True)
class NormCase:
    name: str
    B: int
    C: int
    HW: int
    seed: int

    @property
    def bytes(self) -> int:
        """Algorithmic HBM bytes: x read once, y written once (2-byte elements)."""
        return 2 * 2 * self.B * self.C * self.HW


@dataclass(frozen=True)
class GegluCase:
    name: str
    M: int          # token rows (B * L)
    F: int          # output width (4C)
    seed: int

    @property
    def bytes(self) -> int:
        """h read once (2F per row), out written once (F per row), 2-byte elements."""
        return 2 * 3 * self.M * self.F


NORM_CASES = {
    "gn64": NormCase("gn64", BATCH, 320, 4096, SEED0 + 31),
    "gn32": NormCase("gn32", BATCH, 640, 1024, SEED0 + 32),
    "gn16": NormCase("gn16", BATCH, 1280, 256, SEED0 + 33),
    "gn8": NormCase("gn8", BATCH, 1280, 64, SEED0 + 34),
    "gn32_cat": NormCase("gn32_cat", BATCH, 960, 1024, SEED0 + 35),   # decoder concat width
}

GEGLU_CASES = {
    "geglu64": GegluCase("geglu64", BATCH * 4096, 1280, SEED0 + 41),
    "geglu32": GegluCase("geglu32", BATCH * 1024, 2560, SEED0 + 42),
    "geglu16": GegluCase("geglu16", BATCH * 256, 5120, SEED0 + 43),
}


def _cast(a, dtype):
    if dtype == "f16":
        return a.astype(np.float16)
    if dtype == "bf16":
        return to_bf16_bits(a)
    raise ValueError(f"unknown dtype {dtype!r}")


def make_norm(B, C, HW, seed, dtype="f16"):
    """x [B, C, HW] with per-channel offsets and scales (x = m_c + s_c z, z ~ N(0,1),
    m_c ~ N(0, 1), s_c ~ U(0.2, 2)), then gamma ~ 1 + 0.2 N(0,1), beta ~ 0.2 N(0,1),
    drawn in that order from default_rng(seed) in float32."""
    rng = np.random.default_rng(seed)
    m = rng.standard_normal((1, C, 1), dtype=np.float32)
    s = rng.uniform(0.2, 2.0, size=(1, C, 1)).astype(np.float32)
    x = m + s * rng.standard_normal((B, C, HW), dtype=np.float32)
    gamma = 1 + 0.2 * rng.standard_normal(C, dtype=np.float32)
    beta = 0.2 * rng.standard_normal(C, dtype=np.float32)
    return tuple(_cast(t, dtype) for t in (x, gamma, beta))


def norm_inputs(case: NormCase, dtype="f16"):
    return make_norm(case.B, case.C, case.HW, case.seed, dtype)


def make_geglu(M, F, seed, dtype="f16", sigma=1.5):
    """h [M, 2F] ~ N(0, sigma^2) from default_rng(seed) in float32."""
    rng = np.random.default_rng(seed)
    return _cast(rng.standard_normal((M, 2 * F), dtype=np.float32) * np.float32(sigma), dtype)


def geglu_inputs(case: GegluCase, dtype="f16"):
    return make_geglu(case.M, case.F, case.seed, dtype)


# The UNet's 3x3 convolutions (Sec. 3.3): C -> C channels at each latent level.
CONV_LEVELS = {64: 320, 32: 640, 16: 1280, 8: 1280}


def make_conv(B, Ci, Co, H, W, seed, dtype="f16"):
    """x [B, Ci, H, W] ~ N(0, 1), w [Co, Ci, 3, 3] ~ N(0, 1/(9 Ci)), bias ~ N(0, 0.1^2),
    drawn in that order from default_rng(seed) in float32."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((B, Ci, H, W), dtype=np.float32)
    w = rng.standard_normal((Co, Ci, 3, 3), dtype=np.float32) / np.float32(np.sqrt(9 * Ci))
    b = rng.standard_normal(Co, dtype=np.float32) * np.float32(0.1)
    return tuple(_cast(t, dtype) for t in (x, w, b))
