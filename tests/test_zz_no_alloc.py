"""The attention block through the library's static scratch (no workspace,
no allocation) against the same block with a caller workspace: identical
kernels on identical inputs, so identical bits, on two calls in a row with
the second smaller than the first (the workspace block itself is held to the
oracle chain in test_block_gpu.py)."""
import numpy as np
import pytest

import paper_2304_11267_amd as sd
from paper_2304_11267_amd import workloads as wl

from parity_util import to_device

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _needs_gpu():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    sd.load_library()


def _both(case):
    import torch
    x, ctx, wq, wk, wv, wo, bo = (to_device(t) for t in wl.block_inputs(case))
    ws = torch.empty(sd.attention_block_workspace(case.B, case.Lq, case.Lk, case.C), dtype=torch.uint8,
                     device="cuda")
    ref = torch.empty_like(x)
    sd.attention_block(x, ctx, wq, wk, wv, wo, bo, ref, ws, case.H, case.scale)
    got = torch.full_like(x, 7.0)
    sd.attention_block_static(x, ctx, wq, wk, wv, wo, bo, got, case.H, case.scale)
    torch.cuda.synchronize()
    return ref, got


def test_static_scratch_block_matches_workspace_block_twice():
    import torch
    # the 64x64-level self block (21 MB of scratch), then the smaller 16x16-level cross block
    for name in ("blk64_self", "blk16_cross"):
        ref, got = _both(wl.BLOCK_CASES[name])
        assert torch.equal(ref, got), name


def test_static_scratch_refuses_what_does_not_fit():
    import torch
    x = torch.zeros(4, 4096, 320, dtype=torch.float16, device="cuda")
    w = torch.zeros(320, 320, dtype=torch.float16, device="cuda")
    out = torch.empty_like(x)
    with pytest.raises(sd.SdattnError) as e:
        sd.attention_block_static(x, x, w, w, w, w, None, out, 8, 0.158)
    assert e.value.status == sd.STATUS_SCRATCH
