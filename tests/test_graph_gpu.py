"""HIP graph capture of the library's launches.  Every forward path (the tiled
kernel in its 256- and 64-row geometries (the latter with two and with four
key splits), with and without the Eq. 4
statistics, the short-key kernel, the general kernel, bf16) and the
no-allocation attention block record into a graph -- nothing in them
allocates, clears memory or synchronises -- and every replay reproduces the
eager result bit for bit, with eager work and synchronisations between the
replays."""
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


def _replays_match(record, outputs, reps=3):
    """Run `record` eagerly (reference), capture it in a graph, then replay
    `reps` times: outputs cleared by eager work before each replay, each
    replay checked against the reference."""
    import torch
    record(torch.cuda.current_stream())
    torch.cuda.synchronize()
    ref = [o.clone() for o in outputs]
    side = torch.cuda.Stream()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        record(torch.cuda.current_stream())
    for _ in range(reps):
        for o in outputs:
            o.fill_(3.0)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for r, o in zip(ref, outputs):
            assert torch.equal(r, o)


# (B, H, Lq, Lk, D, dtype, with statistics)
FORWARD_CASES = [
    (2, 8, 4096, 4096, 40, "f16", False),   # 256-row workgroups, 128-key tiles
    (1, 2, 300, 333, 40, "f16", True),      # 128-row workgroups with (L, S), ragged tiles
    (2, 8, 1024, 1024, 80, "f16", False),   # 64-row workgroups, keys split four ways
    (2, 8, 1024, 300, 80, "f16", False),    # 64-row workgroups, two key halves
    (2, 8, 4096, 77, 40, "f16", False),     # short-key kernel
    (1, 3, 70, 90, 16, "f16", False),       # general kernel
    (1, 2, 200, 260, 64, "bf16", True),
]


@pytest.mark.parametrize("case", FORWARD_CASES, ids=lambda c: "B{}H{}q{}k{}D{}{}{}".format(
    *c[:6], "_stats" if c[6] else ""))
def test_forward_graph_replays_match_eager(case):
    import torch
    B, H, Lq, Lk, D, dtype, stats = case
    q, k, v = (to_device(t, dtype) for t in wl.make_qkv(B, H, Lq, Lk, D, 9100 + Lq + D, dtype=dtype))
    out = torch.empty_like(q)
    scale = 1.0 / D ** 0.5
    if stats:
        ls = torch.empty(B, H, Lq, 2, dtype=torch.float32, device="cuda")
        _replays_match(lambda s: sd.forward_ex(q, k, v, out, scale, ls=ls, stream=s), [out, ls])
    else:
        _replays_match(lambda s: sd.forward(q, k, v, out, scale, stream=s), [out])


def test_static_block_graph_replays_match_eager():
    import torch
    case = wl.BLOCK_CASES["blk64_self"]
    x, ctx, wq, wk, wv, wo, bo = (to_device(t) for t in wl.block_inputs(case))
    out = torch.empty_like(x)
    _replays_match(lambda s: sd.attention_block_static(x, ctx, wq, wk, wv, wo, bo, out, case.H, case.scale,
                                                       stream=s), [out])
