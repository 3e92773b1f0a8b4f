"""The entry points under HIP graph capture (torch.cuda.CUDAGraph): a serving
loop records one call and replays it with new inputs copied into the same
buffers.  Every replay must equal, bit for bit, an eager call on the same
inputs made just before it (the same kernels on the same data), with eager
work and synchronisations between the replays.  The library records no
memory fills or copies, only kernel launches."""
import numpy as np
import pytest
import torch

from paper_2506_08520_amd import binding as B
from paper_2506_08520_amd import workloads as W
from helpers import to_dev

pytestmark = pytest.mark.gpu

# (n_windows, heads, N, d_h, m, dtype, entry): the 64-token kernel, the
# large-window kernel, the token-split path (workspace and static scratch)
CASES = [
    (64, 6, 64, 30, 16, "f32", "ex"),
    (32, 6, 256, 30, 32, "bf16", "ex"),
    (1, 2, 16384, 32, 64, "bf16", "ws"),
    (1, 2, 16384, 32, 16, "f32", "noalloc"),
]


def call(entry, q, k, v, m, out, ws):
    if entry == "ex":
        return B.nystra_attn_forward_ex(q, k, v, m, out=out)
    if entry == "ws":
        return B.nystra_attn_forward_ws(q, k, v, m, workspace=ws, out=out)
    return B.nystra_attn_forward_noalloc(q, k, v, m, out=out)


@pytest.mark.parametrize("case", CASES, ids=lambda c: "x".join(map(str, c)))
def test_graph_replay_matches_eager(case):
    nw, h, N, d, m, dtype, entry = case
    shape = (nw, h, N, d)
    bufs = [to_dev(x, dtype) for x in W.iid(shape, seed=1, dtype=dtype)]
    code = B.F32 if dtype == "f32" else B.BF16
    ws = None
    if entry == "ws":
        nb = B.nystra_attn_workspace_size(nw, h, N, d, m, code)
        ws = torch.empty(nb, dtype=torch.uint8, device="cuda")
    out = torch.empty_like(bufs[0])
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):          # warm-up call outside the capture
        call(entry, *bufs, m, out, ws)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        call(entry, *bufs, m, out, ws)
    torch.cuda.synchronize()
    for rep in range(4):
        new = [to_dev(x, dtype) for x in W.iid(shape, seed=100 + rep, dtype=dtype)]
        for b, x in zip(bufs, new):
            b.copy_(x)
        ref = call(entry, *bufs, m, torch.empty_like(out), ws)   # eager, same inputs
        torch.cuda.synchronize()
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.isfinite(out).all(), f"{case}: replay {rep} left non-finite outputs"
        assert torch.equal(out, ref), f"{case}: replay {rep} differs from the eager call"
