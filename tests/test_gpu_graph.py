"""The library's calls captured in a HIP graph (torch.cuda.CUDAGraph): every
replay, with eager work and synchronisations in between, must give the eager
results bit for bit (the kernels write every output element exactly once, in
a fixed order, so the results are deterministic)."""
import pytest
import torch

from paper_1904_10509_amd import sparse_attn as sa
from paper_1904_10509_amd.inputs import make_inputs

from gpu_util import device

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("pattern,n,B,l,c", [(sa.SA_STRIDED, 2048, 64, 128, 0), (sa.SA_FIXED, 2048, 64, 256, 32)])
def test_graph_replays_match_eager(pattern, n, B, l, c):
    dev = device()
    x = make_inputs(2, 4, n, 64, torch.bfloat16, seed=n + l)
    q, k, v, dout = (x[name].to(dev) for name in ("q", "k", "v", "dout"))
    lay = sa.build_layout(n, B, l, c, pattern, sa.SA_MODE_MERGED, device=dev)
    o = torch.empty_like(q)
    lse = torch.empty(q.shape[:3], dtype=torch.float32, device=dev)
    grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v))
    ws = torch.empty(sa.sparse_attn_bwd_workspace_size(*lay.pattern_args, 2, 4, 64, sa.SA_BF16), dtype=torch.uint8,
                     device=dev)

    def step():
        sa.forward(q, k, v, lay, out=o, lse=lse)
        sa.backward(q, k, v, o, dout, lse, lay, grads=grads, workspace=ws)

    side = torch.cuda.Stream(device=dev)
    side.wait_stream(torch.cuda.current_stream(dev))
    with torch.cuda.stream(side):
        step()  # eager, on the stream the graph is captured from
    torch.cuda.current_stream(dev).wait_stream(side)
    torch.cuda.synchronize()
    ref = [t.clone() for t in (o, lse) + grads]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(3):
        for t in (o, lse) + grads:
            t.fill_(float("nan"))  # eager work between replays; the replay must overwrite it all
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, got, want in zip(("o", "lse", "dq", "dk", "dv"), (o, lse) + grads, ref):
            assert torch.equal(got, want), (rep, name)
