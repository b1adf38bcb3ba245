"""The backward by stages (sparse_attn_bwd_stage): row statistics, dQ and
dK / dV as three calls give sparse_attn_bwd's results bit for bit, on the
block path, the fixed pattern whose dQ stage recomputes D, and the strided
path by residue classes (band and classes in each stage)."""
import pytest
import torch

from paper_1904_10509_amd import sparse_attn as sa
from paper_1904_10509_amd.inputs import make_inputs

from gpu_util import device

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("pattern,mode,n,B,l,c,d", [
    (sa.SA_FIXED, sa.SA_MODE_MERGED, 2048, 64, 256, 32, 64),   # block path
    (sa.SA_FIXED, sa.SA_MODE_A2, 512, 64, 64, 1, 64),          # D recomputed in the dQ stage
    (sa.SA_STRIDED, sa.SA_MODE_MERGED, 2048, 64, 64, 0, 64),   # band + classes
    (sa.SA_STRIDED, sa.SA_MODE_A2, 1024, 32, 32, 0, 128),      # classes alone
])
def test_stages_equal_whole_backward(pattern, mode, n, B, l, c, d):
    dev = device()
    x = make_inputs(2, 3, n, d, torch.bfloat16, seed=n + l + d)
    q, k, v, dout = (x[name].to(dev) for name in ("q", "k", "v", "dout"))
    lay = sa.build_layout(n, B, l, c, pattern, mode, device=dev)
    o, lse = sa.forward(q, k, v, lay)
    want = sa.backward(q, k, v, o, dout, lse, lay)
    got = tuple(torch.full_like(q, float("nan")) for _ in range(3))
    ws = torch.empty(sa.sparse_attn_bwd_workspace_size(*lay.pattern_args, 2, 3, d, sa.SA_BF16), dtype=torch.uint8,
                     device=dev)
    for st in (sa.SA_BWD_ROW_STATS, sa.SA_BWD_DQ, sa.SA_BWD_DKDV):
        sa.backward(q, k, v, o, dout, lse, lay, grads=got, workspace=ws, stages=st)
    torch.cuda.synchronize()
    for name, g, w in zip(("dq", "dk", "dv"), got, want):
        assert torch.equal(g, w), name
