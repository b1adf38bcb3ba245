"""sparse_attn_bwd_noalloc (the backward without a caller workspace, for
callers that cannot allocate) through the C ABI: two calls in a row, the
second on a smaller input, each bit for bit equal to sparse_attn_bwd with a
caller workspace on the same inputs, and within the parity bar of the fp64
oracle."""
import pytest
import torch

from oracle import oracle as orc_mod
from paper_1904_10509_amd import sparse_attn as sa
from paper_1904_10509_amd.inputs import make_inputs

from gpu_util import check_all, device, oracle_inputs, to64

pytestmark = pytest.mark.gpu


def run_case(pattern, mode, n, B, l, c, d, batch, heads, seed):
    dev = device()
    x = make_inputs(batch, heads, n, d, torch.bfloat16, seed=seed)
    q, k, v, dout = (x[name].to(dev) for name in ("q", "k", "v", "dout"))
    scale = d ** -0.5
    lay = sa.build_layout(n, B, l, c, pattern, mode, device=dev)
    o, lse = sa.forward(q, k, v, lay, scale)
    want = sa.backward(q, k, v, o, dout, lse, lay, scale)
    got = tuple(torch.full_like(q, float("nan")) for _ in range(3))
    strides = sa._strides(q, k, v, o, dout, *got)
    sa.sparse_attn_bwd_noalloc(*lay.pattern_args, *lay.row_args, *lay.col_args, batch, heads, d, sa.SA_BF16,
                               q, k, v, o, dout, lse, strides, scale, *got)
    torch.cuda.synchronize()
    for name, g, w in zip(("dq", "dk", "dv"), got, want):
        assert torch.equal(g, w), name
    ref = orc_mod.backward(*oracle_inputs(x), pattern=pattern, mode=mode, l=l, c=c, scale=scale)
    check_all(f"noalloc p{pattern} m{mode} n{n} {batch}x{heads}",
              {"dq": to64(got[0]), "dk": to64(got[1]), "dv": to64(got[2])}, ref, torch.bfloat16,
              names=("dq", "dk", "dv"))


def test_noalloc_two_calls_second_smaller():
    assert sa.sparse_attn_bwd_noalloc_max_workspace() == 64 << 20
    # fixed pattern, 2 x 4 heads of 64 over 4,096 positions; then smaller calls
    # on the same scratch: one whose products are split in two parts (c = 1),
    # one of the strided pattern
    run_case(sa.SA_FIXED, sa.SA_MODE_MERGED, 4096, 64, 256, 32, 64, 2, 4, seed=71)
    run_case(sa.SA_FIXED, sa.SA_MODE_A2, 512, 64, 64, 1, 64, 1, 8, seed=72)
    run_case(sa.SA_STRIDED, sa.SA_MODE_MERGED, 256, 32, 32, 0, 32, 1, 2, seed=73)
