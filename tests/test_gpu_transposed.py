"""GPU parity of strided A2 computed by transposition (Sec. 5.5): per residue
class, dense causal attention through the same entry points on strided views,
against the fp64 oracle's strided A2 (mode A2) on the same inputs."""
import numpy as np
import pytest
import torch

from oracle import oracle as orc_mod
from paper_1904_10509_amd import sparse_attn as sa
from paper_1904_10509_amd.inputs import make_inputs

from gpu_util import check, check_all, check_lse, device, oracle_inputs, to64

pytestmark = pytest.mark.gpu

# (n, l, block of the class layout, d, dtype, batch, heads)
CASES = [
    (512, 16, 32, 64, torch.float32, 1, 2),
    (2048, 64, 32, 64, torch.bfloat16, 2, 2),
    (4096, 32, 64, 128, torch.bfloat16, 1, 2),
    (1536, 16, 32, 32, torch.bfloat16, 1, 3),
    (12288, 128, 32, 64, torch.bfloat16, 2, 8),  # the text workload's shape: classes of 96
]


@pytest.mark.parametrize("n,l,B,d,dtype,batch,heads", CASES)
def test_transposed_a2_matches_oracle(n, l, B, d, dtype, batch, heads):
    dev = device()
    x = make_inputs(batch, heads, n, d, dtype, seed=n + l + B + d)
    q, k, v, dout = (x[name].to(dev) for name in ("q", "k", "v", "dout"))
    scale = d ** -0.5
    lay = sa.transposed_a2_layout(n, l, B, device=dev)
    o, lse_cls = sa.forward_a2_transposed(q, k, v, l, lay, scale)
    dq, dk, dv = sa.backward_a2_transposed(q, k, v, o, dout, lse_cls, l, lay, scale)
    torch.cuda.synchronize()
    # class order [b*h, l, n/l] back to [b, h, n] (i = m l + r)
    lse = lse_cls.reshape(batch, heads, l, n // l).transpose(2, 3).reshape(batch, heads, n)
    ref = orc_mod.backward(*oracle_inputs(x), pattern=sa.SA_STRIDED, mode=sa.SA_MODE_A2, l=l, c=0, scale=scale)
    got = {"o": to64(o), "lse": to64(lse), "dq": to64(dq), "dk": to64(dk), "dv": to64(dv)}
    check_all(f"transposed A2 n{n} l{l} B{B} d{d}", got, ref, dtype, names=("o", "lse", "dq", "dk", "dv"))


def test_transposed_a2_equals_block_path_closely():
    """Same inputs through the block-sparse strided A2 kernels: both results
    within the bf16 tolerance of each other (the two round P differently)."""
    dev = device()
    n, l, d = 4096, 64, 64
    x = make_inputs(1, 4, n, d, torch.bfloat16, seed=11)
    q, k, v = (x[name].to(dev) for name in ("q", "k", "v"))
    o_t, _ = sa.forward_a2_transposed(q, k, v, l, sa.transposed_a2_layout(n, l, 64, device=dev))
    o_b, _ = sa.forward(q, k, v, sa.build_layout(n, 64, l, 0, sa.SA_STRIDED, sa.SA_MODE_A2, device=dev))
    torch.cuda.synchronize()
    check("transposed A2 against block A2", to64(o_t), to64(o_b), torch.bfloat16)


# Merged strided heads (A1 u A2) with A2 by transposition: the band through the
# strided A1 layout, the rest ({i - k l : k >= 2}) per residue class, merged
# through their log-sum-exps, against the oracle's merged strided pattern.
# (n, l, band block, class block, d, dtype, batch, heads)
MERGED_CASES = [
    (512, 16, 16, 32, 64, torch.float32, 1, 2),
    (1024, 16, 32, 16, 32, torch.bfloat16, 1, 3),
    (2048, 64, 64, 32, 64, torch.bfloat16, 2, 2),
    (4096, 64, 64, 64, 128, torch.bfloat16, 1, 2),
    (4096, 256, 64, 16, 64, torch.bfloat16, 1, 2),  # 16 positions per class: one class block
    (1600, 25, 16, 32, 64, torch.bfloat16, 1, 2),   # a stride that is not a multiple of the block
    (512, 8, 16, 64, 128, torch.float32, 2, 1),
    (256, 1, 16, 64, 32, torch.bfloat16, 1, 2),     # l = 1: one class, the whole sequence
]


def run_merged(x, n, l, B, CB, scale, dev):
    q, k, v, dout = (x[name].to(dev) for name in ("q", "k", "v", "dout"))
    band = sa.band_layout(n, B, l, device=dev)
    o, lse = sa.forward_merged_transposed(q, k, v, band, CB, scale)
    dq, dk, dv = sa.backward_merged_transposed(q, k, v, o, dout, lse, band, CB, scale)
    torch.cuda.synchronize()
    return {"o": to64(o), "lse": to64(lse), "dq": to64(dq), "dk": to64(dk), "dv": to64(dv)}


@pytest.mark.parametrize("n,l,B,CB,d,dtype,batch,heads", MERGED_CASES)
def test_merged_transposed_matches_oracle(n, l, B, CB, d, dtype, batch, heads):
    dev = device()
    x = make_inputs(batch, heads, n, d, dtype, seed=n + l + CB + d + 3)
    scale = d ** -0.5
    got = run_merged(x, n, l, B, CB, scale, dev)
    ref = orc_mod.backward(*oracle_inputs(x), pattern=sa.SA_STRIDED, mode=sa.SA_MODE_MERGED, l=l, c=0, scale=scale)
    check_all(f"transposed merged n{n} l{l} B{B} CB{CB} d{d}", got, ref, dtype, names=("o", "lse", "dq", "dk", "dv"))


def test_merged_transposed_text_workload_sampled():
    """The text workload (12,288 positions, l = 128, 2 x 8 heads of 64): sampled
    rows and columns against the oracle, and all outputs against the block
    path over the merged layout within the bf16 tolerance."""
    from paper_1904_10509_amd.inputs import WORKLOADS, workload_inputs
    from gpu_util import run_gpu
    dev = device()
    w = WORKLOADS["strided_n12288_l128_merged"]
    x = workload_inputs(w)
    got = run_merged(x, w.n, w.stride, w.block, 32, w.scale, dev)
    blk = run_gpu(x, n=w.n, block=w.block, l=w.stride, c=0, pattern=w.pattern, mode=w.mode, scale=w.scale)
    check_all("transposed merged text against merged layout", got, blk, torch.bfloat16,
              names=("o", "lse", "dq", "dk", "dv"))
    rng = np.random.default_rng(5)
    idx = [0, 1, 127, 128, 129, 255, 256, 257, 6000, w.n - 1] + list(rng.integers(0, w.n, 30))
    sel = np.stack([rng.integers(0, w.batch, len(idx)), rng.integers(0, w.heads, len(idx)), np.array(idx)], axis=1)
    xi = oracle_inputs(x)
    kw = dict(pattern=w.pattern, mode=w.mode, l=w.stride, c=0, scale=w.scale)
    o, lse = orc_mod.forward_rows(*xi[:3], sel, **kw)
    dq = orc_mod.backward_rows(*xi, sel, **kw)
    dk, dv = orc_mod.backward_cols(*xi, sel, **kw)
    r = (sel[:, 0], sel[:, 1], sel[:, 2])
    bf = torch.bfloat16
    check("transposed merged text o rows", got["o"][r], o, bf)
    check_lse("transposed merged text lse rows", got["lse"][r], lse, bf)
    check("transposed merged text dq rows", got["dq"][r], dq, bf)
    check("transposed merged text dk cols", got["dk"][r], dk, bf)
    check("transposed merged text dv cols", got["dv"][r], dv, bf)


def test_merged_transposed_autograd_wrapper():
    dev = device()
    n, l, B, CB, d = 1024, 32, 32, 32, 64
    x = make_inputs(1, 2, n, d, torch.bfloat16, seed=27)
    band = sa.band_layout(n, B, l, device=dev)
    q, k, v = (x[name].to(dev).requires_grad_(True) for name in ("q", "k", "v"))
    o = sa.SparseAttentionTransposed.apply(q, k, v, band, CB, None)
    (o.float() * x["dout"].to(dev).float()).sum().backward()
    ref = orc_mod.backward(*oracle_inputs(x), pattern=sa.SA_STRIDED, mode=sa.SA_MODE_MERGED, l=l, c=0,
                           scale=d ** -0.5)
    check("transposed autograd o", to64(o), ref["o"], torch.bfloat16)
    for name, t in (("dq", q), ("dk", k), ("dv", v)):
        check(f"transposed autograd {name}", to64(t.grad), ref[name], torch.bfloat16)


def test_merged_transposed_n1048576_sampled():
    """The audio shape (1,048,576 positions, l = 1,024, 4 heads of 64, classes
    of 1,024 in blocks of 64): sampled rows and columns against the oracle's
    merged strided pattern, gathered on the device."""
    from paper_1904_10509_amd.inputs import WORKLOADS, workload_inputs
    w = WORKLOADS["strided_n1048576_l1024_merged"]
    dev = device()
    x = workload_inputs(w)
    q, k, v, dout = (x[name].to(dev) for name in ("q", "k", "v", "dout"))
    band = sa.band_layout(w.n, w.block, w.stride, device=dev)
    o, lse = sa.forward_merged_transposed(q, k, v, band, 64, w.scale)
    dq, dk, dv = sa.backward_merged_transposed(q, k, v, o, dout, lse, band, 64, w.scale)
    torch.cuda.synchronize()
    for t in (o, dq, dk, dv):
        assert bool(torch.isfinite(t).all())
    rng = np.random.default_rng(w.seed + 1)
    idx = [0, 1, 1023, 1024, 2047, 2048, 2049, 3072, w.n // 2, w.n - 1] + list(rng.integers(0, w.n, 22))
    sel = np.stack([rng.integers(0, w.batch, len(idx)), rng.integers(0, w.heads, len(idx)), np.array(idx)], axis=1)

    def gather(t):
        ix = torch.as_tensor(sel, device=dev)
        return to64(t[ix[:, 0], ix[:, 1], ix[:, 2]])

    xi = oracle_inputs(x)
    kw = dict(pattern=w.pattern, mode=w.mode, l=w.stride, c=0, scale=w.scale)
    o_ref, lse_ref = orc_mod.forward_rows(*xi[:3], sel, **kw)
    dq_ref = orc_mod.backward_rows(*xi, sel, **kw)
    dk_ref, dv_ref = orc_mod.backward_cols(*xi, sel, **kw)
    bf = torch.bfloat16
    check("transposed merged n1048576 o rows", gather(o), o_ref, bf)
    check_lse("transposed merged n1048576 lse rows", gather(lse), lse_ref, bf)
    check("transposed merged n1048576 dq rows", gather(dq), dq_ref, bf)
    check("transposed merged n1048576 dk cols", gather(dk), dk_ref, bf)
    check("transposed merged n1048576 dv cols", gather(dv), dv_ref, bf)
