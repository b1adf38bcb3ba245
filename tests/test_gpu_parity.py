"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Layouts must match bitwise.  Outputs and gradients must match the fp64
oracle on the same inputs elementwise within the tolerance of the element
type plus half an ulp of the stored output (tests/gpu_util.py): 1e-5 for fp32
and 2e-2 for bf16 on O, dQ, dK, dV, and 1e-5 / 1e-3 on the fp32 LSE.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as orc_mod
from paper_1904_10509_amd import sparse_attn as sa
from paper_1904_10509_amd.inputs import WORKLOADS, make_inputs, workload_inputs

from gpu_util import check, check_all, check_lse, device, oracle_inputs, run_gpu, to64

pytestmark = pytest.mark.gpu

S, F, P = sa.SA_STRIDED, sa.SA_FIXED, sa.SA_FIXED_PER_HEAD
A1, A2, MG, IL = sa.SA_MODE_A1, sa.SA_MODE_A2, sa.SA_MODE_MERGED, sa.SA_MODE_INTERLEAVED


def layout_to_cpu(lay):
    return {k: getattr(lay, k).cpu().numpy() for k in ("row_ptr", "col_idx", "kind", "col_ptr", "row_idx", "kind_t")}


LAYOUT_CASES = [
    (S, 256, 16, 16, 0), (S, 256, 16, 24, 0), (S, 192, 32, 7, 0), (S, 128, 16, 1, 0), (S, 128, 32, 500, 0),
    (S, 64, 64, 9, 0), (S, 384, 64, 128, 0), (F, 256, 16, 32, 8), (F, 256, 32, 32, 32), (F, 240, 16, 20, 1),
    (F, 192, 64, 24, 10), (F, 128, 16, 500, 3), (F, 64, 64, 16, 4), (F, 384, 32, 128, 32),
    (F, 512, 64, 256, 32), (S, 3072, 32, 128, 0), (F, 3072, 32, 128, 32), (S, 12288, 64, 128, 0),
    (F, 65536, 64, 256, 32),
    # a distinct summary subblock per head: one layout per subblock
    (P, 256, 16, 32, 8), (P, 256, 64, 128, 32), (P, 240, 16, 20, 6), (P, 512, 64, 256, 32), (P, 192, 32, 48, 10),
    (P, 1024, 64, 128, 2),
    (P, 16384, 64, 128, 32),
]


@pytest.mark.parametrize("pattern,n,B,l,c", LAYOUT_CASES)
@pytest.mark.parametrize("mode", [A1, A2, MG, IL])
def test_layout_bitwise(pattern, n, B, l, c, mode):
    dev = device()
    lay = sa.build_layout(n, B, l, c, pattern, mode, device=dev)
    got = layout_to_cpu(lay)
    ref = orc_mod.layout(n, B, l, c, pattern, mode)
    assert lay.n_layouts == ref["n_layouts"] and list(lay.nnz) == list(ref["nnz"])
    total = int(sum(ref["nnz"]))
    for key in ("row_ptr", "col_ptr"):
        np.testing.assert_array_equal(got[key], ref[key], err_msg=key)
    for key in ("col_idx", "kind", "row_idx", "kind_t"):
        np.testing.assert_array_equal(got[key][:total], ref[key], err_msg=key)


# (pattern, mode, n, B, l, c, d, dtype, batch, heads)
SMALL_CASES = [
    (S, MG, 256, 16, 16, 0, 32, torch.float32, 1, 1),
    (S, A1, 256, 16, 16, 0, 32, torch.float32, 1, 2),
    (S, A2, 256, 16, 16, 0, 64, torch.float32, 2, 1),
    (F, IL, 256, 32, 64, 16, 128, torch.float32, 1, 3),
    (F, A2, 192, 16, 32, 8, 32, torch.float32, 1, 1),
    (S, MG, 512, 64, 64, 0, 64, torch.bfloat16, 2, 2),
    (S, MG, 512, 64, 100, 0, 64, torch.bfloat16, 1, 2),
    (S, A1, 384, 64, 128, 0, 128, torch.bfloat16, 1, 2),
    (S, A2, 384, 32, 48, 0, 64, torch.bfloat16, 1, 2),
    (S, MG, 256, 16, 1, 0, 32, torch.bfloat16, 1, 1),
    (S, MG, 320, 32, 1000, 0, 64, torch.bfloat16, 1, 1),
    (S, MG, 64, 64, 8, 0, 64, torch.bfloat16, 1, 1),
    (F, MG, 1024, 64, 256, 32, 64, torch.bfloat16, 1, 2),
    (F, MG, 512, 64, 96, 40, 64, torch.bfloat16, 2, 1),
    (F, A1, 512, 32, 128, 32, 128, torch.bfloat16, 1, 2),
    (F, A2, 512, 32, 128, 32, 128, torch.bfloat16, 1, 2),
    (F, IL, 768, 32, 128, 32, 128, torch.bfloat16, 2, 3),
    (F, A2, 256, 16, 64, 1, 32, torch.bfloat16, 1, 1),
    (F, MG, 256, 64, 64, 64, 64, torch.bfloat16, 1, 1),
    (F, IL, 512, 16, 48, 12, 64, torch.bfloat16, 1, 2),
    # d = 128 with 16-wide blocks (two waves per SIMD in the backward)
    (S, MG, 256, 16, 32, 0, 128, torch.bfloat16, 1, 2),
    (F, IL, 256, 16, 64, 16, 128, torch.bfloat16, 1, 2),
    # fixed, B = 64, c = 32: rows whose far blocks pair up (even and odd counts)
    (F, A2, 1024, 64, 128, 32, 64, torch.bfloat16, 1, 2),
    (F, MG, 512, 64, 64, 32, 64, torch.bfloat16, 1, 1),
    (F, IL, 1024, 64, 128, 32, 128, torch.bfloat16, 2, 2),
    # an odd number of summary key blocks: one upper half left without a partner
    (F, MG, 768, 64, 256, 32, 64, torch.bfloat16, 1, 2),
    # the short columns of an l-block walked as one dK / dV item: groups of 6
    # and 8 key blocks (l = 384, 512), with and without summary pairs
    (F, MG, 1536, 64, 384, 32, 64, torch.bfloat16, 1, 2),
    (F, A2, 2048, 64, 512, 32, 64, torch.bfloat16, 1, 2),
    # d = 32 with pairs and half items; l = 96 (blocks straddle l-blocks): half
    # items without pairs
    (F, MG, 512, 64, 128, 32, 32, torch.bfloat16, 1, 2),
    (F, MG, 768, 64, 96, 32, 64, torch.bfloat16, 1, 1),
    # more (batch, head) pairs than the dK / dV kernel has queues, not a multiple of them
    (S, MG, 256, 32, 32, 0, 32, torch.bfloat16, 3, 5),
    (F, IL, 256, 16, 64, 16, 32, torch.bfloat16, 3, 3),
    # strided with l a multiple of B: blocks before the band are single
    # diagonals, taken as rank-1 steps (A2 alone, merged, alternating heads,
    # B = 16 / 32 / 64, d = 32 / 64 / 128, l = B and l = 4B)
    (S, A2, 512, 32, 64, 0, 64, torch.bfloat16, 1, 2),
    (S, IL, 768, 64, 128, 0, 128, torch.bfloat16, 2, 2),
    (S, MG, 1024, 16, 32, 0, 32, torch.bfloat16, 1, 2),
    (S, MG, 1024, 64, 256, 0, 64, torch.bfloat16, 1, 3),
    (S, A2, 1024, 64, 64, 0, 128, torch.bfloat16, 2, 1),
    # a distinct summary subblock per head, heads covering every subblock: with
    # B = 64 and c = 32 the windows alternate between the upper and the lower
    # halves of blocks (pairs of upper or of lower halves, split key blocks of
    # either kind); l = 96 (blocks straddle l-blocks); l <= 64 (summary words
    # built per head); fp32; more heads than subblocks
    (P, MG, 1024, 64, 128, 32, 64, torch.bfloat16, 1, 4),
    (P, A2, 1024, 64, 128, 32, 64, torch.bfloat16, 2, 4),
    (P, IL, 1024, 64, 128, 32, 128, torch.bfloat16, 1, 8),
    (P, MG, 768, 64, 256, 32, 64, torch.bfloat16, 1, 8),
    (P, MG, 512, 64, 192, 32, 32, torch.bfloat16, 1, 6),
    (P, MG, 768, 64, 96, 32, 64, torch.bfloat16, 1, 3),
    (P, MG, 512, 32, 64, 16, 64, torch.bfloat16, 1, 5),
    (P, A2, 512, 16, 48, 12, 32, torch.bfloat16, 1, 4),
    (P, MG, 512, 64, 48, 10, 64, torch.bfloat16, 1, 4),
    (P, IL, 256, 32, 64, 16, 128, torch.float32, 1, 4),
    (P, A1, 256, 32, 64, 16, 64, torch.bfloat16, 1, 3),
    # the largest number of subblocks (64, l = 128, c = 2), and eight with l <= 64
    (P, MG, 1024, 64, 128, 2, 32, torch.bfloat16, 1, 64),
    (P, A2, 512, 16, 64, 8, 32, torch.bfloat16, 1, 8),
    # strided merged and A2 heads with l | n and n / l a multiple of 16 take
    # A2 by residue classes (the band over the layout, then dense causal
    # attention inside each class, merged in place): classes of 16, 32, 48,
    # 64, 96, 128 and 256 positions (class blocks of 16, 32, 16, 32, 32, 32,
    # 64), l / B of 1, 2, 4, A2 alone with l < B, d = 32 / 64 / 128, several
    # (batch, head) pairs.  Classes of 32 to 128 positions (a multiple of 32)
    # run their backward as one launch per class, except 128 positions at
    # d = 128 (too large for LDS), which keeps the separate dQ and dK / dV
    # launches; 16, 48 and 256 positions keep them too.
    (S, MG, 1024, 32, 64, 0, 64, torch.bfloat16, 2, 3),
    (S, MG, 2048, 64, 64, 0, 128, torch.bfloat16, 1, 2),
    (S, MG, 3072, 16, 32, 0, 32, torch.bfloat16, 1, 2),
    (S, MG, 4096, 16, 16, 0, 64, torch.bfloat16, 1, 2),
    (S, MG, 8192, 32, 128, 0, 64, torch.bfloat16, 1, 2),
    # band columns of l / B + 1 = 9 blocks: the band's dK / dV takes one
    # workgroup per column instead of the persistent grid
    (S, MG, 8192, 64, 512, 0, 64, torch.bfloat16, 1, 2),
    (S, MG, 4096, 16, 128, 0, 64, torch.bfloat16, 1, 2),
    # classes of 512 and 1,024 positions (8 and 16 class blocks of 64): their
    # dK / dV take one workgroup per column too
    (S, MG, 8192, 16, 16, 0, 64, torch.bfloat16, 1, 2),
    (S, A2, 16384, 16, 16, 0, 32, torch.bfloat16, 1, 1),
    (S, A2, 1536, 64, 32, 0, 64, torch.bfloat16, 2, 2),
    (S, A2, 2048, 32, 8, 0, 32, torch.bfloat16, 1, 2),
    (S, A2, 3072, 64, 32, 0, 128, torch.bfloat16, 1, 1),
    (S, MG, 4096, 32, 32, 0, 64, torch.bfloat16, 1, 2),
    (S, A2, 4096, 32, 32, 0, 128, torch.bfloat16, 1, 1),
    (S, A2, 2048, 32, 32, 0, 32, torch.bfloat16, 2, 2),
    # few summary keys per row (c = 1, 2), A2 alone, many heads: the summary
    # columns sum hundreds of large weights, so the dV / dK products take P and
    # dS in two bf16 parts (shared window and a subblock per head; B = 64 with
    # half items, B = 32 without)
    (F, A2, 512, 64, 64, 1, 64, torch.bfloat16, 1, 32),
    (F, A2, 512, 64, 64, 2, 64, torch.bfloat16, 1, 64),
    (P, A2, 512, 64, 64, 1, 64, torch.bfloat16, 1, 64),
    (P, A2, 512, 64, 64, 2, 64, torch.bfloat16, 1, 32),
    (F, A2, 512, 32, 64, 1, 32, torch.bfloat16, 2, 32),
    (F, MG, 512, 64, 64, 1, 64, torch.bfloat16, 1, 32),
    (F, IL, 512, 64, 64, 2, 128, torch.bfloat16, 1, 32),
]


@pytest.mark.parametrize("pattern,mode,n,B,l,c,d,dtype,batch,heads", SMALL_CASES)
def test_parity_small(pattern, mode, n, B, l, c, d, dtype, batch, heads):
    x = make_inputs(batch, heads, n, d, dtype, seed=n + l + c + d)
    scale = d ** -0.5
    got = run_gpu(x, n=n, block=B, l=l, c=c, pattern=pattern, mode=mode, scale=scale)
    ref = orc_mod.backward(*oracle_inputs(x), pattern=pattern, mode=mode, l=l, c=c, scale=scale)
    label = f"p{pattern} m{mode} n{n} B{B} l{l} c{c} d{d} {str(dtype)[6:]} {batch}x{heads}"
    check_all(label, got, ref, dtype, names=("o", "lse", "dq", "dk", "dv"))


def test_parity_dkdv_work_orders():
    """The dK / dV kernel takes its work in one of three orders: round-robin
    (strided, or columns of at most 8 blocks), serpentine per head (fixed, at
    least four workgroups per (batch, head)) and atomic queues (fixed with
    more (batch, head) pairs than a quarter of the resident workgroups).  The
    last needs many heads: 16 x 16 here.  Each order must cover every column
    exactly once, so all must match the oracle.  With many heads the summary
    halves of the fixed pattern are also walked in pairs (at least 2.5 of them
    per workgroup of a head): under the queues (16 x 16 heads, shared and
    distinct subblocks) and under the serpentine order (2 x 96 heads, l = 64)."""
    dev = device()
    for pattern, n, B, l, c, batch, heads in [(F, 1024, 64, 128, 32, 16, 16),   # queues, pairs
                                               (P, 1024, 64, 128, 32, 16, 16),  # queues, pairs of either half
                                               (F, 1024, 64, 64, 32, 2, 96),    # serpentine, pairs
                                               (F, 1024, 64, 128, 32, 1, 3),    # serpentine
                                               (S, 1024, 64, 128, 0, 2, 5),     # round-robin
                                               (F, 512, 64, 128, 32, 2, 2)]:    # 8 key blocks: round-robin
        x = make_inputs(batch, heads, n, 32, torch.bfloat16, seed=batch * heads + n)
        got = run_gpu(x, n=n, block=B, l=l, c=c, pattern=pattern, mode=MG, scale=32 ** -0.5, dev=dev)
        ref = orc_mod.backward(*oracle_inputs(x), pattern=pattern, mode=MG, l=l, c=c, scale=32 ** -0.5)
        check_all(f"work order p{pattern} n{n} l{l} {batch}x{heads}", got, ref, torch.bfloat16)


def test_workload_fp32_full():
    w = WORKLOADS["strided_n256_l16_f32"]
    x = workload_inputs(w)
    for mode in (MG, A1, A2):
        got = run_gpu(x, n=w.n, block=w.block, l=w.stride, c=w.summary, pattern=w.pattern, mode=mode, scale=w.scale)
        ref = orc_mod.backward(*oracle_inputs(x), pattern=w.pattern, mode=mode, l=w.stride, c=w.summary,
                               scale=w.scale)
        check_all(f"{w.name} mode {mode}", got, ref, torch.float32, names=("o", "lse", "dq", "dk", "dv"))


def test_workload_interleaved_full():
    w = WORKLOADS["fixed_n3072_l128_c32_interleaved"]
    x = workload_inputs(w)
    got = run_gpu(x, n=w.n, block=w.block, l=w.stride, c=w.summary, pattern=w.pattern, mode=w.mode, scale=w.scale)
    ref = orc_mod.backward(*oracle_inputs(x), pattern=w.pattern, mode=w.mode, l=w.stride, c=w.summary,
                           scale=w.scale)
    check_all(w.name, got, ref, torch.bfloat16, names=("o", "lse", "dq", "dk", "dv"))
    empty = np.isneginf(ref["lse"])
    assert empty.sum() == w.batch * (w.heads // 2) * (w.stride - w.summary)  # head 1, first block
    assert np.all(got["o"][np.broadcast_to(empty[..., None], got["o"].shape)] == 0)


def sample_index(w, rng, count):
    """(b, h, i) triples: first and last rows, tile and l-block edges, random."""
    idx = [0, 1, w.block - 1, w.block, w.stride - 1, w.stride, w.stride + 1, w.n // 2, w.n - w.block, w.n - 1]
    idx = [min(i, w.n - 1) for i in idx]  # a dense-limit stride equals n
    idx += list(rng.integers(0, w.n, count - len(idx)))
    b = rng.integers(0, w.batch, len(idx))
    h = rng.integers(0, w.heads, len(idx))
    return np.stack([b, h, np.array(idx)], axis=1)


@pytest.mark.parametrize("name", ["strided_n12288_l128_merged", "fixed_n65536_l256_c32_merged",
                                  "dense_n12288_merged", "fixed_n12288_l128_c32_merged", "dense_n3072_merged",
                                  "fixed_n3072_l128_c32_merged", "strided_n3072_l128_merged",
                                  "fixed_per_head_n65536_l256_c32_merged", "fixed_per_head_n12288_l128_c32_merged"])
def test_workload_sampled(name):
    w = WORKLOADS[name]
    x = workload_inputs(w)
    got = run_gpu(x, n=w.n, block=w.block, l=w.stride, c=w.summary, pattern=w.pattern, mode=w.mode, scale=w.scale)
    rng = np.random.default_rng(w.seed)
    rows = sample_index(w, rng, 48)
    cols = sample_index(w, rng, 24)
    xi = oracle_inputs(x)
    kw = dict(pattern=w.pattern, mode=w.mode, l=w.stride, c=w.summary, scale=w.scale)
    o, lse = orc_mod.forward_rows(*xi[:3], rows, **kw)
    dq = orc_mod.backward_rows(*xi, rows, **kw)
    dk, dv = orc_mod.backward_cols(*xi, cols, **kw)
    r = (rows[:, 0], rows[:, 1], rows[:, 2])
    cc = (cols[:, 0], cols[:, 1], cols[:, 2])
    bf = torch.bfloat16
    check(f"{name} o rows", got["o"][r], o, bf)
    check_lse(f"{name} lse rows", got["lse"][r], lse, bf)
    check(f"{name} dq rows", got["dq"][r], dq, bf)
    check(f"{name} dk cols", got["dk"][cc], dk, bf)
    check(f"{name} dv cols", got["dv"][cc], dv, bf)
    for key in ("o", "dq", "dk", "dv", "lse"):
        assert np.all(np.isfinite(got[key])), key


# Full size, element by element: every (batch, head) slice of the strided text
# workload (n = 12,288, 2 x 8 heads), and two whole slices of the fixed audio
# workload (n = 65,536, all 65,536 rows and columns of heads 0 and 5), in the
# launch configuration the benchmark times (all heads in one call).
def test_workload_strided_n12288_full():
    w = WORKLOADS["strided_n12288_l128_merged"]
    x = workload_inputs(w)
    got = run_gpu(x, n=w.n, block=w.block, l=w.stride, c=w.summary, pattern=w.pattern, mode=w.mode, scale=w.scale)
    ref = orc_mod.backward(*oracle_inputs(x), pattern=w.pattern, mode=w.mode, l=w.stride, c=w.summary,
                           scale=w.scale)
    check_all(f"{w.name} full", got, ref, torch.bfloat16, names=("o", "lse", "dq", "dk", "dv"))


@pytest.mark.parametrize("name", ["fixed_n65536_l256_c32_merged", "fixed_per_head_n65536_l256_c32_merged"])
def test_workload_fixed_n65536_two_slices_full(name):
    w = WORKLOADS[name]
    x = workload_inputs(w)
    got = run_gpu(x, n=w.n, block=w.block, l=w.stride, c=w.summary, pattern=w.pattern, mode=w.mode, scale=w.scale)
    xi = oracle_inputs(x)
    kw = dict(pattern=w.pattern, mode=w.mode, l=w.stride, c=w.summary, scale=w.scale)
    if w.pattern == P:
        # head h's window is subblock h mod (l / c), so the oracle sees heads 0
        # and 1 as such (the upper and the lower half of a key block)
        ref = orc_mod.backward(*[a[:1, 0:2] for a in xi], **kw)
        check_all(f"{name} heads 0, 1 full", {k_: v_[:1, 0:2] for k_, v_ in got.items()}, ref, torch.bfloat16,
                  names=("o", "lse", "dq", "dk", "dv"))
        return
    for h in (0, 5):
        ref = orc_mod.backward(*[a[:1, h:h + 1] for a in xi], **kw)
        check_all(f"{name} head {h} full", {k_: v_[:1, h:h + 1] for k_, v_ in got.items()}, ref, torch.bfloat16,
                  names=("o", "lse", "dq", "dk", "dv"))


def test_ones_value_gives_ones_output():
    dev = device()
    for pattern, mode, l, c in ((S, MG, 64, 0), (F, MG, 64, 16), (F, A2, 64, 16)):
        n, B, d = 512, 64, 64
        x = make_inputs(1, 2, n, d, torch.bfloat16, seed=5)
        x["v"] = torch.ones_like(x["v"])
        got = run_gpu(x, n=n, block=B, l=l, c=c, pattern=pattern, mode=mode, scale=d ** -0.5, backward=False, dev=dev)
        nonempty = np.isfinite(got["lse"])
        check(f"V = 1 p{pattern} m{mode}", got["o"][nonempty], np.ones(int(nonempty.sum()) * d).reshape(-1, d),
              torch.bfloat16)
        assert np.all(got["o"][~nonempty] == 0)


def test_forward_and_layout_are_deterministic():
    dev = device()
    w = WORKLOADS["strided_n12288_l128_merged"]
    x = make_inputs(1, 2, w.n, w.d_head, torch.bfloat16, seed=9)
    q, k, v = (x[n_].to(dev) for n_ in ("q", "k", "v"))
    lay1 = sa.build_layout(w.n, w.block, w.stride, 0, w.pattern, w.mode, device=dev)
    lay2 = sa.build_layout(w.n, w.block, w.stride, 0, w.pattern, w.mode, device=dev)
    for key in ("row_ptr", "col_idx", "kind", "col_ptr", "row_idx", "kind_t"):
        assert torch.equal(getattr(lay1, key), getattr(lay2, key))
    o1, l1 = sa.forward(q, k, v, lay1)
    o2, l2 = sa.forward(q, k, v, lay1)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_strided_views_match_contiguous():
    dev = device()
    b, h, n, d, B = 2, 3, 256, 64, 32
    base = torch.randn(b, n, h, d, generator=torch.Generator().manual_seed(3)).to(torch.bfloat16).to(dev)
    q = base.transpose(1, 2)  # strides (n*h*d, d, h*d, 1)
    k = (base * 0.5).transpose(1, 2)
    v = (base - 0.25).transpose(1, 2)
    lay = sa.build_layout(n, B, 32, 8, F, IL, device=dev)
    o_v, lse_v = sa.forward(q, k, v, lay)
    o_c, lse_c = sa.forward(q.contiguous(), k.contiguous(), v.contiguous(), lay)
    assert torch.equal(o_v.contiguous(), o_c) and torch.equal(lse_v, lse_c)
    dout = torch.randn_like(o_v)
    g_v = sa.backward(q, k, v, o_v, dout, lse_v, lay)
    g_c = sa.backward(q.contiguous(), k.contiguous(), v.contiguous(), o_c, dout.contiguous(), lse_c, lay)
    for a_, b_ in zip(g_v, g_c):
        assert (a_.contiguous().float() - b_.float()).abs().max().item() <= 1e-2


def test_autograd_wrapper():
    dev = device()
    n, B, d = 256, 32, 64
    x = make_inputs(1, 2, n, d, torch.bfloat16, seed=21)
    lay = sa.build_layout(n, B, 32, 0, S, MG, device=dev)
    q, k, v = (x[n_].to(dev).requires_grad_(True) for n_ in ("q", "k", "v"))
    o = sa.SparseAttention.apply(q, k, v, lay, None)
    (o.float() * x["dout"].to(dev).float()).sum().backward()
    ref = orc_mod.backward(*oracle_inputs(x), pattern=S, mode=MG, l=32, c=0, scale=d ** -0.5)
    check("autograd o", to64(o), ref["o"], torch.bfloat16)
    check("autograd dq", to64(q.grad), ref["dq"], torch.bfloat16)
    check("autograd dk", to64(k.grad), ref["dk"], torch.bfloat16)
    check("autograd dv", to64(v.grad), ref["dv"], torch.bfloat16)


def test_strided_classes_with_views():
    """The strided merged path by residue classes on [b, n, h, d] storage seen
    as [b, h, n, d] (batch 1: heads and rows in one stride pattern), against
    the oracle."""
    dev = device()
    n, l, B, d, h = 2048, 64, 64, 64, 3
    x = make_inputs(1, h, n, d, torch.bfloat16, seed=29)
    lay = sa.build_layout(n, B, l, 0, S, MG, device=dev)
    q, k, v, dout = (x[n_].transpose(1, 2).contiguous().to(dev).transpose(1, 2) for n_ in ("q", "k", "v", "dout"))
    assert not q.is_contiguous()
    o, lse = sa.forward(q, k, v, lay)
    dq, dk, dv = sa.backward(q, k, v, o, dout, lse, lay)
    torch.cuda.synchronize()
    ref = orc_mod.backward(*oracle_inputs(x), pattern=S, mode=MG, l=l, c=0, scale=d ** -0.5)
    got = {"o": to64(o), "lse": to64(lse), "dq": to64(dq), "dk": to64(dk), "dv": to64(dv)}
    check_all("strided classes, [b, n, h, d] views", got, ref, torch.bfloat16, names=("o", "lse", "dq", "dk", "dv"))


def test_autograd_wrapper_transposed_views():
    """q, k, v as [b, n, h, d].transpose(1, 2) views (not contiguous): the
    wrapper hands the incoming gradient over with q's strides."""
    dev = device()
    b, n, h, d = 1, 256, 2, 64
    x = make_inputs(b, h, n, d, torch.bfloat16, seed=23)
    lay = sa.build_layout(n, 32, 32, 8, F, IL, device=dev)
    leaves = [x[n_].transpose(1, 2).contiguous().to(dev).requires_grad_(True) for n_ in ("q", "k", "v")]
    q, k, v = (t.transpose(1, 2) for t in leaves)  # [b, h, n, d] views of [b, n, h, d] storage
    assert not q.is_contiguous()
    o = sa.SparseAttention.apply(q, k, v, lay, None)
    (o.float() * x["dout"].to(dev).float()).sum().backward()
    ref = orc_mod.backward(*oracle_inputs(x), pattern=F, mode=IL, l=32, c=8, scale=d ** -0.5)
    check("autograd views o", to64(o), ref["o"], torch.bfloat16)
    for name, t in (("dq", leaves[0]), ("dk", leaves[1]), ("dv", leaves[2])):
        check(f"autograd views {name}", to64(t.grad.transpose(1, 2)), ref[name], torch.bfloat16)


def test_binding_rejects_mismatched_tensors():
    """Shapes, dtypes, devices and the sequence length are checked before the
    C ABI is called: a smaller or differently typed tensor never reaches a
    kernel."""
    dev = device()
    n, d = 256, 64
    x = make_inputs(2, 2, n, d, torch.bfloat16, seed=4)
    q, k, v, dout = (x[n_].to(dev) for n_ in ("q", "k", "v", "dout"))
    lay = sa.build_layout(n, 64, 64, 0, S, MG, device=dev)
    o, lse = sa.forward(q, k, v, lay)
    bad = [
        lambda: sa.forward(q, k[:1].contiguous(), v, lay),                    # batch
        lambda: sa.forward(q, k, v[:, :, : n - 64].contiguous(), lay),        # sequence
        lambda: sa.forward(q, k.float(), v, lay),                             # dtype
        lambda: sa.forward(q, k.cpu(), v, lay),                               # device
        lambda: sa.forward(q[:, :, :128].contiguous(), k[:, :, :128].contiguous(),
                           v[:, :, :128].contiguous(), lay),                  # n against the layout
        lambda: sa.forward(q, k, v, lay, out=torch.empty_like(q[:1])),
        lambda: sa.forward(q, k, v, lay, lse=torch.empty(2, 2, n - 1, device=dev)),
        lambda: sa.backward(q, k, v, o, dout[:1].contiguous(), lse, lay),
        lambda: sa.backward(q, k, v, o.float(), dout, lse, lay),
        lambda: sa.backward(q, k, v, o, dout, lse[:, :, 1:], lay),
        lambda: sa.backward(q, k, v, o, dout, lse.to(torch.bfloat16), lay),
        lambda: sa.backward(q[:, :, :128].contiguous(), k[:, :, :128].contiguous(), v[:, :, :128].contiguous(),
                            o[:, :, :128].contiguous(), dout[:, :, :128].contiguous(),
                            lse[:, :, :128].contiguous(), lay),
        lambda: sa.backward(q, k, v, o, dout, lse, lay, grads=(torch.empty_like(q), torch.empty_like(k[:1]),
                                                               torch.empty_like(v))),
    ]
    for i, f in enumerate(bad):
        with pytest.raises(ValueError):
            f()
            print("not rejected:", i)
    torch.cuda.synchronize()


# ---------------------------------------------------------------------------
# n = 1,048,576 (strided l = 1024, B = 64, 4 merged heads of 64): the layout
# bitwise, and forward / backward on sampled rows and columns; outputs are
# gathered on the device so that nothing of the full size is copied back in
# float64.
# ---------------------------------------------------------------------------
def test_layout_n1048576_bitwise():
    w = WORKLOADS["strided_n1048576_l1024_merged"]
    dev = device()
    lay = sa.build_layout(w.n, w.block, w.stride, w.summary, w.pattern, w.mode, device=dev)
    got = layout_to_cpu(lay)
    ref = orc_mod.layout(w.n, w.block, w.stride, w.summary, w.pattern, w.mode)
    assert list(lay.nnz) == list(ref["nnz"])
    total = int(sum(ref["nnz"]))
    for key in ("row_ptr", "col_ptr"):
        np.testing.assert_array_equal(got[key], ref[key], err_msg=key)
    for key in ("col_idx", "kind", "row_idx", "kind_t"):
        np.testing.assert_array_equal(got[key][:total], ref[key], err_msg=key)


def test_workload_n1048576_sampled():
    w = WORKLOADS["strided_n1048576_l1024_merged"]
    dev = device()
    x = workload_inputs(w)
    lay = sa.build_layout(w.n, w.block, w.stride, w.summary, w.pattern, w.mode, device=dev)
    q, k, v, dout = (x[name].to(dev) for name in ("q", "k", "v", "dout"))
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    ev[0].record()
    o, lse = sa.forward(q, k, v, lay, w.scale)
    ev[1].record()
    dq, dk, dv = sa.backward(q, k, v, o, dout, lse, lay, w.scale)
    ev[2].record()
    torch.cuda.synchronize()
    print(f"n=1048576: forward {ev[0].elapsed_time(ev[1]):.1f} ms, backward {ev[1].elapsed_time(ev[2]):.1f} ms "
          f"(first call)", flush=True)
    for t in (o, dq, dk, dv):
        assert bool(torch.isfinite(t).all())
    rng = np.random.default_rng(w.seed)
    rows = sample_index(w, rng, 32)
    cols = sample_index(w, rng, 16)

    def gather(t, idx):
        ix = torch.as_tensor(idx, device=dev)
        return to64(t[ix[:, 0], ix[:, 1], ix[:, 2]])

    xi = oracle_inputs(x)
    kw = dict(pattern=w.pattern, mode=w.mode, l=w.stride, c=w.summary, scale=w.scale)
    o_ref, lse_ref = orc_mod.forward_rows(*xi[:3], rows, **kw)
    dq_ref = orc_mod.backward_rows(*xi, rows, **kw)
    dk_ref, dv_ref = orc_mod.backward_cols(*xi, cols, **kw)
    bf = torch.bfloat16
    check("n1048576 o rows", gather(o, rows), o_ref, bf)
    check_lse("n1048576 lse rows", gather(lse, rows), lse_ref, bf)
    check("n1048576 dq rows", gather(dq, rows), dq_ref, bf)
    check("n1048576 dk cols", gather(dk, cols), dk_ref, bf)
    check("n1048576 dv cols", gather(dv, cols), dv_ref, bf)
