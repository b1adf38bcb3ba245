"""Pins of the fp64 oracle against what the paper and mathematics fix.

Nothing here compares the oracle with itself: every expectation comes from the
paper's set-builder definitions (Sec. 4.3), its worked example, closed forms
derived from those definitions, validity (Sec. 4.2), textbook identities of
softmax attention, library routines (PyTorch's scaled-dot-product attention and
autograd, on the CPU in fp64) or finite differences.
"""
import json
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import dense

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
STRIDED, FIXED = 0, 1
A1, A2, MERGED, INTERLEAVED = 0, 1, 2, 3

SMALL_SHAPES = [  # (n, l, c) covering l | n, l not dividing n, l = 1, c = 1, c = l, l >= n
    (64, 8, 2), (96, 16, 4), (100, 7, 3), (64, 1, 1), (48, 48, 48), (40, 64, 5), (128, 12, 12),
]


def closed_form_count(pattern, part, i, l, c):
    """|S_i| derived from the Sec. 4.3 definitions (0-based, causal)."""
    if pattern == STRIDED:
        if part == A1:
            return min(i, l) + 1
        if part == A2:
            return i // l + 1
        return min(i, l) + 1 + max(0, i // l - 1)
    if part == A1:
        return i % l + 1
    if part == A2:
        return c * (i // l) + max(0, i % l - (l - c) + 1)
    return i % l + 1 + c * (i // l)


@pytest.mark.parametrize("pattern", [STRIDED, FIXED])
@pytest.mark.parametrize("part", [A1, A2, MERGED])
@pytest.mark.parametrize("n,l,c", SMALL_SHAPES)
def test_row_sets_equal_set_builder_definition(orc, pattern, part, n, l, c):
    mask = dense.part_mask(pattern, part, n, l, c)
    for i in range(n):
        got = orc.row_set(pattern, part, n, l, c, i)
        np.testing.assert_array_equal(got, np.nonzero(mask[i])[0])
        assert len(got) == closed_form_count(pattern, part, i, l, c)


@pytest.mark.parametrize("pattern", [STRIDED, FIXED])
@pytest.mark.parametrize("part", [A1, A2, MERGED])
@pytest.mark.parametrize("n,l,c", SMALL_SHAPES)
def test_col_sets_are_the_transpose(orc, pattern, part, n, l, c):
    mask = dense.part_mask(pattern, part, n, l, c)
    for j in range(n):
        np.testing.assert_array_equal(orc.col_set(pattern, part, n, l, c, j), np.nonzero(mask[:, j])[0])


@pytest.mark.parametrize("pattern,l,c", [(STRIDED, 128, 0), (STRIDED, 1024, 0), (FIXED, 128, 32),
                                         (FIXED, 256, 32), (FIXED, 128, 8)])
def test_row_counts_closed_form_at_workload_strides(orc, pattern, l, c):
    n = 8 * l
    rng = np.random.default_rng(0)
    for part in (A1, A2, MERGED):
        for i in list(range(0, 3 * l + 2)) + list(rng.integers(0, n, 64)):
            assert len(orc.row_set(pattern, part, n, l, c, int(i))) == closed_form_count(pattern, part, int(i), l, c)


def test_fixed_worked_example(orc):
    ex = json.load(open(os.path.join(GOLDEN, "fixed_l128_c8_example.json")))
    l, c = ex["l"], ex["c"]
    n = 4 * l
    for case in ex["cases"]:
        lo, hi = case["rows"]
        for i in range(lo, hi + 1):
            block_start = (i // l) * l
            for part in (A2, MERGED):
                s = orc.row_set(FIXED, part, n, l, c, i)
                np.testing.assert_array_equal(s[s < block_start], case["earlier_block_columns"])


def test_stride_cost_ratio(orc):
    """Fixed A2 costs about c times strided A2 (Sec. 4.3): compare total set sizes."""
    n, l, c = 4096, 64, 16
    strided = sum(len(orc.row_set(STRIDED, A2, n, l, 0, i)) for i in range(n))
    fixed = sum(len(orc.row_set(FIXED, A2, n, l, c, i)) for i in range(n))
    assert abs(fixed / strided - c) / c < 0.1


@pytest.mark.parametrize("pattern,n,l,c", [(STRIDED, 256, 16, 0), (STRIDED, 300, 17, 0), (FIXED, 256, 16, 1),
                                           (FIXED, 256, 16, 4), (FIXED, 250, 32, 8)])
def test_two_step_reachability(orc, pattern, n, l, c):
    """Validity (Sec. 4.2): every j <= i reaches i in at most p = 2 steps, first
    through A1 (j in A1 of a), then through A2 (a in A2 of i)."""
    m1 = np.zeros((n, n), dtype=np.int64)
    m2 = np.zeros((n, n), dtype=np.int64)
    for i in range(n):
        m1[i, orc.row_set(pattern, A1, n, l, c, i)] = 1
        m2[i, orc.row_set(pattern, A2, n, l, c, i)] = 1
    reach = (m1 + m2 @ m1) > 0
    np.testing.assert_array_equal(reach, np.tril(np.ones((n, n), dtype=bool)))


def _inputs(b, h, n, d, seed, dtype=torch.float64):
    g = torch.Generator().manual_seed(seed)
    return [torch.randn((b, h, n, d), generator=g, dtype=torch.float64).to(dtype) for _ in range(4)]


def _np(t):
    return t.detach().numpy()


def _sdpa_causal_with_grads(q, k, v, dout, scale):
    q, k, v = (x.clone().requires_grad_(True) for x in (q, k, v))
    o = F.scaled_dot_product_attention(q, k, v, is_causal=True, scale=scale)
    (o * dout).sum().backward()
    return o.detach(), q.grad, k.grad, v.grad


def _causal_lse(q, k, scale):
    n = q.shape[-2]
    s = scale * q @ k.transpose(-1, -2)
    s = s.masked_fill(~torch.ones(n, n, dtype=torch.bool).tril(), float("-inf"))
    return torch.logsumexp(s, dim=-1)


@pytest.mark.parametrize("pattern,mode,l,c", [
    (STRIDED, A1, 300, 0), (STRIDED, MERGED, 300, 0), (STRIDED, MERGED, 1, 0),
    (FIXED, A1, 300, 7), (FIXED, MERGED, 300, 7), (FIXED, MERGED, 16, 16),
])
def test_dense_causal_special_cases(orc, pattern, mode, l, c):
    """l >= n (A1 or merged), fixed merged with c = l and strided merged with l = 1
    all attend to every j <= i: the result is dense causal attention (Sec. 4.2)."""
    b, h, n, d = 1, 2, 160, 16
    scale = d ** -0.5
    q, k, v, dout = _inputs(b, h, n, d, seed=7)
    res = orc.backward(_np(q), _np(k), _np(v), _np(dout), pattern=pattern, mode=mode, l=l, c=c, scale=scale)
    o_ref, dq_ref, dk_ref, dv_ref = _sdpa_causal_with_grads(q, k, v, dout, scale)
    np.testing.assert_allclose(res["o"], _np(o_ref), atol=1e-12, rtol=0)
    np.testing.assert_allclose(res["lse"], _np(_causal_lse(q, k, scale)), atol=1e-12, rtol=0)
    for name, ref in (("dq", dq_ref), ("dk", dk_ref), ("dv", dv_ref)):
        np.testing.assert_allclose(res[name], _np(ref), atol=1e-11, rtol=0, err_msg=name)
    o_only, lse_only = orc.forward(_np(q), _np(k), _np(v), pattern=pattern, mode=mode, l=l, c=c, scale=scale)
    np.testing.assert_array_equal(o_only, res["o"])
    np.testing.assert_array_equal(lse_only, res["lse"])


def test_fixed_a1_is_blockwise_dense_causal(orc):
    b, h, n, d, l = 1, 1, 192, 16, 48
    scale = d ** -0.5
    q, k, v, dout = _inputs(b, h, n, d, seed=11)
    res = orc.backward(_np(q), _np(k), _np(v), _np(dout), pattern=FIXED, mode=A1, l=l, c=4, scale=scale)
    for L in range(n // l):
        sl = slice(L * l, (L + 1) * l)
        o, dq, dk, dv = _sdpa_causal_with_grads(q[..., sl, :], k[..., sl, :], v[..., sl, :], dout[..., sl, :], scale)
        np.testing.assert_allclose(res["o"][..., sl, :], _np(o), atol=1e-12, rtol=0)
        np.testing.assert_allclose(res["dq"][..., sl, :], _np(dq), atol=1e-11, rtol=0)
        np.testing.assert_allclose(res["dk"][..., sl, :], _np(dk), atol=1e-11, rtol=0)
        np.testing.assert_allclose(res["dv"][..., sl, :], _np(dv), atol=1e-11, rtol=0)


def test_strided_a2_is_dense_causal_after_transpose(orc):
    """Sec. 5.5: attention with stride l is a local (here: full causal) window
    after regrouping positions by residue class i mod l."""
    b, h, n, d, l = 1, 2, 240, 8, 12
    scale = d ** -0.5
    q, k, v, dout = _inputs(b, h, n, d, seed=13)
    res = orc.backward(_np(q), _np(k), _np(v), _np(dout), pattern=STRIDED, mode=A2, l=l, c=0, scale=scale)
    for r in range(l):
        sl = slice(r, n, l)
        o, dq, dk, dv = _sdpa_causal_with_grads(q[..., sl, :], k[..., sl, :], v[..., sl, :], dout[..., sl, :], scale)
        np.testing.assert_allclose(res["o"][..., sl, :], _np(o), atol=1e-12, rtol=0)
        np.testing.assert_allclose(res["lse"][..., sl], _np(_causal_lse(q[..., sl, :], k[..., sl, :], scale)),
                                   atol=1e-12, rtol=0)
        np.testing.assert_allclose(res["dq"][..., sl, :], _np(dq), atol=1e-11, rtol=0)
        np.testing.assert_allclose(res["dk"][..., sl, :], _np(dk), atol=1e-11, rtol=0)
        np.testing.assert_allclose(res["dv"][..., sl, :], _np(dv), atol=1e-11, rtol=0)


def test_strided_a1_is_a_band(orc):
    b, h, n, d, l = 1, 1, 200, 16, 23
    scale = d ** -0.5
    q, k, v, _ = _inputs(b, h, n, d, seed=17)
    i = torch.arange(n)[:, None]
    j = torch.arange(n)[None, :]
    band = (i - j >= 0) & (i - j <= l)
    ref = F.scaled_dot_product_attention(q, k, v, attn_mask=band, scale=scale)
    o, _ = orc.forward(_np(q), _np(k), _np(v), pattern=STRIDED, mode=A1, l=l, c=0, scale=scale)
    np.testing.assert_allclose(o, _np(ref), atol=1e-12, rtol=0)


@pytest.mark.parametrize("pattern,l,c", [(STRIDED, 8, 0), (STRIDED, 5, 0), (FIXED, 16, 4), (FIXED, 12, 5)])
def test_merged_is_softmax_over_disjoint_union(orc, pattern, l, c):
    """Merged head (Sec. 5.1, eq. mergedmat): softmax over A1 u A2 equals the
    log-sum-exp combination of the attentions over A1 and over A2 minus A1."""
    b, h, n, d = 1, 1, 120, 8
    scale = d ** -0.5
    q, k, v, _ = _inputs(b, h, n, d, seed=19)
    s = scale * q[0, 0] @ k[0, 0].T
    m1 = torch.from_numpy(dense.part_mask(pattern, A1, n, l, c))
    m2 = torch.from_numpy(dense.part_mask(pattern, A2, n, l, c)) & ~m1

    def part(mask):
        sm = s.masked_fill(~mask, float("-inf"))
        lse = torch.logsumexp(sm, dim=-1)
        p = torch.exp(sm - lse[:, None]).nan_to_num(0.0)
        return p @ v[0, 0], lse

    o1, l1 = part(m1)
    o2, l2 = part(m2)
    lse = torch.logaddexp(l1, l2)
    o = torch.exp(l1 - lse)[:, None] * o1 + torch.exp(l2 - lse)[:, None].nan_to_num(0.0) * o2.nan_to_num(0.0)
    got_o, got_lse = orc.forward(_np(q), _np(k), _np(v), pattern=pattern, mode=MERGED, l=l, c=c, scale=scale)
    np.testing.assert_allclose(got_o[0, 0], _np(o), atol=1e-12, rtol=0)
    np.testing.assert_allclose(got_lse[0, 0], _np(lse), atol=1e-12, rtol=0)


@pytest.mark.parametrize("pattern,mode,l,c", [(STRIDED, MERGED, 16, 0), (STRIDED, A2, 7, 0),
                                              (FIXED, A2, 32, 8), (FIXED, INTERLEAVED, 32, 8)])
def test_rows_sum_to_one_and_empty_rows(orc, pattern, mode, l, c):
    """Softmax weights of a non-empty row sum to 1, so V = 1 gives O = 1; an
    empty row (fixed A2 alone, first block) gives O = 0 and LSE = -inf."""
    b, h, n, d = 1, 2, 128, 8
    q, k, _, _ = _inputs(b, h, n, d, seed=23)
    ones = np.ones((b, h, n, d))
    o, lse = orc.forward(_np(q), _np(k), ones, pattern=pattern, mode=mode, l=l, c=c, scale=0.3)
    for hh in range(h):
        mask = dense.head_mask(pattern, mode, hh, n, l, c)
        empty = ~mask.any(axis=1)
        np.testing.assert_allclose(o[0, hh][~empty], 1.0, atol=1e-13, rtol=0)
        np.testing.assert_array_equal(o[0, hh][empty], 0.0)
        assert np.all(np.isneginf(lse[0, hh][empty])) and np.all(np.isfinite(lse[0, hh][~empty]))
        if pattern == FIXED and (mode == A2 or (mode == INTERLEAVED and hh == 1)):
            assert empty.sum() == l - c  # the first block's non-summary rows


@pytest.mark.parametrize("pattern,l,c", [(STRIDED, 8, 0), (STRIDED, 6, 0), (FIXED, 8, 2), (FIXED, 16, 3)])
@pytest.mark.parametrize("mode", [A1, A2, MERGED, INTERLEAVED])
def test_backward_against_central_differences(orc, pattern, l, c, mode):
    b, h, n, d = 1, 2, 48, 8
    scale = d ** -0.5
    q, k, v, dout = (_np(x) for x in _inputs(b, h, n, d, seed=29))
    res = orc.backward(q, k, v, dout, pattern=pattern, mode=mode, l=l, c=c, scale=scale)

    def loss(qq, kk, vv):
        o, _ = orc.forward(qq, kk, vv, pattern=pattern, mode=mode, l=l, c=c, scale=scale)
        return float((o * dout).sum())

    rng = np.random.default_rng(31)
    eps = 1e-5
    for name, arr in (("dq", q), ("dk", k), ("dv", v)):
        for _ in range(24):
            idx = tuple(int(rng.integers(0, s)) for s in arr.shape)
            plus, minus = arr.copy(), arr.copy()
            plus[idx] += eps
            minus[idx] -= eps
            args_p = [plus if a is arr else a for a in (q, k, v)]
            args_m = [minus if a is arr else a for a in (q, k, v)]
            fd = (loss(*args_p) - loss(*args_m)) / (2 * eps)
            assert abs(fd - res[name][idx]) <= 1e-7 * max(1.0, abs(fd)), (name, idx, fd, res[name][idx])


@pytest.mark.parametrize("pattern,mode,l,c", [(STRIDED, MERGED, 16, 0), (FIXED, MERGED, 32, 8),
                                              (FIXED, A2, 32, 8), (STRIDED, A1, 9, 0)])
def test_gradient_shift_invariances(orc, pattern, mode, l, c):
    """Adding one vector to every key leaves each row's softmax unchanged, so
    sum_j dk_j = 0; the weights of a non-empty row sum to 1, so
    sum_j dv_j = sum over non-empty rows of dO_i."""
    b, h, n, d = 2, 2, 128, 8
    q, k, v, dout = (_np(x) for x in _inputs(b, h, n, d, seed=37))
    res = orc.backward(q, k, v, dout, pattern=pattern, mode=mode, l=l, c=c, scale=0.4)
    np.testing.assert_allclose(res["dk"].sum(axis=2), 0.0, atol=1e-11)
    for hh in range(h):
        empty = ~dense.head_mask(pattern, mode, hh, n, l, c).any(axis=1)
        np.testing.assert_allclose(res["dv"][:, hh].sum(axis=1), dout[:, hh][:, ~empty].sum(axis=1), atol=1e-11)


@pytest.mark.parametrize("pattern,mode,n,l,c", [(STRIDED, MERGED, 256, 16, 0), (STRIDED, INTERLEAVED, 200, 9, 0),
                                                (FIXED, INTERLEAVED, 256, 32, 8), (FIXED, A2, 192, 64, 64)])
def test_oracle_matches_dense_numpy(orc, pattern, mode, n, l, c):
    b, h, d = 1, 2, 16
    scale = d ** -0.5
    q, k, v, dout = (_np(x) for x in _inputs(b, h, n, d, seed=41))
    res = orc.backward(q, k, v, dout, pattern=pattern, mode=mode, l=l, c=c, scale=scale)
    for hh in range(h):
        mask = dense.head_mask(pattern, mode, hh, n, l, c)
        o, lse, dq, dk, dv = dense.attention_grads(q[0, hh], k[0, hh], v[0, hh], dout[0, hh], mask, scale)
        np.testing.assert_allclose(res["o"][0, hh], o, atol=1e-12, rtol=0)
        np.testing.assert_array_equal(np.isneginf(res["lse"][0, hh]), np.isneginf(lse))
        fin = np.isfinite(lse)
        np.testing.assert_allclose(res["lse"][0, hh][fin], lse[fin], atol=1e-12, rtol=0)
        for name, ref in (("dq", dq), ("dk", dk), ("dv", dv)):
            np.testing.assert_allclose(res[name][0, hh], ref, atol=1e-11, rtol=0, err_msg=name)


def test_sampled_rows_and_columns_match_full_pass(orc):
    b, h, n, d = 2, 2, 192, 16
    scale = d ** -0.5
    q, k, v, dout = (_np(x) for x in _inputs(b, h, n, d, seed=43, dtype=torch.float32))
    kw = dict(pattern=FIXED, mode=INTERLEAVED, l=32, c=8, scale=scale)
    full = orc.backward(q, k, v, dout, **kw)
    rng = np.random.default_rng(0)
    idx = np.stack([rng.integers(0, b, 40), rng.integers(0, h, 40), rng.integers(0, n, 40)], axis=1)
    o, lse = orc.forward_rows(q, k, v, idx, **kw)
    dq = orc.backward_rows(q, k, v, dout, idx, **kw)
    dk, dv = orc.backward_cols(q, k, v, dout, idx, **kw)
    sel = (idx[:, 0], idx[:, 1], idx[:, 2])
    np.testing.assert_allclose(o, full["o"][sel], atol=1e-13, rtol=0)
    np.testing.assert_array_equal(np.isneginf(lse), np.isneginf(full["lse"][sel]))
    np.testing.assert_allclose(dq, full["dq"][sel], atol=1e-13, rtol=0)
    np.testing.assert_allclose(dk, full["dk"][sel], atol=1e-13, rtol=0)
    np.testing.assert_allclose(dv, full["dv"][sel], atol=1e-13, rtol=0)


def test_bf16_inputs_are_read_exactly(orc):
    t = torch.randn(1, 1, 64, 8, generator=torch.Generator().manual_seed(3)).to(torch.bfloat16)
    bits = t.view(torch.int16).numpy().view(np.uint16)
    as64 = t.to(torch.float64).numpy()
    kw = dict(pattern=STRIDED, mode=MERGED, l=8, c=0, scale=0.5)
    o_bits, lse_bits = orc.forward(bits, bits, bits, **kw)
    o_64, lse_64 = orc.forward(as64, as64, as64, **kw)
    np.testing.assert_array_equal(o_bits, o_64)
    np.testing.assert_array_equal(lse_bits, lse_64)


# ---------------------------------------------------------------------------
# Distinct summary subblocks per head (pattern 2, Sec. 4.3 closing remark)
# ---------------------------------------------------------------------------
FIXED_PER_HEAD = 2
PER_HEAD_SHAPES = [(64, 8, 2), (96, 16, 4), (100, 12, 5), (48, 48, 48), (40, 64, 5), (64, 8, 1)]


def test_per_head_worked_example(orc):
    ex = json.load(open(os.path.join(GOLDEN, "fixed_per_head_l8_c2_example.json")))
    l, c = ex["l"], ex["c"]
    n = 4 * l
    for h, cols in ex["windows"].items():
        h = int(h)
        # the window shows in A2 of the last row as the first block's members
        s = orc.head_row_set(FIXED_PER_HEAD, A2, n, l, c, h, n - 1)
        np.testing.assert_array_equal(s[s < l], cols)
    for case in ex["a2_rows"]:
        np.testing.assert_array_equal(orc.head_row_set(FIXED_PER_HEAD, A2, n, l, c, case["head"], case["row"]),
                                      case["set"])
    for case in ex["merged_rows"]:
        np.testing.assert_array_equal(orc.head_row_set(FIXED_PER_HEAD, MERGED, n, l, c, case["head"], case["row"]),
                                      case["set"])


@pytest.mark.parametrize("mode", [A1, A2, MERGED, INTERLEAVED])
@pytest.mark.parametrize("n,l,c", PER_HEAD_SHAPES)
def test_per_head_sets_equal_predicate_and_transpose(orc, mode, n, l, c):
    for h in range(l // c + 2):
        mask = dense.head_mask(FIXED_PER_HEAD, mode, h, n, l, c)
        for i in range(n):
            np.testing.assert_array_equal(orc.head_row_set(FIXED_PER_HEAD, mode, n, l, c, h, i), np.nonzero(mask[i])[0])
        for j in range(n):
            np.testing.assert_array_equal(orc.head_col_set(FIXED_PER_HEAD, mode, n, l, c, h, j),
                                          np.nonzero(mask[:, j])[0])


@pytest.mark.parametrize("n,l,c", [(96, 16, 4), (64, 8, 2), (90, 9, 3), (64, 8, 8)])
def test_per_head_windows_partition_earlier_blocks(orc, n, l, c):
    """With c | l the l/c heads' windows tile each block: over heads 0 .. l/c - 1,
    every position of an earlier block is in exactly one head's A2, and head 0
    (and every head h = 0 mod l/c) has the plain fixed pattern's set."""
    S = l // c
    for i in range(n):
        blk0 = (i // l) * l
        hits = np.zeros(blk0, dtype=np.int64)
        for h in range(S):
            s = orc.head_row_set(FIXED_PER_HEAD, A2, n, l, c, h, i)
            hits[s[s < blk0]] += 1
        np.testing.assert_array_equal(hits, 1)
        for h in (0, S, 2 * S):
            for part in (A2, MERGED):
                np.testing.assert_array_equal(orc.head_row_set(FIXED_PER_HEAD, part, n, l, c, h, i),
                                              orc.row_set(FIXED, part, n, l, c, i))


@pytest.mark.parametrize("n,l,c", [(256, 16, 4), (250, 32, 8), (192, 12, 4)])
def test_per_head_two_step_reachability(orc, n, l, c):
    """Validity (Sec. 4.2) across the heads: with A2 the union of the heads'
    windows (they tile the block when c | l), every j <= i reaches i in two
    steps.  One head alone is valid only for subblock 0: positions of an
    earlier block after its window reach no later block through A2."""
    S = l // c

    def masks(h):
        m1 = np.zeros((n, n), dtype=np.int64)
        m2 = np.zeros((n, n), dtype=np.int64)
        for i in range(n):
            m1[i, orc.head_row_set(FIXED_PER_HEAD, A1, n, l, c, h, i)] = 1
            m2[i, orc.head_row_set(FIXED_PER_HEAD, A2, n, l, c, h, i)] = 1
        return m1, m2

    tril = np.tril(np.ones((n, n), dtype=bool))
    m1, m2u = masks(0)
    np.testing.assert_array_equal((m1 + m2u @ m1) > 0, tril)
    for h in range(1, S):
        m1h, m2 = masks(h)
        np.testing.assert_array_equal(m1h, m1)
        assert not np.array_equal((m1 + m2 @ m1) > 0, tril)
        m2u = m2u + m2
    np.testing.assert_array_equal((m1 + m2u @ m1) > 0, tril)


@pytest.mark.parametrize("mode,n,l,c", [(A2, 128, 16, 4), (MERGED, 192, 32, 8), (INTERLEAVED, 160, 16, 4)])
def test_per_head_oracle_matches_dense_numpy(orc, mode, n, l, c):
    b, h, d = 1, 5, 16
    scale = d ** -0.5
    q, k, v, dout = (_np(x) for x in _inputs(b, h, n, d, seed=47))
    res = orc.backward(q, k, v, dout, pattern=FIXED_PER_HEAD, mode=mode, l=l, c=c, scale=scale)
    for hh in range(h):
        mask = dense.head_mask(FIXED_PER_HEAD, mode, hh, n, l, c)
        o, lse, dq, dk, dv = dense.attention_grads(q[0, hh], k[0, hh], v[0, hh], dout[0, hh], mask, scale)
        np.testing.assert_allclose(res["o"][0, hh], o, atol=1e-12, rtol=0)
        np.testing.assert_array_equal(np.isneginf(res["lse"][0, hh]), np.isneginf(lse))
        fin = np.isfinite(lse)
        np.testing.assert_allclose(res["lse"][0, hh][fin], lse[fin], atol=1e-12, rtol=0)
        for name, ref in (("dq", dq), ("dk", dk), ("dv", dv)):
            np.testing.assert_allclose(res[name][0, hh], ref, atol=1e-11, rtol=0, err_msg=name)
    idx = np.array([[0, hh, i] for hh in range(h) for i in (0, 3, n // 2 + 1, n - 1)])
    o_r, _ = orc.forward_rows(q, k, v, idx, pattern=FIXED_PER_HEAD, mode=mode, l=l, c=c, scale=scale)
    dk_c, dv_c = orc.backward_cols(q, k, v, dout, idx, pattern=FIXED_PER_HEAD, mode=mode, l=l, c=c, scale=scale)
    sel = (idx[:, 0], idx[:, 1], idx[:, 2])
    np.testing.assert_allclose(o_r, res["o"][sel], atol=1e-13, rtol=0)
    np.testing.assert_allclose(dk_c, res["dk"][sel], atol=1e-13, rtol=0)
    np.testing.assert_allclose(dv_c, res["dv"][sel], atol=1e-13, rtol=0)
