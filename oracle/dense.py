"""Dense NumPy cross-check of the oracle, for small n (test infrastructure only).

The connectivity mask is built straight from the set-builder definitions of
Sec. 4.3 as elementwise predicates over all (i, j) pairs, intersected with the
causal set {j <= i} of Sec. 4.2; attention is then a dense masked softmax.
It has nothing in common with the interval enumeration of the C oracle.
"""
import numpy as np

STRIDED, FIXED, FIXED_PER_HEAD = 0, 1, 2


def part_mask(pattern, part, n, l, c, s=0):
    """Boolean [n, n] mask, mask[i, j] = j in S_i, for part 0=A1, 1=A2, 2=merged.
    Fixed pattern: s picks the summary subblock, positions l-(s+1)c .. l-sc-1
    of each block (s = 0: the last c positions)."""
    i = np.arange(n)[:, None]
    j = np.arange(n)[None, :]
    causal = j <= i
    if pattern == STRIDED:
        a1 = (j >= np.maximum(0, i - l)) & (j <= i)
        a2 = ((i - j) % l) == 0
    else:
        a1 = (j // l) == (i // l)
        a2 = ((j % l) >= (l - (s + 1) * c)) & ((j % l) < (l - s * c))
    if part == 0:
        m = a1
    elif part == 1:
        m = a2
    else:
        m = a1 | a2
    return m & causal


def head_mask(pattern, mode, h, n, l, c):
    part = mode if mode < 3 else (0 if h % 2 == 0 else 1)
    s = h % (l // c) if pattern == FIXED_PER_HEAD else 0
    return part_mask(pattern, part, n, l, c, s)


def attention(q, k, v, mask, scale):
    """Dense masked softmax attention of one head, fp64; empty rows give O=0, LSE=-inf."""
    s = scale * (q @ k.T)
    s = np.where(mask, s, -np.inf)
    m = s.max(axis=1, keepdims=True)
    empty = ~mask.any(axis=1)
    m = np.where(empty[:, None], 0.0, m)
    e = np.where(mask, np.exp(s - m), 0.0)
    z = e.sum(axis=1, keepdims=True)
    p = np.where(empty[:, None], 0.0, e / np.where(z == 0, 1.0, z))
    o = p @ v
    with np.errstate(divide="ignore"):
        lse = np.where(empty, -np.inf, m[:, 0] + np.log(np.where(z[:, 0] == 0, 1.0, z[:, 0])))
    return o, lse, p


def attention_grads(q, k, v, dout, mask, scale):
    """Dense gradients of sum(O * dout) for one head, fp64."""
    o, lse, p = attention(q, k, v, mask, scale)
    dv = p.T @ dout
    dp = dout @ v.T
    delta = (dout * o).sum(axis=1, keepdims=True)
    ds = p * (dp - delta)
    dq = scale * ds @ k
    dk = scale * ds.T @ q
    return o, lse, dq, dk, dv
