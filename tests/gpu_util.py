"""Helpers for the GPU parity tests: run the HIP path through the C ABI, bring
results back as float64 numpy arrays, and compare them with the oracle.

The bar: elementwise, |gpu - oracle| <= tol + half an ulp of the output's
element type at |oracle|, with tol = 1e-5 (fp32) or 2e-2 (bf16) for O, dQ,
dK, dV and 1e-5 / 1e-3 for the fp32 LSE.  The half ulp is the rounding of
the stored output itself (a bf16 value of magnitude 2 .. 4 is stored to
within 2^-7); everything else must fit the absolute tolerance.  Every check
prints, and records for the session summary, the max-abs error per tensor.
"""
import numpy as np
import torch

from paper_1904_10509_amd import sparse_attn as sa
from paper_1904_10509_amd.inputs import as_oracle_array, make_inputs  # noqa: F401

TOL = {torch.float32: 1e-5, torch.bfloat16: 2e-2}
LSE_TOL = {torch.float32: 1e-5, torch.bfloat16: 1e-3}
_PRECISION = {torch.float32: 24, torch.bfloat16: 8}  # significand bits, implicit bit included

# (label, max-abs error, tolerance, worst margin) of every check, in order
RESULTS = []


def device():
    if not torch.cuda.is_available():
        import pytest
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def to64(t):
    return t.detach().float().cpu().numpy().astype(np.float64) if t.dtype != torch.float32 else \
        t.detach().cpu().numpy().astype(np.float64)


def run_gpu(x, *, n, block, l, c, pattern, mode, scale, backward=True, dev=None):
    """x: dict of CPU tensors q, k, v, dout.  Returns dict of float64 arrays."""
    dev = dev or device()
    lay = sa.build_layout(n, block, l, c, pattern, mode, device=dev)
    q, k, v, dout = (x[name].to(dev) for name in ("q", "k", "v", "dout"))
    o, lse = sa.forward(q, k, v, lay, scale)
    out = {"o": o, "lse": lse}
    if backward:
        dq, dk, dv = sa.backward(q, k, v, o, dout, lse, lay, scale)
        out.update(dq=dq, dk=dk, dv=dv)
    torch.cuda.synchronize()
    return {name: to64(t) for name, t in out.items()}


def oracle_inputs(x):
    return [as_oracle_array(x[name]) for name in ("q", "k", "v", "dout")]


def half_ulp(ref, dtype):
    """Half a unit in the last place of `dtype` at |ref| (0 at ref = 0)."""
    a = np.abs(np.asarray(ref, dtype=np.float64))
    e = np.floor(np.log2(np.where(a > 0, a, 1.0))).astype(np.int64)
    return np.where(a > 0, np.ldexp(1.0, e - _PRECISION[dtype]), 0.0)


def compare(got, ref, tol, dtype):
    """(max |got - ref|, max of |got - ref| - tol - half_ulp(ref)) over the
    elements; -inf must meet -inf exactly (empty rows' LSE), NaN fails."""
    g = np.asarray(got, dtype=np.float64)
    r = np.asarray(ref, dtype=np.float64)
    if g.shape != r.shape:
        raise AssertionError(f"shape {g.shape} against {r.shape}")
    if np.any(np.isneginf(g) != np.isneginf(r)):
        return float("inf"), float("inf")
    fin = ~np.isneginf(r)
    d = np.abs(g[fin] - r[fin])
    if d.size == 0:
        return 0.0, -tol
    if np.isnan(d).any():
        return float("nan"), float("inf")
    excess = d - tol - half_ulp(r[fin], dtype)
    return float(d.max()), float(excess.max())


def check(label, got, ref, dtype, tol=None, out_dtype=None):
    """Assert the bar above for one tensor; prints and records its max-abs error.
    dtype: the input element type (picks tol); out_dtype: the stored output's
    element type (picks the half ulp), dtype unless given."""
    tol = TOL[dtype] if tol is None else tol
    md, ex = compare(got, ref, tol, dtype if out_dtype is None else out_dtype)
    RESULTS.append((label, md, tol, -ex))
    print(f"parity {label}: max-abs err {md:.3e} (tol {tol:g} + half ulp), margin {-ex:.3e}", flush=True)
    assert ex <= 0.0, f"{label}: max-abs err {md:.3e}, exceeds tol {tol:g} + half ulp by {ex:.3e}"
    return md


def check_lse(label, got, ref, dtype):
    """LSE is stored in fp32 whatever the input type."""
    return check(label, got, ref, dtype, tol=LSE_TOL[dtype], out_dtype=torch.float32)


def check_all(label, got, ref, dtype, names=("o", "dq", "dk", "dv")):
    for name in names:
        if name == "lse":
            check_lse(f"{label} lse", got[name], ref[name], dtype)
        else:
            check(f"{label} {name}", got[name], ref[name], dtype)
