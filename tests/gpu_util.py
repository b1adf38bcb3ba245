"""Helpers for the GPU parity tests: run the HIP path through the C ABI and
bring results back as float64 numpy arrays."""
import numpy as np
import torch

from paper_1904_10509_amd import sparse_attn as sa
from paper_1904_10509_amd.inputs import as_oracle_array, make_inputs

TOL = {torch.float32: 1e-5, torch.bfloat16: 2e-2}
LSE_TOL = {torch.float32: 1e-5, torch.bfloat16: 1e-3}


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


def max_err(a, b):
    """Largest |a - b| / max(1, |b|) with b the oracle: an absolute error for
    values up to 1 and a relative one above (a bf16 value of magnitude 2..4
    alone carries a rounding error of up to 2^-7).  -inf must meet -inf."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    both_inf = np.isneginf(a) & np.isneginf(b)
    if np.any(np.isneginf(a) != np.isneginf(b)):
        return float("inf")
    a0, b0 = np.where(both_inf, 0.0, a), np.where(both_inf, 0.0, b)
    d = np.abs(a0 - b0) / np.maximum(1.0, np.abs(b0))
    return float(d.max()) if d.size else 0.0
