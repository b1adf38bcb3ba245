"""Seeded synthetic inputs and the named workloads.

This module holds no attention arithmetic.  It is the one piece shared by the
GPU path's callers and the oracle's callers: both receive the same tensors.

Recipe: a CPU ``torch.Generator`` seeded with the workload's seed draws
``randn`` for Q, K, V and dO, in that order, as fp32 of shape [b, h, n, d];
the tensors are then cast to the workload's dtype (round to nearest even for
bf16).  These N(0, 1) tensors stand in for projected activations of the
datasets the paper trains on (CIFAR-10 images, EnWik8 text, classical-music
audio), whose sequence shapes the workloads reuse.
"""
from dataclasses import dataclass, field

import numpy as np
import torch

STRIDED, FIXED, FIXED_PER_HEAD = 0, 1, 2
MODE_A1, MODE_A2, MODE_MERGED, MODE_INTERLEAVED = 0, 1, 2, 3
F32, BF16 = 0, 1


@dataclass(frozen=True)
class Workload:
    name: str
    pattern: int
    mode: int
    n: int
    stride: int
    summary: int
    block: int
    batch: int
    heads: int
    d_head: int
    dtype: int
    seed: int
    note: str = field(default="", compare=False)

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == F32 else torch.bfloat16

    @property
    def scale(self) -> float:
        return 1.0 / float(self.d_head) ** 0.5

    def describe(self) -> dict:
        return {
            "workload": self.name,
            "pattern": ["strided", "fixed", "fixed_per_head"][self.pattern],
            "mode": ["A1", "A2", "merged", "interleaved"][self.mode],
            "n": self.n, "stride": self.stride, "summary": self.summary,
            "block": self.block, "batch": self.batch, "heads": self.heads,
            "d_head": self.d_head, "dtype": "f32" if self.dtype == F32 else "bf16",
            "seed": self.seed,
        }


WORKLOADS = {
    w.name: w for w in [
        Workload("strided_n256_l16_f32", STRIDED, MODE_MERGED, 256, 16, 0, 16, 1, 1, 32, F32, 1,
                 "small parity / finite-difference case"),
        Workload("fixed_n3072_l128_c32_interleaved", FIXED, MODE_INTERLEAVED, 3072, 128, 32, 32,
                 4, 2, 128, BF16, 2, "32x32x3 image raster; head 0 uses A1, head 1 uses A2"),
        Workload("strided_n12288_l128_merged", STRIDED, MODE_MERGED, 12288, 128, 0, 64, 2, 8, 64,
                 BF16, 3, "text context of 12,288 with 8 heads of 64"),
        Workload("fixed_n65536_l256_c32_merged", FIXED, MODE_MERGED, 65536, 256, 32, 64, 1, 8, 64,
                 BF16, 4, "audio sequence of 65,536"),
        Workload("strided_n1048576_l1024_merged", STRIDED, MODE_MERGED, 1048576, 1024, 0, 64, 1, 4,
                 64, BF16, 5, "audio sequence of 1,048,576"),
        # dense against sparse at the two contexts of the paper's Table 2 (text of
        # 12,288: 8 heads of 64; image of 3,072: 2 heads of 128); dense causal
        # attention is the strided pattern with a stride of n (A1 then covers j <= i)
        Workload("dense_n12288_merged", STRIDED, MODE_MERGED, 12288, 12288, 0, 64, 2, 8, 64, BF16, 6,
                 "dense causal limit at the text context of 12,288"),
        Workload("fixed_n12288_l128_c32_merged", FIXED, MODE_MERGED, 12288, 128, 32, 64, 2, 8, 64, BF16, 7,
                 "text context of 12,288, fixed pattern with the paper's text settings"),
        Workload("dense_n3072_merged", STRIDED, MODE_MERGED, 3072, 3072, 0, 64, 4, 2, 128, BF16, 8,
                 "dense causal limit at the image context of 3,072"),
        Workload("fixed_n3072_l128_c32_merged", FIXED, MODE_MERGED, 3072, 128, 32, 64, 4, 2, 128, BF16, 9,
                 "image context of 3,072, fixed pattern"),
        Workload("strided_n3072_l128_merged", STRIDED, MODE_MERGED, 3072, 128, 0, 64, 4, 2, 128, BF16, 10,
                 "image context of 3,072, strided pattern"),
        # the fixed pattern with a distinct summary subblock per head (head h
        # uses positions l-(s+1)c .. l-sc-1 of each block, s = h mod l/c)
        Workload("fixed_per_head_n65536_l256_c32_merged", FIXED_PER_HEAD, MODE_MERGED, 65536, 256, 32, 64, 1, 8,
                 64, BF16, 11, "audio sequence of 65,536; the 8 heads take the 8 subblocks of each block"),
        Workload("fixed_per_head_n12288_l128_c32_merged", FIXED_PER_HEAD, MODE_MERGED, 12288, 128, 32, 64, 2, 8,
                 64, BF16, 12, "text context of 12,288; 8 heads over 4 subblocks"),
    ]
}


def make_inputs(batch, heads, n, d, dtype=torch.bfloat16, seed=0):
    """Q, K, V, dO as CPU tensors [b, h, n, d] of the given dtype."""
    g = torch.Generator().manual_seed(int(seed))
    shape = (batch, heads, n, d)
    out = {}
    for name in ("q", "k", "v", "dout"):
        out[name] = torch.randn(shape, generator=g, dtype=torch.float32).to(dtype)
    return out


def workload_inputs(w: Workload):
    return make_inputs(w.batch, w.heads, w.n, w.d_head, w.torch_dtype, w.seed)


def as_oracle_array(t: torch.Tensor) -> np.ndarray:
    """CPU tensor -> numpy array the oracle reads (bf16 as raw uint16 bits)."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    if t.dtype in (torch.float32, torch.float64):
        return t.numpy()
    raise TypeError(f"unsupported dtype {t.dtype}")
