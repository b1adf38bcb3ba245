"""C-ABI checks that need no GPU: the library loads, exports every function
the header declares, validates arguments before touching device memory, and
its host-side layout size query agrees with the oracle's brute force."""
import ctypes
import os
import re

import pytest

from paper_1904_10509_amd import sparse_attn as sa

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sparse_attn.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(sa.LIB_PATH):
        from paper_1904_10509_amd import build
        build.build()
    return sa.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(sparse_attn_\w+)\s*\(", text, flags=re.M)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert set(names) == set(sa.EXPORTED), names
    for name in names:
        assert hasattr(L, name), name


def test_status_strings(L):
    assert sa.status_string(0) == "success"
    for code in (-1, -2, -3, -4):
        assert sa.status_string(code) not in ("success", "unknown status")
    assert sa.status_string(7) == "unknown status"


SIZE_CASES = [
    (256, 16, 16, 0, 0, 2), (256, 16, 16, 0, 0, 0), (256, 16, 16, 0, 0, 1), (256, 16, 16, 0, 0, 3),
    (384, 32, 7, 0, 0, 2), (128, 16, 1, 0, 0, 2), (128, 32, 500, 0, 0, 0), (64, 64, 9, 0, 0, 1),
    (3072, 32, 128, 32, 1, 3), (240, 16, 20, 1, 1, 2), (192, 64, 24, 10, 1, 1), (128, 16, 500, 3, 1, 2),
    (512, 64, 256, 32, 1, 2), (512, 16, 48, 48, 1, 3), (12288, 64, 128, 0, 0, 2),
    (65536, 64, 256, 32, 1, 2),
    # distinct summary subblocks per head (pattern 2)
    (256, 16, 32, 8, 2, 0), (256, 16, 32, 8, 2, 1), (256, 64, 128, 32, 2, 2), (240, 16, 20, 6, 2, 3),
    (512, 64, 256, 32, 2, 3), (65536, 64, 128, 32, 2, 2), (128, 16, 16, 16, 2, 2),
]


@pytest.mark.parametrize("n,B,l,c,pattern,mode", SIZE_CASES)
def test_layout_size_matches_oracle(L, orc, n, B, l, c, pattern, mode):
    ng, nnz = sa.sparse_attn_layout_size(n, B, l, c, pattern, mode)
    lay = orc.layout(n, B, l, c, pattern, mode)
    assert ng == lay["n_layouts"]
    assert list(nnz) == list(lay["nnz"])


@pytest.mark.parametrize("args", [
    (100, 16, 8, 0, 0, 2),    # n not a multiple of block
    (256, 24, 8, 0, 0, 2),    # block not supported
    (256, 16, 0, 0, 0, 2),    # l < 1
    (256, 16, 8, 3, 0, 2),    # c given for strided
    (256, 16, 8, 0, 1, 2),    # c = 0 for fixed
    (256, 16, 8, 9, 1, 2),    # c > l
    (256, 16, 8, 0, 2, 2),    # c = 0 for fixed with subblocks per head
    (256, 16, 8, 9, 2, 2),    # c > l
    (256, 16, 8, 0, 3, 2),    # unknown pattern
    (256, 16, 8, 0, 0, 4),    # unknown mode
    (0, 16, 8, 0, 0, 2),      # n < 1
])
def test_layout_size_rejects_invalid(L, args):
    ng = ctypes.c_int32(0)
    nnz = (ctypes.c_int64 * 2)()
    assert L.sparse_attn_layout_size(*args, ctypes.byref(ng), nnz) == sa.SA_ERR_INVALID


def test_layout_count(L):
    ng = ctypes.c_int32(0)
    for (l, c, pattern, mode), expect in [((16, 0, 0, 2), 1), ((16, 0, 0, 3), 2), ((16, 4, 1, 3), 2),
                                          ((16, 4, 2, 0), 1), ((16, 4, 2, 1), 4), ((16, 4, 2, 2), 4),
                                          ((16, 4, 2, 3), 5), ((20, 6, 2, 2), 3), ((128, 2, 2, 3), 65)]:
        assert L.sparse_attn_layout_count(l, c, pattern, mode, ctypes.byref(ng)) == 0
        assert ng.value == expect, (l, c, pattern, mode)
    # more than 64 subblocks per block, or a missing output
    assert L.sparse_attn_layout_count(130, 2, 2, 2, ctypes.byref(ng)) == sa.SA_ERR_UNSUPPORTED
    assert L.sparse_attn_layout_count(16, 4, 2, 2, None) == sa.SA_ERR_INVALID
    nnz = (ctypes.c_int64 * 2)()
    assert L.sparse_attn_layout_size(256, 16, 130, 2, 2, 2, ctypes.byref(ng), nnz) == sa.SA_ERR_UNSUPPORTED


FAKE = 0x100000  # never dereferenced: every call below fails validation first


def _fwd(L, **over):
    args = dict(n=256, block=16, l=16, c=0, pattern=0, mode=2, row_ptr=FAKE, col_idx=FAKE, kind=FAKE,
                batch=1, heads=1, d=32, dtype=sa.SA_BF16, q=FAKE, k=FAKE, v=FAKE,
                strides=(ctypes.c_int64 * 3)(8192, 8192, 32), scale=0.25, o=FAKE, lse=FAKE, stream=None)
    args.update(over)
    return L.sparse_attn_fwd(*args.values())


@pytest.mark.parametrize("over,expect", [
    (dict(n=250), sa.SA_ERR_INVALID),
    (dict(c=4), sa.SA_ERR_INVALID),
    (dict(d=48), sa.SA_ERR_UNSUPPORTED),
    (dict(dtype=5), sa.SA_ERR_INVALID),
    (dict(batch=0), sa.SA_ERR_INVALID),
    (dict(q=None), sa.SA_ERR_INVALID),
    (dict(lse=None), sa.SA_ERR_INVALID),
    (dict(row_ptr=None), sa.SA_ERR_INVALID),
    (dict(o=FAKE + 8), sa.SA_ERR_INVALID),                                  # misaligned
    (dict(strides=(ctypes.c_int64 * 3)(8192, 8192, 36)), sa.SA_ERR_INVALID),  # stride not 16-byte
    (dict(strides=(ctypes.c_int64 * 3)(8192, 8192, 16)), sa.SA_ERR_INVALID),  # rows overlap
    (dict(strides=None), sa.SA_ERR_INVALID),
    # bf16 tiles are staged with 32-bit byte offsets: block rows of the sequence stride must span < 4 GiB
    (dict(strides=(ctypes.c_int64 * 3)(1 << 40, 1 << 40, 1 << 27)), sa.SA_ERR_UNSUPPORTED),
    (dict(scale=float("nan")), sa.SA_ERR_INVALID),
])
def test_fwd_rejects_invalid(L, over, expect):
    assert _fwd(L, **over) == expect


def test_bwd_workspace_and_errors(L):
    out = ctypes.c_size_t(0)
    assert L.sparse_attn_bwd_workspace_size(256, 16, 16, 0, 0, 2, 2, 3, 64, sa.SA_BF16, ctypes.byref(out)) == 0
    # D_i and the base-2 LSE per row, 8 queue counters, the item count of the
    # one layout, its item order (two slots per key block)
    assert out.value == 2 * 2 * 3 * 256 * 4 + 8 * 8 + 4 + 2 * 4 * (256 // 16)
    assert L.sparse_attn_bwd_workspace_size(256, 16, 16, 0, 0, 2, 2, 3, 64, sa.SA_F32, ctypes.byref(out)) == 0
    assert out.value == 2 * 2 * 3 * 256 * 4 + 8 * 8 + 4 + 2 * 4 * (256 // 16)
    assert L.sparse_attn_bwd_workspace_size(256, 16, 16, 8, 1, 3, 2, 3, 64, sa.SA_BF16, ctypes.byref(out)) == 0
    assert out.value == 2 * 2 * 3 * 256 * 4 + 8 * 8 + 2 * (4 + 2 * 4 * (256 // 16))  # interleaved: two layouts
    assert L.sparse_attn_bwd_workspace_size(256, 16, 16, 4, 2, 3, 2, 3, 64, sa.SA_BF16, ctypes.byref(out)) == 0
    assert out.value == 2 * 2 * 3 * 256 * 4 + 8 * 8 + 5 * (4 + 2 * 4 * (256 // 16))  # A1 + four subblocks
    assert L.sparse_attn_bwd_workspace_size(256, 16, 16, 0, 0, 2, 2, 3, 40, sa.SA_F32, ctypes.byref(out)) == \
        sa.SA_ERR_UNSUPPORTED
    strides = (ctypes.c_int64 * 3)(256 * 64, 256 * 64, 64)
    common = [256, 16, 16, 0, 0, 2] + [FAKE] * 6 + [1, 1, 64, sa.SA_BF16] + [FAKE] * 6 + [strides, 0.125] + [FAKE] * 3
    need = 2 * 256 * 4 + 8 * 8 + 4 + 2 * 4 * (256 // 16)
    assert L.sparse_attn_bwd(*common, FAKE, need - 1, None) == sa.SA_ERR_BUFFER_TOO_SMALL
    assert L.sparse_attn_bwd(*common, None, need, None) == sa.SA_ERR_INVALID
    bad = list(common)
    bad[6 + 3] = None  # col_ptr
    assert L.sparse_attn_bwd(*bad, FAKE, need, None) == sa.SA_ERR_INVALID


def test_layout_rejects_small_capacity(L):
    _, nnz = sa.sparse_attn_layout_size(256, 16, 16, 0, 0, 2)
    assert L.sparse_attn_layout(256, 16, 16, 0, 0, 2, *([FAKE] * 6), nnz[0] - 1, None) == sa.SA_ERR_BUFFER_TOO_SMALL
    assert L.sparse_attn_layout(256, 16, 16, 0, 0, 2, *([FAKE] * 5), None, nnz[0], None) == sa.SA_ERR_INVALID


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(sa, "_lib", None)
    monkeypatch.setattr(sa, "LIB_PATH", str(tmp_path / "absent.so"))
    with pytest.raises(RuntimeError, match="not built"):
        sa.lib()



def test_decode_workspace_and_errors(L):
    out = ctypes.c_size_t(0)
    # fixed, pos 65,535, l 256, c 32: |S_pos| = 256 + 255 * 32 = 8,416 keys, 33 ranges of up to 256 keys,
    # (64 + 2) fp32 per range and (batch, head)
    assert L.sparse_attn_decode_workspace_size(65535, 256, 32, sa.SA_FIXED, sa.SA_MODE_MERGED, 1, 8, 64, sa.SA_BF16,
                                               ctypes.byref(out)) == 0
    assert out.value == 8 * 33 * 66 * 4
    # a single range when the set is small; ranges capped at 4,096 workgroups in all
    assert L.sparse_attn_decode_workspace_size(5, 16, 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, 2, 3, 32, sa.SA_F32,
                                               ctypes.byref(out)) == 0
    assert out.value == 6 * 1 * 34 * 4
    assert L.sparse_attn_decode_workspace_size(2**31 - 1, 2**31 - 1, 0, sa.SA_STRIDED, sa.SA_MODE_A1, 64, 8, 128,
                                               sa.SA_BF16, ctypes.byref(out)) == 0
    assert out.value == 64 * 8 * 8 * 130 * 4
    # subblocks per head, A2 at pos 65,335 (position 55 of its block): subblock 7 (positions 0..31) holds
    # 255 * 32 + 32 = 8,192 keys, the most of any head: 32 ranges
    assert L.sparse_attn_decode_workspace_size(65335, 256, 32, sa.SA_FIXED_PER_HEAD, sa.SA_MODE_A2, 1, 8, 64,
                                               sa.SA_BF16, ctypes.byref(out)) == 0
    assert out.value == 8 * 32 * 66 * 4
    assert L.sparse_attn_decode_workspace_size(10, 256, 2, sa.SA_FIXED_PER_HEAD, sa.SA_MODE_A2, 1, 8, 64,
                                               sa.SA_BF16, ctypes.byref(out)) == sa.SA_ERR_UNSUPPORTED
    bad = [
        (-1, 16, 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, 1, 1, 64, sa.SA_BF16, sa.SA_ERR_INVALID),
        (2**31, 16, 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, 1, 1, 64, sa.SA_BF16, sa.SA_ERR_INVALID),
        (10, 0, 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, 1, 1, 64, sa.SA_BF16, sa.SA_ERR_INVALID),
        (10, 16, 0, sa.SA_FIXED, sa.SA_MODE_MERGED, 1, 1, 64, sa.SA_BF16, sa.SA_ERR_INVALID),
        (10, 16, 17, sa.SA_FIXED, sa.SA_MODE_MERGED, 1, 1, 64, sa.SA_BF16, sa.SA_ERR_INVALID),
        (10, 16, 4, sa.SA_STRIDED, sa.SA_MODE_MERGED, 1, 1, 64, sa.SA_BF16, sa.SA_ERR_INVALID),
        (10, 16, 0, sa.SA_STRIDED, 4, 1, 1, 64, sa.SA_BF16, sa.SA_ERR_INVALID),
        (10, 16, 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, 0, 1, 64, sa.SA_BF16, sa.SA_ERR_INVALID),
        (10, 16, 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, 1, 1, 48, sa.SA_BF16, sa.SA_ERR_UNSUPPORTED),
        (10, 16, 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, 1, 1, 64, 7, sa.SA_ERR_INVALID),
    ]
    for *args, expect in bad:
        assert L.sparse_attn_decode_workspace_size(*args, ctypes.byref(out)) == expect, args
    assert L.sparse_attn_decode_workspace_size(10, 16, 0, 0, 2, 1, 1, 64, 1, None) == sa.SA_ERR_INVALID
    # validation before any launch: bad strides, alignment, workspace, scale (fake device pointers)
    qs = (ctypes.c_int64 * 2)(64, 64)
    ks = (ctypes.c_int64 * 3)(64 * 64, 64 * 64, 64)
    need = 1 * 1 * 1 * 66 * 4
    base = [10, 16, 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, 1, 1, 64, sa.SA_BF16]

    def call(q=FAKE, qst=qs, k=FAKE, v=FAKE, kst=ks, scale=0.125, o=FAKE, lse=FAKE, ws=FAKE, wsb=need):
        return L.sparse_attn_decode(*base, q, qst, k, v, kst, scale, o, lse, ws, wsb, None)

    assert call(q=None) == sa.SA_ERR_INVALID
    assert call(q=FAKE + 2) == sa.SA_ERR_INVALID
    assert call(qst=(ctypes.c_int64 * 2)(60, 64)) == sa.SA_ERR_INVALID
    assert call(kst=(ctypes.c_int64 * 3)(64 * 64, 64 * 64, 32)) == sa.SA_ERR_INVALID
    assert call(scale=float("nan")) == sa.SA_ERR_INVALID
    assert call(scale=-1.0) == sa.SA_ERR_INVALID
    assert call(wsb=need - 1) == sa.SA_ERR_BUFFER_TOO_SMALL
    assert call(ws=None) == sa.SA_ERR_INVALID


def test_transposed_workspace_and_errors(L):
    """Workspace of the merged transposed path: the band backward's (row
    statistics and dK / dV schedule, as sparse_attn_bwd); the class kernels
    read the same row statistics in place."""
    def bwd_ws(rows, nq):
        return (8 * rows + 15) // 16 * 16 + 8 * 8 + 4 + 2 * 4 * nq

    out = ctypes.c_size_t(0)
    n, B, l, CB, b, h, d = 12288, 64, 128, 32, 2, 8, 64
    assert L.sparse_attn_transposed_workspace_size(n, B, l, CB, b, h, d, sa.SA_BF16, ctypes.byref(out)) == 0
    rows = b * h * n
    assert out.value == bwd_ws(rows, n // B)
    bad = [
        ((12288, 64, 100, 32, 2, 8, 64, sa.SA_BF16), sa.SA_ERR_INVALID),      # l does not divide n
        ((12288, 64, 128, 24, 2, 8, 64, sa.SA_BF16), sa.SA_ERR_INVALID),      # class block not supported
        ((12288, 64, 256, 64, 2, 8, 64, sa.SA_BF16), sa.SA_ERR_INVALID),      # 48 class positions, blocks of 64
        ((12288, 64, 128, 32, 2, 8, 48, sa.SA_BF16), sa.SA_ERR_UNSUPPORTED),  # d
        ((12288, 64, 128, 32, 0, 8, 64, sa.SA_BF16), sa.SA_ERR_INVALID),      # batch
        ((12288, 64, 128, 32, 256, 256, 64, sa.SA_BF16), sa.SA_ERR_UNSUPPORTED),  # batch * heads > 65,535
        ((2 ** 20 * 16, 64, 16, 16, 1, 1, 64, sa.SA_BF16), sa.SA_ERR_UNSUPPORTED),  # 65,536 class block rows
    ]
    for args, expect in bad:
        assert L.sparse_attn_transposed_workspace_size(*args, ctypes.byref(out)) == expect, args
    assert L.sparse_attn_transposed_workspace_size(n, B, l, CB, b, h, d, sa.SA_BF16, None) == sa.SA_ERR_INVALID
    # validation before any launch: workspace size and alignment, scale, pointers (fake device pointers)
    L.sparse_attn_transposed_workspace_size(n, B, l, CB, b, h, d, sa.SA_BF16, ctypes.byref(out))
    need = out.value
    fwd = [n, B, l, CB] + [FAKE] * 3 + [b, h, d, sa.SA_BF16] + [FAKE] * 3 + [0.125] + [FAKE] * 2
    assert L.sparse_attn_fwd_transposed(*fwd, FAKE, need - 1, None) == sa.SA_ERR_BUFFER_TOO_SMALL
    assert L.sparse_attn_fwd_transposed(*fwd, FAKE + 16, need, None) == sa.SA_ERR_INVALID  # not 256-aligned
    assert L.sparse_attn_fwd_transposed(*fwd, None, need, None) == sa.SA_ERR_INVALID
    bad_scale = list(fwd)
    bad_scale[14] = 0.0
    assert L.sparse_attn_fwd_transposed(*bad_scale, FAKE, need, None) == sa.SA_ERR_INVALID
    bwd = [n, B, l, CB] + [FAKE] * 6 + [b, h, d, sa.SA_BF16] + [FAKE] * 6 + [0.125] + [FAKE] * 3
    assert L.sparse_attn_bwd_transposed(*bwd, FAKE, need - 1, None) == sa.SA_ERR_BUFFER_TOO_SMALL
    no_col = list(bwd)
    no_col[7] = None
    assert L.sparse_attn_bwd_transposed(*no_col, FAKE, need, None) == sa.SA_ERR_INVALID


def test_transposed_binding_rejects_strided_views():
    """The transposed entry points take no strides; the binding refuses views
    that are not contiguous before anything reaches the library."""
    import torch
    q = torch.zeros(1, 2, 64, 32, dtype=torch.bfloat16)
    band = sa.Layout(64, 16, 16, 0, sa.SA_STRIDED, sa.SA_MODE_A1, 1, [1], *([torch.zeros(1)] * 6))
    view = torch.zeros(1, 2, 64, 64, dtype=torch.bfloat16)[..., :32]
    with pytest.raises(ValueError, match="contiguous"):
        sa.forward_merged_transposed(q, view, q, band, 16)
    with pytest.raises(ValueError, match="strided A1"):
        sa.forward_merged_transposed(q, q, q, sa.Layout(64, 16, 16, 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, 1, [1],
                                                        *([torch.zeros(1)] * 6)), 16)


def test_noalloc_rejects_workspace_beyond_scratch(L):
    """The allocation-free backward refuses a call whose workspace would exceed
    its fixed scratch (here 16 heads x 2^20 rows, 8 bytes of row statistics
    each: 128 MiB), before touching any memory or the device."""
    n, heads, d = 1 << 20, 16, 64
    need = sa.sparse_attn_bwd_workspace_size(n, 64, 1024, 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, 1, heads, d,
                                             sa.SA_BF16)
    assert need > sa.sparse_attn_bwd_noalloc_max_workspace()
    fake = ctypes.c_void_p(1 << 20)  # never dereferenced: the size check comes first
    strides = (ctypes.c_int64 * 3)(heads * n * d, n * d, d)
    st = L.sparse_attn_bwd_noalloc(n, 64, 1024, 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, *([fake] * 6), 1, heads, d,
                                   sa.SA_BF16, *([fake] * 6), strides, ctypes.c_float(0.125), *([fake] * 3), None)
    assert st == sa.SA_ERR_BUFFER_TOO_SMALL


def test_bwd_stage_validation(L):
    """Stage sets: empty or unknown sets are invalid; fp32 runs only whole."""
    n, B, l, b, h, d = 256, 32, 32, 1, 2, 64
    need = sa.sparse_attn_bwd_workspace_size(n, B, l, 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, b, h, d, sa.SA_BF16)
    fake = ctypes.c_void_p(1 << 20)
    strides = (ctypes.c_int64 * 3)(h * n * d, n * d, d)

    def call(stages, dtype=sa.SA_BF16):
        return L.sparse_attn_bwd_stage(n, B, l, 0, sa.SA_STRIDED, sa.SA_MODE_MERGED, *([fake] * 6), b, h, d, dtype,
                                       *([fake] * 6), strides, ctypes.c_float(0.125), *([fake] * 3), fake, need,
                                       stages, None)
    assert call(0) == sa.SA_ERR_INVALID
    assert call(8) == sa.SA_ERR_INVALID
    assert call(-1) == sa.SA_ERR_INVALID
    assert call(sa.SA_BWD_DQ, sa.SA_F32) == sa.SA_ERR_UNSUPPORTED


def test_probe_library_exports(L):
    """The measurement probes bench.py loads (matrix-core rate and clock, LDS
    read rate, XCD placement, direct-to-LDS read calibration) are exported and
    reject invalid launches before touching a GPU."""
    path = os.path.join(ROOT, "paper_1904_10509_amd", "libsa_probe.so")
    if not os.path.exists(path):
        from paper_1904_10509_amd import build
        build.build()
    P = ctypes.CDLL(path)
    for sym in ("sa_probe_mfma_flop", "sa_probe_mfma_launch", "sa_probe_lds_bytes", "sa_probe_lds_launch",
                "sa_probe_xcd_map_launch", "sa_probe_dma_read_launch"):
        assert hasattr(P, sym), sym
    P.sa_probe_lds_bytes.restype = ctypes.c_double
    P.sa_probe_lds_bytes.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int]
    assert P.sa_probe_lds_bytes(0, 2, 3) == 2 * 256 * 3 * 8 * 16
    assert P.sa_probe_lds_bytes(1, 2, 3) == 2 * 256 * 3 * 8 * 8
    P.sa_probe_lds_launch.restype = ctypes.c_int
    P.sa_probe_lds_launch.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_void_p]
    assert P.sa_probe_lds_launch(2, 1, 1, None, None, None) == -1  # unknown read form
    assert P.sa_probe_lds_launch(0, 0, 1, None, None, None) == -1  # no workgroups
    P.sa_probe_xcd_map_launch.restype = ctypes.c_int
    P.sa_probe_xcd_map_launch.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    assert P.sa_probe_xcd_map_launch(0, None, None, None) == -1
    P.sa_probe_dma_read_launch.restype = ctypes.c_int
    P.sa_probe_dma_read_launch.argtypes = [ctypes.c_int, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p,
                                           ctypes.c_void_p]
    assert P.sa_probe_dma_read_launch(1, 0, None, None, None) == -1
