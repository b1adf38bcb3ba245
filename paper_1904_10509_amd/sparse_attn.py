"""ctypes binding of libsparse_attn.so (include/sparse_attn.h).

The functions named like the C entry points only marshal arguments: every
step of the computation runs in the library's HIP kernels.  PyTorch supplies
device memory and the current stream.  The convenience layer below them
(``build_layout``, ``forward``, ``backward``, ``SparseAttention``) allocates
outputs with torch and calls those same entry points.

Loading fails loudly when the library has not been built; there is no
fallback implementation.
"""
import ctypes
import math
import os
from dataclasses import dataclass

import torch

# SPARSE_ATTN_LIB names another build of the same sources to load instead (the
# sanitizer test loads one whose host code is built with ASan and UBSan).
LIB_PATH = os.environ.get("SPARSE_ATTN_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)),
                                                              "libsparse_attn.so")

SA_OK, SA_ERR_INVALID, SA_ERR_UNSUPPORTED, SA_ERR_BUFFER_TOO_SMALL, SA_ERR_HIP = 0, -1, -2, -3, -4
SA_STRIDED, SA_FIXED, SA_FIXED_PER_HEAD = 0, 1, 2
SA_MODE_A1, SA_MODE_A2, SA_MODE_MERGED, SA_MODE_INTERLEAVED = 0, 1, 2, 3
SA_F32, SA_BF16 = 0, 1
SA_TILE_FULL, SA_TILE_MASKED = 0, 1
SA_BWD_ROW_STATS, SA_BWD_DQ, SA_BWD_DKDV, SA_BWD_ALL_STAGES = 1, 2, 4, 7

EXPORTED = (
    "sparse_attn_layout_count",
    "sparse_attn_layout_size",
    "sparse_attn_layout",
    "sparse_attn_fwd",
    "sparse_attn_bwd_workspace_size",
    "sparse_attn_bwd",
    "sparse_attn_decode_workspace_size",
    "sparse_attn_decode",
    "sparse_attn_transposed_workspace_size",
    "sparse_attn_fwd_transposed",
    "sparse_attn_bwd_transposed",
    "sparse_attn_bwd_stage",
    "sparse_attn_bwd_noalloc_max_workspace",
    "sparse_attn_bwd_noalloc",
    "sparse_attn_status_string",
)

_lib = None
_i32, _i64, _f32, _vp, _sz = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t
_PAT = [_i64, _i32, _i32, _i32, _i32, _i32]  # n, block, stride_l, summary_c, pattern, head_mode


class SparseAttnError(RuntimeError):
    def __init__(self, func, status):
        self.status = status
        super().__init__(f"{func} failed: {status_string(status)} ({status})")


def lib():
    """Load the built library (raises if it is missing)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        L.sparse_attn_layout_count.argtypes = [_i32, _i32, _i32, _i32, _vp]
        L.sparse_attn_layout_size.argtypes = _PAT + [_vp, _vp]
        L.sparse_attn_layout.argtypes = _PAT + [_vp] * 6 + [_i64, _vp]
        L.sparse_attn_fwd.argtypes = _PAT + [_vp] * 3 + [_i32] * 4 + [_vp] * 4 + [_f32, _vp, _vp, _vp]
        L.sparse_attn_bwd_workspace_size.argtypes = _PAT + [_i32] * 4 + [_vp]
        L.sparse_attn_bwd.argtypes = (_PAT + [_vp] * 6 + [_i32] * 4 + [_vp] * 7 + [_f32]
                                      + [_vp] * 4 + [_sz, _vp])
        _DEC = [_i64, _i32, _i32, _i32, _i32]  # pos, stride_l, summary_c, pattern, head_mode
        L.sparse_attn_decode_workspace_size.argtypes = _DEC + [_i32] * 4 + [_vp]
        L.sparse_attn_decode.argtypes = _DEC + [_i32] * 4 + [_vp] * 5 + [_f32] + [_vp] * 3 + [_sz, _vp]
        _TR = [_i64, _i32, _i32, _i32]  # n, block, stride_l, class_block
        L.sparse_attn_transposed_workspace_size.argtypes = _TR + [_i32] * 4 + [_vp]
        L.sparse_attn_fwd_transposed.argtypes = _TR + [_vp] * 3 + [_i32] * 4 + [_vp] * 3 + [_f32] + [_vp] * 3 + [_sz, _vp]
        L.sparse_attn_bwd_transposed.argtypes = (_TR + [_vp] * 6 + [_i32] * 4 + [_vp] * 6 + [_f32] + [_vp] * 4
                                                 + [_sz, _vp])
        L.sparse_attn_bwd_stage.argtypes = (_PAT + [_vp] * 6 + [_i32] * 4 + [_vp] * 7 + [_f32]
                                            + [_vp] * 4 + [_sz, _i32, _vp])
        L.sparse_attn_bwd_noalloc_max_workspace.argtypes = [_vp]
        L.sparse_attn_bwd_noalloc.argtypes = (_PAT + [_vp] * 6 + [_i32] * 4 + [_vp] * 7 + [_f32] + [_vp] * 4)
        L.sparse_attn_status_string.argtypes = [ctypes.c_int]
        L.sparse_attn_status_string.restype = ctypes.c_char_p
        for name in EXPORTED[:-1]:
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().sparse_attn_status_string(int(status)).decode()


def _check(func, status):
    if status != SA_OK:
        raise SparseAttnError(func, status)


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream, device):
    if stream is None:
        stream = torch.cuda.current_stream(device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else stream


def _strides(*tensors):
    """Element strides of [batch, heads, n, d] tensors that agree with the
    first in shape, element type, device and strides (d contiguous); raises
    ValueError otherwise, before anything reaches the library."""
    ref = tensors[0]
    if ref.dim() != 4:
        raise ValueError("tensors must be [batch, heads, n, d]")
    st = ref.stride()
    for t in tensors:
        if t.dim() != 4 or t.shape != ref.shape:
            raise ValueError(f"tensor of shape {tuple(t.shape)} where {tuple(ref.shape)} is expected")
        if t.dtype != ref.dtype:
            raise ValueError(f"tensor of type {t.dtype} where {ref.dtype} is expected")
        if t.device != ref.device or t.device.type != "cuda":
            raise ValueError("every tensor must be on the same GPU")
        if t.stride() != st or t.stride(3) != 1:
            raise ValueError("tensors must have d contiguous and identical strides")
    return (ctypes.c_int64 * 3)(st[0], st[1], st[2])


def _check_lse(lse, q):
    b, h, n, _ = q.shape
    if lse.dtype != torch.float32 or tuple(lse.shape) != (b, h, n) or not lse.is_contiguous():
        raise ValueError("lse must be a contiguous float32 [batch, heads, n] tensor")
    if lse.device != q.device:
        raise ValueError("lse must be on q's device")


def _check_layout(layout, q):
    if q.shape[2] != layout.n:
        raise ValueError("sequence length differs from the layout's")
    if layout.row_ptr.device != q.device:
        raise ValueError("the layout must be on q's device")


def _dtype_code(t):
    if t.dtype == torch.bfloat16:
        return SA_BF16
    if t.dtype == torch.float32:
        return SA_F32
    raise TypeError(f"unsupported dtype {t.dtype}")


# ---------------------------------------------------------------------------
# Entry points, same names and argument order as the C ABI
# ---------------------------------------------------------------------------
def sparse_attn_layout_count(stride_l, summary_c, pattern, head_mode):
    ng = ctypes.c_int32(0)
    st = lib().sparse_attn_layout_count(stride_l, summary_c, pattern, head_mode, ctypes.byref(ng))
    _check("sparse_attn_layout_count", st)
    return ng.value


def sparse_attn_layout_size(n, block, stride_l, summary_c, pattern, head_mode):
    entries = max(2, sparse_attn_layout_count(stride_l, summary_c, pattern, head_mode))
    ng = ctypes.c_int32(0)
    nnz = (ctypes.c_int64 * entries)()
    st = lib().sparse_attn_layout_size(n, block, stride_l, summary_c, pattern, head_mode,
                                       ctypes.byref(ng), nnz)
    _check("sparse_attn_layout_size", st)
    return ng.value, list(nnz)[: ng.value]


def sparse_attn_layout(n, block, stride_l, summary_c, pattern, head_mode, row_ptr, col_idx, kind,
                       col_ptr, row_idx, kind_t, capacity, stream=None):
    st = lib().sparse_attn_layout(n, block, stride_l, summary_c, pattern, head_mode, _ptr(row_ptr),
                                  _ptr(col_idx), _ptr(kind), _ptr(col_ptr), _ptr(row_idx), _ptr(kind_t),
                                  capacity, _stream(stream, row_ptr.device))
    _check("sparse_attn_layout", st)


def sparse_attn_fwd(n, block, stride_l, summary_c, pattern, head_mode, row_ptr, col_idx, kind,
                    batch, heads, d_head, dtype, q, k, v, strides, softmax_scale, o, lse, stream=None):
    st = lib().sparse_attn_fwd(n, block, stride_l, summary_c, pattern, head_mode, _ptr(row_ptr),
                               _ptr(col_idx), _ptr(kind), batch, heads, d_head, dtype, _ptr(q), _ptr(k),
                               _ptr(v), strides, softmax_scale, _ptr(o), _ptr(lse),
                               _stream(stream, q.device))
    _check("sparse_attn_fwd", st)


def sparse_attn_bwd_workspace_size(n, block, stride_l, summary_c, pattern, head_mode, batch, heads,
                                   d_head, dtype):
    out = ctypes.c_size_t(0)
    st = lib().sparse_attn_bwd_workspace_size(n, block, stride_l, summary_c, pattern, head_mode, batch,
                                              heads, d_head, dtype, ctypes.byref(out))
    _check("sparse_attn_bwd_workspace_size", st)
    return out.value


def sparse_attn_bwd(n, block, stride_l, summary_c, pattern, head_mode, row_ptr, col_idx, kind,
                    col_ptr, row_idx, kind_t, batch, heads, d_head, dtype, q, k, v, o, dout, lse,
                    strides, softmax_scale, dq, dk, dv, workspace, workspace_bytes, stream=None):
    st = lib().sparse_attn_bwd(n, block, stride_l, summary_c, pattern, head_mode, _ptr(row_ptr),
                               _ptr(col_idx), _ptr(kind), _ptr(col_ptr), _ptr(row_idx), _ptr(kind_t),
                               batch, heads, d_head, dtype, _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                               _ptr(dout), _ptr(lse), strides, softmax_scale, _ptr(dq), _ptr(dk),
                               _ptr(dv), _ptr(workspace), workspace_bytes, _stream(stream, q.device))
    _check("sparse_attn_bwd", st)


def sparse_attn_bwd_stage(n, block, stride_l, summary_c, pattern, head_mode, row_ptr, col_idx, kind,
                          col_ptr, row_idx, kind_t, batch, heads, d_head, dtype, q, k, v, o, dout, lse,
                          strides, softmax_scale, dq, dk, dv, workspace, workspace_bytes, stages, stream=None):
    st = lib().sparse_attn_bwd_stage(n, block, stride_l, summary_c, pattern, head_mode, _ptr(row_ptr),
                                     _ptr(col_idx), _ptr(kind), _ptr(col_ptr), _ptr(row_idx), _ptr(kind_t),
                                     batch, heads, d_head, dtype, _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                                     _ptr(dout), _ptr(lse), strides, softmax_scale, _ptr(dq), _ptr(dk),
                                     _ptr(dv), _ptr(workspace), workspace_bytes, stages, _stream(stream, q.device))
    _check("sparse_attn_bwd_stage", st)


def sparse_attn_bwd_noalloc_max_workspace():
    out = ctypes.c_size_t(0)
    _check("sparse_attn_bwd_noalloc_max_workspace", lib().sparse_attn_bwd_noalloc_max_workspace(ctypes.byref(out)))
    return out.value


def sparse_attn_bwd_noalloc(n, block, stride_l, summary_c, pattern, head_mode, row_ptr, col_idx, kind,
                            col_ptr, row_idx, kind_t, batch, heads, d_head, dtype, q, k, v, o, dout, lse,
                            strides, softmax_scale, dq, dk, dv, stream=None):
    st = lib().sparse_attn_bwd_noalloc(n, block, stride_l, summary_c, pattern, head_mode, _ptr(row_ptr),
                                       _ptr(col_idx), _ptr(kind), _ptr(col_ptr), _ptr(row_idx), _ptr(kind_t),
                                       batch, heads, d_head, dtype, _ptr(q), _ptr(k), _ptr(v), _ptr(o),
                                       _ptr(dout), _ptr(lse), strides, softmax_scale, _ptr(dq), _ptr(dk),
                                       _ptr(dv), _stream(stream, q.device))
    _check("sparse_attn_bwd_noalloc", st)


def sparse_attn_decode_workspace_size(pos, stride_l, summary_c, pattern, head_mode, batch, heads, d_head, dtype):
    out = ctypes.c_size_t(0)
    st = lib().sparse_attn_decode_workspace_size(pos, stride_l, summary_c, pattern, head_mode, batch, heads,
                                                 d_head, dtype, ctypes.byref(out))
    _check("sparse_attn_decode_workspace_size", st)
    return out.value


def sparse_attn_decode(pos, stride_l, summary_c, pattern, head_mode, batch, heads, d_head, dtype, q, q_strides,
                       k_cache, v_cache, kv_strides, softmax_scale, o, lse, workspace, workspace_bytes,
                       stream=None):
    st = lib().sparse_attn_decode(pos, stride_l, summary_c, pattern, head_mode, batch, heads, d_head, dtype,
                                  _ptr(q), q_strides, _ptr(k_cache), _ptr(v_cache), kv_strides, softmax_scale,
                                  _ptr(o), _ptr(lse), _ptr(workspace), workspace_bytes, _stream(stream, q.device))
    _check("sparse_attn_decode", st)


# ---------------------------------------------------------------------------
# Convenience layer: torch allocates, the entry points above compute
# ---------------------------------------------------------------------------
@dataclass
class Layout:
    n: int
    block: int
    stride_l: int
    summary_c: int
    pattern: int
    head_mode: int
    n_layouts: int
    nnz: list
    row_ptr: torch.Tensor
    col_idx: torch.Tensor
    kind: torch.Tensor
    col_ptr: torch.Tensor
    row_idx: torch.Tensor
    kind_t: torch.Tensor

    @property
    def pattern_args(self):
        return (self.n, self.block, self.stride_l, self.summary_c, self.pattern, self.head_mode)

    @property
    def row_args(self):
        return (self.row_ptr, self.col_idx, self.kind)

    @property
    def col_args(self):
        return (self.col_ptr, self.row_idx, self.kind_t)


def build_layout(n, block, stride_l, summary_c, pattern, head_mode, device="cuda", stream=None):
    ng, nnz = sparse_attn_layout_size(n, block, stride_l, summary_c, pattern, head_mode)
    nq = n // block
    total = max(1, sum(nnz))
    dev = torch.device(device)
    lay = Layout(n, block, stride_l, summary_c, pattern, head_mode, ng, nnz,
                 row_ptr=torch.empty(ng * (nq + 1), dtype=torch.int32, device=dev),
                 col_idx=torch.empty(total, dtype=torch.int32, device=dev),
                 kind=torch.empty(total, dtype=torch.uint8, device=dev),
                 col_ptr=torch.empty(ng * (nq + 1), dtype=torch.int32, device=dev),
                 row_idx=torch.empty(total, dtype=torch.int32, device=dev),
                 kind_t=torch.empty(total, dtype=torch.uint8, device=dev))
    sparse_attn_layout(*lay.pattern_args, lay.row_ptr, lay.col_idx, lay.kind, lay.col_ptr, lay.row_idx,
                       lay.kind_t, total, stream)
    return lay


def _scale(softmax_scale, d):
    return float(1.0 / math.sqrt(d) if softmax_scale is None else softmax_scale)


def forward(q, k, v, layout: Layout, softmax_scale=None, out=None, lse=None, stream=None):
    """O and LSE of sparse attention over ``layout``; q, k, v are [b, h, n, d] on the GPU."""
    b, h, n, d = q.shape
    strides = _strides(q, k, v)
    _check_layout(layout, q)
    o = torch.empty_like(q) if out is None else out
    _strides(q, o)
    lse = torch.empty((b, h, n), dtype=torch.float32, device=q.device) if lse is None else lse
    _check_lse(lse, q)
    sparse_attn_fwd(*layout.pattern_args, *layout.row_args, b, h, d, _dtype_code(q), q, k, v, strides,
                    _scale(softmax_scale, d), o, lse, stream)
    return o, lse


def backward(q, k, v, o, dout, lse, layout: Layout, softmax_scale=None, grads=None, workspace=None,
             stream=None, stages=None):
    """dq, dk, dv of sparse attention given the forward's o and lse (``stages``:
    a subset of the SA_BWD_* stages, through sparse_attn_bwd_stage)."""
    b, h, n, d = q.shape
    strides = _strides(q, k, v, o, dout)
    _check_layout(layout, q)
    _check_lse(lse, q)
    dq, dk, dv = grads if grads is not None else (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v))
    _strides(q, dq, dk, dv)
    dtype = _dtype_code(q)
    need = sparse_attn_bwd_workspace_size(*layout.pattern_args, b, h, d, dtype)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    elif workspace.device != q.device:
        raise ValueError("workspace must be on q's device")
    if stages is not None:
        sparse_attn_bwd_stage(*layout.pattern_args, *layout.row_args, *layout.col_args, b, h, d, dtype, q, k, v, o,
                              dout, lse, strides, _scale(softmax_scale, d), dq, dk, dv, workspace,
                              workspace.numel() * workspace.element_size(), stages, stream)
        return dq, dk, dv
    sparse_attn_bwd(*layout.pattern_args, *layout.row_args, *layout.col_args, b, h, d, dtype, q, k, v, o,
                    dout, lse, strides, _scale(softmax_scale, d), dq, dk, dv, workspace,
                    workspace.numel() * workspace.element_size(), stream)
    return dq, dk, dv


def decode(q, k_cache, v_cache, pos, stride_l, summary_c, pattern, head_mode, softmax_scale=None, out=None,
           lse=None, workspace=None, stream=None):
    """Output of query position ``pos`` (q: [b, h, d]) over the cache ([b, h, >= pos + 1, d]) and S_pos."""
    b, h, d = q.shape
    if k_cache.dim() != 4 or k_cache.shape[:2] != (b, h) or k_cache.shape[3] != d or k_cache.shape[2] <= pos:
        raise ValueError("cache must be [batch, heads, >= pos + 1, d] matching q")
    if v_cache.shape != k_cache.shape or v_cache.stride() != k_cache.stride() or k_cache.stride(3) != 1:
        raise ValueError("k_cache and v_cache must share shape and strides, d contiguous")
    if q.stride(2) != 1:
        raise ValueError("q must have d contiguous")
    o = torch.empty_like(q) if out is None else out
    if o.shape != q.shape or o.stride() != q.stride():
        raise ValueError("out must match q in shape and strides")
    lse = torch.empty((b, h), dtype=torch.float32, device=q.device) if lse is None else lse
    dtype = _dtype_code(q)
    need = sparse_attn_decode_workspace_size(pos, stride_l, summary_c, pattern, head_mode, b, h, d, dtype)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    qs = (ctypes.c_int64 * 2)(q.stride(0), q.stride(1))
    ks = (ctypes.c_int64 * 3)(k_cache.stride(0), k_cache.stride(1), k_cache.stride(2))
    sparse_attn_decode(pos, stride_l, summary_c, pattern, head_mode, b, h, d, dtype, q, qs, k_cache, v_cache, ks,
                       _scale(softmax_scale, d), o, lse, workspace, workspace.numel() * workspace.element_size(),
                       stream)
    return o, lse


# ---------------------------------------------------------------------------
# Strided A2 by transposition (Sec. 5.5).  With l dividing n, write positions
# as i = m l + r (class r = i mod l, index m = i div l): j is in A2 of i iff
# j has the same class and m_j <= m_i.  In class order A2 is therefore dense
# causal attention inside each of the l classes of n / l positions.  A class is
# a strided view of a [b, h, n, d] tensor (first row r, a step of l rows), so
# the entry points above compute it unchanged: "batch" = the b * h heads (the
# stride of one head), "heads" = the l classes (a stride of d elements),
# sequence stride l rows, and the dense causal layout of n / l positions (the
# strided pattern with a stride of n / l).  O and the gradients land in place
# in the original layout; LSE comes out in class order, [b * h, l, n / l].
# ---------------------------------------------------------------------------
def transposed_a2_layout(n, stride_l, block, device="cuda", stream=None):
    """Dense causal layout of one class: n / l positions in blocks of ``block``."""
    if n % stride_l != 0 or (n // stride_l) % block != 0:
        raise ValueError("needs l | n and block | n / l")
    m = n // stride_l
    return build_layout(m, block, m, 0, SA_STRIDED, SA_MODE_A1, device=device, stream=stream)


def _class_view_strides(t, stride_l):
    b, h, n, d = t.shape
    if not t.is_contiguous():
        raise ValueError("the transposed path takes contiguous [b, h, n, d] tensors")
    return (ctypes.c_int64 * 3)(n * d, d, stride_l * d)  # a head, a class, a step within a class


def forward_a2_transposed(q, k, v, stride_l, class_layout: Layout, softmax_scale=None, out=None, lse=None,
                          stream=None):
    """O (original layout) and LSE (class order) of strided A2 attention, computed per class."""
    b, h, n, d = q.shape
    strides = _class_view_strides(q, stride_l)
    for t in (k, v):
        if t.shape != q.shape:
            raise ValueError("q, k, v must have one shape")
        _class_view_strides(t, stride_l)
    m = n // stride_l
    if class_layout.n != m:
        raise ValueError("class layout is for another n / l")
    o = torch.empty_like(q) if out is None else out
    _class_view_strides(o, stride_l)
    lse = torch.empty((b * h, stride_l, m), dtype=torch.float32, device=q.device) if lse is None else lse
    sparse_attn_fwd(*class_layout.pattern_args, *class_layout.row_args, b * h, stride_l, d, _dtype_code(q), q, k,
                    v, strides, _scale(softmax_scale, d), o, lse, stream)
    return o, lse


def backward_a2_transposed(q, k, v, o, dout, lse, stride_l, class_layout: Layout, softmax_scale=None, grads=None,
                           workspace=None, stream=None):
    """dq, dk, dv (original layout) of strided A2 attention, given the class-order LSE."""
    b, h, n, d = q.shape
    strides = _class_view_strides(q, stride_l)
    for t in (k, v, o, dout):
        _class_view_strides(t, stride_l)
    dq, dk, dv = grads if grads is not None else (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v))
    dtype = _dtype_code(q)
    need = sparse_attn_bwd_workspace_size(*class_layout.pattern_args, b * h, stride_l, d, dtype)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
    sparse_attn_bwd(*class_layout.pattern_args, *class_layout.row_args, *class_layout.col_args, b * h, stride_l,
                    d, dtype, q, k, v, o, dout, lse, strides, _scale(softmax_scale, d), dq, dk, dv, workspace,
                    workspace.numel() * workspace.element_size(), stream)
    return dq, dk, dv


def sparse_attn_transposed_workspace_size(n, block, stride_l, class_block, batch, heads, d_head, dtype):
    out = ctypes.c_size_t(0)
    st = lib().sparse_attn_transposed_workspace_size(n, block, stride_l, class_block, batch, heads, d_head, dtype,
                                                     ctypes.byref(out))
    _check("sparse_attn_transposed_workspace_size", st)
    return out.value


def sparse_attn_fwd_transposed(n, block, stride_l, class_block, row_ptr, col_idx, kind, batch, heads, d_head, dtype,
                               q, k, v, softmax_scale, o, lse, workspace, workspace_bytes, stream=None):
    st = lib().sparse_attn_fwd_transposed(n, block, stride_l, class_block, _ptr(row_ptr), _ptr(col_idx), _ptr(kind),
                                          batch, heads, d_head, dtype, _ptr(q), _ptr(k), _ptr(v), softmax_scale,
                                          _ptr(o), _ptr(lse), _ptr(workspace), workspace_bytes,
                                          _stream(stream, q.device))
    _check("sparse_attn_fwd_transposed", st)


def sparse_attn_bwd_transposed(n, block, stride_l, class_block, row_ptr, col_idx, kind, col_ptr, row_idx, kind_t,
                               batch, heads, d_head, dtype, q, k, v, o, dout, lse, softmax_scale, dq, dk, dv,
                               workspace, workspace_bytes, stream=None):
    st = lib().sparse_attn_bwd_transposed(n, block, stride_l, class_block, _ptr(row_ptr), _ptr(col_idx), _ptr(kind),
                                          _ptr(col_ptr), _ptr(row_idx), _ptr(kind_t), batch, heads, d_head, dtype,
                                          _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(dout), _ptr(lse), softmax_scale,
                                          _ptr(dq), _ptr(dk), _ptr(dv), _ptr(workspace), workspace_bytes,
                                          _stream(stream, q.device))
    _check("sparse_attn_bwd_transposed", st)


def band_layout(n, block, stride_l, device="cuda", stream=None):
    """The strided A1 layout the merged transposed path takes for its band."""
    return build_layout(n, block, stride_l, 0, SA_STRIDED, SA_MODE_A1, device=device, stream=stream)


def _check_contiguous(*tensors):
    """The transposed entry points take no strides: [b, h, n, d] contiguous, one shape."""
    shape = tensors[0].shape
    for t in tensors:
        if t.dim() != 4 or t.shape != shape or not t.is_contiguous():
            raise ValueError("the transposed path takes contiguous [batch, heads, n, d] tensors of one shape")


def _transposed_workspace(q, band: Layout, class_block, workspace):
    b, h, n, d = q.shape
    need = sparse_attn_transposed_workspace_size(n, band.block, band.stride_l, class_block, b, h, d, _dtype_code(q))
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=q.device)
    return workspace, workspace.numel() * workspace.element_size()


def forward_merged_transposed(q, k, v, band: Layout, class_block, softmax_scale=None, out=None, lse=None,
                              workspace=None, stream=None):
    """O and LSE of strided merged attention, A2 by transposition; contiguous [b, h, n, d] tensors."""
    b, h, n, d = q.shape
    if band.pattern != SA_STRIDED or band.head_mode != SA_MODE_A1 or band.n != n:
        raise ValueError("band must be the strided A1 layout of this n")
    o = torch.empty_like(q) if out is None else out
    _check_contiguous(q, k, v, o)
    lse = torch.empty((b, h, n), dtype=torch.float32, device=q.device) if lse is None else lse
    if not lse.is_contiguous() or lse.shape != (b, h, n):
        raise ValueError("lse must be a contiguous [batch, heads, n] tensor")
    ws, nbytes = _transposed_workspace(q, band, class_block, workspace)
    sparse_attn_fwd_transposed(n, band.block, band.stride_l, class_block, *band.row_args, b, h, d, _dtype_code(q),
                               q, k, v, _scale(softmax_scale, d), o, lse, ws, nbytes, stream)
    return o, lse


def backward_merged_transposed(q, k, v, o, dout, lse, band: Layout, class_block, softmax_scale=None, grads=None,
                               workspace=None, stream=None):
    """dq, dk, dv of strided merged attention, A2 by transposition."""
    b, h, n, d = q.shape
    if band.pattern != SA_STRIDED or band.head_mode != SA_MODE_A1 or band.n != n:
        raise ValueError("band must be the strided A1 layout of this n")
    dq, dk, dv = grads if grads is not None else (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v))
    _check_contiguous(q, k, v, o, dout, dq, dk, dv)
    if not lse.is_contiguous() or lse.shape != (b, h, n):
        raise ValueError("lse must be a contiguous [batch, heads, n] tensor")
    ws, nbytes = _transposed_workspace(q, band, class_block, workspace)
    sparse_attn_bwd_transposed(n, band.block, band.stride_l, class_block, *band.row_args, *band.col_args, b, h, d,
                               _dtype_code(q), q, k, v, o, dout, lse, _scale(softmax_scale, d), dq, dk, dv, ws,
                               nbytes, stream)
    return dq, dk, dv


class SparseAttention(torch.autograd.Function):
    """Autograd wrapper: saves O and LSE, recomputes attention weights in backward."""

    @staticmethod
    def forward(ctx, q, k, v, layout, softmax_scale=None):
        o, lse = forward(q, k, v, layout, softmax_scale)
        ctx.save_for_backward(q, k, v, o, lse)
        ctx.layout = layout
        ctx.softmax_scale = softmax_scale
        return o

    @staticmethod
    def backward(ctx, dout):
        q, k, v, o, lse = ctx.saved_tensors
        # the entry point takes one set of strides for all tensors: q's
        if dout.stride() != q.stride():
            dout = torch.empty_like(q).copy_(dout)
        dq, dk, dv = backward(q, k, v, o, dout, lse, ctx.layout, ctx.softmax_scale)
        return dq, dk, dv, None, None


class SparseAttentionTransposed(torch.autograd.Function):
    """Autograd wrapper of strided merged attention with A2 by transposition
    (band = the strided A1 layout, class_block = the block of the per-class
    dense causal attention); saves O and LSE, recomputes the weights."""

    @staticmethod
    def forward(ctx, q, k, v, band, class_block, softmax_scale=None):
        q, k, v = q.contiguous(), k.contiguous(), v.contiguous()
        o, lse = forward_merged_transposed(q, k, v, band, class_block, softmax_scale)
        ctx.save_for_backward(q, k, v, o, lse)
        ctx.band = band
        ctx.class_block = class_block
        ctx.softmax_scale = softmax_scale
        return o

    @staticmethod
    def backward(ctx, dout):
        q, k, v, o, lse = ctx.saved_tensors
        dq, dk, dv = backward_merged_transposed(q, k, v, o, dout.contiguous(), lse, ctx.band, ctx.class_block,
                                                ctx.softmax_scale)
        return dq, dk, dv, None, None, None
