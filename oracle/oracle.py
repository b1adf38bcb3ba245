"""ctypes wrapper of the fp64 C oracle (test infrastructure only).

Every function takes numpy arrays laid out [b, h, n, d] (d contiguous) in
float64, float32, or bfloat16 stored as raw uint16 bit patterns; the C side
converts each element exactly to fp64.  Outputs are float64.

Pattern / mode codes follow the paper's vocabulary (Sec. 4.3 and Sec. 5.1):
pattern 0 = strided, 1 = fixed, 2 = fixed with a distinct summary subblock
per head (head h attends positions l-(s+1)c .. l-sc-1 of every l-block, with
s = h mod floor(l/c)); mode 0 = A1 only, 1 = A2 only, 2 = merged
(union of A1 and A2), 3 = interleaved over heads (even heads A1, odd heads A2).
"""
import ctypes
import numpy as np

from .build import ensure_built

STRIDED, FIXED, FIXED_PER_HEAD = 0, 1, 2
MODE_A1, MODE_A2, MODE_MERGED, MODE_INTERLEAVED = 0, 1, 2, 3
PART_A1, PART_A2, PART_MERGED = 0, 1, 2

_lib = None
_i64 = ctypes.c_int64
_int = ctypes.c_int
_dbl = ctypes.c_double
_vp = ctypes.c_void_p


def lib():
    global _lib
    if _lib is None:
        L = ctypes.CDLL(ensure_built())
        L.oracle_num_threads.restype = _int
        L.oracle_row_set.restype = _i64
        L.oracle_row_set.argtypes = [_int, _int, _i64, _i64, _i64, _i64, _vp]
        L.oracle_col_set.restype = _i64
        L.oracle_col_set.argtypes = [_int, _int, _i64, _i64, _i64, _i64, _vp]
        L.oracle_head_row_set.restype = _i64
        L.oracle_head_row_set.argtypes = [_int, _int, _i64, _i64, _i64, _i64, _i64, _vp]
        L.oracle_head_col_set.restype = _i64
        L.oracle_head_col_set.argtypes = [_int, _int, _i64, _i64, _i64, _i64, _i64, _vp]
        L.oracle_num_layouts.restype = _int
        L.oracle_num_layouts.argtypes = [_i64, _i64, _int, _int]
        L.oracle_forward.restype = _int
        L.oracle_forward.argtypes = [_int, _int, _i64, _i64, _i64, _i64, _i64, _i64, _int,
                                     _vp, _vp, _vp, _dbl, _vp, _vp]
        L.oracle_backward.restype = _int
        L.oracle_backward.argtypes = [_int, _int, _i64, _i64, _i64, _i64, _i64, _i64, _int,
                                      _vp, _vp, _vp, _vp, _dbl, _vp, _vp, _vp, _vp, _vp, _vp]
        L.oracle_forward_rows.restype = _int
        L.oracle_forward_rows.argtypes = [_int, _int, _i64, _i64, _i64, _i64, _i64, _int,
                                          _vp, _vp, _vp, _dbl, _i64, _vp, _vp, _vp]
        L.oracle_backward_rows.restype = _int
        L.oracle_backward_rows.argtypes = [_int, _int, _i64, _i64, _i64, _i64, _i64, _int,
                                           _vp, _vp, _vp, _vp, _dbl, _i64, _vp, _vp]
        L.oracle_backward_cols.restype = _int
        L.oracle_backward_cols.argtypes = [_int, _int, _i64, _i64, _i64, _i64, _i64, _int,
                                           _vp, _vp, _vp, _vp, _dbl, _i64, _vp, _vp, _vp]
        L.oracle_layout_count.restype = _int
        L.oracle_layout_count.argtypes = [_i64, _i64, _i64, _i64, _int, _int, _vp, _vp]
        L.oracle_layout_fill.restype = _int
        L.oracle_layout_fill.argtypes = [_i64, _i64, _i64, _i64, _int, _int,
                                         _vp, _vp, _vp, _vp, _vp, _vp]
        _lib = L
    return _lib


def num_threads() -> int:
    return lib().oracle_num_threads()


def _ptr(a):
    return a.ctypes.data_as(_vp) if a is not None else None


def _dtype_code(a):
    if a.dtype == np.float64:
        return 0
    if a.dtype == np.float32:
        return 1
    if a.dtype == np.uint16:
        return 2
    raise TypeError(f"oracle inputs must be float64, float32 or bf16 bits (uint16), got {a.dtype}")


def _prep(*arrays):
    out = [np.ascontiguousarray(a) for a in arrays]
    codes = {_dtype_code(a) for a in out}
    if len(codes) != 1:
        raise TypeError("all inputs must share one dtype")
    return out, codes.pop()


def row_set(pattern, part, n, l, c, i):
    """S_i for one factor (part 0 = A1, 1 = A2, 2 = merged), ascending."""
    m = lib().oracle_row_set(pattern, part, n, l, c, i, None)
    out = np.empty(max(m, 1), dtype=np.int64)
    lib().oracle_row_set(pattern, part, n, l, c, i, _ptr(out))
    return out[:m]


def col_set(pattern, part, n, l, c, j):
    """T_j = {i : j in S_i}, ascending."""
    m = lib().oracle_col_set(pattern, part, n, l, c, j, None)
    out = np.empty(max(m, 1), dtype=np.int64)
    lib().oracle_col_set(pattern, part, n, l, c, j, _ptr(out))
    return out[:m]


def head_row_set(pattern, mode, n, l, c, h, i):
    """S_i of head h of a multi-head call (its factor and summary window)."""
    m = lib().oracle_head_row_set(pattern, mode, n, l, c, h, i, None)
    out = np.empty(max(m, 1), dtype=np.int64)
    lib().oracle_head_row_set(pattern, mode, n, l, c, h, i, _ptr(out))
    return out[:m]


def head_col_set(pattern, mode, n, l, c, h, j):
    """T_j of head h, ascending."""
    m = lib().oracle_head_col_set(pattern, mode, n, l, c, h, j, None)
    out = np.empty(max(m, 1), dtype=np.int64)
    lib().oracle_head_col_set(pattern, mode, n, l, c, h, j, _ptr(out))
    return out[:m]


def num_layouts(l, c, pattern, mode):
    return int(lib().oracle_num_layouts(l, c, pattern, mode))


def forward(q, k, v, *, pattern, mode, l, c, scale):
    """O [b,h,n,d] and LSE [b,h,n] in fp64."""
    (q, k, v), code = _prep(q, k, v)
    b, h, n, d = q.shape
    o = np.empty((b, h, n, d), dtype=np.float64)
    lse = np.empty((b, h, n), dtype=np.float64)
    rc = lib().oracle_forward(pattern, mode, n, l, c, b, h, d, code, _ptr(q), _ptr(k), _ptr(v),
                              float(scale), _ptr(o), _ptr(lse))
    if rc:
        raise ValueError(f"oracle_forward failed ({rc})")
    return o, lse


def backward(q, k, v, dout, *, pattern, mode, l, c, scale):
    """Gradients of sum(O * dout): returns dict with o, lse, delta, dq, dk, dv."""
    (q, k, v, dout), code = _prep(q, k, v, dout)
    b, h, n, d = q.shape
    res = {name: np.empty((b, h, n, d), dtype=np.float64) for name in ("o", "dq", "dk", "dv")}
    res["lse"] = np.empty((b, h, n), dtype=np.float64)
    res["delta"] = np.empty((b, h, n), dtype=np.float64)
    rc = lib().oracle_backward(pattern, mode, n, l, c, b, h, d, code, _ptr(q), _ptr(k), _ptr(v),
                               _ptr(dout), float(scale), _ptr(res["o"]), _ptr(res["lse"]),
                               _ptr(res["delta"]), _ptr(res["dq"]), _ptr(res["dk"]),
                               _ptr(res["dv"]))
    if rc:
        raise ValueError(f"oracle_backward failed ({rc})")
    return res


def _flat_index(shape, bhi):
    b, h, n, _ = shape
    bhi = np.asarray(bhi, dtype=np.int64).reshape(-1, 3)
    return np.ascontiguousarray((bhi[:, 0] * h + bhi[:, 1]) * n + bhi[:, 2])


def forward_rows(q, k, v, rows, *, pattern, mode, l, c, scale):
    """O and LSE of the listed rows; rows is an array of (b, h, i) triples."""
    (q, k, v), code = _prep(q, k, v)
    b, h, n, d = q.shape
    flat = _flat_index(q.shape, rows)
    o = np.empty((len(flat), d), dtype=np.float64)
    lse = np.empty(len(flat), dtype=np.float64)
    rc = lib().oracle_forward_rows(pattern, mode, n, l, c, h, d, code, _ptr(q), _ptr(k), _ptr(v),
                                   float(scale), len(flat), _ptr(flat), _ptr(o), _ptr(lse))
    if rc:
        raise ValueError(f"oracle_forward_rows failed ({rc})")
    return o, lse


def backward_rows(q, k, v, dout, rows, *, pattern, mode, l, c, scale):
    """dq of the listed (b, h, i) rows."""
    (q, k, v, dout), code = _prep(q, k, v, dout)
    b, h, n, d = q.shape
    flat = _flat_index(q.shape, rows)
    dq = np.empty((len(flat), d), dtype=np.float64)
    rc = lib().oracle_backward_rows(pattern, mode, n, l, c, h, d, code, _ptr(q), _ptr(k), _ptr(v),
                                    _ptr(dout), float(scale), len(flat), _ptr(flat), _ptr(dq))
    if rc:
        raise ValueError(f"oracle_backward_rows failed ({rc})")
    return dq


def backward_cols(q, k, v, dout, cols, *, pattern, mode, l, c, scale):
    """dk, dv of the listed (b, h, j) columns."""
    (q, k, v, dout), code = _prep(q, k, v, dout)
    b, h, n, d = q.shape
    flat = _flat_index(q.shape, cols)
    dk = np.empty((len(flat), d), dtype=np.float64)
    dv = np.empty((len(flat), d), dtype=np.float64)
    rc = lib().oracle_backward_cols(pattern, mode, n, l, c, h, d, code, _ptr(q), _ptr(k), _ptr(v),
                                    _ptr(dout), float(scale), len(flat), _ptr(flat), _ptr(dk),
                                    _ptr(dv))
    if rc:
        raise ValueError(f"oracle_backward_cols failed ({rc})")
    return dk, dv


def layout(n, block, l, c, pattern, mode):
    """Brute-force block layout: dict of numpy arrays (CSR rows + transpose)."""
    ng = np.zeros(1, dtype=np.int64)
    nnz = np.zeros(max(2, num_layouts(l, c, pattern, mode)), dtype=np.int64)
    rc = lib().oracle_layout_count(n, block, l, c, pattern, mode, _ptr(ng), _ptr(nnz))
    if rc:
        raise ValueError(f"oracle_layout_count failed ({rc})")
    ng = int(ng[0])
    nq = n // block
    total = int(nnz[:ng].sum())
    out = {
        "n_layouts": ng,
        "nnz": nnz[:ng].copy(),
        "row_ptr": np.zeros(ng * (nq + 1), dtype=np.int32),
        "col_idx": np.zeros(max(total, 1), dtype=np.int32),
        "kind": np.zeros(max(total, 1), dtype=np.uint8),
        "col_ptr": np.zeros(ng * (nq + 1), dtype=np.int32),
        "row_idx": np.zeros(max(total, 1), dtype=np.int32),
        "kind_t": np.zeros(max(total, 1), dtype=np.uint8),
    }
    rc = lib().oracle_layout_fill(n, block, l, c, pattern, mode, _ptr(out["row_ptr"]),
                                  _ptr(out["col_idx"]), _ptr(out["kind"]), _ptr(out["col_ptr"]),
                                  _ptr(out["row_idx"]), _ptr(out["kind_t"]))
    if rc:
        raise ValueError(f"oracle_layout_fill failed ({rc})")
    for key in ("col_idx", "kind", "row_idx", "kind_t"):
        out[key] = out[key][:total]
    return out
