// C ABI (include/sparse_attn.h): argument validation, launch configuration and
// status codes.  Nothing is enqueued unless every argument is valid.
#include <math.h>

#include "sparse_attn.h"
#include "sa_internal.h"
#include "sa_mask.h"

namespace {

using sa::Pattern;

// Summary subblocks per l-block that heads can be spread over; beyond this the
// per-subblock layouts would outgrow any useful head count.
constexpr int kMaxSubblocks = 64;

struct PatternArgs {
    int64_t n;
    int32_t block, l, c;
    int32_t pattern;  // STRIDED or FIXED (SA_FIXED_PER_HEAD is FIXED with sub > 0)
    int32_t mode;
    int32_t sub;      // summary subblocks, 0 = one window for all heads
    int64_t nq;
    int n_layouts;
};

// Pattern, stride and summary width (shared by the block and decoding entry
// points): internal pattern and subblock count.
int check_pattern_code(int32_t l, int32_t c, int32_t pattern, int32_t mode, int32_t* internal, int32_t* sub) {
    if (l < 1) return SA_ERR_INVALID;
    if (pattern != SA_STRIDED && pattern != SA_FIXED && pattern != SA_FIXED_PER_HEAD) return SA_ERR_INVALID;
    if (mode < SA_MODE_A1 || mode > SA_MODE_INTERLEAVED) return SA_ERR_INVALID;
    if (pattern != SA_STRIDED && (c < 1 || c > l)) return SA_ERR_INVALID;
    if (pattern == SA_STRIDED && c != 0) return SA_ERR_INVALID;
    *internal = pattern == SA_STRIDED ? sa::STRIDED : sa::FIXED;
    *sub = 0;
    if (pattern == SA_FIXED_PER_HEAD) {
        if (l / c > kMaxSubblocks) return SA_ERR_UNSUPPORTED;
        *sub = l / c;
    }
    return SA_OK;
}

int check_pattern(int64_t n, int32_t block, int32_t l, int32_t c, int32_t pattern, int32_t mode,
                  PatternArgs* out) {
    if (block != 16 && block != 32 && block != 64) return SA_ERR_INVALID;
    if (n < 1 || n > INT32_MAX || n % block != 0) return SA_ERR_INVALID;
    int32_t internal = 0, sub = 0;
    const int st = check_pattern_code(l, c, pattern, mode, &internal, &sub);
    if (st != SA_OK) return st;
    out->n = n;
    out->block = block;
    out->l = l;
    out->c = c;
    out->pattern = internal;
    out->mode = mode;
    out->sub = sub;
    out->nq = n / block;
    out->n_layouts = sa::layout_count(mode, sub);
    return SA_OK;
}

Pattern pattern_of_layout(const PatternArgs& p, int g) {
    Pattern s;
    s.pattern = p.pattern;
    s.part = sa::part_of_layout(p.mode, g);
    s.l = p.l;
    s.c = p.c;
    s.w = sa::summary_start(p.l, p.c, sa::subblock_of_layout(p.mode, p.sub, g));
    return s;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_tensor_args(const PatternArgs& p, int32_t batch, int32_t heads, int32_t d, int32_t dtype,
                      const int64_t* strides) {
    if (batch < 1 || heads < 1) return SA_ERR_INVALID;
    if (dtype != SA_F32 && dtype != SA_BF16) return SA_ERR_INVALID;
    if (d != 32 && d != 64 && d != 128) return SA_ERR_UNSUPPORTED;
    if (!strides) return SA_ERR_INVALID;
    const int64_t unit = dtype == SA_BF16 ? 8 : 4;  // elements per 16 bytes
    for (int t = 0; t < 3; ++t)
        if (strides[t] < 0 || strides[t] % unit != 0) return SA_ERR_INVALID;
    if (strides[2] < d) return SA_ERR_INVALID;
    if ((int64_t)batch * heads > INT32_MAX / 2) return SA_ERR_INVALID;
    // the bf16 kernels stage a B x d tile with 32-bit byte offsets from its first row
    if (dtype == SA_BF16 && strides[2] * 2 * p.block >= ((int64_t)1 << 32)) return SA_ERR_UNSUPPORTED;
    return SA_OK;
}

sa::AttnArgs make_args(const PatternArgs& p, int32_t batch, int32_t heads, int32_t d,
                       const int64_t* strides, float scale, const int32_t* row_ptr,
                       const int32_t* col_idx, const uint8_t* kind, const int32_t* col_ptr,
                       const int32_t* row_idx, const uint8_t* kind_t) {
    sa::AttnArgs a;
    a.pattern = p.pattern;
    a.mode = p.mode;
    a.l = p.l;
    a.c = p.c;
    a.n = (int32_t)p.n;
    a.nq = (int32_t)p.nq;
    a.block = p.block;
    a.batch = batch;
    a.heads = heads;
    a.d = d;
    a.sb = strides[0];
    a.sh = strides[1];
    a.ss = strides[2];
    a.scale = scale;
    a.scale_log2 = scale * sa::kLog2eHost;
    a.period_bits = sa::host_period_bits(p.l);
    sa::summary_words(p.l, p.c, p.l - p.c, &a.sum_lo, &a.sum_hi);
    a.sub = p.sub;
    a.dl = sa::make_divl(p.l);
    a.row_ptr = row_ptr;
    a.col_idx = col_idx;
    a.kind = kind;
    a.col_ptr = col_ptr;
    a.row_idx = row_idx;
    a.kind_t = kind_t;
    return a;
}

// Pattern arguments of a decoding step (no block size: S_pos is enumerated).
int check_decode_pattern(int64_t pos, int32_t l, int32_t c, int32_t pattern, int32_t mode, int32_t* internal,
                         int32_t* sub) {
    if (pos < 0 || pos > INT32_MAX) return SA_ERR_INVALID;
    return check_pattern_code(l, c, pattern, mode, internal, sub);
}
int check_decode_shape(int32_t batch, int32_t heads, int32_t d, int32_t dtype) {
    if (batch < 1 || heads < 1 || (int64_t)batch * heads > INT32_MAX / 2) return SA_ERR_INVALID;
    if (dtype != SA_F32 && dtype != SA_BF16) return SA_ERR_INVALID;
    if (d != 32 && d != 64 && d != 128) return SA_ERR_UNSUPPORTED;
    return SA_OK;
}

}  // namespace

extern "C" {

int sparse_attn_layout_size(int64_t n, int32_t block, int32_t stride_l, int32_t summary_c,
                            int32_t pattern, int32_t head_mode, int32_t* n_layouts,
                            int64_t* nnz) {
    PatternArgs p;
    int st = check_pattern(n, block, stride_l, summary_c, pattern, head_mode, &p);
    if (st != SA_OK) return st;
    if (!n_layouts || !nnz) return SA_ERR_INVALID;
    int64_t counts[1 + kMaxSubblocks] = {0};
    int64_t total = 0;
    for (int g = 0; g < p.n_layouts; ++g) {
        counts[g] = sa::layout_count_host(pattern_of_layout(p, g), n, block);
        total += counts[g];
    }
    if (total > INT32_MAX) return SA_ERR_UNSUPPORTED;  // int32 layout indices
    *n_layouts = p.n_layouts;
    const int entries = p.n_layouts > 2 ? p.n_layouts : 2;
    for (int g = 0; g < entries; ++g) nnz[g] = counts[g];
    return SA_OK;
}

int sparse_attn_layout_count(int32_t stride_l, int32_t summary_c, int32_t pattern, int32_t head_mode,
                             int32_t* n_layouts) {
    int32_t internal = 0, sub = 0;
    const int st = check_pattern_code(stride_l, summary_c, pattern, head_mode, &internal, &sub);
    if (st != SA_OK) return st;
    if (!n_layouts) return SA_ERR_INVALID;
    *n_layouts = sa::layout_count(head_mode, sub);
    return SA_OK;
}

int sparse_attn_layout(int64_t n, int32_t block, int32_t stride_l, int32_t summary_c,
                       int32_t pattern, int32_t head_mode, int32_t* row_ptr, int32_t* col_idx,
                       uint8_t* kind, int32_t* col_ptr, int32_t* row_idx, uint8_t* kind_t,
                       int64_t capacity, void* stream) {
    PatternArgs p;
    int st = check_pattern(n, block, stride_l, summary_c, pattern, head_mode, &p);
    if (st != SA_OK) return st;
    if (!row_ptr || !col_idx || !kind || !col_ptr || !row_idx || !kind_t) return SA_ERR_INVALID;
    int64_t total = 0;
    for (int g = 0; g < p.n_layouts; ++g) total += sa::layout_count_host(pattern_of_layout(p, g), n, block);
    if (total > INT32_MAX) return SA_ERR_UNSUPPORTED;
    if (capacity < total) return SA_ERR_BUFFER_TOO_SMALL;
    hipError_t e = sa::layout_launch(n, block, p.pattern, head_mode, p.sub, stride_l, summary_c, p.n_layouts,
                                     row_ptr, col_idx, kind, col_ptr, row_idx, kind_t,
                                     static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

int sparse_attn_fwd(int64_t n, int32_t block, int32_t stride_l, int32_t summary_c,
                    int32_t pattern, int32_t head_mode, const int32_t* row_ptr,
                    const int32_t* col_idx, const uint8_t* kind, int32_t batch, int32_t heads,
                    int32_t d_head, int32_t dtype, const void* q, const void* k, const void* v,
                    const int64_t* strides, float softmax_scale, void* o, float* lse,
                    void* stream) {
    PatternArgs p;
    int st = check_pattern(n, block, stride_l, summary_c, pattern, head_mode, &p);
    if (st != SA_OK) return st;
    st = check_tensor_args(p, batch, heads, d_head, dtype, strides);
    if (st != SA_OK) return st;
    if (!row_ptr || !col_idx || !kind || !q || !k || !v || !o || !lse) return SA_ERR_INVALID;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o)) return SA_ERR_INVALID;
    if (!isfinite(softmax_scale) || !(softmax_scale > 0.f)) return SA_ERR_INVALID;
    sa::AttnArgs a = make_args(p, batch, heads, d_head, strides, softmax_scale, row_ptr, col_idx,
                               kind, nullptr, nullptr, nullptr);
    hipError_t e = sa::fwd_launch(a, dtype, q, k, v, o, lse, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

int sparse_attn_bwd_workspace_size(int64_t n, int32_t block, int32_t stride_l,
                                   int32_t summary_c, int32_t pattern, int32_t head_mode,
                                   int32_t batch, int32_t heads, int32_t d_head, int32_t dtype,
                                   size_t* bytes) {
    PatternArgs p;
    int st = check_pattern(n, block, stride_l, summary_c, pattern, head_mode, &p);
    if (st != SA_OK) return st;
    if (batch < 1 || heads < 1 || (dtype != SA_F32 && dtype != SA_BF16) || !bytes) return SA_ERR_INVALID;
    if (d_head != 32 && d_head != 64 && d_head != 128) return SA_ERR_UNSUPPORTED;
    *bytes = sa::bwd_workspace_bytes(batch, heads, n, p.nq, p.n_layouts);
    return SA_OK;
}

int sparse_attn_bwd(int64_t n, int32_t block, int32_t stride_l, int32_t summary_c,
                    int32_t pattern, int32_t head_mode, const int32_t* row_ptr,
                    const int32_t* col_idx, const uint8_t* kind, const int32_t* col_ptr,
                    const int32_t* row_idx, const uint8_t* kind_t, int32_t batch,
                    int32_t heads, int32_t d_head, int32_t dtype, const void* q, const void* k,
                    const void* v, const void* o, const void* dout, const float* lse,
                    const int64_t* strides, float softmax_scale, void* dq, void* dk, void* dv,
                    void* workspace, size_t workspace_bytes, void* stream) {
    PatternArgs p;
    int st = check_pattern(n, block, stride_l, summary_c, pattern, head_mode, &p);
    if (st != SA_OK) return st;
    st = check_tensor_args(p, batch, heads, d_head, dtype, strides);
    if (st != SA_OK) return st;
    if (!row_ptr || !col_idx || !kind || !col_ptr || !row_idx || !kind_t) return SA_ERR_INVALID;
    if (!q || !k || !v || !o || !dout || !lse || !dq || !dk || !dv) return SA_ERR_INVALID;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(dout) ||
        !aligned16(dq) || !aligned16(dk) || !aligned16(dv))
        return SA_ERR_INVALID;
    if (!isfinite(softmax_scale) || !(softmax_scale > 0.f)) return SA_ERR_INVALID;
    const size_t need = sa::bwd_workspace_bytes(batch, heads, n, p.nq, p.n_layouts);
    if (workspace_bytes < need) return SA_ERR_BUFFER_TOO_SMALL;
    if (need > 0 && (!workspace || !aligned16(workspace))) return SA_ERR_INVALID;
    sa::AttnArgs a = make_args(p, batch, heads, d_head, strides, softmax_scale, row_ptr, col_idx,
                               kind, col_ptr, row_idx, kind_t);
    hipError_t e = sa::bwd_launch(a, dtype, q, k, v, o, dout, lse, dq, dk, dv, workspace,
                                  static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}


int sparse_attn_decode_workspace_size(int64_t pos, int32_t stride_l, int32_t summary_c, int32_t pattern,
                                      int32_t head_mode, int32_t batch, int32_t heads, int32_t d_head,
                                      int32_t dtype, size_t* bytes) {
    int32_t internal = 0, sub = 0;
    int st = check_decode_pattern(pos, stride_l, summary_c, pattern, head_mode, &internal, &sub);
    if (st != SA_OK) return st;
    st = check_decode_shape(batch, heads, d_head, dtype);
    if (st != SA_OK) return st;
    if (!bytes) return SA_ERR_INVALID;
    *bytes = sa::decode_workspace_bytes(internal, head_mode, sub, (int32_t)pos, stride_l, summary_c, batch, heads,
                                        d_head);
    return SA_OK;
}

int sparse_attn_decode(int64_t pos, int32_t stride_l, int32_t summary_c, int32_t pattern, int32_t head_mode,
                       int32_t batch, int32_t heads, int32_t d_head, int32_t dtype, const void* q,
                       const int64_t* q_strides, const void* k_cache, const void* v_cache,
                       const int64_t* kv_strides, float softmax_scale, void* o, float* lse, void* workspace,
                       size_t workspace_bytes, void* stream) {
    int32_t internal = 0, sub = 0;
    int st = check_decode_pattern(pos, stride_l, summary_c, pattern, head_mode, &internal, &sub);
    if (st != SA_OK) return st;
    st = check_decode_shape(batch, heads, d_head, dtype);
    if (st != SA_OK) return st;
    if (!q || !q_strides || !k_cache || !v_cache || !kv_strides || !o || !lse) return SA_ERR_INVALID;
    if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned16(o)) return SA_ERR_INVALID;
    const int64_t unit = dtype == SA_BF16 ? 8 : 4;  // elements per 16 bytes
    for (int t = 0; t < 2; ++t)
        if (q_strides[t] < 0 || q_strides[t] % unit != 0) return SA_ERR_INVALID;
    for (int t = 0; t < 3; ++t)
        if (kv_strides[t] < 0 || kv_strides[t] % unit != 0) return SA_ERR_INVALID;
    if (kv_strides[2] < d_head) return SA_ERR_INVALID;
    if (!isfinite(softmax_scale) || !(softmax_scale > 0.f)) return SA_ERR_INVALID;
    const size_t need = sa::decode_workspace_bytes(internal, head_mode, sub, (int32_t)pos, stride_l, summary_c, batch,
                                                   heads, d_head);
    if (workspace_bytes < need) return SA_ERR_BUFFER_TOO_SMALL;
    if (!workspace || !aligned16(workspace)) return SA_ERR_INVALID;
    hipError_t e = sa::decode_launch(internal, head_mode, sub, (int32_t)pos, stride_l, summary_c, batch, heads, d_head,
                                     dtype, q, q_strides, k_cache, v_cache, kv_strides, softmax_scale, o, lse,
                                     workspace, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

const char* sparse_attn_status_string(int status) {
    switch (status) {
    case SA_OK: return "success";
    case SA_ERR_INVALID: return "invalid argument";
    case SA_ERR_UNSUPPORTED: return "unsupported configuration";
    case SA_ERR_BUFFER_TOO_SMALL: return "buffer too small";
    case SA_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
    }
}

}  // extern "C"
