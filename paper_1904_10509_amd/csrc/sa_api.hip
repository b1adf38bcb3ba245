// C ABI (include/sparse_attn.h): argument validation, launch configuration and
// status codes.  Nothing is enqueued unless every argument is valid.
#include <math.h>

#include <mutex>

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
    a.claim_mode = sa::CLAIM_QUEUES;
    a.pairs = 0;
    a.row_stats = 0;
    a.dl = sa::make_divl(p.l);
    a.walk = sa::WALK_LAYOUT;
    a.qshift = 0;
    a.epilogue = sa::EPI_STORE;
    a.lse_sb = (int64_t)heads * p.n;  // LSE and row statistics: [batch, heads, n]
    a.lse_sh = p.n;
    a.lse_ss = 1;
    a.row_ptr = row_ptr;
    a.col_idx = col_idx;
    a.kind = kind;
    a.col_ptr = col_ptr;
    a.row_idx = row_idx;
    a.kind_t = kind_t;
    return a;
}

// Strided pattern, merged heads or A2 alone, bf16: A2 by residue classes
// (Sec. 5.5, a stride becomes a local window once positions are reordered by
// their residue mod l).  With l dividing n, position i = m l + r (class r,
// step m) meets j = m' l + r of its own class only, and A2 \ A1 of the merged
// set is {m' <= m - 2}: dense causal attention inside each class, with the
// queries' causal limit moved back by two steps (A2 alone: by none).  The
// classes are strided views of the [b, h, n, d] tensors, so the block kernels
// walk them unchanged: batch = the b h pairs (stride of one head), heads = the
// l classes (stride of one row), sequence stride l rows, every block kb <= qb
// present (no layout), LSE and row statistics read back in row order.  The
// merged set's band A1 runs first over the caller's layout (only its band
// blocks: with B dividing l, A2 \ A1 never meets them), and the class kernels
// then combine their part into its O and LSE (forward) or add it to its
// gradients (backward).  class_args builds the class view's kernel arguments
// for class blocks of cb positions (merged: queries shifted by two steps);
// class_plan picks the class block and returns false where the block path
// stays: fp32, l not dividing n, n / l not a multiple of 16, batch and head
// strides that do not merge, or sizes the class grid cannot hold.
int class_args(int64_t n, int32_t l, int32_t cb, int32_t mode, int32_t batch, int32_t heads, int32_t d,
               int32_t dtype, const int64_t* strides, float scale, sa::AttnArgs* cls) {
    if (n % l != 0) return SA_ERR_INVALID;
    const int64_t M = n / l;  // positions per class
    if (cb != 16 && cb != 32 && cb != 64) return SA_ERR_INVALID;
    if (M % cb != 0) return SA_ERR_INVALID;
    if (M / cb > 65535 || (int64_t)batch * heads > 65535) return SA_ERR_UNSUPPORTED;  // grid dimensions
    if (batch > 1 && strides[0] != (int64_t)heads * strides[1]) return SA_ERR_UNSUPPORTED;  // (b, h) as one index
    const int64_t cls_strides[3] = {strides[1], strides[2], (int64_t)l * strides[2]};
    PatternArgs c;
    int st = check_pattern(M, cb, (int32_t)M, 0, SA_STRIDED, SA_MODE_A1, &c);
    if (st != SA_OK) return st;
    st = check_tensor_args(c, batch * heads, l, d, dtype, cls_strides);
    if (st != SA_OK) return st;
    *cls = make_args(c, batch * heads, l, d, cls_strides, scale, nullptr, nullptr, nullptr, nullptr, nullptr,
                     nullptr);
    cls->walk = sa::WALK_DENSE;
    cls->qshift = mode == SA_MODE_MERGED ? 2 : 0;
    cls->lse_sb = n;  // row i = m l + r of pair bh sits at bh n + r + m l
    cls->lse_sh = 1;
    cls->lse_ss = l;
    return SA_OK;
}

bool class_plan(const PatternArgs& p, int32_t batch, int32_t heads, int32_t d, int32_t dtype, const int64_t* strides,
                float scale, sa::AttnArgs* cls) {
    if (p.pattern != sa::STRIDED || dtype != SA_BF16) return false;
    if (p.mode != SA_MODE_MERGED && p.mode != SA_MODE_A2) return false;
    if (p.n % p.l != 0 || (p.mode == SA_MODE_MERGED && p.l % p.block != 0)) return false;
    const int64_t M = p.n / p.l;
    const int32_t cb = (M % 64 == 0 && M >= 256) ? 64 : (M % 32 == 0 ? 32 : (M % 16 == 0 ? 16 : 0));
    if (cb == 0) return false;
    return class_args(p.n, p.l, cb, p.mode, batch, heads, d, dtype, strides, scale, cls) == SA_OK;
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

// Merged strided heads by transposition through the explicit entry points:
// the band over the caller's strided A1 layout, the classes in blocks of
// class_block (see class_args); tensors contiguous.
struct TransposedPlan {
    PatternArgs band;
    int64_t strides[3];
    sa::AttnArgs cls;
    size_t workspace;  // bytes: the band backward's workspace
};

int plan_transposed(int64_t n, int32_t block, int32_t l, int32_t class_block, int32_t batch, int32_t heads, int32_t d,
                    int32_t dtype, float scale, TransposedPlan* p) {
    int st = check_pattern(n, block, l, 0, SA_STRIDED, SA_MODE_A1, &p->band);
    if (st != SA_OK) return st;
    if (batch < 1 || heads < 1) return SA_ERR_INVALID;
    p->strides[0] = (int64_t)heads * n * d;
    p->strides[1] = n * d;
    p->strides[2] = d;
    st = check_tensor_args(p->band, batch, heads, d, dtype, p->strides);
    if (st != SA_OK) return st;
    st = class_args(n, l, class_block, SA_MODE_MERGED, batch, heads, d, dtype, p->strides, scale, &p->cls);
    if (st != SA_OK) return st;
    p->workspace = sa::bwd_workspace_bytes(batch, heads, n, p->band.nq, 1);
    return SA_OK;
}

// Arguments of a backward call, shared by sparse_attn_bwd and
// sparse_attn_bwd_noalloc: everything but the workspace.  Fills the kernel
// arguments and the workspace size the call needs.
int check_bwd(int64_t n, int32_t block, int32_t stride_l, int32_t summary_c, int32_t pattern, int32_t head_mode,
              const int32_t* row_ptr, const int32_t* col_idx, const uint8_t* kind, const int32_t* col_ptr,
              const int32_t* row_idx, const uint8_t* kind_t, int32_t batch, int32_t heads, int32_t d_head,
              int32_t dtype, const void* q, const void* k, const void* v, const void* o, const void* dout,
              const float* lse, const int64_t* strides, float softmax_scale, void* dq, void* dk, void* dv,
              sa::AttnArgs* a, size_t* need, bool* by_classes, sa::AttnArgs* cls) {
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
    *need = sa::bwd_workspace_bytes(batch, heads, n, p.nq, p.n_layouts);
    *a = make_args(p, batch, heads, d_head, strides, softmax_scale, row_ptr, col_idx, kind, col_ptr, row_idx,
                   kind_t);
    *by_classes = class_plan(p, batch, heads, d_head, dtype, strides, softmax_scale, cls);
    return SA_OK;
}

// The launches of a validated backward call (see class_plan): the band's
// backward, then the classes' dQ and dK / dV added to it; A2 alone: the row
// statistics, then the classes' dQ and dK / dV.
// `parts`: the stages to launch (sa::BWD_*), in their order.
hipError_t launch_bwd(sa::AttnArgs a, bool by_classes, sa::AttnArgs cls, int dtype, const void* q, const void* k,
                      const void* v, const void* o, const void* dout, const float* lse, void* dq, void* dk, void* dv,
                      void* ws, hipStream_t s, int parts = sa::BWD_ALL) {
    if (!by_classes) return sa::bwd_launch(a, dtype, q, k, v, o, dout, lse, dq, dk, dv, ws, s, parts);
    // the band's stages first (merged; the row statistics, in row order, go
    // with the band's dQ), or the row statistics alone (A2: no band)
    const bool merged = a.mode == sa::MODE_MERGED;
    if (merged) {
        a.walk = sa::WALK_BAND;
        cls.epilogue = sa::EPI_ADD;
    }
    hipError_t e = hipSuccess;
    // the classes' dQ and dK / dV last and together (short classes run them
    // as one launch)
    const int band = merged ? parts : parts & sa::BWD_PRE;
    if (band) e = sa::bwd_launch(a, dtype, q, k, v, o, dout, lse, dq, dk, dv, ws, s, band);
    const int classes = parts & (sa::BWD_DQ | sa::BWD_DKDV);
    if (e == hipSuccess && classes)
        e = sa::bwd_launch(cls, dtype, q, k, v, o, dout, lse, dq, dk, dv, ws, s, classes);
    return e;
}

}  // namespace

// ---------------------------------------------------------------------------
// Scratch of sparse_attn_bwd_noalloc: a fixed device array in place of the
// caller's workspace, one copy per device, held until the process ends.  In
// host code `scratch` names a host-side stand-in, not device memory, so its
// device address is looked up once per device (with that device current)
// and only that address is ever passed on.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices];  // device address of `scratch` per device, guarded by g_scratch_mutex

// Device address of the scratch array on the device of `stream`, which must
// be the current device.
int scratch_address(hipStream_t stream, void** out) {
    int dev = -1, stream_dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return SA_ERR_HIP;
    if (hipStreamGetDevice(stream, &stream_dev) != hipSuccess) return SA_ERR_HIP;
    if (stream_dev != dev) return SA_ERR_INVALID;
    if (dev < 0 || dev >= kMaxDevices) return SA_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return SA_ERR_HIP;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
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
    const hipStream_t s = static_cast<hipStream_t>(stream);
    sa::AttnArgs cls;
    if (class_plan(p, batch, heads, d_head, dtype, strides, softmax_scale, &cls)) {
        hipError_t e = hipSuccess;
        if (p.mode == SA_MODE_MERGED) {  // the band first, then the classes merged into it
            a.walk = sa::WALK_BAND;
            e = sa::fwd_launch(a, dtype, q, k, v, o, lse, s);
            cls.epilogue = sa::EPI_MERGE;
        }
        if (e == hipSuccess) e = sa::fwd_launch(cls, dtype, q, k, v, o, lse, s);
        return e == hipSuccess ? SA_OK : SA_ERR_HIP;
    }
    hipError_t e = sa::fwd_launch(a, dtype, q, k, v, o, lse, s);
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
    sa::AttnArgs a, cls;
    size_t need = 0;
    bool by_classes = false;
    const int st = check_bwd(n, block, stride_l, summary_c, pattern, head_mode, row_ptr, col_idx, kind, col_ptr,
                             row_idx, kind_t, batch, heads, d_head, dtype, q, k, v, o, dout, lse, strides,
                             softmax_scale, dq, dk, dv, &a, &need, &by_classes, &cls);
    if (st != SA_OK) return st;
    if (workspace_bytes < need) return SA_ERR_BUFFER_TOO_SMALL;
    if (need > 0 && (!workspace || !aligned16(workspace))) return SA_ERR_INVALID;
    hipError_t e = launch_bwd(a, by_classes, cls, dtype, q, k, v, o, dout, lse, dq, dk, dv, workspace,
                              static_cast<hipStream_t>(stream));
    return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

int sparse_attn_bwd_stage(int64_t n, int32_t block, int32_t stride_l, int32_t summary_c, int32_t pattern,
                          int32_t head_mode, const int32_t* row_ptr, const int32_t* col_idx, const uint8_t* kind,
                          const int32_t* col_ptr, const int32_t* row_idx, const uint8_t* kind_t, int32_t batch,
                          int32_t heads, int32_t d_head, int32_t dtype, const void* q, const void* k, const void* v,
                          const void* o, const void* dout, const float* lse, const int64_t* strides,
                          float softmax_scale, void* dq, void* dk, void* dv, void* workspace, size_t workspace_bytes,
                          int32_t stages, void* stream) {
    if (stages < 1 || stages > SA_BWD_ALL_STAGES) return SA_ERR_INVALID;
    sa::AttnArgs a, cls;
    size_t need = 0;
    bool by_classes = false;
    const int st = check_bwd(n, block, stride_l, summary_c, pattern, head_mode, row_ptr, col_idx, kind, col_ptr,
                             row_idx, kind_t, batch, heads, d_head, dtype, q, k, v, o, dout, lse, strides,
                             softmax_scale, dq, dk, dv, &a, &need, &by_classes, &cls);
    if (st != SA_OK) return st;
    if (workspace_bytes < need) return SA_ERR_BUFFER_TOO_SMALL;
    if (need > 0 && (!workspace || !aligned16(workspace))) return SA_ERR_INVALID;
    // the fp32 path has no separate stages
    const int parts = dtype == SA_BF16 ? stages : sa::BWD_ALL;
    if (dtype != SA_BF16 && stages != SA_BWD_ALL_STAGES) return SA_ERR_UNSUPPORTED;
    hipError_t e = launch_bwd(a, by_classes, cls, dtype, q, k, v, o, dout, lse, dq, dk, dv, workspace,
                              static_cast<hipStream_t>(stream), parts);
    return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

int sparse_attn_bwd_noalloc_max_workspace(size_t* bytes) {
    if (!bytes) return SA_ERR_INVALID;
    *bytes = kScratchBytes;
    return SA_OK;
}

int sparse_attn_bwd_noalloc(int64_t n, int32_t block, int32_t stride_l, int32_t summary_c, int32_t pattern,
                            int32_t head_mode, const int32_t* row_ptr, const int32_t* col_idx, const uint8_t* kind,
                            const int32_t* col_ptr, const int32_t* row_idx, const uint8_t* kind_t, int32_t batch,
                            int32_t heads, int32_t d_head, int32_t dtype, const void* q, const void* k, const void* v,
                            const void* o, const void* dout, const float* lse, const int64_t* strides,
                            float softmax_scale, void* dq, void* dk, void* dv, void* stream) {
    sa::AttnArgs a, cls;
    size_t need = 0;
    bool by_classes = false;
    int st = check_bwd(n, block, stride_l, summary_c, pattern, head_mode, row_ptr, col_idx, kind, col_ptr, row_idx,
                       kind_t, batch, heads, d_head, dtype, q, k, v, o, dout, lse, strides, softmax_scale, dq, dk,
                       dv, &a, &need, &by_classes, &cls);
    if (st != SA_OK) return st;
    if (need > kScratchBytes) return SA_ERR_BUFFER_TOO_SMALL;
    hipStream_t s = static_cast<hipStream_t>(stream);
    void* ws = nullptr;
    st = scratch_address(s, &ws);
    if (st != SA_OK) return st;
    // the workspace's contents on entry are ignored: the pre kernel writes the
    // row statistics and empties the work counters before anything reads them
    hipError_t e = launch_bwd(a, by_classes, cls, dtype, q, k, v, o, dout, lse, dq, dk, dv, ws, s);
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

int sparse_attn_transposed_workspace_size(int64_t n, int32_t block, int32_t stride_l, int32_t class_block,
                                          int32_t batch, int32_t heads, int32_t d_head, int32_t dtype, size_t* bytes) {
    TransposedPlan p;
    const int st = plan_transposed(n, block, stride_l, class_block, batch, heads, d_head, dtype, 1.f, &p);
    if (st != SA_OK) return st;
    if (!bytes) return SA_ERR_INVALID;
    *bytes = p.workspace;
    return SA_OK;
}

int sparse_attn_fwd_transposed(int64_t n, int32_t block, int32_t stride_l, int32_t class_block,
                               const int32_t* row_ptr, const int32_t* col_idx, const uint8_t* kind, int32_t batch,
                               int32_t heads, int32_t d_head, int32_t dtype, const void* q, const void* k,
                               const void* v, float softmax_scale, void* o, float* lse, void* workspace,
                               size_t workspace_bytes, void* stream) {
    if (!isfinite(softmax_scale) || !(softmax_scale > 0.f)) return SA_ERR_INVALID;
    TransposedPlan p;
    const int st = plan_transposed(n, block, stride_l, class_block, batch, heads, d_head, dtype, softmax_scale, &p);
    if (st != SA_OK) return st;
    if (!row_ptr || !col_idx || !kind || !q || !k || !v || !o || !lse) return SA_ERR_INVALID;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o)) return SA_ERR_INVALID;
    if (workspace_bytes < p.workspace) return SA_ERR_BUFFER_TOO_SMALL;
    if (p.workspace > 0 && (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)) return SA_ERR_INVALID;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    // the band (strided A1 layout), then the classes merged into it
    const sa::AttnArgs band = make_args(p.band, batch, heads, d_head, p.strides, softmax_scale, row_ptr, col_idx,
                                        kind, nullptr, nullptr, nullptr);
    sa::AttnArgs cls = p.cls;
    cls.epilogue = sa::EPI_MERGE;
    hipError_t e = sa::fwd_launch(band, dtype, q, k, v, o, lse, s);
    if (e == hipSuccess) e = sa::fwd_launch(cls, dtype, q, k, v, o, lse, s);
    return e == hipSuccess ? SA_OK : SA_ERR_HIP;
}

int sparse_attn_bwd_transposed(int64_t n, int32_t block, int32_t stride_l, int32_t class_block,
                               const int32_t* row_ptr, const int32_t* col_idx, const uint8_t* kind,
                               const int32_t* col_ptr, const int32_t* row_idx, const uint8_t* kind_t, int32_t batch,
                               int32_t heads, int32_t d_head, int32_t dtype, const void* q, const void* k,
                               const void* v, const void* o, const void* dout, const float* lse, float softmax_scale,
                               void* dq, void* dk, void* dv, void* workspace, size_t workspace_bytes, void* stream) {
    if (!isfinite(softmax_scale) || !(softmax_scale > 0.f)) return SA_ERR_INVALID;
    TransposedPlan p;
    const int st = plan_transposed(n, block, stride_l, class_block, batch, heads, d_head, dtype, softmax_scale, &p);
    if (st != SA_OK) return st;
    if (!row_ptr || !col_idx || !kind || !col_ptr || !row_idx || !kind_t) return SA_ERR_INVALID;
    if (!q || !k || !v || !o || !dout || !lse || !dq || !dk || !dv) return SA_ERR_INVALID;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(dout) || !aligned16(dq) ||
        !aligned16(dk) || !aligned16(dv))
        return SA_ERR_INVALID;
    if (workspace_bytes < p.workspace) return SA_ERR_BUFFER_TOO_SMALL;
    if (p.workspace > 0 && (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)) return SA_ERR_INVALID;
    const hipStream_t s = static_cast<hipStream_t>(stream);
    // the band's backward given the merged O and LSE, then the classes' dQ and
    // dK / dV added to it
    const sa::AttnArgs band = make_args(p.band, batch, heads, d_head, p.strides, softmax_scale, row_ptr, col_idx,
                                        kind, col_ptr, row_idx, kind_t);
    sa::AttnArgs cls = p.cls;
    cls.epilogue = sa::EPI_ADD;
    hipError_t e = sa::bwd_launch(band, dtype, q, k, v, o, dout, lse, dq, dk, dv, workspace, s);
    if (e == hipSuccess)
        e = sa::bwd_launch(cls, dtype, q, k, v, o, dout, lse, dq, dk, dv, workspace, s, sa::BWD_DQ | sa::BWD_DKDV);
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
