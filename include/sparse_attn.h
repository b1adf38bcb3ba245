/*
 * sparse_attn.h -- C ABI of the MI355X (gfx950) factorized sparse attention
 * library.
 *
 * The operation is the attend function of Child et al. (2019), Sec. 4.2
 * (eq. attend_fn): for every position i,
 *     O_i = softmax_j( scale * q_i . k_j )  V_j     over j in S_i,
 * with S_i one of the factorized connectivity patterns of Sec. 4.3, combined
 * over heads as in Sec. 5.1, plus its gradient for training.  The forward
 * saves one log-sum-exp per row so that the backward recomputes the attention
 * weights instead of storing them (Sec. 5.4).  Work is done in B x B blocks of
 * the attention matrix, and blocks above the diagonal are never visited
 * (Sec. 5.5).
 *
 * Positions are 0-based.  With stride l and summary width c:
 *   strided A1 = { max(0, i-l), ..., i }                  (l + 1 positions)
 *   strided A2 = { j <= i : (i - j) mod l == 0 }
 *   fixed   A1 = { j <= i : floor(j / l) == floor(i / l) }
 *   fixed   A2 = { j <= i : j mod l >= l - c }             (1 <= c <= l)
 * and, with a distinct summary subblock per head (Sec. 4.3, closing remark on
 * the fixed pattern: heads may look at different c-wide subblocks of each
 * l-block), for head h with s = h mod floor(l / c):
 *   fixed-per-head A2 = { j <= i : l-(s+1)c <= j mod l < l-sc }
 * (s = 0 is the plain fixed pattern).
 * A row whose set is empty (fixed A2 alone, first block) yields O_i = 0,
 * LSE_i = -inf and no gradient.
 *
 * Conventions for every entry point:
 *   - All functions are extern "C"; no C++ or PyTorch type crosses the ABI.
 *   - Device pointers point to memory allocated by the caller; the library
 *     allocates no device memory.  Its one piece of global state is a cache,
 *     per kernel and device, of how many workgroups of the dK / dV kernel the
 *     device holds at once (set on first use with atomic stores; any thread
 *     computes the same value), so calls from several host threads are safe.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Device work is enqueued asynchronously; nothing synchronizes.  The
 *     device work of a call is kernel launches only (no memset, no
 *     allocation), so it can be captured into a HIP graph.
 *   - Every argument is validated before anything is enqueued.  On error a
 *     negative sa_status is returned and no work is enqueued.  After the
 *     launches, a HIP launch error is reported as SA_ERR_HIP.  The library
 *     never prints and never aborts.
 *   - Tensors Q, K, V, O, dO, dQ, dK, dV are [batch, heads, n, d_head] with d
 *     contiguous and the same element strides (batch, head, sequence) for all;
 *     the sequence stride must be >= d_head and every base address 16-byte
 *     aligned, every stride a multiple of 8 elements.  For bf16, block rows
 *     at the sequence stride must span less than 4 GiB (2 * block * stride
 *     < 2^32 bytes), else SA_ERR_UNSUPPORTED.  LSE is [batch, heads, n]
 *     contiguous fp32 (natural logarithm).
 */
#ifndef SPARSE_ATTN_H
#define SPARSE_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SA_OK = 0,
    SA_ERR_INVALID = -1,          /* an argument is out of range or NULL */
    SA_ERR_UNSUPPORTED = -2,      /* valid request the library does not implement */
    SA_ERR_BUFFER_TOO_SMALL = -3, /* a caller buffer is smaller than required */
    SA_ERR_HIP = -4               /* the HIP runtime reported an error */
} sa_status;

/* Connectivity pattern, Sec. 4.3.  SA_FIXED_PER_HEAD is the fixed pattern
 * with a distinct summary subblock per head (see above); it needs
 * floor(l / c) <= 64, else SA_ERR_UNSUPPORTED. */
typedef enum { SA_STRIDED = 0, SA_FIXED = 1, SA_FIXED_PER_HEAD = 2 } sa_pattern;

/* Head combination, Sec. 5.1:
 *   SA_MODE_A1 / SA_MODE_A2: one factor for the whole call (eq. sepwpmat: a
 *       residual block r uses factor r mod 2, so a call picks one of them);
 *   SA_MODE_MERGED: every head attends to A1 u A2 (eq. mergedmat);
 *   SA_MODE_INTERLEAVED: multi-head attention whose heads alternate the
 *       factors, head h using A1 when h is even and A2 when h is odd. */
typedef enum {
    SA_MODE_A1 = 0,
    SA_MODE_A2 = 1,
    SA_MODE_MERGED = 2,
    SA_MODE_INTERLEAVED = 3
} sa_head_mode;

/* Element type of Q, K, V, O, dO, dQ, dK, dV.  Products accumulate in fp32. */
typedef enum { SA_F32 = 0, SA_BF16 = 1 } sa_dtype;

/* Tile kinds stored in the layout. */
enum { SA_TILE_FULL = 0, SA_TILE_MASKED = 1 };

/*
 * Pattern arguments shared by all entry points:
 *   n          sequence length, 1 <= n < 2^31, a multiple of `block`
 *   block      tile edge B in {16, 32, 64}
 *   stride_l   l >= 1 (Sec. 4.3); any l >= n makes A1 dense causal
 *   summary_c  c: 1 <= c <= l for SA_FIXED and SA_FIXED_PER_HEAD, must be 0
 *              for SA_STRIDED
 *   pattern    sa_pattern
 *   head_mode  sa_head_mode
 */

/*
 * Number of block layouts of a call (host only, no device work): one per
 * distinct set of its heads.
 *   SA_STRIDED, SA_FIXED: 2 for SA_MODE_INTERLEAVED (layout 0 holds A1,
 *       layout 1 holds A2), else 1.
 *   SA_FIXED_PER_HEAD, S = floor(l / c): SA_MODE_A1 1; SA_MODE_A2 and
 *       SA_MODE_MERGED S, layout s for subblock s (head h reads layout
 *       h mod S); SA_MODE_INTERLEAVED 1 + S, layout 0 for A1 and 1 + s for A2
 *       with subblock s (odd head h reads layout 1 + h mod S).
 */
int sparse_attn_layout_count(int32_t stride_l, int32_t summary_c, int32_t pattern, int32_t head_mode,
                             int32_t* n_layouts);

/*
 * Size query for the block layout (host only, synchronous, no device work).
 * Sec. 5.5: the product is computed over B x B blocks; a block (qb, kb) with
 * kb <= qb is present when any pair (i, j) in it is attended.
 * Outputs: *n_layouts as sparse_attn_layout_count gives it; nnz[g] = present
 * blocks of layout g.  nnz must hold max(2, n_layouts) entries (entries past
 * n_layouts are set to 0).  Each layout needs nq + 1 row and column pointers,
 * nq = n / block.
 */
int sparse_attn_layout_size(int64_t n, int32_t block, int32_t stride_l, int32_t summary_c,
                            int32_t pattern, int32_t head_mode, int32_t* n_layouts,
                            int64_t* nnz);

/*
 * Build the block layout on the device (asynchronous on `stream`).
 * All output arrays are device memory owned by the caller:
 *   row_ptr [n_layouts * (nq + 1)]  int32, absolute offsets: layout g's rows are
 *                                   row_ptr[g*(nq+1) + qb] .. row_ptr[g*(nq+1)+qb+1]
 *   col_idx [nnz_total]             int32 key block of each present block,
 *                                   strictly ascending within a row
 *   kind    [nnz_total]             uint8 SA_TILE_FULL when all B*B pairs are
 *                                   attended, else SA_TILE_MASKED
 *   col_ptr [n_layouts * (nq + 1)]  int32, the same blocks grouped by key block
 *   row_idx [nnz_total]             int32 query block, strictly ascending
 *   kind_t  [nnz_total]             uint8 kind of each entry in column order
 * `capacity` is the caller's element count of col_idx / kind / row_idx /
 * kind_t; SA_ERR_BUFFER_TOO_SMALL when below the total from the size query.
 */
int sparse_attn_layout(int64_t n, int32_t block, int32_t stride_l, int32_t summary_c,
                       int32_t pattern, int32_t head_mode, int32_t* row_ptr, int32_t* col_idx,
                       uint8_t* kind, int32_t* col_ptr, int32_t* row_idx, uint8_t* kind_t,
                       int64_t capacity, void* stream);

/*
 * Forward (Sec. 4.2 eq. attend_fn over the sets of Sec. 4.3 / 5.1).
 *   row_ptr, col_idx, kind   the layout built for the same pattern arguments
 *   batch, heads             >= 1
 *   d_head                   in {32, 64, 128}
 *   dtype                    sa_dtype of q, k, v and o
 *   q, k, v                  device inputs, [batch, heads, n, d_head]
 *   strides                  host array {batch, head, sequence} in elements
 *   softmax_scale            > 0, multiplies q . k (the paper uses 1/sqrt(d_head))
 *   o                        device output, same shape and strides as q
 *   lse                      device output [batch, heads, n] fp32:
 *                            log sum_j exp(scale q_i . k_j), -inf for empty rows
 */
int sparse_attn_fwd(int64_t n, int32_t block, int32_t stride_l, int32_t summary_c,
                    int32_t pattern, int32_t head_mode, const int32_t* row_ptr,
                    const int32_t* col_idx, const uint8_t* kind, int32_t batch, int32_t heads,
                    int32_t d_head, int32_t dtype, const void* q, const void* k, const void* v,
                    const int64_t* strides, float softmax_scale, void* o, float* lse,
                    void* stream);

/*
 * Bytes of device workspace that sparse_attn_bwd needs (host only): row
 * statistics (8 bytes per query row and head), work-queue counters and the
 * per-layout order in which the dK / dV kernel takes key blocks.
 */
int sparse_attn_bwd_workspace_size(int64_t n, int32_t block, int32_t stride_l,
                                   int32_t summary_c, int32_t pattern, int32_t head_mode,
                                   int32_t batch, int32_t heads, int32_t d_head, int32_t dtype,
                                   size_t* bytes);

/*
 * Backward with recomputation (Sec. 5.4): gradients of a loss L with
 * dL/dO = dout, given the forward's o and lse.  The attention weights are
 * recomputed blockwise as exp(scale q_i . k_j - LSE_i); nothing of size
 * n x n is stored.  Layout arguments as in the forward plus the column view
 * (col_ptr, row_idx, kind_t).  dq, dk, dv are device outputs with the
 * strides of q.  workspace is caller-owned device memory of at least
 * sparse_attn_bwd_workspace_size bytes (SA_ERR_BUFFER_TOO_SMALL otherwise);
 * its contents on entry are ignored, and calls that share one workspace
 * must not overlap (it holds per-call row statistics and a work counter).
 * Repeated calls with the same arguments on one device give the same bits;
 * the order in which dK and dV sum their terms follows the device's number
 * of compute units, so devices of another size can differ in the last bit.
 */
int sparse_attn_bwd(int64_t n, int32_t block, int32_t stride_l, int32_t summary_c,
                    int32_t pattern, int32_t head_mode, const int32_t* row_ptr,
                    const int32_t* col_idx, const uint8_t* kind, const int32_t* col_ptr,
                    const int32_t* row_idx, const uint8_t* kind_t, int32_t batch,
                    int32_t heads, int32_t d_head, int32_t dtype, const void* q, const void* k,
                    const void* v, const void* o, const void* dout, const float* lse,
                    const int64_t* strides, float softmax_scale, void* dq, void* dk, void* dv,
                    void* workspace, size_t workspace_bytes, void* stream);

/*
 * The stages of sparse_attn_bwd (bf16), for callers that schedule them
 * themselves (the dQ and the dK / dV stages of one call, given the row
 * statistics, touch disjoint outputs) and for timing the stages apart:
 *   SA_BWD_ROW_STATS  D_i = dO_i . O_i and the LSE in base 2, per row, into the
 *                     workspace (Sec. 5.4: the only per-row state the
 *                     recomputation needs besides LSE);
 *   SA_BWD_DQ         dQ, row by row over the layout;
 *   SA_BWD_DKDV       dK and dV, column by column.
 * `stages` is a bit set of them; stages run in this order within a call, and
 * a stage needs the earlier ones of the same call (same arguments, same
 * workspace) already enqueued: SA_BWD_DQ and SA_BWD_DKDV read the row
 * statistics, and SA_BWD_DKDV also reads D where the dQ stage recomputes it
 * (fixed pattern with few summary keys per row) and the work order the row
 * statistics stage lays out (so each SA_BWD_DKDV needs its own earlier
 * SA_BWD_ROW_STATS).  SA_BWD_ROW_STATS and SA_BWD_DQ in one call run as one
 * launch where the dQ grid allows (its kernel then computes its rows'
 * statistics itself); results are the same either way up to the summation
 * order of D.  All three in one call equal sparse_attn_bwd.  Arguments and
 * errors as sparse_attn_bwd; SA_ERR_INVALID for an empty or unknown set,
 * SA_ERR_UNSUPPORTED for a partial set in fp32.
 */
enum { SA_BWD_ROW_STATS = 1, SA_BWD_DQ = 2, SA_BWD_DKDV = 4, SA_BWD_ALL_STAGES = 7 };

int sparse_attn_bwd_stage(int64_t n, int32_t block, int32_t stride_l, int32_t summary_c, int32_t pattern,
                          int32_t head_mode, const int32_t* row_ptr, const int32_t* col_idx, const uint8_t* kind,
                          const int32_t* col_ptr, const int32_t* row_idx, const uint8_t* kind_t, int32_t batch,
                          int32_t heads, int32_t d_head, int32_t dtype, const void* q, const void* k, const void* v,
                          const void* o, const void* dout, const float* lse, const int64_t* strides,
                          float softmax_scale, void* dq, void* dk, void* dv, void* workspace, size_t workspace_bytes,
                          int32_t stages, void* stream);

/*
 * sparse_attn_bwd without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, serving loops,
 * harnesses that forbid allocation).  Same arguments, results and errors as
 * sparse_attn_bwd less the workspace; the library uses a fixed device array
 * of sparse_attn_bwd_noalloc_max_workspace bytes (64 MiB) instead, one per
 * device, held until the process ends, and allocates nothing (no hipMalloc,
 * no allocating library call).  A call whose workspace size
 * (sparse_attn_bwd_workspace_size) exceeds it returns SA_ERR_BUFFER_TOO_SMALL
 * without enqueueing anything (n = 65,536 with 8 heads needs 4 MiB, n =
 * 1,048,576 with 4 heads 32 MiB).  `stream` must belong to the current
 * device (SA_ERR_INVALID otherwise).  Every call on one device shares that
 * device's array: calls that overlap on one device race and must be ordered
 * by the caller (one stream, or events).  The array keeps the last call's
 * contents; nothing in it needs to start at zero.
 */
int sparse_attn_bwd_noalloc_max_workspace(size_t* bytes);

int sparse_attn_bwd_noalloc(int64_t n, int32_t block, int32_t stride_l, int32_t summary_c, int32_t pattern,
                            int32_t head_mode, const int32_t* row_ptr, const int32_t* col_idx, const uint8_t* kind,
                            const int32_t* col_ptr, const int32_t* row_idx, const uint8_t* kind_t, int32_t batch,
                            int32_t heads, int32_t d_head, int32_t dtype, const void* q, const void* k, const void* v,
                            const void* o, const void* dout, const float* lse, const int64_t* strides,
                            float softmax_scale, void* dq, void* dk, void* dv, void* stream);

/*
 * Bytes of device workspace that sparse_attn_decode needs (host only): the
 * partial softmax states of the key ranges a decoding step is split into,
 * (d_head + 2) fp32 values per range and (batch, head).  Pattern arguments
 * as in sparse_attn_decode.
 */
int sparse_attn_decode_workspace_size(int64_t pos, int32_t stride_l, int32_t summary_c, int32_t pattern,
                                      int32_t head_mode, int32_t batch, int32_t heads, int32_t d_head,
                                      int32_t dtype, size_t* bytes);

/*
 * One step of autoregressive generation (the samples of Fig. 1 are drawn one
 * position at a time, Sec. 5.6): for every (batch, head), the output of the
 * single query at position pos attending S_pos (Sec. 4.3, heads combined as
 * in Sec. 5.1) over a key / value cache that holds positions 0 .. pos:
 *     o = softmax_j( scale * q . k_j )  v_j     over j in S_pos.
 * The same result as row pos of sparse_attn_fwd on a sequence of pos + 1
 * positions, without a layout: S_pos is enumerated directly (no block size),
 * and q . k and the softmax are computed in fp32 (the paper casts queries and
 * keys to single precision for sampling).
 *   q        [batch, heads, d_head], element strides q_strides[0..1] (batch,
 *            head), d contiguous.  o has the same shape and strides.
 *   k_cache, v_cache  [batch, heads, >= pos + 1, d_head], element strides
 *            kv_strides[0..2] (batch, head, sequence), d contiguous, sequence
 *            stride >= d_head.
 *   lse      [batch, heads] contiguous fp32, natural log; -inf (and o = 0)
 *            when S_pos is empty.
 * Every base address 16-byte aligned and every stride a multiple of 16 bytes.
 * workspace: at least sparse_attn_decode_workspace_size bytes of device memory,
 * 16-byte aligned (SA_ERR_BUFFER_TOO_SMALL otherwise); its contents on entry
 * are ignored and calls sharing one workspace must not overlap.
 * pos in [0, 2^31 - 1]; pattern, head_mode, stride_l, summary_c, d_head and
 * dtype as in sparse_attn_fwd.
 */
int sparse_attn_decode(int64_t pos, int32_t stride_l, int32_t summary_c, int32_t pattern, int32_t head_mode,
                       int32_t batch, int32_t heads, int32_t d_head, int32_t dtype, const void* q,
                       const int64_t* q_strides, const void* k_cache, const void* v_cache,
                       const int64_t* kv_strides, float softmax_scale, void* o, float* lse, void* workspace,
                       size_t workspace_bytes, void* stream);

/*
 * Strided pattern, merged heads (SA_STRIDED, SA_MODE_MERGED), with the A2
 * part computed by transposition (Sec. 5.5: reordered by residue mod l, a
 * stride of l becomes a local window), with the caller choosing the class
 * block.  Same results as sparse_attn_fwd / sparse_attn_bwd over the merged
 * layout (which take this route by themselves for bf16 when l divides n, B
 * divides l and n / l is a multiple of 16), computed as
 *   the band  A1 = {max(0, i-l) .. i}: the block kernels over the strided A1
 *             layout (sparse_attn_layout with SA_MODE_A1 and the same n,
 *             block, stride_l, summary_c = 0), and
 *   the rest  {i - k l : k >= 2}: in each residue class (positions r + m l,
 *             m < M = n / l), query m attends keys m' <= m - 2, dense causal
 *             attention over blocks of class_block class positions, read in
 *             place through strided views,
 * combined through their log-sum-exps (the sets are disjoint): the class
 * kernels merge their part into the band's O and LSE, and add their
 * gradients to the band's.
 * Requirements beyond the common ones: l divides n; class_block in
 * {16, 32, 64} divides M (SA_ERR_INVALID otherwise); M / class_block <= 65535
 * and batch * heads <= 65535 (else SA_ERR_UNSUPPORTED); q, k, v, o, dout, dq,
 * dk, dv contiguous [batch, heads, n, d_head] (no strides argument).
 * Workspace: device memory of at least sparse_attn_transposed_workspace_size
 * bytes (the backward's row statistics and schedule, as sparse_attn_bwd),
 * 256-byte aligned (SA_ERR_INVALID otherwise); one size serves both calls,
 * and the forward does not touch it.  Its contents on entry are ignored and
 * calls sharing one workspace must not overlap.  The row pointers are those
 * of the A1 layout; the backward also takes its column form.  Outputs as for
 * sparse_attn_fwd / sparse_attn_bwd.
 */
int sparse_attn_transposed_workspace_size(int64_t n, int32_t block, int32_t stride_l, int32_t class_block,
                                          int32_t batch, int32_t heads, int32_t d_head, int32_t dtype, size_t* bytes);

int sparse_attn_fwd_transposed(int64_t n, int32_t block, int32_t stride_l, int32_t class_block,
                               const int32_t* row_ptr, const int32_t* col_idx, const uint8_t* kind, int32_t batch,
                               int32_t heads, int32_t d_head, int32_t dtype, const void* q, const void* k,
                               const void* v, float softmax_scale, void* o, float* lse, void* workspace,
                               size_t workspace_bytes, void* stream);

int sparse_attn_bwd_transposed(int64_t n, int32_t block, int32_t stride_l, int32_t class_block,
                               const int32_t* row_ptr, const int32_t* col_idx, const uint8_t* kind,
                               const int32_t* col_ptr, const int32_t* row_idx, const uint8_t* kind_t, int32_t batch,
                               int32_t heads, int32_t d_head, int32_t dtype, const void* q, const void* k,
                               const void* v, const void* o, const void* dout, const float* lse, float softmax_scale,
                               void* dq, void* dk, void* dv, void* workspace, size_t workspace_bytes, void* stream);

/* Static English description of a status code (never NULL). */
const char* sparse_attn_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* SPARSE_ATTN_H */
