/*
 * Oracle for factorized sparse causal attention (Child et al., 2019,
 * "Generating Long Sequences with Sparse Transformers").
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow, fp64 CPU reference
 * that the GPU library is checked against.  Only the tests, the smoke check and
 * the CPU-baseline leg of the benchmark may load it.  It shares no code, header,
 * table or helper with the GPU library, and the GPU library never calls it.
 *
 * Everything here follows the paper's definitions directly:
 *   - the attend function, Sec. 4.2 (eq. attend_fn): for each output i,
 *     softmax over j in S_i of (q_i . k_j)/sqrt(d), applied to v_j;
 *   - the factorized sets, Sec. 4.3: strided A1 = {max(0,i-l) .. i},
 *     strided A2 = {j : (i-j) mod l = 0}, fixed A1 = {j : floor(j/l) = floor(i/l)},
 *     fixed A2 = {j : j mod l in {l-c .. l-1}}; every set is intersected with
 *     {j : j <= i} (Sec. 4.2, factorized self-attention);
 *   - the head-combination modes, Sec. 5.1: one factor per call (eq. sepwpmat),
 *     the merged union (eq. mergedmat), and per-head factors inside multi-head
 *     attention (heads alternate A1, A2);
 *   - recomputation, Sec. 5.4: the backward pass needs only the saved
 *     log-sum-exp of each row; the attention weights are recomputed.
 *
 * The forward is a two-pass softmax per row (max, then sum).  The backward is
 * the textbook gradient of L = sum(O * dO):
 *   D_i = dO_i . O_i,  dP_ij = dO_i . v_j,  dS_ij = P_ij (dP_ij - D_i),
 *   dq_i = scale sum_j dS_ij k_j,  dk_j = scale sum_i dS_ij q_i,
 *   dv_j = sum_i P_ij dO_i,
 * computed row by row for dq and column by column for dk, dv, so that nothing
 * of size n x n is ever stored.
 *
 * Readings of points the paper leaves open (indices are 0-based):
 *   - strided A1 has l+1 elements, as the set formula gives;
 *   - fixed A2 keeps the summary columns of the query's own block when j <= i;
 *   - a row whose set is empty (fixed A2 alone, first block) has O = 0,
 *     LSE = -inf, and contributes no gradient;
 *   - a merged set is a set union: each j is counted once;
 *   - distinct summary subblocks per head (Sec. 4.3, the remark closing the
 *     fixed pattern: heads may look at different c-wide subblocks of each
 *     l-block): pattern code 2.  The floor(l/c) subblocks are numbered from
 *     the end of the block, subblock s holding the positions l-(s+1)c ..
 *     l-sc-1 of every block, and head h takes s = h mod floor(l/c).  s = 0 is
 *     the shared window of the plain fixed pattern.
 *
 * Inputs are read as fp64, fp32 or bf16 (raw 16-bit patterns), each converted
 * exactly to fp64.  Outputs are fp64.  Layout of every tensor: [b, h, n, d],
 * d contiguous.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { O_STRIDED = 0, O_FIXED = 1, O_FIXED_PER_HEAD = 2 };
enum { O_MODE_A1 = 0, O_MODE_A2 = 1, O_MODE_MERGED = 2, O_MODE_INTERLEAVED = 3 };
enum { O_PART_A1 = 0, O_PART_A2 = 1, O_PART_MERGED = 2 };
enum { O_F64 = 0, O_F32 = 1, O_BF16 = 2 };

int oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ---------------------------------------------------------------------------
 * Sets.  Which factor a head uses (Sec. 5.1): A1 or A2 for the whole call,
 * their union when merged, and A1 on even heads / A2 on odd heads when the
 * factors are spread over the heads of one multi-head call.
 * ------------------------------------------------------------------------- */
static int head_part(int mode, int64_t h) {
    switch (mode) {
    case O_MODE_A1: return O_PART_A1;
    case O_MODE_A2: return O_PART_A2;
    case O_MODE_MERGED: return O_PART_MERGED;
    default: return (h % 2 == 0) ? O_PART_A1 : O_PART_A2;
    }
}

/* First position, inside each l-block, of the c summary columns head h
 * attends (Sec. 4.3): the last c positions, or with distinct subblocks per
 * head subblock s = h mod floor(l/c), counted from the end of the block. */
static int64_t summary_start(int pattern, int64_t l, int64_t c, int64_t h) {
    if (pattern != O_FIXED_PER_HEAD) return l - c;
    return l - (h % (l / c) + 1) * c;
}

static int64_t imax(int64_t a, int64_t b) { return a > b ? a : b; }
static int64_t imin(int64_t a, int64_t b) { return a < b ? a : b; }

/* Append the integers lo..hi (inclusive) to out, if any.  Returns new count. */
static int64_t put_range(int64_t* out, int64_t cnt, int64_t lo, int64_t hi) {
    for (int64_t j = lo; j <= hi; ++j) {
        if (out) out[cnt] = j;
        ++cnt;
    }
    return cnt;
}

/* S_i for one part, ascending j, all within [0, i] (Sec. 4.3); w is the
 * first summary position inside a block (fixed pattern).  Returns |S_i|;
 * writes the members to out when out is not NULL. */
static int64_t row_set_w(int pattern, int part, int64_t l, int64_t c, int64_t w, int64_t i,
                         int64_t* out) {
    int64_t cnt = 0;
    if (pattern == O_STRIDED) {
        int64_t t = imax(0, i - l); /* A1 = {t, ..., i} */
        if (part == O_PART_A1) return put_range(out, 0, t, i);
        if (part == O_PART_A2) {
            /* (i - j) mod l = 0 and 0 <= j <= i: j = i mod l, i mod l + l, ..., i */
            for (int64_t j = i % l; j <= i; j += l) {
                if (out) out[cnt] = j;
                ++cnt;
            }
            return cnt;
        }
        /* union: the A2 members below t, then all of A1 */
        for (int64_t j = i % l; j < t; j += l) {
            if (out) out[cnt] = j;
            ++cnt;
        }
        return put_range(out, cnt, t, i);
    }
    /* fixed: A1 is the query's own l-block up to i, A2 the columns at
     * positions w .. w+c-1 of every block */
    int64_t blk = i / l;
    if (part == O_PART_A1) return put_range(out, 0, blk * l, i);
    if (part == O_PART_A2) {
        for (int64_t L = 0; L <= blk; ++L)
            cnt = put_range(out, cnt, L * l + w, imin(L * l + w + c - 1, i));
        return cnt;
    }
    /* union: the summary columns of the earlier blocks, then all of A1 (the
     * own block's summary columns up to i lie inside A1) */
    for (int64_t L = 0; L < blk; ++L)
        cnt = put_range(out, cnt, L * l + w, L * l + w + c - 1);
    return put_range(out, cnt, blk * l, i);
}

/* T_j = {i : j in S_i}, ascending i, within [j, n-1]. */
static int64_t col_set_w(int pattern, int part, int64_t n, int64_t l, int64_t c, int64_t w,
                         int64_t j, int64_t* out) {
    int64_t cnt = 0;
    if (pattern == O_STRIDED) {
        int64_t a1_hi = imin(n - 1, j + l); /* i - l <= j <= i */
        if (part == O_PART_A1) return put_range(out, 0, j, a1_hi);
        if (part == O_PART_A2) {
            for (int64_t i = j; i < n; i += l) {
                if (out) out[cnt] = i;
                ++cnt;
            }
            return cnt;
        }
        cnt = put_range(out, 0, j, a1_hi);
        for (int64_t i = j + 2 * l; i < n; i += l) { /* j + l is already in A1 */
            if (out) out[cnt] = i;
            ++cnt;
        }
        return cnt;
    }
    int summary = (j % l) >= w && (j % l) < w + c;
    int64_t blk_hi = imin(n - 1, (j / l) * l + l - 1);
    if (part == O_PART_A1) return put_range(out, 0, j, blk_hi);
    if (part == O_PART_A2) return summary ? put_range(out, 0, j, n - 1) : 0;
    return put_range(out, 0, j, summary ? n - 1 : blk_hi);
}

/* S_i of one factor with the shared summary window (patterns 0 and 1; any
 * other code is read as the fixed pattern). */
int64_t oracle_row_set(int pattern, int part, int64_t n, int64_t l, int64_t c,
                       int64_t i, int64_t* out) {
    (void)n;
    return row_set_w(pattern, part, l, c, summary_start(O_FIXED, l, c, 0), i, out);
}

int64_t oracle_col_set(int pattern, int part, int64_t n, int64_t l, int64_t c,
                       int64_t j, int64_t* out) {
    return col_set_w(pattern, part, n, l, c, summary_start(O_FIXED, l, c, 0), j, out);
}

/* S_i and T_j of head h of a multi-head call: its factor (Sec. 5.1) and, for
 * pattern 2, its own summary subblock. */
int64_t oracle_head_row_set(int pattern, int mode, int64_t n, int64_t l, int64_t c, int64_t h,
                            int64_t i, int64_t* out) {
    (void)n;
    return row_set_w(pattern, head_part(mode, h), l, c, summary_start(pattern, l, c, h), i, out);
}

int64_t oracle_head_col_set(int pattern, int mode, int64_t n, int64_t l, int64_t c, int64_t h,
                            int64_t j, int64_t* out) {
    return col_set_w(pattern, head_part(mode, h), n, l, c, summary_start(pattern, l, c, h), j, out);
}

/* ---------------------------------------------------------------------------
 * Input access: element e of a tensor stored as fp64, fp32 or bf16 bits.
 * ------------------------------------------------------------------------- */
static double load_elem(const void* p, int dtype, int64_t e) {
    if (dtype == O_F64) return ((const double*)p)[e];
    if (dtype == O_F32) return (double)((const float*)p)[e];
    uint32_t bits = (uint32_t)((const uint16_t*)p)[e] << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

typedef struct {
    int pattern, mode;
    int64_t n, l, c, heads, d;
    int dtype;
    const void *q, *k, *v, *dout;
    double scale;
} problem;

static int64_t row_base(const problem* P, int64_t bh, int64_t i) {
    return (bh * P->n + i) * P->d;
}

static double dot_qk(const problem* P, int64_t bh, int64_t i, int64_t j) {
    double s = 0.0;
    int64_t qi = row_base(P, bh, i), kj = row_base(P, bh, j);
    for (int64_t t = 0; t < P->d; ++t)
        s += load_elem(P->q, P->dtype, qi + t) * load_elem(P->k, P->dtype, kj + t);
    return s;
}

static double dot_dov(const problem* P, int64_t bh, int64_t i, int64_t j) {
    double s = 0.0;
    int64_t oi = row_base(P, bh, i), vj = row_base(P, bh, j);
    for (int64_t t = 0; t < P->d; ++t)
        s += load_elem(P->dout, P->dtype, oi + t) * load_elem(P->v, P->dtype, vj + t);
    return s;
}

/* Forward for one row (Sec. 4.2): a(x_i, S_i) with a two-pass softmax.
 * jbuf and sbuf hold at least n entries.  Writes o[0..d) and *lse. */
static void row_forward(const problem* P, int64_t bh, int64_t i, int64_t* jbuf,
                        double* sbuf, double* o, double* lse) {
    int64_t cnt = oracle_head_row_set(P->pattern, P->mode, P->n, P->l, P->c, bh % P->heads, i, jbuf);
    for (int64_t t = 0; t < P->d; ++t) o[t] = 0.0;
    if (cnt == 0) {
        *lse = -INFINITY;
        return;
    }
    double m = -INFINITY;
    for (int64_t a = 0; a < cnt; ++a) {
        sbuf[a] = P->scale * dot_qk(P, bh, i, jbuf[a]);
        if (sbuf[a] > m) m = sbuf[a];
    }
    double z = 0.0;
    for (int64_t a = 0; a < cnt; ++a) z += exp(sbuf[a] - m);
    for (int64_t a = 0; a < cnt; ++a) {
        double p = exp(sbuf[a] - m) / z;
        int64_t vj = row_base(P, bh, jbuf[a]);
        for (int64_t t = 0; t < P->d; ++t) o[t] += p * load_elem(P->v, P->dtype, vj + t);
    }
    *lse = m + log(z);
}

/* D_i = dO_i . O_i, with the oracle's own fp64 O. */
static double row_delta(const problem* P, int64_t bh, int64_t i, const double* o) {
    double s = 0.0;
    int64_t oi = row_base(P, bh, i);
    for (int64_t t = 0; t < P->d; ++t) s += load_elem(P->dout, P->dtype, oi + t) * o[t];
    return s;
}

/* dq_i = scale * sum_{j in S_i} P_ij (dP_ij - D_i) k_j, with P recomputed from
 * the saved LSE (Sec. 5.4). */
static void row_dq(const problem* P, int64_t bh, int64_t i, int64_t* jbuf,
                   double lse, double delta, double* dq) {
    int64_t cnt = oracle_head_row_set(P->pattern, P->mode, P->n, P->l, P->c, bh % P->heads, i, jbuf);
    for (int64_t t = 0; t < P->d; ++t) dq[t] = 0.0;
    for (int64_t a = 0; a < cnt; ++a) {
        int64_t j = jbuf[a];
        double p = exp(P->scale * dot_qk(P, bh, i, j) - lse);
        double ds = p * (dot_dov(P, bh, i, j) - delta);
        int64_t kj = row_base(P, bh, j);
        for (int64_t t = 0; t < P->d; ++t)
            dq[t] += P->scale * ds * load_elem(P->k, P->dtype, kj + t);
    }
}

/* dk_j, dv_j by the column pass over T_j; lse[] and delta[] indexed by row. */
static void col_dkdv(const problem* P, int64_t bh, int64_t j, int64_t* ibuf,
                     const double* lse, const double* delta, double* dk, double* dv) {
    int64_t cnt = oracle_head_col_set(P->pattern, P->mode, P->n, P->l, P->c, bh % P->heads, j, ibuf);
    for (int64_t t = 0; t < P->d; ++t) dk[t] = dv[t] = 0.0;
    for (int64_t a = 0; a < cnt; ++a) {
        int64_t i = ibuf[a];
        double p = exp(P->scale * dot_qk(P, bh, i, j) - lse[i]);
        double ds = p * (dot_dov(P, bh, i, j) - delta[i]);
        int64_t qi = row_base(P, bh, i);
        for (int64_t t = 0; t < P->d; ++t) {
            dv[t] += p * load_elem(P->dout, P->dtype, qi + t);
            dk[t] += P->scale * ds * load_elem(P->q, P->dtype, qi + t);
        }
    }
}

static int check_problem(const problem* P) {
    if (P->n < 1 || P->l < 1 || P->d < 1 || P->heads < 1) return -1;
    if (P->pattern < O_STRIDED || P->pattern > O_FIXED_PER_HEAD) return -1;
    if (P->mode < O_MODE_A1 || P->mode > O_MODE_INTERLEAVED) return -1;
    if (P->pattern != O_STRIDED && (P->c < 1 || P->c > P->l)) return -1;
    if (P->dtype < O_F64 || P->dtype > O_BF16) return -1;
    return 0;
}

static problem make_problem(int pattern, int mode, int64_t n, int64_t l, int64_t c,
                            int64_t heads, int64_t d, int dtype, const void* q,
                            const void* k, const void* v, const void* dout, double scale) {
    problem P;
    P.pattern = pattern; P.mode = mode; P.n = n; P.l = l; P.c = c;
    P.heads = heads; P.d = d; P.dtype = dtype;
    P.q = q; P.k = k; P.v = v; P.dout = dout; P.scale = scale;
    return P;
}

/* Full forward: o[b,h,n,d], lse[b,h,n]. */
int oracle_forward(int pattern, int mode, int64_t n, int64_t l, int64_t c, int64_t batch,
                   int64_t heads, int64_t d, int dtype, const void* q, const void* k,
                   const void* v, double scale, double* o, double* lse) {
    problem P = make_problem(pattern, mode, n, l, c, heads, d, dtype, q, k, v, NULL, scale);
    if (check_problem(&P) || batch < 1) return -1;
    int64_t rows = batch * heads * n;
    int err = 0;
#pragma omp parallel
    {
        int64_t* jbuf = malloc(sizeof(int64_t) * n);
        double* sbuf = malloc(sizeof(double) * n);
        if (!jbuf || !sbuf) {
#pragma omp atomic write
            err = -2;
        } else {
#pragma omp for schedule(dynamic, 64)
            for (int64_t r = 0; r < rows; ++r)
                row_forward(&P, r / n, r % n, jbuf, sbuf, o + r * d, lse + r);
        }
        free(jbuf);
        free(sbuf);
    }
    return err;
}

/* Full backward of L = sum(O * dout).  Recomputes the forward itself; o, lse,
 * delta (each may be NULL) receive the oracle's own O, LSE and D. */
int oracle_backward(int pattern, int mode, int64_t n, int64_t l, int64_t c, int64_t batch,
                    int64_t heads, int64_t d, int dtype, const void* q, const void* k,
                    const void* v, const void* dout, double scale, double* o_out,
                    double* lse_out, double* delta_out, double* dq, double* dk, double* dv) {
    problem P = make_problem(pattern, mode, n, l, c, heads, d, dtype, q, k, v, dout, scale);
    if (check_problem(&P) || batch < 1) return -1;
    int64_t rows = batch * heads * n;
    double* lse = malloc(sizeof(double) * rows);
    double* delta = malloc(sizeof(double) * rows);
    if (!lse || !delta) {
        free(lse);
        free(delta);
        return -2;
    }
    int err = 0;
    /* row pass: O, LSE, D, dq */
#pragma omp parallel
    {
        int64_t* jbuf = malloc(sizeof(int64_t) * n);
        double* sbuf = malloc(sizeof(double) * n);
        double* orow = malloc(sizeof(double) * d);
        if (!jbuf || !sbuf || !orow) {
#pragma omp atomic write
            err = -2;
        } else {
#pragma omp for schedule(dynamic, 64)
            for (int64_t r = 0; r < rows; ++r) {
                int64_t bh = r / n, i = r % n;
                row_forward(&P, bh, i, jbuf, sbuf, orow, &lse[r]);
                delta[r] = row_delta(&P, bh, i, orow);
                if (o_out) memcpy(o_out + r * d, orow, sizeof(double) * d);
                row_dq(&P, bh, i, jbuf, lse[r], delta[r], dq + r * d);
            }
        }
        free(jbuf);
        free(sbuf);
        free(orow);
    }
    /* column pass: dk, dv */
    if (!err) {
#pragma omp parallel
        {
            int64_t* ibuf = malloc(sizeof(int64_t) * n);
            if (!ibuf) {
#pragma omp atomic write
                err = -2;
            } else {
#pragma omp for schedule(dynamic, 64)
                for (int64_t r = 0; r < rows; ++r) {
                    int64_t bh = r / n;
                    col_dkdv(&P, bh, r % n, ibuf, lse + bh * n, delta + bh * n,
                             dk + r * d, dv + r * d);
                }
            }
            free(ibuf);
        }
    }
    if (lse_out) memcpy(lse_out, lse, sizeof(double) * rows);
    if (delta_out) memcpy(delta_out, delta, sizeof(double) * rows);
    free(lse);
    free(delta);
    return err;
}

/* Sampled forward: rows[r] = (b*heads + h)*n + i; o is [nrows, d]. */
int oracle_forward_rows(int pattern, int mode, int64_t n, int64_t l, int64_t c,
                        int64_t heads, int64_t d, int dtype, const void* q, const void* k,
                        const void* v, double scale, int64_t nrows, const int64_t* rows,
                        double* o, double* lse) {
    problem P = make_problem(pattern, mode, n, l, c, heads, d, dtype, q, k, v, NULL, scale);
    if (check_problem(&P)) return -1;
    int err = 0;
#pragma omp parallel
    {
        int64_t* jbuf = malloc(sizeof(int64_t) * n);
        double* sbuf = malloc(sizeof(double) * n);
        if (!jbuf || !sbuf) {
#pragma omp atomic write
            err = -2;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t r = 0; r < nrows; ++r)
                row_forward(&P, rows[r] / n, rows[r] % n, jbuf, sbuf, o + r * d, lse + r);
        }
        free(jbuf);
        free(sbuf);
    }
    return err;
}

/* Sampled dq: rows as in oracle_forward_rows; dq is [nrows, d]. */
int oracle_backward_rows(int pattern, int mode, int64_t n, int64_t l, int64_t c,
                         int64_t heads, int64_t d, int dtype, const void* q, const void* k,
                         const void* v, const void* dout, double scale, int64_t nrows,
                         const int64_t* rows, double* dq) {
    problem P = make_problem(pattern, mode, n, l, c, heads, d, dtype, q, k, v, dout, scale);
    if (check_problem(&P)) return -1;
    int err = 0;
#pragma omp parallel
    {
        int64_t* jbuf = malloc(sizeof(int64_t) * n);
        double* sbuf = malloc(sizeof(double) * n);
        double* orow = malloc(sizeof(double) * d);
        if (!jbuf || !sbuf || !orow) {
#pragma omp atomic write
            err = -2;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t r = 0; r < nrows; ++r) {
                int64_t bh = rows[r] / n, i = rows[r] % n;
                double lse;
                row_forward(&P, bh, i, jbuf, sbuf, orow, &lse);
                double delta = row_delta(&P, bh, i, orow);
                row_dq(&P, bh, i, jbuf, lse, delta, dq + r * d);
            }
        }
        free(jbuf);
        free(sbuf);
        free(orow);
    }
    return err;
}

/* Sampled dk, dv: cols[r] = (b*heads + h)*n + j; dk, dv are [ncols, d].  The
 * LSE and D of every row in T_j are recomputed for each sampled column. */
int oracle_backward_cols(int pattern, int mode, int64_t n, int64_t l, int64_t c,
                         int64_t heads, int64_t d, int dtype, const void* q, const void* k,
                         const void* v, const void* dout, double scale, int64_t ncols,
                         const int64_t* cols, double* dk, double* dv) {
    problem P = make_problem(pattern, mode, n, l, c, heads, d, dtype, q, k, v, dout, scale);
    if (check_problem(&P)) return -1;
    int err = 0;
    for (int64_t r = 0; r < ncols && !err; ++r) {
        int64_t bh = cols[r] / n, j = cols[r] % n;
        int64_t* ibuf = malloc(sizeof(int64_t) * n);
        double* lse = calloc((size_t)n, sizeof(double));
        double* delta = calloc((size_t)n, sizeof(double));
        if (!ibuf || !lse || !delta) {
            err = -2;
        } else {
            int64_t cnt = oracle_head_col_set(P.pattern, P.mode, n, l, c, bh % P.heads, j, ibuf);
#pragma omp parallel
            {
                int64_t* jbuf = malloc(sizeof(int64_t) * n);
                double* sbuf = malloc(sizeof(double) * n);
                double* orow = malloc(sizeof(double) * d);
                if (!jbuf || !sbuf || !orow) {
#pragma omp atomic write
                    err = -2;
                } else {
#pragma omp for schedule(dynamic, 4)
                    for (int64_t a = 0; a < cnt; ++a) {
                        int64_t i = ibuf[a];
                        row_forward(&P, bh, i, jbuf, sbuf, orow, &lse[i]);
                        delta[i] = row_delta(&P, bh, i, orow);
                    }
                }
                free(jbuf);
                free(sbuf);
                free(orow);
            }
            if (!err) col_dkdv(&P, bh, j, ibuf, lse, delta, dk + r * d, dv + r * d);
        }
        free(ibuf);
        free(lse);
        free(delta);
    }
    return err;
}

/* ---------------------------------------------------------------------------
 * Block layout by brute force (Sec. 5.5: the product is computed in blocks,
 * and the upper triangle is never touched).  For each layout g and each query
 * tile qb, every attended pair (i, j) with i in the tile increments a counter
 * for key tile j / B.  A tile is present iff its counter is positive, and is
 * FULL (kind 0) iff all B*B of its pairs are attended, else MASKED (kind 1).
 *
 * Layouts, one per distinct set of the heads of a call:
 *   - shared summary window (patterns 0 and 1): one layout, except when heads
 *     alternate the two factors, where layout 0 is A1 and layout 1 is A2;
 *   - distinct subblocks (pattern 2), S = floor(l/c): A1 alone has one
 *     layout (A1 has no summary columns); A2 or merged has S layouts, layout
 *     s for subblock s (head h uses layout h mod S); alternating heads have
 *     1 + S, layout 0 for A1 and layout 1 + s for A2 with subblock s (odd
 *     head h uses layout 1 + h mod S).
 * Rows of all layouts are concatenated; row_ptr[g*(nq+1) + qb] is an
 * absolute offset into col_idx.  col_ptr / row_idx / kind_t are the same
 * tiles in column order.
 * ------------------------------------------------------------------------- */
int oracle_num_layouts(int64_t l, int64_t c, int pattern, int mode) {
    if (pattern != O_FIXED_PER_HEAD || mode == O_MODE_A1)
        return mode == O_MODE_INTERLEAVED ? 2 : 1;
    int64_t S = l / c;
    return (int)(mode == O_MODE_INTERLEAVED ? 1 + S : S);
}

/* Factor and summary window start of layout g. */
static void layout_set(int64_t l, int64_t c, int pattern, int mode, int g, int* part, int64_t* w) {
    int s = 0;
    if (mode == O_MODE_INTERLEAVED) {
        *part = g == 0 ? O_PART_A1 : O_PART_A2;
        s = g == 0 ? 0 : g - 1;
    } else {
        *part = head_part(mode, 0);
        s = g;
    }
    *w = pattern == O_FIXED_PER_HEAD ? l - (s + 1) * c : l - c;
}

static int check_layout_args(int64_t n, int64_t B, int64_t l, int64_t c, int pattern, int mode) {
    if (n < 1 || B < 1 || n % B != 0 || l < 1) return -1;
    if (pattern < O_STRIDED || pattern > O_FIXED_PER_HEAD) return -1;
    if (mode < O_MODE_A1 || mode > O_MODE_INTERLEAVED) return -1;
    if (pattern != O_STRIDED && (c < 1 || c > l)) return -1;
    return 0;
}

/* Count attended pairs of query tile qb per key tile into cnt[0..nq). */
static void tile_row_counts(int pattern, int part, int64_t w, int64_t n, int64_t B, int64_t l,
                            int64_t c, int64_t qb, int64_t* cnt, int64_t* jbuf) {
    int64_t nq = n / B;
    for (int64_t kb = 0; kb < nq; ++kb) cnt[kb] = 0;
    for (int64_t i = qb * B; i < qb * B + B; ++i) {
        int64_t m = row_set_w(pattern, part, l, c, w, i, jbuf);
        for (int64_t a = 0; a < m; ++a) cnt[jbuf[a] / B] += 1;
    }
}

/* n_layouts and nnz per layout; nnz holds max(2, oracle_num_layouts(...))
 * entries (unused ones are set to 0). */
int oracle_layout_count(int64_t n, int64_t B, int64_t l, int64_t c, int pattern, int mode,
                        int64_t* n_layouts, int64_t* nnz) {
    if (check_layout_args(n, B, l, c, pattern, mode)) return -1;
    int ng = oracle_num_layouts(l, c, pattern, mode);
    int64_t nq = n / B;
    nnz[0] = nnz[1] = 0;
    for (int g = 0; g < ng; ++g) {
        int part;
        int64_t w;
        layout_set(l, c, pattern, mode, g, &part, &w);
        int64_t total = 0;
#pragma omp parallel
        {
            int64_t* cnt = malloc(sizeof(int64_t) * nq);
            int64_t* jbuf = malloc(sizeof(int64_t) * n);
#pragma omp for schedule(dynamic, 1) reduction(+ : total)
            for (int64_t qb = 0; qb < nq; ++qb) {
                tile_row_counts(pattern, part, w, n, B, l, c, qb, cnt, jbuf);
                for (int64_t kb = 0; kb < nq; ++kb) total += cnt[kb] > 0;
            }
            free(cnt);
            free(jbuf);
        }
        nnz[g] = total;
    }
    *n_layouts = ng;
    return 0;
}

int oracle_layout_fill(int64_t n, int64_t B, int64_t l, int64_t c, int pattern, int mode,
                       int32_t* row_ptr, int32_t* col_idx, uint8_t* kind, int32_t* col_ptr,
                       int32_t* row_idx, uint8_t* kind_t) {
    if (check_layout_args(n, B, l, c, pattern, mode)) return -1;
    int ng = oracle_num_layouts(l, c, pattern, mode);
    int64_t nq = n / B;
    int64_t base = 0;
    for (int g = 0; g < ng; ++g) {
        int part;
        int64_t w;
        layout_set(l, c, pattern, mode, g, &part, &w);
        int32_t* rp = row_ptr + g * (nq + 1);
        int32_t* cp = col_ptr + g * (nq + 1);
        /* pass 1: tiles per query tile */
        int64_t* rowcnt = calloc((size_t)nq, sizeof(int64_t));
#pragma omp parallel
        {
            int64_t* cnt = malloc(sizeof(int64_t) * nq);
            int64_t* jbuf = malloc(sizeof(int64_t) * n);
#pragma omp for schedule(dynamic, 1)
            for (int64_t qb = 0; qb < nq; ++qb) {
                tile_row_counts(pattern, part, w, n, B, l, c, qb, cnt, jbuf);
                int64_t m = 0;
                for (int64_t kb = 0; kb < nq; ++kb) m += cnt[kb] > 0;
                rowcnt[qb] = m;
            }
            free(cnt);
            free(jbuf);
        }
        rp[0] = (int32_t)base;
        for (int64_t qb = 0; qb < nq; ++qb) rp[qb + 1] = (int32_t)(rp[qb] + rowcnt[qb]);
        free(rowcnt);
        /* pass 2: fill each row in ascending key-tile order */
#pragma omp parallel
        {
            int64_t* cnt = malloc(sizeof(int64_t) * nq);
            int64_t* jbuf = malloc(sizeof(int64_t) * n);
#pragma omp for schedule(dynamic, 1)
            for (int64_t qb = 0; qb < nq; ++qb) {
                tile_row_counts(pattern, part, w, n, B, l, c, qb, cnt, jbuf);
                int64_t e = rp[qb];
                for (int64_t kb = 0; kb < nq; ++kb) {
                    if (cnt[kb] == 0) continue;
                    col_idx[e] = (int32_t)kb;
                    kind[e] = (uint8_t)(cnt[kb] == B * B ? 0 : 1);
                    ++e;
                }
            }
            free(cnt);
            free(jbuf);
        }
        /* transpose: stable counting sort of the row-ordered tiles by column */
        int64_t end = rp[nq];
        int64_t* colcnt = calloc((size_t)nq + 1, sizeof(int64_t));
        for (int64_t e = base; e < end; ++e) colcnt[col_idx[e] + 1] += 1;
        cp[0] = (int32_t)base;
        for (int64_t kb = 0; kb < nq; ++kb) cp[kb + 1] = (int32_t)(cp[kb] + colcnt[kb + 1]);
        for (int64_t kb = 0; kb < nq; ++kb) colcnt[kb] = cp[kb];
        for (int64_t qb = 0; qb < nq; ++qb)
            for (int64_t e = rp[qb]; e < rp[qb + 1]; ++e) {
                int64_t pos = colcnt[col_idx[e]]++;
                row_idx[pos] = (int32_t)qb;
                kind_t[pos] = kind[e];
            }
        free(colcnt);
        base = end;
    }
    return 0;
}
