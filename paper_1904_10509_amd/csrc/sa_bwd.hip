// Backward entry of the library (Sec. 5.4, recomputation): workspace size,
// dispatch to the bf16 kernels of each head size (sa_bwd_kernels.h,
// sa_bwd_bf16_d*.hip) and the fp32 kernels below.
//
// fp32 path: the same quantities as the bf16 kernels on the VALU, one thread
// per row for dq and one thread per column for dk / dv, using the element
// predicate; it serves the small fp32 parity case.
#include "sa_bwd_kernels.h"

namespace sa {

namespace {

// ---------------------------------------------------------------------------
// fp32, VALU
// ---------------------------------------------------------------------------
// The blocks a walk visits (see WALK_*): row qb as entries e0 .. e1 of the
// layout, column kb as entries e0 .. e0 + len (WALK_DENSE: e is the block).
__device__ inline void row_entries(const AttnArgs& a, int lay, int qb, int* e0, int* e1) {
    if (a.walk == WALK_DENSE) {
        *e0 = 0;
        *e1 = qb + 1;
        return;
    }
    const int64_t rp = (int64_t)lay * (a.nq + 1) + qb;
    *e0 = a.row_ptr[rp];
    *e1 = a.row_ptr[rp + 1];
    if (a.walk == WALK_BAND) *e0 = max(*e0, *e1 - (a.l / a.block + 1));
}
__device__ inline void col_entries(const AttnArgs& a, int lay, int kb, int* e0, int* e1) {
    if (a.walk == WALK_DENSE) {
        *e0 = kb;
        *e1 = a.nq;
        return;
    }
    const int64_t cp = (int64_t)lay * (a.nq + 1) + kb;
    *e0 = a.col_ptr[cp];
    *e1 = a.col_ptr[cp + 1];
    if (a.walk == WALK_BAND) *e1 = min(*e1, *e0 + a.l / a.block + 1);
}

template <int D>
__global__ void __launch_bounds__(64)
bwd_dq_f32_kernel(AttnArgs a, const float* __restrict__ q, const float* __restrict__ k,
                  const float* __restrict__ v, const float* __restrict__ dout,
                  const float* __restrict__ lse, const float* __restrict__ ndelta,
                  float* __restrict__ dq) {
    const int h = blockIdx.y, b = blockIdx.z;
    const int i = blockIdx.x * 64 + threadIdx.x;
    if (i >= a.n) return;
    const int qb = i / a.block;
    const int lay = head_layout(a, h);
    const int part = part_of_head(a.mode, h);
    const int32_t wst = window_start(a, subblock_of_head(a.sub, h));
    const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;
    const int64_t rowid = stat_index(a, b, h, i);
    const float L = lse[rowid], nDi = ndelta[rowid];
    const float* qr = q + base + (int64_t)i * a.ss;
    const float* gr = dout + base + (int64_t)i * a.ss;
    float acc[D];
    for (int t = 0; t < D; ++t) acc[t] = 0.f;
    int e0, e1;
    row_entries(a, lay, qb, &e0, &e1);
    for (int e = e0; e < e1; ++e) {
        const int kb = a.walk == WALK_DENSE ? e : a.col_idx[e];
        const bool full = a.walk != WALK_DENSE && a.kind[e] == TILE_FULL;
        for (int jj = 0; jj < a.block; ++jj) {
            const int jx = kb * a.block + jj;
            if (!full && !attended(a.pattern, part, a.l, a.c, wst, i - a.qshift, jx)) continue;
            const float* kr = k + base + (int64_t)jx * a.ss;
            const float* vr = v + base + (int64_t)jx * a.ss;
            float s = 0.f, dp = 0.f;
            for (int t = 0; t < D; ++t) {
                s = fmaf(qr[t], kr[t], s);
                dp = fmaf(gr[t], vr[t], dp);
            }
            const float p = expf(s * a.scale - L);
            const float dsv = p * (dp + nDi);
            for (int t = 0; t < D; ++t) acc[t] = fmaf(dsv, kr[t], acc[t]);
        }
    }
    float* drow = dq + base + (int64_t)i * a.ss;
    for (int t = 0; t < D; ++t) drow[t] = (a.epilogue == EPI_ADD ? drow[t] : 0.f) + acc[t] * a.scale;
}

template <int D>
__global__ void __launch_bounds__(64)
bwd_dkdv_f32_kernel(AttnArgs a, const float* __restrict__ q, const float* __restrict__ k,
                    const float* __restrict__ v, const float* __restrict__ dout,
                    const float* __restrict__ lse, const float* __restrict__ ndelta,
                    float* __restrict__ dk, float* __restrict__ dv) {
    const int h = blockIdx.y, b = blockIdx.z;
    const int jx = blockIdx.x * 64 + threadIdx.x;
    if (jx >= a.n) return;
    const int kb = jx / a.block;
    const int lay = head_layout(a, h);
    const int part = part_of_head(a.mode, h);
    const int32_t wst = window_start(a, subblock_of_head(a.sub, h));
    const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;
    const float* kr = k + base + (int64_t)jx * a.ss;
    const float* vr = v + base + (int64_t)jx * a.ss;
    float ak[D], av[D];
    for (int t = 0; t < D; ++t) ak[t] = av[t] = 0.f;
    int e0, e1;
    col_entries(a, lay, kb, &e0, &e1);
    for (int e = e0; e < e1; ++e) {
        const int qb = a.walk == WALK_DENSE ? e : a.row_idx[e];
        const bool full = a.walk != WALK_DENSE && a.kind_t[e] == TILE_FULL;
        for (int ii = 0; ii < a.block; ++ii) {
            const int i = qb * a.block + ii;
            if (!full && !attended(a.pattern, part, a.l, a.c, wst, i - a.qshift, jx)) continue;
            const float* qr = q + base + (int64_t)i * a.ss;
            const float* gr = dout + base + (int64_t)i * a.ss;
            float s = 0.f, dp = 0.f;
            for (int t = 0; t < D; ++t) {
                s = fmaf(qr[t], kr[t], s);
                dp = fmaf(gr[t], vr[t], dp);
            }
            const int64_t rowid = stat_index(a, b, h, i);
            const float p = expf(s * a.scale - lse[rowid]);
            const float dsv = p * (dp + ndelta[rowid]);
            for (int t = 0; t < D; ++t) {
                av[t] = fmaf(p, gr[t], av[t]);
                ak[t] = fmaf(dsv, qr[t], ak[t]);
            }
        }
    }
    float* dkrow = dk + base + (int64_t)jx * a.ss;
    float* dvrow = dv + base + (int64_t)jx * a.ss;
    const bool add = a.epilogue == EPI_ADD;
    for (int t = 0; t < D; ++t) {
        dkrow[t] = (add ? dkrow[t] : 0.f) + ak[t] * a.scale;
        dvrow[t] = (add ? dvrow[t] : 0.f) + av[t];
    }
}

template <int D>
hipError_t launch_bwd_f32(const AttnArgs& a, const void* q, const void* k, const void* v,
                          const void* o, const void* dout, const float* lse, void* dq, void* dk,
                          void* dv, const BwdWorkspace& ws, hipStream_t stream, int parts) {
    const int64_t rows = (int64_t)a.batch * a.heads * a.n;
    float* ndelta = ws.ndelta;
    if (parts & BWD_PRE)
        hipLaunchKernelGGL((bwd_pre_kernel<D, float>), dim3((unsigned)((rows + 255) / 256)), dim3(256),
                           0, stream, a, (const float*)o, (const float*)dout, lse, ndelta, ws.nlse2,
                           (unsigned long long*)nullptr, (int32_t*)nullptr, (int32_t*)nullptr);
    dim3 grid((unsigned)((a.n + 63) / 64), (unsigned)a.heads, (unsigned)a.batch);
    if (parts & BWD_DQ)
        hipLaunchKernelGGL((bwd_dq_f32_kernel<D>), grid, dim3(64), 0, stream, a, (const float*)q,
                           (const float*)k, (const float*)v, (const float*)dout, lse, ndelta, (float*)dq);
    if (parts & BWD_DKDV)
        hipLaunchKernelGGL((bwd_dkdv_f32_kernel<D>), grid, dim3(64), 0, stream, a, (const float*)q,
                           (const float*)k, (const float*)v, (const float*)dout, lse, ndelta, (float*)dk,
                           (float*)dv);
    return hipGetLastError();
}

}  // namespace

size_t bwd_workspace_bytes(int64_t batch, int64_t heads, int64_t n, int64_t nq, int n_layouts) {
    return (size_t)bwd_workspace_size(batch * heads * n, nq, n_layouts);
}

hipError_t bwd_launch(const AttnArgs& a, int dtype, const void* q, const void* k, const void* v,
                      const void* o, const void* dout, const float* lse, void* dq, void* dk,
                      void* dv, void* workspace, hipStream_t stream, int parts) {
    const BwdWorkspace ws = bwd_workspace(workspace, (int64_t)a.batch * a.heads * a.n, layout_count(a.mode, a.sub));
    if (dtype == 1) {
        switch (a.d) {
        case 32: return bwd_bf16_d32(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream, parts);
        case 64: return bwd_bf16_d64(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream, parts);
        default: return bwd_bf16_d128(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream, parts);
        }
    }
    switch (a.d) {
    case 32: return launch_bwd_f32<32>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream, parts);
    case 64: return launch_bwd_f32<64>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream, parts);
    default: return launch_bwd_f32<128>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream, parts);
    }
}

}  // namespace sa
