// Backward of factorized sparse attention with recomputation (Sec. 5.4): the
// attention weights are rebuilt block by block as P = exp(scale q.k - LSE)
// from the LSE the forward saved, so nothing of size n x n is ever stored.
// For L with dL/dO = dO:
//   D_i  = dO_i . O_i
//   dP   = dO V^T,  dS = P * (dP - D_i)
//   dV   = P^T dO,  dK = scale dS^T Q,  dQ = scale dS K
//
// bf16 path, three launches:
//   1. pre:   D_i into the workspace, and the fp32 dQ accumulator cleared;
//   2. dkdv:  one workgroup per (key block kb, head, batch), B/16 waves of 16
//             keys each, walking the column view of the layout.  dK and dV
//             stay in registers; the block's dQ contribution goes through
//             LDS into fp32 atomics on the accumulator;
//   3. dq:    the accumulator rounded to bf16 into dq.
// fp32 path: the same quantities on the VALU, one thread per row for dq and
// one thread per column for dk / dv, with no atomics.
#include "sa_internal.h"
#include "sa_mfma.h"

namespace sa {

namespace {

// ---------------------------------------------------------------------------
// shared pieces
// ---------------------------------------------------------------------------
struct Workspace {
    float* dq_acc;  // [b, h, n, d]
    float* delta;   // [b, h, n]
};

inline Workspace carve(void* ws, int64_t rows, int64_t d) {
    Workspace w;
    w.dq_acc = static_cast<float*>(ws);
    w.delta = w.dq_acc + rows * d;
    return w;
}

// One thread per row: D_i = sum_t dO[i,t] O[i,t] (fp32), and the dq
// accumulator row cleared.
template <int D, typename T>
__global__ void __launch_bounds__(256)
bwd_pre_kernel(AttnArgs a, const T* __restrict__ o, const T* __restrict__ dout,
               float* __restrict__ delta, float* __restrict__ dq_acc) {
    const int64_t row = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t rows = (int64_t)a.batch * a.heads * a.n;
    if (row >= rows) return;
    const int64_t bh = row / a.n, i = row % a.n;
    const int64_t off = (bh / a.heads) * a.sb + (bh % a.heads) * a.sh + i * a.ss;
    float acc = 0.f;
#pragma unroll 8
    for (int t = 0; t < D; ++t) {
        float x, y;
        if constexpr (sizeof(T) == 2) {
            x = bf16_to_f32(o[off + t]);
            y = bf16_to_f32(dout[off + t]);
        } else {
            x = o[off + t];
            y = dout[off + t];
        }
        acc = fmaf(x, y, acc);
    }
    delta[row] = acc;
    if (dq_acc) {
        float4* dst = reinterpret_cast<float4*>(dq_acc + row * D);
#pragma unroll
        for (int t = 0; t < D / 4; ++t) dst[t] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
}

// ---------------------------------------------------------------------------
// bf16, matrix cores
// ---------------------------------------------------------------------------
template <int D, int BLK>
struct BwdCfg {
    static constexpr int NW = BLK / 16;         // waves; wave w owns keys 16w .. 16w+15
    static constexpr int NT = NW * 64;
    static constexpr int KS = D / 32;           // 32-deep steps over d
    static constexpr int QB = BLK / 16;         // 16-query blocks per tile
    static constexpr int QC = (BLK + 31) / 32;  // 32-query chunks (contraction over queries)
    static constexpr int DB = D / 16;
    static constexpr int RP = D + 8;            // pitch of row-major [BLK][D] tiles
    static constexpr int TP = BLK + 8;          // pitch of transposed [D][BLK] tiles and sdS
};

// Stage rows [row0, row0 + BLK) of a [.., D] bf16 tensor into LDS twice:
// row-major (pitch RP) and transposed (pitch TP).
template <int D, int BLK>
__device__ inline void stage_both(const uint16_t* __restrict__ src, int64_t row0, int64_t ss,
                                  uint16_t* dst, uint16_t* dstT, int tid) {
    using C = BwdCfg<D, BLK>;
    uint32_t* dstT32 = reinterpret_cast<uint32_t*>(dstT);
    for (int u = tid; u < (BLK / 2) * (D / 8); u += C::NT) {
        const int pr = u / (D / 8), col = (u % (D / 8)) * 8;
        u32x4 r0 = *reinterpret_cast<const u32x4*>(src + (row0 + 2 * pr) * ss + col);
        u32x4 r1 = *reinterpret_cast<const u32x4*>(src + (row0 + 2 * pr + 1) * ss + col);
        *reinterpret_cast<u32x4*>(dst + (2 * pr) * C::RP + col) = r0;
        *reinterpret_cast<u32x4*>(dst + (2 * pr + 1) * C::RP + col) = r1;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            uint32_t lo = (r0[e >> 1] >> (16 * (e & 1))) & 0xffffu;
            uint32_t hi = (r1[e >> 1] >> (16 * (e & 1))) & 0xffffu;
            dstT32[((col + e) * C::TP) / 2 + pr] = lo | (hi << 16);
        }
    }
}

// Operand over a 32-query (or 32-key) chunk read from a transposed tile row,
// in the chunk_row() order; zero-padded when the tile has only 16 entries.
template <int BLK>
__device__ inline bf16x8 ld_chunk_T(const uint16_t* row, int chunk, int g) {
    const uint16_t* p = row + chunk * 32 + 4 * g;
    if constexpr (BLK >= 32) {
        return ld_bf16x4x2(p, p + 16);
    } else {
        u32x2 lo = *reinterpret_cast<const u32x2*>(p);
        return __builtin_bit_cast(bf16x8, u32x4{lo.x, lo.y, 0u, 0u});
    }
}

template <int BLK>
__device__ inline bf16x8 pack_chunk(const f32x4* x, int chunk) {
    if constexpr (BLK >= 32) {
        return pack_bf16x8(x[2 * chunk], x[2 * chunk + 1]);
    } else {
        return pack_bf16x8(x[0], zero4());
    }
}

template <int D, int BLK>
__global__ void __launch_bounds__(BLK * 4)
bwd_dkdv_bf16_kernel(AttnArgs a, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                     const uint16_t* __restrict__ v, const uint16_t* __restrict__ dout,
                     const float* __restrict__ lse, const float* __restrict__ delta,
                     float* __restrict__ dq_acc, uint16_t* __restrict__ dk,
                     uint16_t* __restrict__ dv) {
    using C = BwdCfg<D, BLK>;
    __shared__ __attribute__((aligned(16))) uint16_t sQ[BLK * C::RP];
    __shared__ __attribute__((aligned(16))) uint16_t sQt[D * C::TP];
    __shared__ __attribute__((aligned(16))) uint16_t sdO[BLK * C::RP];
    __shared__ __attribute__((aligned(16))) uint16_t sdOt[D * C::TP];
    __shared__ __attribute__((aligned(16))) uint16_t sKt[D * C::TP];
    __shared__ __attribute__((aligned(16))) uint16_t sdS[BLK * C::TP];
    __shared__ float sL[BLK];
    __shared__ float sDelta[BLK];

    const int kb = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, w = tid / 64, lane = tid % 64, g = lane / 16, r = lane % 16;
    const int lay = a.mode == MODE_INTERLEAVED ? (h & 1) : 0;
    const int part = part_of_head(a.mode, h);
    const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;
    const int64_t rowbase = ((int64_t)b * a.heads + h) * a.n;  // LSE / D / dq_acc rows
    const int j = kb * BLK + w * 16 + r;                        // this lane's key

    // K and V rows of this lane's key, as B operands (d in 8g .. 8g+7 of each step)
    bf16x8 kf[C::KS], vf[C::KS];
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
        kf[ks] = ld_bf16x8(k + base + (int64_t)j * a.ss + ks * 32 + 8 * g);
        vf[ks] = ld_bf16x8(v + base + (int64_t)j * a.ss + ks * 32 + 8 * g);
    }
    // K^T of the whole key block for the dQ product
    {
        uint32_t* sKt32 = reinterpret_cast<uint32_t*>(sKt);
        for (int u = tid; u < (BLK / 2) * (D / 8); u += C::NT) {
            const int pr = u / (D / 8), col = (u % (D / 8)) * 8;
            const int64_t r0 = base + (int64_t)(kb * BLK + 2 * pr) * a.ss + col;
            u32x4 x0 = *reinterpret_cast<const u32x4*>(k + r0);
            u32x4 x1 = *reinterpret_cast<const u32x4*>(k + r0 + a.ss);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                uint32_t lo = (x0[e >> 1] >> (16 * (e & 1))) & 0xffffu;
                uint32_t hi = (x1[e >> 1] >> (16 * (e & 1))) & 0xffffu;
                sKt32[((col + e) * C::TP) / 2 + pr] = lo | (hi << 16);
            }
        }
    }

    f32x4 dvacc[C::DB], dkacc[C::DB];
#pragma unroll
    for (int db = 0; db < C::DB; ++db) {
        dvacc[db] = zero4();
        dkacc[db] = zero4();
    }

    const int64_t cp = (int64_t)lay * (a.nq + 1) + kb;
    const int e0 = a.col_ptr[cp], e1 = a.col_ptr[cp + 1];
    for (int e = e0; e < e1; ++e) {
        const int qb = a.row_idx[e];
        const bool masked = a.kind_t[e] != TILE_FULL;
        const int64_t row0 = (int64_t)qb * BLK;
        __syncthreads();  // every wave is done with the previous query block
        stage_both<D, BLK>(q + base, row0, a.ss, sQ, sQt, tid);
        stage_both<D, BLK>(dout + base, row0, a.ss, sdO, sdOt, tid);
        for (int t = tid; t < BLK; t += C::NT) {
            float L = lse[rowbase + row0 + t];
            sL[t] = L * kLog2e;  // -inf stays -inf
            sDelta[t] = delta[rowbase + row0 + t];
        }
        __syncthreads();

        // S and dP for the 16-query blocks: x[qblk][t] is query 16*qblk + 4g + t, key j
        f32x4 p[C::QB], ds[C::QB];
#pragma unroll
        for (int qblk = 0; qblk < C::QB; ++qblk) {
            f32x4 s = zero4(), dp = zero4();
#pragma unroll
            for (int ks = 0; ks < C::KS; ++ks) {
                bf16x8 qa = ld_bf16x8(sQ + (qblk * 16 + r) * C::RP + ks * 32 + 8 * g);
                bf16x8 oa = ld_bf16x8(sdO + (qblk * 16 + r) * C::RP + ks * 32 + 8 * g);
                s = mfma_16x16x32(qa, kf[ks], s);
                dp = mfma_16x16x32(oa, vf[ks], dp);
            }
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int qi = qblk * 16 + 4 * g + t;
                const float L = sL[qi];
                bool on = true;
                if (masked) on = attended(a.pattern, part, a.l, a.c, (int)row0 + qi, j);
                const float pv = on ? exp2_fast(s[t] * a.scale_log2 - L) : 0.f;
                p[qblk][t] = pv;
                ds[qblk][t] = pv * (dp[t] - sDelta[qi]);
            }
        }

        // dV^T += dO^T P and dK^T += Q^T dS, contracting over the block's queries
#pragma unroll
        for (int qc = 0; qc < C::QC; ++qc) {
            bf16x8 pb = pack_chunk<BLK>(p, qc);
            bf16x8 sb = pack_chunk<BLK>(ds, qc);
#pragma unroll
            for (int db = 0; db < C::DB; ++db) {
                bf16x8 oa = ld_chunk_T<BLK>(sdOt + (db * 16 + r) * C::TP, qc, g);
                bf16x8 qa = ld_chunk_T<BLK>(sQt + (db * 16 + r) * C::TP, qc, g);
                dvacc[db] = mfma_16x16x32(oa, pb, dvacc[db]);
                dkacc[db] = mfma_16x16x32(qa, sb, dkacc[db]);
            }
        }

        // dS to LDS as [query][key] for the dQ product
#pragma unroll
        for (int qblk = 0; qblk < C::QB; ++qblk)
#pragma unroll
            for (int t = 0; t < 4; ++t)
                sdS[(qblk * 16 + 4 * g + t) * C::TP + w * 16 + r] = bf16_bits(ds[qblk][t]);
        __syncthreads();

        // dQ rows 16w .. 16w+15 of this query block: dS[q][:] K[:][d]
        f32x4 dqa[C::DB];
#pragma unroll
        for (int db = 0; db < C::DB; ++db) dqa[db] = zero4();
#pragma unroll
        for (int kc = 0; kc < C::QC; ++kc) {
            bf16x8 sa;
            if (BLK >= 32 || g < 2) sa = ld_bf16x8(sdS + (w * 16 + r) * C::TP + kc * 32 + 8 * g);
            else sa = zero_bf16x8();
#pragma unroll
            for (int db = 0; db < C::DB; ++db) {
                bf16x8 kt;
                if (BLK >= 32 || g < 2) kt = ld_bf16x8(sKt + (db * 16 + r) * C::TP + kc * 32 + 8 * g);
                else kt = zero_bf16x8();
                dqa[db] = mfma_16x16x32(sa, kt, dqa[db]);
            }
        }
        float* dst = dq_acc + (rowbase + row0 + w * 16) * D;
#pragma unroll
        for (int db = 0; db < C::DB; ++db)
#pragma unroll
            for (int t = 0; t < 4; ++t)
                atomicAdd(dst + (4 * g + t) * D + db * 16 + r, a.scale * dqa[db][t]);
    }

    // this lane holds dV^T / dK^T at d = 16 db + 4g + t for key j
    uint16_t* dvrow = dv + base + (int64_t)j * a.ss;
    uint16_t* dkrow = dk + base + (int64_t)j * a.ss;
#pragma unroll
    for (int db = 0; db < C::DB; ++db) {
        *reinterpret_cast<uint2*>(dvrow + db * 16 + 4 * g) = pack_bf16x4_bits(dvacc[db]);
        *reinterpret_cast<uint2*>(dkrow + db * 16 + 4 * g) = pack_bf16x4_bits(dkacc[db] * a.scale);
    }
}

template <int D>
__global__ void __launch_bounds__(256)
bwd_dq_convert_kernel(AttnArgs a, const float* __restrict__ dq_acc, uint16_t* __restrict__ dq) {
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;  // one thread per 4 elements
    const int64_t rows = (int64_t)a.batch * a.heads * a.n;
    if (idx >= rows * (D / 4)) return;
    const int64_t row = idx / (D / 4);
    const int c4 = (int)(idx % (D / 4)) * 4;
    const int64_t bh = row / a.n, i = row % a.n;
    const int64_t off = (bh / a.heads) * a.sb + (bh % a.heads) * a.sh + i * a.ss + c4;
    f32x4 x = *reinterpret_cast<const f32x4*>(dq_acc + row * D + c4);
    *reinterpret_cast<uint2*>(dq + off) = pack_bf16x4_bits(x);
}

// ---------------------------------------------------------------------------
// fp32, VALU
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(64)
bwd_dq_f32_kernel(AttnArgs a, const float* __restrict__ q, const float* __restrict__ k,
                  const float* __restrict__ v, const float* __restrict__ dout,
                  const float* __restrict__ lse, const float* __restrict__ delta,
                  float* __restrict__ dq) {
    const int h = blockIdx.y, b = blockIdx.z;
    const int i = blockIdx.x * 64 + threadIdx.x;
    if (i >= a.n) return;
    const int qb = i / a.block;
    const int lay = a.mode == MODE_INTERLEAVED ? (h & 1) : 0;
    const int part = part_of_head(a.mode, h);
    const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;
    const int64_t rowid = ((int64_t)b * a.heads + h) * a.n + i;
    const float L = lse[rowid], Di = delta[rowid];
    const float* qr = q + base + (int64_t)i * a.ss;
    const float* gr = dout + base + (int64_t)i * a.ss;
    float acc[D];
    for (int t = 0; t < D; ++t) acc[t] = 0.f;
    const int64_t rp = (int64_t)lay * (a.nq + 1) + qb;
    for (int e = a.row_ptr[rp]; e < a.row_ptr[rp + 1]; ++e) {
        const int kb = a.col_idx[e];
        const bool full = a.kind[e] == TILE_FULL;
        for (int jj = 0; jj < a.block; ++jj) {
            const int jx = kb * a.block + jj;
            if (!full && !attended(a.pattern, part, a.l, a.c, i, jx)) continue;
            const float* kr = k + base + (int64_t)jx * a.ss;
            const float* vr = v + base + (int64_t)jx * a.ss;
            float s = 0.f, dp = 0.f;
            for (int t = 0; t < D; ++t) {
                s = fmaf(qr[t], kr[t], s);
                dp = fmaf(gr[t], vr[t], dp);
            }
            const float p = expf(s * a.scale - L);
            const float dsv = p * (dp - Di);
            for (int t = 0; t < D; ++t) acc[t] = fmaf(dsv, kr[t], acc[t]);
        }
    }
    for (int t = 0; t < D; ++t) dq[base + (int64_t)i * a.ss + t] = acc[t] * a.scale;
}

template <int D>
__global__ void __launch_bounds__(64)
bwd_dkdv_f32_kernel(AttnArgs a, const float* __restrict__ q, const float* __restrict__ k,
                    const float* __restrict__ v, const float* __restrict__ dout,
                    const float* __restrict__ lse, const float* __restrict__ delta,
                    float* __restrict__ dk, float* __restrict__ dv) {
    const int h = blockIdx.y, b = blockIdx.z;
    const int jx = blockIdx.x * 64 + threadIdx.x;
    if (jx >= a.n) return;
    const int kb = jx / a.block;
    const int lay = a.mode == MODE_INTERLEAVED ? (h & 1) : 0;
    const int part = part_of_head(a.mode, h);
    const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;
    const int64_t rowbase = ((int64_t)b * a.heads + h) * a.n;
    const float* kr = k + base + (int64_t)jx * a.ss;
    const float* vr = v + base + (int64_t)jx * a.ss;
    float ak[D], av[D];
    for (int t = 0; t < D; ++t) ak[t] = av[t] = 0.f;
    const int64_t cp = (int64_t)lay * (a.nq + 1) + kb;
    for (int e = a.col_ptr[cp]; e < a.col_ptr[cp + 1]; ++e) {
        const int qb = a.row_idx[e];
        const bool full = a.kind_t[e] == TILE_FULL;
        for (int ii = 0; ii < a.block; ++ii) {
            const int i = qb * a.block + ii;
            if (!full && !attended(a.pattern, part, a.l, a.c, i, jx)) continue;
            const float* qr = q + base + (int64_t)i * a.ss;
            const float* gr = dout + base + (int64_t)i * a.ss;
            float s = 0.f, dp = 0.f;
            for (int t = 0; t < D; ++t) {
                s = fmaf(qr[t], kr[t], s);
                dp = fmaf(gr[t], vr[t], dp);
            }
            const float p = expf(s * a.scale - lse[rowbase + i]);
            const float dsv = p * (dp - delta[rowbase + i]);
            for (int t = 0; t < D; ++t) {
                av[t] = fmaf(p, gr[t], av[t]);
                ak[t] = fmaf(dsv, qr[t], ak[t]);
            }
        }
    }
    for (int t = 0; t < D; ++t) {
        dk[base + (int64_t)jx * a.ss + t] = ak[t] * a.scale;
        dv[base + (int64_t)jx * a.ss + t] = av[t];
    }
}

template <int D>
hipError_t launch_bwd_f32(const AttnArgs& a, const void* q, const void* k, const void* v,
                          const void* o, const void* dout, const float* lse, void* dq, void* dk,
                          void* dv, Workspace ws, hipStream_t stream) {
    const int64_t rows = (int64_t)a.batch * a.heads * a.n;
    hipLaunchKernelGGL((bwd_pre_kernel<D, float>), dim3((unsigned)((rows + 255) / 256)), dim3(256),
                       0, stream, a, (const float*)o, (const float*)dout, ws.delta, (float*)nullptr);
    dim3 grid((unsigned)((a.n + 63) / 64), (unsigned)a.heads, (unsigned)a.batch);
    hipLaunchKernelGGL((bwd_dq_f32_kernel<D>), grid, dim3(64), 0, stream, a, (const float*)q,
                       (const float*)k, (const float*)v, (const float*)dout, lse, ws.delta,
                       (float*)dq);
    hipLaunchKernelGGL((bwd_dkdv_f32_kernel<D>), grid, dim3(64), 0, stream, a, (const float*)q,
                       (const float*)k, (const float*)v, (const float*)dout, lse, ws.delta,
                       (float*)dk, (float*)dv);
    return hipGetLastError();
}

template <int D, int BLK>
hipError_t launch_bwd_bf16(const AttnArgs& a, const void* q, const void* k, const void* v,
                           const void* o, const void* dout, const float* lse, void* dq, void* dk,
                           void* dv, Workspace ws, hipStream_t stream) {
    const int64_t rows = (int64_t)a.batch * a.heads * a.n;
    hipLaunchKernelGGL((bwd_pre_kernel<D, uint16_t>), dim3((unsigned)((rows + 255) / 256)),
                       dim3(256), 0, stream, a, (const uint16_t*)o, (const uint16_t*)dout, ws.delta,
                       ws.dq_acc);
    dim3 grid((unsigned)a.nq, (unsigned)a.heads, (unsigned)a.batch);
    hipLaunchKernelGGL((bwd_dkdv_bf16_kernel<D, BLK>), grid, dim3(BwdCfg<D, BLK>::NT), 0, stream,
                       a, (const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)v,
                       (const uint16_t*)dout, lse, ws.delta, ws.dq_acc, (uint16_t*)dk,
                       (uint16_t*)dv);
    const int64_t quads = rows * (D / 4);
    hipLaunchKernelGGL((bwd_dq_convert_kernel<D>), dim3((unsigned)((quads + 255) / 256)), dim3(256),
                       0, stream, a, ws.dq_acc, (uint16_t*)dq);
    return hipGetLastError();
}

template <int D>
hipError_t launch_bwd_bf16_d(const AttnArgs& a, const void* q, const void* k, const void* v,
                             const void* o, const void* dout, const float* lse, void* dq,
                             void* dk, void* dv, Workspace ws, hipStream_t stream) {
    switch (a.block) {
    case 16: return launch_bwd_bf16<D, 16>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream);
    case 32: return launch_bwd_bf16<D, 32>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream);
    default: return launch_bwd_bf16<D, 64>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream);
    }
}

}  // namespace

size_t bwd_workspace_bytes(int64_t batch, int64_t heads, int64_t n, int64_t d, int dtype) {
    const int64_t rows = batch * heads * n;
    const int64_t acc = dtype == 1 ? rows * d : 0;  // fp32 dq accumulator (bf16 path only)
    return (size_t)((acc + rows) * (int64_t)sizeof(float));
}

hipError_t bwd_launch(const AttnArgs& a, int dtype, const void* q, const void* k, const void* v,
                      const void* o, const void* dout, const float* lse, void* dq, void* dk,
                      void* dv, void* workspace, hipStream_t stream) {
    const int64_t rows = (int64_t)a.batch * a.heads * a.n;
    if (dtype == 1) {
        Workspace ws = carve(workspace, rows, a.d);
        switch (a.d) {
        case 32: return launch_bwd_bf16_d<32>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream);
        case 64: return launch_bwd_bf16_d<64>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream);
        default: return launch_bwd_bf16_d<128>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream);
        }
    }
    Workspace ws = carve(workspace, rows, 0);
    switch (a.d) {
    case 32: return launch_bwd_f32<32>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream);
    case 64: return launch_bwd_f32<64>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream);
    default: return launch_bwd_f32<128>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream);
    }
}

}  // namespace sa
