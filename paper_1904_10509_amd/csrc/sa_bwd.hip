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
#include "sa_mask.h"
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
    static constexpr int KW = BLK < 32 ? BLK : 32;  // keys per wave
    static constexpr int KBW = KW / 16;             // 16-key blocks per wave
    static constexpr int NW = BLK / KW;             // waves
    static constexpr int NT = NW * 64;
    static constexpr int KS = D / 32;               // 32-deep steps over d
    static constexpr int QB = BLK / 16;             // 16-query blocks per tile
    static constexpr int QC = (BLK + 31) / 32;      // 32-query chunks (contraction over queries)
    static constexpr int DB = D / 16;
    static constexpr int P = D + 8;                 // pitch of row-major [BLK][D] tiles
    static constexpr int SP = BLK + 8;              // pitch of dS [query][key]
    static constexpr int CH = BLK * D / 8;          // 16-byte chunks per Q (or dO) tile
    static constexpr int CPT = (CH + NT - 1) / NT;
    static constexpr int QRW = BLK / NW;            // dQ rows per wave
    static constexpr int QBQ = QRW / 16;            // their 16-row blocks
};

template <int D, int BLK>
__global__ void __launch_bounds__(BLK < 32 ? 64 : 2 * BLK)
bwd_dkdv_bf16_kernel(AttnArgs a, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                     const uint16_t* __restrict__ v, const uint16_t* __restrict__ dout,
                     const float* __restrict__ lse, const float* __restrict__ delta,
                     float* __restrict__ dq_acc, uint16_t* __restrict__ dk,
                     uint16_t* __restrict__ dv) {
    using C = BwdCfg<D, BLK>;
    __shared__ __attribute__((aligned(16))) uint16_t sQ[2][BLK * C::P];
    __shared__ __attribute__((aligned(16))) uint16_t sdO[2][BLK * C::P];
    __shared__ __attribute__((aligned(16))) uint16_t sK[BLK * C::P];
    __shared__ __attribute__((aligned(16))) uint16_t sdS[BLK * C::SP];
    __shared__ __attribute__((aligned(16))) float sL[2][BLK];
    __shared__ __attribute__((aligned(16))) float sDl[2][BLK];

    const int kb = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, w = tid / 64, lane = tid % 64, g = lane / 16, r = lane % 16;
    const int lay = a.mode == MODE_INTERLEAVED ? (h & 1) : 0;
    MaskParams mp{a.pattern, part_of_head(a.mode, h), a.l, a.c, a.period_bits};
    const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;
    const int64_t rowbase = ((int64_t)b * a.heads + h) * a.n;  // LSE / D / dq_acc rows
    const int key0 = kb * BLK + w * C::KW;                      // first key of this wave

    // this lane's keys j = key0 + 16 kbw + r as B operands (d = 32 ks + 8g + t)
    bf16x8 kf[C::KBW][C::KS], vf[C::KBW][C::KS];
    bool summary[C::KBW];
#pragma unroll
    for (int kbw = 0; kbw < C::KBW; ++kbw) {
        const int j = key0 + 16 * kbw + r;
#pragma unroll
        for (int ks = 0; ks < C::KS; ++ks) {
            kf[kbw][ks] = ld_bf16x8(k + base + (int64_t)j * a.ss + ks * 32 + 8 * g);
            vf[kbw][ks] = ld_bf16x8(v + base + (int64_t)j * a.ss + ks * 32 + 8 * g);
        }
        summary[kbw] = a.pattern == FIXED && (j % a.l) >= a.l - a.c;
    }
    // the key block row-major, for the transposed operand of dQ = dS K
    for (int ch = tid; ch < C::CH; ch += C::NT) {
        const int row = ch / (D / 8), col = (ch % (D / 8)) * 8;
        *reinterpret_cast<u32x4*>(&sK[row * C::P + col]) =
            *reinterpret_cast<const u32x4*>(k + base + (int64_t)(kb * BLK + row) * a.ss + col);
    }

    f32x4 dvacc[C::KBW][C::DB], dkacc[C::KBW][C::DB];
#pragma unroll
    for (int kbw = 0; kbw < C::KBW; ++kbw)
#pragma unroll
        for (int db = 0; db < C::DB; ++db) {
            dvacc[kbw][db] = zero4();
            dkacc[kbw][db] = zero4();
        }

    const int64_t cp = (int64_t)lay * (a.nq + 1) + kb;
    const int e0 = a.col_ptr[cp], e1 = a.col_ptr[cp + 1];
    const int len = e1 - e0;
    // Start each column at its own offset so that the workgroups running at
    // the same time add into different dQ rows.
    const int rot = len > 0 ? (int)(((int64_t)kb * 37 + h * 11) % len) : 0;
    auto entry = [&](int s) { int x = s + rot; return e0 + (x >= len ? x - len : x); };

    u32x4 qreg[C::CPT], oreg[C::CPT];
    float lreg = 0.f, dreg = 0.f;
    auto load_block = [&](int qb) {
        const int64_t qbase = base + (int64_t)qb * BLK * a.ss;
#pragma unroll
        for (int t = 0; t < C::CPT; ++t) {
            const int ch = tid + t * C::NT;
            if (C::CH % C::NT == 0 || ch < C::CH) {
                const int row = ch / (D / 8), col = (ch % (D / 8)) * 8;
                qreg[t] = *reinterpret_cast<const u32x4*>(q + qbase + (int64_t)row * a.ss + col);
                oreg[t] = *reinterpret_cast<const u32x4*>(dout + qbase + (int64_t)row * a.ss + col);
            }
        }
        if (tid < BLK) {
            lreg = lse[rowbase + (int64_t)qb * BLK + tid];
            dreg = delta[rowbase + (int64_t)qb * BLK + tid];
        }
    };
    auto store_block = [&](int buf) {
#pragma unroll
        for (int t = 0; t < C::CPT; ++t) {
            const int ch = tid + t * C::NT;
            if (C::CH % C::NT == 0 || ch < C::CH) {
                const int row = ch / (D / 8), col = (ch % (D / 8)) * 8;
                *reinterpret_cast<u32x4*>(&sQ[buf][row * C::P + col]) = qreg[t];
                *reinterpret_cast<u32x4*>(&sdO[buf][row * C::P + col]) = oreg[t];
            }
        }
        if (tid < BLK) {
            sL[buf][tid] = lreg * kLog2e;  // -inf stays -inf
            sDl[buf][tid] = dreg;
        }
    };

    if (len > 0) {
        load_block(a.row_idx[entry(0)]);
        store_block(0);
    }
    __syncthreads();
    const float c2 = a.scale_log2;
    for (int st = 0; st < len; ++st) {
        const int buf = st & 1;
        const int e = entry(st);
        const int qb = a.row_idx[e];
        const bool masked = a.kind_t[e] != TILE_FULL;
        const int i0 = qb * BLK;
        if (st + 1 < len) load_block(a.row_idx[entry(st + 1)]);
        const uint16_t* tQ = sQ[buf];
        const uint16_t* tO = sdO[buf];

        // S and dP: x[kbw][qblk][t] is query i0 + 16 qblk + 4g + t against key key0 + 16 kbw + r
        f32x4 p[C::KBW][C::QB], ds[C::KBW][C::QB];
#pragma unroll
        for (int qblk = 0; qblk < C::QB; ++qblk) {
            bf16x8 qa[C::KS], oa[C::KS];
#pragma unroll
            for (int ks = 0; ks < C::KS; ++ks) {
                qa[ks] = ld_bf16x8(tQ + (qblk * 16 + r) * C::P + ks * 32 + 8 * g);
                oa[ks] = ld_bf16x8(tO + (qblk * 16 + r) * C::P + ks * 32 + 8 * g);
            }
#pragma unroll
            for (int kbw = 0; kbw < C::KBW; ++kbw) {
                f32x4 sacc = zero4(), dpacc = zero4();
#pragma unroll
                for (int ks = 0; ks < C::KS; ++ks) {
                    sacc = mfma_16x16x32(qa[ks], kf[kbw][ks], sacc);
                    dpacc = mfma_16x16x32(oa[ks], vf[kbw][ks], dpacc);
                }
                p[kbw][qblk] = sacc;
                ds[kbw][qblk] = dpacc;
            }
        }
#pragma unroll
        for (int kbw = 0; kbw < C::KBW; ++kbw) {
            uint64_t bits = ~0ull;
            if (masked) bits = col_mask(mp, key0 + 16 * kbw + r, i0, summary[kbw]) >> (4 * g);
#pragma unroll
            for (int qblk = 0; qblk < C::QB; ++qblk) {
                const f32x4 L = *reinterpret_cast<const f32x4*>(&sL[buf][qblk * 16 + 4 * g]);
                const f32x4 Dl = *reinterpret_cast<const f32x4*>(&sDl[buf][qblk * 16 + 4 * g]);
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const bool on = (bits >> (16 * qblk + t)) & 1ull;
                    const float pv = on ? exp2_fast(fmaf(p[kbw][qblk][t], c2, -L[t])) : 0.f;
                    p[kbw][qblk][t] = pv;
                    ds[kbw][qblk][t] = pv * (ds[kbw][qblk][t] - Dl[t]);
                }
            }
        }

        // dV^T += dO^T P and dK^T += Q^T dS, contracting over the block's queries;
        // dO^T and Q^T are read transposed from the row-major tiles
#pragma unroll
        for (int qc = 0; qc < C::QC; ++qc) {
#pragma unroll
            for (int db = 0; db < C::DB; ++db) {
                bf16x8 oT, qT;
                if constexpr (BLK >= 32) {
                    oT = ld_tr_operand(tO, C::P, qc * 32 + 4 * g, qc * 32 + 16 + 4 * g, db * 16, r);
                    qT = ld_tr_operand(tQ, C::P, qc * 32 + 4 * g, qc * 32 + 16 + 4 * g, db * 16, r);
                } else {
                    u32x2 lo = ld_tr16(tO + (4 * g + (r >> 2)) * C::P + db * 16 + 4 * (r & 3));
                    u32x2 lq = ld_tr16(tQ + (4 * g + (r >> 2)) * C::P + db * 16 + 4 * (r & 3));
                    oT = __builtin_bit_cast(bf16x8, u32x4{lo.x, lo.y, 0u, 0u});
                    qT = __builtin_bit_cast(bf16x8, u32x4{lq.x, lq.y, 0u, 0u});
                }
#pragma unroll
                for (int kbw = 0; kbw < C::KBW; ++kbw) {
                    bf16x8 pb, sb;
                    if constexpr (BLK >= 32) {
                        pb = pack_bf16x8(p[kbw][2 * qc], p[kbw][2 * qc + 1]);
                        sb = pack_bf16x8(ds[kbw][2 * qc], ds[kbw][2 * qc + 1]);
                    } else {
                        pb = pack_bf16x8(p[kbw][0], zero4());
                        sb = pack_bf16x8(ds[kbw][0], zero4());
                    }
                    dvacc[kbw][db] = mfma_16x16x32(oT, pb, dvacc[kbw][db]);
                    dkacc[kbw][db] = mfma_16x16x32(qT, sb, dkacc[kbw][db]);
                }
            }
        }

        // dS to LDS as [query][key] for the dQ product
#pragma unroll
        for (int kbw = 0; kbw < C::KBW; ++kbw)
#pragma unroll
            for (int qblk = 0; qblk < C::QB; ++qblk)
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    sdS[(qblk * 16 + 4 * g + t) * C::SP + w * C::KW + 16 * kbw + r] = bf16_bits(ds[kbw][qblk][t]);
        __syncthreads();

        // dQ rows w*QRW .. of this query block: dS[q][:] K[:][d], K read transposed
        f32x4 dqa[C::QBQ][C::DB];
#pragma unroll
        for (int u = 0; u < C::QBQ; ++u)
#pragma unroll
            for (int db = 0; db < C::DB; ++db) dqa[u][db] = zero4();
        // With 16-key blocks only lane groups g < 2 carry keys; the others
        // read in-bounds rows and are zeroed by a data mask afterwards: the
        // transposing LDS read is always issued with every lane active.
        const int gk = (BLK >= 32) ? g : (g & 1);
        const uint32_t keep = (BLK >= 32 || g < 2) ? 0xffffffffu : 0u;
#pragma unroll
        for (int kc = 0; kc < C::QC; ++kc) {
            bf16x8 sa[C::QBQ];
#pragma unroll
            for (int u = 0; u < C::QBQ; ++u)
                sa[u] = mask_bf16x8(ld_bf16x8(sdS + (w * C::QRW + 16 * u + r) * C::SP + kc * 32 + 8 * gk), keep);
#pragma unroll
            for (int db = 0; db < C::DB; ++db) {
                const bf16x8 kt =
                    mask_bf16x8(ld_tr_operand(sK, C::P, kc * 32 + 8 * gk, kc * 32 + 8 * gk + 4, db * 16, r), keep);
#pragma unroll
                for (int u = 0; u < C::QBQ; ++u) dqa[u][db] = mfma_16x16x32(sa[u], kt, dqa[u][db]);
            }
        }
#pragma unroll
        for (int u = 0; u < C::QBQ; ++u) {
            float* dst = dq_acc + (rowbase + i0 + w * C::QRW + 16 * u) * D;
#pragma unroll
            for (int db = 0; db < C::DB; ++db)
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    atomicAdd(dst + (4 * g + t) * D + db * 16 + r, a.scale * dqa[u][db][t]);
        }

        if (st + 1 < len) store_block(buf ^ 1);
        __syncthreads();
    }

    // this lane holds dV^T / dK^T at d = 16 db + 4g + t for key key0 + 16 kbw + r
#pragma unroll
    for (int kbw = 0; kbw < C::KBW; ++kbw) {
        const int j = key0 + 16 * kbw + r;
        uint16_t* dvrow = dv + base + (int64_t)j * a.ss;
        uint16_t* dkrow = dk + base + (int64_t)j * a.ss;
#pragma unroll
        for (int db = 0; db < C::DB; ++db) {
            *reinterpret_cast<uint2*>(dvrow + db * 16 + 4 * g) = pack_bf16x4_bits(dvacc[kbw][db]);
            *reinterpret_cast<uint2*>(dkrow + db * 16 + 4 * g) = pack_bf16x4_bits(dkacc[kbw][db] * a.scale);
        }
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
