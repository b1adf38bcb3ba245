// Forward of factorized sparse attention (Sec. 4.2 eq. attend_fn over the
// sets of Sec. 4.3), block by block over the layout (Sec. 5.5), with the
// softmax fused into the same kernel and kept in registers.  The kernel keeps
// one running maximum and sum per row (online softmax) and saves
// LSE = log(sum_j exp(s_ij)) for the recomputing backward (Sec. 5.4).
//
// bf16 path: one workgroup per (query block qb, head, batch), B/16 waves of
// 16 query rows each.  Per present key block kb:
//   S^T = K_kb Q^T        (MFMA 16x16x32, K from LDS, Q fragment in VGPRs)
//   mask (MASKED blocks), running max over the row, P = exp2(S - m)
//   O^T += V_kb^T P^T     (MFMA; P^T is fed from the S^T results directly)
// Each lane owns one query row (r = lane % 16), so the row statistics are
// per lane plus a two-step exchange over the four lane groups.
//
// fp32 path: one thread per query row, same online softmax on the VALU.
#include "sa_internal.h"
#include "sa_mfma.h"

namespace sa {

namespace {

// ---------------------------------------------------------------------------
// bf16, matrix cores
// ---------------------------------------------------------------------------
template <int D, int BLK>
struct FwdCfg {
    static constexpr int NW = BLK / 16;          // waves per workgroup
    static constexpr int NT = NW * 64;           // threads
    static constexpr int KS = D / 32;            // 32-deep steps over d for S
    static constexpr int KB = BLK / 16;          // 16-key blocks per tile
    static constexpr int KC = (BLK + 31) / 32;   // 32-key chunks for P V
    static constexpr int DB = D / 16;            // 16-wide d blocks of O
    static constexpr int KP = D + 8;             // sK row pitch (elements)
    static constexpr int VP = BLK + 8;           // sVt row pitch (elements)
    static constexpr int KCH = (BLK * D / 8 + NT - 1) / NT;        // 16-byte K chunks per thread
    static constexpr int VU = ((BLK / 2) * (D / 8) + NT - 1) / NT;  // V (pair, chunk) units per thread
};

template <int D, int BLK>
__global__ void __launch_bounds__(BLK * 4)
fwd_bf16_kernel(AttnArgs a, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                const uint16_t* __restrict__ v, uint16_t* __restrict__ o, float* __restrict__ lse) {
    using C = FwdCfg<D, BLK>;
    __shared__ __attribute__((aligned(16))) uint16_t sK[BLK * C::KP];
    __shared__ __attribute__((aligned(16))) uint16_t sVt[D * C::VP];

    const int qb = a.nq - 1 - (int)blockIdx.x;  // longest rows first
    const int h = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, w = tid / 64, lane = tid % 64, g = lane / 16, r = lane % 16;
    const int lay = a.mode == MODE_INTERLEAVED ? (h & 1) : 0;
    const int part = part_of_head(a.mode, h);
    const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;
    const int i = qb * BLK + w * 16 + r;  // this lane's query row

    bf16x8 qf[C::KS];
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) qf[ks] = ld_bf16x8(q + base + (int64_t)i * a.ss + ks * 32 + 8 * g);

    f32x4 oacc[C::DB];
#pragma unroll
    for (int db = 0; db < C::DB; ++db) oacc[db] = zero4();
    float m_run = -INFINITY, l_run = 0.f;

    const int64_t rp = (int64_t)lay * (a.nq + 1) + qb;
    const int e0 = a.row_ptr[rp], e1 = a.row_ptr[rp + 1];

    // register staging of the next K / V block
    u32x4 kreg[C::KCH];
    u32x4 vreg[C::VU][2];
    auto load_block = [&](int kb) {
        const int64_t kbase = base + (int64_t)kb * BLK * a.ss;
#pragma unroll
        for (int t = 0; t < C::KCH; ++t) {
            int ch = tid + t * C::NT;
            if (ch < BLK * D / 8) {
                int row = ch / (D / 8), col = (ch % (D / 8)) * 8;
                kreg[t] = *reinterpret_cast<const u32x4*>(k + kbase + (int64_t)row * a.ss + col);
            }
        }
#pragma unroll
        for (int t = 0; t < C::VU; ++t) {
            int u = tid + t * C::NT;
            if (u < (BLK / 2) * (D / 8)) {
                int pr = u / (D / 8), col = (u % (D / 8)) * 8;
                vreg[t][0] = *reinterpret_cast<const u32x4*>(v + kbase + (int64_t)(2 * pr) * a.ss + col);
                vreg[t][1] = *reinterpret_cast<const u32x4*>(v + kbase + (int64_t)(2 * pr + 1) * a.ss + col);
            }
        }
    };
    auto store_block = [&]() {
#pragma unroll
        for (int t = 0; t < C::KCH; ++t) {
            int ch = tid + t * C::NT;
            if (ch < BLK * D / 8) {
                int row = ch / (D / 8), col = (ch % (D / 8)) * 8;
                *reinterpret_cast<u32x4*>(sK + row * C::KP + col) = kreg[t];
            }
        }
        uint32_t* sVt32 = reinterpret_cast<uint32_t*>(sVt);
#pragma unroll
        for (int t = 0; t < C::VU; ++t) {
            int u = tid + t * C::NT;
            if (u < (BLK / 2) * (D / 8)) {
                int pr = u / (D / 8), col = (u % (D / 8)) * 8;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    uint32_t lo = (vreg[t][0][e >> 1] >> (16 * (e & 1))) & 0xffffu;
                    uint32_t hi = (vreg[t][1][e >> 1] >> (16 * (e & 1))) & 0xffffu;
                    sVt32[((col + e) * C::VP) / 2 + pr] = lo | (hi << 16);
                }
            }
        }
    };

    if (e0 < e1) load_block(a.col_idx[e0]);
    for (int e = e0; e < e1; ++e) {
        const int kb = a.col_idx[e];
        const bool masked = a.kind[e] != TILE_FULL;
        __syncthreads();  // previous block's LDS reads are done
        store_block();
        __syncthreads();
        if (e + 1 < e1) load_block(a.col_idx[e + 1]);

        // S^T blocks: s[kblk][t] = score of key kb*BLK + 16*kblk + 4g + t against row i
        f32x4 s[C::KB];
#pragma unroll
        for (int kblk = 0; kblk < C::KB; ++kblk) {
            s[kblk] = zero4();
#pragma unroll
            for (int ks = 0; ks < C::KS; ++ks) {
                bf16x8 kf = ld_bf16x8(sK + (kblk * 16 + r) * C::KP + ks * 32 + 8 * g);
                s[kblk] = mfma_16x16x32(kf, qf[ks], s[kblk]);
            }
        }
        float mloc = -INFINITY;
#pragma unroll
        for (int kblk = 0; kblk < C::KB; ++kblk) {
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                float x = s[kblk][t] * a.scale_log2;
                if (masked) {
                    int j = kb * BLK + kblk * 16 + 4 * g + t;
                    if (!attended(a.pattern, part, a.l, a.c, i, j)) x = -INFINITY;
                }
                s[kblk][t] = x;
                mloc = fmaxf(mloc, x);
            }
        }
        mloc = max_over_g(mloc);
        const float m_new = fmaxf(m_run, mloc);
        // A row with nothing attended so far keeps m = -inf; using 0 as its
        // reference gives p = 0 and alpha = 0 without any branch around the MFMAs.
        const float m_ref = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = exp2_fast(m_run - m_ref);
        m_run = m_new;
        float psum = 0.f;
#pragma unroll
        for (int kblk = 0; kblk < C::KB; ++kblk) {
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                float p = exp2_fast(s[kblk][t] - m_ref);
                s[kblk][t] = p;
                psum += p;
            }
        }
        l_run = l_run * alpha + psum;
#pragma unroll
        for (int db = 0; db < C::DB; ++db) oacc[db] *= alpha;

#pragma unroll
        for (int kc = 0; kc < C::KC; ++kc) {
            bf16x8 pf;
            if constexpr (BLK >= 32) pf = pack_bf16x8(s[2 * kc], s[2 * kc + 1]);
            else pf = pack_bf16x8(s[0], zero4());
#pragma unroll
            for (int db = 0; db < C::DB; ++db) {
                const uint16_t* row = sVt + (db * 16 + r) * C::VP + kc * 32 + 4 * g;
                bf16x8 vf;
                if constexpr (BLK >= 32) {
                    vf = ld_bf16x4x2(row, row + 16);
                } else {
                    u32x2 lo = *reinterpret_cast<const u32x2*>(row);
                    vf = __builtin_bit_cast(bf16x8, u32x4{lo.x, lo.y, 0u, 0u});
                }
                oacc[db] = mfma_16x16x32(vf, pf, oacc[db]);
            }
        }
    }

    const float l_tot = sum_over_g(l_run);
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    uint16_t* orow = o + base + (int64_t)i * a.ss;
#pragma unroll
    for (int db = 0; db < C::DB; ++db) {
        uint2 bits = pack_bf16x4_bits(oacc[db] * inv);
        *reinterpret_cast<uint2*>(orow + db * 16 + 4 * g) = bits;
    }
    if (g == 0) {
        float val = l_tot > 0.f ? (m_run + __log2f(l_tot)) * kLn2 : -INFINITY;
        lse[((int64_t)b * a.heads + h) * a.n + i] = val;
    }
}

// ---------------------------------------------------------------------------
// fp32, VALU: one thread per query row
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(64)
fwd_f32_kernel(AttnArgs a, const float* __restrict__ q, const float* __restrict__ k,
               const float* __restrict__ v, float* __restrict__ o, float* __restrict__ lse) {
    const int h = blockIdx.y, b = blockIdx.z;
    const int i = blockIdx.x * 64 + threadIdx.x;
    if (i >= a.n) return;
    const int qb = i / a.block;
    const int lay = a.mode == MODE_INTERLEAVED ? (h & 1) : 0;
    const int part = part_of_head(a.mode, h);
    const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;

    float qr[D], acc[D];
    for (int t = 0; t < D; ++t) {
        qr[t] = q[base + (int64_t)i * a.ss + t];
        acc[t] = 0.f;
    }
    float m = -INFINITY, l = 0.f;
    const int64_t rp = (int64_t)lay * (a.nq + 1) + qb;
    for (int e = a.row_ptr[rp]; e < a.row_ptr[rp + 1]; ++e) {
        const int kb = a.col_idx[e];
        const bool full = a.kind[e] == TILE_FULL;
        for (int jj = 0; jj < a.block; ++jj) {
            const int j = kb * a.block + jj;
            if (!full && !attended(a.pattern, part, a.l, a.c, i, j)) continue;
            const float* kr = k + base + (int64_t)j * a.ss;
            float s = 0.f;
            for (int t = 0; t < D; ++t) s = fmaf(qr[t], kr[t], s);
            s *= a.scale;
            if (s > m) {
                float alpha = expf(m - s);
                l *= alpha;
                for (int t = 0; t < D; ++t) acc[t] *= alpha;
                m = s;
            }
            float p = expf(s - m);
            l += p;
            const float* vr = v + base + (int64_t)j * a.ss;
            for (int t = 0; t < D; ++t) acc[t] = fmaf(p, vr[t], acc[t]);
        }
    }
    float inv = l > 0.f ? 1.f / l : 0.f;
    for (int t = 0; t < D; ++t) o[base + (int64_t)i * a.ss + t] = acc[t] * inv;
    lse[((int64_t)b * a.heads + h) * a.n + i] = l > 0.f ? m + logf(l) : -INFINITY;
}

template <int D, int BLK>
hipError_t launch_bf16(const AttnArgs& a, const void* q, const void* k, const void* v, void* o,
                       float* lse, hipStream_t stream) {
    dim3 grid((unsigned)a.nq, (unsigned)a.heads, (unsigned)a.batch);
    hipLaunchKernelGGL((fwd_bf16_kernel<D, BLK>), grid, dim3(FwdCfg<D, BLK>::NT), 0, stream, a,
                       (const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)v, (uint16_t*)o, lse);
    return hipGetLastError();
}

template <int D>
hipError_t launch_bf16_d(const AttnArgs& a, const void* q, const void* k, const void* v, void* o,
                         float* lse, hipStream_t stream) {
    switch (a.block) {
    case 16: return launch_bf16<D, 16>(a, q, k, v, o, lse, stream);
    case 32: return launch_bf16<D, 32>(a, q, k, v, o, lse, stream);
    default: return launch_bf16<D, 64>(a, q, k, v, o, lse, stream);
    }
}

template <int D>
hipError_t launch_f32(const AttnArgs& a, const void* q, const void* k, const void* v, void* o,
                      float* lse, hipStream_t stream) {
    dim3 grid((unsigned)((a.n + 63) / 64), (unsigned)a.heads, (unsigned)a.batch);
    hipLaunchKernelGGL((fwd_f32_kernel<D>), grid, dim3(64), 0, stream, a, (const float*)q,
                       (const float*)k, (const float*)v, (float*)o, lse);
    return hipGetLastError();
}

}  // namespace

hipError_t fwd_launch(const AttnArgs& a, int dtype, const void* q, const void* k, const void* v,
                      void* o, float* lse, hipStream_t stream) {
    if (dtype == 1) {
        switch (a.d) {
        case 32: return launch_bf16_d<32>(a, q, k, v, o, lse, stream);
        case 64: return launch_bf16_d<64>(a, q, k, v, o, lse, stream);
        default: return launch_bf16_d<128>(a, q, k, v, o, lse, stream);
        }
    }
    switch (a.d) {
    case 32: return launch_f32<32>(a, q, k, v, o, lse, stream);
    case 64: return launch_f32<64>(a, q, k, v, o, lse, stream);
    default: return launch_f32<128>(a, q, k, v, o, lse, stream);
    }
}

}  // namespace sa
