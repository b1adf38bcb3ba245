// Forward of factorized sparse attention (Sec. 4.2 eq. attend_fn over the
// sets of Sec. 4.3), block by block over the layout (Sec. 5.5), with the
// softmax fused into the same kernel and kept in registers.  The kernel keeps
// one running maximum and sum per row (online softmax) and saves
// LSE = log(sum_j exp(s_ij)) for the recomputing backward (Sec. 5.4).
//
// bf16 path: one workgroup per (query block qb, head, batch), waves of 32
// query rows (one wave of 16 rows for B = 16).  Per present key block kb:
//   S^T = K_kb Q^T        (MFMA 16x16x32, K from LDS, Q fragment in VGPRs)
//   mask (MASKED blocks), running max over the row, P = exp2(S - m)
//   O^T += V_kb^T P^T     (MFMA; P^T is fed from the S^T results directly)
// Each lane owns one query row (r = lane % 16), so the row statistics are
// per lane plus a two-step exchange over the four lane groups.
//
// fp32 path: one thread per query row, same online softmax on the VALU.
#include "sa_internal.h"
#include "sa_mask.h"
#include "sa_mfma.h"
#include "sa_tile.h"

namespace sa {

namespace {

// ---------------------------------------------------------------------------
// bf16, matrix cores
// ---------------------------------------------------------------------------
// Waves of 16 query rows: with four waves per 64-wide block the workgroup holds
// more waves per SIMD (fewer registers each), and in the strided pattern a
// block that holds one diagonal leaves each 16-row wave a single live chunk.
template <int D, int BLK, int PAT>
struct FwdCfg {
    // query rows per wave.  (32 rows per wave in the fixed pattern, each K / V
    // operand read feeding two row blocks at two waves per SIMD, made the
    // forward at n = 65,536 slower: 0.83 against 0.77 ms.)
    static constexpr int RW = 16;
    static constexpr int QBW = RW / 16;             // 16-row blocks per wave
    static constexpr int NW = BLK / RW;             // waves per workgroup
    static constexpr int NT = NW * 64;              // threads
    static constexpr int KS = D / 32;               // 32-deep steps over d for S
    static constexpr int KB = BLK / 16;             // 16-key blocks per tile
    static constexpr int KC = (BLK + 31) / 32;      // 32-key chunks for P V
    static constexpr int DB = D / 16;               // 16-wide d blocks of O
    static constexpr int NS = 2;                    // K / V ring stages
    static constexpr int WAVES_PER_EU = RW == 32 ? 2 : 3;
};

// grid: (heads, nq, batch).  Consecutive workgroups (dispatched round-robin
// over the XCDs) share a query block index across heads, so with heads a
// multiple of 8 each head stays on one XCD and its keys stay in that L2; a
// dense walk takes a head's query blocks together instead (row_grid_item).
template <int D, int BLK, int PAT, int MODE, bool FULL_BODY>
__global__ void __launch_bounds__((FwdCfg<D, BLK, PAT>::NT)) __attribute__((amdgpu_waves_per_eu(FwdCfg<D, BLK, PAT>::WAVES_PER_EU)))
fwd_bf16_kernel(AttnArgs a, const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ col_idx,
                const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                const uint16_t* __restrict__ v, uint16_t* __restrict__ o, float* __restrict__ lse) {
    using C = FwdCfg<D, BLK, PAT>;
    // K and V tiles in a two-stage ring: the next key block is in flight
    // while one is computed; one barrier per key block
    __shared__ __attribute__((aligned(16))) uint16_t sK[C::NS][BLK * D];
    __shared__ __attribute__((aligned(16))) uint16_t sV[C::NS][BLK * D];
    constexpr uint32_t kTileBytes = BLK * D * 2;
    constexpr uint64_t kTileBits = BLK == 64 ? ~0ull : (1ull << BLK) - 1;
    const uint32_t sK_base = lds_addr(&sK[0][0]), sV_base = lds_addr(&sV[0][0]);

    const GridItem gi = row_grid_item(a);  // longest rows first
    const int h = __builtin_amdgcn_readfirstlane(gi.h), qb = __builtin_amdgcn_readfirstlane(gi.qb),
              b = __builtin_amdgcn_readfirstlane(gi.b);
    const int tid = threadIdx.x, lane = tid % 64, g = lane / 16, r = lane % 16;
    const int w = __builtin_amdgcn_readfirstlane(tid / 64);
    const int lay = head_layout(a, h);
    const MaskParams mp = head_mask_params(a, PAT, MODE, h);
    const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;
    const int row0 = qb * BLK + w * C::RW;  // first query row of this wave
    const int qs0 = qb * BLK - a.qshift;    // first query row of the block as the masks see it

    bf16x8 qf[C::QBW][C::KS];
    f32x4 oacc[C::QBW][C::DB];
    float m_run[C::QBW], l_run[C::QBW];
    RowLane rl[C::QBW];
#pragma unroll
    for (int u = 0; u < C::QBW; ++u) {
#pragma unroll
        for (int ks = 0; ks < C::KS; ++ks)
            qf[u][ks] = ld_bf16x8(q + base + (int64_t)(row0 + 16 * u + r) * a.ss + ks * 32 + 8 * g);
#pragma unroll
        for (int db = 0; db < C::DB; ++db) oacc[u][db] = zero4();
        m_run[u] = -INFINITY;
        l_run[u] = 0.f;
        rl[u] = row_lane(row0 + 16 * u + r - a.qshift, a.dl);
    }

    int e0 = 0, e1 = qb + 1;  // WALK_DENSE: key blocks 0 .. qb
    if (a.walk != WALK_DENSE) {
        const int64_t rp = (int64_t)lay * (a.nq + 1) + qb;
        e0 = __builtin_amdgcn_readfirstlane(row_ptr[rp]);
        e1 = __builtin_amdgcn_readfirstlane(row_ptr[rp + 1]);
        if (a.walk == WALK_BAND) e0 = max(e0, e1 - (a.l / BLK + 1));
    }
    TileLoader<D, BLK, C::NW> ld;
    ld.init(a.ss, w, lane);
    // A step stages one block, or two summary halves (see RowStepper) as one tile
    constexpr bool kPairs = PAT == FIXED && BLK == 64;
    auto load_step = [&](RowStep s, int stage) {
        const uint32_t kdst = sK_base + stage * kTileBytes, vdst = sV_base + stage * kTileBytes;
        if (!kPairs || s.b < 0) {
            const int64_t kbase = base + (int64_t)s.a * BLK * a.ss;
            ld.issue(k + kbase, kdst);
            ld.issue(v + kbase, vdst);
        } else if constexpr (kPairs) {
            // the summary halves: upper (window at 32 mod 64) or lower (at 0 mod
            // 64); issue_halves takes tile rows 0..31 from lo and 32..63 from hi
            const int half_off = (mp.w & 63) == 0 ? 0 : BLK / 2;
            const int64_t lo = base + ((int64_t)s.a * BLK + half_off) * a.ss;
            const int64_t hi = base + ((int64_t)s.b * BLK - (BLK / 2 - half_off)) * a.ss;
            ld.issue_halves(k + lo, k + hi, kdst);
            ld.issue_halves(v + lo, v + hi, vdst);
        }
    };

    // The register loads above complete before the ring starts, so no
    // compiler-tracked load is outstanding inside the loop (a wait for one
    // would also drain the ring).
    wait_loads_upto<0>();
    const float c2 = a.scale_log2;
    // two-stage ring; the next step's blocks are read one step ahead (scalar
    // loads, off the vector-memory counter the ring waits on)
    RowStepper<kPairs> steps{col_idx, e0, e1, RowStepper<kPairs>::pair_bound(mp, a.dl, qb * BLK),
                             a.walk == WALK_DENSE};
    // strided blocks away from the band are single diagonals (see the step)
    const bool diag_far = PAT == STRIDED && mp.part != PART_A1 && a.l % BLK == 0;
    RowStep cur = steps.next();
    if (cur.a >= 0) load_step(cur, 0);
    TileReader<D> rd;
    rd.init(g, r);
    two_stage_while([&](auto stage) {
        constexpr int st = decltype(stage)::value;  // ring stage of the current step
        if (cur.a < 0) return false;
        const RowStep nxt = steps.next();
        const int kb = cur.a;
        const int j0 = kb * BLK;
        // a pair of summary halves is attended everywhere
        const bool masked =
            cur.b < 0 && !block_full32(PAT, mp.part, a.dl, a.c, mp.w, qs0, qs0 + BLK - 1, j0, j0 + BLK - 1);
        wait_loads_upto<0>();
        __syncthreads();  // this step is in LDS everywhere; the other stage is free
        if (nxt.a >= 0) load_step(nxt, st ^ 1);
        const uint16_t* tK = sK[st];
        const uint16_t* tV = sV[st];
        if constexpr (PAT == STRIDED) {
            // A strided block away from the band, with l a multiple of B, holds
            // exactly its main diagonal (row i0 + t attends key j0 + t): each row
            // gains one score, so the online softmax takes a rank-1 step in
            // registers, q . k and O += p v, instead of a masked chunk of
            // products.
            if (diag_far && far_block(PAT, a.dl, qs0, j0, BLK)) {
#pragma unroll
                for (int u = 0; u < C::QBW; ++u) {
                    const int kk = w * C::RW + 16 * u + r;  // this lane's row, and its key, in the block
                    float part = 0.f;
#pragma unroll
                    for (int ks = 0; ks < C::KS; ++ks)
                        part += dot_bf16x8(qf[u][ks], ld_bf16x8(tK + Swz<D>::off(kk, 32 * ks + 8 * g)));
                    bf16x4 vv[C::DB];  // read now, used after the softmax update
#pragma unroll
                    for (int db = 0; db < C::DB; ++db)
                        vv[db] = __builtin_bit_cast(bf16x4, *reinterpret_cast<const uint2*>(tV + Swz<D>::off(kk, 16 * db + 4 * g)));
                    const float sc = sum_over_g(part);
                    const bool grew = sc > m_run[u];
                    const float m_new = grew ? sc : m_run[u];
                    const float alpha = exp2_fast((m_run[u] - m_new) * c2);  // 0 while m was -inf
                    const float pr = exp2_fast((sc - m_new) * c2);
                    l_run[u] = fmaf(l_run[u], alpha, g == 0 ? pr : 0.f);  // one lane of the row counts p
                    m_run[u] = m_new;
                    // O is rescaled only where some row's maximum grew (a wave-uniform branch)
                    if (__builtin_amdgcn_ballot_w64(grew) != 0ull) {
#pragma unroll
                        for (int db = 0; db < C::DB; ++db) oacc[u][db] *= alpha;
                    }
#pragma unroll
                    for (int db = 0; db < C::DB; ++db)
#pragma unroll
                        for (int t = 0; t < 4; ++t) oacc[u][db][t] = fmaf(pr, (float)vv[db][t], oacc[u][db][t]);
                }
                cur = nxt;
                return true;
            }
        }
        // With FULL_BODY the step body exists twice: for blocks attended
        // everywhere (every chunk class a compile-time ALL, no mask and no
        // branch on classes) and for the others (see with_full_body).
        auto compute = [&](auto full) {
            // mask bits of this lane's rows (bit 16 kb16 + t after the shift), and
            // the treatment of each 32-key chunk
            uint64_t bits[C::QBW];
            int cls[C::QBW][C::KC];
#pragma unroll
            for (int u = 0; u < C::QBW; ++u) {
                bits[u] = ~0ull;
#pragma unroll
                for (int kc = 0; kc < C::KC; ++kc) cls[u][kc] = CHUNK_ALL;
            }
            if constexpr (!decltype(full)::value) {
                const int j0_mod = mod_l(a.dl, j0);
                const uint64_t sum = PAT == FIXED ? summary_bits(mp, j0_mod) : 0ull;
                const bool far = far_block(PAT, a.dl, qs0, j0, BLK);
                if (PAT == FIXED && far && mp.part != PART_A1) {
                    // every row attends exactly the summary keys: one mask for the wave
                    const uint64_t sb = sum & kTileBits;
#pragma unroll
                    for (int u = 0; u < C::QBW; ++u) {
                        bits[u] = sb >> (4 * g);
#pragma unroll
                        for (int kc = 0; kc < C::KC; ++kc) cls[u][kc] = uniform_chunk_class(sb, kc, C::KB >= 2);
                    }
                } else {
                    if (far) {
#pragma unroll
                        for (int u = 0; u < C::QBW; ++u) bits[u] = (row_mask_far(mp, rl[u], j0_mod, sum) & kTileBits) >> (4 * g);
                    } else {
#pragma unroll
                        for (int u = 0; u < C::QBW; ++u) bits[u] = (row_mask(mp, rl[u], j0, j0_mod, sum) & kTileBits) >> (4 * g);
                    }
#pragma unroll
                    for (int u = 0; u < C::QBW; ++u)
#pragma unroll
                        for (int kc = 0; kc < C::KC; ++kc)
                            cls[u][kc] = chunk_class(chunk_bits(bits[u], kc, C::KB >= 2), C::KB >= 2);
                }
            }

            // A 32-key chunk enters the products only where some row of the wave
            // attends one of its keys; elsewhere its probabilities are zero and
            // its operands are neither read nor multiplied (wave-uniform branches)
            constexpr int HK = C::KB >= 2 ? 2 : 1;  // 16-key blocks per 32-key chunk
            bool kc_live[C::KC];
#pragma unroll
            for (int kc = 0; kc < C::KC; ++kc) {
                kc_live[kc] = false;
#pragma unroll
                for (int u = 0; u < C::QBW; ++u) kc_live[kc] = kc_live[kc] || cls[u][kc] != CHUNK_NONE;
            }
            // V^T operands of this block, read now: their LDS latency then hides
            // behind the S products and the softmax
            bf16x8 vt[C::KC][C::DB];
#pragma unroll
            for (int kc = 0; kc < C::KC; ++kc) {
                if (!kc_live[kc]) continue;
#pragma unroll
                for (int db = 0; db < C::DB; ++db) {
                    if constexpr (BLK >= 32) vt[kc][db] = rd.tr(tV, kc * 32, kc * 32 + 16, db);
                    else vt[kc][db] = rd.tr_half(tV, 0, db);
                }
            }

            // S^T blocks: s[u][kb16][t] = q_(row0+16u+r) . k_(j0 + 16 kb16 + 4g + t).
            // The wave's priority is raised while it issues them, so that the
            // matrix cores get the products early while the other waves of the
            // SIMD run their softmax (0.5-1% on the forward; raised around the
            // PV products too it was slower).
            __builtin_amdgcn_s_setprio(1);
            f32x4 s[C::QBW][C::KB];
#pragma unroll
            for (int kblk = 0; kblk < C::KB; ++kblk) {
                const int kc = kblk / HK;
#pragma unroll
                for (int u = 0; u < C::QBW; ++u) s[u][kblk] = zero4();
                if (!kc_live[kc]) continue;
                bf16x8 kf[C::KS];
#pragma unroll
                for (int ks = 0; ks < C::KS; ++ks) kf[ks] = rd.row(tK, kblk * 16, ks);
#pragma unroll
                for (int u = 0; u < C::QBW; ++u) {
                    if (cls[u][kc] == CHUNK_NONE) continue;
#pragma unroll
                    for (int ks = 0; ks < C::KS; ++ks) s[u][kblk] = mfma_16x16x32(kf[ks], qf[u][ks], s[u][kblk]);
                }
            }

            __builtin_amdgcn_s_setprio(0);
            bf16x8 pf[C::QBW][C::KC];
#pragma unroll
            for (int u = 0; u < C::QBW; ++u) {
                // running max in raw score units (the scale is positive) over the
                // chunks that hold attended keys; masked items become -inf
                float mloc = -INFINITY;
#pragma unroll
                for (int kc = 0; kc < C::KC; ++kc) {
                    if (cls[u][kc] == CHUNK_NONE) continue;
                    if (cls[u][kc] == CHUNK_PART) {
#pragma unroll
                        for (int hk = 0; hk < HK; ++hk)
#pragma unroll
                            for (int t = 0; t < 4; ++t)
                                s[u][2 * kc + hk][t] =
                                    select_or_neg_inf(bit_lane_mask(bits[u], 16 * (2 * kc + hk) + t), s[u][2 * kc + hk][t]);
                    }
#pragma unroll
                    for (int hk = 0; hk < HK; ++hk) {
                        // a chain of three-way maxima: two instructions per four scores
                        const f32x4 x = s[u][2 * kc + hk];
                        mloc = fmaxf(fmaxf(mloc, x[0]), x[1]);
                        mloc = fmaxf(fmaxf(mloc, x[2]), x[3]);
                    }
                }
                mloc = max_over_g(mloc);
                // The reference is the exact running maximum, so the largest
                // probability of a row is exactly 1 in bf16 as in fp32.
                const bool grew = mloc > m_run[u];
                const float m_new = grew ? mloc : m_run[u];
                // rows with nothing attended so far keep m = -inf; 0 as reference
                // gives p = 0 without a branch around the MFMAs
                const float m_ref = m_new == -INFINITY ? 0.f : m_new;
                const float neg = -m_ref * c2;
                float psum = 0.f;
#pragma unroll
                for (int kc = 0; kc < C::KC; ++kc) {
                    if (cls[u][kc] != CHUNK_NONE) {
#pragma unroll
                        for (int hk = 0; hk < HK; ++hk) {
#pragma unroll
                            for (int t = 0; t < 4; ++t) {
                                const float pv = exp2_fast(fmaf(s[u][2 * kc + hk][t], c2, neg));
                                s[u][2 * kc + hk][t] = pv;
                                psum += pv;
                            }
                        }
                    } else {
#pragma unroll
                        for (int hk = 0; hk < HK; ++hk) s[u][2 * kc + hk] = zero4();
                    }
                    if constexpr (BLK >= 32) pf[u][kc] = pack_bf16x8(s[u][2 * kc], s[u][2 * kc + 1]);
                    else pf[u][kc] = pack_bf16x8(s[u][0], zero4());
                }
                // alpha rescales the state kept for the old maximum (0 when it was -inf)
                const float alpha = exp2_fast((m_run[u] - m_ref) * c2);
                l_run[u] = fmaf(l_run[u], alpha, psum);
                m_run[u] = m_new;
                // O is rescaled on every step: where no row's maximum grew alpha
                // is exactly 1 and O keeps its bits.  (Behind a branch on the
                // growth the compiler kept O in other registers on the two sides
                // and copied it back every step, which cost more than the
                // multiplies: n = 1,048,576 forward 2.94 -> 2.90 ms.)
#pragma unroll
                for (int db = 0; db < C::DB; ++db) oacc[u][db] *= alpha;
            }

            // O^T += V^T P^T
#pragma unroll
            for (int kc = 0; kc < C::KC; ++kc) {
#pragma unroll
                for (int u = 0; u < C::QBW; ++u) {
                    if (cls[u][kc] == CHUNK_NONE) continue;
#pragma unroll
                    for (int db = 0; db < C::DB; ++db) oacc[u][db] = mfma_16x16x32(vt[kc][db], pf[u][kc], oacc[u][db]);
                }
            }
        };
        if (masked || !FULL_BODY) compute(std::false_type{});
        else compute(std::true_type{});
        cur = nxt;
        return true;
    });

#pragma unroll
    for (int u = 0; u < C::QBW; ++u) {
        const int i = row0 + 16 * u + r;
        const float l_tot = sum_over_g(l_run[u]);
        uint16_t* orow = o + base + (int64_t)i * a.ss;
        float* lrow = lse + stat_index(a, b, h, i);
        if (a.epilogue == EPI_MERGE) {
            // O and LSE of another, disjoint part of the row's set are already
            // there: with weights exp(LSE_part - LSE) the union's softmax is
            // O = (w1 O1 + exp(m scale - mx) acc) / z, LSE = mx + log z
            const float lse1 = *lrow;
            const float lse2 = l_tot > 0.f ? m_run[u] * a.scale + __logf(l_tot) : -INFINITY;
            const float mx = fmaxf(lse1, lse2);
            const float w1 = lse1 == -INFINITY ? 0.f : __expf(lse1 - mx);
            const float w2 = l_tot > 0.f ? __expf(m_run[u] * a.scale - mx) : 0.f;  // weight of acc
            const float z = w1 + w2 * l_tot;
            const float inv = z > 0.f ? 1.f / z : 0.f;
#pragma unroll
            for (int db = 0; db < C::DB; ++db) {
                uint2* dst = reinterpret_cast<uint2*>(orow + db * 16 + 4 * g);
                const bf16x4 o1 = __builtin_bit_cast(bf16x4, *dst);
                f32x4 x;
#pragma unroll
                for (int t = 0; t < 4; ++t) x[t] = (w1 * (float)o1[t] + w2 * oacc[u][db][t]) * inv;
                *dst = pack_bf16x4_bits(x);
            }
            if (g == 0) *lrow = z > 0.f ? mx + __logf(z) : -INFINITY;
            continue;
        }
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
#pragma unroll
        for (int db = 0; db < C::DB; ++db)
            *reinterpret_cast<uint2*>(orow + db * 16 + 4 * g) = pack_bf16x4_bits(oacc[u][db] * inv);
        if (g == 0) *lrow = l_tot > 0.f ? m_run[u] * a.scale + __logf(l_tot) : -INFINITY;
    }
}

// ---------------------------------------------------------------------------
// fp32, VALU: one thread per query row
// ---------------------------------------------------------------------------
// The blocks of row qb a walk visits (see WALK_*), as entries e0 .. e1 of the
// layout (WALK_DENSE: e is the key block itself).
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

template <int D>
__global__ void __launch_bounds__(64)
fwd_f32_kernel(AttnArgs a, const float* __restrict__ q, const float* __restrict__ k,
               const float* __restrict__ v, float* __restrict__ o, float* __restrict__ lse) {
    const int h = blockIdx.y, b = blockIdx.z;
    const int i = blockIdx.x * 64 + threadIdx.x;
    if (i >= a.n) return;
    const int qb = i / a.block;
    const int lay = head_layout(a, h);
    const int part = part_of_head(a.mode, h);
    const int32_t wst = window_start(a, subblock_of_head(a.sub, h));
    const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;

    float qr[D], acc[D];
    for (int t = 0; t < D; ++t) {
        qr[t] = q[base + (int64_t)i * a.ss + t];
        acc[t] = 0.f;
    }
    float m = -INFINITY, l = 0.f;
    int e0, e1;
    row_entries(a, lay, qb, &e0, &e1);
    for (int e = e0; e < e1; ++e) {
        const int kb = a.walk == WALK_DENSE ? e : a.col_idx[e];
        const bool full = a.walk != WALK_DENSE && a.kind[e] == TILE_FULL;
        for (int jj = 0; jj < a.block; ++jj) {
            const int j = kb * a.block + jj;
            if (!full && !attended(a.pattern, part, a.l, a.c, wst, i - a.qshift, j)) continue;
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
    float* orow = o + base + (int64_t)i * a.ss;
    float* lrow = lse + stat_index(a, b, h, i);
    if (a.epilogue == EPI_MERGE) {
        // combine with the O and LSE of the disjoint part already there
        const float lse1 = *lrow, lse2 = l > 0.f ? m + logf(l) : -INFINITY;
        const float mx = fmaxf(lse1, lse2);
        const float w1 = lse1 == -INFINITY ? 0.f : expf(lse1 - mx);
        const float w2 = l > 0.f ? expf(m - mx) : 0.f;  // weight of acc
        const float z = w1 + w2 * l;
        const float inv = z > 0.f ? 1.f / z : 0.f;
        for (int t = 0; t < D; ++t) orow[t] = (w1 * orow[t] + w2 * acc[t]) * inv;
        *lrow = z > 0.f ? mx + logf(z) : -INFINITY;
        return;
    }
    float inv = l > 0.f ? 1.f / l : 0.f;
    for (int t = 0; t < D; ++t) orow[t] = acc[t] * inv;
    *lrow = l > 0.f ? m + logf(l) : -INFINITY;
}

template <int D, int BLK>
hipError_t launch_bf16(const AttnArgs& a, const void* q, const void* k, const void* v, void* o,
                       float* lse, hipStream_t stream) {
    dim3 grid((unsigned)a.heads, (unsigned)a.nq, (unsigned)a.batch);
    return with_pattern_mode(a.pattern, a.mode, [&](auto pat, auto mode) {
        constexpr int PAT = decltype(pat)::value, MODE = decltype(mode)::value;
        return with_full_body<PAT>(a, [&](auto fb) {
            hipLaunchKernelGGL((fwd_bf16_kernel<D, BLK, PAT, MODE, decltype(fb)::value>), grid,
                               dim3(FwdCfg<D, BLK, PAT>::NT), 0, stream, a, a.row_ptr, a.col_idx, (const uint16_t*)q,
                               (const uint16_t*)k, (const uint16_t*)v, (uint16_t*)o, lse);
            return hipGetLastError();
        });
    });
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
