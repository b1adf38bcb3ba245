// Backward of factorized sparse attention with recomputation (Sec. 5.4): the
// attention weights are rebuilt block by block as P = exp(scale q.k - LSE)
// from the LSE the forward saved, so nothing of size n x n is ever stored.
// For L with dL/dO = dO:
//   D_i  = dO_i . O_i
//   dP   = dO V^T,  dS = P * (dP - D_i)
//   dV   = P^T dO,  dK = scale dS^T Q,  dQ = scale dS K
//
// bf16 path, three launches, no atomics (every output element has exactly
// one writer, so results are reproducible bit for bit):
//   1. pre:   D_i into the workspace;
//   2. dq:    one workgroup per (head, query block, batch) walks the row view
//             of the layout like the forward: S^T and dP^T recomputed, dS^T
//             formed in registers and contracted with K into dQ;
//   3. dkdv:  a workgroup takes one (key block, batch, head) column at a
//             time from a queue and walks its column view: S and dP
//             recomputed, dV += P^T dO and dK += dS^T Q held in registers for
//             the whole column.
// In the fixed pattern with B = 64 a key block that is half summary keys is
// split into its two halves, and summary halves one l-block apart are walked
// as pairs (see split_column, pair_partner).
// Column lengths can vary with a short period (in the fixed pattern only the
// key blocks holding summary columns are long), and a hardware placement of
// one workgroup per column can then pile the long columns onto a few compute
// units.  The dkdv grid is therefore sized to the resident capacity of the
// device, the pre kernel sorts the key blocks of each layout by column length
// (longest first, so the long columns of a head start together and walk the
// same Q / dO tiles at about the same time), and each workgroup takes its
// columns in one of three orders chosen per call:
//   - serpentine per head (fixed pattern, a few workgroups per head): one
//     head per workgroup, ranks j, 2J - 1 - j, 2J + j, ... over the head's J
//     workgroups, which evens out the sums of the sorted lengths;
//   - round-robin over the rank-major order (strided pattern, short columns);
//   - atomic counters, one queue per XCD holding the heads bh = x (mod 8),
//     with stealing once a queue is dry (the remaining cases).
// The first two use no atomics: claims on one counter are serialised across
// the device and, with short columns, take longer than the columns.
// The dq kernel repeats the S and dP products of the dkdv kernel; those two
// extra products per block are the price of having no reduction across
// workgroups.
// fp32 path: the same quantities on the VALU, one thread per row for dq and
// one thread per column for dk / dv.
#pragma once

#include <atomic>
#include <type_traits>

#include "sa_internal.h"
#include "sa_mask.h"
#include "sa_mfma.h"
#include "sa_tile.h"

namespace sa {

// Workspace: -D [rows] and -LSE log2 e [rows] (fp32), then (16-byte aligned)
// the kQueues queue counters (uint64), the item count of each layout
// (int32), and the item order of each layout (2 nq int32 slots).
struct BwdWorkspace {
    float* ndelta;  // -D
    float* nlse2;   // -LSE log2 e
    unsigned long long* queue;
    int32_t* items;
    int32_t* order;
};

// bf16 backward of one head size (one translation unit each, sa_bwd_bf16_d*.hip).
hipError_t bwd_bf16_d32(const AttnArgs& a, const void* q, const void* k, const void* v, const void* o,
                        const void* dout, const float* lse, void* dq, void* dk, void* dv, const BwdWorkspace& ws,
                        hipStream_t stream, int parts);
hipError_t bwd_bf16_d64(const AttnArgs& a, const void* q, const void* k, const void* v, const void* o,
                        const void* dout, const float* lse, void* dq, void* dk, void* dv, const BwdWorkspace& ws,
                        hipStream_t stream, int parts);
hipError_t bwd_bf16_d128(const AttnArgs& a, const void* q, const void* k, const void* v, const void* o,
                         const void* dout, const float* lse, void* dq, void* dk, void* dv, const BwdWorkspace& ws,
                         hipStream_t stream, int parts);

namespace {

// ---------------------------------------------------------------------------
// shared pieces
// ---------------------------------------------------------------------------
// One thread per row: -D_i = -sum_t dO[i,t] O[i,t] (fp32), and the saved LSE
// in base-2 units, negated (-LSE * log2 e), for the exp2 recomputation of P.
// Both are stored negated because the kernels add them: -D_i is where the
// dP accumulation starts, and P = exp2(scale log2 e * s - LSE log2 e) is one
// fused multiply-add.
// Schedule of the dK / dV kernel.
constexpr int kQueues = 8;          // one per XCD
constexpr int kLengthClasses = 128;  // four per octave of column length

// Length class of a column of `len` blocks; longer columns get lower classes.
__device__ inline int length_class(int len) {
    if (len <= 0) return kLengthClasses - 1;
    const int lg = 31 - __builtin_clz((unsigned)len);
    const int frac = lg >= 2 ? (len >> (lg - 2)) & 3 : (len << (2 - lg)) & 3;
    return kLengthClasses - 2 - (4 * lg + frac);
}

// Queue x holds the (batch, head) pairs bh = x (mod kQueues).
__device__ inline int64_t queue_heads(int64_t bh_count, int x) {
    return bh_count > x ? (bh_count - 1 - x) / kQueues + 1 : 0;
}

// Items of the dK / dV schedule: key block kb whole (kind 0), one 32-key
// half of a 64-wide block (kind 1: keys 0..31, kind 2: keys 32..63), a
// pair of such halves (kind 3: keys 0..31, kind 4: keys 32..63, of kb and of
// kb + l / 64), or the short columns of the l-block that starts at kb
// (kind 5, kGroupKind below); -1 is an empty slot.  kb < 2^27 (n < 2^31,
// B >= 16).
constexpr int kItemShift = 28;
__device__ inline int32_t item_code(int kb, int kind) { return kb | (kind << kItemShift); }

// In the fixed pattern with B = 64, a key block half of whose keys (the
// upper or the lower 32) are summary keys and the other half not is split
// into its two halves: the other keys meet only the blocks of their own
// l-block, the summary keys every block of the column.  Each half is then
// shared by all four waves (its two 16-key groups times the two 32-query
// halves of a block), where the whole block would leave the two waves of the
// other keys idle on every block away from the diagonal.  Returns 0 (no
// split), 1 (upper keys are the summary keys) or 2 (lower keys are).
__device__ inline int split_column(const AttnArgs& a, int g, int kb) {
    if (a.pattern != FIXED || a.block != 64) return 0;
    const MaskParams mp = mask_params(a, a.pattern, part_of_layout(a.mode, g), subblock_of_layout(a.mode, a.sub, g));
    if (mp.part == PART_A1) return 0;
    const uint64_t bits = summary_bits(mp, mod_l(a.dl, 64 * kb));
    return bits == 0xFFFFFFFF00000000ull ? 1 : (bits == 0x00000000FFFFFFFFull ? 2 : 0);
}

// When l is a multiple of 64 the summary halves of split blocks recur every
// l / 64 blocks at the same place, and two of them, one l-block apart, can be
// walked as one item (a.pairs, chosen by the launcher): a split block of an
// even l-block takes the summary half of the block l / 64 further along.  The
// column of the first holds the second's (summary keys meet every later
// query), and each staged Q / dO tile then serves 64 keys, where a single
// half uses it for 32.  Returns the partner block of split block kb's summary
// half, kb when that half is walked alone, or -1 when it is the second half
// of kb - l / 64's pair.
__device__ inline int pair_partner(const AttnArgs& a, int kb) {
    if (!a.pairs || a.l % 64 != 0) return kb;
    const int step = a.l / 64;
    if ((kb / step) & 1) return -1;
    return kb + step < a.nq ? kb + step : kb;
}

// In the fixed pattern with B = 64 and l a multiple of 128, the short
// columns of one l-block (whole blocks attended only inside it, and the
// other-key halves of split blocks) form one item, kind kGroupKind, coded by
// the l-block's first key block: one workgroup walks them one after the
// other, so the l-block's Q / dO tiles are fetched once and then hit in L2
// (as separate items they ran on different workgroups at different times
// and were fetched again).  Returns the key blocks per l-block, or 0 where
// columns are not grouped.
constexpr int kGroupKind = 5;
__device__ inline int group_blocks(const AttnArgs& a) {
    return a.pattern == FIXED && a.block == 64 && a.l % 128 == 0 ? a.l / 64 : 0;
}
// The item kind key block kb takes inside its l-block's group (0: the whole
// block, 1 / 2: its lower / upper 32 keys), or -1 when it has no short
// column (its column is walked as an item of its own).  cp: layout g's
// column pointers.
__device__ inline int group_member(const AttnArgs& a, int g, int kb, const int32_t* cp) {
    const int split = split_column(a, g, kb);
    if (split) return split;  // the other half of a split block is short
    return cp[kb + 1] - cp[kb] <= group_blocks(a) ? 0 : -1;
}

// Workgroup g < n_layouts of the row-statistics step (the pre kernel, or
// the dQ kernel where it computes the statistics): layout g's items (2 nq
// slots) ordered by length class, empty slots last, and its item count in
// items[g].  Inside a class the items follow their key blocks (and a block's
// items the order below), the same on every run: in the serpentine orders
// an item's place decides which round walks its column and so the
// direction, and with it the rounding of dK and dV.  Workgroup 0 also
// empties the queues.
__device__ void build_schedule(const AttnArgs& a, int g, unsigned long long* queue, int32_t* items_out,
                               int32_t* order) {
    __shared__ int cls_pos[kLengthClasses];
    __shared__ int items;
    const int tid = threadIdx.x;
    if (g == 0 && tid < kQueues) queue[tid] = 0ull;
    // Columns no longer than an l-block (the local columns, and the halves of
    // non-summary keys) share one class: inside a class items sit in about
    // the order of their key blocks, so the local columns of one l-block stay
    // adjacent, run at about the same time on neighbouring workgroups and
    // share that l-block's Q / dO tiles in L2 (in length classes of their own,
    // 1 .. l/B blocks long, they ran far apart and each re-read them).
    const int short_len = a.l / a.block > 2 ? a.l / a.block : 2;
    const int lower_cls = length_class(short_len);
    auto cls_of = [&](int len) { return len <= short_len ? lower_cls : length_class(len); };
    const int32_t* cp = a.col_ptr + (int64_t)g * (a.nq + 1);
    int32_t* ord = order + (int64_t)g * 2 * a.nq;
    for (int i = tid; i < kLengthClasses; i += blockDim.x) cls_pos[i] = 0;
    __syncthreads();
    const int G = group_blocks(a);
    // a group's class follows the sum of its members' walks (a split block's
    // short half walks at most the l-block's blocks)
    auto group_len = [&](int kb0) {
        int total = 0;
        for (int kb = kb0; kb < kb0 + G && kb < a.nq; ++kb)
            if (group_member(a, g, kb, cp) >= 0) total += min(cp[kb + 1] - cp[kb], G);
        return total;
    };
    // (the counting pass takes the same decisions as the placing pass below)
    for (int kb = tid; kb < a.nq; kb += blockDim.x) {
        const int split = split_column(a, g, kb), partner = split ? pair_partner(a, kb) : kb;
        const bool member = G && group_member(a, g, kb, cp) >= 0;
        if (split == 0) {
            if (!member) atomicAdd(&cls_pos[cls_of(cp[kb + 1] - cp[kb])], 1);
        } else if (partner >= 0) {
            atomicAdd(&cls_pos[cls_of(cp[kb + 1] - cp[kb])], 1);
        }
        if (!G && split) atomicAdd(&cls_pos[lower_cls], 1);
        if (G && kb % G == 0) {
            const int total = group_len(kb);
            if (total > 0) atomicAdd(&cls_pos[cls_of(total)], 1);
        }
    }
    __syncthreads();
    if (tid == 0) {
        int run = 0;
        for (int i = 0; i < kLengthClasses; ++i) {
            const int c = cls_pos[i];
            cls_pos[i] = run;
            run += c;
        }
        items = run;
    }
    __syncthreads();
    // Placing pass, by wave 0 alone: 64 key blocks at a time, in order, each
    // lane holding block kb's up to three items (code, class; class -1: none).
    // The items of one class in the chunk go to consecutive places ranked by
    // (lane, item), a stable counting sort.
    if (tid < 64) {
        const int lane = tid;
        const uint64_t below = lane == 0 ? 0ull : ~0ull >> (64 - lane);
        for (int kb0 = 0; kb0 < a.nq; kb0 += 64) {
            const int kb = kb0 + lane;
            int32_t code[3] = {-1, -1, -1};
            int cls[3] = {-1, -1, -1};
            if (kb < a.nq) {
                const int split = split_column(a, g, kb);
                // the summary half (alone or with its partner) takes the
                // column's class, the other half the short one (or its
                // l-block's group)
                const int sum_half = split == 1 ? 2 : 1, partner = split ? pair_partner(a, kb) : kb;
                const bool member = G && group_member(a, g, kb, cp) >= 0;
                if (split == 0) {
                    if (!member) {
                        code[0] = item_code(kb, 0);
                        cls[0] = cls_of(cp[kb + 1] - cp[kb]);
                    }
                } else if (partner >= 0) {
                    code[0] = item_code(kb, partner == kb ? sum_half : sum_half + 2);
                    cls[0] = cls_of(cp[kb + 1] - cp[kb]);
                }
                if (!G && split) {
                    code[1] = item_code(kb, 3 - sum_half);
                    cls[1] = lower_cls;
                }
                if (G && kb % G == 0) {
                    const int total = group_len(kb);
                    if (total > 0) {
                        code[2] = item_code(kb, kGroupKind);
                        cls[2] = cls_of(total);
                    }
                }
            }
            uint64_t left[3];
#pragma unroll
            for (int i = 0; i < 3; ++i) left[i] = __ballot(cls[i] >= 0);
            while (left[0] | left[1] | left[2]) {
                // the next class: that of the first lane still holding an item
                const int i0 = left[0] ? 0 : (left[1] ? 1 : 2);
                const int c0 = i0 == 0 ? cls[0] : (i0 == 1 ? cls[1] : cls[2]);
                const int c = __builtin_amdgcn_readlane(c0, __builtin_ctzll(left[i0]));
                uint64_t m[3];
                int before = 0, count = 0;
#pragma unroll
                for (int i = 0; i < 3; ++i) {
                    m[i] = __ballot(cls[i] == c);
                    before += __popcll(m[i] & below);
                    count += __popcll(m[i]);
                    left[i] &= ~m[i];
                }
                const int base = cls_pos[c];
                int pos = base + before;
#pragma unroll
                for (int i = 0; i < 3; ++i)
                    if (cls[i] == c) ord[pos++] = code[i];
                if (lane == 0) cls_pos[c] = base + count;
            }
        }
    }
    for (int i = items + tid; i < 2 * a.nq; i += blockDim.x) ord[i] = -1;
    if (tid == 0) items_out[g] = items;
}

// Rows of the row-statistics kernel per 256-thread workgroup: one thread per
// row in fp32; in bf16 four lanes per row, lane g reading the 16-byte chunks
// 8 g + 32 ks (ks = 0 .. D/32 - 1), the chunks the dQ kernel's lane g holds, so
// that D sums in the dQ kernel's order (see bwd_dq_bf16_kernel's row_stats):
// the same bits whichever kernel computes it.
template <int D, typename T>
constexpr int pre_rows_per_group() {
    return sizeof(T) == 2 ? 64 : 256;
}

template <int D, typename T>
__global__ void __launch_bounds__(256)
bwd_pre_kernel(AttnArgs a, const T* __restrict__ o, const T* __restrict__ dout, const float* __restrict__ lse,
               float* __restrict__ ndelta, float* __restrict__ nlse2, unsigned long long* __restrict__ queue,
               int32_t* __restrict__ items, int32_t* __restrict__ order) {
    if (queue && (int)blockIdx.x < layout_count(a.mode, a.sub)) build_schedule(a, blockIdx.x, queue, items, order);
    constexpr int kLanes = sizeof(T) == 2 ? 4 : 1;  // lanes per row
    const int64_t row = (int64_t)blockIdx.x * pre_rows_per_group<D, T>() + threadIdx.x / kLanes;
    const int g = threadIdx.x % kLanes;
    const int64_t rows = (int64_t)a.batch * a.heads * a.n;
    // (the four lanes of a row share their wave and its exit, so every lane
    // of a row reaches the reduction below)
    if (row >= rows) return;
    const int64_t bh = row / a.n, i = row % a.n;
    const int64_t off = (bh / a.heads) * a.sb + (bh % a.heads) * a.sh + i * a.ss;
    float acc = 0.f;
    if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks)
            acc += dot_bf16x8(ld_bf16x8(dout + off + ks * 32 + 8 * g), ld_bf16x8(o + off + ks * 32 + 8 * g));
        acc += __shfl_xor(acc, 1);  // (g0 + g1) and (g2 + g3), then their sum
        acc += __shfl_xor(acc, 2);
    } else {
        for (int t = 0; t < D; ++t) acc = fmaf(o[off + t], dout[off + t], acc);
    }
    if (g != 0) return;
    ndelta[row] = -acc;
    nlse2[row] = -lse[row] * kLog2e;  // an empty row (LSE = -inf) gives +inf; its items are all masked
}

// ---------------------------------------------------------------------------
// bf16, matrix cores: dQ, row-parallel
// ---------------------------------------------------------------------------
// Query rows per wave.  Strided: 16, so that in a block holding one diagonal
// each wave has a single live 32-key chunk and four waves share the block.
// Fixed: 32, where most steps are fully attended blocks (the summary pairs)
// and each K / V operand read from LDS then serves 32 rows (16 rows at three
// waves per SIMD made the fixed backward at n = 65,536 slower: 2.30 against
// 2.24 ms).
template <int D, int BLK, int PAT>
struct DqCfg {
    static constexpr int RW = BLK < 32 || PAT == STRIDED ? 16 : 32;  // query rows per wave
    static constexpr int QBW = RW / 16;
    static constexpr int NW = BLK / RW;
    static constexpr int NT = NW * 64;
    static constexpr int KS = D / 32;
    static constexpr int KB = BLK / 16;
    static constexpr int KC = (BLK + 31) / 32;
    static constexpr int DB = D / 16;
    static constexpr int NS = 2;  // K / V ring stages
    // (d = 128 with 16-key blocks spilled 16 to 30 registers at three waves)
    static constexpr int WAVES_PER_EU = RW == 16 && !(D == 128 && BLK == 16) ? 3 : 2;
};

// SPLIT (see split_products): the row is walked twice.  The first walk
// recomputes S and dP and sums D_i = sum_j P_ij dP_ij, which is dO_i . O_i for
// the exact O rather than for the O rounded to bf16 that the pre kernel
// reads, and stores it for the dK / dV kernel; the second forms dS from it
// and takes dS into the dQ product in a high and a low bf16 part.
//
// a.row_stats: the kernel does the pre kernel's work for its own rows, D_i =
// dO_i . O_i and the LSE in base 2 (it holds dO_i already), and writes both for
// the dK / dV kernel; its first layout_count workgroups build the dK / dV
// schedule.  The launcher sets it when the grid covers every row and at least
// that many workgroups, and then launches no pre kernel.
template <int D, int BLK, int PAT, int MODE, bool FULL_BODY, bool SPLIT>
__global__ void __launch_bounds__((DqCfg<D, BLK, PAT>::NT))
    __attribute__((amdgpu_waves_per_eu(DqCfg<D, BLK, PAT>::WAVES_PER_EU)))
bwd_dq_bf16_kernel(AttnArgs a, const int32_t* __restrict__ row_ptr, const int32_t* __restrict__ col_idx,
                   const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                   const uint16_t* __restrict__ v, const uint16_t* __restrict__ dout,
                   float* __restrict__ nlse2, float* __restrict__ ndelta,
                   uint16_t* __restrict__ dq, const uint16_t* __restrict__ o, const float* __restrict__ lse,
                   unsigned long long* __restrict__ queue, int32_t* __restrict__ items,
                   int32_t* __restrict__ order) {
    using C = DqCfg<D, BLK, PAT>;
    if (a.row_stats && queue) {  // uniform over the workgroup
        const int64_t wg = blockIdx.x + (int64_t)gridDim.x * (blockIdx.y + (int64_t)gridDim.y * blockIdx.z);
        if (wg < layout_count(a.mode, a.sub)) build_schedule(a, (int)wg, queue, items, order);
    }
    __shared__ __attribute__((aligned(16))) uint16_t sK[C::NS][BLK * D];
    __shared__ __attribute__((aligned(16))) uint16_t sV[C::NS][BLK * D];
    constexpr uint32_t kTileBytes = BLK * D * 2;
    const uint32_t sK_base = lds_addr(&sK[0][0]), sV_base = lds_addr(&sV[0][0]);

    const GridItem gi = row_grid_item(a);  // longest rows first
    const int h = __builtin_amdgcn_readfirstlane(gi.h), qb = __builtin_amdgcn_readfirstlane(gi.qb),
              b = __builtin_amdgcn_readfirstlane(gi.b);
    const int tid = threadIdx.x, lane = tid % 64, g = lane / 16, r = lane % 16;
    const int w = __builtin_amdgcn_readfirstlane(tid / 64);
    const int lay = head_layout(a, h);
    const MaskParams mp = head_mask_params(a, PAT, MODE, h);
    const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;
    const int row0 = qb * BLK + w * C::RW;
    const int qs0 = qb * BLK - a.qshift;  // first query row of the block as the masks see it
    const float c2 = a.scale_log2;
    constexpr uint64_t kTileBits = BLK == 64 ? ~0ull : (1ull << BLK) - 1;

    // this lane's query rows row0 + 16u + r: Q and dO as B operands, -LSE log2 e,
    // and -D splat over a D-result quad (where dP^T accumulation starts)
    bf16x8 qf[C::QBW][C::KS], of[C::QBW][C::KS];
    float nl2[C::QBW];
    f32x4 nd4[C::QBW];
    RowLane rl[C::QBW];
    f32x4 dqacc[C::QBW][C::DB];
#pragma unroll
    for (int u = 0; u < C::QBW; ++u) {
        const int i = row0 + 16 * u + r;
#pragma unroll
        for (int ks = 0; ks < C::KS; ++ks) {
            qf[u][ks] = ld_bf16x8(q + base + (int64_t)i * a.ss + ks * 32 + 8 * g);
            of[u][ks] = ld_bf16x8(dout + base + (int64_t)i * a.ss + ks * 32 + 8 * g);
        }
        const int64_t si = stat_index(a, b, h, i);
        float nd;
        if (a.row_stats) {
            // D_i over the lanes of row i (each holds 8 g .. 8 g + 7 of every
            // 32-wide chunk), and -LSE_i log2 e, as the pre kernel writes them
            float part = 0.f;
#pragma unroll
            for (int ks = 0; ks < C::KS; ++ks)
                part += dot_bf16x8(of[u][ks], ld_bf16x8(o + base + (int64_t)i * a.ss + ks * 32 + 8 * g));
            nd = -sum_over_g(part);
            nl2[u] = -lse[si] * kLog2e;  // an empty row (LSE = -inf) gives +inf; its items are all masked
            if (g == 0) {
                ndelta[si] = nd;
                nlse2[si] = nl2[u];
            }
        } else {
            nl2[u] = nlse2[si];
            nd = ndelta[si];
        }
        nd4[u] = f32x4{nd, nd, nd, nd};
        rl[u] = row_lane(i - a.qshift, a.dl);
#pragma unroll
        for (int db = 0; db < C::DB; ++db) dqacc[u][db] = zero4();
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
    wait_loads_upto<0>();  // register loads done before the ring starts
    // strided blocks away from the band are single diagonals (see the step)
    const bool diag_far = PAT == STRIDED && mp.part != PART_A1 && a.l % BLK == 0;
    TileReader<D> rd;
    rd.init(g, r);
    float dsum[C::QBW];  // first walk of SPLIT: this lane's share of sum_j P_ij dP_ij
#pragma unroll
    for (int u = 0; u < C::QBW; ++u) dsum[u] = 0.f;
    auto walk = [&](auto pass) {
    constexpr bool kSumD = decltype(pass)::value == 0;  // the walk that sums D
    // two-stage ring; the next step's blocks are read one step ahead
    RowStepper<kPairs> steps{col_idx, e0, e1, RowStepper<kPairs>::pair_bound(mp, a.dl, qb * BLK),
                             a.walk == WALK_DENSE};
    RowStep cur = steps.next();
    if (cur.a >= 0) load_step(cur, 0);
    two_stage_while([&](auto stage) {
        constexpr int st = decltype(stage)::value;
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
            // a single diagonal (see the forward): per row one score, one dS and
            // dQ += dS k as a rank-1 step in registers
            if (diag_far && far_block(PAT, a.dl, qs0, j0, BLK)) {
#pragma unroll
                for (int u = 0; u < C::QBW; ++u) {
                    const int kk = w * C::RW + 16 * u + r;  // this lane's row, and its key, in the block
                    float sp = 0.f, dpp = 0.f;
#pragma unroll
                    for (int ks = 0; ks < C::KS; ++ks) {
                        sp += dot_bf16x8(qf[u][ks], ld_bf16x8(tK + Swz<D>::off(kk, 32 * ks + 8 * g)));
                        dpp += dot_bf16x8(of[u][ks], ld_bf16x8(tV + Swz<D>::off(kk, 32 * ks + 8 * g)));
                    }
                    const float pr = exp2_fast(fmaf(sum_over_g(sp), c2, nl2[u]));
                    const float ds = pr * (sum_over_g(dpp) + nd4[u][0]);
#pragma unroll
                    for (int db = 0; db < C::DB; ++db) {
                        const bf16x4 kq =
                            __builtin_bit_cast(bf16x4, *reinterpret_cast<const uint2*>(tK + Swz<D>::off(kk, 16 * db + 4 * g)));
#pragma unroll
                        for (int t = 0; t < 4; ++t) dqacc[u][db][t] = fmaf(ds, (float)kq[t], dqacc[u][db][t]);
                    }
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
            // attends one of its keys; elsewhere dS is zero and the chunk's
            // operands are neither read nor multiplied (wave-uniform branches)
            constexpr int HK = C::KB >= 2 ? 2 : 1;  // 16-key blocks per 32-key chunk
            bool kc_live[C::KC];
#pragma unroll
            for (int kc = 0; kc < C::KC; ++kc) {
                kc_live[kc] = false;
#pragma unroll
                for (int u = 0; u < C::QBW; ++u) kc_live[kc] = kc_live[kc] || cls[u][kc] != CHUNK_NONE;
            }
            // K^T operands of this block, read now: their LDS latency then hides
            // behind the S and dP products and the softmax
            bf16x8 ktr[C::KC][C::DB];
#pragma unroll
            for (int kc = 0; kc < C::KC; ++kc) {
                if (kSumD || !kc_live[kc]) continue;
#pragma unroll
                for (int db = 0; db < C::DB; ++db) {
                    if constexpr (BLK >= 32) ktr[kc][db] = rd.tr(tK, kc * 32, kc * 32 + 16, db);
                    else ktr[kc][db] = rd.tr_half(tK, 0, db);
                }
            }

            // S^T and dP^T - D: x[u][kb16][t] for key j0 + 16 kb16 + 4g + t, query row0 + 16u + r
            f32x4 s[C::QBW][C::KB], dp[C::QBW][C::KB];
#pragma unroll
            for (int kblk = 0; kblk < C::KB; ++kblk) {
                const int kc = kblk / HK;
#pragma unroll
                for (int u = 0; u < C::QBW; ++u) {
                    s[u][kblk] = zero4();
                    dp[u][kblk] = kSumD ? zero4() : nd4[u];
                }
                if (!kc_live[kc]) continue;
                bf16x8 kf[C::KS], vf[C::KS];
#pragma unroll
                for (int ks = 0; ks < C::KS; ++ks) {
                    kf[ks] = rd.row(tK, kblk * 16, ks);
                    vf[ks] = rd.row(tV, kblk * 16, ks);
                }
#pragma unroll
                for (int u = 0; u < C::QBW; ++u) {
                    if (cls[u][kc] == CHUNK_NONE) continue;
#pragma unroll
                    for (int ks = 0; ks < C::KS; ++ks) {
                        s[u][kblk] = mfma_16x16x32(kf[ks], qf[u][ks], s[u][kblk]);
                        dp[u][kblk] = mfma_16x16x32(vf[ks], of[u][ks], dp[u][kblk]);
                    }
                }
            }

            // dS^T = P^T (dP^T - D), P^T = exp2(S^T c2 - LSE log2 e); in the walk
            // that sums D, P^T dP^T instead
            bf16x8 dsf[C::QBW][C::KC], dsl[C::QBW][C::KC];  // dS^T (high and, SPLIT, low parts)
#pragma unroll
            for (int u = 0; u < C::QBW; ++u) {
#pragma unroll
                for (int kc = 0; kc < C::KC; ++kc) {
                    auto chunk = [&](auto part) {
#pragma unroll
                        for (int hk = 0; hk < HK; ++hk) {
                            const int kblk = 2 * kc + hk;
#pragma unroll
                            for (int t = 0; t < 4; ++t) {
                                float pv = exp2_fast(fmaf(s[u][kblk][t], c2, nl2[u]));
                                if constexpr (decltype(part)::value)
                                    pv = select_or_zero(bit_lane_mask(bits[u], 16 * kblk + t), pv);
                                if constexpr (kSumD) dsum[u] = fmaf(pv, dp[u][kblk][t], dsum[u]);
                                else s[u][kblk][t] = pv * dp[u][kblk][t];
                            }
                        }
                    };
                    if (cls[u][kc] == CHUNK_ALL) {
                        chunk(std::false_type{});
                    } else if (cls[u][kc] == CHUNK_PART) {
                        chunk(std::true_type{});
                    } else {
#pragma unroll
                        for (int hk = 0; hk < HK; ++hk) s[u][2 * kc + hk] = zero4();
                    }
                    if constexpr (kSumD) continue;
                    if constexpr (BLK >= 32 && SPLIT) split_bf16x8(s[u][2 * kc], s[u][2 * kc + 1], dsf[u][kc], dsl[u][kc]);
                    else if constexpr (BLK >= 32) dsf[u][kc] = pack_bf16x8(s[u][2 * kc], s[u][2 * kc + 1]);
                    else if constexpr (SPLIT) split_bf16x8(s[u][0], zero4(), dsf[u][kc], dsl[u][kc]);
                    else dsf[u][kc] = pack_bf16x8(s[u][0], zero4());
                }
            }
            if constexpr (kSumD) return;
            // dQ^T += K^T dS^T
#pragma unroll
            for (int kc = 0; kc < C::KC; ++kc) {
#pragma unroll
                for (int u = 0; u < C::QBW; ++u) {
                    if (cls[u][kc] == CHUNK_NONE) continue;
#pragma unroll
                    for (int db = 0; db < C::DB; ++db) dqacc[u][db] = mfma_16x16x32(ktr[kc][db], dsf[u][kc], dqacc[u][db]);
                }
            }
            if constexpr (SPLIT) {
#pragma unroll
                for (int kc = 0; kc < C::KC; ++kc) {
#pragma unroll
                    for (int u = 0; u < C::QBW; ++u) {
                        if (cls[u][kc] == CHUNK_NONE) continue;
#pragma unroll
                        for (int db = 0; db < C::DB; ++db)
                            dqacc[u][db] = mfma_16x16x32(ktr[kc][db], dsl[u][kc], dqacc[u][db]);
                    }
                }
            }
        };
        if (masked || !FULL_BODY) compute(std::false_type{});
        else compute(std::true_type{});
        cur = nxt;
        return true;
    });
    };
    if constexpr (SPLIT) {
        walk(std::integral_constant<int, 0>{});
        // the lanes of a row hold disjoint keys: D_i is the sum over them
#pragma unroll
        for (int u = 0; u < C::QBW; ++u) {
            const float nd = -sum_over_g(dsum[u]);
            nd4[u] = f32x4{nd, nd, nd, nd};
            if (g == 0) ndelta[stat_index(a, b, h, row0 + 16 * u + r)] = nd;
        }
        __syncthreads();  // every wave is done with the ring before it is refilled
    }
    walk(std::integral_constant<int, 1>{});

    // this lane holds dQ^T at d = 16 db + 4g + t for query row0 + 16u + r
#pragma unroll
    for (int u = 0; u < C::QBW; ++u) {
        uint16_t* drow = dq + base + (int64_t)(row0 + 16 * u + r) * a.ss;
#pragma unroll
        for (int db = 0; db < C::DB; ++db) {
            uint2* dst = reinterpret_cast<uint2*>(drow + db * 16 + 4 * g);
            f32x4 x = dqacc[u][db] * a.scale;
            if (a.epilogue == EPI_ADD) x += bf16x4_to_f32x4(*dst);
            *dst = pack_bf16x4_bits(x);
        }
    }
}

// ---------------------------------------------------------------------------
// bf16, matrix cores: dK and dV, column-parallel
// ---------------------------------------------------------------------------
// Waves of 16 keys, four per 64-wide block, three waves per SIMD.  In the
// fixed pattern a block away from the diagonal is uniform over each 16-key
// group (all of its keys are summary keys or none is), so whole waves skip
// their products; in the strided pattern a block holding one diagonal leaves
// each 16-key wave a single live 32-query chunk.
template <int D, int BLK, int PAT>
struct DkvCfg {
    // keys per wave.  (32 keys per wave, two key groups sharing every Q / dO
    // operand read, needs about 290 registers: at one wave per SIMD it made the
    // fixed backward at n = 65,536 slower, 1.68 against 1.45 ms, and at two
    // with spills 2.10 ms; at two with the step body free of spills, 2.80
    // against 2.18 ms; the half and pair logic below handles both widths.)
    static constexpr int KW = 16;
    static constexpr int KBW = KW / 16;         // 16-key blocks per wave
    static constexpr int NW = BLK / KW;         // waves
    static constexpr int NT = NW * 64;
    static constexpr int KS = D / 32;           // 32-deep steps over d
    static constexpr int QB = BLK / 16;         // 16-query blocks per tile
    static constexpr int QC = (BLK + 31) / 32;  // 32-query chunks (contraction over queries)
    static constexpr int DB = D / 16;
    static constexpr int NS = 2;  // Q / dO (and row statistics) ring stages
    // (d = 128 with 16-query blocks spilled 51 to 90 registers at three waves)
    static constexpr int WAVES_PER_EU = KW == 32 || (D == 128 && BLK == 16) ? 2 : 3;
};

// SPLIT: P and dS enter the dV and dK products as a high and a low bf16 part
// (two products each), for calls whose long key columns are attended by rows
// with few keys (see split_products).
template <int D, int BLK, int PAT, int MODE, bool SPLIT>
__global__ void __launch_bounds__((DkvCfg<D, BLK, PAT>::NT))
    __attribute__((amdgpu_waves_per_eu(DkvCfg<D, BLK, PAT>::WAVES_PER_EU)))
bwd_dkdv_bf16_kernel(AttnArgs a, const int32_t* __restrict__ col_ptr, const int32_t* __restrict__ row_idx,
                     const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                     const uint16_t* __restrict__ v, const uint16_t* __restrict__ dout,
                     const float* __restrict__ nlse2, const float* __restrict__ ndelta,
                     uint16_t* __restrict__ dk, uint16_t* __restrict__ dv,
                     unsigned long long* __restrict__ queue, const int32_t* __restrict__ items,
                     const int32_t* __restrict__ order) {
    using C = DkvCfg<D, BLK, PAT>;
    constexpr bool kHalves = PAT == FIXED && BLK == 64;  // items may be 32-key halves
    static_assert(!kHalves || (C::QC == 2 && ((C::NW == 4 && C::KBW == 1) || (C::NW == 2 && C::KBW == 2))),
                  "half items: 4 waves of 16 keys or 2 of 32");
    constexpr int kHalfWaves = C::NW >= 2 ? C::NW / 2 : 1;  // waves per 32-key half in a pair
    __shared__ __attribute__((aligned(16))) uint16_t sQ[C::NS][BLK * D];
    __shared__ __attribute__((aligned(16))) uint16_t sdO[C::NS][BLK * D];
    __shared__ __attribute__((aligned(16))) float sL[C::NS][64];
    __shared__ __attribute__((aligned(16))) float sDl[C::NS][64];
    __shared__ unsigned long long sItem[2];
    constexpr uint32_t kTileBytes = BLK * D * 2;
    constexpr uint64_t kTileBits = BLK == 64 ? ~0ull : (1ull << BLK) - 1;
    const uint32_t sQ_base = lds_addr(&sQ[0][0]), sdO_base = lds_addr(&sdO[0][0]);
    const uint32_t sL_base = lds_addr(&sL[0][0]), sDl_base = lds_addr(&sDl[0][0]);

    const int tid = threadIdx.x, lane = tid % 64, g = lane / 16, r = lane % 16;
    const int w = __builtin_amdgcn_readfirstlane(tid / 64);
    const int64_t bh_count = (int64_t)a.batch * a.heads;
    const float c2 = a.scale_log2;
    TileLoader<D, BLK, C::NW> ld;
    ld.init(a.ss, w, lane);
    TileReader<D> rd;
    rd.init(g, r);
    // Claims are made by thread 0, which walks the queues from its own XCD's
    // on; a claim is (queue << 56 | index), with bit kAscend set when the
    // column is walked upwards (below), kNoWork once all queues are dry.
    constexpr unsigned long long kNoWork = ~0ull;
    constexpr unsigned long long kAscend = 1ull << 55;
    int qx = 0, q_left = kQueues;
    uint64_t per_layout = 0;  // item slots taken per (batch, head): the largest item count of a layout
    if (tid == 0) {
        const int n_layouts = layout_count(a.mode, a.sub);
        // walks of the band or of every block take the key blocks whole, in
        // order (the longest columns first when dense); no item order is built
        if (a.walk != WALK_LAYOUT) per_layout = (uint64_t)a.nq;
        else
            for (int gl = 0; gl < n_layouts; ++gl)
                per_layout = (uint64_t)items[gl] > per_layout ? (uint64_t)items[gl] : per_layout;
        unsigned xcc;
        asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID, 0, 4)" : "=s"(xcc));
        qx = (int)(xcc % kQueues);
    }
    // How thread 0 finds the next slot (a.claim_mode, chosen by the launcher):
    //   CLAIM_QUEUES: from the queue counters, one atomic per slot, stealing
    //     from the other queues once its own is dry;
    //   CLAIM_ROUND_ROBIN: workgroup w takes the slots w, w + G, w + 2G, ... (G
    //     workgroups) of the rank-major order (every (batch, head) of the
    //     longest columns first), with no atomics;
    //   CLAIM_SERPENTINE: workgroup w serves head w mod (batch heads) alone and
    //     takes that head's ranks in serpentine order over the J workgroups of
    //     the head (j, 2J - 1 - j, 2J + j, ...), which evens out the sums of
    //     sorted column lengths, with no atomics; after the first round the
    //     first J / 16 places drop out of the serpentine (below);
    //   CLAIM_XCD_SERPENTINE: workgroup w (on XCD x = w mod 8, the j-th of
    //     its J there) serves the heads bh = x (mod 8), head by head with
    //     every column of a head, longest first, before the next: places
    //     kJ + j for even k, kJ + J - 1 - j for odd k of that sequence.  The
    //     J workgroups of an XCD thus walk the columns of J / nq heads at a
    //     time, whose Q and dO stay in that XCD's L2 (the residue classes:
    //     many short dense heads read at a stride of l rows).  Needs the grid
    //     and batch x heads multiples of 8 (the launcher checks).
    // The atomics of all workgroups on one counter are serialised
    // device-wide; with many short columns a claim waits longer than a column
    // takes, hence the fixed orders.  Every mode yields queue-encoded slots.
    //   In the two serpentine orders the workgroups of a head start each
    // round at about the same time, since their earlier columns' lengths
    // sum to about the same.  Columns of even rounds are walked from their
    // last query block down, of odd rounds from their first up: a column of
    // length L started at time T then reads query block (last - L + 1) +
    // (t - T), and T + L is about the same for every workgroup of the
    // round, so they all read the same Q / dO tile at the same time and it
    // is fetched into L2 once.  (Downwards in every round, the second
    // round's walks start at staggered times from the same last block; the
    // tiles between them outgrow an XCD's L2 and were fetched again by each.)
    uint64_t next_slot = blockIdx.x, sweep = 0;
    auto encode = [&](uint64_t rank, int bh) -> unsigned long long {
        const int x = bh % kQueues;
        return ((uint64_t)x << 56) | (rank * (uint64_t)queue_heads(bh_count, x) + (uint64_t)(bh / kQueues));
    };
    auto claim = [&]() -> unsigned long long {
        if (a.claim_mode == CLAIM_ROUND_ROBIN) {
            if (next_slot >= per_layout * (uint64_t)bh_count) return kNoWork;
            const uint64_t s = next_slot;
            next_slot += gridDim.x;
            const uint64_t rank = s / (uint64_t)bh_count;
            return encode(rank, (int)(s - rank * (uint64_t)bh_count));
        }
        if (a.claim_mode == CLAIM_XCD_SERPENTINE) {
            const uint64_t J = gridDim.x / kQueues, j = blockIdx.x / kQueues;
            const int x = (int)(blockIdx.x % kQueues);
            const uint64_t k = sweep++;
            const uint64_t p = k * J + ((k & 1) ? J - 1 - j : j);
            const uint64_t i = p / per_layout;  // the i-th head of this XCD
            if (i >= (uint64_t)(bh_count / kQueues)) return kNoWork;
            return encode(p - i * per_layout, x + kQueues * (int)i) | ((k & 1) ? kAscend : 0ull);
        }
        if (a.claim_mode == CLAIM_SERPENTINE) {
            const int bh = (int)(blockIdx.x % (uint64_t)bh_count);
            const uint64_t j = blockIdx.x / (uint64_t)bh_count;
            const uint64_t J = (gridDim.x - bh + bh_count - 1) / bh_count;  // workgroups of this head
            const uint64_t k = sweep++;
            // The first sixteenth of the places (the head's longest columns)
            // take nothing after their first: with long summary columns the
            // longest chain is the first place's column plus what follows it,
            // and the later rounds serpentine over the other places.  (More
            // places left out, an eighth or a quarter, crowded the short
            // columns into fewer workgroups and fetched more.)
            uint64_t rank = j;
            if (k > 0) {
                const uint64_t S = J / 16;
                if (j < S) return kNoWork;
                const uint64_t J2 = J - S, j2 = j - S, kk = k - 1;
                rank = J + kk * J2 + ((kk & 1) ? j2 : J2 - 1 - j2);
            }
            return rank < per_layout ? encode(rank, bh) | ((k & 1) ? kAscend : 0ull) : kNoWork;
        }
        while (q_left > 0) {
            const uint64_t t = atomicAdd(queue + qx, 1ull);
            if (t < per_layout * (uint64_t)queue_heads(bh_count, qx)) return ((uint64_t)qx << 56) | t;
            qx = qx + 1 == kQueues ? 0 : qx + 1;
            --q_left;
        }
        return kNoWork;
    };
    if (tid == 0) sItem[0] = claim();
    __syncthreads();
    // Every wave leaves the loop at the same claim: the claim is shared
    // through LDS and is kNoWork once every queue has run dry.  A group item
    // takes one pass of the loop per key block of its l-block (grp_kb ..
    // grp_end - 1 still to come, wave-uniform); the claim after it is made
    // when the group starts and published after its last block.
    int ci = 0, grp_kb = 0, grp_end = 0;
    int h = 0, b = 0, lay = 0;
    bool ascend = false;
    unsigned long long next = 0ull;
    for (;;) {
        int kb = 0, kind = -1;
        if (grp_kb < grp_end) {
            kb = grp_kb++;
            kind = __builtin_amdgcn_readfirstlane(group_member(a, lay, kb, col_ptr + (int64_t)lay * (a.nq + 1)));
        } else {
            const uint64_t item = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(sItem[ci & 1] >> 32)) << 32) |
                                  __builtin_amdgcn_readfirstlane((uint32_t)sItem[ci & 1]);
            if (item == kNoWork) break;
            if (tid == 0) next = claim();  // claimed now, published after the column (or group)
            const int x = (int)(item >> 56);
            ascend = (item & kAscend) != 0ull;
            const uint64_t t = item & (kAscend - 1);
            const int64_t nx = queue_heads(bh_count, x);
            // (the scalar unit holds every index of the column walk; the
            // readfirstlane calls only tell the compiler so)
            const int rank = __builtin_amdgcn_readfirstlane((int)(t / (uint64_t)nx));  // position in the length order
            const int bh = __builtin_amdgcn_readfirstlane(x + kQueues * (int)(t - (uint64_t)rank * nx));
            h = bh % a.heads;
            b = bh / a.heads;
            lay = head_layout(a, h);
            const int32_t code = a.walk != WALK_LAYOUT
                                     ? item_code(rank, 0)
                                     : __builtin_amdgcn_readfirstlane(order[(int64_t)lay * 2 * a.nq + rank]);
            // code < 0: an empty slot (a layout with fewer items than another)
            if (code >= 0) {
                kb = code & ((1 << kItemShift) - 1);
                kind = kHalves ? code >> kItemShift : 0;
                if (kHalves && kind == kGroupKind) {
                    grp_kb = kb + 1;
                    grp_end = min(kb + group_blocks(a), a.nq);
                    kind = __builtin_amdgcn_readfirstlane(
                        group_member(a, lay, kb, col_ptr + (int64_t)lay * (a.nq + 1)));
                }
            }
        }
        // kind < 0: an empty slot, or a block of a group whose column is long
        // (an item of its own)
        if (kind >= 0) {
        // In a pair the first half of the waves takes the summary half of kb,
        // the second half that of kb + l / 64, each for all queries of a block;
        // a single half is shared by all waves: with four waves of 16 keys, two
        // key groups times two query halves; with two waves of 32 keys, both
        // key groups times one query half each.
        const bool pair = kind >= 3;
        const int half = pair ? kind - 2 : kind;  // 32-key half walked; 0: the whole block
        const bool single = half != 0 && !pair;
        const int kb_w = pair && w >= kHalfWaves ? kb + a.l / 64 : kb;  // this wave's key block
        const int qhalf = w / kHalfWaves;  // single half: the 32-query half of each block this wave takes
        const MaskParams mp = head_mask_params(a, PAT, MODE, h);
        const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;
        // This wave's keys are the 16-key groups w, w + NW, ...: interleaved, so
        // that the waves share the summary columns of the fixed pattern (which
        // sit at the end of a block) and with them the softmax work.  In a
        // single half the wave takes key group w mod 2 of the half (both with
        // 32 keys per wave), for the queries of one 32-query half (qhalf) of
        // every block; in a pair, the same groups of its block's half, for
        // every query.
        auto kgrp = [&](int kbw) {
            return half == 0 ? C::NW * kbw + w : 2 * (half - 1) + (C::KBW == 2 ? kbw : (w & 1));
        };
        auto key_of = [&](int kbw) { return kb_w * BLK + 16 * kgrp(kbw) + r; };

        // this lane's keys j = key_of(kbw) as B operands (d = 32 ks + 8g + t)
        bf16x8 kf[C::KBW][C::KS], vf[C::KBW][C::KS];
        ColLane cl[C::KBW];
#pragma unroll
        for (int kbw = 0; kbw < C::KBW; ++kbw) {
            const int j = key_of(kbw);
#pragma unroll
            for (int ks = 0; ks < C::KS; ++ks) {
                // In the fixed pattern these rows are read once, and kept out
                // of L2 they leave it to the Q / dO tiles the walks share (510 ->
                // 499 MiB fetched per launch at n = 65,536, the same time); the
                // strided band reads them just after the dQ kernel did and
                // takes them from the caches (non-temporal: 2-4% slower).
                if constexpr (PAT == FIXED) {
                    kf[kbw][ks] = ld_bf16x8_once(k + base + (int64_t)j * a.ss + ks * 32 + 8 * g);
                    vf[kbw][ks] = ld_bf16x8_once(v + base + (int64_t)j * a.ss + ks * 32 + 8 * g);
                } else {
                    kf[kbw][ks] = ld_bf16x8(k + base + (int64_t)j * a.ss + ks * 32 + 8 * g);
                    vf[kbw][ks] = ld_bf16x8(v + base + (int64_t)j * a.ss + ks * 32 + 8 * g);
                }
            }
            cl[kbw] = col_lane(j, a.dl, a.c, mp.w);
        }
        // summary keys of this key block (fixed pattern), bit = key offset in the block
        const uint64_t key_summary = PAT == FIXED ? summary_bits(mp, mod_l(a.dl, kb_w * BLK)) & kTileBits : 0ull;
        f32x4 dvacc[C::KBW][C::DB], dkacc[C::KBW][C::DB];
#pragma unroll
        for (int kbw = 0; kbw < C::KBW; ++kbw)
#pragma unroll
            for (int db = 0; db < C::DB; ++db) {
                dvacc[kbw][db] = zero4();
                dkacc[kbw][db] = zero4();
            }

        int e0 = 0, len = a.nq - kb;  // WALK_DENSE: query blocks kb .. nq - 1
        if (a.walk != WALK_DENSE) {
            const int64_t cp = (int64_t)lay * (a.nq + 1) + kb;
            e0 = __builtin_amdgcn_readfirstlane(col_ptr[cp]);
            len = __builtin_amdgcn_readfirstlane(col_ptr[cp + 1]) - e0;
            if (a.walk == WALK_BAND) len = min(len, a.l / BLK + 1);
        }
        if (single && ((key_summary >> (32 * (half - 1))) & 0xFFFFFFFFull) == 0ull) {
            // the non-summary half is attended only inside its own l-block:
            // the column's first entries (the query blocks ascend)
            int near = 0;
            while (near < len &&
                   !far_block(FIXED, a.dl, BLK * __builtin_amdgcn_readfirstlane(row_idx[e0 + near]), kb * BLK, BLK))
                ++near;
            len = near;
        }
        // strided blocks away from the band are single diagonals (see the step)
        const bool diag_far = PAT == STRIDED && mp.part != PART_A1 && a.l % BLK == 0;
        // The column is walked from its last query block down (or, in odd
        // serpentine rounds, from its first up; see the claims): the long
        // columns of a head, started together, then visit the same query
        // blocks at about the same time and share those Q / dO tiles in L2.
        auto query_block = [&](int sidx) {
            const int e = ascend ? sidx : len - 1 - sidx;
            return a.walk == WALK_DENSE ? kb + e : __builtin_amdgcn_readfirstlane(row_idx[e0 + e]);
        };
        auto load_block = [&](int qb, int stage) {
            const int64_t qbase = base + (int64_t)qb * BLK * a.ss;
            ld.issue(q + qbase, sQ_base + stage * kTileBytes);
            ld.issue(dout + qbase, sdO_base + stage * kTileBytes);
            const int64_t st0 = stat_index(a, b, h, (int64_t)qb * BLK);
            if (w == 0) load_row_stats_async(nlse2 + st0, BLK, sL_base + stage * 256u, lane, (uint32_t)a.lse_ss);
            if (w == C::NW - 1)
                load_row_stats_async(ndelta + st0, BLK, sDl_base + stage * 256u, lane, (uint32_t)a.lse_ss);
        };

        wait_loads_upto<0>();  // register loads done before the ring starts
        // two-stage ring: the next block's index is read one step ahead (a
        // scalar load, off the vector-memory counter the ring waits on)
        int qb_next = len > 0 ? query_block(0) : 0;
        if (len > 0) load_block(qb_next, 0);
        two_stage_loop(len, [&](auto stage, int sidx) {
            constexpr int st = decltype(stage)::value;
            const int qb = qb_next;
            qb_next = sidx + 1 < len ? query_block(sidx + 1) : 0;
            const int i0 = qb * BLK - a.qshift;  // first query row of the block as the masks see it
            // a pair's keys are summary keys, attended by every query of a block
            // away from both key blocks' l-blocks
            const bool masked =
                pair ? !far_block(PAT, a.dl, i0, (kb + a.l / 64) * BLK, BLK)
                     : !block_full32(PAT, mp.part, a.dl, a.c, mp.w, i0, i0 + BLK - 1, kb * BLK, kb * BLK + BLK - 1);
            wait_loads_upto<0>();
            __syncthreads();  // block sidx is in LDS everywhere; the other stage is free
            if (sidx + 1 < len) load_block(qb_next, st ^ 1);
            const uint16_t* tQ = sQ[st];
            const uint16_t* tO = sdO[st];
            const float* tL = sL[st];
            const float* tD = sDl[st];
            if constexpr (PAT == STRIDED) {
                // a single diagonal (see the forward): key kk of the block meets
                // query kk only, so dV += p dO and dK += dS q are rank-1 steps in
                // registers
                if (diag_far && far_block(PAT, a.dl, i0, kb * BLK, BLK)) {
#pragma unroll
                    for (int kbw = 0; kbw < C::KBW; ++kbw) {
                        const int kk = 16 * kgrp(kbw) + r;  // this lane's key, and its query, in the block
                        float sp = 0.f, dpp = 0.f;
#pragma unroll
                        for (int ks = 0; ks < C::KS; ++ks) {
                            sp += dot_bf16x8(kf[kbw][ks], ld_bf16x8(tQ + Swz<D>::off(kk, 32 * ks + 8 * g)));
                            dpp += dot_bf16x8(vf[kbw][ks], ld_bf16x8(tO + Swz<D>::off(kk, 32 * ks + 8 * g)));
                        }
                        const float pr = exp2_fast(fmaf(sum_over_g(sp), c2, tL[kk]));
                        const float ds = pr * (sum_over_g(dpp) + tD[kk]);
#pragma unroll
                        for (int db = 0; db < C::DB; ++db) {
                            const bf16x4 oq = __builtin_bit_cast(
                                bf16x4, *reinterpret_cast<const uint2*>(tO + Swz<D>::off(kk, 16 * db + 4 * g)));
                            const bf16x4 qq = __builtin_bit_cast(
                                bf16x4, *reinterpret_cast<const uint2*>(tQ + Swz<D>::off(kk, 16 * db + 4 * g)));
#pragma unroll
                            for (int t = 0; t < 4; ++t) {
                                dvacc[kbw][db][t] = fmaf(pr, (float)oq[t], dvacc[kbw][db][t]);
                                dkacc[kbw][db][t] = fmaf(ds, (float)qq[t], dkacc[kbw][db][t]);
                            }
                        }
                    }
                    return;
                }
            }
            // The step body exists for blocks attended everywhere (every chunk
            // class a compile-time ALL, no mask; with one_half, a single half
            // leaves one query half to the other waves) and for the others, in
            // both patterns.
            auto compute = [&](auto full, auto one_half) {

                // -LSE log2 e and -D of queries i0 + 16 qblk + 4g + t
                auto row_stat = [&](const float* tile, int qblk) {
                    return *reinterpret_cast<const f32x4*>(&tile[qblk * 16 + 4 * g]);
                };
                // mask bits of this lane's column (bit 16 qblk + t after the shift),
                // and which 32-query chunks hold an attended item anywhere in the wave
                uint64_t bits[C::KBW];
                int cls[C::KBW][C::QC];
#pragma unroll
                for (int kbw = 0; kbw < C::KBW; ++kbw) {
                    bits[kbw] = ~0ull;
#pragma unroll
                    for (int qc = 0; qc < C::QC; ++qc) cls[kbw][qc] = CHUNK_ALL;
                }
                if constexpr (!decltype(full)::value) {
                    const int i0_mod = mod_l(a.dl, i0);
                    const bool far = far_block(PAT, a.dl, i0, kb_w * BLK, BLK);
                    if (PAT == FIXED && far && mp.part != PART_A1) {
                        // a summary key is attended by every row, any other key by none
#pragma unroll
                        for (int kbw = 0; kbw < C::KBW; ++kbw) {
                            bits[kbw] = cl[kbw].summary ? (kTileBits >> (4 * g)) : 0ull;
                            const uint32_t keys = (uint32_t)(key_summary >> (16 * kgrp(kbw))) & 0xFFFFu;
                            const int k_cls = keys == 0u ? CHUNK_NONE : (keys == 0xFFFFu ? CHUNK_ALL : CHUNK_PART);
#pragma unroll
                            for (int qc = 0; qc < C::QC; ++qc) cls[kbw][qc] = k_cls;
                        }
                    } else if (far) {
#pragma unroll
                        for (int kbw = 0; kbw < C::KBW; ++kbw)
                            bits[kbw] = (col_mask_far(mp, cl[kbw], i0_mod) & kTileBits) >> (4 * g);
                    } else {
#pragma unroll
                        for (int kbw = 0; kbw < C::KBW; ++kbw)
                            bits[kbw] = (col_mask(mp, cl[kbw], i0, i0_mod) & kTileBits) >> (4 * g);
                    }
                    if (!(PAT == FIXED && far && mp.part != PART_A1)) {
#pragma unroll
                        for (int kbw = 0; kbw < C::KBW; ++kbw)
#pragma unroll
                            for (int qc = 0; qc < C::QC; ++qc)
                                cls[kbw][qc] = chunk_class(chunk_bits(bits[kbw], qc, C::QB >= 2), C::QB >= 2);
                    }
                }

                if (decltype(one_half)::value || (!decltype(full)::value && single)) {
                    // a single half: this wave takes one 32-query half of the block
#pragma unroll
                    for (int kbw = 0; kbw < C::KBW; ++kbw)
#pragma unroll
                        for (int qc = 0; qc < C::QC; ++qc)
                            if (qc != qhalf) cls[kbw][qc] = CHUNK_NONE;
                }
                // A 32-query chunk enters the products only where some key of the
                // wave is attended by one of its queries; elsewhere P and dS are zero
                // and its operands are neither read nor multiplied (wave-uniform
                // branches)
                constexpr int HQ = C::QB >= 2 ? 2 : 1;  // 16-query blocks per 32-query chunk
                // unmasked steps: ask the scheduler to interleave the exponentials
                // with the matrix products (its strategy for attention-like loops)
                if constexpr (decltype(full)::value && !decltype(one_half)::value && C::KW == 16)
                    __builtin_amdgcn_iglp_opt(2);
                bool qc_live[C::QC];
#pragma unroll
                for (int qc = 0; qc < C::QC; ++qc) {
                    qc_live[qc] = false;
#pragma unroll
                    for (int kbw = 0; kbw < C::KBW; ++kbw) qc_live[qc] = qc_live[qc] || cls[kbw][qc] != CHUNK_NONE;
                }
                // Per 32-query chunk: S and dP - D, then P = exp2(S c2 - LSE log2 e)
                // and dS = P (dP - D), then dV^T += dO^T P and dK^T += Q^T dS,
                // contracting over the chunk's queries (dO^T and Q^T read
                // transposed from the row-major tiles).  A chunk is finished before
                // the next starts, so only its P and dS are live.
#pragma unroll
                for (int qc = 0; qc < C::QC; ++qc) {
                    if (!qc_live[qc]) continue;
                    // x[kbw][hq][t]: query i0 + 16 (2 qc + hq) + 4g + t against key key_of(kbw)
                    f32x4 p[C::KBW][HQ], ds[C::KBW][HQ];
#pragma unroll
                    for (int hq = 0; hq < HQ; ++hq) {
                        const int qblk = HQ * qc + hq;
                        bf16x8 qa[C::KS], oa[C::KS];
#pragma unroll
                        for (int ks = 0; ks < C::KS; ++ks) {
                            qa[ks] = rd.row(tQ, qblk * 16, ks);
                            oa[ks] = rd.row(tO, qblk * 16, ks);
                        }
#pragma unroll
                        for (int kbw = 0; kbw < C::KBW; ++kbw) {
                            if (cls[kbw][qc] == CHUNK_NONE) continue;
                            f32x4 sacc = zero4(), dpacc = row_stat(tD, qblk);
#pragma unroll
                            for (int ks = 0; ks < C::KS; ++ks) {
                                sacc = mfma_16x16x32(qa[ks], kf[kbw][ks], sacc);
                                dpacc = mfma_16x16x32(oa[ks], vf[kbw][ks], dpacc);
                            }
                            p[kbw][hq] = sacc;
                            ds[kbw][hq] = dpacc;
                        }
                    }
                    // (SPLIT: every transposed operand is kept for the low parts,
                    // issued after every high part so that no product waits on the
                    // one just issued; otherwise each is read one d-block ahead of
                    // its products, in the fixed pattern the first before the
                    // exponentials, so that the products do not wait on the LDS: the
                    // fixed backward at n = 65,536 took 4% and then another 1.5% less
                    // than with each read just before its use.  The strided kernels
                    // read the first after the exponentials: earlier, its registers
                    // made them spill.)
                    constexpr int kKeep = SPLIT ? C::DB : 2;
                    bf16x8 oT[kKeep], qT[kKeep];
                    auto read_tr = [&](int db, int x) {
                        if constexpr (BLK >= 32) {
                            oT[x] = rd.tr(tO, qc * 32, qc * 32 + 16, db);
                            qT[x] = rd.tr(tQ, qc * 32, qc * 32 + 16, db);
                        } else {
                            oT[x] = rd.tr_half(tO, 0, db);
                            qT[x] = rd.tr_half(tQ, 0, db);
                        }
                    };
                    constexpr bool kEarly = !SPLIT && PAT == FIXED;
                    if constexpr (kEarly) read_tr(0, 0);
                    bf16x8 pb[C::KBW], sb[C::KBW];
                    bf16x8 pbl[C::KBW], sbl[C::KBW];  // low parts (SPLIT)
#pragma unroll
                    for (int kbw = 0; kbw < C::KBW; ++kbw) {
                        auto chunk = [&](auto part) {
#pragma unroll
                            for (int hq = 0; hq < HQ; ++hq) {
                                const int qblk = HQ * qc + hq;
                                const f32x4 nl = row_stat(tL, qblk);
#pragma unroll
                                for (int t = 0; t < 4; ++t) {
                                    float pv = exp2_fast(fmaf(p[kbw][hq][t], c2, nl[t]));
                                    if constexpr (decltype(part)::value)
                                        pv = select_or_zero(bit_lane_mask(bits[kbw], 16 * qblk + t), pv);
                                    p[kbw][hq][t] = pv;
                                    ds[kbw][hq][t] = pv * ds[kbw][hq][t];
                                }
                            }
                            if constexpr (HQ == 2 && SPLIT) {
                                split_bf16x8(p[kbw][0], p[kbw][1], pb[kbw], pbl[kbw]);
                                split_bf16x8(ds[kbw][0], ds[kbw][1], sb[kbw], sbl[kbw]);
                            } else if constexpr (HQ == 2) {
                                pb[kbw] = pack_bf16x8(p[kbw][0], p[kbw][1]);
                                sb[kbw] = pack_bf16x8(ds[kbw][0], ds[kbw][1]);
                            } else if constexpr (SPLIT) {
                                split_bf16x8(p[kbw][0], zero4(), pb[kbw], pbl[kbw]);
                                split_bf16x8(ds[kbw][0], zero4(), sb[kbw], sbl[kbw]);
                            } else {
                                pb[kbw] = pack_bf16x8(p[kbw][0], zero4());
                                sb[kbw] = pack_bf16x8(ds[kbw][0], zero4());
                            }
                        };
                        if (cls[kbw][qc] == CHUNK_ALL) chunk(std::false_type{});
                        else if (cls[kbw][qc] == CHUNK_PART) chunk(std::true_type{});
                    }
                    if constexpr (!SPLIT && !kEarly) read_tr(0, 0);
#pragma unroll
                    for (int db = 0; db < C::DB; ++db) {
                        const int x = SPLIT ? db : (db & 1);
                        if constexpr (SPLIT) read_tr(db, db);
                        else if (db + 1 < C::DB) read_tr(db + 1, (db + 1) & 1);
#pragma unroll
                        for (int kbw = 0; kbw < C::KBW; ++kbw) {
                            if (cls[kbw][qc] == CHUNK_NONE) continue;
                            dvacc[kbw][db] = mfma_16x16x32(oT[x], pb[kbw], dvacc[kbw][db]);
                            dkacc[kbw][db] = mfma_16x16x32(qT[x], sb[kbw], dkacc[kbw][db]);
                        }
                    }
                    if constexpr (SPLIT) {
#pragma unroll
                        for (int db = 0; db < C::DB; ++db) {
#pragma unroll
                            for (int kbw = 0; kbw < C::KBW; ++kbw) {
                                if (cls[kbw][qc] == CHUNK_NONE) continue;
                                dvacc[kbw][db] = mfma_16x16x32(oT[db % kKeep], pbl[kbw], dvacc[kbw][db]);
                                dkacc[kbw][db] = mfma_16x16x32(qT[db % kKeep], sbl[kbw], dkacc[kbw][db]);
                            }
                        }
                    }
                    // with 32 keys per wave, chunks are kept apart: scheduled
                    // together their live values outgrow two waves' registers
                    if constexpr (C::KW == 32) __builtin_amdgcn_sched_barrier(0);
                }
            };
            // unmasked steps of whole blocks and pairs run without a runtime
            // chunk class (straight-line code over both query chunks)
            if (masked) {
                compute(std::false_type{}, std::false_type{});
            } else if constexpr (kHalves) {
                if (single) compute(std::true_type{}, std::true_type{});
                else compute(std::true_type{}, std::false_type{});
            } else {
                compute(std::true_type{}, std::false_type{});
            }
        });

        if constexpr (kHalves) {
            if (single) {
                // the two query halves of each key group are summed through LDS
                // (the ring is idle once every wave has passed the last step)
                static_assert(sizeof(sQ) >= (size_t)kHalfWaves * C::KBW * 2 * C::DB * 64 * sizeof(f32x4),
                              "reduction fits the Q ring");
                __syncthreads();
                f32x4* red = reinterpret_cast<f32x4*>(&sQ[0][0]);
                const int slot0 = (w % kHalfWaves) * C::KBW * 2 * C::DB;
                if (qhalf == 1) {
#pragma unroll
                    for (int kbw = 0; kbw < C::KBW; ++kbw)
#pragma unroll
                        for (int db = 0; db < C::DB; ++db) {
                            red[(slot0 + kbw * 2 * C::DB + db) * 64 + lane] = dvacc[kbw][db];
                            red[(slot0 + kbw * 2 * C::DB + C::DB + db) * 64 + lane] = dkacc[kbw][db];
                        }
                }
                __syncthreads();
                if (qhalf == 0) {
#pragma unroll
                    for (int kbw = 0; kbw < C::KBW; ++kbw)
#pragma unroll
                        for (int db = 0; db < C::DB; ++db) {
                            dvacc[kbw][db] += red[(slot0 + kbw * 2 * C::DB + db) * 64 + lane];
                            dkacc[kbw][db] += red[(slot0 + kbw * 2 * C::DB + C::DB + db) * 64 + lane];
                        }
                }
            }
        }
        // this lane holds dV^T / dK^T at d = 16 db + 4g + t for key key_of(kbw)
#pragma unroll
        for (int kbw = 0; kbw < C::KBW; ++kbw) {
            if (single && qhalf == 1) break;  // written by the wave of the other query half
            const int j = key_of(kbw);
            uint16_t* dvrow = dv + base + (int64_t)j * a.ss;
            uint16_t* dkrow = dk + base + (int64_t)j * a.ss;
#pragma unroll
            for (int db = 0; db < C::DB; ++db) {
                uint2* dvp = reinterpret_cast<uint2*>(dvrow + db * 16 + 4 * g);
                uint2* dkp = reinterpret_cast<uint2*>(dkrow + db * 16 + 4 * g);
                f32x4 xv = dvacc[kbw][db], xk = dkacc[kbw][db] * a.scale;
                if (a.epilogue == EPI_ADD) {
                    xv += bf16x4_to_f32x4(*dvp);
                    xk += bf16x4_to_f32x4(*dkp);
                }
                *dvp = pack_bf16x4_bits(xv);
                *dkp = pack_bf16x4_bits(xk);
            }
        }
        }  // kind >= 0
        if (grp_kb >= grp_end) {
            if (tid == 0) sItem[(ci + 1) & 1] = next;
            ++ci;
        }
        // the ring is free again and the next claim is visible to every wave
        __syncthreads();
    }
}

constexpr int64_t align16(int64_t x) { return (x + 15) / 16 * 16; }

inline int64_t bwd_workspace_size(int64_t rows, int64_t nq, int n_layouts) {
    return align16(2 * rows * (int64_t)sizeof(float)) + kQueues * 8 + (int64_t)n_layouts * 4 +
           (int64_t)n_layouts * 2 * nq * 4;
}

inline BwdWorkspace bwd_workspace(void* ws, int64_t rows, int n_layouts) {
    char* p = static_cast<char*>(ws);
    BwdWorkspace w;
    w.ndelta = reinterpret_cast<float*>(p);
    w.nlse2 = w.ndelta + rows;
    w.queue = reinterpret_cast<unsigned long long*>(p + align16(2 * rows * (int64_t)sizeof(float)));
    w.items = reinterpret_cast<int32_t*>(w.queue + kQueues);
    w.order = w.items + n_layouts;
    return w;
}

// Workgroups of `Kernel` the current device holds at once (0 if unknown),
// cached per kernel and device (every instantiation of this template has its
// own cache: kernels differ in registers and LDS, hence in occupancy).
template <auto Kernel>
int64_t resident_workgroups(int threads) {
    static std::atomic<int64_t> cache[64];
    const auto kernel = Kernel;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 0;
    if (dev < 64) {
        const int64_t v = cache[dev].load(std::memory_order_relaxed);
        if (v > 0) return v;
    }
    int cus = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess) return 0;
    const int64_t v = (int64_t)cus * per_cu;
    if (dev < 64 && v > 0) cache[dev].store(v, std::memory_order_relaxed);
    return v;
}

// Whether the dK / dV products take P and dS in two bf16 parts.  Rounding
// P_ij (and dS_ij) to bf16 moves each term of dV_j = sum_i P_ij dO_i by up to
// 2^-8 of itself, independently, so over a key column the error grows like
// 2^-8 (sum_i P_ij^2 / 3)^(1/2) |dO|.  A row attending m keys has P_ij of
// about 1/m, so the column weight W = sum_i 1 / m_i^2 over the rows of the
// longest column decides.  The long columns are the summary columns of the
// fixed pattern (Sec. 4.3), attended by every later row: a row of l-block L
// attends c L summary keys (A2 alone), or its own r + 1 keys besides (merged),
// so
//   A2 alone:  W = (l / c^2) sum_{L >= 1} 1 / L^2
//   merged:    W = sum_{L >= 1} sum_{r < l} 1 / (c L + r + 1)^2.
// Strided columns meet rows with at least |A2| = floor(i / l) + 1 keys one
// stride apart, W <= pi^2 / 6 spread over a handful of large weights, and A1
// columns are short.  Above W = 0.15 (an expected error near 0.003 |dO| per
// column at the one-part products, against a bound of 2e-2 on the largest of
// many columns) the products are split; the configurations of the paper's
// experiments stay below it (l = 128 or 256 with c = 32).
inline bool split_products(const AttnArgs& a) {
    if (a.pattern != FIXED || a.mode == MODE_A1) return false;
    const int64_t blocks = ((int64_t)a.n + a.l - 1) / a.l;  // l-blocks
    const double l = a.l, c = a.c;
    double w = 0.0;
    const int64_t last = blocks - 1 < (1 << 20) ? blocks - 1 : (1 << 20);
    const bool a2_alone = a.mode == MODE_A2 || a.mode == MODE_INTERLEAVED;
    for (int64_t L = 1; L <= last; ++L) {
        const double cl = c * (double)L;
        // sum_{m = cL+1}^{cL+l} 1/m^2, by the midpoint rule of 1/x^2
        w += a2_alone ? l / (cl * cl) : 1.0 / (cl + 0.5) - 1.0 / (cl + l + 0.5);
    }
    return w > 0.15;
}

template <int D, int BLK>
hipError_t launch_bwd_bf16(const AttnArgs& a, const void* q, const void* k, const void* v,
                           const void* o, const void* dout, const float* lse, void* dq, void* dk,
                           void* dv, const BwdWorkspace& ws, hipStream_t stream, int parts) {
    const int64_t rows = (int64_t)a.batch * a.heads * a.n;
    float* ndelta = ws.ndelta;
    float* nlse2 = ws.nlse2;
    constexpr int kPreRows = pre_rows_per_group<D, uint16_t>();
    const int64_t pre_groups = (rows + kPreRows - 1) / kPreRows > layout_count(a.mode, a.sub)
                                   ? (rows + kPreRows - 1) / kPreRows
                                   : layout_count(a.mode, a.sub);
    dim3 grid((unsigned)a.heads, (unsigned)a.nq, (unsigned)a.batch);
    const int64_t items = (int64_t)a.nq * a.batch * a.heads;
    AttnArgs ak = a;
    const bool split = split_products(a);
    return with_pattern_mode(a.pattern, a.mode, [&](auto pat, auto mode) {
        constexpr int PAT = decltype(pat)::value, MODE = decltype(mode)::value;
        const int64_t slots =
            split ? resident_workgroups<bwd_dkdv_bf16_kernel<D, BLK, PAT, MODE, PAT == FIXED>>(DkvCfg<D, BLK, PAT>::NT)
                  : resident_workgroups<bwd_dkdv_bf16_kernel<D, BLK, PAT, MODE, false>>(DkvCfg<D, BLK, PAT>::NT);
        // A band walk of long columns, and a dense walk (the residue classes)
        // of at least 8 blocks, take one workgroup per column instead of the
        // persistent grid: the hardware then overlaps one column's register
        // loads with the others' steps (n = 1,048,576: the band's 17-block
        // columns, backward 8.71 -> 8.53 ms; the classes' 16 blocks, 8.39 ->
        // 8.28 ms; with 3-block band columns, at n = 12,288, the persistent
        // grid stays 2% faster).  Under CLAIM_XCD_SERPENTINE such a grid is
        // the first round alone: the columns of a class unit take consecutive
        // places on one XCD.
        const bool per_column = (a.walk == WALK_BAND && a.l / BLK + 1 >= 8) || (a.walk == WALK_DENSE && a.nq >= 8);
        const unsigned qgrid = (unsigned)(slots > 0 && slots < items && !per_column
                                              ? slots
                                              : (items < (1ll << 31) ? items : (1ll << 31) - 1));
        // order of the dK / dV work (see the kernel): head by head on each XCD
        // for a walk of every block (the residue classes); a fixed order where
        // column lengths change smoothly (strided: a band and a stride's worth
        // of rows per column) or columns are a few blocks long; serpentine per
        // head where long summary columns alternate with short ones (fixed) and
        // each head has a few workgroups; the queues otherwise
        const int64_t bh_count = (int64_t)a.batch * a.heads;
        ak.claim_mode = a.walk == WALK_DENSE && qgrid % kQueues == 0 && bh_count % kQueues == 0
                            ? CLAIM_XCD_SERPENTINE
                        : (PAT == STRIDED || a.nq <= 8)
                            ? CLAIM_ROUND_ROBIN
                            : (bh_count * 4 <= (int64_t)qgrid ? CLAIM_SERPENTINE : CLAIM_QUEUES);
        // Summary halves in pairs (fixed, B = 64, l a multiple of 64: n / l of
        // them per (batch, head)) only where each workgroup of a head gets at
        // least 2.5 of them on average: a pair's column takes one workgroup
        // about 1.45 times as long as a single half's, so with fewer the
        // longest pair sets the kernel's time (fixed, n = 12,288, l = 128,
        // 16 heads: 7% slower), with more the saved staging and steps win
        // (n = 65,536, l = 256, 8 heads: 3% faster).
        const int64_t per_head = (int64_t)qgrid / bh_count;
        ak.pairs = PAT == FIXED && BLK == 64 && a.l % 64 == 0 && 2 * ((int64_t)a.n / a.l) >= 5 * per_head;
        // The row statistics go into the dQ kernel when both are asked for and
        // its grid (every row) holds a workgroup per layout for the schedule.
        AttnArgs aq = ak;
        aq.row_stats = (parts & BWD_PRE) && (parts & BWD_DQ) &&
                       (int64_t)a.heads * a.nq * a.batch >= layout_count(a.mode, a.sub);
        if ((parts & BWD_PRE) && !aq.row_stats)
            hipLaunchKernelGGL((bwd_pre_kernel<D, uint16_t>), dim3((unsigned)pre_groups), dim3(256), 0, stream, ak,
                               (const uint16_t*)o, (const uint16_t*)dout, lse, ndelta, nlse2, ws.queue, ws.items,
                               ws.order);
        if (parts & BWD_DQ) (void)with_full_body<PAT>(a, [&](auto fb) {
            auto dq_kernel = [&](auto sp) {
                hipLaunchKernelGGL((bwd_dq_bf16_kernel<D, BLK, PAT, MODE, decltype(fb)::value, decltype(sp)::value>),
                                   grid, dim3(DqCfg<D, BLK, PAT>::NT), 0, stream, aq, a.row_ptr, a.col_idx,
                                   (const uint16_t*)q, (const uint16_t*)k, (const uint16_t*)v, (const uint16_t*)dout,
                                   nlse2, ndelta, (uint16_t*)dq, (const uint16_t*)o, lse, ws.queue, ws.items,
                                   ws.order);
            };
            if constexpr (PAT == FIXED) {
                if (split) dq_kernel(std::true_type{});
                else dq_kernel(std::false_type{});
            } else {
                dq_kernel(std::false_type{});
            }
            return hipSuccess;
        });
        auto dkdv = [&](auto sp) {
            hipLaunchKernelGGL((bwd_dkdv_bf16_kernel<D, BLK, PAT, MODE, decltype(sp)::value>), dim3(qgrid),
                               dim3(DkvCfg<D, BLK, PAT>::NT), 0, stream, ak, a.col_ptr, a.row_idx, (const uint16_t*)q,
                               (const uint16_t*)k, (const uint16_t*)v, (const uint16_t*)dout, nlse2, ndelta,
                               (uint16_t*)dk, (uint16_t*)dv, ws.queue, ws.items, ws.order);
        };
        if (!(parts & BWD_DKDV)) {
        } else if constexpr (PAT == FIXED) {
            if (split) dkdv(std::true_type{});
            else dkdv(std::false_type{});
        } else {
            dkdv(std::false_type{});
        }
        return hipGetLastError();
    });
}

// ---------------------------------------------------------------------------
// bf16, matrix cores: the whole backward of one short residue class
// ---------------------------------------------------------------------------
// In the class view of a strided call each (batch x head, class) unit is
// dense causal attention over M positions with the causal limit moved back
// a.qshift steps.  Where M <= 128 (a multiple of 32), one workgroup of M / 16
// waves takes a unit whole: its Q, K, V, dO and row statistics go into LDS
// once, and
//   phase 1: wave w takes keys 16 w .. 16 w + 15 and walks the 32-query chunks
//     that attend them, forming S and dP once per pair: dV and dK accumulate
//     in registers, dS (bf16, the values the dK product takes) goes to LDS
//     transposed, dS^T[key][query];
//   phase 2: wave w takes queries 16 w .. 16 w + 15: dQ^T = K^T dS^T over the
//     keys they attend, both operands read back from LDS.
// The separate dQ and dK / dV kernels form S and dP twice and read the four
// tensors twice.  No atomics: every output row has one writer.
template <int D, int M>
struct ClassBwdCfg {
    static constexpr int NW = M / 16;       // waves
    static constexpr int NT = NW * 64;
    static constexpr int KS = D / 32;
    static constexpr int DB = D / 16;
    static constexpr int MP = M + 8;         // row stride of dS^T in LDS (elements, rows 16-byte aligned)
    static constexpr int MS = (M + 63) / 64 * 64;  // row statistics, whole 64-row loads
    static_assert(M % 32 == 0 && M <= 128, "classes of 32, 64, 96 or 128 positions");
};

template <int D, int M>
__global__ void __launch_bounds__((ClassBwdCfg<D, M>::NT))
bwd_class_bf16_kernel(AttnArgs a, const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                      const uint16_t* __restrict__ v, const uint16_t* __restrict__ dout,
                      const float* __restrict__ nlse2, const float* __restrict__ ndelta,
                      uint16_t* __restrict__ dq, uint16_t* __restrict__ dk, uint16_t* __restrict__ dv) {
    using C = ClassBwdCfg<D, M>;
    __shared__ __attribute__((aligned(16))) uint16_t sQ[M * D];
    __shared__ __attribute__((aligned(16))) uint16_t sK[M * D];
    __shared__ __attribute__((aligned(16))) uint16_t sV[M * D];
    __shared__ __attribute__((aligned(16))) uint16_t sO[M * D];       // dO
    __shared__ __attribute__((aligned(16))) uint16_t sST[M * C::MP];  // dS^T
    __shared__ __attribute__((aligned(16))) float sL[C::MS];          // -LSE log2 e
    __shared__ __attribute__((aligned(16))) float sD[C::MS];          // -D

    const int h = blockIdx.x, b = blockIdx.z;  // class, batch x head
    const int tid = threadIdx.x, lane = tid % 64, g = lane / 16, r = lane % 16;
    const int w = __builtin_amdgcn_readfirstlane(tid / 64);
    const int64_t base = (int64_t)b * a.sb + (int64_t)h * a.sh;
    const int shift = a.qshift;
    const float c2 = a.scale_log2;

    // The unit's four tensors, M x D each in the swizzled tile layout, by
    // direct-to-LDS loads: wave w takes the 1 KiB windows w, w + NW, ...
    // (D / 32 per tensor); the launcher keeps (M - 1) ss + D inside 32-bit
    // byte offsets.  Waves 0 and 1 load the row statistics, 64 rows a load.
    constexpr int kWin = M * D / 512;
    static_assert(kWin % C::NW == 0, "every wave issues the same number of loads");
#pragma unroll
    for (int kk = 0; kk < kWin / C::NW; ++kk) {
        const int win = w + C::NW * kk;
        const int oe = 512 * win + 8 * lane;  // element offset of this lane's slot
        const int row = oe / D, chunk = ((oe % D) / 8) ^ Swz<D>::perm(row);
        const uint32_t off = (uint32_t)(((int64_t)row * a.ss + 8 * chunk) * 2);
        dma_b128(uniform_ptr(q + base), off, lds_addr(sQ) + 1024 * win);
        dma_b128(uniform_ptr(k + base), off, lds_addr(sK) + 1024 * win);
        dma_b128(uniform_ptr(v + base), off, lds_addr(sV) + 1024 * win);
        dma_b128(uniform_ptr(dout + base), off, lds_addr(sO) + 1024 * win);
    }
    if (64 * w < M) {
        const int m0 = 64 * w, nv = M - m0 < 64 ? M - m0 : 64;
        const int64_t st0 = stat_index(a, b, h, m0);
        load_row_stats_async(nlse2 + st0, nv, lds_addr(sL) + 4 * m0, lane, (uint32_t)a.lse_ss);
        load_row_stats_async(ndelta + st0, nv, lds_addr(sD) + 4 * m0, lane, (uint32_t)a.lse_ss);
    }
    // dS^T starts at zero: pairs no chunk visits stay zero for phase 2
    for (int i = tid; i < M * C::MP / 8; i += C::NT) reinterpret_cast<u32x4*>(sST)[i] = u32x4{0u, 0u, 0u, 0u};
    wait_loads_upto<0>();
    __syncthreads();

    TileReader<D> rd;
    rd.init(g, r);

    // phase 1: this lane's key j; S^T blocks s[t] = q_(16 qblk + 4 g + t) . k_j
    const int j = 16 * w + r;
    bf16x8 kf[C::KS], vf[C::KS];
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
        kf[ks] = rd.row(sK, 16 * w, ks);
        vf[ks] = rd.row(sV, 16 * w, ks);
    }
    f32x4 dvacc[C::DB], dkacc[C::DB];
#pragma unroll
    for (int db = 0; db < C::DB; ++db) {
        dvacc[db] = zero4();
        dkacc[db] = zero4();
    }
    // the first 32-query chunk holding a query i >= 16 w + shift (one that
    // attends a key of this wave)
    for (int qc = (16 * w + shift) / 32; qc < M / 32; ++qc) {
        f32x4 p[2], ds[2];
#pragma unroll
        for (int hq = 0; hq < 2; ++hq) {
            const int qblk = 2 * qc + hq;
            bf16x8 qa[C::KS], oa[C::KS];
#pragma unroll
            for (int ks = 0; ks < C::KS; ++ks) {
                qa[ks] = rd.row(sQ, 16 * qblk, ks);
                oa[ks] = rd.row(sO, 16 * qblk, ks);
            }
            f32x4 sacc = zero4(), dpacc = *reinterpret_cast<const f32x4*>(&sD[16 * qblk + 4 * g]);
#pragma unroll
            for (int ks = 0; ks < C::KS; ++ks) {
                sacc = mfma_16x16x32(qa[ks], kf[ks], sacc);
                dpacc = mfma_16x16x32(oa[ks], vf[ks], dpacc);
            }
            const f32x4 nl = *reinterpret_cast<const f32x4*>(&sL[16 * qblk + 4 * g]);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int i = 16 * qblk + 4 * g + t;  // query; pair (i, j) attended when j <= i - shift
                const float pv = j <= i - shift ? exp2_fast(fmaf(sacc[t], c2, nl[t])) : 0.f;
                p[hq][t] = pv;
                ds[hq][t] = pv * dpacc[t];
            }
        }
        const bf16x8 pb = pack_bf16x8(p[0], p[1]), sb = pack_bf16x8(ds[0], ds[1]);
        // transposed operands one d-block ahead of their products
        bf16x8 oT[2], qT[2];
        oT[0] = rd.tr(sO, 32 * qc, 32 * qc + 16, 0);
        qT[0] = rd.tr(sQ, 32 * qc, 32 * qc + 16, 0);
#pragma unroll
        for (int db = 0; db < C::DB; ++db) {
            if (db + 1 < C::DB) {
                oT[(db + 1) & 1] = rd.tr(sO, 32 * qc, 32 * qc + 16, db + 1);
                qT[(db + 1) & 1] = rd.tr(sQ, 32 * qc, 32 * qc + 16, db + 1);
            }
            dvacc[db] = mfma_16x16x32(oT[db & 1], pb, dvacc[db]);
            dkacc[db] = mfma_16x16x32(qT[db & 1], sb, dkacc[db]);
        }
        // dS^T row j, queries 32 qc + 16 hq + 4 g .. +3
        *reinterpret_cast<uint2*>(&sST[j * C::MP + 32 * qc + 4 * g]) = pack_bf16x4_bits(ds[0]);
        *reinterpret_cast<uint2*>(&sST[j * C::MP + 32 * qc + 16 + 4 * g]) = pack_bf16x4_bits(ds[1]);
    }
    // this lane holds dV^T / dK^T at d = 16 db + 4 g + t for key j
    {
        uint16_t* dvrow = dv + base + (int64_t)j * a.ss;
        uint16_t* dkrow = dk + base + (int64_t)j * a.ss;
#pragma unroll
        for (int db = 0; db < C::DB; ++db) {
            uint2* dvp = reinterpret_cast<uint2*>(dvrow + db * 16 + 4 * g);
            uint2* dkp = reinterpret_cast<uint2*>(dkrow + db * 16 + 4 * g);
            f32x4 xv = dvacc[db], xk = dkacc[db] * a.scale;
            if (a.epilogue == EPI_ADD) {
                xv += bf16x4_to_f32x4(*dvp);
                xk += bf16x4_to_f32x4(*dkp);
            }
            *dvp = pack_bf16x4_bits(xv);
            *dkp = pack_bf16x4_bits(xk);
        }
    }
    __syncthreads();  // dS^T complete

    // phase 2: queries q0 + r; dQ^T = K^T dS^T over the 32-key chunks up to the
    // last key the wave's queries attend (q0 + 15 - shift)
    const int q0 = 16 * w, last = q0 + 15 - shift;
    f32x4 dqacc[C::DB];
#pragma unroll
    for (int db = 0; db < C::DB; ++db) dqacc[db] = zero4();
    for (int kc = 0; last >= 0 && kc <= last / 32; ++kc) {
        // dS^T rows 32 kc + 4 g + u and 32 kc + 16 + 4 g + u of query column
        // q0 + r (transposing reads), the key order of rd.tr below
        const uint16_t* t = &sST[(32 * kc + 4 * g + r / 4) * C::MP + q0 + 4 * (r & 3)];
        const u32x2 lo = ld_tr16(t), hi = ld_tr16(t + 16 * C::MP);
        const bf16x8 dsb = __builtin_bit_cast(bf16x8, u32x4{lo.x, lo.y, hi.x, hi.y});
        bf16x8 kT[2];  // one d-block ahead of its product
        kT[0] = rd.tr(sK, 32 * kc, 32 * kc + 16, 0);
#pragma unroll
        for (int db = 0; db < C::DB; ++db) {
            if (db + 1 < C::DB) kT[(db + 1) & 1] = rd.tr(sK, 32 * kc, 32 * kc + 16, db + 1);
            dqacc[db] = mfma_16x16x32(kT[db & 1], dsb, dqacc[db]);
        }
    }
    uint16_t* drow = dq + base + (int64_t)(q0 + r) * a.ss;
#pragma unroll
    for (int db = 0; db < C::DB; ++db) {
        uint2* dst = reinterpret_cast<uint2*>(drow + db * 16 + 4 * g);
        f32x4 x = dqacc[db] * a.scale;
        if (a.epilogue == EPI_ADD) x += bf16x4_to_f32x4(*dst);
        *dst = pack_bf16x4_bits(x);
    }
}

// Whether a call's dQ and dK / dV can run as one bwd_class_bf16_kernel per
// unit: the class view (a dense walk of a strided A1 view) with M a multiple
// of 32 up to 128 whose tensors fit LDS, and row offsets inside 32 bits.
template <int D>
inline bool class_bwd_fits(const AttnArgs& a) {
    if (a.walk != WALK_DENSE || a.pattern != STRIDED || a.mode != MODE_A1) return false;
    const int M = a.n;
    if (M % 32 != 0 || M > 128 || (D == 128 && M > 96)) return false;  // 4 M D + M (M + 8) bf16 within 160 KiB
    return ((int64_t)(M - 1) * a.ss + D) * 2 < ((int64_t)1 << 32) && a.lse_ss * 64 < ((int64_t)1 << 30);
}

template <int D, int M>
hipError_t launch_class_bwd(const AttnArgs& a, const void* q, const void* k, const void* v, const void* dout,
                            void* dq, void* dk, void* dv, const BwdWorkspace& ws, hipStream_t stream) {
    hipLaunchKernelGGL((bwd_class_bf16_kernel<D, M>), dim3((unsigned)a.heads, 1, (unsigned)a.batch),
                       dim3(ClassBwdCfg<D, M>::NT), 0, stream, a, (const uint16_t*)q, (const uint16_t*)k,
                       (const uint16_t*)v, (const uint16_t*)dout, ws.nlse2, ws.ndelta, (uint16_t*)dq,
                       (uint16_t*)dk, (uint16_t*)dv);
    return hipGetLastError();
}

template <int D>
hipError_t launch_bwd_bf16_d(const AttnArgs& a, const void* q, const void* k, const void* v,
                             const void* o, const void* dout, const float* lse, void* dq,
                             void* dk, void* dv, const BwdWorkspace& ws, hipStream_t stream, int parts) {
    if ((parts & BWD_DQ) && (parts & BWD_DKDV) && class_bwd_fits<D>(a)) {
        hipError_t e = hipSuccess;
        if (parts & BWD_PRE)
            e = launch_bwd_bf16_d<D>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream, BWD_PRE);
        if (e != hipSuccess) return e;
        switch (a.n) {
        case 32: return launch_class_bwd<D, 32>(a, q, k, v, dout, dq, dk, dv, ws, stream);
        case 64: return launch_class_bwd<D, 64>(a, q, k, v, dout, dq, dk, dv, ws, stream);
        case 96: return launch_class_bwd<D, 96>(a, q, k, v, dout, dq, dk, dv, ws, stream);
        default:
            if constexpr (D != 128) return launch_class_bwd<D, 128>(a, q, k, v, dout, dq, dk, dv, ws, stream);
            return hipErrorInvalidValue;  // unreachable: class_bwd_fits keeps M <= 96 for D = 128
        }
    }
    switch (a.block) {
    case 16: return launch_bwd_bf16<D, 16>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream, parts);
    case 32: return launch_bwd_bf16<D, 32>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream, parts);
    default: return launch_bwd_bf16<D, 64>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream, parts);
    }
}

}  // namespace

}  // namespace sa
