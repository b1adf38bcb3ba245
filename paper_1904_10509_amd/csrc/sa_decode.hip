// One decoding step: the output of a single query position pos attending S_pos
// (Sec. 4.3) over a key / value cache, for every (batch, head).  Autoregressive
// sampling (Fig. 1, Sec. 5.6) runs one such step per generated position.
//
// The work is a gather and two dot products per key, so it is bound by reading
// the K and V rows of S_pos from HBM; there is no matrix product to put on the
// matrix cores.  Split-key (two kernels, no atomics):
//   1. split: S_pos, as the index space of DecodeSet, is cut into `splits`
//      contiguous ranges per (batch, head); a workgroup walks one range with
//      D/8 lanes per key (16-byte loads of 8 elements per lane, whole rows per
//      group of lanes), keeps a running max / sum / weighted V sum per key
//      slot in fp32, and merges them into one partial state;
//   2. combine: per (batch, head) the partial states are merged into o and
//      LSE.
// Scores are kept in base-2 units (q pre-scaled by scale * log2 e).
#include <math.h>

#include "sa_internal.h"
#include "sa_mfma.h"
#include "sa_pattern.h"

namespace sa {

namespace {

constexpr int kDecodeThreads = 256;  // four waves
constexpr int kKeysPerSplit = 256;    // target keys per workgroup
constexpr int kMaxWorkgroups = 4096;  // splits are capped at this over all (batch, head)

struct DecodeArgs {
    int pattern, mode, heads, splits;
    int32_t sub;  // summary subblocks (0: one window for all heads)
    int32_t pos, l, c;
    DivL dc;
    int64_t qsb, qsh;        // q and o strides
    int64_t ksb, ksh, kss;   // cache strides
    float scale_log2;
};

// 8 consecutive elements as fp32 (16-byte aligned source).
__device__ inline void load8(const uint16_t* p, float* x) {
    const u32x4 u = *reinterpret_cast<const u32x4*>(p);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        x[2 * e] = __uint_as_float(u[e] << 16);
        x[2 * e + 1] = __uint_as_float(u[e] & 0xffff0000u);
    }
}
__device__ inline void load8(const float* p, float* x) {
    const f32x4 a = *reinterpret_cast<const f32x4*>(p);
    const f32x4 b = *reinterpret_cast<const f32x4*>(p + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        x[e] = a[e];
        x[4 + e] = b[e];
    }
}

// The same for the K / V cache rows, with non-temporal loads: a step reads each
// row once, and marked so the rows do not displace other lines in the caches
// (fixed n = 65,536, 32 sequences: 108 -> 95 us per step).
__device__ inline void load8_once(const uint16_t* p, float* x) {
    const u32x4 u = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        x[2 * e] = __uint_as_float(u[e] << 16);
        x[2 * e + 1] = __uint_as_float(u[e] & 0xffff0000u);
    }
}
__device__ inline void load8_once(const float* p, float* x) {
    const f32x4 a = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
    const f32x4 b = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p + 4));
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        x[e] = a[e];
        x[4 + e] = b[e];
    }
}

// Merge softmax state (m2, l2, acc2) into (m, l, acc); m = -inf is the empty state.
template <int N>
__device__ inline void merge_state(float& m, float& l, float* acc, float m2, float l2, const float* acc2) {
    const float mx = fmaxf(m, m2);
    const float a1 = m == -INFINITY ? 0.f : exp2_fast(m - mx);
    const float a2 = m2 == -INFINITY ? 0.f : exp2_fast(m2 - mx);
    l = l * a1 + l2 * a2;
#pragma unroll
    for (int e = 0; e < N; ++e) acc[e] = acc[e] * a1 + acc2[e] * a2;
    m = mx;
}

// part: [batch * heads][splits][D + 2] fp32: D weighted V sums, running max, sum
template <int D, typename T>
__global__ void __launch_bounds__(kDecodeThreads)
decode_split_kernel(DecodeArgs a, const T* __restrict__ q, const T* __restrict__ kc, const T* __restrict__ vc,
                    float* __restrict__ part) {
    constexpr int LPK = D / 8;     // lanes per key
    constexpr int KPW = 64 / LPK;  // keys per wave per pass
    constexpr int NWV = kDecodeThreads / 64;
    __shared__ float s_m[NWV], s_l[NWV];
    __shared__ float s_acc[NWV][D];

    const int split = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int tid = threadIdx.x, lane = tid % 64, w = tid / 64;
    const int slot = lane / LPK, ds = lane % LPK;  // key slot of the lane; its elements are 8 ds .. 8 ds + 7
    const DecodeSet S(a.pattern, part_of_head(a.mode, h), a.pos, a.l, a.c,
                      (int32_t)summary_start(a.l, a.c, subblock_of_head(a.sub, h)), a.dc);
    const int64_t per = (S.count + a.splits - 1) / a.splits;
    const int64_t t0 = (int64_t)split * per < S.count ? (int64_t)split * per : S.count;
    const int64_t t1 = t0 + per < S.count ? t0 + per : S.count;

    float qv[8];
    load8(q + b * a.qsb + h * a.qsh + 8 * ds, qv);
#pragma unroll
    for (int e = 0; e < 8; ++e) qv[e] *= a.scale_log2;
    const int64_t cbase = (int64_t)b * a.ksb + (int64_t)h * a.ksh + 8 * ds;

    float m = -INFINITY, lsum = 0.f, acc[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] = 0.f;
    // the loop bound is the same for the whole wave, so every shuffle runs with
    // all lanes active; lanes past the range contribute nothing
    for (int64_t first = t0 + (int64_t)w * KPW; first < t1; first += (int64_t)NWV * KPW) {
        const int64_t t = first + slot;
        const bool valid = t < t1;
        float kx[8], vx[8];
        float s = 0.f;
        if (valid) {
            const int64_t row = (int64_t)S.at(t) * a.kss;
            load8_once(kc + cbase + row, kx);
            load8_once(vc + cbase + row, vx);
#pragma unroll
            for (int e = 0; e < 8; ++e) s = fmaf(qv[e], kx[e], s);
        }
#pragma unroll
        for (int off = 1; off < LPK; off <<= 1) s += __shfl_xor(s, off);
        if (valid) {
            const float mx = fmaxf(m, s);
            const float alpha = exp2_fast(m - mx);  // 0 while m = -inf
            const float p = exp2_fast(s - mx);
            lsum = fmaf(lsum, alpha, p);
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] = fmaf(acc[e], alpha, p * vx[e]);
            m = mx;
        }
    }
    // merge the key slots of the wave (lanes with the same d slice)
#pragma unroll
    for (int off = LPK; off < 64; off <<= 1) {
        float acc2[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc2[e] = __shfl_xor(acc[e], off);
        const float m2 = __shfl_xor(m, off), l2 = __shfl_xor(lsum, off);
        merge_state<8>(m, lsum, acc, m2, l2, acc2);
    }
    if (slot == 0) {
#pragma unroll
        for (int e = 0; e < 8; ++e) s_acc[w][8 * ds + e] = acc[e];
        if (ds == 0) {
            s_m[w] = m;
            s_l[w] = lsum;
        }
    }
    __syncthreads();
    // merge the waves: thread d owns element d of the output state
    if (tid < D) {
        float mm = -INFINITY, ll = 0.f, x = 0.f;
#pragma unroll
        for (int v = 0; v < NWV; ++v) {
            float xv = s_acc[v][tid];
            merge_state<1>(mm, ll, &x, s_m[v], s_l[v], &xv);
        }
        float* dst = part + (((int64_t)b * a.heads + h) * a.splits + split) * (D + 2);
        dst[tid] = x;
        if (tid == 0) {
            dst[D] = mm;
            dst[D + 1] = ll;
        }
    }
}

template <int D, typename T>
__global__ void __launch_bounds__(128)
decode_combine_kernel(DecodeArgs a, const float* __restrict__ part, T* __restrict__ o, float* __restrict__ lse) {
    const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
    const float* src = part + ((int64_t)b * a.heads + h) * a.splits * (D + 2);
    float m = -INFINITY, l = 0.f, x = 0.f;
    for (int s = 0; s < a.splits; ++s) {
        const float* p = src + (int64_t)s * (D + 2);
        float xv = tid < D ? p[tid] : 0.f;
        merge_state<1>(m, l, &x, p[D], p[D + 1], &xv);
    }
    const float inv = l > 0.f ? 1.f / l : 0.f;  // an empty set gives o = 0
    if (tid < D) {
        const float val = x * inv;
        T* dst = o + b * a.qsb + h * a.qsh + tid;
        if constexpr (sizeof(T) == 2) {
            const __bf16 bv = (__bf16)val;
            *reinterpret_cast<__bf16*>(dst) = bv;
        } else {
            *dst = val;
        }
    }
    if (tid == 0) lse[(int64_t)b * a.heads + h] = l > 0.f ? (m + __log2f(l)) / kLog2e : -INFINITY;
}

template <int D, typename T>
hipError_t launch(const DecodeArgs& a, int batch, const void* q, const void* k, const void* v, void* o,
                  float* lse, float* part, hipStream_t stream) {
    hipLaunchKernelGGL((decode_split_kernel<D, T>), dim3((unsigned)a.splits, (unsigned)a.heads, (unsigned)batch),
                       dim3(kDecodeThreads), 0, stream, a, (const T*)q, (const T*)k, (const T*)v, part);
    hipLaunchKernelGGL((decode_combine_kernel<D, T>), dim3((unsigned)a.heads, (unsigned)batch), dim3(128), 0,
                       stream, a, (const float*)part, (T*)o, lse);
    return hipGetLastError();
}

}  // namespace

// Ranges per (batch, head): about kKeysPerSplit keys each (for the largest
// set of a head), at most kMaxWorkgroups workgroups in all (and at least one
// range).
int decode_splits(int pattern, int mode, int32_t sub, int32_t pos, int32_t l, int32_t c, int64_t batch,
                  int64_t heads) {
    const DivL dc = make_divl(c > 0 ? c : 1);
    int64_t count = 0;
    const int sets = layout_count(mode, sub);
    for (int g = 0; g < sets; ++g) {
        const int32_t w = (int32_t)summary_start(l, c, subblock_of_layout(mode, sub, g));
        const DecodeSet S(pattern, part_of_layout(mode, g), pos, l, c, w, dc);
        count = S.count > count ? S.count : count;
    }
    int64_t splits = (count + kKeysPerSplit - 1) / kKeysPerSplit;
    const int64_t cap = kMaxWorkgroups / (batch * heads);
    if (splits > cap) splits = cap;
    if (splits < 1) splits = 1;
    return (int)splits;
}

size_t decode_workspace_bytes(int pattern, int mode, int32_t sub, int32_t pos, int32_t l, int32_t c,
                              int64_t batch, int64_t heads, int d) {
    return (size_t)batch * heads * decode_splits(pattern, mode, sub, pos, l, c, batch, heads) * (d + 2) *
           sizeof(float);
}

hipError_t decode_launch(int pattern, int mode, int32_t sub, int32_t pos, int32_t l, int32_t c, int batch, int heads,
                         int d, int dtype, const void* q, const int64_t* q_strides, const void* k, const void* v,
                         const int64_t* kv_strides, float scale, void* o, float* lse, void* workspace,
                         hipStream_t stream) {
    DecodeArgs a;
    a.pattern = pattern;
    a.mode = mode;
    a.heads = heads;
    a.sub = sub;
    a.splits = decode_splits(pattern, mode, sub, pos, l, c, batch, heads);
    a.pos = pos;
    a.l = l;
    a.c = c;
    a.dc = make_divl(c > 0 ? c : 1);
    a.qsb = q_strides[0];
    a.qsh = q_strides[1];
    a.ksb = kv_strides[0];
    a.ksh = kv_strides[1];
    a.kss = kv_strides[2];
    a.scale_log2 = scale * kLog2eHost;
    float* part = static_cast<float*>(workspace);
    if (dtype == 1) {
        switch (d) {
        case 32: return launch<32, uint16_t>(a, batch, q, k, v, o, lse, part, stream);
        case 64: return launch<64, uint16_t>(a, batch, q, k, v, o, lse, part, stream);
        default: return launch<128, uint16_t>(a, batch, q, k, v, o, lse, part, stream);
        }
    }
    switch (d) {
    case 32: return launch<32, float>(a, batch, q, k, v, o, lse, part, stream);
    case 64: return launch<64, float>(a, batch, q, k, v, o, lse, part, stream);
    default: return launch<128, float>(a, batch, q, k, v, o, lse, part, stream);
    }
}

}  // namespace sa
