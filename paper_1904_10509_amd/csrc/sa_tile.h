// B x D bf16 tiles in LDS, filled straight from global memory.
//
// A tile is stored unpadded, row-major, with its 16-byte chunks permuted per
// row (chunk c of row R sits at position c ^ perm(R)).  perm is a linear map
// over GF(2) of the low four bits of R, chosen (by exhaustive search over
// such maps) so that no two lanes served together touch one bank twice, for
// the row reads (ds_read_b128: 16 rows at one 16-byte column, taken 8 or 16
// lanes at a time) and for the transposing reads (ds_read_b64_tr_b16: four
// rows of 32 bytes per 16 lanes, taken 16 or 32 lanes at a time), whether a
// cycle serves 128 or 256 bytes.  The plain forms perm(R) = R / rows-per-256
// bytes left the transposing reads two-way conflicted.  perm depending on
// R mod 16 alone keeps it unchanged under row offsets that are multiples of
// 16, which the readers below rely on.
//
// Filling uses global_load_lds_dwordx4: lane L of a wave writes bytes
// [16 L, 16 L + 16) of a 1 KiB LDS window (base in M0), from any global
// address, without passing through registers.  So each lane fetches the
// global chunk that belongs at its slot.  The loads complete asynchronously
// and in issue order; wait_loads_upto<N>() waits until at most N of this
// wave's loads are outstanding, after which a barrier publishes the tile.
//
// The loads are issued from inline assembly on purpose: the compiler then
// does not track them, and so does not put a full wait before every LDS
// read (it cannot tell which ring stage a read touches).  Every read of a
// stage sits behind an explicit wait and a workgroup barrier instead.  A
// compiler-issued wait for its own loads stays correct with these extra
// loads outstanding, since waits count completed loads in issue order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "sa_mfma.h"

namespace sa {

template <int D>
struct Swz {
    static constexpr int CPR = D / 8;  // 16-byte chunks per row
    static_assert(D == 32 || D == 64 || D == 128, "head sizes 32, 64, 128");
    __device__ static int perm(int row) {
        const int b0 = row & 1, b1 = (row >> 1) & 1, b2 = (row >> 2) & 1, b3 = (row >> 3) & 1;
        if constexpr (D == 32) return b2 | ((b1 ^ b2 ^ b3) << 1);
        else if constexpr (D == 64) return b2 | (b1 << 1) | ((b0 ^ b2 ^ b3) << 2);
        else return b2 | (b1 << 1) | (b0 << 2) | ((b2 ^ b3) << 3);
    }
    // element offset of (row, col); col .. col+7 must stay inside one 8-element chunk
    __device__ static int off(int row, int col) {
        return row * D + ((((col >> 3) ^ perm(row))) << 3) + (col & 7);
    }
};

// LDS byte address of a pointer into a __shared__ array, made wave-uniform.
// Ring stages are addressed as this base plus a stage offset: selecting
// between generic pointers to different stages would make the compiler test
// the pointer against the LDS aperture.
__device__ inline uint32_t lds_addr(const void* p) {
    const uint32_t a = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
    return __builtin_amdgcn_readfirstlane(a);
}

// A wave-uniform global pointer, kept in scalar registers.
__device__ inline const void* uniform_ptr(const void* p) {
    const uint64_t v = (uint64_t)(uintptr_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
    return (const void*)(uintptr_t)(((uint64_t)hi << 32) | lo);
}

// One direct-to-LDS load per lane: 16 (or 4) bytes from sbase + voff (sbase
// wave-uniform, voff a 32-bit byte offset) into the LDS window lds_window.
__device__ inline void dma_b128(const void* sbase, uint32_t voff, uint32_t lds_window) {
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" : : "v"(voff), "s"(sbase), "s"(lds_window)
                 : "memory");
}

__device__ inline void dma_b32(const void* sbase, uint32_t voff, uint32_t lds_window) {
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1" : : "v"(voff), "s"(sbase), "s"(lds_window)
                 : "memory");
}

// Issues the direct-to-LDS loads of one BLK x D tile (rows 0..BLK-1 at row
// stride ss elements) spread over NW waves.  Each lane's byte offsets inside
// the tile are the same for every tile and computed once.
template <int D, int BLK, int NW>
struct TileLoader {
    static constexpr int NB = BLK * D / 512;  // 1 KiB windows per tile
    static constexpr int PER = NB / NW;       // windows per wave
    static_assert(NB % NW == 0, "every wave issues the same number of loads");
    uint32_t off[PER];
    int w;

    __device__ void init(int64_t ss, int wave, int lane) {
        w = wave;
#pragma unroll
        for (int kk = 0; kk < PER; ++kk) {
            const int k = w + NW * kk;
            const int oe = 512 * k + 8 * lane;  // element offset of this lane's slot
            const int row = oe / D, pos = (oe % D) / 8;
            const int chunk = pos ^ Swz<D>::perm(row);
            off[kk] = (uint32_t)((row * ss + 8 * chunk) * 2);
        }
    }
    // src: first element of the tile's row 0 (wave-uniform); base: LDS byte
    // address of the tile
    __device__ void issue(const uint16_t* src, uint32_t base) const {
        const void* s = uniform_ptr(src);
#pragma unroll
        for (int kk = 0; kk < PER; ++kk) dma_b128(s, off[kk], base + 1024 * (w + NW * kk));
    }
    // One tile made of two half tiles: rows 0 .. BLK/2-1 from src_lo and rows
    // BLK/2 .. BLK-1 from src_hi, each pointer being where tile row 0 would
    // sit (so tile row R reads row R past its pointer).  A 1 KiB window never
    // straddles the two halves.
    __device__ void issue_halves(const uint16_t* src_lo, const uint16_t* src_hi, uint32_t base) const {
        static_assert((NB / 2) * 512 == (BLK / 2) * D, "windows split at half the tile");
        const void* lo = uniform_ptr(src_lo);
        const void* hi = uniform_ptr(src_hi);
#pragma unroll
        for (int kk = 0; kk < PER; ++kk) {
            const int win = w + NW * kk;
            dma_b128(win < NB / 2 ? lo : hi, off[kk], base + 1024 * win);
        }
    }
};

// 64 fp32 values src[0], src[stride], ... (one per lane, lanes past n_valid
// repeat the last value) to LDS byte address dst: one direct-to-LDS load.
__device__ inline void load_row_stats_async(const float* src, int n_valid, uint32_t dst, int lane,
                                            uint32_t stride = 1) {
    const uint32_t i = (uint32_t)(lane < n_valid ? lane : n_valid - 1);
    dma_b32(uniform_ptr(src), 4u * i * stride, dst);
}

// s_waitcnt vmcnt(N): at most N of this wave's global loads (including the
// ones that write LDS) are still outstanding; loads complete in issue order.
template <int N>
__device__ inline void wait_loads_upto() {
    static_assert(N >= 0 && N < 64, "vmcnt field holds 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Per-lane byte offsets of the operand reads of a swizzled [., D] tile.
// Row block bases that are multiples of 16 leave the chunk permutation of
// a lane unchanged, so an address is one per-lane offset (chosen by the
// d-chunk) plus a constant: the tile's LDS address, its ring stage and the
// row block, all of which fit the immediate offset of the LDS read when the
// caller indexes the tile with compile-time constants.
template <int D>
struct TileReader {
    static constexpr int KS = D / 32;  // 32-wide d chunks (row reads)
    static constexpr int DB = D / 16;  // 16-wide d blocks (transposed reads)
    uint32_t row_off[KS];  // row r, elements 32 ks + 8 g .. +7
    uint32_t tr_off[DB];   // row 4 g + r / 4, elements 16 db + 4 (r % 4) .. +3

    __device__ void init(int g, int r) {
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) row_off[ks] = 2u * (uint32_t)Swz<D>::off(r, 32 * ks + 8 * g);
#pragma unroll
        for (int db = 0; db < DB; ++db) tr_off[db] = 2u * (uint32_t)Swz<D>::off(4 * g + r / 4, 16 * db + 4 * (r & 3));
    }
    // A / B operand: row row0 + r (row0 a multiple of 16), elements 32 ks + 8 g .. +7
    __device__ bf16x8 row(const uint16_t* tile, int row0, int ks) const {
        return ld_bf16x8(reinterpret_cast<const uint16_t*>(reinterpret_cast<const char*>(tile) + row_off[ks]) +
                         row0 * D);
    }
    // Transposed operand over the 32 rows lo .. lo+15 and hi .. hi+15
    // (multiples of 16) of column 16 db + r (see ld_tr16)
    __device__ bf16x8 tr(const uint16_t* tile, int lo, int hi, int db) const {
        const uint16_t* t = reinterpret_cast<const uint16_t*>(reinterpret_cast<const char*>(tile) + tr_off[db]);
        const u32x2 a = ld_tr16(t + lo * D);
        const u32x2 b = ld_tr16(t + hi * D);
        return __builtin_bit_cast(bf16x8, u32x4{a.x, a.y, b.x, b.y});
    }
    // Same over rows lo .. lo+15 only; the upper half of the operand is zero
    __device__ bf16x8 tr_half(const uint16_t* tile, int lo, int db) const {
        const uint16_t* t = reinterpret_cast<const uint16_t*>(reinterpret_cast<const char*>(tile) + tr_off[db]);
        const u32x2 a = ld_tr16(t + lo * D);
        return __builtin_bit_cast(bf16x8, u32x4{a.x, a.y, 0u, 0u});
    }
};

// Runs body(stage, i) for i = 0 .. count-1, stage = i mod 2 passed as a
// compile-time constant, so that ring-stage addresses are constants.
template <typename F>
__device__ inline void two_stage_loop(int count, F&& body) {
    for (int i = 0; i < count; i += 2) {
        body(std::integral_constant<int, 0>{}, i);
        if (i + 1 < count) body(std::integral_constant<int, 1>{}, i + 1);
    }
}

// The same for a loop whose trip count is found on the way: body(stage)
// returns false when there is no further step.
template <typename F>
__device__ inline void two_stage_while(F&& body) {
    while (body(std::integral_constant<int, 0>{}) && body(std::integral_constant<int, 1>{})) {
    }
}

}  // namespace sa
