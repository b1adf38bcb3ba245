// B x D bf16 tiles in LDS, filled straight from global memory.
//
// A tile is stored unpadded, row-major, with its 16-byte chunks permuted per
// row (chunk c of row R sits at position c ^ perm(R)).  The permutation puts
// the 16 rows that one 16-lane group reads at the same column into 16
// distinct 16-byte slots of every 256-byte bank window, for both the row
// reads (ds_read_b128) and the transposing reads (ds_read_b64_tr_b16).
//
// Filling uses global_load_lds_dwordx4: lane L of a wave writes bytes
// [16 L, 16 L + 16) of a 1 KiB LDS window, from any global address, without
// passing through registers.  So each lane fetches the global chunk that
// belongs at its slot.  The loads complete asynchronously; wait_tile_loads()
// waits for this wave's loads, after which a barrier publishes the tile.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sa_mfma.h"

namespace sa {

template <int D>
struct Swz {
    static constexpr int CPR = D / 8;                            // 16-byte chunks per row
    static constexpr int RPW = (2 * D >= 256) ? 1 : 256 / (2 * D);  // rows per 256-byte window
    __device__ static int perm(int row) { return (row / RPW) % CPR; }
    // element offset of (row, col); col .. col+7 must stay inside one 8-element chunk
    __device__ static int off(int row, int col) {
        return row * D + ((((col >> 3) ^ perm(row))) << 3) + (col & 7);
    }
};

// Issue the loads of rows [0, BLK) of a [., D] bf16 tensor whose row 0 is at
// `src` (row stride `ss` elements) into `tile`, spread over the NW waves.
template <int D, int BLK, int NW>
__device__ inline void load_tile_async(const uint16_t* src, int64_t ss, uint16_t* tile, int w, int lane) {
    constexpr int NB = BLK * D / 512;  // 1 KiB windows per tile
#pragma unroll
    for (int k = w; k < NB; k += NW) {
        const int oe = 512 * k + 8 * lane;  // element offset of this lane's slot
        const int row = oe / D, pos = (oe % D) / 8;
        const int chunk = pos ^ Swz<D>::perm(row);
        __builtin_amdgcn_global_load_lds(src + row * ss + 8 * chunk,
                                         (__attribute__((address_space(3))) void*)(tile + 512 * k), 16, 0,
                                         0);
    }
}

// 64 consecutive fp32 values (one per lane) into `dst`, by wave 0 only.
__device__ inline void load_row_stats_async(const float* src, int n_valid, float* dst, int w, int lane) {
    if (w == 0) {
        const int i = lane < n_valid ? lane : n_valid - 1;
        __builtin_amdgcn_global_load_lds(src + i, (__attribute__((address_space(3))) void*)dst, 4, 0, 0);
    }
}

// s_waitcnt vmcnt(0): this wave's outstanding global loads (including the
// ones that write LDS) have completed.
__device__ inline void wait_tile_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Transposed operand over 32 rows of column col0 + (lane % 16): the first
// four contraction items from rows row_lo .. row_lo+3, the last four from
// row_hi .. row_hi+3 (see ld_tr16).
template <int D>
__device__ inline bf16x8 ld_tr_swz(const uint16_t* tile, int row_lo, int row_hi, int col0, int r) {
    const int dr = r >> 2, dc = col0 + 4 * (r & 3);
    u32x2 lo = ld_tr16(tile + Swz<D>::off(row_lo + dr, dc));
    u32x2 hi = ld_tr16(tile + Swz<D>::off(row_hi + dr, dc));
    return __builtin_bit_cast(bf16x8, u32x4{lo.x, lo.y, hi.x, hi.y});
}

// Same for a 16-row tile: rows row_lo .. row_lo+3 only, upper half zero.
template <int D>
__device__ inline bf16x8 ld_tr_swz_half(const uint16_t* tile, int row_lo, int col0, int r) {
    u32x2 lo = ld_tr16(tile + Swz<D>::off(row_lo + (r >> 2), col0 + 4 * (r & 3)));
    return __builtin_bit_cast(bf16x8, u32x4{lo.x, lo.y, 0u, 0u});
}

// Row read: 8 consecutive elements of one row.
template <int D>
__device__ inline bf16x8 ld_row_swz(const uint16_t* tile, int row, int col) {
    return ld_bf16x8(tile + Swz<D>::off(row, col));
}

}  // namespace sa
