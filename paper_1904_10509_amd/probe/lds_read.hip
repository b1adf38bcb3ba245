// Measurement probe for the benchmark (not part of the attention library):
// the LDS read rate per compute unit for the two read forms the attention
// kernels use: ds_read_b128 (16 bytes a lane, the row operands) and
// ds_read_b64_tr_b16 (8 bytes a lane, transposed, the operands whose
// contraction runs over a tile's rows).  Each 256-thread workgroup fills 16 KiB
// of LDS, small enough for eight workgroups (32 waves, the most a CU holds) to
// be resident, since with fewer waves the rate measured is their latency, not
// the LDS's; every lane issues 8 independent reads per iteration at
// consecutive, conflict-free 16-byte slots and folds them into a checksum; one
// wave reads the shader-cycle and real-time counters around its loop, as in
// the matrix-core probe.  Built into libsa_probe.so; bench.py times the launch.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

constexpr int kWords = 4096;  // 16 KiB of LDS per workgroup
constexpr int kReads = 8;      // independent reads per lane and iteration

template <int KIND>
__global__ void __launch_bounds__(256) lds_read_kernel(int iters, uint32_t* __restrict__ sink,
                                                       unsigned long long* __restrict__ clocks) {
    __shared__ __attribute__((aligned(16))) uint32_t buf[kWords];
    const int tid = threadIdx.x;
    for (int i = tid; i < kWords; i += 256) buf[i] = (uint32_t)i * 2654435761u;
    __syncthreads();
    uint32_t acc[kReads];
#pragma unroll
    for (int u = 0; u < kReads; ++u) acc[u] = 0u;
    const bool timer = blockIdx.x == 0 && tid == 0;
    uint64_t t0 = 0, r0 = 0;
    if (timer) {
        t0 = __builtin_amdgcn_s_memtime();
        r0 = __builtin_amdgcn_s_memrealtime();
    }
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int u = 0; u < kReads; ++u) {
            // 16-byte slot (tid + 256 u + 64 it) mod kWords / 4: a wave's lanes
            // take consecutive slots; the highest word read is kWords - 1
            const int slot = (tid + 256 * u + 64 * it) & (kWords / 4 - 1);
            if constexpr (KIND == 0) {
                const u32x4 x = *reinterpret_cast<const u32x4*>(&buf[4 * slot]);
                acc[u] ^= x[0] ^ x[1] ^ x[2] ^ x[3];
            } else {
                // 8 bytes at word 2 * slot (at most kWords / 2 - 1)
                const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                    (__attribute__((address_space(3))) s16x4*)(&buf[2 * slot]));
                acc[u] ^= (uint32_t)(uint16_t)v[0] ^ ((uint32_t)(uint16_t)v[1] << 16) ^ (uint32_t)(uint16_t)v[2] ^
                          ((uint32_t)(uint16_t)v[3] << 16);
            }
        }
    }
    if (timer) {
        const uint64_t t1 = __builtin_amdgcn_s_memtime();
        const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
        clocks[0] = t1 - t0;
        clocks[1] = r1 - r0;
    }
    uint32_t s = 0u;
#pragma unroll
    for (int u = 0; u < kReads; ++u) s ^= acc[u];
    sink[(int64_t)blockIdx.x * 256 + tid] = s;  // keeps the reads live
}

extern "C" {

// Bytes read from LDS by one launch: workgroups x 256 lanes x iters x 8 reads
// x (16 bytes for kind 0, ds_read_b128; 8 bytes for kind 1, ds_read_b64_tr_b16).
double sa_probe_lds_bytes(int kind, int workgroups, int iters) {
    return (double)workgroups * 256.0 * (double)iters * kReads * (kind == 0 ? 16.0 : 8.0);
}

// sink: workgroups * 256 words; clocks: 2 values (shader cycles, 100 MHz ticks).
int sa_probe_lds_launch(int kind, int workgroups, int iters, uint32_t* sink, unsigned long long* clocks,
                        void* stream) {
    if ((kind != 0 && kind != 1) || workgroups < 1 || iters < 1 || !sink || !clocks) return -1;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (kind == 0) hipLaunchKernelGGL(lds_read_kernel<0>, dim3((unsigned)workgroups), dim3(256), 0, s, iters, sink, clocks);
    else hipLaunchKernelGGL(lds_read_kernel<1>, dim3((unsigned)workgroups), dim3(256), 0, s, iters, sink, clocks);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
