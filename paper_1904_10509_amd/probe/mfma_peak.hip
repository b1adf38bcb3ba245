// Measurement probe for the benchmark (not part of the attention library):
// the achievable rate of the bf16 matrix cores and the shader clock while
// they run.  Every wave issues v_mfma_f32_16x16x32_bf16 (16 x 16 x 32, 16,384
// FLOP) on eight independent accumulators, nothing else in its loop; one wave
// reads the 64-bit shader-cycle counter (s_memtime) and the 100 MHz real-time
// counter (s_memrealtime) before and after its loop, so that cycles over time
// give the clock.  Built into libsa_probe.so; bench.py times the launch.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kChains = 8;

__global__ void __launch_bounds__(256) mfma_peak_kernel(int iters, float* __restrict__ sink,
                                                        unsigned long long* __restrict__ clocks) {
    const int tid = threadIdx.x;
    bf16x8 a, b;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        a[e] = (__bf16)(0.001f * (float)((tid + e) & 7));
        b[e] = (__bf16)(0.002f * (float)((tid * 3 + e) & 7));
    }
    f32x4 acc[kChains];
#pragma unroll
    for (int c = 0; c < kChains; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
    const bool timer = blockIdx.x == 0 && tid == 0;
    uint64_t t0 = 0, r0 = 0;
    if (timer) {
        t0 = __builtin_amdgcn_s_memtime();
        r0 = __builtin_amdgcn_s_memrealtime();
    }
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int c = 0; c < kChains; ++c) acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc[c], 0, 0, 0);
    }
    if (timer) {
        const uint64_t t1 = __builtin_amdgcn_s_memtime();
        const uint64_t r1 = __builtin_amdgcn_s_memrealtime();
        clocks[0] = t1 - t0;
        clocks[1] = r1 - r0;
    }
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < kChains; ++c) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
    sink[(int64_t)blockIdx.x * 256 + tid] = s;  // keeps the products live
}

extern "C" {

// FLOP of one launch: workgroups x 4 waves x iters x 8 chains x 16,384.
double sa_probe_mfma_flop(int workgroups, int iters) {
    return (double)workgroups * 4.0 * (double)iters * kChains * 16384.0;
}

// sink: workgroups * 256 floats; clocks: 2 values (shader cycles, 100 MHz ticks).
int sa_probe_mfma_launch(int workgroups, int iters, float* sink, unsigned long long* clocks, void* stream) {
    if (workgroups < 1 || iters < 1 || !sink || !clocks) return -1;
    hipLaunchKernelGGL(mfma_peak_kernel, dim3((unsigned)workgroups), dim3(256), 0, static_cast<hipStream_t>(stream),
                       iters, sink, clocks);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
