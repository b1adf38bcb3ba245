// Measurement probe for the benchmark (not part of the attention library): a
// read of known size through the direct-to-LDS loads (global_load_lds_dwordx4)
// the attention kernels stage their tiles with, so that the HBM byte
// counters can be scaled for that kind of load as they are for ordinary
// loads by the copy calibration.  Every wave streams its own contiguous share
// of the source, 1 KiB (64 lanes x 16 bytes) a load into its own LDS window,
// and folds one word of each window into a checksum.  Built into
// libsa_probe.so.
#include <hip/hip_runtime.h>
#include <stdint.h>

__global__ void __launch_bounds__(256) dma_read_kernel(const uint8_t* __restrict__ src, int64_t kib_per_wave,
                                                       uint32_t* __restrict__ sink) {
    __shared__ __attribute__((aligned(16))) uint32_t win[4][256];  // 1 KiB per wave
    const int lane = threadIdx.x % 64;
    const int w = threadIdx.x / 64;
    const int64_t wave = (int64_t)blockIdx.x * 4 + w;
    const uint8_t* base = src + wave * kib_per_wave * 1024;
    const uint32_t lds = (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)&win[w][0];
    uint32_t acc = 0u;
    for (int64_t i = 0; i < kib_per_wave; ++i) {
        const uint8_t* p = base + i * 1024;
        const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)p);
        const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uintptr_t)p >> 32));
        const void* sp = (const void*)(uintptr_t)(((uint64_t)hi << 32) | lo);
        const uint32_t voff = 16u * (uint32_t)lane;
        const uint32_t m0 = __builtin_amdgcn_readfirstlane(lds);
        asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" : : "v"(voff), "s"(sp), "s"(m0) : "memory");
        asm volatile("s_waitcnt vmcnt(0)" : : : "memory");
        acc ^= win[w][lane * 4];
        __builtin_amdgcn_wave_barrier();  // every lane has read the window before the next load overwrites it
    }
    sink[wave * 64 + lane] = acc;
}

extern "C" {

// Reads workgroups x 4 waves x kib_per_wave KiB from src (that many bytes,
// contiguous); sink: workgroups x 256 words.
int sa_probe_dma_read_launch(int workgroups, int64_t kib_per_wave, const void* src, uint32_t* sink, void* stream) {
    if (workgroups < 1 || kib_per_wave < 1 || !src || !sink) return -1;
    hipLaunchKernelGGL(dma_read_kernel, dim3((unsigned)workgroups), dim3(256), 0, static_cast<hipStream_t>(stream),
                       (const uint8_t*)src, kib_per_wave, sink);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
