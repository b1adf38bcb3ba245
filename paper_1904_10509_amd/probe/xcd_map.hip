// Measurement probe for the benchmark (not part of the attention library):
// the XCD each workgroup of a grid runs on, read from the hardware register
// HW_REG_XCC_ID.  The attention kernels' work orders assume that the
// dispatcher hands workgroup L to XCD L mod 8 (consecutive workgroups go to
// the XCDs in turn); this records it.  Each workgroup does a little work so
// that the grid is spread as a real one is.  Built into libsa_probe.so.
#include <hip/hip_runtime.h>
#include <stdint.h>

__global__ void __launch_bounds__(256) xcd_map_kernel(uint32_t* __restrict__ xcd, float* __restrict__ sink,
                                                      int iters) {
    uint32_t id;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID, 0, 4)" : "=s"(id));
    float x = (float)threadIdx.x;
    for (int i = 0; i < iters; ++i) x = x * 1.0001f + 0.5f;
    if (threadIdx.x == 0) xcd[blockIdx.x] = id;
    sink[(int64_t)blockIdx.x * 256 + threadIdx.x] = x;
}

extern "C" {

// xcd: workgroups words; sink: workgroups * 256 floats.
int sa_probe_xcd_map_launch(int workgroups, uint32_t* xcd, float* sink, void* stream) {
    if (workgroups < 1 || !xcd || !sink) return -1;
    hipLaunchKernelGGL(xcd_map_kernel, dim3((unsigned)workgroups), dim3(256), 0, static_cast<hipStream_t>(stream),
                       xcd, sink, 2000);
    return hipGetLastError() == hipSuccess ? 0 : -4;
}

}  // extern "C"
