// bf16 backward kernels (sa_bwd_kernels.h) instantiated for d = 64: one
// translation unit per head size, so that they compile in parallel.
#include "sa_bwd_kernels.h"

namespace sa {

hipError_t bwd_bf16_d64(const AttnArgs& a, const void* q, const void* k, const void* v, const void* o,
                        const void* dout, const float* lse, void* dq, void* dk, void* dv, const BwdWorkspace& ws,
                        hipStream_t stream, int parts) {
    return launch_bwd_bf16_d<64>(a, q, k, v, o, dout, lse, dq, dk, dv, ws, stream, parts);
}

}  // namespace sa
