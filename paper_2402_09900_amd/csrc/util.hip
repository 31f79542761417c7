// util.hip -- workspace initialisation.
#include "scan_common.hpp"
#include "kernels.hpp"

namespace memoroid {

__global__ __launch_bounds__(256) void ws_init_kernel(u32x4* zero, int64_t z16, u32x4* ones, int64_t o16) {
    const u32x4 z = {0u, 0u, 0u, 0u};
    const u32x4 o = {kEmpty32, kEmpty32, kEmpty32, kEmpty32};
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < z16 + o16; i += stride) {
        if (i < z16)
            zero[i] = z;
        else
            ones[i - z16] = o;
    }
}

hipError_t ws_init_launch(void* zero, size_t zero_bytes, void* ones, size_t ones_bytes, hipStream_t s) {
    const int64_t z16 = (int64_t)(zero_bytes / 16), o16 = (int64_t)(ones_bytes / 16);
    int64_t blocks = (z16 + o16 + 255) / 256;
    if (blocks < 1) blocks = 1;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(ws_init_kernel, dim3((unsigned)blocks), dim3(256), 0, s, (u32x4*)zero, z16, (u32x4*)ones,
                       o16);
    return hipGetLastError();
}

// One int64 store: outputs that must be written even when there is no work
// (a fill kernel rather than a memset, so that the call can be captured).
__global__ void store_i64_kernel(int64_t* p, int64_t v) {
    if (threadIdx.x == 0) *p = v;
}

hipError_t store_i64_launch(int64_t* p, int64_t v, hipStream_t s) {
    hipLaunchKernelGGL(store_i64_kernel, dim3(1), dim3(64), 0, s, p, v);
    return hipGetLastError();
}

}  // namespace memoroid
