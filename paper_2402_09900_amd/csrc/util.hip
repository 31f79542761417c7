// util.hip -- workspace initialisation.
#include "scan_common.hpp"
#include "kernels.hpp"

namespace memoroid {

__global__ __launch_bounds__(256) void ws_init_kernel(uint32_t* hdr, u32x4* p, int64_t n16) {
    if (blockIdx.x == 0 && threadIdx.x < 64) hdr[threadIdx.x] = 0u;
    const u32x4 ones = {kEmpty32, kEmpty32, kEmpty32, kEmpty32};
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16; i += (int64_t)gridDim.x * 256)
        p[i] = ones;
}

hipError_t ws_init_launch(void* hdr, void* p, size_t bytes, hipStream_t s) {
    const int64_t n16 = (int64_t)(bytes / 16);
    int64_t blocks = (n16 + 255) / 256;
    if (blocks < 1) blocks = 1;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(ws_init_kernel, dim3((unsigned)blocks), dim3(256), 0, s, (uint32_t*)hdr,
                       (u32x4*)p, n16);
    return hipGetLastError();
}

}  // namespace memoroid
