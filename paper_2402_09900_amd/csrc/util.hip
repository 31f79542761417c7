// util.hip -- workspace initialisation and the episode-index scan.
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

// ------------------------------------------------------------ episode index
// Three passes over the begin flags of each tape: count begins per block of
// kEpBlock steps, turn the counts into exclusive offsets per tape, and write
// every step's index.  Integer arithmetic only, so the result is exact.

constexpr int kEpPerThread = kEpBlock / 256;

__device__ __forceinline__ int ep_is_begin(const uint8_t* st, int64_t t) { return t == 0 || st[t] != 0; }

__global__ __launch_bounds__(256) void ep_count_kernel(const uint8_t* start, int32_t* counts, int64_t T,
                                                       int64_t nblk) {
    __shared__ int32_t red[256];
    const int64_t b = blockIdx.y, blk = blockIdx.x;
    const uint8_t* st = start + b * T;
    const int64_t t0 = blk * kEpBlock + (int64_t)threadIdx.x * kEpPerThread;
    int32_t c = 0;
    for (int i = 0; i < kEpPerThread; ++i) {
        const int64_t t = t0 + i;
        if (t < T) c += ep_is_begin(st, t);
    }
    red[threadIdx.x] = c;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) red[threadIdx.x] += red[threadIdx.x + off];
        __syncthreads();
    }
    if (threadIdx.x == 0) counts[b * nblk + blk] = red[0];
}

__global__ __launch_bounds__(256) void ep_offsets_kernel(int32_t* counts, int64_t B, int64_t nblk) {
    const int64_t b = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (b >= B) return;
    int32_t run = 0;
    for (int64_t i = 0; i < nblk; ++i) {
        const int32_t c = counts[b * nblk + i];
        counts[b * nblk + i] = run;
        run += c;
    }
}

__global__ __launch_bounds__(256) void ep_write_kernel(const uint8_t* start, const int32_t* offsets,
                                                       int32_t* idx, int64_t T, int64_t nblk) {
    __shared__ int32_t scan[2][256];
    const int64_t b = blockIdx.y, blk = blockIdx.x;
    const uint8_t* st = start + b * T;
    const int64_t t0 = blk * kEpBlock + (int64_t)threadIdx.x * kEpPerThread;
    int32_t c = 0;
    for (int i = 0; i < kEpPerThread; ++i) {
        const int64_t t = t0 + i;
        if (t < T) c += ep_is_begin(st, t);
    }
    // inclusive Hillis-Steele scan of the per-thread counts
    int cur = 0;
    scan[cur][threadIdx.x] = c;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
        const int32_t v = scan[cur][threadIdx.x] + ((int)threadIdx.x >= off ? scan[cur][threadIdx.x - off] : 0);
        scan[cur ^ 1][threadIdx.x] = v;
        cur ^= 1;
        __syncthreads();
    }
    int32_t run = offsets[b * nblk + blk] + scan[cur][threadIdx.x] - c - 1;
    for (int i = 0; i < kEpPerThread; ++i) {
        const int64_t t = t0 + i;
        if (t < T) {
            run += ep_is_begin(st, t);
            idx[b * T + t] = run;
        }
    }
}

hipError_t episode_idx_launch(const uint8_t* start, int32_t* idx, int64_t B, int64_t T, int32_t* counts,
                              hipStream_t s) {
    const int64_t nblk = (T + kEpBlock - 1) / kEpBlock;
    dim3 grid((unsigned)nblk, (unsigned)B);
    hipLaunchKernelGGL(ep_count_kernel, grid, dim3(256), 0, s, start, counts, T, nblk);
    hipLaunchKernelGGL(ep_offsets_kernel, dim3((unsigned)((B + 255) / 256)), dim3(256), 0, s, counts, B, nblk);
    hipLaunchKernelGGL(ep_write_kernel, grid, dim3(256), 0, s, start, (const int32_t*)counts, idx, T, nblk);
    return hipGetLastError();
}

}  // namespace memoroid
