// linattn_common.hpp -- shared pieces of the linear-attention kernels: chunk
// and LDS geometry, phi, LDS staging of 64-row chunks, and 64x64x64
// contractions on v_mfma_f32_16x16x4_f32.
//
// In one MFMA the four k-slots take k = 16*slot + s, a permutation of the
// contraction index applied to both operands, so an operand stored with k
// contiguous is read with 16-byte LDS loads; one stored with k as its row
// index is read with 4-byte loads whose rows are rotated by 16 columns per 16
// rows, which spreads the four k-slots over different LDS banks.
#pragma once

#include "scan_common.hpp"
#include "kernels.hpp"

namespace memoroid {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kC = 64;                      // chunk length (steps) and head width
constexpr int kLD = 68;                     // LDS row stride in floats (16-byte aligned rows)
constexpr int kStateWords = kC * kC + kC;   // S^T (64x64) followed by z (64)

// phi(u) = 1 + ELU(u): u + 1 for u > 0, exp(u) otherwise.  exp uses the
// hardware base-2 exponential (relative error a few ulp, far inside the fp32
// tolerance of the readout).
__device__ __forceinline__ float phi(float u) { return u > 0.0f ? u + 1.0f : __expf(u); }

// column of element (row, col) in a rotated buffer
__device__ __forceinline__ int rot_col(int row, int col) { return (col + 16 * (row >> 4)) & (kC - 1); }

// Fetch one chunk of a [T][H][64] tensor into registers (4 float4 per
// thread, rows outside [lo, hi) as zeros) and write it to LDS later with
// store_rows; returns nonzero if a value is not finite.
__device__ __forceinline__ int fetch_rows(f32x4 (&v)[4], const float* src, int64_t t0, int64_t H, int64_t h, int lo,
                                          int hi) {
    int bad = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int f = threadIdx.x + 256 * u;
        const int row = f >> 4, c4 = (f & 15) * 4;
        v[u] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        if (row >= lo && row < hi) {
            v[u] = *(const f32x4*)(src + ((t0 + row) * H + h) * kC + c4);
            bad |= !(__builtin_isfinite(v[u].x) && __builtin_isfinite(v[u].y) && __builtin_isfinite(v[u].z) &&
                     __builtin_isfinite(v[u].w));
        }
    }
    return bad;
}

template <bool ROT>
__device__ __forceinline__ void store_rows(float* s, const f32x4 (&v)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int f = threadIdx.x + 256 * u;
        const int row = f >> 4, c4 = (f & 15) * 4;
        *(f32x4*)(s + row * kLD + (ROT ? rot_col(row, c4) : c4)) = v[u];
    }
}

// Stage one chunk (64 rows) of a [T][H][64] tensor into LDS, row-major,
// applying phi if requested; rows outside [lo, hi) are written as zeros (a
// select, so non-finite values in excluded rows never enter).  ROT rotates
// each row as rot_col does.  Returns nonzero if a staged value is not finite.
template <bool PHI, bool ROT>
__device__ __forceinline__ int stage(float* s, const float* src, int64_t t0, int64_t H, int64_t h, int lo, int hi) {
    int bad = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int f = threadIdx.x + 256 * u;   // float4 index within the 64x64 tile
        const int row = f >> 4, c4 = (f & 15) * 4;
        f32x4 v = {0.0f, 0.0f, 0.0f, 0.0f};
        if (row >= lo && row < hi) {
            v = *(const f32x4*)(src + ((t0 + row) * H + h) * kC + c4);
            if (PHI) {
                v.x = phi(v.x); v.y = phi(v.y); v.z = phi(v.z); v.w = phi(v.w);
            }
            bad |= !(__builtin_isfinite(v.x) && __builtin_isfinite(v.y) && __builtin_isfinite(v.z) &&
                     __builtin_isfinite(v.w));
        }
        *(f32x4*)(s + row * kLD + (ROT ? rot_col(row, c4) : c4)) = v;
    }
    return bad;
}

// acc += A * B for 64x64 LDS tiles.  Wave w computes rows 16w .. 16w+15; on
// return acc[jt][r] = C[16w + 4*(lane/16) + r][16*jt + lane%16].
//   A_ROWS: A[i][k] = sA[i*kLD + k]          else A[i][k] = sA[k*kLD + rot_col(k, i)]
//   B_ROWS: B[k][j] = sB[j*kLD + k]          else B[k][j] = sB[k*kLD + rot_col(k, j)]
template <bool A_ROWS, bool B_ROWS>
__device__ __forceinline__ void mfma_64x64x64(const float* sA, const float* sB, f32x4 acc[4]) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int i = 16 * w + (lane & 15), kk = (lane >> 4) * 16;
    float af[16];
    if constexpr (A_ROWS) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const f32x4 v = *(const f32x4*)(sA + i * kLD + kk + 4 * u);
            af[4 * u] = v.x; af[4 * u + 1] = v.y; af[4 * u + 2] = v.z; af[4 * u + 3] = v.w;
        }
    } else {
        const int c = rot_col(kk, i);            // (kk + s) >> 4 == kk >> 4 for s < 16
#pragma unroll
        for (int s = 0; s < 16; ++s) af[s] = sA[(kk + s) * kLD + c];
    }
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
        const int j = 16 * jt + (lane & 15);
        float bf[16];
        if constexpr (B_ROWS) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const f32x4 v = *(const f32x4*)(sB + j * kLD + kk + 4 * u);
                bf[4 * u] = v.x; bf[4 * u + 1] = v.y; bf[4 * u + 2] = v.z; bf[4 * u + 3] = v.w;
            }
        } else {
            const int c = rot_col(kk, j);
#pragma unroll
            for (int s = 0; s < 16; ++s) bf[s] = sB[(kk + s) * kLD + c];
        }
#pragma unroll
        for (int s = 0; s < 16; ++s) acc[jt] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[s], bf[s], acc[jt], 0, 0, 0);
    }
}

__device__ __forceinline__ bool is_begin(const uint8_t* st, int64_t t) { return t == 0 || st[t] != 0; }

// sum over the 16 lanes that share lane / 16
__device__ __forceinline__ float sum16(float v) {
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) v += __shfl_xor(v, off, 64);
    return v;
}

}  // namespace memoroid
