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

// Rows [lo, hi) of one chunk of a [T][H][64] tensor as a buffer resource
// based at row lo: a row outside the range has an offset past the end (rows
// below lo wrap to huge unsigned offsets), so the hardware reads it as zeros
// and no load needs a branch.  off(row, c4) is the byte offset.
struct ChunkRows {
    Rsrc r;
    uint32_t row_bytes;
    int lo;
    __device__ __forceinline__ uint32_t off(int row, int c4) const {
        return (uint32_t)(row - lo) * row_bytes + (uint32_t)c4 * 4u;
    }
    __device__ __forceinline__ f32x4 load(int row, int c4) const {
        const u32x4 w = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off(row, c4), 0, 0);
        return f32x4{__uint_as_float(w.x), __uint_as_float(w.y), __uint_as_float(w.z), __uint_as_float(w.w)};
    }
};
__device__ __forceinline__ ChunkRows chunk_rows(const float* src, int64_t t0, int64_t H, int64_t h, int lo, int hi) {
    const uint32_t rb = (uint32_t)(H * kC * 4);
    const int n = hi > lo ? hi - lo : 0;
    const int64_t bytes = n > 0 ? (int64_t)(n - 1) * rb + kC * 4 : 0;
    return ChunkRows{make_rsrc(src + ((t0 + lo) * H + h) * kC, bytes), rb, lo};
}

__device__ __forceinline__ bool finite4(f32x4 v) {
    return __builtin_isfinite(v.x) && __builtin_isfinite(v.y) && __builtin_isfinite(v.z) && __builtin_isfinite(v.w);
}

// Fetch one chunk of a [T][H][64] tensor into registers (4 float4 per
// thread, rows outside [lo, hi) as zeros) and write it to LDS later with
// store_rows; returns nonzero if a value is not finite.
__device__ __forceinline__ int fetch_rows(f32x4 (&v)[4], const float* src, int64_t t0, int64_t H, int64_t h, int lo,
                                          int hi) {
    const ChunkRows cr = chunk_rows(src, t0, H, h, lo, hi);
    int bad = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int f = threadIdx.x + 256 * u;
        v[u] = cr.load(f >> 4, (f & 15) * 4);
        bad |= !finite4(v[u]);
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
    const ChunkRows cr = chunk_rows(src, t0, H, h, lo, hi);
    f32x4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int f = threadIdx.x + 256 * u;   // float4 index within the 64x64 tile
        v[u] = cr.load(f >> 4, (f & 15) * 4);
    }
    int bad = 0;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int f = threadIdx.x + 256 * u;
        const int row = f >> 4, c4 = (f & 15) * 4;
        if (PHI) {
            // phi(0) = 1: rows outside the range are selected back to zeros
            const bool in = row >= lo && row < hi;
            v[u].x = in ? phi(v[u].x) : 0.0f;
            v[u].y = in ? phi(v[u].y) : 0.0f;
            v[u].z = in ? phi(v[u].z) : 0.0f;
            v[u].w = in ? phi(v[u].w) : 0.0f;
        }
        bad |= !finite4(v[u]);
        *(f32x4*)(s + row * kLD + (ROT ? rot_col(row, c4) : c4)) = v[u];
    }
    return bad;
}

// acc += A * B for 64x64 LDS tiles.  The wavefront computes rows 16w .. 16w+15
// of C, w = rb if given (else the wavefront's index in the workgroup); on
// return acc[jt][r] = C[16w + 4*(lane/16) + r][16*jt + lane%16].
//   A_ROWS: A[i][k] = sA[i*kLD + k]          else A[i][k] = sA[k*kLD + rot_col(k, i)]
//   B_ROWS: B[k][j] = sB[j*kLD + k]          else B[k][j] = sB[k*kLD + rot_col(k, j)]
// jt_last < 3 leaves the output column tiles past it untouched (a wave of a
// causally masked product skips the tiles above the diagonal).
template <bool A_ROWS, bool B_ROWS>
__device__ __forceinline__ void mfma_64x64x64(const float* sA, const float* sB, f32x4 acc[4], int jt_last = 3,
                                              int rb = -1) {
    const int lane = threadIdx.x & 63, w = rb >= 0 ? rb : (int)(threadIdx.x >> 6);
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
        if (jt > jt_last) break;
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

// acc += A * B for a lower-triangular A (A[i][k] = 0 for k > i), rows
// 16rb .. 16rb+15 of C as above; A row-major, B stored with k as its row
// index (rotated).  Here MFMA number 4q + r takes k = 16q + 4*(lane/16) + r in
// its four k-slots, so each k-block q holds whole columns of A and the blocks
// past the row block (all zeros in its rows) are skipped.  The A reads are
// 16-byte loads; for the B reads the four k-slots sit 4 rows apart, which the
// 68-float row stride already places in different LDS banks.
__device__ __forceinline__ void mfma_64x64x64_tril(const float* sA, const float* sB, f32x4 acc[4], int rb) {
    const int lane = threadIdx.x & 63;
    const int i = 16 * rb + (lane & 15), g = lane >> 4;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        if (q > rb) break;
        const f32x4 a4 = *(const f32x4*)(sA + i * kLD + 16 * q + 4 * g);
        const float af[4] = {a4.x, a4.y, a4.z, a4.w};
        float bf[4][4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int k = 16 * q + 4 * g + r;
#pragma unroll
            for (int jt = 0; jt < 4; ++jt) bf[r][jt] = sB[k * kLD + rot_col(k, 16 * jt + (lane & 15))];
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
#pragma unroll
            for (int jt = 0; jt < 4; ++jt) acc[jt] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[r], bf[r][jt], acc[jt], 0, 0, 0);
        }
    }
}

__device__ __forceinline__ bool is_begin(const uint8_t* st, int64_t t) { return t == 0 || st[t] != 0; }

// sum over the 16 lanes that share lane / 16, with DPP moves inside each
// 16-lane row: lane ^ 1, lane ^ 2 (quad permutations), then the mirror of
// each 8-lane half and of the row; every step adds two equal partial sums in
// either order, so all 16 lanes hold the bit-identical total
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float sum16(float v) {
    v += dpp_f32<0xB1>(v);     // quad_perm [1, 0, 3, 2]
    v += dpp_f32<0x4E>(v);     // quad_perm [2, 3, 0, 1]
    v += dpp_f32<0x141>(v);    // row_half_mirror
    v += dpp_f32<0x140>(v);    // row_mirror
    return v;
}

}  // namespace memoroid
