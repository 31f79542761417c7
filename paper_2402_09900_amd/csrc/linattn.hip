// linattn.hip -- chunked kernels of the linear-transformer memoroid (App. G.1)
// over a tape with resets, for gfx950.
//
// The memoroid's monoid is a plain sum, (S, z) . (S', z') = (S + S', z + z'),
// of outer products phi(k) v^T and of phi(k); under the reset transform the
// state of step t sums only the steps of t's episode up to t.  Chunks of C = 64
// steps are processed as dense 64x64x64 contractions on the fp32 matrix cores:
//
//   summary kernel (one workgroup per chunk and head):
//     dS^T = V^T phi(K)  over the rows after the chunk's last begin step
//     dz   = column sums of those phi(K) rows;  R = "chunk holds a begin"
//   the chunk states are then scanned with the resettable diagonal scan
//   (a = 1: the sum monoid), giving S_inc(c) = state after chunk c;
//   output kernel (one workgroup per chunk and head), with r_i the last begin
//   step <= i inside the chunk (-1 if none):
//     A   = phi(Q) phi(K)^T,  masked to j <= i and j >= r_i
//     num = A V + [r_i < 0] phi(Q) S_inc(c-1),  den = rowsum(A) + [r_i < 0] phi(Q).z
//     out = num / den.
//
// Contractions use v_mfma_f32_16x16x4_f32.  Operands are staged in LDS with
// the contraction index contiguous, so one lane's 16 k-values of a fragment
// come from four 16-byte LDS reads; within one MFMA the four k-slots of the
// instruction take k = 16*slot + s, a permutation of the contraction index
// applied identically to both operands.
#include "scan_common.hpp"
#include "kernels.hpp"

namespace memoroid {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kC = 64;            // chunk length (steps) and head width
constexpr int kLD = 68;           // LDS row stride in floats (16-byte aligned rows)
constexpr int kStateWords = kC * kC + kC;   // S^T (64x64) followed by z (64)

__device__ __forceinline__ float phi(float u) { return u > 0.0f ? u + 1.0f : expf(u); }

// Stage rows [0, 64) of one chunk of a [T][H][64] tensor into LDS, applying
// phi if requested; rows outside [lo, hi) are written as zeros (a select, so
// non-finite values in excluded rows never enter).  TRANS stores element
// (row, col) at s[col * kLD + row], otherwise at s[row * kLD + col].
// Returns nonzero if a staged value is not finite.
template <bool PHI, bool TRANS>
__device__ __forceinline__ int stage(float* s, const float* src, int64_t t0, int64_t H, int64_t h,
                                     int lo, int hi) {
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
        if (TRANS) {
            s[(c4 + 0) * kLD + row] = v.x;
            s[(c4 + 1) * kLD + row] = v.y;
            s[(c4 + 2) * kLD + row] = v.z;
            s[(c4 + 3) * kLD + row] = v.w;
        } else {
            *(f32x4*)(s + row * kLD + c4) = v;
        }
    }
    return bad;
}

// C = A * Bt^T for 64x64 LDS tiles: A[i][k] = sA[i*kLD + k], Bt[j][k] =
// sBt[j*kLD + k].  Wave w computes rows 16w .. 16w+15; on return
// acc[jt][r] = C[16w + 4*(lane/16) + r][16*jt + lane%16].
__device__ __forceinline__ void mfma_64x64x64(const float* sA, const float* sBt, f32x4 acc[4]) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int i = 16 * w + (lane & 15), kk = (lane >> 4) * 16;
    float af[16];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const f32x4 v = *(const f32x4*)(sA + i * kLD + kk + 4 * u);
        af[4 * u] = v.x; af[4 * u + 1] = v.y; af[4 * u + 2] = v.z; af[4 * u + 3] = v.w;
    }
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
        const int j = 16 * jt + (lane & 15);
        float bf[16];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const f32x4 v = *(const f32x4*)(sBt + j * kLD + kk + 4 * u);
            bf[4 * u] = v.x; bf[4 * u + 1] = v.y; bf[4 * u + 2] = v.z; bf[4 * u + 3] = v.w;
        }
#pragma unroll
        for (int s = 0; s < 16; ++s) acc[jt] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[s], bf[s], acc[jt], 0, 0, 0);
    }
}

__device__ __forceinline__ bool is_begin(const uint8_t* st, int64_t t) { return t == 0 || st[t] != 0; }

// ---------------------------------------------------------------- summaries

__global__ __launch_bounds__(256) void linattn_summary_kernel(const float* __restrict__ k,
                                                              const float* __restrict__ v,
                                                              const uint8_t* __restrict__ start,
                                                              float* __restrict__ dS, uint8_t* __restrict__ R,
                                                              int64_t T, int64_t H) {
    __shared__ __attribute__((aligned(16))) float sKt[kC * kLD];
    __shared__ __attribute__((aligned(16))) float sVt[kC * kLD];
    __shared__ int s_last;
    const int64_t c = blockIdx.x, h = blockIdx.y;
    const int64_t t0 = c * kC;
    const int nvalid = (int)(T - t0 < kC ? T - t0 : kC);
    if (threadIdx.x == 0) s_last = -1;
    __syncthreads();
    if ((int)threadIdx.x < nvalid && is_begin(start, t0 + threadIdx.x)) atomicMax(&s_last, (int)threadIdx.x);
    __syncthreads();
    const int last = s_last;
    const int lo = last > 0 ? last : 0;
    stage<true, true>(sKt, k, t0, H, h, lo, nvalid);
    stage<false, true>(sVt, v, t0, H, h, lo, nvalid);
    __syncthreads();

    f32x4 acc[4];
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) acc[jt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    mfma_64x64x64(sVt, sKt, acc);   // C[n][kd] = sum_j V[j][n] phi(K)[j][kd] = dS^T

    float* out = dS + (c * H + h) * kStateWords;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int n = 16 * w + 4 * (lane >> 4) + r;
            const int kd = 16 * jt + (lane & 15);
            out[n * kC + kd] = acc[jt][r];
        }
    }
    if (threadIdx.x < kC) {
        float z = 0.0f;
        for (int j = 0; j < kC; ++j) z += sKt[threadIdx.x * kLD + j];
        out[kC * kC + threadIdx.x] = z;
    }
    if (h == 0 && threadIdx.x == 0) R[c] = last >= 0 ? 1 : 0;
}

// ------------------------------------------------------------------- output

__global__ __launch_bounds__(256) void linattn_output_kernel(const float* __restrict__ q,
                                                             const float* __restrict__ k,
                                                             const float* __restrict__ v,
                                                             const uint8_t* __restrict__ start,
                                                             const float* __restrict__ Sinc,
                                                             float* __restrict__ out, int64_t T, int64_t H) {
    __shared__ __attribute__((aligned(16))) float sQ[kC * kLD];   // phi(Q), later V^T
    __shared__ __attribute__((aligned(16))) float sK[kC * kLD];   // phi(K), later masked A
    __shared__ __attribute__((aligned(16))) float sS[kC * kLD];   // S_in^T
    __shared__ float sZ[kC], sQZ[kC], sDen[kC];
    __shared__ int sR[kC];
    __shared__ uint8_t sBeg[kC];
    __shared__ int s_bad;

    const int64_t c = blockIdx.x, h = blockIdx.y;
    const int64_t t0 = c * kC;
    const int nvalid = (int)(T - t0 < kC ? T - t0 : kC);
    const int tid = threadIdx.x;
    if (tid < kC) sBeg[tid] = tid < nvalid && is_begin(start, t0 + tid);
    if (tid == 0) s_bad = 0;
    stage<true, false>(sQ, q, t0, H, h, 0, nvalid);
    stage<true, false>(sK, k, t0, H, h, 0, nvalid);
    if (c > 0) {
        const float* src = Sinc + ((c - 1) * H + h) * kStateWords;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int f = tid + 256 * u;
            const int row = f >> 4, c4 = (f & 15) * 4;
            *(f32x4*)(sS + row * kLD + c4) = *(const f32x4*)(src + row * kC + c4);
        }
        if (tid < kC) sZ[tid] = src[kC * kC + tid];
    } else {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const int f = tid + 256 * u;
            const int row = f >> 4, c4 = (f & 15) * 4;
            *(f32x4*)(sS + row * kLD + c4) = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        }
        if (tid < kC) sZ[tid] = 0.0f;
    }
    __syncthreads();

    if (tid < kC) {
        int r = -1;
        for (int j = tid; j >= 0; --j)
            if (sBeg[j]) { r = j; break; }
        sR[tid] = r;
        float qz = 0.0f;
        for (int kd = 0; kd < kC; ++kd) qz += sQ[tid * kLD + kd] * sZ[kd];
        sQZ[tid] = qz;
    }
    f32x4 accA[4], accS[4];
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
        accA[jt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        accS[jt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    mfma_64x64x64(sQ, sK, accA);    // A[i][j]   = phi(q_i) . phi(k_j)
    mfma_64x64x64(sQ, sS, accS);    // QS[i][n]  = sum_kd phi(q_i)[kd] S_in[kd][n]
    __syncthreads();

    const int lane = tid & 63, w = tid >> 6;
    // masked A into sK (select: excluded entries are exact zeros)
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int i = 16 * w + 4 * (lane >> 4) + r;
            const int j = 16 * jt + (lane & 15);
            const int ri = sR[i];
            const bool keep = i < nvalid && j <= i && j >= (ri > 0 ? ri : 0);
            sK[i * kLD + j] = keep ? accA[jt][r] : 0.0f;
        }
    }
    const int bad = stage<false, true>(sQ, v, t0, H, h, 0, nvalid);   // V^T
    if (bad) atomicOr(&s_bad, 1);
    __syncthreads();

    if (tid < kC) {
        float den = 0.0f;
        for (int j = 0; j < kC; ++j) den += sK[tid * kLD + j];
        sDen[tid] = den + (sR[tid] < 0 ? sQZ[tid] : 0.0f);
    }
    f32x4 accO[4];
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) accO[jt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    const bool nonfinite_v = s_bad != 0;
    if (!nonfinite_v) {
        mfma_64x64x64(sK, sQ, accO);    // num[i][n] = sum_j Am[i][j] V[j][n]
    } else {
        // A non-finite value in V would reach other episodes of this chunk
        // through the dense product (0 * NaN = NaN); sum only each row's own
        // episode instead.
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int i = 16 * w + 4 * (lane >> 4) + r;
                const int n = 16 * jt + (lane & 15);
                const int ri = sR[i];
                float s = 0.0f;
                for (int j = (ri > 0 ? ri : 0); j <= i && j < nvalid; ++j) s += sK[i * kLD + j] * sQ[n * kLD + j];
                accO[jt][r] = s;
            }
        }
    }
    __syncthreads();

#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int i = 16 * w + 4 * (lane >> 4) + r;
            const int n = 16 * jt + (lane & 15);
            if (i < nvalid) {
                const float num = accO[jt][r] + (sR[i] < 0 ? accS[jt][r] : 0.0f);
                out[((t0 + i) * H + h) * kC + n] = num / sDen[i];
            }
        }
    }
}

__global__ __launch_bounds__(256) void fill_f32_kernel(float* p, int64_t n, float value) {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = value;
}

// ------------------------------------------------------------------ launch

hipError_t linattn_summary_launch(const float* k, const float* v, const uint8_t* start, float* dS, uint8_t* R,
                                  int64_t T, int64_t H, hipStream_t s) {
    const int64_t nch = (T + kC - 1) / kC;
    hipLaunchKernelGGL(linattn_summary_kernel, dim3((unsigned)nch, (unsigned)H), dim3(256), 0, s, k, v, start, dS,
                       R, T, H);
    return hipGetLastError();
}

hipError_t linattn_output_launch(const float* q, const float* k, const float* v, const uint8_t* start,
                                 const float* Sinc, float* out, int64_t T, int64_t H, hipStream_t s) {
    const int64_t nch = (T + kC - 1) / kC;
    hipLaunchKernelGGL(linattn_output_kernel, dim3((unsigned)nch, (unsigned)H), dim3(256), 0, s, q, k, v, start,
                       Sinc, out, T, H);
    return hipGetLastError();
}

hipError_t fill_f32_launch(float* p, int64_t n, float value, hipStream_t s) {
    int64_t blocks = (n + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(fill_f32_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n, value);
    return hipGetLastError();
}

}  // namespace memoroid
