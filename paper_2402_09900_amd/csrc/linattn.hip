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
//     (it also initialises the state scan's workspace);
//   the chunk states are then scanned with the resettable diagonal scan
//   (a = 1: the sum monoid), giving S_inc(c) = state after chunk c;
//   output kernel (one workgroup per chunk and head), with r_i the last begin
//   step <= i inside the chunk (-1 if none):
//     A   = phi(Q) phi(K)^T,  masked to j <= i and j >= r_i
//     num = A V + [r_i < 0] phi(Q) S_inc(c-1),  den = rowsum(A) + [r_i < 0] phi(Q).z
//     out = num / den;
//   the head-0 workgroups also produce the episode index of the chunk's steps.
//
// Contractions use v_mfma_f32_16x16x4_f32 on operands staged in LDS in their
// natural (row-major) layout.  In one MFMA the four k-slots take k = 16*slot
// + s, a permutation of the contraction index applied to both operands, so
// an operand stored with k contiguous is read with 16-byte LDS loads; one
// stored with k as its row index is read with 4-byte loads whose rows are
// rotated by 16 columns per 16 rows, which spreads the four k-slots over
// different LDS banks.
#include "linattn_common.hpp"

namespace memoroid {

// ---------------------------------------------------------------- summaries

__global__ __launch_bounds__(256) void linattn_summary_kernel(LinSummaryArgs p) {
    __shared__ __attribute__((aligned(16))) float sK[kC * kLD];   // phi(K), rotated
    __shared__ __attribute__((aligned(16))) float sV[kC * kLD];   // V, rotated
    __shared__ __attribute__((aligned(16))) float sZ[4][kC];      // dz, one partial per wavefront
    const int64_t c = blockIdx.x, h = blockIdx.y;
    const int64_t t0 = c * kC;
    const int nvalid = (int)(p.T - t0 < kC ? p.T - t0 : kC);

    // workspace of the state scan and the episode-index count words are
    // prepared (all-ones bytes) here, so that the later kernels find them
    // ready (stream order)
    {
        const int64_t nblk = (int64_t)gridDim.x * gridDim.y;
        const int64_t gid = (int64_t)(blockIdx.y * gridDim.x + blockIdx.x) * 256 + threadIdx.x;
        const u32x4 ones = {kEmpty32, kEmpty32, kEmpty32, kEmpty32};
        for (int64_t i = gid; i < p.fill16; i += nblk * 256) p.fill[i] = ones;
    }

    // K, V rows and the begin flags are all loaded at once; every wavefront
    // finds the chunk's last begin step with one ballot (lane = row), and
    // rows before it are then selected to zeros in both phi(K) and V (a
    // select, so non-finite values there never enter)
    f32x4 kreg[4], vreg[4];
    fetch_rows(kreg, p.k, t0, p.H, h, 0, nvalid);
    fetch_rows(vreg, p.v, t0, p.H, h, 0, nvalid);
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const uint64_t bm = __ballot(lane < nvalid && is_begin(p.start, t0 + lane));
    const int last = bm ? 63 - __builtin_clzll(bm) : -1;
    const int lo = last > 0 ? last : 0;
    // dz: each thread sums its four rows of phi(K) per column, then the four
    // lanes of a wavefront that hold the same columns (lane ^ 16, lane ^ 32)
    f32x4 zp = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int f = threadIdx.x + 256 * u;
        const int row = f >> 4, c4 = (f & 15) * 4;
        const bool in = row >= lo && row < nvalid;
        f32x4 kv = kreg[u], vv = vreg[u];
        kv.x = in ? phi(kv.x) : 0.0f; kv.y = in ? phi(kv.y) : 0.0f;
        kv.z = in ? phi(kv.z) : 0.0f; kv.w = in ? phi(kv.w) : 0.0f;
        vv.x = in ? vv.x : 0.0f; vv.y = in ? vv.y : 0.0f; vv.z = in ? vv.z : 0.0f; vv.w = in ? vv.w : 0.0f;
        *(f32x4*)(sK + row * kLD + rot_col(row, c4)) = kv;
        *(f32x4*)(sV + row * kLD + rot_col(row, c4)) = vv;
        zp.x += kv.x; zp.y += kv.y; zp.z += kv.z; zp.w += kv.w;
    }
#pragma unroll
    for (int m = 16; m < 64; m <<= 1) {
        zp.x += __shfl_xor(zp.x, m, 64); zp.y += __shfl_xor(zp.y, m, 64);
        zp.z += __shfl_xor(zp.z, m, 64); zp.w += __shfl_xor(zp.w, m, 64);
    }
    if (lane < 16) *(f32x4*)(&sZ[w][lane * 4]) = zp;
    __syncthreads();

    f32x4 acc[4];
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) acc[jt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    // C[n][kd] = sum_j V[j][n] phi(K)[j][kd] = dS^T: A = V^T, B = phi(K), both k-major
    mfma_64x64x64<false, false>(sV, sK, acc);

    float* out = p.dS + (c * p.H + h) * kStateWords;
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
        const int t = threadIdx.x;
        out[kC * kC + t] = (sZ[0][t] + sZ[1][t]) + (sZ[2][t] + sZ[3][t]);
    }
    if (h == 0 && threadIdx.x == 0) p.R[c] = last >= 0 ? 1 : 0;
}

// ------------------------------------------------------------------- output

__global__ __launch_bounds__(256, 4) void linattn_output_kernel(LinOutputArgs p) {
    // two LDS tiles, reused in turn: (phi(Q), phi(K)) -> (phi(Q), S_in^T) ->
    // (masked A, V rotated); 35 KB per workgroup, four workgroups per CU
    __shared__ __attribute__((aligned(16))) float X0[kC * kLD];
    __shared__ __attribute__((aligned(16))) float X1[kC * kLD];
    __shared__ float sZ[kC];

    const int64_t c = blockIdx.x, h = blockIdx.y;
    const int64_t t0 = c * kC;
    const int nvalid = (int)(p.T - t0 < kC ? p.T - t0 : kC);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    // the causal products give the wavefront of row block rb (rb + 1) / 4 of
    // a full product's work, and wavefront w of a workgroup usually runs on
    // SIMD w: row blocks rotate with the chunk so that the SIMDs of a CU
    // share the triangle evenly across its workgroups
    const int rb = (w + (int)blockIdx.x) & 3;

    // row `lane` of the chunk: begin flag, and the last begin at or before it
    // (an inclusive max-scan across the wavefront; every wavefront has all 64)
    const bool beg = lane < nvalid && is_begin(p.start, t0 + lane);
    int rmax = beg ? lane : -1;
#pragma unroll
    for (int k = 1; k < 64; k <<= 1) {
        const int o = __shfl_up(rmax, k, 64);
        if (lane >= k) rmax = rmax > o ? rmax : o;
    }

    // every global load of the workgroup is issued before any LDS store: q,
    // k, v and S_in into registers (S and V wait there for their turn in LDS)
    f32x4 qreg[4], kreg[4], vreg[4], sreg[4];
    fetch_rows(qreg, p.q, t0, p.H, h, 0, nvalid);
    fetch_rows(kreg, p.k, t0, p.H, h, 0, nvalid);
    const int bad = fetch_rows(vreg, p.v, t0, p.H, h, 0, nvalid);
    // S_in: the state after the previous chunk (an empty range, read as
    // zeros, for the first chunk)
    const Rsrc rs_s = make_rsrc(p.Sinc + (c > 0 ? ((c - 1) * p.H + h) * kStateWords : 0),
                                c > 0 ? kStateWords * 4 : 0);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int f = tid + 256 * u;
        const u32x4 wv = __builtin_amdgcn_raw_buffer_load_b128(rs_s, ((f >> 4) * kC + (f & 15) * 4) * 4, 0, 0);
        sreg[u] = f32x4{__uint_as_float(wv.x), __uint_as_float(wv.y), __uint_as_float(wv.z), __uint_as_float(wv.w)};
    }
    const float zin = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rs_s, (kC * kC + (tid & (kC - 1))) * 4, 0, 0));
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int f = tid + 256 * u;
        const int row = f >> 4, c4 = (f & 15) * 4;
        // phi of every row: rows past T read zeros (phi = 1), and their
        // entries are masked out of A or belong to outputs never stored
        f32x4 qv = qreg[u], kv = kreg[u];
        qv.x = phi(qv.x); qv.y = phi(qv.y); qv.z = phi(qv.z); qv.w = phi(qv.w);
        kv.x = phi(kv.x); kv.y = phi(kv.y); kv.z = phi(kv.z); kv.w = phi(kv.w);
        *(f32x4*)(X0 + row * kLD + c4) = qv;
        *(f32x4*)(X1 + row * kLD + c4) = kv;
    }
    if (tid < kC) sZ[tid] = zin;
    const bool nonfinite_v = __syncthreads_or(bad) != 0;

    // episode index of the chunk's steps (head-0 workgroups): wavefront 2
    // publishes the chunk's own begin count at once, wavefront 1 looks back
    // for the count before the chunk, publishes the running count and writes
    // the indices (publishing and polling use different wavefronts)
    if (p.idx != nullptr && h == 0 && (w == 1 || w == 2)) {
        const uint64_t m = __ballot(beg);
        const uint32_t c_chunk = (uint32_t)__builtin_popcountll(m);
        if (w == 2) {
            if (lane == 0) publish64(p.cnt + c, (c == 0 ? kCountIncl : kCountOwn) | c_chunk);
        } else {
            const uint32_t before = c == 0 ? 0u : count_lookback(p.cnt, c - 1, 1, p.timeout);
            if (lane == 0 && c > 0) publish64(p.cnt + c, kCountIncl | (before + c_chunk));
            const uint32_t upto = (uint32_t)__builtin_popcountll(m & ((2ull << lane) - 1ull));
            if (lane < nvalid) p.idx[t0 + lane] = (int32_t)(before + upto) - 1;
        }
    }

    f32x4 accA[4], accS[4];
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
        accA[jt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
        accS[jt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    // A[i][j] = phi(q_i) . phi(k_j); column tiles above the diagonal are
    // masked out entirely and skipped
    mfma_64x64x64<true, true>(X0, X1, accA, rb, rb);
    __syncthreads();                            // every wavefront is done with phi(K)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int f = tid + 256 * u;
        *(f32x4*)(X1 + (f >> 4) * kLD + (f & 15) * 4) = sreg[u];
    }
    __syncthreads();
    // QS[i][n] = sum_kd phi(q_i)[kd] S_in[kd][n], needed only by rows before
    // the chunk's first begin (their episode started in an earlier chunk)
    const uint64_t bmask = __ballot(beg);
    const int fbeg = bmask ? __builtin_ctzll(bmask) : kC;
    if (16 * rb < fbeg) mfma_64x64x64<true, true>(X0, X1, accS, 3, rb);

    // mask A to each row's episode (a select: excluded entries are exact
    // zeros), then the row sums and phi(q_i).z_in, reduced across lanes
    int ri[4];
    float den[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int i = 16 * rb + 4 * (lane >> 4) + r;
        ri[r] = __shfl(rmax, i, 64);
        float rs = 0.0f;
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
            const int j = 16 * jt + (lane & 15);
            const bool keep = i < nvalid && j <= i && j >= (ri[r] > 0 ? ri[r] : 0);
            accA[jt][r] = keep ? accA[jt][r] : 0.0f;
            rs += accA[jt][r];
        }
        const int kd = 4 * (lane & 15);
        const f32x4 qv = *(const f32x4*)(X0 + i * kLD + kd);
        float qz = qv.x * sZ[kd] + qv.y * sZ[kd + 1] + qv.z * sZ[kd + 2] + qv.w * sZ[kd + 3];
        rs = sum16(rs);
        qz = sum16(qz);
        den[r] = rs + (ri[r] < 0 ? qz : 0.0f);
    }
    __syncthreads();                            // every wavefront is done with phi(Q) and S
    float* const sA = X0;
    float* const sV = X1;
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) {
#pragma unroll
        for (int r = 0; r < 4; ++r) sA[(16 * rb + 4 * (lane >> 4) + r) * kLD + 16 * jt + (lane & 15)] = accA[jt][r];
    }
    store_rows<true>(sV, vreg);
    __syncthreads();

    f32x4 accO[4];
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) accO[jt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    if (!nonfinite_v) {
        mfma_64x64x64_tril(sA, sV, accO, rb);       // num[i][n] = sum_{j <= i} A[i][j] V[j][n]
    } else {
        // A non-finite value in V would reach other episodes of this chunk
        // through the dense product (0 * NaN = NaN); sum each row's own
        // episode explicitly instead.
#pragma unroll
        for (int jt = 0; jt < 4; ++jt) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int i = 16 * rb + 4 * (lane >> 4) + r;
                const int n = 16 * jt + (lane & 15);
                float s = 0.0f;
                for (int j = (ri[r] > 0 ? ri[r] : 0); j <= i && j < nvalid; ++j)
                    s += sA[i * kLD + j] * sV[j * kLD + rot_col(j, n)];
                accO[jt][r] = s;
            }
        }
    }

    // one reciprocal per row (correctly rounded) and a product per output
    float rden[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) rden[r] = 1.0f / den[r];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int i = 16 * rb + 4 * (lane >> 4) + r;
        if (i < nvalid) {
            float* orow = p.out + ((t0 + i) * p.H + h) * kC + (lane & 15);
#pragma unroll
            for (int jt = 0; jt < 4; ++jt) {
                const float num = accO[jt][r] + (ri[r] < 0 ? accS[jt][r] : 0.0f);
                __builtin_nontemporal_store(num * rden[r], &orow[16 * jt]);   // written once, read by no later kernel
            }
        }
    }
}

// ------------------------------------------------------------------ launch

hipError_t linattn_summary_launch(const LinSummaryArgs& a, hipStream_t s) {
    const int64_t nch = (a.T + kC - 1) / kC;
    hipLaunchKernelGGL(linattn_summary_kernel, dim3((unsigned)nch, (unsigned)a.H), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t linattn_output_launch(const LinOutputArgs& a, hipStream_t s) {
    const int64_t nch = (a.T + kC - 1) / kC;
    hipLaunchKernelGGL(linattn_output_kernel, dim3((unsigned)nch, (unsigned)a.H), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace memoroid
