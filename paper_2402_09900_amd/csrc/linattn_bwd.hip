// linattn_bwd.hip -- gradient of the linear-transformer memoroid readout
// (App. G.1) over a tape with resets, chunked like the forward pass, for
// gfx950.
//
// With Q = phi(q), K = phi(k), the forward states (S, z) and g = dL/dout:
//   dnum_i = g_i / den_i,  dden_i = -(g_i . out_i) / den_i,
//   dP     = (dnum V^T + dden 1^T) masked to the forward pattern M (j <= i,
//            j >= r_i: row i's episode inside the chunk),
//   dQ     = dP K + [r_i < 0] (S_in dnum_i + dden_i z_in),
//   dK     = dP^T Q + [row j's episode runs past the chunk] (U_out v_j + w_out),
//   dV     = (A (.) M)^T dnum + [same] U_out^T K_j,
// where (U, w) are reverse states: sums of Q_t dnum_t^T and dden_t Q_t over
// the later steps of the episode.  Per chunk the reverse summary is
// dU = sum of Q_i dnum_i^T over the rows before the chunk's first begin step
// (the rows whose episode continues into the previous chunk), and the chunk
// states are scanned right to left with the resettable reverse scan (a = 1),
// cut at every chunk that holds a begin step.
//
// Kernels: the forward summary and state scan (shared with the forward
// pass) give S_in, z_in; the backward summary computes den, dnum, dden for
// every row (kept in the workspace) and dU; the reverse state scan gives
// U_out; then one kernel forms dq, dk and dv.  Each of its workgroups (one
// chunk of one head) uses four 64x64 LDS tiles, all stored rotated so that
// either index of a tile can serve as the contraction index.
#include "linattn_common.hpp"

namespace memoroid {

namespace {

// Row `lane` of the chunk: its begin flag and the last begin at or before it
// (an inclusive max-scan across the wavefront; every wavefront has all 64).
__device__ __forceinline__ int row_last_begin(const uint8_t* start, int64_t t0, int nvalid, bool& beg) {
    const int lane = threadIdx.x & 63;
    beg = lane < nvalid && is_begin(start, t0 + lane);
    int rmax = beg ? lane : -1;
#pragma unroll
    for (int k = 1; k < 64; k <<= 1) {
        const int o = __shfl_up(rmax, k, 64);
        if (lane >= k) rmax = rmax > o ? rmax : o;
    }
    return rmax;
}

// Mask of the forward pattern for the accumulator element (i, j) of this
// lane: j <= i, j >= max(r_i, 0), i a valid row.
__device__ __forceinline__ bool keep_ij(int i, int j, int ri, int nvalid) {
    return i < nvalid && j <= i && j >= (ri > 0 ? ri : 0);
}

// phi of a fetched tile, rows outside [lo, hi) selected to zeros
__device__ __forceinline__ void phi_rows(f32x4 (&v)[4], int lo, int hi) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int row = (threadIdx.x + 256 * u) >> 4;
        const bool in = row >= lo && row < hi;
        v[u].x = in ? phi(v[u].x) : 0.0f; v[u].y = in ? phi(v[u].y) : 0.0f;
        v[u].z = in ? phi(v[u].z) : 0.0f; v[u].w = in ? phi(v[u].w) : 0.0f;
    }
}

// rows outside [lo, hi) selected to zeros (store_rows writes the result)
__device__ __forceinline__ f32x4 rows_in(const f32x4& v, int u, int lo, int hi) {
    const int row = (threadIdx.x + 256 * u) >> 4;
    const bool in = row >= lo && row < hi;
    return f32x4{in ? v.x : 0.0f, in ? v.y : 0.0f, in ? v.z : 0.0f, in ? v.w : 0.0f};
}

// phi'(u) from phi(u): 1 for u > 0 (phi = u + 1 >= 1), exp(u) = phi(u) <= 1
// otherwise, i.e. min(phi(u), 1), bit for bit; a NaN stays NaN
__device__ __forceinline__ float phi_prime_of_phi(float ph) { return ph > 1.0f ? 1.0f : ph; }

__device__ __forceinline__ void zero_acc(f32x4 (&acc)[4]) {
#pragma unroll
    for (int jt = 0; jt < 4; ++jt) acc[jt] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
}

}  // namespace

// ------------------------------------------------------------- summaries
// den, dnum, dden of every row (to the workspace), the reverse summary
// (dU, dw) of the rows before the chunk's first begin, and the shifted chunk
// flag of the reverse scan.  Also initialises the reverse scan's workspace.
__global__ __launch_bounds__(256) void linattn_bwd_summary_kernel(LinBwdArgs p) {
    __shared__ __attribute__((aligned(16))) float sQ[kC * kLD];   // phi(Q), later rotated rows < fb
    __shared__ __attribute__((aligned(16))) float sK[kC * kLD];   // phi(K), later dnum rotated rows < fb
    __shared__ float sZ[kC], sDen[kC], sDd[kC];
    __shared__ __attribute__((aligned(16))) float sDw[4][kC];      // dw, one partial per wavefront
    const int64_t c = blockIdx.x, h = blockIdx.y;
    const int64_t t0 = c * kC;
    const int nvalid = (int)(p.T - t0 < kC ? p.T - t0 : kC);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    // row block of the causal product A, rotated with the chunk so that the
    // triangle's uneven work spreads over the SIMDs of a CU
    const int rb = (w + (int)blockIdx.x) & 3;

    {   // reverse-scan workspace prepared: all-ones bytes
        const int64_t nblk = (int64_t)gridDim.x * gridDim.y;
        const int64_t gid = (int64_t)(blockIdx.y * gridDim.x + blockIdx.x) * 256 + tid;
        const u32x4 ones = {kEmpty32, kEmpty32, kEmpty32, kEmpty32};
        for (int64_t i = gid; i < p.fill16; i += nblk * 256) p.fill[i] = ones;
    }

    bool beg;
    const int rmax = row_last_begin(p.start, t0, nvalid, beg);
    const uint64_t mb = __ballot(beg);
    const int fb = mb ? __builtin_ctzll(mb) : kC;        // first begin row (64: none)

    // every global load up front: q, k, z_in; g and out of this thread's
    // row quarter (four threads per row, 16 columns each)
    f32x4 qreg[4], kreg[4], gv[4], ov[4];
    fetch_rows(qreg, p.q, t0, p.H, h, 0, nvalid);
    fetch_rows(kreg, p.k, t0, p.H, h, 0, nvalid);
    const float zin = tid < kC && c > 0 ? p.Sinc[((c - 1) * p.H + h) * kStateWords + kC * kC + tid] : 0.0f;
    const int grow = tid >> 2, gc0 = (tid & 3) * 16;
    {
        const ChunkRows cr_g = chunk_rows(p.g, t0, p.H, h, 0, nvalid);
        const ChunkRows cr_o = chunk_rows(p.out, t0, p.H, h, 0, nvalid);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            gv[u] = cr_g.load(grow, gc0 + 4 * u);
            ov[u] = cr_o.load(grow, gc0 + 4 * u);
        }
    }
    phi_rows(qreg, 0, nvalid);
    phi_rows(kreg, 0, nvalid);
    store_rows<false>(sQ, qreg);
    store_rows<false>(sK, kreg);
    if (tid < kC) sZ[tid] = zin;
    __syncthreads();

    f32x4 accA[4];
    zero_acc(accA);
    // A[i][j] = phi(q_i) . phi(k_j), only the column tiles that reach j <= i
    mfma_64x64x64<true, true>(sQ, sK, accA, rb, rb);
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int i = 16 * rb + 4 * (lane >> 4) + r;
        const int ri = __shfl(rmax, i, 64);
        float rs = 0.0f;
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
            rs += keep_ij(i, 16 * jt + (lane & 15), ri, nvalid) ? accA[jt][r] : 0.0f;
        const int kd = 4 * (lane & 15);
        const f32x4 qv = *(const f32x4*)(sQ + i * kLD + kd);
        float qz = qv.x * sZ[kd] + qv.y * sZ[kd + 1] + qv.z * sZ[kd + 2] + qv.w * sZ[kd + 3];
        rs = sum16(rs);
        qz = sum16(qz);
        if ((lane & 15) == 0) sDen[i] = rs + (ri < 0 ? qz : 0.0f);
    }
    __syncthreads();                                         // den ready; sQ/sK reads done

    // dnum = g / den and dden = -(g . out) / den: four threads per row, 16
    // columns each
    {
        const int row = grow, c0 = gc0;
        float dot = 0.0f;
        const bool ok = row < nvalid;
        const int64_t base = ((t0 + row) * p.H + h) * kC + c0;
#pragma unroll
        for (int u = 0; u < 4; ++u)
            dot += gv[u].x * ov[u].x + gv[u].y * ov[u].y + gv[u].z * ov[u].z + gv[u].w * ov[u].w;
        dot += __shfl_xor(dot, 1, 64);
        dot += __shfl_xor(dot, 2, 64);
        const float den = sDen[row];
        const float dd = -dot / den;
        const bool in_du = row < fb;                         // row's episode continues to the left
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            f32x4 dn;
            dn.x = gv[u].x / den; dn.y = gv[u].y / den; dn.z = gv[u].z / den; dn.w = gv[u].w / den;
            if (ok) *(f32x4*)(p.dnum + base + 4 * u) = dn;
            const f32x4 zz = {0.0f, 0.0f, 0.0f, 0.0f};
            *(f32x4*)(sK + row * kLD + rot_col(row, c0 + 4 * u)) = (ok && in_du) ? dn : zz;
        }
        if ((tid & 3) == 0) {
            if (ok) p.dden[(t0 + row) * p.H + h] = dd;
            sDd[row] = (ok && in_du) ? dd : 0.0f;
        }
    }
    // phi(Q) rows < fb, rotated, from the registers
    f32x4 qr[4];
    {
        const int hi = fb < nvalid ? fb : nvalid;
#pragma unroll
        for (int u = 0; u < 4; ++u) qr[u] = rows_in(qreg[u], u, 0, hi);
        store_rows<true>(sQ, qr);
    }
    __syncthreads();
    {   // dw[kd] = sum_i dden_i phi(Q)[i][kd]: each thread's four rows, then
        // the lanes holding the same columns (lane ^ 16, lane ^ 32)
        f32x4 zp = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const float d = sDd[(tid >> 4) + 16 * u];
            zp.x += d * qr[u].x; zp.y += d * qr[u].y; zp.z += d * qr[u].z; zp.w += d * qr[u].w;
        }
#pragma unroll
        for (int m = 16; m < 64; m <<= 1) {
            zp.x += __shfl_xor(zp.x, m, 64); zp.y += __shfl_xor(zp.y, m, 64);
            zp.z += __shfl_xor(zp.z, m, 64); zp.w += __shfl_xor(zp.w, m, 64);
        }
        if (lane < 16) *(f32x4*)(&sDw[w][lane * 4]) = zp;
    }

    f32x4 accU[4];
    zero_acc(accU);
    // dU[kd][n] = sum_i Q[i][kd] dnum[i][n]: A = Q^T, B = dnum, both k-major
    mfma_64x64x64<false, false>(sQ, sK, accU);
    float* du = p.dU + (c * p.H + h) * kStateWords;
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
        for (int r = 0; r < 4; ++r)
            du[(16 * w + 4 * (lane >> 4) + r) * kC + 16 * jt + (lane & 15)] = accU[jt][r];
    __syncthreads();                                         // dw partials ready
    if (tid < kC) du[kC * kC + tid] = (sDw[0][tid] + sDw[1][tid]) + (sDw[2][tid] + sDw[3][tid]);
    if (h == 0 && tid == 0) {
        if (c == 0) p.Rs[0] = 1;
        if (c + 1 < p.nch) p.Rs[c + 1] = mb ? 1 : 0;
    }
}

// ------------------------------------------------------------- dq, dk, dv
// The gradient kernel runs eight wavefronts per (chunk, head): wavefront w
// owns rows 16 rb .. 16 rb + 15 and the column half ch = w / 4 (column tiles
// 2 ch, 2 ch + 1) of every 64x64 product, with rb = w % 4 for ch = 0 and
// 3 - w % 4 for ch = 1.  The hardware places wavefront w on SIMD w % 4, so
// each SIMD gets one row block from each end of the causal triangle and the
// triangular products (dP, A) load the four SIMDs about evenly.  Eight
// wavefronts with at most 128 VGPRs each give two workgroups, four
// wavefronts per SIMD, on a CU.
constexpr int kGradThreads = 512;
constexpr int kGradPer = kC * kC / 4 / kGradThreads;    // float4 per thread per 64x64 tile

__device__ __forceinline__ void grad_block(int& rb, int& ch) {
    const int w = threadIdx.x >> 6;
    ch = w >> 2;
    rb = ch ? 3 - (w & 3) : (w & 3);
}

// rows [0, nvalid) of one chunk of a [T][H][64] tensor (zeros past them)
__device__ __forceinline__ void grad_fetch_rows(f32x4 (&v)[kGradPer], const float* src, int64_t t0, int64_t H,
                                                int64_t h, int nvalid) {
    const ChunkRows cr = chunk_rows(src, t0, H, h, 0, nvalid);
#pragma unroll
    for (int u = 0; u < kGradPer; ++u) {
        const int f = threadIdx.x + kGradThreads * u;
        v[u] = cr.load(f >> 4, (f & 15) * 4);
    }
}

// a 64x64 state block stored row-major (zeros when `have` is false)
__device__ __forceinline__ void grad_fetch_state(f32x4 (&v)[kGradPer], const float* src, bool have) {
    const Rsrc r = make_rsrc(src, have ? kC * kC * 4 : 0);
#pragma unroll
    for (int u = 0; u < kGradPer; ++u) {
        const int f = threadIdx.x + kGradThreads * u;
        const u32x4 wv = __builtin_amdgcn_raw_buffer_load_b128(r, ((f >> 4) * kC + (f & 15) * 4) * 4, 0, 0);
        v[u] = f32x4{__uint_as_float(wv.x), __uint_as_float(wv.y), __uint_as_float(wv.z), __uint_as_float(wv.w)};
    }
}

// phi of fetched rows, rows at or past nvalid selected to zeros
__device__ __forceinline__ void grad_phi(f32x4 (&v)[kGradPer], int nvalid) {
#pragma unroll
    for (int u = 0; u < kGradPer; ++u) {
        const bool in = (int)((threadIdx.x + kGradThreads * u) >> 4) < nvalid;
        v[u].x = in ? phi(v[u].x) : 0.0f; v[u].y = in ? phi(v[u].y) : 0.0f;
        v[u].z = in ? phi(v[u].z) : 0.0f; v[u].w = in ? phi(v[u].w) : 0.0f;
    }
}

__device__ __forceinline__ void grad_store(float* s, const f32x4 (&v)[kGradPer]) {
#pragma unroll
    for (int u = 0; u < kGradPer; ++u) {
        const int f = threadIdx.x + kGradThreads * u;
        const int row = f >> 4, c4 = (f & 15) * 4;
        *(f32x4*)(s + row * kLD + rot_col(row, c4)) = v[u];
    }
}

// acc[jj][r] = C[16 rb + 4 (lane / 16) + r][16 (2 ch + jj) + lane % 16]
__device__ __forceinline__ void grad_acc_to_lds(float* s, const f32x4 (&acc)[2], int rb, int ch) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = 16 * rb + 4 * (lane >> 4) + r, col = 16 * (2 * ch + jj) + (lane & 15);
            s[row * kLD + rot_col(row, col)] = acc[jj][r];
        }
}

// acc += A * B on this wavefront's row block and column half, for 64x64 LDS
// tiles all stored rotated (rot_col).
//   A_ROWS: A[i][k] is element (i, k) of the A tile, else element (k, i);
//   B_ROWS: B[k][j] is element (j, k) of the B tile, else element (k, j).
// Read along its rows, a rotated tile still gives 16-byte runs (the rotation
// moves whole 16-column blocks, the same for the 16 rows a wavefront
// reads), so either index of a tile can be the contraction index and no
// tile is staged twice.  Column tiles past jt_last are left untouched.
template <bool A_ROWS, bool B_ROWS>
__device__ __forceinline__ void grad_mfma(const float* sA, const float* sB, f32x4 (&acc)[2], int rb, int ch,
                                          int jt_last = 3) {
    if (2 * ch > jt_last) return;
    const int lane = threadIdx.x & 63;
    const int i = 16 * rb + (lane & 15), kk = (lane >> 4) * 16;
    float af[16];
    if constexpr (A_ROWS) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const f32x4 v = *(const f32x4*)(sA + i * kLD + rot_col(i, kk + 4 * u));
            af[4 * u] = v.x; af[4 * u + 1] = v.y; af[4 * u + 2] = v.z; af[4 * u + 3] = v.w;
        }
    } else {
        const int c = rot_col(kk, i);
#pragma unroll
        for (int s = 0; s < 16; ++s) af[s] = sA[(kk + s) * kLD + c];
    }
#pragma unroll
    for (int jj = 0; jj < 2; ++jj) {
        const int jt = 2 * ch + jj;
        if (jt > jt_last) break;
        const int j = 16 * jt + (lane & 15);
        float bf[16];
        if constexpr (B_ROWS) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const f32x4 v = *(const f32x4*)(sB + j * kLD + rot_col(j, kk + 4 * u));
                bf[4 * u] = v.x; bf[4 * u + 1] = v.y; bf[4 * u + 2] = v.z; bf[4 * u + 3] = v.w;
            }
        } else {
            const int c = rot_col(kk, j);
#pragma unroll
            for (int s = 0; s < 16; ++s) bf[s] = sB[(kk + s) * kLD + c];
        }
#pragma unroll
        for (int s = 0; s < 16; ++s) acc[jj] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[s], bf[s], acc[jj], 0, 0, 0);
    }
}

// grad_mfma over the k-blocks q_lo .. q_hi only (k in [16 q_lo, 16 q_hi + 16)),
// for products whose A is zero outside them in this row block (a causal
// factor: dP or A, read along either index).  MFMA number 4q + r takes k = 16q
// + 4 (lane / 16) + r in its four k-slots, so each k-block is whole in its
// own four MFMAs; A_ROWS reads stay 16-byte runs (4 (lane / 16) + 3 < 16, and
// the rotation moves whole 16-column blocks), and the k-rows read by the
// other mode sit 4 rows apart, which the 68-float stride puts in different
// LDS banks.
template <bool A_ROWS, bool B_ROWS>
__device__ __forceinline__ void grad_mfma_kblocks(const float* sA, const float* sB, f32x4 (&acc)[2], int rb, int ch,
                                                  int q_lo, int q_hi) {
    const int lane = threadIdx.x & 63, g = lane >> 4;
    const int i = 16 * rb + (lane & 15);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        if (q < q_lo || q > q_hi) continue;
        const int k0 = 16 * q + 4 * g;
        float af[4], bf[4][2];
        if constexpr (A_ROWS) {
            const f32x4 v = *(const f32x4*)(sA + i * kLD + rot_col(i, k0));
            af[0] = v.x; af[1] = v.y; af[2] = v.z; af[3] = v.w;
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r) af[r] = sA[(k0 + r) * kLD + rot_col(k0 + r, i)];
        }
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
            const int j = 16 * (2 * ch + jj) + (lane & 15);
            if constexpr (B_ROWS) {
                const f32x4 v = *(const f32x4*)(sB + j * kLD + rot_col(j, k0));
                bf[0][jj] = v.x; bf[1][jj] = v.y; bf[2][jj] = v.z; bf[3][jj] = v.w;
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r) bf[r][jj] = sB[(k0 + r) * kLD + rot_col(k0 + r, j)];
            }
        }
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int jj = 0; jj < 2; ++jj)
                acc[jj] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[r], bf[r][jj], acc[jj], 0, 0, 0);
    }
}

// any value of the fetched rows that is not finite
__device__ __forceinline__ bool grad_nonfinite(const f32x4 (&v)[kGradPer]) {
    bool bad = false;
#pragma unroll
    for (int u = 0; u < kGradPer; ++u) bad |= !finite4(v[u]);
    return bad;
}

// Products of a causal factor P (masked to the episodes: exact zeros outside
// them) with a row operand Y, summed over each row's own episode only, for
// chunks holding a value that is not finite, where the dense product would
// carry it to other episodes through 0 * NaN.  Both tiles are rotated.
//   rows of P:    out[i][col] = sum over j in [lo_i, i]   of P[i][j] Y[j][col]
//   columns of P: out[j][col] = sum over i in [j, end_j)  of P[i][j] Y[i][col]
// (lo_i: row i's episode start in the chunk; end_j: the first begin after
// row j, or the chunk's valid rows).
__device__ __forceinline__ float episode_row_sum(const float* sP, const float* sY, int i, int lo, int col) {
    float acc = 0.0f;
    for (int j = lo; j <= i; ++j) acc += sP[i * kLD + rot_col(i, j)] * sY[j * kLD + rot_col(j, col)];
    return acc;
}
__device__ __forceinline__ float episode_col_sum(const float* sP, const float* sY, int j, int end, int col) {
    float acc = 0.0f;
    for (int i = j; i < end; ++i) acc += sP[i * kLD + rot_col(i, j)] * sY[i * kLD + rot_col(i, col)];
    return acc;
}

__device__ __forceinline__ void zero2(f32x4 (&acc)[2]) {
    acc[0] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    acc[1] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
}

// One workgroup per (chunk, head) forms dq, dk and dv from four rotated LDS
// tiles, each written once per phase:
//   phase 1 (U_out, phi(K), V, dnum): dK2 = V U_out^T, dV2 = phi(K) U_out,
//                                     dP = (dnum V^T + dden) masked
//   phase 2 (phi(Q), phi(K), dP, dnum): A = phi(Q) phi(K)^T masked,
//                                       dQ1 = dP phi(K), dK1 = dP^T phi(Q) -> dk
//   phase 3 (S_in^T, phi(K), A, dnum): dV1 = A^T dnum -> dv, dQ2 = dnum S_in^T -> dq
// The state products are skipped by wavefronts none of whose rows take them
// (dK2, dV2: rows at or after the chunk's last begin; dQ2: rows before its
// first), dP, A skip their column tiles above the diagonal, and dQ1, dK1,
// dV1 the k-blocks where their causal factor is zero.  A chunk whose phi(K),
// phi(Q) or dnum holds a value that is not finite forms dQ1, dK1 and dV1 as
// explicit sums over each row's own episode instead (the masked factor's
// zeros would otherwise meet that value in the dense product).
__global__ __launch_bounds__(kGradThreads, 2) void linattn_bwd_grad_kernel(LinBwdArgs p) {
    __shared__ __attribute__((aligned(16))) float X0[kC * kLD];   // U_out [kd][n], then phi(Q), then S_in^T [n][kd]
    __shared__ __attribute__((aligned(16))) float X1[kC * kLD];   // phi(K)
    __shared__ __attribute__((aligned(16))) float X2[kC * kLD];   // V, then dP, then A
    __shared__ __attribute__((aligned(16))) float X3[kC * kLD];   // dnum
    __shared__ float sW[kC], sZ[kC];
    const int64_t c = blockIdx.x, h = blockIdx.y;
    const int64_t t0 = c * kC;
    const int nvalid = (int)(p.T - t0 < kC ? p.T - t0 : kC);
    const int tid = threadIdx.x, lane = tid & 63;
    int rb, ch;
    grad_block(rb, ch);
    bool beg;
    const int rmax = row_last_begin(p.start, t0, nvalid, beg);
    const uint64_t mb = __ballot(beg);
    const int lastb = mb ? 63 - __builtin_clzll(mb) : -1;    // rows >= lastb continue past the chunk
    const int firstb = mb ? __builtin_ctzll(mb) : kC;        // rows < firstb continue from the previous chunk
    const bool have_u = c + 1 < p.nch, have_s = c > 0;
    const float* uo = p.Y + (have_u ? ((c + 1) * p.H + h) * kStateWords : 0);
    const float* si = p.Sinc + (have_s ? ((c - 1) * p.H + h) * kStateWords : 0);

    // every global load up front
    f32x4 ureg[kGradPer], kreg[kGradPer], vreg[kGradPer], dnreg[kGradPer], qreg[kGradPer], sreg[kGradPer];
    grad_fetch_state(ureg, uo, have_u);
    grad_fetch_rows(kreg, p.k, t0, p.H, h, nvalid);
    grad_fetch_rows(vreg, p.v, t0, p.H, h, nvalid);
    grad_fetch_rows(dnreg, p.dnum, t0, p.H, h, nvalid);
    grad_fetch_rows(qreg, p.q, t0, p.H, h, nvalid);
    grad_fetch_state(sreg, si, have_s);
    if (tid < kC) {
        sW[tid] = have_u ? uo[kC * kC + tid] : 0.0f;
        sZ[tid] = have_s ? si[kC * kC + tid] : 0.0f;
    }
    float dd[4];
    int ri[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int i = 16 * rb + 4 * (lane >> 4) + r;
        dd[r] = i < nvalid ? p.dden[(t0 + i) * p.H + h] : 0.0f;
        ri[r] = __shfl(rmax, i, 64);
    }
    grad_phi(kreg, nvalid);
    grad_store(X0, ureg);
    grad_store(X1, kreg);
    grad_store(X2, vreg);
    grad_store(X3, dnreg);
    __syncthreads();

    // ---- phase 1
    f32x4 accK2[2], accV2[2], accP[2];
    zero2(accK2);
    zero2(accV2);
    zero2(accP);
    if (have_u && 16 * rb + 15 >= lastb) {
        grad_mfma<true, true>(X2, X0, accK2, rb, ch);        // sum_n V[j][n] U[kd][n]
        grad_mfma<true, false>(X1, X0, accV2, rb, ch);       // sum_kd K[j][kd] U[kd][n]
    }
    grad_mfma<true, true>(X3, X2, accP, rb, ch, rb);         // sum_n dnum[i][n] V[j][n]
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = 16 * rb + 4 * (lane >> 4) + r, col = 16 * (2 * ch + jj) + (lane & 15);
            accP[jj][r] = keep_ij(row, col, ri[r], nvalid) ? accP[jj][r] + dd[r] : 0.0f;
        }
    grad_phi(qreg, nvalid);
    const bool nonfinite =
        __syncthreads_or(grad_nonfinite(kreg) || grad_nonfinite(qreg) || grad_nonfinite(dnreg)) != 0;
    // X0 (U_out), X2 (V) free
    grad_store(X0, qreg);
    grad_acc_to_lds(X2, accP, rb, ch);
    __syncthreads();

    // ---- phase 2
    f32x4 accA[2], accQ1[2], accK1[2];
    zero2(accA);
    zero2(accQ1);
    zero2(accK1);
    grad_mfma<true, true>(X0, X1, accA, rb, ch, rb);         // sum_kd Q[i][kd] K[j][kd]
    // episode bounds of this lane's rows, for the explicit sums
    int lo_r[4], end_r[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int row = 16 * rb + 4 * (lane >> 4) + r;
        lo_r[r] = ri[r] > 0 ? ri[r] : 0;
        const uint64_t later = row < 63 ? mb & ~((2ull << row) - 1ull) : 0ull;   // begins after row
        end_r[r] = later ? __builtin_ctzll(later) : nvalid;
    }
    if (!nonfinite) {
        // dP[i][j] = 0 for j > i: row block rb of dQ1 takes j < 16 rb + 16,
        // and of dK1 (rows j) takes i >= 16 rb
        grad_mfma_kblocks<true, false>(X2, X1, accQ1, rb, ch, 0, rb);    // sum_j dP[i][j] K[j][kd]
        grad_mfma_kblocks<false, false>(X2, X0, accK1, rb, ch, rb, 3);   // sum_i dP[i][j] Q[i][kd]
    } else {
#pragma unroll
        for (int jj = 0; jj < 2; ++jj)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = 16 * rb + 4 * (lane >> 4) + r, col = 16 * (2 * ch + jj) + (lane & 15);
                if (row < nvalid) {
                    accQ1[jj][r] = episode_row_sum(X2, X1, row, lo_r[r], col);
                    accK1[jj][r] = episode_col_sum(X2, X0, row, end_r[r], col);
                }
            }
    }
    // this lane's accumulator elements (row, col): A masked; phi'(q) kept for
    // dq; dk (rows j, columns kd) written, with phi'(k) from phi(K)
    float pq[2][4];
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = 16 * rb + 4 * (lane >> 4) + r, col = 16 * (2 * ch + jj) + (lane & 15);
            accA[jj][r] = keep_ij(row, col, ri[r], nvalid) ? accA[jj][r] : 0.0f;
            pq[jj][r] = phi_prime_of_phi(X0[row * kLD + rot_col(row, col)]);
            if (row < nvalid) {
                const float dK = accK1[jj][r] + (row >= lastb ? accK2[jj][r] + sW[col] : 0.0f);
                p.dk[((t0 + row) * p.H + h) * kC + col] = dK * phi_prime_of_phi(X1[row * kLD + rot_col(row, col)]);
            }
        }
    __syncthreads();                                         // X0 (phi(Q)), X2 (dP) free
    grad_store(X0, sreg);
    grad_acc_to_lds(X2, accA, rb, ch);
    __syncthreads();

    // ---- phase 3
    f32x4 accV1[2], accQ2[2];
    zero2(accV1);
    zero2(accQ2);
    if (!nonfinite) {
        grad_mfma_kblocks<false, false>(X2, X3, accV1, rb, ch, rb, 3);   // sum_{i >= j} A[i][j] dnum[i][n]
    } else {
#pragma unroll
        for (int jj = 0; jj < 2; ++jj)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int row = 16 * rb + 4 * (lane >> 4) + r, col = 16 * (2 * ch + jj) + (lane & 15);
                if (row < nvalid) accV1[jj][r] = episode_col_sum(X2, X3, row, end_r[r], col);
            }
    }
    if (have_s && 16 * rb < firstb) grad_mfma<true, false>(X3, X0, accQ2, rb, ch);   // sum_n dnum[i][n] S_in[kd][n]
#pragma unroll
    for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int i = 16 * rb + 4 * (lane >> 4) + r, col = 16 * (2 * ch + jj) + (lane & 15);
            if (i < nvalid) {
                p.dv[((t0 + i) * p.H + h) * kC + col] = accV1[jj][r] + (i >= lastb ? accV2[jj][r] : 0.0f);
                const float dQ = accQ1[jj][r] + (ri[r] < 0 ? accQ2[jj][r] + dd[r] * sZ[col] : 0.0f);
                p.dq[((t0 + i) * p.H + h) * kC + col] = dQ * pq[jj][r];
            }
        }
}

hipError_t linattn_bwd_summary_launch(const LinBwdArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(linattn_bwd_summary_kernel, dim3((unsigned)a.nch, (unsigned)a.H), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t linattn_bwd_grad_launch(const LinBwdArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(linattn_bwd_grad_kernel, dim3((unsigned)a.nch, (unsigned)a.H), dim3(kGradThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace memoroid
