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

// Write a 64x64 accumulator tile (acc[jt][r] = C[16w + 4(lane/16) + r][16 jt + lane%16])
// to LDS, natural or rotated.
template <bool ROT>
__device__ __forceinline__ void acc_to_lds(float* s, const f32x4 (&acc)[4]) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = 16 * w + 4 * (lane >> 4) + r, col = 16 * jt + (lane & 15);
            s[row * kLD + (ROT ? rot_col(row, col) : col)] = acc[jt][r];
        }
}

// Load a 64x64 state block stored row-major at src into registers (the
// fetch_rows layout); zeros when `have` is false.
__device__ __forceinline__ void fetch_state(f32x4 (&v)[4], const float* src, bool have) {
    const Rsrc r = make_rsrc(src, have ? kC * kC * 4 : 0);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int f = threadIdx.x + 256 * u;
        const u32x4 wv = __builtin_amdgcn_raw_buffer_load_b128(r, ((f >> 4) * kC + (f & 15) * 4) * 4, 0, 0);
        v[u] = f32x4{__uint_as_float(wv.x), __uint_as_float(wv.y), __uint_as_float(wv.z), __uint_as_float(wv.w)};
    }
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
    const int64_t c = blockIdx.x, h = blockIdx.y;
    const int64_t t0 = c * kC;
    const int nvalid = (int)(p.T - t0 < kC ? p.T - t0 : kC);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;

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
    mfma_64x64x64<true, true>(sQ, sK, accA);               // A[i][j] = phi(q_i) . phi(k_j)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int i = 16 * w + 4 * (lane >> 4) + r;
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
    {   // phi(Q) rows < fb, rotated, from the registers
        const int hi = fb < nvalid ? fb : nvalid;
        f32x4 qr[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) qr[u] = rows_in(qreg[u], u, 0, hi);
        store_rows<true>(sQ, qr);
    }
    __syncthreads();

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
    if (tid < kC) {
        float s = 0.0f;
        for (int i = 0; i < kC; ++i) s += sDd[i] * sQ[i * kLD + rot_col(i, tid)];
        du[kC * kC + tid] = s;
    }
    if (h == 0 && tid == 0) {
        if (c == 0) p.Rs[0] = 1;
        if (c + 1 < p.nch) p.Rs[c + 1] = mb ? 1 : 0;
    }
}

// ------------------------------------------------------------- dq, dk, dv
// acc += A * B for 64x64 LDS tiles that are all stored rotated (rot_col).
//   A_ROWS: A[i][k] is element (i, k) of the A tile, else element (k, i);
//   B_ROWS: B[k][j] is element (j, k) of the B tile, else element (k, j).
// Read along its rows, a rotated tile still gives 16-byte runs (the rotation
// moves whole 16-column blocks, the same for the 16 rows of a wavefront), so
// either index of a tile can be the contraction index and no tile is staged
// twice.  jt_last as in mfma_64x64x64.
template <bool A_ROWS, bool B_ROWS>
__device__ __forceinline__ void mfma_rot(const float* sA, const float* sB, f32x4 acc[4], int jt_last = 3) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int i = 16 * w + (lane & 15), kk = (lane >> 4) * 16;
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
    for (int jt = 0; jt < 4; ++jt) {
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
        for (int s = 0; s < 16; ++s) acc[jt] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[s], bf[s], acc[jt], 0, 0, 0);
    }
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
// first), and dP, A skip their column tiles above the diagonal.
__global__ __launch_bounds__(256, 2) void linattn_bwd_grad_kernel(LinBwdArgs p) {
    __shared__ __attribute__((aligned(16))) float X0[kC * kLD];   // U_out [kd][n], then phi(Q), then S_in^T [n][kd]
    __shared__ __attribute__((aligned(16))) float X1[kC * kLD];   // phi(K)
    __shared__ __attribute__((aligned(16))) float X2[kC * kLD];   // V, then dP, then A
    __shared__ __attribute__((aligned(16))) float X3[kC * kLD];   // dnum
    __shared__ float sW[kC], sZ[kC];
    const int64_t c = blockIdx.x, h = blockIdx.y;
    const int64_t t0 = c * kC;
    const int nvalid = (int)(p.T - t0 < kC ? p.T - t0 : kC);
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    bool beg;
    const int rmax = row_last_begin(p.start, t0, nvalid, beg);
    const uint64_t mb = __ballot(beg);
    const int lastb = mb ? 63 - __builtin_clzll(mb) : -1;    // rows >= lastb continue past the chunk
    const int firstb = mb ? __builtin_ctzll(mb) : kC;        // rows < firstb continue from the previous chunk
    const bool have_u = c + 1 < p.nch, have_s = c > 0;
    const float* uo = p.Y + (have_u ? ((c + 1) * p.H + h) * kStateWords : 0);
    const float* si = p.Sinc + (have_s ? ((c - 1) * p.H + h) * kStateWords : 0);

    // every global load up front
    f32x4 ureg[4], kreg[4], vreg[4], dnreg[4], qreg[4], sreg[4];
    fetch_state(ureg, uo, have_u);
    fetch_rows(kreg, p.k, t0, p.H, h, 0, nvalid);
    fetch_rows(vreg, p.v, t0, p.H, h, 0, nvalid);
    fetch_rows(dnreg, p.dnum, t0, p.H, h, 0, nvalid);
    fetch_rows(qreg, p.q, t0, p.H, h, 0, nvalid);
    fetch_state(sreg, si, have_s);
    if (tid < kC) {
        sW[tid] = have_u ? uo[kC * kC + tid] : 0.0f;
        sZ[tid] = have_s ? si[kC * kC + tid] : 0.0f;
    }
    float dd[4];
    int ri[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int i = 16 * w + 4 * (lane >> 4) + r;
        dd[r] = i < nvalid ? p.dden[(t0 + i) * p.H + h] : 0.0f;
        ri[r] = __shfl(rmax, i, 64);
    }
    phi_rows(kreg, 0, nvalid);
    store_rows<true>(X0, ureg);
    store_rows<true>(X1, kreg);
    store_rows<true>(X2, vreg);
    store_rows<true>(X3, dnreg);
    __syncthreads();

    // ---- phase 1
    f32x4 accK2[4], accV2[4], accP[4];
    zero_acc(accK2);
    zero_acc(accV2);
    zero_acc(accP);
    if (have_u && 16 * w + 15 >= lastb) {
        mfma_rot<true, true>(X2, X0, accK2);                 // sum_n V[j][n] U[kd][n]
        mfma_rot<true, false>(X1, X0, accV2);                // sum_kd K[j][kd] U[kd][n]
    }
    mfma_rot<true, true>(X3, X2, accP, w);                   // sum_n dnum[i][n] V[j][n]
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int i = 16 * w + 4 * (lane >> 4) + r;
#pragma unroll
        for (int jt = 0; jt < 4; ++jt)
            accP[jt][r] = keep_ij(i, 16 * jt + (lane & 15), ri[r], nvalid) ? accP[jt][r] + dd[r] : 0.0f;
    }
    phi_rows(qreg, 0, nvalid);
    __syncthreads();                                         // X0 (U_out), X2 (V) free
    store_rows<true>(X0, qreg);
    acc_to_lds<true>(X2, accP);
    __syncthreads();

    // ---- phase 2
    f32x4 accA[4], accQ1[4], accK1[4];
    zero_acc(accA);
    zero_acc(accQ1);
    zero_acc(accK1);
    mfma_rot<true, true>(X0, X1, accA, w);                   // sum_kd Q[i][kd] K[j][kd]
    mfma_rot<true, false>(X2, X1, accQ1);                    // sum_j dP[i][j] K[j][kd]
    mfma_rot<false, false>(X2, X0, accK1);                   // sum_i dP[i][j] Q[i][kd]
    // this lane's accumulator elements (row, col): A masked; phi'(q) kept for
    // dq; dk (rows j, columns kd) written, with phi'(k) from phi(K)
    float pq[4][4];
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = 16 * w + 4 * (lane >> 4) + r, col = 16 * jt + (lane & 15);
            accA[jt][r] = keep_ij(row, col, ri[r], nvalid) ? accA[jt][r] : 0.0f;
            pq[jt][r] = phi_prime_of_phi(X0[row * kLD + rot_col(row, col)]);
            if (row < nvalid) {
                const float dK = accK1[jt][r] + (row >= lastb ? accK2[jt][r] + sW[col] : 0.0f);
                p.dk[((t0 + row) * p.H + h) * kC + col] = dK * phi_prime_of_phi(X1[row * kLD + rot_col(row, col)]);
            }
        }
    __syncthreads();                                         // X0 (phi(Q)), X2 (dP) free
    store_rows<true>(X0, sreg);
    acc_to_lds<true>(X2, accA);
    __syncthreads();

    // ---- phase 3
    f32x4 accV1[4], accQ2[4];
    zero_acc(accV1);
    zero_acc(accQ2);
    mfma_rot<false, false>(X2, X3, accV1);                   // sum_i A[i][j] dnum[i][n]
    if (have_s && 16 * w < firstb) mfma_rot<true, false>(X3, X0, accQ2);   // sum_n dnum[i][n] S_in[kd][n]
#pragma unroll
    for (int jt = 0; jt < 4; ++jt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int i = 16 * w + 4 * (lane >> 4) + r, col = 16 * jt + (lane & 15);
            if (i < nvalid) {
                p.dv[((t0 + i) * p.H + h) * kC + col] = accV1[jt][r] + (i >= lastb ? accV2[jt][r] : 0.0f);
                const float dQ = accQ1[jt][r] + (ri[r] < 0 ? accQ2[jt][r] + dd[r] * sZ[col] : 0.0f);
                p.dq[((t0 + i) * p.H + h) * kC + col] = dQ * pq[jt][r];
            }
        }
}

hipError_t linattn_bwd_summary_launch(const LinBwdArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(linattn_bwd_summary_kernel, dim3((unsigned)a.nch, (unsigned)a.H), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t linattn_bwd_grad_launch(const LinBwdArgs& a, hipStream_t s) {
    hipLaunchKernelGGL(linattn_bwd_grad_kernel, dim3((unsigned)a.nch, (unsigned)a.H), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace memoroid
