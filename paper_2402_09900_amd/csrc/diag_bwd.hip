// diag_bwd.hip -- single-pass resettable reverse scan of the diagonal
// memoroid (the gradient of diag_fwd.hip), for gfx950.
//
// The derivative of h_t = a_t h_{t-1} + x_t (conjugate convention of complex
// autograd) back-propagates the upstream gradient g = dL/dh as
//     lam_t = g_t                                if t is an episode end,
//     lam_t = conj(a_{t+1}) * lam_{t+1} + g_t    otherwise,
// where an episode end is the last step of the tape or a step followed by a
// begin step; then dx_t = lam_t and da_t = [t not a begin] lam_t conj(h_{t-1}).
// This is the forward scan's machinery mirrored in time: the same tiles, but
// handed out from the end of the tape, each step's coefficient taken from the
// step after it, and episode ends acting as resets.
//
// For a time-invariant a, da is the sum over all tapes and steps; each tile
// writes one deterministic partial per feature and colsum kernels (below) add
// them up in a fixed order.
#include "scan_common.hpp"
#include "kernels.hpp"

namespace memoroid {

template <Kind K, int VEC, int R, bool AINV>
__global__ __launch_bounds__(256) void diag_bwd_kernel(DiagBwdArgs p) {
    using S = typename StateOf<K>::type;
    using C = Codec<K, VEC>;
    constexpr int NT = 256;
    constexpr int EB = KindInfo<K>::bytes;

    __shared__ uint32_t s_ticket;
    __shared__ S sA[NT * VEC];
    __shared__ S sH[NT * VEC];
    __shared__ uint8_t sF[NT];
    __shared__ S sCarry[64 * VEC];

    const int tid = threadIdx.x;
    if (tid == 0) s_ticket = atomicAdd(&p.hdr->ticket, 1u);
    __syncthreads();
    const uint32_t ticket = s_ticket;
    const int chain = (int)(ticket % (uint32_t)p.nchains);
    const int64_t k = ticket / (uint32_t)p.nchains;
    const int64_t tile = p.nt - 1 - k;              // tiles run from the tape end
    const int b = chain / p.nfb;
    const int fb = chain - b * p.nfb;
    const int Qp = p.Qp;
    const int G = NT / Qp;
    const int q = tid & (Qp - 1);
    const int g = tid / Qp;
    const int Dp = Qp * VEC;
    const int64_t L = (int64_t)G * R;
    const int64_t tile_row0 = tile * L;
    const int64_t row0 = tile_row0 + (int64_t)g * R;
    const int64_t f0 = (int64_t)fb * Dp + (int64_t)q * VEC;
    const bool active = f0 < p.d;
    const uint8_t* st = p.start + (int64_t)b * p.T;
    const int64_t T = p.T;
    const int64_t rowbase = (int64_t)b * T;

    // ---- loads: g_t, a_{t+1}, and the flags of steps t and t+1
    RawVec<K, VEC> rg[R];
    RawVec<K, VEC> ra[AINV ? 1 : R];
    uint32_t ends = 0, begins = 0, valid = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t t = row0 + r;
        if (t < T) {
            valid |= 1u << r;
            if (t == 0 || st[t] != 0) begins |= 1u << r;
            const bool end = (t + 1 == T) || st[t + 1] != 0;
            if (end) ends |= 1u << r;
            if (active) {
                raw_load(rg[r], (const char*)p.g + ((rowbase + t) * p.d + f0) * EB);
                if constexpr (!AINV) {
                    if (!end) raw_load(ra[r], (const char*)p.a + ((rowbase + t + 1) * p.d + f0) * EB);
                }
            }
        }
    }
    S ainv[VEC];
    if constexpr (AINV) {
        RawVec<K, VEC> r0;
        if (active) raw_load(r0, (const char*)p.a + f0 * EB);
#pragma unroll
        for (int v = 0; v < VEC; ++v) ainv[v] = active ? conj(C::get(r0, v)) : s_one<S>();
    }
    auto coef = [&](int r, int v) -> S {      // conj(a_{t+1})
        if constexpr (AINV) return ainv[v];
        else return conj(C::get(ra[r], v));
    };

    // ---- per-lane summary, walking its R steps backwards
    S A[VEC], H[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) { A[v] = s_one<S>(); H[v] = s_zero<S>(); }
#pragma unroll
    for (int r = R - 1; r >= 0; --r) {
        if (!((valid >> r) & 1u)) continue;
        const bool e = (ends >> r) & 1u;
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            const S gv = C::get(rg[r], v);
            if (e) {
                A[v] = s_one<S>();
                H[v] = gv;
            } else {
                const S cv = coef(r, v);
                H[v] = mad(cv, H[v], gv);
                A[v] = A[v] * cv;
            }
        }
    }
    const bool f_own = ends != 0;

    // ---- combine groups (later groups come first in scan order)
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        sA[tid * VEC + v] = A[v];
        sH[tid * VEC + v] = H[v];
    }
    sF[tid] = f_own;
    __syncthreads();

    S eA[VEC], eH[VEC];
    bool ef = false;
#pragma unroll
    for (int v = 0; v < VEC; ++v) { eA[v] = s_one<S>(); eH[v] = s_zero<S>(); }
    for (int gg = G - 1; gg > g; --gg) {
        const int j = gg * Qp + q;
        const bool fj = sF[j];
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            const S Aj = sA[j * VEC + v], Hj = sH[j * VEC + v];
            if (fj) {
                eA[v] = Aj;
                eH[v] = Hj;
            } else {
                eH[v] = mad(Aj, eH[v], Hj);
                eA[v] = Aj * eA[v];
            }
        }
        ef = ef || fj;
    }

    // ---- group 0 (earliest steps) holds the tile summary: publish, look back
    if (g == 0) {
        S iA[VEC], iH[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            if (f_own) {
                iA[v] = A[v];
                iH[v] = H[v];
            } else {
                iH[v] = mad(A[v], eH[v], H[v]);
                iA[v] = A[v] * eA[v];
            }
        }
        const bool tile_any = ef || f_own;
        const int64_t di = (int64_t)ticket * Dp + (int64_t)q * VEC;
        if (active) {
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                if (tile_any) Desc<S>::put_incl(p.incl, di + v, iH[v]);
                else Desc<S>::put_agg(p.agg, di + v, iA[v], iH[v]);
            }
        }
        S carry[VEC];
#pragma unroll
        for (int v = 0; v < VEC; ++v) carry[v] = s_zero<S>();
        const int64_t t_last = (tile_row0 + L < T ? tile_row0 + L : T) - 1;
        const bool need_carry = !((t_last + 1 == T) || st[t_last + 1] != 0);
        if (active && need_carry) {
            S accA[VEC], accH[VEC];
#pragma unroll
            for (int v = 0; v < VEC; ++v) { accA[v] = s_one<S>(); accH[v] = s_zero<S>(); }
            int64_t pred = (int64_t)ticket - p.nchains;
            uint32_t polls = 0;
            while (true) {
                const int64_t pi = pred * Dp + (int64_t)q * VEC;
                S ih[VEC];
                bool ok = true;
#pragma unroll
                for (int v = 0; v < VEC; ++v) ok = Desc<S>::get_incl(p.incl, pi + v, ih[v]) && ok;
                if (ok) {
#pragma unroll
                    for (int v = 0; v < VEC; ++v) carry[v] = mad(accA[v], ih[v], accH[v]);
                    break;
                }
                S ga[VEC], gh[VEC];
                ok = true;
#pragma unroll
                for (int v = 0; v < VEC; ++v) ok = Desc<S>::get_agg(p.agg, pi + v, ga[v], gh[v]) && ok;
                if (ok) {
#pragma unroll
                    for (int v = 0; v < VEC; ++v) {
                        accH[v] = mad(accA[v], gh[v], accH[v]);
                        accA[v] = accA[v] * ga[v];
                    }
                    pred -= p.nchains;
                    continue;
                }
                if (++polls > kMaxPolls) {
                    __hip_atomic_store(&p.hdr->timeout, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                __builtin_amdgcn_s_sleep(1);
            }
        }
        if (active && !tile_any) {
#pragma unroll
            for (int v = 0; v < VEC; ++v) Desc<S>::put_incl(p.incl, di + v, mad(iA[v], carry[v], iH[v]));
        }
#pragma unroll
        for (int v = 0; v < VEC; ++v) sCarry[q * VEC + v] = carry[v];
    }
    __syncthreads();

    // ---- replay backwards from the carry-in; emit dx, da
    S lam[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        const S c = sCarry[q * VEC + v];
        lam[v] = ef ? eH[v] : mad(eA[v], c, eH[v]);
    }
    S dsum[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) dsum[v] = s_zero<S>();
    const bool want_da = AINV ? p.da_part != nullptr : p.da != nullptr;
    if (active) {
#pragma unroll
        for (int r = R - 1; r >= 0; --r) {
            if (!((valid >> r) & 1u)) continue;
            const int64_t t = row0 + r;
            const bool e = (ends >> r) & 1u;
            const bool bg = (begins >> r) & 1u;
            RawVec<K, VEC> hprev;
            if (want_da && !bg) raw_load(hprev, (const char*)p.h + ((rowbase + t - 1) * p.d + f0) * EB);
            RawVec<K, VEC> odx, oda;
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                const S gv = C::get(rg[r], v);
                lam[v] = e ? gv : mad(coef(r, v), lam[v], gv);
                C::put(odx, v, lam[v]);
                const S dav = bg ? s_zero<S>() : lam[v] * conj(C::get(hprev, v));
                if constexpr (AINV) dsum[v] = dsum[v] + dav;
                else C::put(oda, v, dav);
            }
            const int64_t off = ((rowbase + t) * p.d + f0) * EB;
            raw_store_nt((char*)p.dx + off, odx);
            if constexpr (!AINV) {
                if (want_da) raw_store_nt((char*)p.da + off, oda);
            }
        }
    }
    if constexpr (AINV) {
        if (want_da) {
            // deterministic per-tile partial: sum the groups in a fixed order
            __syncthreads();
#pragma unroll
            for (int v = 0; v < VEC; ++v) sH[tid * VEC + v] = dsum[v];
            __syncthreads();
            if (g == 0 && active) {
                RawVec<K, VEC> o;
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    S s = s_zero<S>();
                    for (int gg = 0; gg < G; ++gg) s = s + sH[(gg * Qp + q) * VEC + v];
                    C::put(o, v, s);
                }
                // partial row = (tile, tape); columns = the d features
                const int64_t prow = tile * (p.nchains / p.nfb) + b;
                raw_store_nt((char*)p.da_part + (prow * p.d + f0) * EB, o);
            }
        }
    }
}

// Column sums of a row-major [rows][cols] float matrix, `chunk` rows per
// thread, in row order: out[(r / chunk)][c] = sum of rows r .. r+chunk-1.
__global__ __launch_bounds__(256) void colsum_kernel(const float* in, float* out, int64_t rows,
                                                     int64_t cols, int64_t chunk) {
    const int64_t c = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t r0 = (int64_t)blockIdx.y * chunk;
    if (c >= cols) return;
    const int64_t r1 = r0 + chunk < rows ? r0 + chunk : rows;
    float s = 0.0f;
    for (int64_t r = r0; r < r1; ++r) s += in[r * cols + c];
    out[(int64_t)blockIdx.y * cols + c] = s;
}

// ------------------------------------------------------------------ launch

template <Kind K, int VEC, int R>
static hipError_t launch_bwd(const DiagBwdArgs& args, int64_t ntiles, bool ainv, hipStream_t s) {
    if (ainv)
        hipLaunchKernelGGL((diag_bwd_kernel<K, VEC, R, true>), dim3((unsigned)ntiles), dim3(256), 0, s, args);
    else
        hipLaunchKernelGGL((diag_bwd_kernel<K, VEC, R, false>), dim3((unsigned)ntiles), dim3(256), 0, s, args);
    return hipGetLastError();
}

hipError_t diag_bwd_launch(int kind, bool vec, bool ainv, const DiagBwdArgs& args, int64_t ntiles,
                           hipStream_t s) {
    constexpr int R = kBwdRows;
    if (kind == K_F32)
        return vec ? launch_bwd<K_F32, 4, R>(args, ntiles, ainv, s) : launch_bwd<K_F32, 1, R>(args, ntiles, ainv, s);
    if (kind == K_C64)
        return vec ? launch_bwd<K_C64, 2, R>(args, ntiles, ainv, s) : launch_bwd<K_C64, 1, R>(args, ntiles, ainv, s);
    return hipErrorInvalidValue;
}

hipError_t colsum_launch(const float* in, float* out, int64_t rows, int64_t cols, int64_t chunk,
                         hipStream_t s) {
    const int64_t nchunks = (rows + chunk - 1) / chunk;
    dim3 grid((unsigned)((cols + 255) / 256), (unsigned)nchunks);
    hipLaunchKernelGGL(colsum_kernel, grid, dim3(256), 0, s, in, out, rows, cols, chunk);
    return hipGetLastError();
}

}  // namespace memoroid
