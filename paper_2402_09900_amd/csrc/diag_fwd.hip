// diag_fwd.hip -- single-pass resettable scan of the diagonal memoroid,
// forward direction, for gfx950.
//
// Recurrence (S5 / LRU / FFM memoroids of App. G.2-G.4 with a diagonal
// transition, under the reset transform of the Section 4 theorem):
//     h_t = x_t                   at a begin step,
//     h_t = a_t * h_{t-1} + x_t   otherwise.
//
// Work decomposition
//   chain  = (tape b, feature block fb): an independent scan over T steps of
//            Dp = Qp * VEC features; blocks are as wide as one wavefront row
//            (64 lanes x 16 bytes) so every row access is a coalesced burst.
//   tile   = L = G * R consecutive steps of one chain, one workgroup.  Lane q
//            of group g owns VEC features and R consecutive steps; groups are
//            consecutive in time (for Qp = 64 a group is one wavefront).
//   ticket = tiles are numbered by an atomic counter in launch order,
//            interleaving chains (ticket = tile * nchains + chain), so every
//            tile a workgroup waits for was handed to a workgroup that is
//            already running or finished.
//
// Per tile: (1) load a, x for all R steps into registers with one wide load
// per step; (2) each lane folds its R steps into a summary (A, H, any-begin);
// (3) groups combine their summaries through LDS into exclusive prefixes and
// the tile summary; (4) the last group publishes the tile summary to the
// workspace at once -- as the inclusive prefix if the tile holds a begin step
// (nothing older can reach past it), else as an aggregate -- then looks back
// over predecessor tiles of its chain, folding aggregates until it meets an
// inclusive prefix, and publishes its own inclusive prefix; (5) every lane
// replays its R steps from its carry-in and streams h out.  a and x are read
// from HBM once and h written once; the cross-tile traffic is a few words per
// feature per tile.
#include "scan_common.hpp"
#include "kernels.hpp"

namespace memoroid {

template <Kind IN, Kind OUT, int VEC, int R, bool AINV>
__global__ __launch_bounds__(256) void diag_fwd_kernel(DiagFwdArgs p) {
    using S = typename StateOf<IN>::type;
    using CIn = Codec<IN, VEC>;
    using COut = Codec<OUT, VEC>;
    constexpr int NT = 256;
    constexpr int IB = KindInfo<IN>::bytes;
    constexpr int OB = KindInfo<OUT>::bytes;

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
    const int64_t tile = ticket / (uint32_t)p.nchains;
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

    // ---- (1) loads: one wide access per step and tensor
    RawVec<IN, VEC> ra[AINV ? 1 : R];
    RawVec<IN, VEC> rx[R];
    uint32_t begins = 0, valid = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t t = row0 + r;
        if (t < p.T) {
            valid |= 1u << r;
            if (t == 0 || st[t] != 0) begins |= 1u << r;
            if (active) {
                const int64_t off = ((int64_t)b * p.T + t) * p.d + f0;
                raw_load(rx[r], (const char*)p.x + off * IB);
                if constexpr (!AINV) raw_load(ra[r], (const char*)p.a + off * IB);
            }
        }
    }
    S ainv[VEC];
    if constexpr (AINV) {
        RawVec<IN, VEC> r0;
        if (active) raw_load(r0, (const char*)p.a + f0 * IB);
#pragma unroll
        for (int v = 0; v < VEC; ++v) ainv[v] = active ? CIn::get(r0, v) : s_one<S>();
    }
    auto a_at = [&](int r, int v) -> S {
        if constexpr (AINV) return ainv[v];
        else return CIn::get(ra[r], v);
    };

    // ---- (2) per-lane summary of R steps
    S A[VEC], H[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) { A[v] = s_one<S>(); H[v] = s_zero<S>(); }
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if (!((valid >> r) & 1u)) continue;
        const bool bg = (begins >> r) & 1u;
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            const S xv = CIn::get(rx[r], v);
            if (bg) {
                A[v] = s_one<S>();
                H[v] = xv;
            } else {
                const S av = a_at(r, v);
                H[v] = mad(av, H[v], xv);
                A[v] = A[v] * av;
            }
        }
    }
    const bool f_own = begins != 0;

    // ---- (3) combine groups through LDS
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
    for (int gg = 0; gg < g; ++gg) {
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

    // ---- (4) publish, look back, publish inclusive
    if (g == G - 1) {
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
        const bool need_carry = !(tile_row0 == 0 || st[tile_row0] != 0);
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

    // ---- (5) replay from the carry-in and stream h out
    S hv[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        const S c = sCarry[q * VEC + v];
        hv[v] = ef ? eH[v] : mad(eA[v], c, eH[v]);
    }
    if (!active) return;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if (!((valid >> r) & 1u)) continue;
        const bool bg = (begins >> r) & 1u;
        RawVec<OUT, VEC> o;
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            const S xv = CIn::get(rx[r], v);
            hv[v] = bg ? xv : mad(a_at(r, v), hv[v], xv);
            COut::put(o, v, hv[v]);
        }
        const int64_t off = ((int64_t)b * p.T + row0 + r) * p.d + f0;
        raw_store_nt((char*)p.h + off * OB, o);
    }
}

// ------------------------------------------------------------------ launch

template <Kind IN, Kind OUT, int VEC, int R>
static hipError_t launch_fwd(const DiagFwdArgs& args, int64_t ntiles, bool ainv, hipStream_t s) {
    if (ainv)
        hipLaunchKernelGGL((diag_fwd_kernel<IN, OUT, VEC, R, true>), dim3((unsigned)ntiles), dim3(256), 0, s, args);
    else
        hipLaunchKernelGGL((diag_fwd_kernel<IN, OUT, VEC, R, false>), dim3((unsigned)ntiles), dim3(256), 0, s, args);
    return hipGetLastError();
}

int diag_fwd_rows_per_lane(int in_kind) {
    (void)in_kind;
    return kFwdRows;
}

hipError_t diag_fwd_launch(int in_kind, int out_kind, bool vec, bool ainv,
                           const DiagFwdArgs& args, int64_t ntiles, hipStream_t s) {
    constexpr int R = kFwdRows;
    if (in_kind == K_F32 && out_kind == K_F32)
        return vec ? launch_fwd<K_F32, K_F32, 4, R>(args, ntiles, ainv, s)
                   : launch_fwd<K_F32, K_F32, 1, R>(args, ntiles, ainv, s);
    if (in_kind == K_BF16 && out_kind == K_BF16)
        return vec ? launch_fwd<K_BF16, K_BF16, 8, R>(args, ntiles, ainv, s)
                   : launch_fwd<K_BF16, K_BF16, 1, R>(args, ntiles, ainv, s);
    if (in_kind == K_BF16 && out_kind == K_F32)
        return vec ? launch_fwd<K_BF16, K_F32, 8, R>(args, ntiles, ainv, s)
                   : launch_fwd<K_BF16, K_F32, 1, R>(args, ntiles, ainv, s);
    if (in_kind == K_C64 && out_kind == K_C64)
        return vec ? launch_fwd<K_C64, K_C64, 2, R>(args, ntiles, ainv, s)
                   : launch_fwd<K_C64, K_C64, 1, R>(args, ntiles, ainv, s);
    return hipErrorInvalidValue;
}

}  // namespace memoroid
