// diag_bwd.hip -- single-pass resettable reverse scan of the diagonal
// memoroid (the gradient of diag_fwd.hip), for gfx950.
//
// The derivative of h_t = a_t h_{t-1} + x_t (conjugate convention of complex
// autograd) back-propagates the upstream gradient g = dL/dh as
//     lam_t = g_t                                if t is an episode end,
//     lam_t = conj(a_{t+1}) * lam_{t+1} + g_t    otherwise,
// where an episode end is the last step of the tape or a step followed by a
// begin step; then dx_t = lam_t and da_t = [t not a begin] lam_t conj(h_{t-1}).
// This is the forward scan's machinery (diag_fwd.hip) mirrored in time: the
// same tiles, handed out from the end of the tape, each step's coefficient
// taken from the step after it, and episode ends acting as resets; the same
// never-reset counters, epoch banks and workspace binding.
//
// For a time-invariant a, da is the sum over all tapes and steps; each tile
// writes one partial per feature, summed inside the tile in a fixed order, and
// colsum kernels (below) add the partials up in a fixed order too, so the
// result does not depend on timing.
#include <type_traits>

#include "scan_common.hpp"
#include "kernels.hpp"

namespace memoroid {

template <Kind K, int VEC, int R, bool AINV, bool FFM = false>
__global__ __launch_bounds__(256) void diag_bwd_kernel(DiagBwdArgs p) {
    static_assert(!FFM || (K == K_C64 && AINV), "FFM: complex state, generated a");
    static_assert(R >= 1 && R <= 32, "a lane's steps are bits of 32-bit masks");
    using S = typename StateOf<K>::type;
    using C = Codec<K, VEC>;
    using SegT = Seg<S, VEC>;
    constexpr int NT = 256;
    constexpr int NW = NT / 64;
    constexpr int EB = KindInfo<K>::bytes;
    // widest lane group of this kernel's plans: one chain row of VEC-wide lanes
    constexpr int kQpMax = kChainRowBytes / (VEC * EB) > 0 ? (int)(kChainRowBytes / (VEC * EB)) : 1;

    __shared__ uint32_t s_ticket;          // place in the chain; all ones: stand down
    __shared__ uint32_t s_bank;
    __shared__ S sWA[NW][64 * VEC];
    __shared__ S sWH[NW][64 * VEC];
    __shared__ uint32_t sWF[NW];
    __shared__ S sCarry[64 * VEC];
    __shared__ LookbackLds<S, VEC> sLb;
    __shared__ cf sFfm[FFM ? 64 : 1];      // FFM conj(a) of the chain's features

    const int tid = threadIdx.x;
    // the workgroup's chain is fixed by its index (each run of nchains
    // consecutive workgroups covers every chain once, rotated by one per run
    // so that no chain stays on one XCD); its place in the chain comes from
    // the chain's own counter, in the order tiles start
    const uint32_t nch = (uint32_t)p.nchains;
    const int chain = (int)((blockIdx.x % nch + blockIdx.x / nch) % nch);
    if (tid == 0) {
        // the signature load goes first: the compiler waits for the atomic's
        // result right after issuing it, and both round trips then overlap
        const uint64_t seen = peek_sig(p.hdr);
        const Claim c = claim_of(take_ticket(p.ctr + (size_t)chain * kCtrStride, (uint32_t)p.nt), (uint32_t)p.nt);
        const bool bound = ws_bound_to(p.hdr, p.sig, seen, chain == 0 && c.pos == 0);
        s_ticket = bound ? c.pos : kEmpty32;
        s_bank = c.bank;
    }
    barrier_lds();
    const uint32_t claimed = __builtin_amdgcn_readfirstlane(s_ticket);
    if (claimed == kEmpty32) return;       // workspace bound to another call: every tile stands down
    const int64_t k = (int64_t)claimed;
    const uint32_t ticket = (uint32_t)(k * p.nchains + chain);
    const int64_t boff = __builtin_amdgcn_readfirstlane(s_bank) ? p.bank : 0;
    const int64_t bidle = p.bank - boff;
    void* const agg = (char*)p.agg + boff;
    void* const incl = (char*)p.incl + boff;
    const int64_t tile = p.nt - 1 - k;              // tiles run from the tape end
    const int b = chain / p.nfb;
    const int fb = chain - b * p.nfb;
    const int Qp = p.Qp;
    const int qsh = __builtin_ctz((unsigned)Qp);   // Qp is a power of two
    const int Gw = 64 >> qsh;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    const int q = lane & (Qp - 1);
    const int j = lane >> qsh;
    const int Dp = Qp * VEC;
    const int64_t L = (int64_t)NW * Gw * R;
    const int64_t tile_row0 = tile * L;
    const int64_t row0 = tile_row0 + (int64_t)(wave * Gw + j) * R;
    const int64_t f0 = (int64_t)fb * Dp + (int64_t)q * VEC;
    const bool active = f0 < p.d;
    const uint8_t* st = p.start + (int64_t)b * p.T;
    const int64_t T = p.T;
    const int64_t rowbase = (int64_t)b * T;
    const bool want_da = AINV ? p.da_part != nullptr : p.da != nullptr;

    // ---- loads, through buffer resources based at the tile's first step of
    // this tape: rows past T and lanes past d read zeros and their stores are
    // dropped, and so are a_{t+1} at t + 1 = T and h_{t-1} at t = 0 (offsets
    // out of range; both are unused there).  The begin flags of the lane's
    // steps t and t+1 (and of the step after the tile) go first, so that
    // waiting for them leaves every data load in flight; then g_t, a_{t+1}
    // and h_{t-1} of every step, one wide access each.
    const int64_t rows_left = T - tile_row0;
    const int64_t tape_row0 = rowbase + tile_row0;
    const int64_t rowB = p.d * EB;
    const uint32_t lrow = (uint32_t)((wave * Gw + j) * R);
    const Rsrc rs_st = make_rsrc(st + tile_row0, rows_left);
    const Rsrc rs_g = make_rsrc((const char*)p.g + tape_row0 * rowB, rows_left * rowB);
    const Rsrc rs_a = make_rsrc(AINV ? p.g : (const char*)p.a + tape_row0 * rowB, AINV ? 0 : rows_left * rowB);
    // h_{t-1}: based one step before the tile (when there is one), so the
    // tile's first step reads the previous tile's last h
    const int64_t h_back = tile_row0 > 0 ? 1 : 0;
    const Rsrc rs_h = make_rsrc(want_da ? (const char*)p.h + (tape_row0 - h_back) * rowB : p.g,
                                want_da ? (rows_left + h_back) * rowB : 0);
    const uint32_t step = active ? (uint32_t)rowB : 0u;
    const uint32_t off0 = active ? (uint32_t)((int64_t)lrow * rowB + f0 * EB) : kOob;
    // the previous tile's inclusive words, ahead of everything else (the
    // look-back below is skipped when they were all published)
    S spec[VEC];
    bool spec_ok = false;
    if (wave == NW - 1 && j == 0 && active && k > 0)
        spec_ok = peek_incl_ahead<S, VEC>(incl, (int64_t)ticket - p.nchains, Dp, Qp, q, spec);
    // FFM: the parameters of the chain's transitions, ahead of the tile's
    // loads, so that the table need not wait for them
    FfmParam fpar{0.f, 0.f};
    if constexpr (FFM) fpar = ffm_param_load(p.alpha, p.omega, p.d, p.ffm_c, (int64_t)fb * Dp, Dp);
    uint32_t fl[R + 1];
#pragma unroll
    for (int r = 0; r <= R; ++r) fl[r] = bload_u8(rs_st, lrow + r);
    const int64_t t_last = (tile_row0 + L < T ? tile_row0 + L : T) - 1;
    const uint32_t fl_after = bload_u8(rs_st, (uint32_t)(t_last + 1 - tile_row0));
    __builtin_amdgcn_sched_barrier(0);
    RawVec<K, VEC> rg[R];
    RawVec<K, VEC> ra[AINV ? 1 : R];
    RawVec<K, VEC> rh[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const uint32_t off = off0 + r * step;
        raw_bload(rg[r], rs_g, off);
        if constexpr (!AINV) raw_bload(ra[r], rs_a, off + step);
        if (want_da) raw_bload(rh[r], rs_h, h_back ? off : off - step);
    }
    __builtin_amdgcn_sched_barrier(0);
    uint32_t ends = 0, begins = 0, valid = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t t = row0 + r;
        const uint32_t in = t < T ? 1u : 0u;
        valid |= in << r;
        begins |= (in & ((t == 0 ? 1u : 0u) | (fl[r] != 0u ? 1u : 0u))) << r;
        ends |= (in & ((t + 1 == T ? 1u : 0u) | (fl[r + 1] != 0u ? 1u : 0u))) << r;
    }
    S ainv[VEC];
    if constexpr (FFM) {
        // conj(a) of the chain's features, evaluated once per tile as in the
        // forward pass
        if constexpr (std::is_same<S, cf>::value) {
            ffm_table_store(sFfm, fpar, Dp, true);
            barrier_lds();
#pragma unroll
            for (int v = 0; v < VEC; ++v) ainv[v] = sFfm[q * VEC + v];
        }
    } else if constexpr (AINV) {
        // a NULL time-invariant a stands for a = 1 (the reverse sum, used by
        // the linear-attention gradient's state scan)
        RawVec<K, VEC> r0;
        const bool have = active && p.a != nullptr;
        if (have) raw_load(r0, (const char*)p.a + f0 * EB);
#pragma unroll
        for (int v = 0; v < VEC; ++v) ainv[v] = have ? conj(C::get(r0, v)) : s_one<S>();
    }
    auto coef = [&](int r, int v) -> S {      // conj(a_{t+1})
        if constexpr (AINV) return ainv[v];
        else return conj(C::get(ra[r], v));
    };

    // ---- per-lane summary, walking its R steps backwards.  Steps past T
    // hold zeros and come before the tape's last step, which ends an episode,
    // so they never reach a real output.
    //
    // With a time-invariant complex a the fold also takes from h all that da
    // needs, so h is not held across the look-back (and for FFM neither is
    // g); the real kernels keep the plain replay, whose registers this would
    // raise.
    // With lam_in the adjoint that enters the lane's last step,
    // lam_t = l_t + c_t lam_in, where l_t is the lane's own recurrence from
    // zero (own.H after step t) and c_t the product of conj(a) over steps t..
    // up to the lane's last, zero from its first end downwards.  Kept:
    // D1 = sum_t l_t conj(h_{t-1}) and D2 = sum_t c_t conj(h_{t-1}) (da's
    // partial is D1 + lam_in D2), and for FFM sum_v Re(l_t) per step (the
    // input gradient adds Re over the lane's features, which share one row j).
    constexpr bool kFoldDa = AINV && std::is_same<S, cf>::value;
    constexpr int RF = FFM ? R : 1;
    float lre[RF];
    S d1[VEC], d2[VEC], cp[VEC];
    bool alive = true, d2_live = false;      // c_t not forced to zero yet / some term of D2 counts
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        d1[v] = s_zero<S>();
        d2[v] = s_zero<S>();
        cp[v] = s_one<S>();
    }
    SegT own = seg_identity<S, VEC>();
#pragma unroll
    for (int r = R - 1; r >= 0; --r) {
        const bool e = (ends >> r) & 1u;
        // no da at a begin step, nor past T (a select: the step T reads
        // h_{T-1}, and 0 * Inf would reach the sum)
        const bool no_da = ((begins | ~valid) >> r) & 1u;
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            const S gv = C::get(rg[r], v);
            const S cv = coef(r, v);
            const S nh = mad(cv, own.H[v], gv);
            const S na = own.A[v] * cv;
            own.H[v] = e ? gv : nh;
            own.A[v] = e ? s_one<S>() : na;
            if constexpr (kFoldDa) {
                const S ncp = cv * cp[v];
                cp[v] = e ? s_zero<S>() : ncp;
                if (want_da) {
                    const S hc = conj(C::get(rh[r], v));
                    d1[v] = no_da ? d1[v] : mad(own.H[v], hc, d1[v]);
                    d2[v] = no_da ? d2[v] : mad(cp[v], hc, d2[v]);
                }
            }
        }
        if constexpr (kFoldDa) {
            alive = alive && !e;
            d2_live = d2_live || (alive && !no_da);
        }
        if constexpr (FFM) {
            float sre = 0.0f;
#pragma unroll
            for (int v = 0; v < VEC; ++v) sre += re_part(own.H[v]);
            lre[r] = sre;
        }
    }
    own.f = ends != 0;

    // ---- scan the wavefront's groups (later groups first), then combine the
    // wavefront totals (later wavefronts first) through LDS
    SegT inc = own, exc;
    wave_group_scan<S, VEC, true, kQpMax>(inc, exc, Qp);
    if (j == 0) {
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            sWA[wave][q * VEC + v] = inc.A[v];
            sWH[wave][q * VEC + v] = inc.H[v];
        }
        if (q == 0) sWF[wave] = inc.f;
    }
    barrier_lds();
    auto wave_total = [&](int w) -> SegT {
        SegT t;
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            t.A[v] = sWA[w][q * VEC + v];
            t.H[v] = sWH[w][q * VEC + v];
        }
        t.f = sWF[w] != 0;
        return t;
    };
    SegT before = seg_identity<S, VEC>();        // later steps of the tile, in scan order
    for (int w = NW - 1; w > wave; --w) before = seg_then<S, VEC>(before, wave_total(w));
    const SegT pre = seg_then<S, VEC>(before, exc);

    // ---- wavefront 0 publishes the tile summary; the last wavefront looks
    // back for the carry from the later tiles (publishing and polling use
    // different wavefronts: loads and stores share one completion counter)
    const bool summary_lane = wave == 0 && j == 0 && active;
    SegT tot = seg_identity<S, VEC>();
    if (wave == 0) {
        tot = seg_then<S, VEC>(before, wave_total(0));
        if (summary_lane) {
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                if (tot.f) Desc<S>::put_incl(incl, desc_slot(ticket, Dp, Qp, q, v), tot.H[v]);
                else Desc<S>::put_agg(agg, desc_slot(ticket, Dp, Qp, q, v), tot.A[v], tot.H[v]);
            }
#pragma unroll
            for (int v = 0; v < VEC; ++v)
                Desc<S>::clear((char*)p.agg + bidle, (char*)p.incl + bidle, desc_slot(ticket, Dp, Qp, q, v));
        }
    }
    if (wave == NW - 1) {
        const bool need_carry = !((t_last + 1 == T) || fl_after != 0);
        S carry[VEC];
        if (need_carry && __all(j != 0 || !active || spec_ok)) {
#pragma unroll
            for (int v = 0; v < VEC; ++v) carry[v] = active ? spec[v] : s_zero<S>();
        } else {
            lookback<S, VEC>(agg, incl, (int64_t)ticket - p.nchains, p.nchains, Dp, Qp, need_carry && active, carry,
                             sLb, &p.hdr->timeout);
        }
        if (j == 0) {
#pragma unroll
            for (int v = 0; v < VEC; ++v) sCarry[q * VEC + v] = carry[v];
        }
    }
    barrier_lds();

    // ---- the tile's inclusive prefix goes out first; then replay backwards
    // from the carry-in and emit dx (built in the registers that held g) and
    // da (in those that held a), so no store waits on another
    S lam[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        const S c = sCarry[q * VEC + v];
        if (summary_lane && !tot.f)
            Desc<S>::put_incl(incl, desc_slot(ticket, Dp, Qp, q, v), mad(tot.A[v], c, tot.H[v]));
        lam[v] = seg_apply<S, VEC>(pre, v, c);
    }
    S dsum[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) dsum[v] = s_zero<S>();
    if (active) {
        // the adjoint entering the lane's last step, lam_in, completes what
        // the fold kept: da adds lam_in D2 (a select: when no term of D2
        // counts, a non-finite lam_in cut off by an end stays out)
        if constexpr (kFoldDa) {
#pragma unroll
            for (int v = 0; v < VEC; ++v) dsum[v] = d2_live ? mad(lam[v], d2[v], d1[v]) : d1[v];
        }
        if constexpr (FFM) {
            // lam_t = l_t + m_t with m_t = c_t lam_in, run down from lam_in
            // (reset to zero by a select at an end)
            // x is real and broadcast over the c columns of its row j: its
            // gradient is the sum of Re(lam) over those columns.  c is a power
            // of two and at least VEC (the host picks one feature per lane
            // otherwise), so a lane's features share one j and groups of
            // c / VEC lanes are combined by shuffles.  The chain's jpc = Dp / c
            // rows go to the chain-major workspace [chain][T][jpc], so that a
            // tile writes whole lines (ffm_bwd_finish_kernel puts them in
            // [B][T][m] order).
            const int64_t cc = p.ffm_c;
            const int csh = __builtin_ctzll((uint64_t)cc);
            const int64_t jpc = Dp >> csh;
            const int gsz = (int)(cc / VEC);
            float* const dxw = p.dxr + (int64_t)chain * T * jpc;
#pragma unroll
            for (int r = R - 1; r >= 0; --r) {
                const int64_t t = row0 + r;
                const bool e = (ends >> r) & 1u;
                float part = lre[r];
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    const S nm = coef(r, v) * lam[v];
                    lam[v] = e ? s_zero<S>() : nm;
                    part += re_part(lam[v]);
                }
                for (int off = 1; off < gsz; off <<= 1) part += lanes_xor(part, off);
                if (t < T && (q & (gsz - 1)) == 0) dxw[t * jpc + ((q * VEC) >> csh)] = part;
            }
        } else {
#pragma unroll
            for (int r = R - 1; r >= 0; --r) {
                const bool e = (ends >> r) & 1u;
                // no da at a begin step, nor past T: there lam is 0, but the
                // step T reads h_{T-1}, and 0 * Inf would reach the sum
                const bool no_da = ((begins | ~valid) >> r) & 1u;
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    const S gv = C::get(rg[r], v);
                    lam[v] = e ? gv : mad(coef(r, v), lam[v], gv);
                    if constexpr (!kFoldDa) {
                        const S dav = no_da ? s_zero<S>() : lam[v] * conj(C::get(rh[r], v));
                        if constexpr (AINV) dsum[v] = dsum[v] + dav;
                        else C::put(ra[r], v, dav);
                    }
                    C::put(rg[r], v, lam[v]);
                }
            }
            const Rsrc rs_dx = make_rsrc((char*)p.dx + tape_row0 * rowB, rows_left * rowB);
            const Rsrc rs_da = make_rsrc(AINV ? p.dx : (char*)p.da + tape_row0 * rowB, AINV ? 0 : rows_left * rowB);
#pragma unroll
            for (int r = R - 1; r >= 0; --r) {
                raw_bstore_nt(rs_dx, off0 + r * step, rg[r]);
                if constexpr (!AINV) {
                    if (want_da) raw_bstore_nt(rs_da, off0 + r * step, ra[r]);
                }
            }
        }
    }
    if constexpr (AINV) {
        if (want_da) {
            // per-tile partial of da, summed over the tile's lanes in a fixed
            // order (wavefront, then group)
            __syncthreads();
#pragma unroll
            for (int v = 0; v < VEC; ++v) sWH[wave][lane * VEC + v] = dsum[v];
            __syncthreads();
            if (wave == 0 && j == 0 && active) {
                RawVec<K, VEC> o;
                S sv[VEC];
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    S s = s_zero<S>();
                    for (int w = 0; w < NW; ++w)
                        for (int jj = 0; jj < Gw; ++jj) s = s + sWH[w][(jj * Qp + q) * VEC + v];
                    sv[v] = s;
                    C::put(o, v, s);
                }
                // partial row = (tile, tape); columns = the d features
                const int64_t prow = tile * (p.nchains / p.nfb) + b;
                if (p.da_out) {
                    // self-validating words, banked like the descriptors
                    uint64_t* const cur = (uint64_t*)((char*)p.da_part + boff);
                    uint64_t* const idle = (uint64_t*)((char*)p.da_part + bidle);
#pragma unroll
                    for (int v = 0; v < VEC; ++v) {
                        publish64(cur + prow * p.d + f0 + v, pack_state(sv[v]));
                        idle[prow * p.d + f0 + v] = kEmpty64;
                    }
                } else {
                    raw_store_nt((char*)p.da_part + (prow * p.d + f0) * EB, o);
                }
            }
            if (p.da_out && k == p.nt - 1) {
                // the chain's last tile (its ticket was handed out last, so
                // every other tile of the chain is running or done) sums the
                // chain's partial rows.  Thread (group g, slot fs) takes the
                // feature fb * Dp + fs of tiles g, g + G, ... (G = 256 / Dp),
                // eight loads in flight at a time; the groups are then added
                // in order through LDS, so the result does not depend on timing.
                const int fs = tid % Dp, G = NT / Dp, grp = tid / Dp;
                const int64_t f = (int64_t)fb * Dp + fs;
                const bool fin = f < p.d;
                const uint64_t* const part = (const uint64_t*)((const char*)p.da_part + boff);
                S acc = s_zero<S>();
                uint32_t polls = 0;
                for (int64_t base = grp; base < p.nt; base += 8 * (int64_t)G) {
                    uint64_t wd[8];
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        const int64_t tl = base + (int64_t)i * G;
                        wd[i] = (fin && tl < p.nt) ? peek64(part + tl * p.d + f) : 0ull;
                    }
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        const int64_t tl = base + (int64_t)i * G;
                        while (wd[i] == kEmpty64) {
                            if (++polls > kMaxPolls) {
                                flag_timeout(&p.hdr->timeout);
                                wd[i] = 0ull;
                            } else {
                                __builtin_amdgcn_s_sleep(1);
                                wd[i] = peek64(part + tl * p.d + f);
                            }
                        }
                        acc = acc + unpack_state<S>(wd[i]);
                    }
                }
                __syncthreads();                     // sWH is free again
                S* red = &sWH[0][0];
                red[tid] = acc;
                __syncthreads();
                if (grp == 0 && fin) {
                    S tot2 = s_zero<S>();
                    for (int g2 = 0; g2 < G; ++g2) tot2 = tot2 + red[g2 * Dp + fs];
                    if constexpr (std::is_same<S, cf>::value) {
                        ((float*)p.da_out)[2 * f] = tot2.re;
                        ((float*)p.da_out)[2 * f + 1] = tot2.im;
                    } else {
                        ((float*)p.da_out)[f] = tot2;
                    }
                }
            }
        }
    }
}

// Column sums of a row-major [rows][cols] float matrix over blocks of
// 4 * rpw rows: out[r / (4 rpw)][c] = sum of rows r .. r + 4 rpw - 1 of column
// c.  A workgroup takes 64 columns; each of its four wavefronts adds rpw
// consecutive rows (loads issued 16 at a time), then the four partial sums
// are added in wavefront order, so the result does not depend on timing.
__global__ __launch_bounds__(256) void colsum_kernel(const float* in, float* out, int64_t rows,
                                                     int64_t cols, int64_t rpw) {
    __shared__ float part[4][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int64_t c = (int64_t)blockIdx.x * 64 + lane;
    const int64_t r0 = (int64_t)blockIdx.y * 4 * rpw + w * rpw;
    float s = 0.0f;
    if (c < cols) {
        for (int64_t i0 = 0; i0 < rpw; i0 += 16) {
            float v[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int64_t r = r0 + i0 + i;
                v[i] = (i0 + i < rpw && r < rows) ? in[r * cols + c] : 0.0f;
            }
#pragma unroll
            for (int i = 0; i < 16; ++i) s += v[i];
        }
    }
    part[w][lane] = s;
    __syncthreads();
    if (w == 0 && c < cols) out[(int64_t)blockIdx.y * cols + c] = ((part[0][lane] + part[1][lane]) + part[2][lane]) + part[3][lane];
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

hipError_t ffm_bwd_launch(bool vec, const DiagBwdArgs& args, int64_t ntiles, hipStream_t s) {
    constexpr int RI = kFfmBwdRows;
    if (vec)
        hipLaunchKernelGGL((diag_bwd_kernel<K_C64, KindInfo<K_C64>::vec, RI, true, true>), dim3((unsigned)ntiles),
                           dim3(256), 0, s, args);
    else
        hipLaunchKernelGGL((diag_bwd_kernel<K_C64, 1, RI, true, true>), dim3((unsigned)ntiles), dim3(256), 0, s, args);
    return hipGetLastError();
}

// One workgroup: thread j < m forms dalpha[j], thread k < c forms domega[k]
// (loops over the other index), from the summed complex da[m][c].
// dα_j = -sign(α_j) Σ_k Re(conj(γ_jk) da_jk) and dω_k = Σ_j Im(conj(γ_jk) da_jk)
// with γ_jk = exp(-|α_j|) e^{iω_k}, in double.  One workgroup (all 256
// threads call it): |γ| per row and (cos, sin) per column are evaluated once
// into LDS, in parallel, so that the sums are plain multiply-adds (the same
// operations in the same order as evaluating them inside the sums).
constexpr int kParamRows = 1024, kParamCols = 256, kParamDa = 4096;
// The finish kernel's LDS, shared by its two kinds of workgroup: the
// parameter tables (and da) of the last one, the row block of the others.
constexpr int kFinRows = 256;          // steps per copying workgroup
constexpr int kFinLdsCols = 32;        // m up to this: rows gathered in LDS
constexpr int kFinBatch = 16;          // gather loads in flight per thread
constexpr int kParamLdsBytes = kParamRows * 8 + 2 * kParamCols * 8 + kParamDa * 4;
constexpr int kBlockLdsBytes = kFinRows * kFinLdsCols * 4;
constexpr int kFinLdsBytes = kParamLdsBytes > kBlockLdsBytes ? kParamLdsBytes : kBlockLdsBytes;

__device__ void ffm_param_grad(const float* alpha, const float* omega, const float* da_g, int64_t m, int64_t c,
                               float* dalpha, float* domega, unsigned char* lds) {
    double* const s_mag = (double*)lds;
    double* const s_cs = s_mag + kParamRows;
    double* const s_sn = s_cs + kParamCols;
    float* const s_da = (float*)(s_sn + kParamCols);   // da as well, when it fits (loaded once, coalesced)
    const bool tab = m <= kParamRows && c <= kParamCols;
    const bool lds_da = 2 * m * c <= kParamDa;
    if (tab) {
        for (int64_t j = threadIdx.x; j < m; j += 256) s_mag[j] = exp(-fabs((double)alpha[j]));
        for (int64_t k = threadIdx.x; k < c; k += 256) sincos((double)omega[k], &s_sn[k], &s_cs[k]);
    }
    if (lds_da)
        for (int64_t e = threadIdx.x; e < 2 * m * c; e += 256) s_da[e] = da_g[e];
    __syncthreads();
    const float* da = lds_da ? s_da : da_g;
    auto mag_of = [&](int64_t j) { return tab ? s_mag[j] : exp(-fabs((double)alpha[j])); };
    auto trig_of = [&](int64_t k, double& sn, double& cs) {
        if (tab) {
            sn = s_sn[k];
            cs = s_cs[k];
        } else {
            sincos((double)omega[k], &sn, &cs);
        }
    };
    for (int64_t j = threadIdx.x; dalpha && j < m; j += 256) {
        const double mag = mag_of(j);
        const double sgn = alpha[j] > 0.0f ? 1.0 : (alpha[j] < 0.0f ? -1.0 : 0.0);
        double acc = 0.0;
        for (int64_t k = 0; k < c; ++k) {
            double sn, cs;
            trig_of(k, sn, cs);
            const double dr = da[2 * (j * c + k)], di = da[2 * (j * c + k) + 1];
            acc += mag * (cs * dr + sn * di);                 // Re(conj(a) da)
        }
        dalpha[j] = (float)(-sgn * acc);
    }
    for (int64_t k = threadIdx.x; domega && k < c; k += 256) {
        double sn, cs;
        trig_of(k, sn, cs);
        double acc = 0.0;
        for (int64_t j = 0; j < m; ++j) {
            const double mag = mag_of(j);
            const double dr = da[2 * (j * c + k)], di = da[2 * (j * c + k) + 1];
            acc += mag * (cs * di - sn * dr);                 // Im(conj(a) da)
        }
        domega[k] = (float)acc;
    }
}

// The FFM gradient's last step: workgroups below nblk copy the chain-major
// input gradient dxw[B][nfb][T][jpc] into dx[B][T][m], 256 steps of one tape
// each (the chains' rows of those steps are whole lines, read once); the
// last workgroup forms the parameter gradients from the summed da when asked.
__global__ __launch_bounds__(256) void ffm_bwd_finish_kernel(FfmFinishArgs p) {
    __shared__ __attribute__((aligned(16))) unsigned char s_lds[kFinLdsBytes];
    const int64_t nblk_t = (p.T + kFinRows - 1) / kFinRows;
    if ((int64_t)blockIdx.x == p.B * nblk_t) {
        if (p.dalpha || p.domega) ffm_param_grad(p.alpha, p.omega, p.da, p.m, p.c, p.dalpha, p.domega, s_lds);
        return;
    }
    const int64_t b = blockIdx.x / nblk_t;
    const int64_t t0 = (blockIdx.x - b * nblk_t) * kFinRows;
    const int rows = (int)(p.T - t0 < kFinRows ? p.T - t0 : kFinRows);
    const int64_t nfb = (p.m + p.jpc - 1) / p.jpc;
    if (p.m <= kFinLdsCols) {
        // the block's rows are gathered in LDS: each chain's run of
        // rows * jpc floats is contiguous, read with consecutive threads on
        // consecutive words, and every row of dx then goes out whole.  Row r
        // keeps column j at r * 32 + (j ^ (r & 31)), so neither the gather
        // (rows across the lanes) nor the row reads meet bank conflicts.
        float* const blk = (float*)s_lds;
        const int jpc = (int)p.jpc, m = (int)p.m;
        const int lj = __builtin_ctz((unsigned)jpc);     // jpc = Dp / c, a power of two
        const int run = rows << lj;
        // thread t takes the words t, t + 256, ... of the chains' runs laid
        // end to end; (fb, w) is advanced by subtraction, not division
        int fb = 0, w = (int)threadIdx.x;
        while (fb < (int)nfb && w >= run) {
            w -= run;
            ++fb;
        }
        while (fb < (int)nfb) {
            float v[kFinBatch];
            int at[kFinBatch];
#pragma unroll
            for (int u = 0; u < kFinBatch; ++u) {
                v[u] = 0.0f;
                at[u] = -1;
                if (fb < (int)nfb) {
                    const int r = w >> lj, j = (fb << lj) + (w & (jpc - 1));
                    v[u] = p.dxw[((b * nfb + fb) * p.T + t0) * jpc + w];
                    if (j < m) at[u] = r * kFinLdsCols + (j ^ (r & (kFinLdsCols - 1)));
                    w += 256;
                    while (fb < (int)nfb && w >= run) {
                        w -= run;
                        ++fb;
                    }
                }
            }
#pragma unroll
            for (int u = 0; u < kFinBatch; ++u)
                if (at[u] >= 0) blk[at[u]] = v[u];
        }
        __syncthreads();
        // thread (r0, j) writes column j of rows r0, r0 + per, ...
        float* const dst = p.dx + (b * p.T + t0) * p.m;
        const int per = 256 / m, r0 = (int)threadIdx.x / m, jc = (int)threadIdx.x - r0 * m;
        if (r0 < per) {
            for (int r = r0; r < rows; r += per)
                __builtin_nontemporal_store(blk[r * kFinLdsCols + (jc ^ (r & (kFinLdsCols - 1)))], &dst[r * m + jc]);
        }
        return;
    }
    // thread (r0, j) copies column j of rows r0, r0 + per, ...; for m > 256
    // one row per pass and several columns per thread
    const int64_t per = p.m <= 256 ? 256 / p.m : 1;
    const int64_t r0 = p.m <= 256 ? threadIdx.x / p.m : 0;
    if (r0 >= per) return;
    for (int64_t j = p.m <= 256 ? threadIdx.x % p.m : threadIdx.x; j < p.m; j += 256) {
        const int64_t fb = j / p.jpc;
        const float* src = p.dxw + ((b * nfb + fb) * p.T + t0) * p.jpc + (j - fb * p.jpc);
        float* dst = p.dx + (b * p.T + t0) * p.m + j;
        const int64_t ss = p.jpc, ds = p.m;
        int64_t r = r0;
        for (; r + 3 * per < rows; r += 4 * per) {
            const float v0 = src[r * ss], v1 = src[(r + per) * ss];
            const float v2 = src[(r + 2 * per) * ss], v3 = src[(r + 3 * per) * ss];
            dst[r * ds] = v0;
            dst[(r + per) * ds] = v1;
            dst[(r + 2 * per) * ds] = v2;
            dst[(r + 3 * per) * ds] = v3;
        }
        for (; r < rows; r += per) dst[r * ds] = src[r * ss];
        if (p.m <= 256) break;
    }
}

hipError_t ffm_bwd_finish_launch(const FfmFinishArgs& a, hipStream_t s) {
    const int64_t nblk = a.B * ((a.T + kFinRows - 1) / kFinRows) + 1;
    hipLaunchKernelGGL(ffm_bwd_finish_kernel, dim3((unsigned)nblk), dim3(256), 0, s, a);
    return hipGetLastError();
}

hipError_t diag_bwd_launch(int kind, bool vec, bool ainv, const DiagBwdArgs& args, int64_t ntiles,
                           hipStream_t s) {
    constexpr int RI = diag_rows(true, true), RS = diag_rows(true, false);
    if (kind == K_F32) {
        if (ainv) return vec ? launch_bwd<K_F32, KindInfo<K_F32>::vec, RI>(args, ntiles, true, s) : launch_bwd<K_F32, 1, RI>(args, ntiles, true, s);
        return vec ? launch_bwd<K_F32, KindInfo<K_F32>::vec, RS>(args, ntiles, false, s) : launch_bwd<K_F32, 1, RS>(args, ntiles, false, s);
    }
    if (kind == K_C64) {
        if (ainv) return vec ? launch_bwd<K_C64, KindInfo<K_C64>::vec, kBwdRowsC64Inv>(args, ntiles, true, s) : launch_bwd<K_C64, 1, RI>(args, ntiles, true, s);
        return vec ? launch_bwd<K_C64, KindInfo<K_C64>::vec, RS>(args, ntiles, false, s) : launch_bwd<K_C64, 1, RS>(args, ntiles, false, s);
    }
    return hipErrorInvalidValue;
}

hipError_t colsum_launch(const float* in, float* out, int64_t rows, int64_t cols, int64_t rpw, hipStream_t s) {
    dim3 grid((unsigned)((cols + 63) / 64), (unsigned)((rows + 4 * rpw - 1) / (4 * rpw)));
    hipLaunchKernelGGL(colsum_kernel, grid, dim3(256), 0, s, in, out, rows, cols, rpw);
    return hipGetLastError();
}

}  // namespace memoroid
