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
//            Dp = Qp * VEC features.  Qp lanes of VEC features each cover one
//            step's block; a block is one 128-byte line of the feature row
//            (narrow chains make the tiles long in time, so an episode spans
//            few tiles and the carry rarely has far to travel).
//   tile   = one workgroup of 4 wavefronts.  Lane (j, q) of wavefront w
//            (lane = j * Qp + q) owns the VEC features at q and R consecutive
//            steps; its group is w * Gw + j with Gw = 64 / Qp, groups being
//            consecutive in time: L = 4 * Gw * R steps per tile.
//   ticket = workgroup g works on chain (g + g / nchains) mod nchains (every
//            chain once per run of nchains workgroups, rotated so that no
//            chain is tied to one XCD); its tile within the
//            chain is drawn from that chain's own atomic counter in the order
//            workgroups start, so every tile a workgroup waits for (an
//            earlier tile of its chain) was handed to a workgroup that is
//            already running or finished.  Descriptors are indexed by
//            ticket = tile * nchains + chain.  One counter per chain, each on
//            its own 128-byte line, keeps the counters from serialising.
//            The counters are never reset: they wrap every two calls, so a
//            ticket also tells the call's epoch parity, which picks the
//            descriptor bank (the tile clears its words of the other bank
//            for the next call).  The FFM aggregator keeps one counter per
//            (chain, XCD group) instead, so that every chain's tile at a
//            position runs on one XCD (its chains share the input rows).
//
// Per tile: (1) every load is issued up front: the begin flags of the lane's
// steps, then a and x, one wide access per step; (2) each lane folds its R
// steps into a segment summary (A, H, has-begin); (3) the groups of a
// wavefront scan their summaries with cross-lane shuffles, and the four
// wavefront totals are combined through LDS; (4) the last wavefront publishes
// the tile summary at once -- as the inclusive prefix if the tile holds a
// begin step (nothing older can reach past it), else as an aggregate -- while
// the first wavefront looks back over predecessor tiles for the carry-in;
// (5) the tile's inclusive prefix is published, and every lane replays its
// steps from its carry-in and streams h out.  The cross-lane moves of (3)
// and of the begin counts are DPP / swizzle / permlane butterflies.  a and x are read from HBM once
// and h written once; cross-tile traffic is a few bytes per feature per tile.
#include <type_traits>

#include "scan_common.hpp"
#include "kernels.hpp"

namespace memoroid {

template <Kind IN, Kind OUT, int VEC, int R, bool AINV, bool FFM = false>
__global__ __launch_bounds__(256) void diag_fwd_kernel(DiagFwdArgs p) {
    static_assert(!FFM || (IN == K_C64 && OUT == K_C64 && AINV), "FFM: complex state, generated a");
    static_assert(R >= 1 && R <= 32, "a lane's steps are bits of 32-bit masks");
    using S = typename StateOf<IN>::type;
    using CIn = Codec<IN, VEC>;
    using COut = Codec<OUT, VEC>;
    using SegT = Seg<S, VEC>;
    constexpr int NT = 256;
    constexpr int NW = NT / 64;
    constexpr int IB = KindInfo<IN>::bytes;
    constexpr int OB = KindInfo<OUT>::bytes;
    // widest lane group of this kernel's plans: one chain row of VEC-wide lanes
    constexpr int kQpMax = kChainRowBytes / (VEC * IB) > 0 ? (int)(kChainRowBytes / (VEC * IB)) : 1;

    __shared__ uint32_t s_ticket;          // place in the chain; all ones: stand down
    __shared__ uint32_t s_bank;
    __shared__ S sWA[NW][64 * VEC];        // wavefront totals, per feature of the block
    __shared__ S sWH[NW][64 * VEC];
    __shared__ uint32_t sWF[NW];
    __shared__ S sCarry[64 * VEC];
    __shared__ LookbackLds<S, VEC> sLb;
    __shared__ uint32_t sWC[NW];           // begin counts per wavefront (episode index)
    __shared__ uint32_t sCntBefore;        // begins on the tape before this tile
    __shared__ cf sFfm[FFM ? 64 : 1];      // FFM transitions of the chain's features

    const int tid = threadIdx.x;
    // the workgroup's chain is fixed by its index (each run of nchains
    // consecutive workgroups covers every chain once, rotated by one per run
    // so that no chain stays on one XCD); its place in the chain comes from
    // the chain's own counter, in the order tiles start
    const uint32_t nch = (uint32_t)p.nchains;
    // FFM: the chains of a tape all read each step's real input row.  The
    // grid runs in groups of kXcds * nchains workgroups; workgroup
    // g = kXcds * i + x takes chain i mod nchains and counter (chain, x),
    // whose n-th ticket is position kXcds * n + x, so every chain's tile at a
    // position runs on the same XCD x and its L2 fetches the input rows once.
    // A counter hands out its positions in the order its workgroups start;
    // those of group x - 1 (and of the group before) come earlier in the
    // grid, so the tile a workgroup waits for was claimed by one that is
    // running or finished.  The grid is padded to whole groups: positions
    // past the last tile stand down.
    int chain;
    uint32_t grp = 0, per_call = (uint32_t)p.nt;
    if constexpr (FFM) {
        chain = (int)((blockIdx.x / kXcds) % nch);
        grp = blockIdx.x % kXcds;
        per_call = (uint32_t)((p.nt + kXcds - 1) / kXcds);
    } else {
        chain = (int)((blockIdx.x % nch + blockIdx.x / nch) % nch);
    }
    if (tid == 0) {
        // the signature load goes first: the compiler waits for the atomic's
        // result right after issuing it, and both round trips then overlap
        const uint64_t seen = peek_sig(p.hdr);
        uint32_t* const ctr = p.ctr + ((size_t)chain * (FFM ? kXcds : 1u) + grp) * kCtrStride;
        const Claim c = claim_of(take_ticket(ctr, per_call), per_call);
        const uint32_t pos = FFM ? c.pos * kXcds + grp : c.pos;
        const bool bound = ws_bound_to(p.hdr, p.sig, seen, chain == 0 && pos == 0);
        s_ticket = bound && pos < (uint32_t)p.nt ? pos : kEmpty32;
        s_bank = c.bank;
    }
    barrier_lds();
    const uint32_t claimed = __builtin_amdgcn_readfirstlane(s_ticket);
    if (claimed == kEmpty32) return;       // workspace bound to another call (every tile stands down), or padding
    const int64_t tile = (int64_t)claimed;
    const uint32_t ticket = (uint32_t)(tile * p.nchains + chain);
    // descriptor banks: this call's (epoch parity) and the idle one
    const int64_t boff = __builtin_amdgcn_readfirstlane(s_bank) ? p.bank : 0;
    const int64_t bidle = p.bank - boff;
    void* const agg = (char*)p.agg + boff;
    void* const incl = (char*)p.incl + boff;
    uint64_t* const cnt = p.cnt ? (uint64_t*)((char*)p.cnt + boff) : nullptr;
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

    // ---- (1) loads, through buffer resources based at the tile's first
    // step of this tape: rows past T and lanes past d read zeros (their
    // offsets are out of range) and their stores are dropped.  Flags of the
    // lane's own steps (and of the tile's first step) go first, so that
    // waiting for them leaves every data load in flight; then one wide access
    // per step and tensor.
    const int64_t rows_left = p.T - tile_row0;             // steps from the tile's first to T
    const int64_t tape_row0 = (int64_t)b * p.T + tile_row0;
    const uint32_t lrow = (uint32_t)((wave * Gw + j) * R);  // lane's first step within the tile
    const Rsrc rs_st = make_rsrc(st + tile_row0, rows_left);
    const Rsrc rs_x = make_rsrc((const char*)p.x + tape_row0 * p.d * IB, rows_left * p.d * IB);
    const Rsrc rs_a = make_rsrc(AINV ? p.a : (const char*)p.a + tape_row0 * p.d * IB, AINV ? 0 : rows_left * p.d * IB);
    const uint32_t in_step = active ? (uint32_t)(p.d * IB) : 0u;
    const uint32_t in_off = active ? (uint32_t)((int64_t)lrow * p.d * IB + f0 * IB) : kOob;
    // the previous tile's inclusive words, ahead of everything else (the
    // look-back below is skipped when they were all published)
    S spec[VEC];
    bool spec_ok = false;
    if (wave == 0 && j == 0 && active && tile > 0)
        spec_ok = peek_incl_ahead<S, VEC>(incl, (int64_t)ticket - p.nchains, Dp, Qp, q, spec);
    // FFM: the parameters of the chain's transitions, ahead of the tile's
    // loads, so that the table need not wait for them
    FfmParam fpar{0.f, 0.f};
    if constexpr (FFM) fpar = ffm_param_load(p.alpha, p.omega, p.d, p.ffm_c, (int64_t)fb * Dp, Dp);
    uint32_t fl[R];
#pragma unroll
    for (int r = 0; r < R; ++r) fl[r] = bload_u8(rs_st, lrow + r);
    const uint32_t fl_tile0 = bload_u8(rs_st, 0);
    __builtin_amdgcn_sched_barrier(0);
    RawVec<IN, VEC> ra[AINV ? 1 : R];
    RawVec<IN, VEC> rx[R];
    if constexpr (FFM) {
        // real x[B][T][m] read once per feature's row j and broadcast over
        // the row's c columns (imaginary parts zero)
        // (VEC > 1 only for even c, so a lane's features share one row j
        // and one load per step serves them all)
        const int64_t m = p.ffm_m;
        const Rsrc rs_xf = make_rsrc((const char*)p.x + tape_row0 * m * 4, rows_left * m * 4);
        const uint32_t xo = active ? (uint32_t)(((int64_t)lrow * m + (int64_t)((uint32_t)f0 / (uint32_t)p.ffm_c)) * 4)
                                   : kOob;
        const uint32_t xstep = active ? (uint32_t)(m * 4) : 0u;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const uint32_t w = __builtin_amdgcn_raw_buffer_load_b32(rs_xf, (int)(xo + r * xstep), 0, 0);
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                rx[r].w[2 * v] = w;
                rx[r].w[2 * v + 1] = 0u;
            }
        }
    } else {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            raw_bload(rx[r], rs_x, in_off + r * in_step);
            if constexpr (!AINV) raw_bload(ra[r], rs_a, in_off + r * in_step);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    uint32_t begins = 0, valid = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int64_t t = row0 + r;
        const uint32_t in = t < p.T ? 1u : 0u;
        valid |= in << r;
        begins |= (in & ((t == 0 ? 1u : 0u) | (fl[r] != 0u ? 1u : 0u))) << r;
    }
    S ainv[VEC];
    if constexpr (FFM) {
        // the chain's transitions, evaluated once per tile by wavefront 0
        // while the loads are in flight
        if constexpr (std::is_same<S, cf>::value) {
            ffm_table_store(sFfm, fpar, Dp, false);
            barrier_lds();
#pragma unroll
            for (int v = 0; v < VEC; ++v) ainv[v] = sFfm[q * VEC + v];
        }
    } else if constexpr (AINV) {
        // a NULL time-invariant a stands for a = 1 (the sum monoid, used by
        // the linear-attention state scan)
        RawVec<IN, VEC> r0;
        const bool have = active && p.a != nullptr;
        if (have) raw_load(r0, (const char*)p.a + f0 * IB);
#pragma unroll
        for (int v = 0; v < VEC; ++v) ainv[v] = have ? CIn::get(r0, v) : s_one<S>();
    }
    auto a_at = [&](int r, int v) -> S {
        if constexpr (AINV) return ainv[v];
        else return CIn::get(ra[r], v);
    };

    // ---- (2) per-lane summary of its R steps.  Steps past T hold zeros and
    // come after every real step, so they only touch summaries that no real
    // output uses.
    SegT own = seg_identity<S, VEC>();
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const bool bg = (begins >> r) & 1u;
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            const S xv = CIn::get(rx[r], v);
            const S av = a_at(r, v);
            const S nh = mad(av, own.H[v], xv);
            const S na = own.A[v] * av;
            own.H[v] = bg ? xv : nh;
            own.A[v] = bg ? s_one<S>() : na;
        }
    }
    own.f = begins != 0;
    // packed inputs (bf16) are decoded again for the replay rather than kept
    // decoded: an empty asm on each stored word hides that the decode would
    // repeat, so only the packed words stay live across the scan
    if constexpr (IB < 4) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
#pragma unroll
            for (int k = 0; k < RawVec<IN, VEC>::WORDS; ++k) {
                asm volatile("" : "+v"(rx[r].w[k]));
                if constexpr (!AINV) asm volatile("" : "+v"(ra[r].w[k]));
            }
        }
    }

    // ---- episode index (optional): the tiles of each tape's first feature
    // block count begin steps; the count of the lane's earlier groups comes
    // from a cross-lane prefix sum over the wavefront's groups
    const bool want_idx = p.idx != nullptr && fb == 0;
    const int B = p.nchains / p.nfb;
    const uint32_t c_own = __builtin_popcount(begins);
    uint32_t c_inc = c_own;
    if (want_idx) {
        c_inc = lanes_prefix_sum(c_own, Qp);
        if (j == Gw - 1 && q == 0) sWC[wave] = c_inc;
    }

    // ---- (3) scan the wavefront's groups; combine wavefront totals in LDS
    SegT inc = own, exc;
    wave_group_scan<S, VEC, false, kQpMax>(inc, exc, Qp);
    if (j == Gw - 1) {
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
    SegT before = seg_identity<S, VEC>();        // tile steps before this wavefront
    for (int w = 0; w < wave; ++w) before = seg_then<S, VEC>(before, wave_total(w));
    const SegT pre = seg_then<S, VEC>(before, exc);   // tile steps before this lane's group

    // ---- (4) publish the tile summary (last wavefront, one group of lanes)
    // and look back for the carry-in (first wavefront).  On this hardware a
    // wavefront's loads and stores share one completion counter, so a
    // wavefront with stores in flight could not see its polls' data before
    // those stores are acknowledged: publishing and polling use different
    // wavefronts.
    const bool summary_lane = wave == NW - 1 && j == 0 && active;
    SegT tot = seg_identity<S, VEC>();
    if (wave == NW - 1) {
        tot = seg_then<S, VEC>(before, wave_total(NW - 1));
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
        // the count word of the idle bank, whether or not this call counts
        if (p.cnt != nullptr && fb == 0 && lane == 0)
            ((uint64_t*)((char*)p.cnt + bidle))[tile * (p.nchains / p.nfb) + b] = kEmpty64;
    }
    uint32_t c_before = 0, c_tile = 0;           // begins before this wavefront / in the tile
    if (want_idx) {
        for (int w = 0; w < NW; ++w) {
            if (w < wave) c_before += sWC[w];
            c_tile += sWC[w];
        }
        if (wave == NW - 1 && lane == 0)
            publish64(cnt + tile * B + b, (tile == 0 ? kCountIncl : kCountOwn) | c_tile);
        if (wave == 1) {
            const uint32_t before_tile =
                tile == 0 ? 0u : count_lookback(cnt, (tile - 1) * B + b, B, &p.hdr->timeout);
            if (lane == 0) sCntBefore = before_tile;
        }
    }
    if (wave == 0) {
        const bool need_carry = !(tile_row0 == 0 || fl_tile0 != 0);
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

    // ---- (5) the tile's inclusive prefix goes out first (successors may be
    // waiting for it); then every lane replays its steps from its carry-in
    // and streams h out.
    S hv[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        const S c = sCarry[q * VEC + v];
        if (summary_lane && !tot.f)
            Desc<S>::put_incl(incl, desc_slot(ticket, Dp, Qp, q, v), mad(tot.A[v], c, tot.H[v]));
        hv[v] = seg_apply<S, VEC>(pre, v, c);
    }
    if (want_idx) {
        const uint32_t base_cnt = sCntBefore;
        if (wave == NW - 1 && lane == 0 && tile > 0) publish64(cnt + tile * B + b, kCountIncl | (base_cnt + c_tile));
        if (q == 0) {
            uint32_t run = base_cnt + c_before + (c_inc - c_own);
#pragma unroll
            for (int r = 0; r < R; ++r) {
                if (!((valid >> r) & 1u)) continue;
                run += (begins >> r) & 1u;
                p.idx[(int64_t)b * p.T + row0 + r] = (int32_t)run - 1;
            }
        }
    }
    const Rsrc rs_h = make_rsrc((char*)p.h + tape_row0 * p.d * OB, rows_left * p.d * OB);
    const uint32_t out_step = active ? (uint32_t)(p.d * OB) : 0u;
    const uint32_t out_off = active ? (uint32_t)((int64_t)lrow * p.d * OB + f0 * OB) : kOob;
    auto replay = [&](int r) {
        const bool bg = (begins >> r) & 1u;
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            const S xv = CIn::get(rx[r], v);
            hv[v] = bg ? xv : mad(a_at(r, v), hv[v], xv);
        }
    };
    if constexpr (FFM) {
        // one real input word per step serves all of a lane's features, so
        // holding every step's output would take several times the input's
        // registers: each step's h is stored as soon as it is known
#pragma unroll
        for (int r = 0; r < R; ++r) {
            replay(r);
            RawVec<OUT, VEC> o1;
            COut::put_all(o1, hv);
            raw_bstore_nt(rs_h, out_off + r * out_step, o1);
        }
    } else {
        // all outputs are computed before any store (in the registers that
        // held x when the dtypes match), so the stores go out in one burst
        // and never wait on one another
        constexpr bool kInPlace = (int)IN == (int)OUT;
        RawVec<OUT, VEC> o[kInPlace ? 1 : R];
#pragma unroll
        for (int r = 0; r < R; ++r) {
            replay(r);
            if constexpr (kInPlace) CIn::put_all(rx[r], hv);
            else COut::put_all(o[r], hv);
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            if constexpr (kInPlace) raw_bstore_nt(rs_h, out_off + r * out_step, rx[r]);
            else raw_bstore_nt(rs_h, out_off + r * out_step, o[r]);
        }
    }
}

// ------------------------------------------------------------------ launch

// R: steps per lane with a time-invariant a; RS with a per-step a (the host
// plans the tiles with the same counts, diag_fwd_rows)
template <Kind IN, Kind OUT, int VEC, int R, int RS = R>
static hipError_t launch_fwd(const DiagFwdArgs& args, int64_t ntiles, bool ainv, hipStream_t s) {
    if (ainv)
        hipLaunchKernelGGL((diag_fwd_kernel<IN, OUT, VEC, R, true>), dim3((unsigned)ntiles), dim3(256), 0, s, args);
    else
        hipLaunchKernelGGL((diag_fwd_kernel<IN, OUT, VEC, RS, false>), dim3((unsigned)ntiles), dim3(256), 0, s, args);
    return hipGetLastError();
}

hipError_t ffm_fwd_launch(bool vec, const DiagFwdArgs& args, int64_t ntiles, hipStream_t s) {
    constexpr int R = kFfmFwdRows;
    constexpr int VC = KindInfo<K_C64>::vec;
    (void)ntiles;
    // whole groups of kXcds positions per chain (see the kernel)
    const int64_t grid = ((args.nt + kXcds - 1) / kXcds) * kXcds * args.nchains;
    if (vec)
        hipLaunchKernelGGL((diag_fwd_kernel<K_C64, K_C64, VC, R, true, true>), dim3((unsigned)grid), dim3(256), 0, s,
                           args);
    else
        hipLaunchKernelGGL((diag_fwd_kernel<K_C64, K_C64, 1, R, true, true>), dim3((unsigned)grid), dim3(256), 0, s,
                           args);
    return hipGetLastError();
}

hipError_t diag_fwd_launch(int in_kind, int out_kind, bool vec, bool ainv,
                           const DiagFwdArgs& args, int64_t ntiles, hipStream_t s) {
    constexpr int R = kFwdRows;
    constexpr int VF = KindInfo<K_F32>::vec, VB = KindInfo<K_BF16>::vec, VC = KindInfo<K_C64>::vec;
    if (in_kind == K_F32 && out_kind == K_F32)
        return vec ? launch_fwd<K_F32, K_F32, VF, R, kFwdRowsF32StepA>(args, ntiles, ainv, s)
                   : launch_fwd<K_F32, K_F32, 1, R>(args, ntiles, ainv, s);
    constexpr int RB = kFwdRowsBf16;
    if (in_kind == K_BF16 && out_kind == K_BF16)
        return vec ? launch_fwd<K_BF16, K_BF16, VB, RB>(args, ntiles, ainv, s)
                   : launch_fwd<K_BF16, K_BF16, 1, R>(args, ntiles, ainv, s);
    if (in_kind == K_BF16 && out_kind == K_F32)
        return vec ? launch_fwd<K_BF16, K_F32, VB, RB>(args, ntiles, ainv, s)
                   : launch_fwd<K_BF16, K_F32, 1, R>(args, ntiles, ainv, s);
    if (in_kind == K_C64 && out_kind == K_C64)
        return vec ? launch_fwd<K_C64, K_C64, VC, R>(args, ntiles, ainv, s)
                   : launch_fwd<K_C64, K_C64, 1, R>(args, ntiles, ainv, s);
    return hipErrorInvalidValue;
}

}  // namespace memoroid
