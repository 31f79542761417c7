// discount.hip -- discounted return and generalized advantage estimate over a
// tape of episodes, for gfx950.
//
// Both are the memoroid (a, r) . (a', r') = (a a', a r' + r) of App. D and
// App. E folded over the rest of each step's episode, i.e. the reverse
// resettable recurrence
//     y_t = x_t                     if t is the last step of its episode
//     y_t = a * y_{t+1} + x_t       otherwise,
// with a = gamma, x = r for the return and a = gamma * lambda, x = delta
// (the TD error, computed in the kernel) for the advantage.  A step is the
// last of its episode when the next step begins an episode or the tape ends.
//
// One tape per row of [B][T]; a tile is 4 wavefronts of 64 lanes, each lane
// owning one contiguous run of disc_rows(GAE) steps (32 for the return, 16
// for the advantage: tiles of 8192 and 4096 steps).  Loads are coalesced
// (load u of a wavefront puts steps VEC*(64u + lane) .. + VEC-1 into lane
// `lane`); each VEC-step chunk's episode-end bits and, for the advantage, TD
// errors are formed there, and the chunks then move through LDS into the
// lanes that own them.  The recurrence is carried as maps "value at the
// run's first step = f ? H : A * (value after the run) + H": a lane folds
// its run, the wavefront scans its 64 lane maps once, the wavefronts combine
// through LDS, and tiles find the value entering from their right with a
// decoupled look-back over the tiles to their right.  Outputs go back
// through LDS to coalesced stores.
//
// Tiles are numbered from the tape's end by their workgroup index, with no
// ticket counter (a single counter serialises every workgroup on one memory
// line).  Waiting for a tile that has not started could then deadlock, so a
// look-back that sees no progress for a while computes the awaited tile's
// aggregate itself from that tile's inputs (a "fallback") and moves on: no
// wait depends on another workgroup having started, and in the usual
// in-order dispatch the fallback never runs.  The descriptor words are
// banked by epoch (see scan_common.hpp); each tile keeps its own epoch word.
#include "scan_common.hpp"
#include "kernels.hpp"

namespace memoroid {

namespace {


struct RMap {
    float A, H;
    bool f;
};

__device__ __forceinline__ RMap rmap_id() { return RMap{1.0f, 0.0f, false}; }

// `left` covers the steps just before `right`; the value entering from the
// right passes through `right` first.
__device__ __forceinline__ RMap rmap_then(const RMap& left, const RMap& right) {
    RMap o;
    o.f = left.f || right.f;
    o.H = left.f ? left.H : __builtin_fmaf(left.A, right.H, left.H);
    o.A = left.A * right.A;
    return o;
}

__device__ __forceinline__ float rmap_apply(const RMap& m, float after) {
    return m.f ? m.H : __builtin_fmaf(m.A, after, m.H);
}

// the value of lane (l & ~(2M - 1)) | M (the first lane of the upper half
// of each block of 2M lanes; see sk_move)
template <int M>
__device__ __forceinline__ RMap rmap_upper_first(const RMap& m) {
    return RMap{sk_move<true, M, 1>(m.A), sk_move<true, M, 1>(m.H), sk_move<true, M, 1>((uint32_t)m.f) != 0u};
}

template <int M>
__device__ __forceinline__ void suffix_steps(RMap& m) {
    if constexpr (M < 64) {
        const int lane = threadIdx.x & 63;
        const RMap o = rmap_upper_first<M>(m);
        const RMap n = rmap_then(m, o);
        // component-wise selects (a select of whole structs would keep them
        // in private memory)
        const bool takes = (lane & M) == 0;
        m.A = takes ? n.A : m.A;
        m.H = takes ? n.H : m.H;
        m.f = takes ? n.f : m.f;
        suffix_steps<2 * M>(m);
    }
}

__device__ __forceinline__ float readlane_f(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}

// The value of lane l + 1 (lane 63 gets its own): one DPP move with the
// whole-wavefront shift wave_shl:1 (gfx9 DPP; lane 63, which has no source,
// keeps the `old` operand, here its own value).  Called with every lane
// active (no ds_bpermute, whose reads of a disabled lane would be undefined).
__device__ __forceinline__ uint32_t lane_next(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x130, 0xF, 0xF, false);   // wave_shl:1
}
__device__ __forceinline__ float lane_next(float v) { return __uint_as_float(lane_next(__float_as_uint(v))); }

// Suffix composition over the wavefront: `exc` gets m_{l+1} . ... . m_63
// (the lanes after lane l; identity for lane 63) and `total` m_0 . ... .
// m_63 (the same in every lane).  A Sklansky scan towards lane 0: at step
// M the lower half of each block of 2M lanes (earlier steps) appends the
// upper half's total, which the upper half's first lane holds -- one partner
// move (ds_swizzle within 32 lanes, a scalar lane read across the halves)
// and one combine per step, no LDS memory; the exclusive suffix is the next
// lane's (lane_next) and the total lane 0's (a scalar read).
__device__ __forceinline__ void wave_suffix(const RMap& m0, RMap& exc, RMap& total) {
    const int lane = threadIdx.x & 63;
    RMap m = m0;
    suffix_steps<1>(m);
    const float na = lane_next(m.A), nh = lane_next(m.H);
    const uint32_t nf = lane_next((uint32_t)m.f);
    const bool last = lane == 63;
    exc.A = last ? 1.0f : na;
    exc.H = last ? 0.0f : nh;
    exc.f = last ? false : nf != 0u;
    total = RMap{readlane_f(m.A, 0), readlane_f(m.H, 0), __builtin_amdgcn_readlane((int)m.f, 0) != 0};
}

// m_0 . ... . m_63 in every lane
__device__ __forceinline__ RMap wave_total(const RMap& m) {
    RMap exc, total;
    wave_suffix(m, exc, total);
    return total;
}

template <int VEC>
struct F;
template <>
struct F<4> {
    typedef float __attribute__((ext_vector_type(4))) T;
};
template <>
struct F<1> {
    typedef float T;
};

template <int VEC>
__device__ __forceinline__ float comp(const typename F<VEC>::T& v, int k) {
    if constexpr (VEC == 1) {
        return v;
    } else {
        return v[k];
    }
}

template <int VEC>
__device__ __forceinline__ void set_comp(typename F<VEC>::T& v, int k, float x) {
    if constexpr (VEC == 1) {
        v = x;
    } else {
        v[k] = x;
    }
}

template <int VEC>
// inputs are read once: non-temporal loads (the return 35.6 -> 33.3 us)
__device__ __forceinline__ typename F<VEC>::T load_vec(const float* p) {
    return __builtin_nontemporal_load((const typename F<VEC>::T*)p);
}

template <int VEC>
__device__ __forceinline__ uint32_t load_flags(const uint8_t* p) {
    if constexpr (VEC == 1) {
        return *p;
    } else {
        return *(const uint32_t*)p;
    }
}

template <int VEC>
__device__ __forceinline__ void store_vec(float* p, const typename F<VEC>::T& v) {
    __builtin_nontemporal_store(v, (typename F<VEC>::T*)p);
}

// Inputs x (delta for the advantage, computed here in place) of one lane's
// VEC steps t0 .. t0+VEC-1; returns bit k set when step k is the last of its
// episode.  next_fl / next_v: begin flag and V(s) of the step after the
// lane's last step.
template <int VEC, bool GAE>
__device__ __forceinline__ uint32_t prep_chunk(const DiscArgs& p, int64_t t0, typename F<VEC>::T& x,
                                               const typename F<VEC>::T& vv, const typename F<VEC>::T& vn,
                                               uint32_t fl, uint32_t dn, uint32_t next_fl, float next_v) {
    // steps k >= lim are the tape's last step or past it
    const int64_t rem = p.T - 1 - t0;
    const int lim = rem <= 0 ? 0 : (rem >= VEC ? VEC : (int)rem);
    uint32_t eb = ((1u << VEC) - 1u) & ~((1u << lim) - 1u);
    if constexpr (VEC == 4) {
        // begin flags of steps t0+1 .. t0+4, one per byte; a byte's top bit
        // set exactly when the byte is nonzero, then the four top bits
        const uint32_t w = __builtin_amdgcn_alignbyte(next_fl, fl, 1);
        const uint32_t hb = (((w & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | w) & 0x80808080u;
        eb |= ((hb >> 7) | (hb >> 14) | (hb >> 21) | (hb >> 28)) & 0xFu;
    } else {
        eb |= (next_fl & 0xFFu) != 0u ? 1u : 0u;
    }
#pragma unroll
    for (int k = 0; k < VEC; ++k) {
        const bool e = (eb >> k) & 1u;
        if constexpr (GAE) {
            float nxt;
            if (p.vn) {
                nxt = comp<VEC>(vn, k);
            } else {
                nxt = k + 1 < VEC ? comp<VEC>(vv, k + 1 < VEC ? k + 1 : k) : next_v;
                nxt = e ? 0.0f : nxt;
            }
            const bool keep = ((dn >> (8 * k)) & 0xFFu) == 0u;
            const float g = keep ? p.gamma : 0.0f;
            set_comp<VEC>(x, k, __builtin_fmaf(g, nxt, comp<VEC>(x, k)) - comp<VEC>(vv, k));
        }
    }
    return eb;
}

// The map of VEC steps with inputs x and episode-end bits eb.
template <int VEC>
__device__ __forceinline__ RMap chunk_map(float a, const typename F<VEC>::T& x, uint32_t eb) {
    RMap m = rmap_id();
#pragma unroll
    for (int k = VEC - 1; k >= 0; --k) m = rmap_then(RMap{a, comp<VEC>(x, k), ((eb >> k) & 1u) != 0u}, m);
    return m;
}

// One step of the reverse recurrence as a bit select (no multiply by zero
// at a reset, so a non-finite value never crosses an episode end): the
// value at step s of a lane's run given the value y after it, with bit s of
// m set when step s ends its episode.
__device__ __forceinline__ float step_back(uint32_t m, int s, float a, float x, float y) {
    const uint32_t mk = (uint32_t)((int32_t)(m << (31 - s)) >> 31);   // v_bfe_i32: all ones or zero
    const float ny = __builtin_fmaf(a, y, x);
    // one v_bfi_b32 (written out: the compiler would turn the bit select
    // into a compare and a v_cndmask, one instruction more per step)
    uint32_t r;
    asm("v_bfi_b32 %0, %1, %2, %3" : "=v"(r) : "v"(mk), "v"(__float_as_uint(x)), "v"(__float_as_uint(ny)));
    return __uint_as_float(r);
}

// Position of chunk k of lane o's run in the wavefront's LDS rows of NC
// chunks: XOR-swizzled within the row, so that an instruction of the
// coalesced side (64 consecutive chunks) and one of the owner side (chunk k
// of every row) both reach distinct banks.
template <int NC>
__device__ __forceinline__ int owner_slot(int o, int k) {
    constexpr int LG = NC == 4 ? 2 : NC == 8 ? 3 : NC == 16 ? 4 : 5;
    static_assert(NC == (1 << LG), "rows of 4, 8, 16 or 32 chunks");
    return o * NC + (k ^ ((o ^ (o >> LG)) & (NC - 1)));
}

// Aggregate map of tile `tile` of tape row `row`, computed by one wavefront
// straight from the inputs (the look-back fallback).  Loads are taken one
// run of 64*VEC steps at a time, right to left; each lane reads the flag and
// value after its own steps directly.
template <int VEC, bool GAE>
__device__ __forceinline__ RMap tile_map_from_inputs(const DiscArgs& p, int64_t row, int64_t tile) {
    typedef typename F<VEC>::T V;
    const int lane = threadIdx.x & 63;
    constexpr int kTile = disc_tile(GAE);
    constexpr int runs = kTile / (64 * VEC);
    RMap TM = rmap_id();
#pragma unroll 1
    for (int s = runs - 1; s >= 0; --s) {
        const int64_t t0 = tile * kTile + (int64_t)64 * VEC * s + VEC * lane;
        const bool ok = t0 < p.T;
        V x{}, vv{}, vn{};
        uint32_t fl = 0, dn = 0, next_fl = 1;
        float next_v = 0.0f;
        if (ok) {
            fl = load_flags<VEC>(p.start + row + t0);
            x = load_vec<VEC>(p.r + row + t0);
            if (t0 + VEC < p.T) next_fl = p.start[row + t0 + VEC];
            if constexpr (GAE) {
                vv = load_vec<VEC>(p.v + row + t0);
                if (p.vn) vn = load_vec<VEC>(p.vn + row + t0);
                if (p.done) dn = load_flags<VEC>(p.done + row + t0);
                if (!p.vn && t0 + VEC < p.T) next_v = p.v[row + t0 + VEC];
            }
        }
        const uint32_t eb = prep_chunk<VEC, GAE>(p, t0, x, vv, vn, fl, dn, next_fl, next_v);
        const RMap m = chunk_map<VEC>(p.a, x, eb);
        TM = rmap_then(wave_total(m), TM);
    }
    return TM;
}

}  // namespace

template <int VEC, bool GAE>
__global__ __launch_bounds__(256) void disc_kernel(DiscArgs p) {
    constexpr int kRows = disc_rows(GAE);     // steps per lane: one contiguous run
    constexpr int kSeg = 64 * kRows;          // steps per wavefront
    constexpr int kTile = disc_tile(GAE);
    constexpr int NC = kRows / VEC;           // chunks of VEC steps per lane (loads per lane)
    typedef typename F<VEC>::T V;
    __shared__ V s_x[4][64 * NC];             // per wavefront: inputs in owner rows, then outputs
    __shared__ __attribute__((aligned(16))) uint8_t s_e[4][64 * NC];   // episode-end bits per chunk
    __shared__ float s_wA[4], s_wH[4];
    __shared__ int s_wf[4];
    __shared__ float s_carry;
    __shared__ uint32_t s_bank;               // epoch parity; all ones: stand down
    __shared__ int s_need;

    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t ticket = blockIdx.x;
    // workspace binding: the signature is loaded first, checked after the loads
    uint64_t sig_seen = 0;
    uint32_t epoch = 0;
    if (tid == 0) sig_seen = peek_sig(p.hdr);
    // tiles counted from the tape's end (fewer than 2^31 tiles: a 32-bit division)
    const int64_t j = (int64_t)((uint32_t)ticket / (uint32_t)p.B);
    const int64_t b = ticket - j * p.B;
    const int64_t i = p.nt - 1 - j;           // tile index from the tape's start
    const int64_t T = p.T;
    const int64_t row = b * T;
    const int64_t t_seg = i * kTile + (int64_t)w * kSeg;
    const int64_t t_after = t_seg + kSeg;     // first step after this wavefront's steps

    // ------------------------------------------------ loads (coalesced)
    // load u of lane l holds chunk 64u + l of the wavefront's run
    V x[NC], vv[NC] = {}, vn[NC] = {};
    uint32_t fl[NC], dn[NC] = {};
#pragma unroll
    for (int u = 0; u < NC; ++u) {
        const int64_t t = t_seg + VEC * (64 * u + lane);
        const bool ok = t < T;
        fl[u] = ok ? load_flags<VEC>(p.start + row + t) : 0u;
        x[u] = ok ? load_vec<VEC>(p.r + row + t) : V{};
        if constexpr (GAE) {
            vv[u] = ok ? load_vec<VEC>(p.v + row + t) : V{};
            vn[u] = (ok && p.vn) ? load_vec<VEC>(p.vn + row + t) : V{};
            dn[u] = (ok && p.done) ? load_flags<VEC>(p.done + row + t) : 0u;
        }
    }
    // the tile's epoch, behind its loads (waiting for the epoch word then
    // leaves them in flight)
    if (tid == 0) epoch = read_epoch(p.epoch + ticket);
    // the step after this wavefront's run: its begin flag (and value)
    const bool after_in = t_after < T;
    const uint32_t fl_after = after_in ? p.start[row + t_after] : 1u;
    float v_after = 0.0f;
    if constexpr (GAE) {
        if (after_in && !p.vn) v_after = p.v[row + t_after];
    }

    // ------------------- per-step inputs, then the transpose to owner rows
    // Each chunk's inputs (delta for the advantage) and episode-end bits are
    // formed where the chunk was loaded, with the step after it taken from
    // the next lane (or the next load's first lane, or the next run); then
    // the chunks go to LDS, where lane o's row holds chunks NC*o .. NC*o+NC-1:
    // its own contiguous run of kRows steps.
#pragma unroll
    for (int u = 0; u < NC; ++u) {
        const int c = 64 * u + lane;
        const int64_t t0 = t_seg + VEC * c;
        const uint32_t next_lane_fl = lane_next(fl[u]);
        const uint32_t fl_next_run =
            u + 1 < NC ? (uint32_t)__builtin_amdgcn_readlane((int)fl[u + 1 < NC ? u + 1 : u], 0) : fl_after;
        const uint32_t next_fl = lane < 63 ? next_lane_fl : fl_next_run;
        float next_v = 0.0f;
        if constexpr (GAE) {
            const float nl = lane_next(comp<VEC>(vv[u], 0));
            const float nr = u + 1 < NC ? readlane_f(comp<VEC>(vv[u + 1 < NC ? u + 1 : u], 0), 0) : v_after;
            next_v = lane < 63 ? nl : nr;
        }
        const uint32_t eb = prep_chunk<VEC, GAE>(p, t0, x[u], vv[u], vn[u], fl[u], dn[u], next_fl, next_v);
        s_x[w][owner_slot<NC>(c / NC, c % NC)] = x[u];
        s_e[w][c] = (uint8_t)eb;
    }
    // the wavefront's own LDS rows only: its LDS operations run in program
    // order, so a compiler-only fence is all the ordering needed
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    V xo[NC];
#pragma unroll
    for (int k = 0; k < NC; ++k) xo[k] = s_x[w][owner_slot<NC>(lane, k)];
    // bit s of m: step s of the lane's run ends its episode
    uint32_t m = 0;
    {
        const uint32_t* ew = (const uint32_t*)&s_e[w][lane * NC];
        uint32_t d[(NC + 3) / 4];
#pragma unroll
        for (int q = 0; q < (NC + 3) / 4; ++q) d[q] = ew[q];
#pragma unroll
        for (int q = 0; q < NC; ++q) m |= ((d[q / 4] >> (8 * (q % 4))) & ((1u << VEC) - 1u)) << (VEC * q);
    }
    const float a = p.a;

    // ------------------------------------------- lane maps, wavefront scan
    // the lane's map: its run folded right to left from a zero after it
    float y = 0.0f;
#pragma unroll
    for (int q = NC - 1; q >= 0; --q)
#pragma unroll
        for (int k = VEC - 1; k >= 0; --k) y = step_back(m, VEC * q + k, a, comp<VEC>(xo[q], k), y);
    float aR = a;                             // a^kRows: the map's factor when no step of the run ends an episode
#pragma unroll
    for (int n = 1; n < kRows; n *= 2) aR *= aR;
    RMap E, Wtot;                             // E: the lanes after this one; Wtot: the whole wavefront
    wave_suffix(RMap{aR, y, m != 0u}, E, Wtot);
    if (lane == 0) {
        s_wA[w] = Wtot.A;
        s_wH[w] = Wtot.H;
        s_wf[w] = (int)Wtot.f;
    }
    // a carry from the next tile is needed unless the tile's last step ends
    // an episode (the last wavefront holds the next tile's first flag)
    if (tid == 192) s_need = (j > 0 && fl_after == 0u) ? 1 : 0;
    const int64_t slot = b * p.nt + j;
    // Wavefront 0 holds the tile's first steps: when they include an episode
    // end it knows the value at the tile's first step already, and publishes
    // it before the barrier, so that a look-back waiting for this tile does
    // not wait for the tile's other wavefronts.
    if (tid == 0) {
        const bool bound = ws_bound_to(p.hdr, p.sig, sig_seen, ticket == 0);
        s_bank = bound ? (epoch & 1u) : kEmpty32;
        if (bound && Wtot.f) publish64((uint64_t*)((char*)p.incl + ((epoch & 1u) ? p.bank : 0)) + slot, pack2(Wtot.H, 0.0f));
    }
    barrier_lds();
    const uint32_t bank = __builtin_amdgcn_readfirstlane(s_bank);
    if (bank == kEmpty32) return;             // workspace bound to another call: every tile stands down
    uint64_t* const agg = (uint64_t*)((char*)p.agg + (bank ? p.bank : 0));
    uint64_t* const incl = (uint64_t*)((char*)p.incl + (bank ? p.bank : 0));
    RMap Wt[4];
#pragma unroll
    for (int ww = 0; ww < 4; ++ww) Wt[ww] = RMap{s_wA[ww], s_wH[ww], s_wf[ww] != 0};
    const RMap TM = rmap_then(Wt[0], rmap_then(Wt[1], rmap_then(Wt[2], Wt[3])));
    const bool need = __builtin_amdgcn_readfirstlane(s_need) != 0;
    // wavefront ww depends on the carry when no later wavefront of the tile
    // holds an episode end (a tile that needs no carry ends one itself)
    bool dep[4];
    dep[3] = need;
#pragma unroll
    for (int ww = 2; ww >= 0; --ww) dep[ww] = dep[ww + 1] && !Wt[ww + 1].f;

    // ------------------------------------------------------------ outputs
    // The value entering the wavefront's last step passes through the later
    // wavefronts' maps from the tile's carry c; each lane takes it through
    // the later lanes' maps, runs its steps right to left, and the results
    // go back through the LDS rows to coalesced stores.
    auto emit = [&](float c) {
#pragma unroll
        for (int ww = 3; ww > 0; --ww)
            if (ww > w) c = rmap_apply(Wt[ww], c);
        float yv = rmap_apply(E, c);
        // the step masks are formed again from an opaque copy of m rather
        // than kept from the lane map's loop (32 of them would not fit)
        uint32_t m2 = m;
        asm volatile("" : "+v"(m2));
#pragma unroll
        for (int q = NC - 1; q >= 0; --q)
#pragma unroll
            for (int k = VEC - 1; k >= 0; --k) {
                yv = step_back(m2, VEC * q + k, a, comp<VEC>(xo[q], k), yv);
                set_comp<VEC>(xo[q], k, yv);
            }
#pragma unroll
        for (int k = 0; k < NC; ++k) s_x[w][owner_slot<NC>(lane, k)] = xo[k];
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
#pragma unroll
        for (int u = 0; u < NC; ++u) {
            const int cc = 64 * u + lane;
            const int64_t t0 = t_seg + VEC * cc;
            const V out = s_x[w][owner_slot<NC>(cc / NC, cc % NC)];
            if (t0 < T) {
                store_vec<VEC>(p.out + row + t0, out);
                if constexpr (GAE) {
                    if (p.target) store_vec<VEC>(p.target + row + t0, out + vv[u]);
                }
            }
        }
    };

    // ------------------------------------------------ publish, look back
    // Wavefront 2 publishes the tile's aggregate (or, when the tile holds an
    // episode end that wavefront 0 did not hold, its value at the first step,
    // which then needs nothing from the right); wavefront 3, the one that
    // needs the carry, looks back; so no wavefront both stores and polls.
    // Wavefronts that do not depend on the carry store their outputs at once.
    if (w == 2 && lane == 0) {
        if (!TM.f)
            publish64(agg + slot, pack2(TM.H, TM.A));
        else if (!Wt[0].f)
            publish64(incl + slot, pack2(TM.H, 0.0f));
        // this tile's words of the idle bank, for the next call
        const int64_t idle = bank ? 0 : p.bank;
        ((uint64_t*)((char*)p.agg + idle))[slot] = kEmpty64;
        ((uint64_t*)((char*)p.incl + idle))[slot] = kEmpty64;
    }
    if (!dep[w]) emit(0.0f);                  // exact: the carry does not reach these steps
    float carry = 0.0f;
    if (w == 3 && need) {
        RMap acc = rmap_id();
        int64_t base = j - 1;
        uint32_t polls = 0;
        while (true) {
            const int64_t pj = base - lane;
            uint64_t wi = pack2(0.0f, 0.0f), wa = kEmpty64;
            if (pj >= 0) {
                wi = peek64(incl + b * p.nt + pj);
                if (wi == kEmpty64) wa = peek64(agg + b * p.nt + pj);
            }
            const bool term = wi != kEmpty64;
            const bool ready = term || wa != kEmpty64;
            const uint64_t m_term = __ballot(term);
            const uint64_t m_nr = __ballot(!ready);
            const int ft = m_term ? __builtin_ctzll(m_term) : 64;
            const int fn = m_nr ? __builtin_ctzll(m_nr) : 64;
            const int upto = ft < fn ? ft : fn;   // lanes before `upto` hold aggregates
            RMap mm = rmap_id();
            if (lane < upto) mm = RMap{unpack_hi(wa), unpack_lo(wa), false};
            if (ft < fn && lane == ft) mm = RMap{1.0f, unpack_lo(wi), true};
            const RMap R = wave_total(mm);
            acc = rmap_then(acc, R);
            if (ft < fn) {
                carry = acc.H;
                break;
            }
            base -= fn;
            if (fn > 0) {
                polls = 0;
            } else if (++polls > p.fallback_polls) {
                // tile `base` has not published: fold its aggregate in
                // from its inputs (tile index from the tape's start)
                const RMap M = tile_map_from_inputs<VEC, GAE>(p, row, p.nt - 1 - base);
                acc = rmap_then(acc, M);
                if (M.f) {
                    carry = acc.H;
                    break;
                }
                base -= 1;
                polls = 0;
            } else {
                __builtin_amdgcn_s_sleep(1);
            }
        }
        if (!TM.f && lane == 0) publish64(incl + slot, pack2(rmap_apply(TM, carry), 0.0f));
        if (dep[2] && lane == 0) s_carry = carry;
    }
    if (dep[2]) {                             // workgroup-uniform: earlier wavefronts wait for the carry too
        barrier_lds();
        carry = s_carry;
    }
    if (dep[w]) emit(carry);
    if (tid == 0) write_epoch(p.epoch + ticket, epoch);
}

hipError_t disc_launch(bool vec, bool gae, const DiscArgs& a, int64_t ntiles, hipStream_t s) {
    const dim3 grid((unsigned)ntiles), block(256);
    if (vec) {
        if (gae)
            hipLaunchKernelGGL((disc_kernel<4, true>), grid, block, 0, s, a);
        else
            hipLaunchKernelGGL((disc_kernel<4, false>), grid, block, 0, s, a);
    } else {
        if (gae)
            hipLaunchKernelGGL((disc_kernel<1, true>), grid, block, 0, s, a);
        else
            hipLaunchKernelGGL((disc_kernel<1, false>), grid, block, 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace memoroid
