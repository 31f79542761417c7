// tbb.hip -- Tape-Based Batching buffer operations (Alg. 1 and Alg. 2), for
// gfx950.
//
// Insertion needs I = offset + where(b): a stream compaction of the begin
// flags.  One pass: a tile (kIdxBlocks blocks of 256 lanes x 64 flags)
// counts its begin steps, publishes the count at once, finds the count
// before it with a look-back over earlier tiles and writes its indices.
// Tiles are ordered by workgroup index; a look-back that sees no progress
// counts the awaited tile's flags itself (a fallback), so no wait depends on
// another workgroup having started.  The count words are banked by epoch
// (see scan_common.hpp); each tile keeps its own epoch word.
//
// Sampling concatenates the drawn episodes D[I[i] : I[i+1]] and cuts the
// batch to B rows.  Two kernels: a row-sum pass over the draws (the same
// one-pass look-back, on sums saturated at B) that records where each draw
// starts in the batch and which draw holds the first row of each group of
// 256 output rows; then a gather in which every group reads its first draw
// from that table, every row finds its draw by binary search over the next
// 256 draws' first rows, and the workgroup copies the rows.  The draws are
// used in order until the batch is full, so the row-sum tiles past the few
// that should fill it (from the buffer's mean episode length) wait for those
// tiles' verdict and, if the batch is already full, skip their loads.
#include <type_traits>

#include "scan_common.hpp"
#include "kernels.hpp"

namespace memoroid {

namespace {

constexpr int kFlagsPerLane = 64;                  // flags per lane and block
constexpr int kIdxBlocks = kTbbBeginBlocks;         // blocks per tile
constexpr int kIdxBlock = 256 * kFlagsPerLane;      // flags per block (one per lane of the workgroup)
constexpr int kIdxTile = kIdxBlocks * kIdxBlock;    // flags per workgroup
static_assert(kIdxTile == kTbbBeginTile, "compaction tile");

// Bit i set when byte i of the lane's 64 flags is nonzero.
template <bool VEC>
__device__ __forceinline__ uint64_t lane_begin_mask(Rsrc rs, uint32_t off) {
    uint64_t m = 0;
    if constexpr (VEC) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(rs, (int)(off + 16u * q), 0, 0);
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
                for (int by = 0; by < 4; ++by)
                    m |= (uint64_t)(((w[e] >> (8 * by)) & 0xFFu) != 0u) << (16 * q + 4 * e + by);
        }
    } else {
#pragma unroll 8
        for (int i = 0; i < kFlagsPerLane; ++i)
            m |= (uint64_t)(bload_u8(rs, off + i) != 0u) << i;
    }
    return m;
}

// inclusive prefix sums over the 64 lanes (DPP / swizzle / permlane butterfly)
__device__ __forceinline__ uint32_t wave_incl_sum(uint32_t v) { return lanes_prefix_sum(v, 1); }

}  // namespace

template <bool VEC>
__global__ __launch_bounds__(256) void tbb_begins_kernel(TbbBeginArgs p) {
    constexpr int NB = kIdxBlocks;
    __shared__ uint32_t s_wave[NB][4];
    __shared__ uint32_t s_before;
    __shared__ uint32_t s_bank;               // epoch parity; all ones: stand down
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t tile = blockIdx.x;
    // workspace binding and epoch, as in the discounted-return kernel
    uint64_t sig_seen = 0;
    uint32_t epoch = 0;
    if (tid == 0) sig_seen = peek_sig(p.hdr);
    const int64_t t0 = tile * kIdxTile;
    const Rsrc rs = make_rsrc(p.start + t0, p.n - t0);
    // block b of the tile: lane tid holds flags (b * 256 + tid) * 64 .. + 63,
    // so that each block is one contiguous, coalesced 16 KB read
    uint64_t mask[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) mask[b] = lane_begin_mask<VEC>(rs, (uint32_t)((b * 256 + tid) * kFlagsPerLane));
    if (tid == 0) epoch = read_epoch(p.epoch + tile);
    uint32_t mine[NB], incl[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        mine[b] = (uint32_t)__builtin_popcountll(mask[b]);
        incl[b] = wave_incl_sum(mine[b]);
        if (lane == 63) s_wave[b][w] = incl[b];
    }
    if (tid == 0) s_bank = ws_bound_to(p.hdr, p.sig, sig_seen, tile == 0) ? (epoch & 1u) : kEmpty32;
    __syncthreads();
    const uint32_t bank = __builtin_amdgcn_readfirstlane(s_bank);
    if (bank == kEmpty32) return;             // workspace bound to another call: every tile stands down
    uint64_t* const cnt = (uint64_t*)((char*)p.cnt + (bank ? p.bank : 0));
    // begin steps of the tile, and those before this lane's chunk of block b
    // (earlier blocks, then earlier wavefronts of block b)
    uint32_t own = 0, before[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        before[b] = own;
#pragma unroll
        for (int ww = 0; ww < 4; ++ww) {
            if (ww < w) before[b] += s_wave[b][ww];
            own += s_wave[b][ww];
        }
    }

    // wavefront 3 publishes the tile's own count (inclusive for tile 0);
    // wavefront 0 looks back (publishing and polling use different waves)
    if (w == 3 && lane == 0) {
        publish64(cnt + tile, (tile == 0 ? kCountIncl : kCountOwn) | own);
        ((uint64_t*)((char*)p.cnt + (bank ? 0 : p.bank)))[tile] = kEmpty64;   // idle bank, next call
    }
    if (w == 0) {
        uint32_t acc = 0;
        if (tile > 0) {
            int64_t base = tile - 1;
            uint32_t polls = 0;
            while (true) {
                uint32_t sum;
                int fe;
                const bool stop = count_window(cnt, base, 1, sum, fe);
                acc += sum;
                if (stop) break;
                base -= fe;
                if (fe > 0) {
                    polls = 0;
                } else if (++polls > p.fallback_polls) {
                    // tile `base` has not published: count its flags here
                    const int64_t tb = base * kIdxTile;
                    const Rsrc rb = make_rsrc(p.start + tb, p.n - tb);
                    uint32_t c = 0;
#pragma unroll 1
                    for (int part = 0; part < 4 * NB; ++part)
                        c += (uint32_t)__builtin_popcountll(
                            lane_begin_mask<VEC>(rb, (uint32_t)((part * 64 + lane) * kFlagsPerLane)));
                    acc += wave_sum_u32(c);
                    base -= 1;
                    polls = 0;
                } else {
                    __builtin_amdgcn_s_sleep(1);
                }
            }
            if (lane == 0) publish64(cnt + tile, kCountIncl | (acc + own));
        }
        if (lane == 0) {
            s_before = acc;
            if (tile == (int64_t)gridDim.x - 1 && p.count) *p.count = (int64_t)(acc + own);
        }
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        uint64_t m = mask[b];
        int64_t k = (int64_t)s_before + before[b] + (incl[b] - mine[b]);
        const int64_t f0 = p.offset + t0 + (int64_t)(b * 256 + tid) * kFlagsPerLane;
        while (m) {
            const int bit = __builtin_ctzll(m);
            p.indices[k++] = f0 + bit;
            m &= m - 1;
        }
    }
    if (tid == 0) write_epoch(p.epoch + tile, epoch);
}

hipError_t tbb_begins_launch(bool vec, const TbbBeginArgs& a, int64_t ntiles, hipStream_t s) {
    if (vec)
        hipLaunchKernelGGL(tbb_begins_kernel<true>, dim3((unsigned)ntiles), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(tbb_begins_kernel<false>, dim3((unsigned)ntiles), dim3(256), 0, s, a);
    return hipGetLastError();
}

// ----------------------------------------------------------------- sampling

namespace {

constexpr int kDrawsPerLane = kTbbDrawTile / 256;
static_assert(kDrawsPerLane * 256 == kTbbDrawTile, "draw tile");

// Episode of draw k: first source row `lo` and length `len` (0 past the last
// draw).  The position is clamped into [0, n_I) and the episode's rows into
// [0, n_D], so no index in I or draws can send a read outside D.
__device__ __forceinline__ void draw_rows(const TbbSampleArgs& p, int64_t k, int64_t& lo, int64_t& len) {
    lo = 0;
    len = 0;
    if (k >= p.n_draws) return;
    int64_t i = p.draws[k];
    i = i < 0 ? 0 : (i >= p.n_I ? p.n_I - 1 : i);
    int64_t a = p.I[i];
    int64_t b = i + 1 < p.n_I ? p.I[i + 1] : p.n_D;
    a = a < 0 ? 0 : (a > p.n_D ? p.n_D : a);
    b = b < a ? a : (b > p.n_D ? p.n_D : b);
    lo = a;
    len = b - a;
}

__device__ __forceinline__ int64_t wave_incl_sum64(int64_t v) { return lanes_prefix_sum(v, 1); }

__device__ __forceinline__ uint64_t min_u64(uint64_t a, uint64_t b) { return a < b ? a : b; }

}  // namespace

// Row sums of the draws: tile = kTbbDrawTile consecutive draws (2 per
// lane).  Each tile sums its episode lengths, publishes the sum, looks back
// over earlier tiles for the rows before it (ordered by workgroup index, with
// the same fallback as the compaction: an awaited tile that has not
// published is summed here), and then, for every draw whose first row falls
// inside the batch, writes that row and the source-row shift, the gather
// groups whose first row it holds, and -- for the draw that reaches the end
// of the batch, or the last tile if the draws fall short -- the rows filled.
// Sums saturate at the batch size (min(a + b, batch) is associative), so they
// stay exact below it and never overflow.
__global__ __launch_bounds__(256) void tbb_rows_kernel(TbbSampleArgs p) {
    constexpr int RW = kTbbRowsPerGroup;
    __shared__ int64_t s_wave[4];
    __shared__ uint64_t s_before;
    __shared__ uint32_t s_bank;               // epoch parity; all ones: stand down
    __shared__ uint32_t s_skip, s_epoch;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t tile = blockIdx.x;
    const uint64_t cap = (uint64_t)p.batch;
    uint64_t sig_seen = 0;
    uint32_t epoch = 0;
    if (tid == 0) sig_seen = peek_sig(p.hdr);
    if (tile >= p.lead) {
        // a tile past the lead ones waits (one lane, bounded) for the last
        // lead tile's verdict; if the lead tiles already fill the batch, every
        // draw here starts past its end and the tile only publishes the
        // saturated sum, with no loads
        if (tid == 0) {
            epoch = read_epoch(p.epoch + tile);
            const bool bound = ws_bound_to(p.hdr, p.sig, sig_seen, false);
            uint32_t skip = 0;
            if (bound) {
                // the last lead tile posts its verdict in 64 copies, one per
                // cache line, so that the waiting tiles do not all poll one
                // memory location
                const uint64_t* dw = p.dec + 16 * (tile & 63);
                uint32_t polls = 0;
                while (true) {
                    const uint64_t v = peek64(dw);
                    if ((uint32_t)(v >> 32) == epoch && (uint32_t)v != kEmpty32) {
                        skip = (uint32_t)v == 1u ? 1u : 0u;
                        break;
                    }
                    if (++polls > p.fallback_polls) break;          // go on without it
                    __builtin_amdgcn_s_sleep(4);
                }
            }
            s_skip = skip;
            s_bank = bound ? (epoch & 1u) : kEmpty32;
        }
        __syncthreads();
        const uint32_t bank = __builtin_amdgcn_readfirstlane(s_bank);
        if (bank == kEmpty32) return;
        if (s_skip) {
            if (tid == 0) {
                publish64((uint64_t*)((char*)p.cnt + (bank ? p.bank : 0)) + tile, kCountIncl | cap);
                ((uint64_t*)((char*)p.cnt + (bank ? 0 : p.bank)))[tile] = kEmpty64;
                write_epoch(p.epoch + tile, epoch);
            }
            return;
        }
        __syncthreads();                      // s_bank is rewritten below
    }
    const int64_t k0 = tile * kTbbDrawTile + (int64_t)tid * kDrawsPerLane;
    int64_t lo[kDrawsPerLane], len[kDrawsPerLane];
    int64_t run = 0;
#pragma unroll
    for (int e = 0; e < kDrawsPerLane; ++e) {
        draw_rows(p, k0 + e, lo[e], len[e]);
        run += len[e];
    }
    if (tid == 0 && tile < p.lead) epoch = read_epoch(p.epoch + tile);
    const int64_t incl = wave_incl_sum64(run);
    if (lane == 63) s_wave[w] = incl;
    if (tid == 0) {
        s_bank = ws_bound_to(p.hdr, p.sig, sig_seen, tile == 0) ? (epoch & 1u) : kEmpty32;
        s_epoch = epoch;
    }
    __syncthreads();
    const uint32_t bank = __builtin_amdgcn_readfirstlane(s_bank);
    if (bank == kEmpty32) return;             // workspace bound to another call: every tile stands down
    uint64_t* const cnt = (uint64_t*)((char*)p.cnt + (bank ? p.bank : 0));
    const uint64_t own = min_u64((uint64_t)(s_wave[0] + s_wave[1] + s_wave[2] + s_wave[3]), cap);
    int64_t before_wave = 0;
#pragma unroll
    for (int ww = 0; ww < 4; ++ww)
        if (ww < w) before_wave += s_wave[ww];

    // wavefront 3 publishes the tile's own sum (inclusive for tile 0);
    // wavefront 0 looks back
    if (w == 3 && lane == 0) {
        publish64(cnt + tile, (tile == 0 ? kCountIncl : kCountOwn) | own);
        ((uint64_t*)((char*)p.cnt + (bank ? 0 : p.bank)))[tile] = kEmpty64;   // idle bank, next call
    }
    if (w == 0) {
        uint64_t acc = 0;
        if (tile > 0) {
            int64_t base = tile - 1;
            uint32_t polls = 0;
            while (true) {
                uint64_t sum;
                int fe;
                const bool stop = count_window(cnt, base, 1, sum, fe);
                acc = min_u64(acc + sum, cap);
                if (stop) break;
                base -= fe;
                if (fe > 0) {
                    polls = 0;
                } else if (++polls > p.fallback_polls) {
                    // tile `base` has not published: sum its episode lengths here
                    uint64_t r = 0;
#pragma unroll 1
                    for (int e = 0; e < kTbbDrawTile / 64; ++e) {
                        int64_t l, n;
                        draw_rows(p, base * kTbbDrawTile + 64 * e + lane, l, n);
                        r += (uint64_t)n;
                    }
                    acc = min_u64(acc + min_u64(wave_sum_u64(r), cap), cap);
                    base -= 1;
                    polls = 0;
                } else {
                    __builtin_amdgcn_s_sleep(1);
                }
            }
            if (lane == 0) publish64(cnt + tile, kCountIncl | min_u64(acc + own, cap));
        }
        if (tile == p.lead - 1 && p.lead < (int64_t)gridDim.x) {
            // the verdict for the tiles past the lead: is the batch full?
            const uint64_t v = ((uint64_t)s_epoch << 32) | (min_u64(acc + own, cap) >= cap ? 1u : 2u);
            __hip_atomic_store(p.dec + 16 * lane, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (lane == 0) {
            s_before = acc;
            const uint64_t total = min_u64(acc + own, cap);
            if (tile == (p.n_draws - 1) / kTbbDrawTile && total < cap) {
                // the draws end inside the batch
                p.meta[0] = (int64_t)total;
                p.meta[1] = p.n_draws;
                if (p.filled) *p.filled = (int64_t)total;
            }
        }
    }
    __syncthreads();

    // first batch row of each of the lane's draws, and the groups whose
    // first row g * RW lies in [row, min(row + length, batch)): a lane writes
    // up to kFewGroups of them itself; the whole wavefront serves a draw
    // whose episode holds more
    constexpr int64_t kFewGroups = 8;
    uint64_t r = min_u64(s_before + (uint64_t)(before_wave + incl - run), cap);
#pragma unroll
    for (int e = 0; e < kDrawsPerLane; ++e) {
        const int64_t k = k0 + e;
        int64_t ga = 0, gb = 0;
        if (k < p.n_draws && r < cap) {
            const uint64_t end = r + (uint64_t)len[e];
            p.row0[k] = (int64_t)r;
            p.shift[k] = lo[e] - (int64_t)r;
            if (end >= cap) {
                // the draw that reaches the end of the batch
                p.meta[0] = (int64_t)cap;
                p.meta[1] = k + 1;
                if (p.filled) *p.filled = (int64_t)cap;
            }
            ga = (int64_t)((r + RW - 1) / RW);
            gb = (int64_t)((min_u64(end, cap) + RW - 1) / RW);
            if (gb - ga <= kFewGroups)
                for (int64_t g = ga; g < gb; ++g) p.first[g] = k;
        }
        uint64_t many = __ballot(gb - ga > kFewGroups);
        while (many) {
            const int L = __builtin_ctzll(many);
            many &= many - 1;
            const int64_t a = __shfl(ga, L, 64), b = __shfl(gb, L, 64), kk = __shfl(k, L, 64);
            for (int64_t g = a + lane; g < b; g += 64) p.first[g] = kk;
        }
        r = min_u64(r + (uint64_t)len[e], cap);
    }
    if (tid == 0) write_epoch(p.epoch + tile, epoch);
}

// Output rows in groups of kTbbRowsPerGroup (RW / 256 per thread).
// The group's first draw comes from the row-sum kernel's table; the first
// rows and shifts of the next kTbbRowsPerGroup draws go to LDS, where every
// row finds its own draw (the last one starting at or before it) by binary
// search; then the workgroup copies the rows in units of U bytes.
template <int U>
__global__ __launch_bounds__(256) void tbb_gather_kernel(TbbSampleArgs p) {
    constexpr int RW = kTbbRowsPerGroup;
    constexpr int RPT = RW / 256;                  // rows (and window draws) per thread
    __shared__ int64_t s_row0[RW];     // first batch rows of draws k0 .. k0 + RW - 1
    __shared__ int64_t s_shift[RW];    // source row minus batch row for those draws
    __shared__ int64_t s_src[RW];
    __shared__ int64_t s_head[4];      // rows filled, k0, draws inside the batch, go
    const int tid = threadIdx.x;
    const int64_t g = blockIdx.x, r0 = g * RW;
    const int64_t nd = p.n_draws;

    if (tid == 0) {
        int64_t fill = 0, k0 = 0, klim = 0, go = 1;
        if (nd > 0) {
            const uint64_t sig = p.hdr->sig;
            const int64_t f = p.meta[0], kl = p.meta[1], first = p.first[g];
            go = sig == p.sig;                     // else the row sums stood down
            // clamped so that even a workspace left stale by an abandoned
            // call keeps every access in bounds
            fill = f < 0 ? 0 : (f > p.batch ? p.batch : f);
            klim = kl < 0 ? 0 : (kl > nd ? nd : kl);
            k0 = r0 < fill ? (first < 0 ? 0 : (first > klim ? klim : first)) : klim;
        } else if (g == 0 && p.filled) {
            *p.filled = 0;
        }
        s_head[0] = fill;
        s_head[1] = k0;
        s_head[2] = klim;
        s_head[3] = go;
    }
    __syncthreads();
    if (!s_head[3]) return;
    const int64_t fill = s_head[0], k0 = s_head[1], klim = s_head[2];

    // ---- the window of draws k0 .. k0 + RW - 1
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
        const int w = tid + 256 * j;
        const int64_t k = k0 + w;
        const bool in = k < klim;
        s_row0[w] = in ? p.row0[k] : INT64_MAX;
        s_shift[w] = in ? p.shift[k] : 0;
    }
    __syncthreads();

    // ---- each row's draw and source row
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
        const int rr = tid + 256 * j;
        const int64_t t = r0 + rr;
        int64_t src = -1;
        if (t < p.batch) {
            uint8_t st = 0;
            if (t < fill) {
                int a = 0, b = RW;                 // first window slot starting after t
                while (a < b) {
                    const int mid = (a + b) >> 1;
                    if (s_row0[mid] > t) b = mid;
                    else a = mid + 1;
                }
                int64_t row0 = -1, shift = 0;
                if (a == RW && k0 + RW < klim) {
                    // more than RW draws begin inside this group (empty
                    // episodes): search the remaining draws directly
                    int64_t gl = k0 + RW, gh = klim;
                    while (gl < gh) {
                        const int64_t mid = (gl + gh) >> 1;
                        if (p.row0[mid] > t) gh = mid;
                        else gl = mid + 1;
                    }
                    row0 = p.row0[gl - 1];
                    shift = p.shift[gl - 1];
                } else if (a > 0) {
                    row0 = s_row0[a - 1];
                    shift = s_shift[a - 1];
                }
                src = t + shift;
                if (row0 < 0 || src < 0 || src >= p.n_D) src = -1;
                st = src >= 0 && row0 == t ? 1 : 0;
            }
            p.out_start[t] = st;
            if (p.out_src) p.out_src[t] = src;
        }
        s_src[rr] = src;
    }
    __syncthreads();

    // ---- copy the rows: up to 8 units per thread in flight (loads first,
    // then stores), 32-bit index arithmetic
    const uint32_t units = (uint32_t)(p.row_bytes / U);
    const uint32_t rows = (uint32_t)(p.batch - r0 < RW ? p.batch - r0 : RW);
    const uint32_t total = rows * units;
    typedef typename std::conditional<U == 16, u32x4, typename std::conditional<U == 4, uint32_t, uint8_t>::type>::type
        Unit;
    for (uint32_t base = 0; base < total; base += 256u * 8u) {
        Unit v[8];
        uint32_t rr[8], uu[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t e = base + 256u * j + (uint32_t)tid;
            rr[j] = e / units;
            uu[j] = e - rr[j] * units;
            v[j] = Unit{};
            const int64_t sr = e < total ? s_src[rr[j]] : -1;
            if (sr >= 0) v[j] = *(const Unit*)((const char*)p.D + sr * p.row_bytes + (int64_t)uu[j] * U);
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t e = base + 256u * j + (uint32_t)tid;
            if (e < total) {
                Unit* dst = (Unit*)((char*)p.out + (r0 + rr[j]) * p.row_bytes + (int64_t)uu[j] * U);
                __builtin_nontemporal_store(v[j], dst);
            }
        }
    }
}

hipError_t tbb_sample_launch(int unit, const TbbSampleArgs& a, int64_t ntiles, hipStream_t s) {
    if (a.n_draws > 0) hipLaunchKernelGGL(tbb_rows_kernel, dim3((unsigned)ntiles), dim3(256), 0, s, a);
    const unsigned groups = (unsigned)((a.batch + kTbbRowsPerGroup - 1) / kTbbRowsPerGroup);
    if (unit == 16)
        hipLaunchKernelGGL(tbb_gather_kernel<16>, dim3(groups), dim3(256), 0, s, a);
    else if (unit == 4)
        hipLaunchKernelGGL(tbb_gather_kernel<4>, dim3(groups), dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL(tbb_gather_kernel<1>, dim3(groups), dim3(256), 0, s, a);
    return hipGetLastError();
}

}  // namespace memoroid
