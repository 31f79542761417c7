// tbb.hip -- Tape-Based Batching buffer operations (Alg. 1 and Alg. 2), for
// gfx950.
//
// Insertion needs I = offset + where(b): a stream compaction of the begin
// flags.  One pass: a tile (256 lanes x 64 flags) counts its begin steps,
// publishes the count at once, finds the count before it with a look-back
// over earlier tiles and writes its indices.  Tiles are ordered by workgroup
// index; a look-back that sees no progress counts the awaited tile's flags
// itself (a fallback), so no wait depends on another workgroup having
// started.  The count words are banked by epoch (see scan_common.hpp);
// each tile keeps its own epoch word.
//
// Sampling concatenates the drawn episodes D[I[i] : I[i+1]] and cuts the
// batch to B rows.  Three kernels: episode lengths with block-local
// inclusive sums; a one-workgroup scan of the block totals; a gather in
// which every output row finds its episode by binary search over the
// running ends and copies its row.
#include <type_traits>

#include "scan_common.hpp"
#include "kernels.hpp"

namespace memoroid {

namespace {

constexpr int kFlagsPerLane = 64;
constexpr int kIdxTile = 256 * kFlagsPerLane;      // flags per workgroup
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

__device__ __forceinline__ uint32_t wave_incl_sum(uint32_t v) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int k = 1; k < 64; k <<= 1) {
        const uint32_t o = (uint32_t)__shfl_up((int)v, k, 64);
        if (lane >= k) v += o;
    }
    return v;
}

}  // namespace

template <bool VEC>
__global__ __launch_bounds__(256) void tbb_begins_kernel(TbbBeginArgs p) {
    __shared__ uint32_t s_wave[4];
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
    const uint32_t loff = (uint32_t)(tid * kFlagsPerLane);
    const uint64_t mask = lane_begin_mask<VEC>(rs, loff);
    if (tid == 0) epoch = read_epoch(p.epoch + tile);
    const uint32_t mine = (uint32_t)__builtin_popcountll(mask);
    const uint32_t incl = wave_incl_sum(mine);
    if (lane == 63) s_wave[w] = incl;
    if (tid == 0) s_bank = ws_bound_to(p.hdr, p.sig, sig_seen, tile == 0) ? (epoch & 1u) : kEmpty32;
    __syncthreads();
    const uint32_t bank = __builtin_amdgcn_readfirstlane(s_bank);
    if (bank == kEmpty32) return;             // workspace bound to another call: every tile stands down
    uint64_t* const cnt = (uint64_t*)((char*)p.cnt + (bank ? p.bank : 0));
    const uint32_t own = s_wave[0] + s_wave[1] + s_wave[2] + s_wave[3];
    uint32_t before_wave = 0;
#pragma unroll
    for (int ww = 0; ww < 4; ++ww)
        if (ww < w) before_wave += s_wave[ww];

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
                    for (int part = 0; part < 4; ++part)
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
    uint64_t m = mask;
    int64_t k = (int64_t)s_before + before_wave + (incl - mine);
    while (m) {
        const int b = __builtin_ctzll(m);
        p.indices[k++] = p.offset + t0 + loff + b;
        m &= m - 1;
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

__device__ __forceinline__ int64_t draw_at(const TbbSampleArgs& p, int64_t k) {
    int64_t i = p.draws[k];
    i = i < 0 ? 0 : (i >= p.n_I ? p.n_I - 1 : i);
    return i;
}

// Rows [lo, hi) of episode i, clamped into [0, n_D] so that no index in I
// can send a read outside D.
__device__ __forceinline__ void episode_rows(const TbbSampleArgs& p, int64_t i, int64_t& lo, int64_t& hi) {
    lo = p.I[i];
    hi = i + 1 < p.n_I ? p.I[i + 1] : p.n_D;
    lo = lo < 0 ? 0 : (lo > p.n_D ? p.n_D : lo);
    hi = hi < lo ? lo : (hi > p.n_D ? p.n_D : hi);
}

__device__ __forceinline__ int64_t episode_len(const TbbSampleArgs& p, int64_t i) {
    int64_t lo, hi;
    episode_rows(p, i, lo, hi);
    return hi - lo;
}

__device__ __forceinline__ int64_t wave_incl_sum64(int64_t v) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int k = 1; k < 64; k <<= 1) {
        const int64_t o = __shfl_up(v, k, 64);
        if (lane >= k) v += o;
    }
    return v;
}

// running end of draw k's episode inside the batch (rows before + its length)
__device__ __forceinline__ int64_t end_at(const TbbSampleArgs& p, int64_t k) {
    return p.ends[k] + p.block_off[k / kTbbDrawBlock];
}

}  // namespace

// Episode lengths of the draws and their inclusive sums within blocks of
// kTbbDrawBlock draws (256 lanes x 16 consecutive draws).
__global__ __launch_bounds__(256) void tbb_lengths_kernel(TbbSampleArgs p) {
    __shared__ int64_t s_wave[4];
    constexpr int PER = kTbbDrawBlock / 256;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t k0 = (int64_t)blockIdx.x * kTbbDrawBlock + (int64_t)tid * PER;
    int64_t len[PER];
    int64_t run = 0;
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        const int64_t k = k0 + e;
        len[e] = k < p.n_draws ? episode_len(p, draw_at(p, k)) : 0;
        run += len[e];
    }
    const int64_t incl = wave_incl_sum64(run);
    if (lane == 63) s_wave[w] = incl;
    __syncthreads();
    int64_t before = incl - run;
    for (int ww = 0; ww < w; ++ww) before += s_wave[ww];
#pragma unroll
    for (int e = 0; e < PER; ++e) {
        before += len[e];
        if (k0 + e < p.n_draws) p.ends[k0 + e] = before;
    }
    if (tid == 255) p.block_tot[blockIdx.x] = before;
}

// Exclusive scan of the block totals (one workgroup of 1024 threads), and
// the number of batch rows the draws fill.
__global__ __launch_bounds__(1024) void tbb_block_scan_kernel(TbbSampleArgs p) {
    __shared__ int64_t s_wave[16];
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int64_t nb = p.nblocks;
    const int64_t per = (nb + 1023) / 1024;
    const int64_t b0 = (int64_t)tid * per;
    int64_t run = 0;
    for (int64_t e = 0; e < per; ++e)
        if (b0 + e < nb) run += p.block_tot[b0 + e];
    const int64_t incl = wave_incl_sum64(run);
    if (lane == 63) s_wave[w] = incl;
    __syncthreads();
    int64_t before = incl - run;
    for (int ww = 0; ww < w; ++ww) before += s_wave[ww];
    for (int64_t e = 0; e < per; ++e) {
        if (b0 + e < nb) {
            p.block_off[b0 + e] = before;
            before += p.block_tot[b0 + e];
        }
    }
    if (tid == 1023 && p.filled) *p.filled = before < p.batch ? before : p.batch;
}

// Output rows in groups of kTbbRowsPerGroup (kRowsPerThread per thread).
// The group's first draw -- the first whose running end passes the group's
// first row -- is found by a 256-way search over the running ends (a few
// rounds of one probe per thread); the ends and first source rows of the
// next kTbbRowsPerGroup draws go to LDS, where every row finds its own draw
// by binary search; then the workgroup copies the rows in units of U bytes.
template <int U>
__global__ __launch_bounds__(256) void tbb_gather_kernel(TbbSampleArgs p) {
    constexpr int RW = kTbbRowsPerGroup;
    constexpr int RPT = RW / 256;                  // rows (and window draws) per thread
    __shared__ int64_t s_q[256];
    __shared__ int s_first;
    __shared__ int64_t s_end[RW];      // running ends of draws k0 .. k0 + RW - 1
    __shared__ int64_t s_lo[RW];       // source row minus batch row for those draws
    __shared__ int64_t s_src[RW];
    const int tid = threadIdx.x;
    const int64_t r0 = (int64_t)blockIdx.x * RW;
    const int64_t nd = p.n_draws;

    // ---- k0 = first k with end(k) > r0 (nd if none).  Invariant: the answer
    // lies in [lo, hi], and position hi is either nd or known to qualify.
    int64_t lo = 0, hi = nd;
    while (hi > lo) {
        const int64_t span = hi - lo;
        const bool last_round = span <= 256;
        const int64_t q = last_round ? lo + tid : lo + (((int64_t)tid + 1) * span) / 256 - 1;
        const bool ok = q < hi && end_at(p, q) > r0;
        if (tid == 0) s_first = 256;
        s_q[tid] = q;
        __syncthreads();
        if (ok) atomicMin(&s_first, tid);
        __syncthreads();
        const int f = s_first;
        if (last_round) {
            hi = f < 256 ? s_q[f] : hi;
            lo = hi;
        } else if (f == 256) {
            lo = hi;                      // nothing in [lo, hi) qualifies
        } else {
            lo = f == 0 ? lo : s_q[f - 1] + 1;
            hi = s_q[f];
        }
        __syncthreads();
    }
    const int64_t k0 = hi;

    // ---- the window of draws k0 .. k0 + RW - 1
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
        const int w = tid + 256 * j;
        const int64_t k = k0 + w;
        int64_t e = INT64_MAX, l = 0;
        if (k < nd) {
            int64_t elo, ehi;
            episode_rows(p, draw_at(p, k), elo, ehi);
            e = end_at(p, k);
            l = elo - (e - (ehi - elo));     // source row minus batch row, constant over the episode
        }
        s_end[w] = e;
        s_lo[w] = l;
    }
    __syncthreads();
    const int64_t prev0 = k0 > 0 && k0 <= nd ? end_at(p, k0 - 1) : 0;   // end of the draw before the window

    // ---- each row's draw and source row
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
        const int rr = tid + 256 * j;
        const int64_t t = r0 + rr;
        int64_t src = -1;
        if (t < p.batch) {
            uint8_t st = 0;
            if (k0 < nd) {
                int a = 0, b = RW;              // first window slot with end > t
                while (a < b) {
                    const int mid = (a + b) >> 1;
                    if (s_end[mid] > t) b = mid;
                    else a = mid + 1;
                }
                if (a < RW && k0 + a < nd) {
                    src = t + s_lo[a];
                    st = (a > 0 ? s_end[a - 1] : prev0) == t ? 1 : 0;
                } else if (a == RW) {
                    // more than RW draws end inside this group (empty
                    // episodes): search the remaining draws directly
                    int64_t gl = k0 + RW, gh = nd;
                    while (gl < gh) {
                        const int64_t mid = (gl + gh) >> 1;
                        if (end_at(p, mid) > t) gh = mid;
                        else gl = mid + 1;
                    }
                    if (gl < nd) {
                        int64_t elo, ehi;
                        episode_rows(p, draw_at(p, gl), elo, ehi);
                        src = elo + (t - (end_at(p, gl) - (ehi - elo)));
                        st = src == elo ? 1 : 0;
                    }
                }
            }
            p.out_start[t] = st;
            if (p.out_src) p.out_src[t] = src;
        }
        s_src[rr] = src;
    }
    if (blockIdx.x == 0 && tid == 0 && nd == 0 && p.filled) *p.filled = 0;
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

hipError_t tbb_sample_launch(int unit, const TbbSampleArgs& a, hipStream_t s) {
    if (a.n_draws > 0) {
        hipLaunchKernelGGL(tbb_lengths_kernel, dim3((unsigned)a.nblocks), dim3(256), 0, s, a);
        hipLaunchKernelGGL(tbb_block_scan_kernel, dim3(1), dim3(1024), 0, s, a);
    }
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
