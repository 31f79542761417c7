// abi.hip -- the extern "C" entry points declared in include/memoroid.h:
// argument validation (before any HIP call), tiling plans, workspace layout
// and kernel launches.
#include <limits.h>
#include <atomic>
#include <mutex>
#include <initializer_list>
#include <stdlib.h>
#include <string.h>

#include "memoroid.h"
#include "memoroid_testing.h"
#include "kernels.hpp"
#include "scan_common.hpp"

using namespace memoroid;

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

int elem_bytes(int dt) { return dt == MEMOROID_F32 ? 4 : dt == MEMOROID_BF16 ? 2 : 8; }
int vec_width(int dt) { return dt == MEMOROID_F32 ? 4 : dt == MEMOROID_BF16 ? 8 : 2; }
// smallest power of two >= v, capped at 2^62 (callers cap it far lower)
int64_t next_pow2(int64_t v) {
    int64_t p = 1;
    while (p < v && p < ((int64_t)1 << 62)) p <<= 1;
    return p;
}
bool aligned(const void* p, size_t n) { return ((uintptr_t)p % n) == 0; }

// Overflow-checked product of non-negative extents.
bool mul_ok(int64_t a, int64_t b, int64_t* out) {
    if (a != 0 && b > INT64_MAX / a) return false;
    *out = a * b;
    return true;
}

struct DiagPlan {
    int VEC = 1;
    int Qp = 1;
    int Dp = 1;
    int nfb = 1;
    int64_t L = 1;
    int64_t nt = 0;
    int64_t nchains = 0;
    int64_t ntiles = 0;
    // offsets of the counters and of bank 0's regions (bank 1: + bank_bytes)
    size_t off_ctr = 0, off_agg = 0, off_incl = 0, off_cnt = 0, off_part = 0, off_sum1 = 0, off_sum2 = 0;
    size_t bank_bytes = 0;
    bool fused_da = false;   // one tape: da summed inside the reverse kernel
    size_t init_bytes = 0;   // what a self-initialising call fills: header, counters, bank 0
    size_t total = 0;
};

// Signature of a call's workspace layout (FNV-1a over the values that fix
// it); never all ones (a fresh workspace) or kSigPoisoned.
uint64_t layout_sig(std::initializer_list<int64_t> vals) {
    uint64_t h = 0xcbf29ce484222325ull;
    for (int64_t v : vals)
        for (int i = 0; i < 8; ++i) {
            h ^= (uint64_t)(v >> (8 * i)) & 0xFFu;
            h *= 0x100000001b3ull;
        }
    if (h == kEmpty64 || h == kSigPoisoned) h ^= 0x9E3779B97F4A7C15ull;
    return h;
}

// entry points in a signature
enum SigKind : int64_t { kSigDiag = 1, kSigDiagBwd, kSigFfm, kSigFfmBwd, kSigDiscount, kSigTbbBegins,
                         kSigLinattn, kSigLinattnBwd, kSigTbbSample };

// Tiling and workspace layout of a diagonal scan.  `vec` selects the
// vectorised lane width; `state_complex` picks the descriptor size.
// ctr_groups: tile counters per chain (the FFM forward keeps one per XCD
// group of workgroups, kXcds)
bool plan_diag(int64_t B, int64_t T, int64_t d, int state_dtype, bool vec, int rows, bool bwd,
               bool ainv, bool want_grad_a, DiagPlan* p, int ctr_groups = 1) {
    // extents no tiling can address (and whose sums below would overflow)
    if (B <= 0 || T <= 0 || d <= 0 || d > (int64_t)INT32_MAX || T > INT64_MAX / 4) return false;
    const int VEC = vec ? vec_width(state_dtype) : 1;
    const int64_t lanes = (d + VEC - 1) / VEC;
    // a chain's row block is (at most) one 128-byte line of the feature row
    const int64_t qp_cap = kChainRowBytes / (VEC * elem_bytes(state_dtype)) > 0 ? kChainRowBytes / (VEC * elem_bytes(state_dtype)) : 1;
    const int64_t Qp = next_pow2(lanes) < qp_cap ? next_pow2(lanes) : qp_cap;
    p->VEC = VEC;
    p->Qp = (int)Qp;
    p->Dp = (int)(Qp * VEC);
    p->nfb = (int)((d + p->Dp - 1) / p->Dp);
    p->L = (256 / Qp) * rows;
    p->nt = (T + p->L - 1) / p->L;
    if (!mul_ok(B, p->nfb, &p->nchains)) return false;
    if (!mul_ok(p->nt, p->nchains, &p->ntiles)) return false;
    if (p->ntiles >= (int64_t)INT32_MAX || p->nchains >= (int64_t)INT32_MAX) return false;
    // a grid padded to whole groups of ctr_groups positions per chain
    if (ctr_groups > 1 && ((p->nt + ctr_groups - 1) / ctr_groups) * ctr_groups > (int64_t)INT32_MAX / p->nchains)
        return false;
    // a tile's rows (plus one step on each side) are addressed with 32-bit
    // buffer offsets below 2^31
    // (4 bytes at least: bf16 input may be written as f32)
    const int64_t wb = elem_bytes(state_dtype) > 4 ? elem_bytes(state_dtype) : 4;
    int64_t tile_bytes;
    if (!mul_ok(p->L + 2, d, &tile_bytes) || !mul_ok(tile_bytes, wb, &tile_bytes) || tile_bytes >= (int64_t)INT32_MAX)
        return false;
    const bool cplx = state_dtype == MEMOROID_C64;
    const size_t agg_b = cplx ? 16 : 8, incl_b = cplx ? 8 : 4;
    int64_t ndesc;
    if (!mul_ok(p->ntiles, p->Dp, &ndesc)) return false;
    if (ndesc > INT64_MAX / 32) return false;
    size_t off = kAlign;                                   // header
    p->off_ctr = off;                                      // per-chain tile counters
    off = align_up(off + (size_t)p->nchains * (size_t)ctr_groups * kCtrStride * 4);
    // bank 0 of the self-validating words, then bank 1 with the same layout
    const size_t bank0 = off;
    p->off_agg = off;
    off = align_up(off + (size_t)ndesc * agg_b);
    p->off_incl = off;
    off = align_up(off + (size_t)ndesc * incl_b);
    p->off_cnt = off;                                      // begin-count words, [tiles per chain][B]
    if (!bwd) off = align_up(off + (size_t)p->nt * (size_t)B * 8);
    const bool fused = bwd && ainv && want_grad_a && B == 1;
    if (fused) {
        // one tape: the partial rows are self-validating 64-bit words, banked
        // with the descriptors, and the chain's last tile sums them
        p->fused_da = true;
        p->off_part = off;
        off = align_up(off + (size_t)p->nt * (size_t)d * 8);
    }
    p->bank_bytes = off - bank0;
    p->init_bytes = off;
    off += p->bank_bytes;
    if (bwd && ainv && want_grad_a && !fused) {
        const size_t sb = cplx ? 8 : 4;
        const int64_t rows_part = p->nt * B;
        p->off_part = off;
        off = align_up(off + (size_t)rows_part * (size_t)d * sb);
        const int64_t r1 = (rows_part + 63) / 64, r2 = (r1 + 63) / 64;
        p->off_sum1 = off;
        off = align_up(off + (size_t)r1 * (size_t)d * sb);
        p->off_sum2 = off;
        off = align_up(off + (size_t)r2 * (size_t)d * sb);
    }
    p->total = off;
    return true;
}

int check_hip(hipError_t e) { return e == hipSuccess ? MEMOROID_OK : MEMOROID_EHIP; }

// How a call treats its workspace (include/memoroid.h): a self-initialising
// call first fills the part its kernels read before writing (header, tile
// counters or epoch words, the bank the first epoch uses) with all-ones
// bytes, which is exactly the state memoroid_workspace_prepare leaves; the
// kernels then run as the first call on a prepared workspace.  A prepared
// call launches the kernels alone.
// kNoAlloc: self-initialising, on the library's own static scratch array
// instead of a caller's workspace (memoroid_scan_diag_noalloc).
enum class WsMode { kSelfInit, kPrepared, kNoAlloc };

int init_if_self(WsMode mode, void* ws, size_t init_bytes, hipStream_t s) {
    if (mode == WsMode::kPrepared) return MEMOROID_OK;
    return check_hip(ws_init_launch(nullptr, 0, ws, init_bytes, s));
}

}  // namespace

// ---------------------------------------------------------- static scratch
// Workspace of memoroid_scan_diag_noalloc: one fixed array in device memory,
// held by every GPU that the library runs on until the process ends.  In
// host code `scratch` names a host-side stand-in, never the device array:
// host code uses only the address hipGetSymbolAddress returns for the
// current device (each GPU holds its own copy at its own address).
constexpr size_t kNoAllocScratchBytes = MEMOROID_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of the current device's scratch array, looked up on the
// first call made with that device current and kept.
int scratch_address(void** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return MEMOROID_EHIP;
    if (dev < 0 || dev >= kMaxDevices) return MEMOROID_EUNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[dev] == nullptr) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || ptr == nullptr) return MEMOROID_EHIP;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return MEMOROID_OK;
}

// Workspace fields of a diagonal scan's arguments: counters and bank-0
// descriptor regions at `base` (the plan's offset 0), header at `hdr`.
template <class Args>
void set_scan_ws(Args& a, const DiagPlan& p, char* base, WsHeader* hdr, uint64_t sig) {
    a.nt = p.nt;
    a.agg = base + p.off_agg;
    a.incl = base + p.off_incl;
    a.bank = (int64_t)p.bank_bytes;
    a.hdr = hdr;
    a.sig = sig;
    a.ctr = (uint32_t*)(base + p.off_ctr);
}

bool diag_dtypes_ok(int in_dt, int out_dt) {
    return (in_dt == MEMOROID_F32 && out_dt == MEMOROID_F32) || (in_dt == MEMOROID_BF16 && out_dt == MEMOROID_BF16) ||
           (in_dt == MEMOROID_BF16 && out_dt == MEMOROID_F32) || (in_dt == MEMOROID_C64 && out_dt == MEMOROID_C64);
}


// Reduce a [rows][cols] float matrix over rows into out[cols] in a fixed
// order: one pass when there are at most 1024 rows (256 per wavefront),
// otherwise passes of 64 rows until that holds.
int reduce_rows(const float* part, float* s1, float* s2, float* out, int64_t rows, int64_t cols,
                hipStream_t s) {
    const float* cur = part;
    float* bufs[2] = {s1, s2};
    int which = 0;
    while (rows > 1024) {
        if (colsum_launch(cur, bufs[which], rows, cols, 16, s) != hipSuccess) return MEMOROID_EHIP;
        cur = bufs[which];
        which ^= 1;
        rows = (rows + 63) / 64;
    }
    const int64_t rpw = rows > 0 ? (rows + 3) / 4 : 1;
    return check_hip(colsum_launch(cur, out, rows, cols, rpw, s));
}

}  // namespace

extern "C" {

int memoroid_abi_version(void) { return MEMOROID_ABI_VERSION; }

const char* memoroid_status_string(int status) {
    switch (status) {
        case MEMOROID_OK: return "ok";
        case MEMOROID_EINVAL: return "invalid argument (pointer, extent, stride, alignment or aliasing)";
        case MEMOROID_EUNSUPPORTED: return "unsupported dtype combination or shape";
        case MEMOROID_EWORKSPACE: return "workspace missing or too small";
        case MEMOROID_EHIP: return "HIP runtime error";
        case MEMOROID_ETIMEOUT: return "a cross-tile wait gave up; outputs are invalid";
        case MEMOROID_EMISMATCH:
            return "workspace prepared for (bound to) another call; outputs are invalid, prepare it again";
        default: return "unknown status";
    }
}

// ------------------------------------------------------------- diag forward

size_t memoroid_scan_diag_workspace_bytes(int64_t B, int64_t T, int64_t d, int in_dtype, int out_dtype) {
    if (B < 0 || T < 0 || d < 0 || !diag_dtypes_ok(in_dtype, out_dtype)) return 0;
    if (B == 0 || T == 0 || d == 0) return 0;
    DiagPlan pv, ps;
    const int sd = in_dtype == MEMOROID_C64 ? MEMOROID_C64 : (in_dtype == MEMOROID_BF16 ? MEMOROID_BF16 : MEMOROID_F32);
    size_t best = 0;
    for (int vec = 0; vec < 2; ++vec) {
        for (int ainv = 0; ainv < 2; ++ainv) {
            DiagPlan& p = vec ? pv : ps;
            if (!plan_diag(B, T, d, sd, vec, diag_fwd_rows(sd, vec, ainv), false, ainv, false, &p)) return 0;
            if (p.total > best) best = p.total;
        }
    }
    return best;
}

static int scan_diag_run(const void* a, int64_t a_stride_t, const void* x, const uint8_t* start, void* h,
                         int32_t* episode_idx, int64_t B, int64_t T, int64_t d, int in_dtype, int out_dtype,
                         void* workspace, size_t workspace_bytes, void* stream, WsMode mode) {
    if (B < 0 || T < 0 || d < 0) return MEMOROID_EINVAL;
    if (!diag_dtypes_ok(in_dtype, out_dtype)) return MEMOROID_EUNSUPPORTED;
    if (B == 0 || T == 0 || d == 0) return MEMOROID_OK;
    int64_t BT, BTd;
    if (!mul_ok(B, T, &BT) || !mul_ok(BT, d, &BTd) || BTd > INT64_MAX / 16) return MEMOROID_EINVAL;
    if (!a || !x || !start || !h) return MEMOROID_EINVAL;
    if (a_stride_t != 0 && a_stride_t != d) return MEMOROID_EINVAL;
    const int ib = elem_bytes(in_dtype), ob = elem_bytes(out_dtype);
    if (!aligned(a, ib) || !aligned(x, ib) || !aligned(h, ob) || (episode_idx && !aligned(episode_idx, 4)))
        return MEMOROID_EINVAL;
    if (h == x || h == a || (const void*)episode_idx == (const void*)h || (const void*)episode_idx == x ||
        (const void*)episode_idx == a || (const void*)episode_idx == (const void*)start)
        return MEMOROID_EINVAL;
    const bool ainv = a_stride_t == 0;
    const int VW = vec_width(in_dtype);
    const bool vec = d % VW == 0 && aligned(x, 16) && aligned(h, 16) && aligned(a, 16);
    const int sd = in_dtype == MEMOROID_C64 ? MEMOROID_C64 : (in_dtype == MEMOROID_BF16 ? MEMOROID_BF16 : MEMOROID_F32);
    DiagPlan p;
    if (!plan_diag(B, T, d, sd, vec, diag_fwd_rows(sd, vec, ainv), false, ainv, false, &p))
        return MEMOROID_EUNSUPPORTED;
    if (mode == WsMode::kNoAlloc) {
        // the plan's own size (the scratch array is never shared with
        // another plan's call in flight, so the query's maximum over plans
        // is not needed)
        if (p.total > kNoAllocScratchBytes) return MEMOROID_EWORKSPACE;
        const int st = scratch_address(&workspace);
        if (st != MEMOROID_OK) return st;
        workspace_bytes = kNoAllocScratchBytes;
    } else {
        if (!workspace) return MEMOROID_EWORKSPACE;
        if (workspace_bytes < memoroid_scan_diag_workspace_bytes(B, T, d, in_dtype, out_dtype) ||
            workspace_bytes < p.total)
            return MEMOROID_EWORKSPACE;
    }
    if (!aligned(workspace, 16)) return MEMOROID_EINVAL;

    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    DiagFwdArgs args{};
    args.a = a;
    args.x = x;
    args.start = start;
    args.h = h;
    args.T = T;
    args.d = d;
    args.Qp = p.Qp;
    args.nfb = p.nfb;
    args.nchains = (int32_t)p.nchains;
    set_scan_ws(args, p, ws, (WsHeader*)ws, layout_sig({kSigDiag, B, T, d, sd, vec, ainv}));
    args.idx = episode_idx;
    args.cnt = (uint64_t*)(ws + p.off_cnt);
    const int ik = in_dtype == MEMOROID_F32 ? K_F32 : in_dtype == MEMOROID_BF16 ? K_BF16 : K_C64;
    const int ok = out_dtype == MEMOROID_F32 ? K_F32 : out_dtype == MEMOROID_BF16 ? K_BF16 : K_C64;
    const int st = init_if_self(mode, ws, p.init_bytes, s);
    if (st != MEMOROID_OK) return st;
    if (diag_fwd_launch(ik, ok, vec, ainv, args, p.ntiles, s) != hipSuccess) return MEMOROID_EHIP;
    return MEMOROID_OK;
}

int memoroid_scan_diag(const void* a, int64_t a_stride_t, const void* x, const uint8_t* start, void* h,
                       int32_t* episode_idx, int64_t B, int64_t T, int64_t d, int in_dtype, int out_dtype,
                       void* workspace, size_t workspace_bytes, void* stream) {
    return scan_diag_run(a, a_stride_t, x, start, h, episode_idx, B, T, d, in_dtype, out_dtype, workspace,
                         workspace_bytes, stream, WsMode::kSelfInit);
}

int memoroid_scan_diag_prepared(const void* a, int64_t a_stride_t, const void* x, const uint8_t* start, void* h,
                                int32_t* episode_idx, int64_t B, int64_t T, int64_t d, int in_dtype,
                                int out_dtype, void* workspace, size_t workspace_bytes, void* stream) {
    return scan_diag_run(a, a_stride_t, x, start, h, episode_idx, B, T, d, in_dtype, out_dtype, workspace,
                         workspace_bytes, stream, WsMode::kPrepared);
}

int memoroid_scan_diag_noalloc(const void* a, int64_t a_stride_t, const void* x, const uint8_t* start, void* h,
                               int32_t* episode_idx, int64_t B, int64_t T, int64_t d, int in_dtype, int out_dtype,
                               void* stream) {
    return scan_diag_run(a, a_stride_t, x, start, h, episode_idx, B, T, d, in_dtype, out_dtype, nullptr, 0, stream,
                         WsMode::kNoAlloc);
}

// ------------------------------------------------------------------- FFM

size_t memoroid_scan_ffm_workspace_bytes(int64_t B, int64_t T, int64_t m, int64_t c) {
    int64_t d;
    if (B <= 0 || T <= 0 || m <= 0 || c <= 0 || !mul_ok(m, c, &d)) return 0;
    size_t best = 0;
    for (int vec = 0; vec < 2; ++vec) {
        DiagPlan p;
        if (!plan_diag(B, T, d, MEMOROID_C64, vec, kFfmFwdRows, false, true, false, &p, (int)kXcds)) return 0;
        if (p.total > best) best = p.total;
    }
    return best;
}

static int scan_ffm_run(const float* alpha, const float* omega, const float* x, const uint8_t* start, void* S,
                        int32_t* episode_idx, int64_t B, int64_t T, int64_t m, int64_t c, void* workspace,
                        size_t workspace_bytes, void* stream, WsMode mode) {
    if (B < 0 || T < 0 || m < 0 || c < 0) return MEMOROID_EINVAL;
    if (B == 0 || T == 0 || m == 0 || c == 0) return MEMOROID_OK;
    int64_t d, BT, BTd;
    if (!mul_ok(m, c, &d) || !mul_ok(B, T, &BT) || !mul_ok(BT, d, &BTd) || BTd > INT64_MAX / 16)
        return MEMOROID_EINVAL;
    if (!alpha || !omega || !x || !start || !S) return MEMOROID_EINVAL;
    if (!aligned(alpha, 4) || !aligned(omega, 4) || !aligned(x, 4) || !aligned(S, 8) ||
        (episode_idx && !aligned(episode_idx, 4)))
        return MEMOROID_EINVAL;
    if (S == (const void*)x || S == (const void*)alpha || S == (const void*)omega || S == (const void*)start ||
        (const void*)episode_idx == S || (const void*)episode_idx == (const void*)x ||
        (const void*)episode_idx == (const void*)start)
        return MEMOROID_EINVAL;
    // two features per lane when they always share a row of x (c even)
    const bool vec = c % 2 == 0 && aligned(S, 16);
    DiagPlan p;
    if (!plan_diag(B, T, d, MEMOROID_C64, vec, kFfmFwdRows, false, true, false, &p, (int)kXcds))
        return MEMOROID_EUNSUPPORTED;
    if (!workspace) return MEMOROID_EWORKSPACE;
    if (workspace_bytes < memoroid_scan_ffm_workspace_bytes(B, T, m, c) || workspace_bytes < p.total)
        return MEMOROID_EWORKSPACE;
    if (!aligned(workspace, 16)) return MEMOROID_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    DiagFwdArgs args{};
    args.a = nullptr;
    args.x = x;
    args.start = start;
    args.h = S;
    args.T = T;
    args.d = d;
    args.Qp = p.Qp;
    args.nfb = p.nfb;
    args.nchains = (int32_t)p.nchains;
    set_scan_ws(args, p, ws, (WsHeader*)ws, layout_sig({kSigFfm, B, T, m, c, vec}));
    args.idx = episode_idx;
    args.cnt = (uint64_t*)(ws + p.off_cnt);
    args.alpha = alpha;
    args.omega = omega;
    args.ffm_m = m;
    args.ffm_c = c;
    const int st = init_if_self(mode, ws, p.init_bytes, s);
    if (st != MEMOROID_OK) return st;
    return check_hip(ffm_fwd_launch(vec, args, p.ntiles, s));
}

int memoroid_scan_ffm(const float* alpha, const float* omega, const float* x, const uint8_t* start, void* S,
                      int32_t* episode_idx, int64_t B, int64_t T, int64_t m, int64_t c, void* workspace,
                      size_t workspace_bytes, void* stream) {
    return scan_ffm_run(alpha, omega, x, start, S, episode_idx, B, T, m, c, workspace, workspace_bytes, stream,
                        WsMode::kSelfInit);
}

int memoroid_scan_ffm_prepared(const float* alpha, const float* omega, const float* x, const uint8_t* start,
                               void* S, int32_t* episode_idx, int64_t B, int64_t T, int64_t m, int64_t c,
                               void* workspace, size_t workspace_bytes, void* stream) {
    return scan_ffm_run(alpha, omega, x, start, S, episode_idx, B, T, m, c, workspace, workspace_bytes, stream,
                        WsMode::kPrepared);
}

// ------------------------------------------------------------ FFM gradient

namespace {

// The scan's workspace, then the summed da (complex [m][c]), then the
// chain-major input gradient [B][nfb][T][Dp / c] (floats).
bool ffm_bwd_plan(int64_t B, int64_t T, int64_t m, int64_t c, bool vec, bool params, DiagPlan* p,
                  size_t* off_da, size_t* off_dxw, size_t* total) {
    int64_t d;
    if (!mul_ok(m, c, &d)) return false;
    if (!plan_diag(B, T, d, MEMOROID_C64, vec, kFfmBwdRows, true, true, params, p)) return false;
    *off_da = align_up(p->total);
    *off_dxw = align_up(*off_da + (size_t)(params ? d : 1) * 8);
    const int64_t jpc = c <= p->Dp ? p->Dp / c : 1;
    int64_t n;
    if (!mul_ok(B * (int64_t)p->nfb, T, &n) || !mul_ok(n, jpc, &n) || n > INT64_MAX / 8) return false;
    *total = align_up(*off_dxw + (size_t)n * 4);
    return true;
}

bool pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

}  // namespace

size_t memoroid_scan_ffm_bwd_workspace_bytes(int64_t B, int64_t T, int64_t m, int64_t c) {
    if (B <= 0 || T <= 0 || m <= 0 || c <= 0) return 0;
    size_t best = 0;
    for (int vec = 0; vec < 2; ++vec) {
        DiagPlan p;
        size_t off_da, off_dxw, total;
        if (!ffm_bwd_plan(B, T, m, c, vec, true, &p, &off_da, &off_dxw, &total)) return 0;
        if (total > best) best = total;
    }
    return best;
}

static int scan_ffm_bwd_run(const float* alpha, const float* omega, const uint8_t* start, const void* S,
                            const void* grad_S, float* grad_x, float* grad_alpha, float* grad_omega, int64_t B,
                            int64_t T, int64_t m, int64_t c, void* workspace, size_t workspace_bytes, void* stream,
                            WsMode mode) {
    if (B < 0 || T < 0 || m < 0 || c < 0) return MEMOROID_EINVAL;
    if (B == 0 || T == 0 || m == 0 || c == 0) return MEMOROID_OK;
    int64_t d, BT, BTd;
    if (!mul_ok(m, c, &d) || !mul_ok(B, T, &BT) || !mul_ok(BT, d, &BTd) || BTd > INT64_MAX / 16)
        return MEMOROID_EINVAL;
    const bool params = grad_alpha || grad_omega;
    if (!alpha || !omega || !start || !grad_S || !grad_x || (params && !S)) return MEMOROID_EINVAL;
    if (!aligned(alpha, 4) || !aligned(omega, 4) || !aligned(grad_S, 8) || !aligned(grad_x, 4) ||
        (S && !aligned(S, 8)) || (grad_alpha && !aligned(grad_alpha, 4)) || (grad_omega && !aligned(grad_omega, 4)))
        return MEMOROID_EINVAL;
    const void* ins[5] = {alpha, omega, start, S, grad_S};
    const void* outs[3] = {grad_x, grad_alpha, grad_omega};
    for (int o = 0; o < 3; ++o) {
        if (!outs[o]) continue;
        for (int i = 0; i < 5; ++i)
            if (ins[i] && outs[o] == ins[i]) return MEMOROID_EINVAL;
        for (int o2 = 0; o2 < o; ++o2)
            if (outs[o2] && outs[o] == outs[o2]) return MEMOROID_EINVAL;
    }
    // two features per lane only when they always share a row of x (c even)
    const bool vec = c % 2 == 0 && aligned(grad_S, 16) && (!S || aligned(S, 16));
    DiagPlan p;
    size_t off_da, off_dxw, total;
    if (!ffm_bwd_plan(B, T, m, c, vec, params, &p, &off_da, &off_dxw, &total)) return MEMOROID_EUNSUPPORTED;
    // the real input's gradient is reduced over the c columns inside the
    // kernel: c must be a power of two that divides the chain width
    if (!pow2(c) || c > p.Dp) return MEMOROID_EUNSUPPORTED;
    if (!workspace || workspace_bytes < total) return MEMOROID_EWORKSPACE;
    if (!aligned(workspace, 16)) return MEMOROID_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    DiagBwdArgs args{};
    args.a = nullptr;
    args.start = start;
    args.h = S;
    args.g = grad_S;
    args.dx = nullptr;
    args.da = nullptr;
    args.da_part = params ? ws + p.off_part : nullptr;
    args.da_out = (params && p.fused_da) ? ws + off_da : nullptr;
    args.T = T;
    args.d = d;
    args.Qp = p.Qp;
    args.nfb = p.nfb;
    args.nchains = (int32_t)p.nchains;
    set_scan_ws(args, p, ws, (WsHeader*)ws, layout_sig({kSigFfmBwd, B, T, m, c, vec, params}));
    args.alpha = alpha;
    args.omega = omega;
    args.ffm_m = m;
    args.ffm_c = c;
    args.dxr = (float*)(ws + off_dxw);
    const int sti = init_if_self(mode, ws, p.init_bytes, s);
    if (sti != MEMOROID_OK) return sti;
    if (ffm_bwd_launch(vec, args, p.ntiles, s) != hipSuccess) return MEMOROID_EHIP;
    float* da = (float*)(ws + off_da);
    if (params && !p.fused_da) {
        const int st = reduce_rows((const float*)(ws + p.off_part), (float*)(ws + p.off_sum1),
                                   (float*)(ws + p.off_sum2), da, p.nt * B, 2 * d, s);
        if (st != MEMOROID_OK) return st;
    }
    FfmFinishArgs fa{};
    fa.dxw = (const float*)(ws + off_dxw);
    fa.dx = grad_x;
    fa.B = B;
    fa.T = T;
    fa.m = m;
    fa.c = c;
    fa.jpc = p.Dp / c;
    fa.alpha = alpha;
    fa.omega = omega;
    fa.da = da;
    fa.dalpha = params ? grad_alpha : nullptr;
    fa.domega = params ? grad_omega : nullptr;
    return check_hip(ffm_bwd_finish_launch(fa, s));
}

int memoroid_scan_ffm_bwd(const float* alpha, const float* omega, const uint8_t* start, const void* S,
                          const void* grad_S, float* grad_x, float* grad_alpha, float* grad_omega, int64_t B,
                          int64_t T, int64_t m, int64_t c, void* workspace, size_t workspace_bytes, void* stream) {
    return scan_ffm_bwd_run(alpha, omega, start, S, grad_S, grad_x, grad_alpha, grad_omega, B, T, m, c, workspace,
                            workspace_bytes, stream, WsMode::kSelfInit);
}

int memoroid_scan_ffm_bwd_prepared(const float* alpha, const float* omega, const uint8_t* start, const void* S,
                                   const void* grad_S, float* grad_x, float* grad_alpha, float* grad_omega,
                                   int64_t B, int64_t T, int64_t m, int64_t c, void* workspace,
                                   size_t workspace_bytes, void* stream) {
    return scan_ffm_bwd_run(alpha, omega, start, S, grad_S, grad_x, grad_alpha, grad_omega, B, T, m, c, workspace,
                            workspace_bytes, stream, WsMode::kPrepared);
}

// ------------------------------------------------------------ diag backward

size_t memoroid_scan_diag_bwd_workspace_bytes(int64_t B, int64_t T, int64_t d, int dtype, int64_t a_stride_t) {
    if (B < 0 || T < 0 || d < 0 || (dtype != MEMOROID_F32 && dtype != MEMOROID_C64)) return 0;
    if (B == 0 || T == 0 || d == 0) return 0;
    size_t best = 0;
    for (int vec = 0; vec < 2; ++vec) {
        DiagPlan p;
        if (!plan_diag(B, T, d, dtype, vec, diag_bwd_rows(dtype, vec, a_stride_t == 0), true, a_stride_t == 0, true,
                       &p))
            return 0;
        if (p.total > best) best = p.total;
    }
    return best;
}

static int scan_diag_bwd_run(const void* a, int64_t a_stride_t, const uint8_t* start, const void* h,
                             const void* grad_h, void* grad_x, void* grad_a, int64_t B, int64_t T, int64_t d,
                             int dtype, void* workspace, size_t workspace_bytes, void* stream, WsMode mode) {
    if (B < 0 || T < 0 || d < 0) return MEMOROID_EINVAL;
    if (dtype != MEMOROID_F32 && dtype != MEMOROID_C64) return MEMOROID_EUNSUPPORTED;
    if (B == 0 || T == 0 || d == 0) return MEMOROID_OK;
    int64_t BT, BTd;
    if (!mul_ok(B, T, &BT) || !mul_ok(BT, d, &BTd) || BTd > INT64_MAX / 16) return MEMOROID_EINVAL;
    if (!a || !start || !grad_h || !grad_x || (grad_a && !h)) return MEMOROID_EINVAL;
    if (a_stride_t != 0 && a_stride_t != d) return MEMOROID_EINVAL;
    const int eb = elem_bytes(dtype);
    if (!aligned(a, eb) || !aligned(grad_h, eb) || !aligned(grad_x, eb) || (h && !aligned(h, eb)) ||
        (grad_a && !aligned(grad_a, eb)))
        return MEMOROID_EINVAL;
    if (grad_x == grad_h || grad_x == a || (h && grad_x == h) ||
        (grad_a && (grad_a == grad_x || grad_a == grad_h || grad_a == a || grad_a == h)))
        return MEMOROID_EINVAL;
    const bool ainv = a_stride_t == 0;
    const int VW = vec_width(dtype);
    const bool vec = d % VW == 0 && aligned(a, 16) && aligned(grad_h, 16) && aligned(grad_x, 16) &&
                     (!h || aligned(h, 16)) && (!grad_a || aligned(grad_a, 16));
    DiagPlan p;
    if (!plan_diag(B, T, d, dtype, vec, diag_bwd_rows(dtype, vec, ainv), true, ainv, grad_a != nullptr, &p))
        return MEMOROID_EUNSUPPORTED;
    if (!workspace) return MEMOROID_EWORKSPACE;
    if (workspace_bytes < memoroid_scan_diag_bwd_workspace_bytes(B, T, d, dtype, a_stride_t) ||
        workspace_bytes < p.total)
        return MEMOROID_EWORKSPACE;
    if (!aligned(workspace, 16)) return MEMOROID_EINVAL;

    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    DiagBwdArgs args{};
    args.a = a;
    args.start = start;
    args.h = h;
    args.g = grad_h;
    args.dx = grad_x;
    args.da = ainv ? nullptr : grad_a;
    args.da_part = (ainv && grad_a) ? ws + p.off_part : nullptr;
    args.da_out = (ainv && grad_a && p.fused_da) ? grad_a : nullptr;
    args.T = T;
    args.d = d;
    args.Qp = p.Qp;
    args.nfb = p.nfb;
    args.nchains = (int32_t)p.nchains;
    set_scan_ws(args, p, ws, (WsHeader*)ws,
                layout_sig({kSigDiagBwd, B, T, d, dtype, vec, ainv, grad_a != nullptr}));
    const int k = dtype == MEMOROID_F32 ? K_F32 : K_C64;
    const int64_t cols = d * (dtype == MEMOROID_C64 ? 2 : 1);
    const int sti = init_if_self(mode, ws, p.init_bytes, s);
    if (sti != MEMOROID_OK) return sti;
    if (diag_bwd_launch(k, vec, ainv, args, p.ntiles, s) != hipSuccess) return MEMOROID_EHIP;
    if (ainv && grad_a && !p.fused_da) {
        const int st = reduce_rows((const float*)(ws + p.off_part), (float*)(ws + p.off_sum1),
                                   (float*)(ws + p.off_sum2), (float*)grad_a, p.nt * B, cols, s);
        if (st != MEMOROID_OK) return st;
    }
    return MEMOROID_OK;
}

int memoroid_scan_diag_bwd(const void* a, int64_t a_stride_t, const uint8_t* start, const void* h,
                           const void* grad_h, void* grad_x, void* grad_a, int64_t B, int64_t T, int64_t d,
                           int dtype, void* workspace, size_t workspace_bytes, void* stream) {
    return scan_diag_bwd_run(a, a_stride_t, start, h, grad_h, grad_x, grad_a, B, T, d, dtype, workspace,
                             workspace_bytes, stream, WsMode::kSelfInit);
}

int memoroid_scan_diag_bwd_prepared(const void* a, int64_t a_stride_t, const uint8_t* start, const void* h,
                                    const void* grad_h, void* grad_x, void* grad_a, int64_t B, int64_t T,
                                    int64_t d, int dtype, void* workspace, size_t workspace_bytes, void* stream) {
    return scan_diag_bwd_run(a, a_stride_t, start, h, grad_h, grad_x, grad_a, B, T, d, dtype, workspace,
                             workspace_bytes, stream, WsMode::kPrepared);
}

// ---------------------------------------------------------- linear attention
// Summaries per (chunk, head) -> resettable sum-scan of the chunk states over
// chunks (the diagonal scan with a = 1, the monoid of App. G.1 being a sum)
// -> outputs per (chunk, head).

namespace {

struct LinPlan {
    int64_t nch = 0, dstate = 0;
    size_t off_dS = 0, off_Sinc = 0, off_R = 0, off_scan = 0, off_cnt = 0, total = 0;
    DiagPlan scan;
};

bool plan_linattn(int64_t T, int64_t H, LinPlan* p) {
    p->nch = (T + kLinChunk - 1) / kLinChunk;
    p->dstate = H * kLinStateWords;
    const size_t states = (size_t)p->nch * (size_t)p->dstate * 4;
    // the state scan's own workspace comes first, so that its header (and
    // timeout word) sits at offset 0 like every other call's; the chunk
    // begin-count words follow its descriptors so one fill covers both
    size_t off = 0;
    p->off_scan = off;
    // the state scan always runs vectorised: dstate % 4 == 0 and every
    // buffer is 256-byte aligned inside the workspace
    if (!plan_diag(1, p->nch, p->dstate, MEMOROID_F32, true, diag_rows(false, true), false, true, false, &p->scan))
        return false;
    off = align_up(off + p->scan.total);
    p->off_cnt = off;
    off = align_up(off + (size_t)p->nch * 8);
    p->off_dS = off;
    off = align_up(off + states);
    p->off_Sinc = off;
    off = align_up(off + states);
    p->off_R = off;
    off = align_up(off + (size_t)p->nch);
    p->total = off;
    return true;
}

}  // namespace

size_t memoroid_scan_linattn_workspace_bytes(int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t chunk) {
    if (T <= 0 || H <= 0 || dk != 64 || dv != 64 || chunk != 64) return 0;
    if (T > (int64_t)INT32_MAX / 2 || H > 65535) return 0;
    LinPlan p;
    if (!plan_linattn(T, H, &p)) return 0;
    return p.total;
}

int memoroid_scan_linattn(const float* q, const float* k, const float* v, const uint8_t* start, float* out,
                          int32_t* episode_idx, int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t chunk,
                          void* workspace, size_t workspace_bytes, void* stream) {
    if (T < 0 || H < 0 || dk < 0 || dv < 0 || chunk < 0) return MEMOROID_EINVAL;
    if (dk != 64 || dv != 64 || chunk != 64) return MEMOROID_EUNSUPPORTED;
    if (T == 0 || H == 0) return MEMOROID_OK;
    if (T > (int64_t)INT32_MAX / 2 || H > 65535) return MEMOROID_EUNSUPPORTED;
    if (!q || !k || !v || !start || !out) return MEMOROID_EINVAL;
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(out, 16) ||
        (episode_idx && !aligned(episode_idx, 4)))
        return MEMOROID_EINVAL;
    if (out == q || out == k || out == v ||
        (episode_idx && ((void*)episode_idx == (void*)out || (const void*)episode_idx == (const void*)start)))
        return MEMOROID_EINVAL;
    LinPlan p;
    if (!plan_linattn(T, H, &p)) return MEMOROID_EUNSUPPORTED;
    if (!workspace) return MEMOROID_EWORKSPACE;
    if (workspace_bytes < p.total) return MEMOROID_EWORKSPACE;
    if (!aligned(workspace, 256)) return MEMOROID_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    char* sw = ws + p.off_scan;
    float* dS = (float*)(ws + p.off_dS);
    float* Sinc = (float*)(ws + p.off_Sinc);
    uint8_t* R = (uint8_t*)(ws + p.off_R);
    LinSummaryArgs sa{};
    sa.k = k;
    sa.v = v;
    sa.start = start;
    sa.dS = dS;
    sa.R = R;
    sa.T = T;
    sa.H = H;
    // the summary kernel prepares the state scan's workspace and the count
    // words (one contiguous run from offset 0) on every call
    sa.fill = (u32x4*)sw;
    sa.fill16 = (int64_t)((p.off_cnt + (size_t)p.nch * 8 - p.off_scan + 15) / 16);
    if (linattn_summary_launch(sa, s) != hipSuccess) return MEMOROID_EHIP;
    DiagFwdArgs args{};
    args.a = nullptr;            // a = 1: the state scan is a resettable sum
    args.x = dS;
    args.start = R;
    args.h = Sinc;
    args.T = p.nch;
    args.d = p.dstate;
    args.Qp = p.scan.Qp;
    args.nfb = p.scan.nfb;
    args.nchains = (int32_t)p.scan.nchains;
    set_scan_ws(args, p.scan, sw, (WsHeader*)sw, layout_sig({kSigLinattn, T, H}));
    args.idx = nullptr;
    args.cnt = nullptr;
    if (diag_fwd_launch(K_F32, K_F32, true, true, args, p.scan.ntiles, s) != hipSuccess) return MEMOROID_EHIP;
    LinOutputArgs oa{};
    oa.q = q;
    oa.k = k;
    oa.v = v;
    oa.start = start;
    oa.Sinc = Sinc;
    oa.out = out;
    oa.T = T;
    oa.H = H;
    oa.idx = episode_idx;
    oa.cnt = (uint64_t*)(ws + p.off_cnt);
    oa.timeout = &((WsHeader*)sw)->timeout;
    if (linattn_output_launch(oa, s) != hipSuccess) return MEMOROID_EHIP;
    return MEMOROID_OK;
}

// ------------------------------------------------- linear attention, grad

namespace {

struct LinBwdPlan {
    LinPlan fwd;                 // the forward summaries and state scan, from offset 0
    DiagPlan rscan;              // the reverse chunk-state scan
    size_t off_dnum = 0, off_dden = 0, off_dU = 0, off_Y = 0, off_Rs = 0, off_rscan = 0, total = 0;
};

bool plan_linattn_bwd(int64_t T, int64_t H, LinBwdPlan* p) {
    if (!plan_linattn(T, H, &p->fwd)) return false;
    const int64_t nch = p->fwd.nch;
    const size_t states = (size_t)nch * (size_t)p->fwd.dstate * 4;
    size_t off = align_up(p->fwd.total);
    p->off_dnum = off;
    off = align_up(off + (size_t)T * (size_t)H * kLinChunk * 4);
    p->off_dden = off;
    off = align_up(off + (size_t)T * (size_t)H * 4);
    p->off_dU = off;
    off = align_up(off + states);
    p->off_Y = off;
    off = align_up(off + states);
    p->off_Rs = off;
    off = align_up(off + (size_t)nch);
    if (!plan_diag(1, nch, p->fwd.dstate, MEMOROID_F32, true, diag_rows(true, true), true, true, false, &p->rscan))
        return false;
    p->off_rscan = off;
    off = align_up(off + p->rscan.total);
    p->total = off;
    return true;
}

}  // namespace

size_t memoroid_scan_linattn_bwd_workspace_bytes(int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t chunk) {
    if (T <= 0 || H <= 0 || dk != 64 || dv != 64 || chunk != 64) return 0;
    if (T > (int64_t)INT32_MAX / 2 || H > 65535) return 0;
    LinBwdPlan p;
    if (!plan_linattn_bwd(T, H, &p)) return 0;
    return p.total;
}

int memoroid_scan_linattn_bwd(const float* q, const float* k, const float* v, const uint8_t* start,
                              const float* out, const float* grad_out, float* grad_q, float* grad_k, float* grad_v,
                              int64_t T, int64_t H, int64_t dk, int64_t dv, int64_t chunk, void* workspace,
                              size_t workspace_bytes, void* stream) {
    if (T < 0 || H < 0 || dk < 0 || dv < 0 || chunk < 0) return MEMOROID_EINVAL;
    if (dk != 64 || dv != 64 || chunk != 64) return MEMOROID_EUNSUPPORTED;
    if (T == 0 || H == 0) return MEMOROID_OK;
    if (T > (int64_t)INT32_MAX / 2 || H > 65535) return MEMOROID_EUNSUPPORTED;
    const float* ins[6] = {q, k, v, out, grad_out, nullptr};
    float* outs[3] = {grad_q, grad_k, grad_v};
    for (int i = 0; i < 5; ++i)
        if (!ins[i] || !aligned(ins[i], 16)) return MEMOROID_EINVAL;
    if (!start) return MEMOROID_EINVAL;
    for (int o = 0; o < 3; ++o) {
        if (!outs[o] || !aligned(outs[o], 16)) return MEMOROID_EINVAL;
        for (int i = 0; i < 5; ++i)
            if ((const float*)outs[o] == ins[i]) return MEMOROID_EINVAL;
        for (int o2 = 0; o2 < o; ++o2)
            if (outs[o] == outs[o2]) return MEMOROID_EINVAL;
    }
    LinBwdPlan p;
    if (!plan_linattn_bwd(T, H, &p)) return MEMOROID_EUNSUPPORTED;
    if (!workspace || workspace_bytes < p.total) return MEMOROID_EWORKSPACE;
    if (!aligned(workspace, 256)) return MEMOROID_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    const LinPlan& f = p.fwd;
    char* sw = ws + f.off_scan;
    float* dS = (float*)(ws + f.off_dS);
    float* Sinc = (float*)(ws + f.off_Sinc);
    uint8_t* R = (uint8_t*)(ws + f.off_R);

    // forward chunk states (as in the forward pass, without the readout)
    LinSummaryArgs sa{};
    sa.k = k;
    sa.v = v;
    sa.start = start;
    sa.dS = dS;
    sa.R = R;
    sa.T = T;
    sa.H = H;
    sa.fill = (u32x4*)sw;
    sa.fill16 = (int64_t)((f.off_cnt + (size_t)f.nch * 8 - f.off_scan + 15) / 16);
    if (linattn_summary_launch(sa, s) != hipSuccess) return MEMOROID_EHIP;
    const uint64_t sig = layout_sig({kSigLinattnBwd, T, H});
    DiagFwdArgs fa{};
    fa.a = nullptr;
    fa.x = dS;
    fa.start = R;
    fa.h = Sinc;
    fa.T = f.nch;
    fa.d = f.dstate;
    fa.Qp = f.scan.Qp;
    fa.nfb = f.scan.nfb;
    fa.nchains = (int32_t)f.scan.nchains;
    set_scan_ws(fa, f.scan, sw, (WsHeader*)sw, sig);
    if (diag_fwd_launch(K_F32, K_F32, true, true, fa, f.scan.ntiles, s) != hipSuccess) return MEMOROID_EHIP;

    // backward summaries (and the reverse scan's workspace set-up)
    char* rw = ws + p.off_rscan;
    LinBwdArgs ba{};
    ba.q = q;
    ba.k = k;
    ba.v = v;
    ba.out = out;
    ba.g = grad_out;
    ba.start = start;
    ba.Sinc = Sinc;
    ba.dnum = (float*)(ws + p.off_dnum);
    ba.dden = (float*)(ws + p.off_dden);
    ba.dU = (float*)(ws + p.off_dU);
    ba.Rs = (uint8_t*)(ws + p.off_Rs);
    ba.Y = (const float*)(ws + p.off_Y);
    ba.dq = grad_q;
    ba.dk = grad_k;
    ba.dv = grad_v;
    ba.T = T;
    ba.H = H;
    ba.nch = f.nch;
    ba.fill = (u32x4*)rw;
    ba.fill16 = (int64_t)(p.rscan.total / 16);
    if (linattn_bwd_summary_launch(ba, s) != hipSuccess) return MEMOROID_EHIP;

    // reverse chunk-state scan: Y_c = dU_c + [chunk c holds no begin] Y_{c+1}
    // (the reverse diagonal scan with a = 1, cut by the shifted chunk flags);
    // a wait that gives up flags the timeout word of the forward header
    DiagBwdArgs ra{};
    ra.a = nullptr;
    ra.start = ba.Rs;
    ra.h = nullptr;
    ra.g = ba.dU;
    ra.dx = (void*)ba.Y;
    ra.da = nullptr;
    ra.da_part = nullptr;
    ra.T = f.nch;
    ra.d = f.dstate;
    ra.Qp = p.rscan.Qp;
    ra.nfb = p.rscan.nfb;
    ra.nchains = (int32_t)p.rscan.nchains;
    set_scan_ws(ra, p.rscan, rw, (WsHeader*)sw, sig);
    if (diag_bwd_launch(K_F32, true, true, ra, p.rscan.ntiles, s) != hipSuccess) return MEMOROID_EHIP;

    return check_hip(linattn_bwd_grad_launch(ba, s));
}

// ------------------------------------------------------------------ status

// ------------------------------------------- discounted return and GAE

namespace {

struct DiscPlan {
    int64_t nt = 0, ntiles = 0;
    size_t off_epoch = 0, off_agg = 0, off_incl = 0, bank_bytes = 0, init_bytes = 0, total = 0;
};

// header, per-tile epoch words, then two banks of tile words
bool plan_disc(int64_t B, int64_t T, bool gae, DiscPlan* p) {
    if (B <= 0 || T <= 0 || T > INT64_MAX / 4) return false;
    p->nt = (T + disc_tile(gae) - 1) / disc_tile(gae);
    if (!mul_ok(B, p->nt, &p->ntiles) || p->ntiles >= (int64_t)INT32_MAX) return false;
    size_t off = kAlign;
    p->off_epoch = off;
    off = align_up(off + (size_t)p->ntiles * 4);
    const size_t bank0 = off;
    p->off_agg = off;
    off = align_up(off + (size_t)p->ntiles * 8);
    p->off_incl = off;
    off = align_up(off + (size_t)p->ntiles * 8);
    p->bank_bytes = off - bank0;
    p->init_bytes = off;
    p->total = off + p->bank_bytes;
    return true;
}

bool unit_interval(float v) { return v >= 0.0f && v <= 1.0f; }   // false for NaN

// Polls of an awaited tile without progress before a look-back computes
// that tile's aggregate from its inputs (memoroid_testing_set_fallback_polls
// lowers it in tests, to run the fallback on every wait).
constexpr uint32_t kDefaultFallbackPolls = 4096u;
std::atomic<uint32_t> g_fallback_polls{kDefaultFallbackPolls};
uint32_t fallback_polls() { return g_fallback_polls.load(std::memory_order_relaxed); }

int disc_run(const float* r, const float* value, const float* value_next, const uint8_t* done,
             const uint8_t* start, float a, float gamma, float* out, float* target, int64_t B, int64_t T,
             void* workspace, size_t workspace_bytes, void* stream, bool gae, WsMode mode) {
    int64_t BT;
    if (!mul_ok(B, T, &BT) || BT > INT64_MAX / 16) return MEMOROID_EINVAL;
    const float* fin[3] = {r, value, value_next};
    const float* fout[2] = {out, target};
    for (const float* q : fin)
        if (q && !aligned(q, 4)) return MEMOROID_EINVAL;
    for (const float* q : fout) {
        if (q && !aligned(q, 4)) return MEMOROID_EINVAL;
        if (q && (q == r || q == value || q == value_next || (const void*)q == (const void*)start ||
                  (const void*)q == (const void*)done))
            return MEMOROID_EINVAL;
    }
    if (target && target == out) return MEMOROID_EINVAL;
    const bool vec = T % 4 == 0 && aligned(r, 16) && aligned(out, 16) && aligned(start, 4) &&
                     (!value || aligned(value, 16)) && (!value_next || aligned(value_next, 16)) &&
                     (!done || aligned(done, 4)) && (!target || aligned(target, 16));
    DiscPlan p;
    if (!plan_disc(B, T, gae, &p)) return MEMOROID_EUNSUPPORTED;
    if (!workspace || workspace_bytes < p.total) return MEMOROID_EWORKSPACE;
    if (!aligned(workspace, 16)) return MEMOROID_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    char* ws = (char*)workspace;
    DiscArgs args{};
    args.r = r;
    args.v = value;
    args.vn = value_next;
    args.done = done;
    args.start = start;
    args.out = out;
    args.target = target;
    args.a = a;
    args.gamma = gamma;
    args.T = T;
    args.nt = p.nt;
    args.B = B;
    args.fallback_polls = fallback_polls();
    args.agg = (uint64_t*)(ws + p.off_agg);
    args.incl = (uint64_t*)(ws + p.off_incl);
    args.bank = (int64_t)p.bank_bytes;
    args.hdr = (WsHeader*)ws;
    // the return and the advantage tile differently: each binds its own workspace
    args.sig = layout_sig({kSigDiscount, B, T, gae});
    args.epoch = (uint32_t*)(ws + p.off_epoch);
    const int st = init_if_self(mode, ws, p.init_bytes, s);
    if (st != MEMOROID_OK) return st;
    return check_hip(disc_launch(vec, gae, args, p.ntiles, s));
}

}  // namespace

size_t memoroid_discount_workspace_bytes(int64_t B, int64_t T) {
    if (B <= 0 || T <= 0) return 0;
    DiscPlan pr, pg;
    if (!plan_disc(B, T, false, &pr) || !plan_disc(B, T, true, &pg)) return 0;
    return pr.total > pg.total ? pr.total : pg.total;
}

static int return_run(const float* r, const uint8_t* start, float gamma, float* G, int64_t B, int64_t T,
                      void* workspace, size_t workspace_bytes, void* stream, WsMode mode) {
    if (B < 0 || T < 0 || !unit_interval(gamma)) return MEMOROID_EINVAL;
    if (B == 0 || T == 0) return MEMOROID_OK;
    if (!r || !start || !G) return MEMOROID_EINVAL;
    return disc_run(r, nullptr, nullptr, nullptr, start, gamma, gamma, G, nullptr, B, T, workspace,
                    workspace_bytes, stream, false, mode);
}

int memoroid_discounted_return(const float* r, const uint8_t* start, float gamma, float* G, int64_t B, int64_t T,
                               void* workspace, size_t workspace_bytes, void* stream) {
    return return_run(r, start, gamma, G, B, T, workspace, workspace_bytes, stream, WsMode::kSelfInit);
}

int memoroid_discounted_return_prepared(const float* r, const uint8_t* start, float gamma, float* G, int64_t B,
                                        int64_t T, void* workspace, size_t workspace_bytes, void* stream) {
    return return_run(r, start, gamma, G, B, T, workspace, workspace_bytes, stream, WsMode::kPrepared);
}

static int gae_run(const float* r, const float* value, const float* value_next, const uint8_t* done,
                   const uint8_t* start, float gamma, float lambda, float* adv, float* target, int64_t B, int64_t T,
                   void* workspace, size_t workspace_bytes, void* stream, WsMode mode) {
    if (B < 0 || T < 0 || !unit_interval(gamma) || !unit_interval(lambda)) return MEMOROID_EINVAL;
    if (B == 0 || T == 0) return MEMOROID_OK;
    if (!r || !value || !start || !adv) return MEMOROID_EINVAL;
    return disc_run(r, value, value_next, done, start, gamma * lambda, gamma, adv, target, B, T, workspace,
                    workspace_bytes, stream, true, mode);
}

int memoroid_gae(const float* r, const float* value, const float* value_next, const uint8_t* done,
                 const uint8_t* start, float gamma, float lambda, float* adv, float* target, int64_t B, int64_t T,
                 void* workspace, size_t workspace_bytes, void* stream) {
    return gae_run(r, value, value_next, done, start, gamma, lambda, adv, target, B, T, workspace, workspace_bytes,
                   stream, WsMode::kSelfInit);
}

int memoroid_gae_prepared(const float* r, const float* value, const float* value_next, const uint8_t* done,
                          const uint8_t* start, float gamma, float lambda, float* adv, float* target, int64_t B,
                          int64_t T, void* workspace, size_t workspace_bytes, void* stream) {
    return gae_run(r, value, value_next, done, start, gamma, lambda, adv, target, B, T, workspace, workspace_bytes,
                   stream, WsMode::kPrepared);
}

// ------------------------------------------------- tape-based batching

namespace {

// header, per-tile epoch words, then two banks of count words
struct TbbPlan {
    int64_t ntiles = 0;
    size_t off_epoch = 0, off_cnt = 0, bank_bytes = 0, init_bytes = 0, total = 0;
};

void plan_tbb(int64_t n, TbbPlan* p) {
    p->ntiles = (n + kTbbBeginTile - 1) / kTbbBeginTile;
    p->off_epoch = kAlign;
    p->off_cnt = align_up(p->off_epoch + (size_t)p->ntiles * 4);
    p->bank_bytes = align_up((size_t)p->ntiles * 8);
    p->init_bytes = p->off_cnt + p->bank_bytes;
    p->total = p->off_cnt + 2 * p->bank_bytes;
}

// Sampling workspace: header, epoch words, two banks of row-sum words, the
// rows filled and draws inside the batch, the lead tiles' verdict words, the
// group table, and each draw's first batch row and source shift.
struct SamplePlan {
    int64_t ntiles = 0, groups = 0;
    size_t off_epoch = 0, off_cnt = 0, bank_bytes = 0, off_meta = 0, off_dec = 0, off_first = 0, off_row0 = 0,
           off_shift = 0, init_bytes = 0, total = 0;
};

constexpr int64_t kSampleMaxRows = (int64_t)1 << 47;   // batch and n_D bound: row sums stay below 2^48

void plan_sample(int64_t n_draws, int64_t batch, SamplePlan* p) {
    p->ntiles = (n_draws + kTbbDrawTile - 1) / kTbbDrawTile;
    p->groups = (batch + kTbbRowsPerGroup - 1) / kTbbRowsPerGroup;
    p->off_epoch = kAlign;
    p->off_cnt = align_up(p->off_epoch + (size_t)p->ntiles * 4);
    p->bank_bytes = align_up((size_t)p->ntiles * 8);
    p->off_meta = p->off_cnt + 2 * p->bank_bytes;
    p->off_dec = align_up(p->off_meta + 16);
    p->off_first = align_up(p->off_dec + 64 * 128);    // 64 verdict words, one per 128-byte line
    // the verdict words carry the call's epoch: a self-initialising call
    // (always epoch 0) clears them too
    p->init_bytes = p->off_first;
    p->off_row0 = align_up(p->off_first + (size_t)p->groups * 8);
    p->off_shift = align_up(p->off_row0 + (size_t)n_draws * 8);
    p->total = align_up(p->off_shift + (size_t)n_draws * 8);
}

}  // namespace

size_t memoroid_tbb_begin_indices_workspace_bytes(int64_t n) {
    if (n <= 0 || n > (int64_t)INT32_MAX) return 0;
    TbbPlan p;
    plan_tbb(n, &p);
    return p.total;
}

static int tbb_begins_run(const uint8_t* start, int64_t n, int64_t offset, int64_t* indices, int64_t* count,
                          void* workspace, size_t workspace_bytes, void* stream, WsMode mode) {
    if (n < 0) return MEMOROID_EINVAL;
    if (n > (int64_t)INT32_MAX) return MEMOROID_EUNSUPPORTED;
    if (!count) return MEMOROID_EINVAL;
    if (!aligned(count, 8) || (indices && !aligned(indices, 8))) return MEMOROID_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    if (n == 0) {
        // nothing to scan, but the count is still an output
        return check_hip(store_i64_launch(count, 0, s));
    }
    if (!start || !indices) return MEMOROID_EINVAL;
    if ((const void*)indices == (const void*)start || (const void*)count == (const void*)start ||
        (const void*)count == (const void*)indices)
        return MEMOROID_EINVAL;
    if (offset > INT64_MAX - n || offset < INT64_MIN + 1) return MEMOROID_EINVAL;
    const size_t need = memoroid_tbb_begin_indices_workspace_bytes(n);
    if (!workspace || workspace_bytes < need) return MEMOROID_EWORKSPACE;
    if (!aligned(workspace, 16)) return MEMOROID_EINVAL;
    char* ws = (char*)workspace;
    TbbPlan p;
    plan_tbb(n, &p);
    TbbBeginArgs a{};
    a.start = start;
    a.n = n;
    a.offset = offset;
    a.indices = indices;
    a.count = count;
    a.cnt = (uint64_t*)(ws + p.off_cnt);
    a.bank = (int64_t)p.bank_bytes;
    a.hdr = (WsHeader*)ws;
    a.sig = layout_sig({kSigTbbBegins, n});
    a.epoch = (uint32_t*)(ws + p.off_epoch);
    a.fallback_polls = fallback_polls();
    const bool vec = aligned(start, 16) && n % 16 == 0;
    const int st = init_if_self(mode, ws, p.init_bytes, s);
    if (st != MEMOROID_OK) return st;
    return check_hip(tbb_begins_launch(vec, a, p.ntiles, s));
}

int memoroid_tbb_begin_indices(const uint8_t* start, int64_t n, int64_t offset, int64_t* indices, int64_t* count,
                               void* workspace, size_t workspace_bytes, void* stream) {
    return tbb_begins_run(start, n, offset, indices, count, workspace, workspace_bytes, stream, WsMode::kSelfInit);
}

int memoroid_tbb_begin_indices_prepared(const uint8_t* start, int64_t n, int64_t offset, int64_t* indices,
                                        int64_t* count, void* workspace, size_t workspace_bytes, void* stream) {
    return tbb_begins_run(start, n, offset, indices, count, workspace, workspace_bytes, stream, WsMode::kPrepared);
}

size_t memoroid_tbb_sample_workspace_bytes(int64_t n_draws, int64_t batch) {
    if (n_draws < 0 || n_draws > ((int64_t)1 << 24) || batch < 0 || batch >= kSampleMaxRows) return 0;
    SamplePlan p;
    plan_sample(n_draws, batch, &p);
    return p.total;
}

static int tbb_sample_run(const void* D, int64_t n_D, int64_t row_bytes, const int64_t* I, int64_t n_I,
                          const int64_t* draws, int64_t n_draws, int64_t batch, void* out, uint8_t* out_start,
                          int64_t* out_src, int64_t* filled, void* workspace, size_t workspace_bytes, void* stream,
                          WsMode mode) {
    if (n_D < 0 || row_bytes <= 0 || n_I < 0 || n_draws < 0 || batch < 0) return MEMOROID_EINVAL;
    if (n_draws > ((int64_t)1 << 24) || row_bytes > ((int64_t)1 << 24)) return MEMOROID_EUNSUPPORTED;
    int64_t tmp;
    if (!mul_ok(batch, row_bytes, &tmp) || !mul_ok(n_D, row_bytes, &tmp)) return MEMOROID_EINVAL;
    if (batch >= kSampleMaxRows || n_D >= kSampleMaxRows) return MEMOROID_EUNSUPPORTED;
    if (n_draws > 0 && (!I || !draws || n_I == 0)) return MEMOROID_EINVAL;
    if (n_draws > 0 && n_D > 0 && !D) return MEMOROID_EINVAL;
    if (batch > 0 && (!out || !out_start)) return MEMOROID_EINVAL;
    if ((I && !aligned(I, 8)) || (draws && !aligned(draws, 8)) || (out_src && !aligned(out_src, 8)) ||
        (filled && !aligned(filled, 8)))
        return MEMOROID_EINVAL;
    if (batch > 0 && (out == D || (const void*)out == (const void*)I || (const void*)out == (const void*)draws ||
                      (const void*)out_start == (const void*)out || (const void*)out_src == (const void*)out))
        return MEMOROID_EINVAL;
    hipStream_t s = (hipStream_t)stream;
    if (batch == 0) return filled ? check_hip(store_i64_launch(filled, 0, s)) : MEMOROID_OK;
    SamplePlan p;
    plan_sample(n_draws, batch, &p);
    if (n_draws > 0 && (!workspace || workspace_bytes < p.total)) return MEMOROID_EWORKSPACE;
    if (workspace && !aligned(workspace, 16)) return MEMOROID_EINVAL;
    TbbSampleArgs a{};
    a.D = D;
    a.n_D = n_D;
    a.row_bytes = row_bytes;
    a.I = I;
    a.n_I = n_I;
    a.draws = draws;
    a.n_draws = n_draws;
    a.batch = batch;
    a.out = out;
    a.out_start = out_start;
    a.out_src = out_src;
    a.filled = filled;
    if (n_draws > 0) {
        char* ws = (char*)workspace;
        a.hdr = (WsHeader*)ws;
        a.sig = layout_sig({kSigTbbSample, n_draws, batch});
        a.epoch = (uint32_t*)(ws + p.off_epoch);
        a.cnt = (uint64_t*)(ws + p.off_cnt);
        a.bank = (int64_t)p.bank_bytes;
        a.meta = (int64_t*)(ws + p.off_meta);
        a.dec = (uint64_t*)(ws + p.off_dec);
        a.first = (int64_t*)(ws + p.off_first);
        a.row0 = (int64_t*)(ws + p.off_row0);
        a.shift = (int64_t*)(ws + p.off_shift);
        a.fallback_polls = fallback_polls();
    }
    const int unit = (row_bytes % 16 == 0 && aligned(out, 16) && (!D || aligned(D, 16))) ? 16
                     : (row_bytes % 4 == 0 && aligned(out, 4) && (!D || aligned(D, 4))) ? 4 : 1;
    // Draws are taken in order until the batch is full: about batch / (mean
    // episode length) = batch * n_I / n_D of them.  The row-sum tiles that
    // twice that many draws need run at once; the later ones wait for them
    // and skip their loads if the batch is already full.
    a.lead = p.ntiles;
    if (n_draws > 0 && n_D > 0) {
        const double need = 2.0 * (double)batch * (double)n_I / (double)n_D;
        const double tiles = need / (double)kTbbDrawTile + 1.0;
        a.lead = tiles < (double)p.ntiles ? (int64_t)tiles : p.ntiles;
        if (a.lead < 1) a.lead = 1;
    }
    if (n_draws > 0) {
        const int st = init_if_self(mode, workspace, p.init_bytes, s);
        if (st != MEMOROID_OK) return st;
    }
    return check_hip(tbb_sample_launch(unit, a, p.ntiles, s));
}

int memoroid_tbb_sample(const void* D, int64_t n_D, int64_t row_bytes, const int64_t* I, int64_t n_I,
                        const int64_t* draws, int64_t n_draws, int64_t batch, void* out, uint8_t* out_start,
                        int64_t* out_src, int64_t* filled, void* workspace, size_t workspace_bytes, void* stream) {
    return tbb_sample_run(D, n_D, row_bytes, I, n_I, draws, n_draws, batch, out, out_start, out_src, filled,
                          workspace, workspace_bytes, stream, WsMode::kSelfInit);
}

int memoroid_tbb_sample_prepared(const void* D, int64_t n_D, int64_t row_bytes, const int64_t* I, int64_t n_I,
                                 const int64_t* draws, int64_t n_draws, int64_t batch, void* out,
                                 uint8_t* out_start, int64_t* out_src, int64_t* filled, void* workspace,
                                 size_t workspace_bytes, void* stream) {
    return tbb_sample_run(D, n_D, row_bytes, I, n_I, draws, n_draws, batch, out, out_start, out_src, filled,
                          workspace, workspace_bytes, stream, WsMode::kPrepared);
}

int memoroid_workspace_prepare(void* workspace, size_t workspace_bytes, void* stream) {
    if (!workspace || workspace_bytes < sizeof(WsHeader) || !aligned(workspace, 16)) return MEMOROID_EINVAL;
    return check_hip(ws_init_launch(nullptr, 0, workspace, workspace_bytes / 16 * 16, (hipStream_t)stream));
}

size_t memoroid_workspace_bytes(memoroid_op op_in, int64_t B, int64_t T, int64_t d_or_H, int64_t dk, int64_t dv,
                                int64_t chunk) {
    // the operation as a plain int: a C caller may pass any value, which a
    // C++ load of the enum type would not allow
    int op;
    static_assert(sizeof op == sizeof op_in, "memoroid_op is int-sized");
    memcpy(&op, &op_in, sizeof op);
    size_t best = 0;
    auto take = [&best](size_t v) {
        if (v > best) best = v;
    };
    switch (op) {
        case MEMOROID_OP_DIAG: {
            const int pairs[4][2] = {{MEMOROID_F32, MEMOROID_F32},
                                     {MEMOROID_BF16, MEMOROID_BF16},
                                     {MEMOROID_BF16, MEMOROID_F32},
                                     {MEMOROID_C64, MEMOROID_C64}};
            for (const auto& pr : pairs) take(memoroid_scan_diag_workspace_bytes(B, T, d_or_H, pr[0], pr[1]));
            return best;
        }
        case MEMOROID_OP_DIAG_BWD:
            for (int dt : {MEMOROID_F32, MEMOROID_C64})
                for (int64_t stride : {(int64_t)0, d_or_H})
                    take(memoroid_scan_diag_bwd_workspace_bytes(B, T, d_or_H, dt, stride));
            return best;
        case MEMOROID_OP_LINATTN:
            return memoroid_scan_linattn_workspace_bytes(T, d_or_H, dk, dv, chunk);
        case MEMOROID_OP_LINATTN_BWD:
            return memoroid_scan_linattn_bwd_workspace_bytes(T, d_or_H, dk, dv, chunk);
        case MEMOROID_OP_FFM:
            return memoroid_scan_ffm_workspace_bytes(B, T, d_or_H, dk);
        case MEMOROID_OP_FFM_BWD:
            return memoroid_scan_ffm_bwd_workspace_bytes(B, T, d_or_H, dk);
        case MEMOROID_OP_RETURN:
        case MEMOROID_OP_GAE:
            return memoroid_discount_workspace_bytes(B, T);
        case MEMOROID_OP_TBB_BEGIN_INDICES:
            return memoroid_tbb_begin_indices_workspace_bytes(T);
        case MEMOROID_OP_TBB_SAMPLE:
            return memoroid_tbb_sample_workspace_bytes(B, T);
    }
    return 0;
}

int64_t memoroid_testing_set_fallback_polls(int64_t polls) {
    const uint32_t v = polls < 0 ? kDefaultFallbackPolls : (polls > 0xFFFFFFFFll ? 0xFFFFFFFFu : (uint32_t)polls);
    return (int64_t)g_fallback_polls.exchange(v, std::memory_order_relaxed);
}

int64_t memoroid_testing_tile_steps(int reverse, int64_t B, int64_t T, int64_t d, int dtype, int64_t a_stride_t,
                                    int vectorised) {
    if (B <= 0 || T <= 0 || d <= 0 || (a_stride_t != 0 && a_stride_t != d)) return 0;
    if (dtype != MEMOROID_F32 && dtype != MEMOROID_BF16 && dtype != MEMOROID_C64) return 0;
    if (reverse && dtype == MEMOROID_BF16) return 0;
    const bool ainv = a_stride_t == 0;
    DiagPlan p;
    const int rows = reverse ? diag_bwd_rows(dtype, vectorised != 0, ainv) : diag_fwd_rows(dtype, vectorised != 0, ainv);
    if (!plan_diag(B, T, d, dtype, vectorised != 0, rows, reverse != 0, ainv, reverse != 0, &p))
        return 0;
    return p.L;
}

int memoroid_workspace_status(const void* workspace, size_t workspace_bytes, void* stream) {
    if (!workspace || workspace_bytes < sizeof(WsHeader)) return MEMOROID_EINVAL;
    WsHeader hdr;
    hipStream_t s = (hipStream_t)stream;
    if (hipMemcpyAsync(&hdr, workspace, 16, hipMemcpyDeviceToHost, s) != hipSuccess) return MEMOROID_EHIP;
    if (hipStreamSynchronize(s) != hipSuccess) return MEMOROID_EHIP;
    if (hdr.sig == kSigPoisoned) return MEMOROID_EMISMATCH;
    return hdr.timeout != kEmpty32 ? MEMOROID_ETIMEOUT : MEMOROID_OK;
}

}  // extern "C"
