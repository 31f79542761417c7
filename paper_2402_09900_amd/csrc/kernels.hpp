// kernels.hpp -- internal interface between the C ABI (abi.hip) and the
// kernel translation units.  Not installed; not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace memoroid {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct WsHeader;

// Steps per lane held in registers by the diagonal scans (a tile is
// 256 / Qp * rows steps long: 64 for full-width feature blocks).  The reverse
// scan with a per-step a keeps three tensors per step (g, a, h) and so holds
// fewer steps, to stay within 256 registers (two workgroups per CU); with a
// time-invariant a it runs 8 (shorter tiles, more of them in flight: the
// linear-attention state scan, one tile per chain at 16, took 21.2 µs
// against 18.5 at 8).
#ifndef MEMOROID_FWD_ROWS
#define MEMOROID_FWD_ROWS 16
#endif
#ifndef MEMOROID_BWD_ROWS
#define MEMOROID_BWD_ROWS 8
#endif
#ifndef MEMOROID_BWD_ROWS_PER_STEP_A
#define MEMOROID_BWD_ROWS_PER_STEP_A 12
#endif
#ifndef MEMOROID_CHAIN_ROW_BYTES
#define MEMOROID_CHAIN_ROW_BYTES 128
#endif
#ifndef MEMOROID_FWD_ROWS_BF16
#define MEMOROID_FWD_ROWS_BF16 12
#endif
#ifndef MEMOROID_FWD_ROWS_F32_STEP_A
#define MEMOROID_FWD_ROWS_F32_STEP_A 18
#endif
constexpr int kFwdRows = MEMOROID_FWD_ROWS;
// bf16 input, vectorised: 8 features per lane (one 16-byte access), so a
// lane's steps hold half the bytes they would in f32 for the same registers
constexpr int kFwdRowsBf16 = MEMOROID_FWD_ROWS_BF16;
// f32 with a per-step a, vectorised: 18 steps still fit two workgroups per CU
// and the longer tiles spread the per-tile fixed cost further
constexpr int kFwdRowsF32StepA = MEMOROID_FWD_ROWS_F32_STEP_A;
constexpr int kBwdRows = MEMOROID_BWD_ROWS;
constexpr int kBwdRowsPerStepA = MEMOROID_BWD_ROWS_PER_STEP_A;
// Bytes of a feature row one chain covers (one 128-byte line by default).
constexpr int64_t kChainRowBytes = MEMOROID_CHAIN_ROW_BYTES;
// Accelerator dies (XCDs, each with its own L2) of an MI355X: the dispatcher
// hands workgroup g to XCD g mod kXcds.
constexpr uint32_t kXcds = 8;
constexpr int diag_rows(bool bwd, bool ainv) { return !bwd ? kFwdRows : (ainv ? kBwdRows : kBwdRowsPerStepA); }
// The reverse scan of complex state with a time-invariant a, vectorised,
// runs shorter tiles: at 8 steps it keeps three workgroups per CU.
#ifndef MEMOROID_BWD_ROWS_C64_INV
#define MEMOROID_BWD_ROWS_C64_INV 8
#endif
constexpr int kBwdRowsC64Inv = MEMOROID_BWD_ROWS_C64_INV;
// steps per lane of the reverse scan of a state dtype (f32 is 0, c64 2)
constexpr int diag_bwd_rows(int state_dtype, bool vec, bool ainv) {
    return state_dtype == 2 && vec && ainv ? kBwdRowsC64Inv : diag_rows(true, ainv);
}
// steps per lane of the forward scan of a state dtype (a memoroid_dtype:
// f32 is 0, bf16 1), vectorised or not, with a time-invariant a or not
constexpr int diag_fwd_rows(int state_dtype, bool vec, bool ainv) {
    return !vec ? kFwdRows : state_dtype == 1 ? kFwdRowsBf16 : (state_dtype == 0 && !ainv) ? kFwdRowsF32StepA : kFwdRows;
}
// The FFM gradient keeps more per-tile state (the input-gradient reduction)
// and runs fastest with shorter tiles and more workgroups per CU.
#ifndef MEMOROID_FFM_BWD_ROWS
#define MEMOROID_FFM_BWD_ROWS 8
#endif
constexpr int kFfmBwdRows = MEMOROID_FFM_BWD_ROWS;
// The FFM forward holds only the real input per step (its outputs stream
// out), so its register count and tile length are set on their own.
#ifndef MEMOROID_FFM_FWD_ROWS
#define MEMOROID_FFM_FWD_ROWS 24
#endif
constexpr int kFfmFwdRows = MEMOROID_FFM_FWD_ROWS;


struct DiagFwdArgs {
    const void* a;
    const void* x;
    const uint8_t* start;
    void* h;
    int64_t T;
    int64_t d;
    int32_t Qp;        // lanes per step row of a tile (power of two, <= 64)
    int32_t nfb;       // feature blocks per tape
    int32_t nchains;   // tapes * feature blocks
    int32_t pad0;
    int64_t nt;        // tiles per chain
    // descriptor words, bank 0 (bank 1 lies `bank` bytes further on)
    void* agg;         // [tiles][Dp] aggregate descriptor words
    void* incl;        // [tiles][Dp] inclusive-prefix descriptor words
    uint64_t* cnt;     // [tiles per chain][B] begin-count descriptor words, or NULL
    int64_t bank;
    WsHeader* hdr;
    uint64_t sig;      // signature of the call (workspace binding)
    uint32_t* ctr;     // per-chain tile counters, kCtrStride words apart
    int32_t* idx;      // episode index out [B][T], or NULL
    // FFM aggregator (complex state, d = m * c): a[j*c + k] =
    // exp(-|alpha_j| + i omega_k) is generated in the kernel and x is real
    // [B][T][m], broadcast over the c columns
    const float* alpha;
    const float* omega;
    int64_t ffm_m, ffm_c;
};

struct DiagBwdArgs {
    const void* a;
    const uint8_t* start;
    const void* h;
    const void* g;
    void* dx;
    void* da;          // per-step da, or NULL
    void* da_part;     // time-invariant a: [tiles per chain * B][d] partial sums
    void* da_out;      // time-invariant a with one tape: da [d], summed in the kernel from
                       // partial words [tiles per chain][d] (64-bit, self-validating, banked
                       // like the descriptors) in da_part
    int64_t T;
    int64_t d;
    int64_t nt;        // tiles per chain
    int32_t Qp;
    int32_t nfb;
    int32_t nchains;
    int32_t pad0;
    void* agg;         // bank 0, as in DiagFwdArgs
    void* incl;
    int64_t bank;
    WsHeader* hdr;
    uint64_t sig;
    uint32_t* ctr;     // per-chain tile counters, kCtrStride words apart
    // FFM aggregator gradient: a generated from alpha, omega (as in the
    // forward pass); dx is reduced over the c columns of each row j into the
    // real dxr[B][T][m] instead of being stored per feature
    const float* alpha;
    const float* omega;
    int64_t ffm_m, ffm_c;
    float* dxr;        // chain-major input gradient [chains][T][Dp / c] (workspace)
};

// Last step of the FFM gradient: dx[B][T][m] from the chain-major dxw, and
// dalpha / domega from the summed da[m][c] (complex), when not NULL.
struct FfmFinishArgs {
    const float* dxw;  // [B][nfb][T][jpc], nfb = ceil(m / jpc)
    float* dx;
    int64_t B, T, m, c, jpc;
    const float* alpha;
    const float* omega;
    const float* da;
    float* dalpha;
    float* domega;
};

hipError_t diag_fwd_launch(int in_kind, int out_kind, bool vec, bool ainv,
                           const DiagFwdArgs& args, int64_t ntiles, hipStream_t s);
hipError_t ffm_fwd_launch(bool vec, const DiagFwdArgs& args, int64_t ntiles, hipStream_t s);
hipError_t ffm_bwd_launch(bool vec, const DiagBwdArgs& args, int64_t ntiles, hipStream_t s);
// dx from the chain-major workspace; dalpha[j] = -sign(alpha_j) sum_k
// Re(conj(a_jk) da_jk), domega[k] = sum_j Im(conj(a_jk) da_jk)
hipError_t ffm_bwd_finish_launch(const FfmFinishArgs& a, hipStream_t s);
hipError_t diag_bwd_launch(int kind, bool vec, bool ainv, const DiagBwdArgs& args,
                           int64_t ntiles, hipStream_t s);
// out[r / (4 rpw)][c] = sum over rows r .. r + 4 rpw - 1 of in[r][c], in a
// fixed order (rpw: rows per wavefront).
hipError_t colsum_launch(const float* in, float* out, int64_t rows, int64_t cols, int64_t rpw, hipStream_t s);

// Per-chain tile counters sit 128 bytes apart: atomics on one cache line
// serialise (about 11 ns each on MI355X), atomics on distinct lines do not.
constexpr int kCtrStride = 32;

// Zero `zero_bytes` from `zero` and fill `ones_bytes` from `ones` with
// all-ones bytes; both sizes multiples of 16.  A kernel, not
// hipMemsetAsync, so that a caller may capture the call in a HIP graph.
hipError_t ws_init_launch(void* zero, size_t zero_bytes, void* ones, size_t ones_bytes, hipStream_t s);
hipError_t store_i64_launch(int64_t* p, int64_t v, hipStream_t s);

// Linear-attention memoroid: per-(chunk, head) state summaries, and outputs
// from the scanned chunk states.  A state is S^T (64x64, row n holds column n
// of S) followed by z (64), kLinStateWords floats.
constexpr int kLinChunk = 64;
constexpr int kLinStateWords = 64 * 64 + 64;

struct LinSummaryArgs {
    const float* k;
    const float* v;
    const uint8_t* start;
    float* dS;          // [chunks][H][kLinStateWords]
    uint8_t* R;         // [chunks] chunk holds a begin step
    int64_t T;
    int64_t H;
    u32x4* fill;        // state-scan workspace to prepare (all-ones bytes, 16-byte units)
    int64_t fill16;
};

struct LinOutputArgs {
    const float* q;
    const float* k;
    const float* v;
    const uint8_t* start;
    const float* Sinc;  // scanned states, [chunks][H][kLinStateWords]
    float* out;
    int64_t T;
    int64_t H;
    int32_t* idx;       // episode index out [T], or NULL
    uint64_t* cnt;      // [chunks] begin-count words (filled by the summary kernel)
    uint32_t* timeout;
};

hipError_t linattn_summary_launch(const LinSummaryArgs& a, hipStream_t s);
hipError_t linattn_output_launch(const LinOutputArgs& a, hipStream_t s);

struct LinBwdArgs {
    const float* q;
    const float* k;
    const float* v;
    const float* out;   // forward readout [T][H][64]
    const float* g;     // dL/dout [T][H][64]
    const uint8_t* start;
    const float* Sinc;  // forward chunk states after each chunk [chunks][H][kLinStateWords]
    float* dnum;        // workspace [T][H][64]
    float* dden;        // workspace [T][H]
    float* dU;          // reverse chunk summaries [chunks][H][kLinStateWords] (U [kd][n], then w)
    uint8_t* Rs;        // [chunks] reverse-scan flags: Rs[c] = chunk c - 1 holds a begin
    const float* Y;     // reverse-scanned states [chunks][H][kLinStateWords]
    float* dq;
    float* dk;
    float* dv;
    int64_t T, H, nch;
    u32x4* fill;        // reverse-scan workspace to prepare (all-ones bytes)
    int64_t fill16;
};

hipError_t linattn_bwd_summary_launch(const LinBwdArgs& a, hipStream_t s);
hipError_t linattn_bwd_grad_launch(const LinBwdArgs& a, hipStream_t s);

// ------------------------------------------- discounted return and GAE
// Steps per lane: 32 for the return (two streams in registers), 16 for the
// advantage (four); a tile is 4 wavefronts of 64 lanes.
#ifndef MEMOROID_RETURN_ROWS
#define MEMOROID_RETURN_ROWS 32
#endif
#ifndef MEMOROID_GAE_ROWS
#define MEMOROID_GAE_ROWS 16
#endif
constexpr int disc_rows(bool gae) { return gae ? MEMOROID_GAE_ROWS : MEMOROID_RETURN_ROWS; }
constexpr int disc_tile(bool gae) { return 4 * 64 * disc_rows(gae); }

struct DiscArgs {
    const float* r;          // [B][T] rewards
    const float* v;          // [B][T] V(s_t) (advantage only)
    const float* vn;         // [B][T] V(s'_t) or NULL (advantage only)
    const uint8_t* done;     // [B][T] terminal flags or NULL (advantage only)
    const uint8_t* start;    // [B][T] begin flags
    float* out;              // [B][T] return or advantage
    float* target;           // [B][T] advantage + V(s_t), or NULL
    float a;                 // recurrence coefficient: gamma, or gamma * lambda
    float gamma;             // discount of the TD error (advantage only)
    int64_t T, nt, B;        // tape length, tiles per tape, tapes
    uint32_t fallback_polls; // polls without progress before a look-back computes the awaited tile itself
    uint64_t* agg;           // [B][nt] tile aggregates (bank 0)
    uint64_t* incl;          // [B][nt] tile values at their first step (bank 0)
    int64_t bank;            // bytes from bank 0 to bank 1
    WsHeader* hdr;
    uint64_t sig;
    uint32_t* epoch;         // [B][nt] per-tile epoch words
};

hipError_t disc_launch(bool vec, bool gae, const DiscArgs& a, int64_t ntiles, hipStream_t s);

// ------------------------------------------------ tape-based batching
#ifndef MEMOROID_TBB_BEGIN_BLOCKS
#define MEMOROID_TBB_BEGIN_BLOCKS 2
#endif
constexpr int kTbbBeginBlocks = MEMOROID_TBB_BEGIN_BLOCKS;    // blocks of 16384 flags per compaction workgroup
constexpr int kTbbBeginTile = 16384 * kTbbBeginBlocks;        // flags per workgroup of the compaction
#ifndef MEMOROID_TBB_DRAW_TILE
#define MEMOROID_TBB_DRAW_TILE 512
#endif
#ifndef MEMOROID_TBB_ROWS_PER_GROUP
#define MEMOROID_TBB_ROWS_PER_GROUP 256
#endif
constexpr int kTbbDrawTile = MEMOROID_TBB_DRAW_TILE;          // draws per workgroup of the row sums
constexpr int kTbbRowsPerGroup = MEMOROID_TBB_ROWS_PER_GROUP; // output rows per workgroup of the gather
// each of the gather's 256 threads owns RW / 256 rows and window draws
static_assert(kTbbRowsPerGroup >= 256 && kTbbRowsPerGroup % 256 == 0, "gather group: a multiple of 256 rows");
static_assert(kTbbDrawTile >= 256 && kTbbDrawTile % 256 == 0, "row-sum tile: a multiple of 256 draws");

struct TbbBeginArgs {
    const uint8_t* start;    // [n] begin flags
    int64_t n;
    int64_t offset;          // added to every index
    int64_t* indices;        // out, room for n
    int64_t* count;          // out, one value (may be NULL)
    uint64_t* cnt;           // [tiles] count descriptor words (bank 0)
    int64_t bank;            // bytes from bank 0 to bank 1
    WsHeader* hdr;
    uint64_t sig;
    uint32_t* epoch;         // [tiles] per-tile epoch words
    uint32_t fallback_polls;
};

hipError_t tbb_begins_launch(bool vec, const TbbBeginArgs& a, int64_t ntiles, hipStream_t s);

struct TbbSampleArgs {
    const void* D;           // [n_D][row_bytes]
    int64_t n_D, row_bytes;
    const int64_t* I;        // [n_I] begin indices
    int64_t n_I;
    const int64_t* draws;    // [n_draws] positions in I
    int64_t n_draws;
    int64_t batch;
    void* out;               // [batch][row_bytes]
    uint8_t* out_start;      // [batch]
    int64_t* out_src;        // [batch] or NULL
    int64_t* filled;         // one value or NULL
    // workspace
    WsHeader* hdr;
    uint64_t sig;
    uint32_t* epoch;         // [tiles] per-tile epoch words
    uint64_t* cnt;           // [tiles] row-sum descriptor words (bank 0)
    int64_t bank;            // bytes from bank 0 to bank 1
    int64_t* meta;           // [2]: rows filled; draws whose first row is inside the batch
    int64_t lead;            // row-sum tiles that run without first waiting for the earlier ones
    uint64_t* dec;           // [64 words, 128 bytes apart]: (epoch << 32) | 1 batch full within the lead tiles, | 2 not
    int64_t* first;          // [groups]: the draw holding each gather group's first row
    int64_t* row0;           // [n_draws]: first batch row of each draw (draws inside the batch)
    int64_t* shift;          // [n_draws]: source row minus batch row (same draws)
    uint32_t fallback_polls;
};

hipError_t tbb_sample_launch(int unit, const TbbSampleArgs& a, int64_t ntiles, hipStream_t s);

}  // namespace memoroid
