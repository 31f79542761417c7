// scan_common.hpp -- device helpers shared by the scan kernels (gfx950).
//
//  * element kinds (f32, bf16, complex64) with exact decode / RNE encode;
//  * register-resident raw vectors loaded and stored with one wide access;
//  * the state algebra of the diagonal memoroid under the reset transform;
//  * self-validating cross-tile descriptor words for the single-pass scan.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kernels.hpp"

namespace memoroid {

typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

enum Kind { K_F32 = 0, K_BF16 = 1, K_C64 = 2 };

template <Kind K> struct KindInfo;
template <> struct KindInfo<K_F32> { static constexpr int bytes = 4; static constexpr int vec = 4; };
template <> struct KindInfo<K_BF16> { static constexpr int bytes = 2; static constexpr int vec = 8; };
template <> struct KindInfo<K_C64> { static constexpr int bytes = 8; static constexpr int vec = 2; };

// ------------------------------------------------------------ complex float

struct cf {
    float re, im;
};

__device__ __forceinline__ cf operator*(cf a, cf b) {
    return cf{a.re * b.re - a.im * b.im, a.re * b.im + a.im * b.re};
}
__device__ __forceinline__ cf operator+(cf a, cf b) { return cf{a.re + b.re, a.im + b.im}; }
__device__ __forceinline__ cf conj(cf a) { return cf{a.re, -a.im}; }
__device__ __forceinline__ float conj(float a) { return a; }
__device__ __forceinline__ float re_part(cf a) { return a.re; }
__device__ __forceinline__ float re_part(float a) { return a; }

// a * b + c, fused per component where the arithmetic allows
__device__ __forceinline__ float mad(float a, float b, float c) { return __builtin_fmaf(a, b, c); }
__device__ __forceinline__ cf mad(cf a, cf b, cf c) {
    return cf{__builtin_fmaf(a.re, b.re, __builtin_fmaf(-a.im, b.im, c.re)),
              __builtin_fmaf(a.re, b.im, __builtin_fmaf(a.im, b.re, c.im))};
}

template <class S> __device__ __forceinline__ S s_one();
template <> __device__ __forceinline__ float s_one<float>() { return 1.0f; }
template <> __device__ __forceinline__ cf s_one<cf>() { return cf{1.0f, 0.0f}; }
template <class S> __device__ __forceinline__ S s_zero();
template <> __device__ __forceinline__ float s_zero<float>() { return 0.0f; }
template <> __device__ __forceinline__ cf s_zero<cf>() { return cf{0.0f, 0.0f}; }

template <Kind K> struct StateOf { using type = float; };
template <> struct StateOf<K_C64> { using type = cf; };

// ---------------------------------------------------------------- bf16 codec

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// float -> bf16 bits, round to nearest even (NaN stays NaN), by the
// hardware conversion; f32x2_to_bf16x2 converts two values with one
// instruction and packs them, the first in the low half.
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t f32x2_to_bf16x2(float lo, float hi) {
    const f32x2_t f = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f, bf16x2_t));
}
__device__ __forceinline__ uint32_t f32_to_bf16(float f) { return f32x2_to_bf16x2(f, 0.0f) & 0xFFFFu; }

// -------------------------------------------------------------- raw vectors
// RawVec<K, VEC> holds VEC elements of kind K in their storage format, in
// ceil(VEC*bytes/4) 32-bit registers, and moves with a single global access.

template <Kind K, int VEC> struct RawVec {
    static constexpr int BYTES = VEC * KindInfo<K>::bytes;
    static constexpr int WORDS = BYTES >= 4 ? BYTES / 4 : 1;
    uint32_t w[WORDS];
};

// ------------------------------------------------------- buffer access
// Raw buffer loads and stores: 32-bit byte offsets from a base held in
// scalar registers, with the range check done by the memory pipeline -- a
// load at or past the resource's byte count returns zeros and a store there
// is dropped -- so the edges of a tile need no branches or masks.  Both use
// the non-temporal cache policy: the scans read and write every element
// once (non-temporal loads took the f32 T = 2^20, d = 256 forward / reverse
// scans from 575 / 946 to 562 / 935 us).  Every offset goes in the per-lane
// (range-checked) operand; the scalar offset, which the check does not
// cover, is always 0.
typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int kRsrcWord3 = 0x00020000;       // gfx9 raw buffer, 32-bit data format
constexpr uint32_t kOob = 0x80000000u;       // an offset past every resource's range
constexpr int kNt = 2;                       // cache policy: non-temporal

__device__ __forceinline__ Rsrc make_rsrc(const void* base, int64_t bytes) {
    const int n = bytes >= 0x7FFFFFFF ? 0x7FFFFFFF : (bytes <= 0 ? 0 : (int)bytes);
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, kRsrcWord3);
}

__device__ __forceinline__ uint32_t bload_u8(Rsrc r, uint32_t off) {
    return (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(r, (int)off, 0, 0);
}

template <int BYTES> struct WideAccess;

template <> struct WideAccess<2> {
    template <int W> __device__ static void bload(uint32_t (&w)[W], Rsrc r, uint32_t off) {
        w[0] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(r, (int)off, 0, kNt);
    }
    template <int W> __device__ static void bstore_nt(Rsrc r, uint32_t off, const uint32_t (&w)[W]) {
        __builtin_amdgcn_raw_buffer_store_b16((unsigned short)w[0], r, (int)off, 0, kNt);
    }
    template <int W> __device__ static void load(uint32_t (&w)[W], const void* p) {
        w[0] = *(const uint16_t*)p;
    }
    template <int W> __device__ static void store_nt(void* p, const uint32_t (&w)[W]) {
        __builtin_nontemporal_store((uint16_t)w[0], (uint16_t*)p);
    }
};
template <> struct WideAccess<4> {
    template <int W> __device__ static void bload(uint32_t (&w)[W], Rsrc r, uint32_t off) {
        w[0] = __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, kNt);
    }
    template <int W> __device__ static void bstore_nt(Rsrc r, uint32_t off, const uint32_t (&w)[W]) {
        __builtin_amdgcn_raw_buffer_store_b32(w[0], r, (int)off, 0, kNt);
    }
    template <int W> __device__ static void load(uint32_t (&w)[W], const void* p) {
        w[0] = *(const uint32_t*)p;
    }
    template <int W> __device__ static void store_nt(void* p, const uint32_t (&w)[W]) {
        __builtin_nontemporal_store(w[0], (uint32_t*)p);
    }
};
template <> struct WideAccess<8> {
    template <int W> __device__ static void bload(uint32_t (&w)[W], Rsrc r, uint32_t off) {
        const u32x2 v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, kNt);
        w[0] = v.x; w[1] = v.y;
    }
    template <int W> __device__ static void bstore_nt(Rsrc r, uint32_t off, const uint32_t (&w)[W]) {
        const u32x2 v = {w[0], w[1]};
        __builtin_amdgcn_raw_buffer_store_b64(v, r, (int)off, 0, kNt);
    }
    template <int W> __device__ static void load(uint32_t (&w)[W], const void* p) {
        u32x2 v = *(const u32x2*)p;
        w[0] = v.x; w[1] = v.y;
    }
    template <int W> __device__ static void store_nt(void* p, const uint32_t (&w)[W]) {
        u32x2 v = {w[0], w[1]};
        __builtin_nontemporal_store(v, (u32x2*)p);
    }
};
template <> struct WideAccess<16> {
    template <int W> __device__ static void bload(uint32_t (&w)[W], Rsrc r, uint32_t off) {
        const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kNt);
        w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
    }
    template <int W> __device__ static void bstore_nt(Rsrc r, uint32_t off, const uint32_t (&w)[W]) {
        const u32x4 v = {w[0], w[1], w[2], w[3]};
        __builtin_amdgcn_raw_buffer_store_b128(v, r, (int)off, 0, kNt);
    }
    template <int W> __device__ static void load(uint32_t (&w)[W], const void* p) {
        u32x4 v = *(const u32x4*)p;
        w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
    }
    template <int W> __device__ static void store_nt(void* p, const uint32_t (&w)[W]) {
        u32x4 v = {w[0], w[1], w[2], w[3]};
        __builtin_nontemporal_store(v, (u32x4*)p);
    }
};
template <> struct WideAccess<32> {
    template <int W> __device__ static void bload(uint32_t (&w)[W], Rsrc r, uint32_t off) {
        const u32x4 v0 = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, kNt);
        const u32x4 v1 = __builtin_amdgcn_raw_buffer_load_b128(r, (int)(off + 16u), 0, kNt);
        w[0] = v0.x; w[1] = v0.y; w[2] = v0.z; w[3] = v0.w;
        w[4] = v1.x; w[5] = v1.y; w[6] = v1.z; w[7] = v1.w;
    }
    template <int W> __device__ static void bstore_nt(Rsrc r, uint32_t off, const uint32_t (&w)[W]) {
        const u32x4 v0 = {w[0], w[1], w[2], w[3]};
        const u32x4 v1 = {w[4], w[5], w[6], w[7]};
        __builtin_amdgcn_raw_buffer_store_b128(v0, r, (int)off, 0, kNt);
        __builtin_amdgcn_raw_buffer_store_b128(v1, r, (int)(off + 16u), 0, kNt);
    }
    template <int W> __device__ static void load(uint32_t (&w)[W], const void* p) {
        u32x4 v0 = ((const u32x4*)p)[0];
        u32x4 v1 = ((const u32x4*)p)[1];
        w[0] = v0.x; w[1] = v0.y; w[2] = v0.z; w[3] = v0.w;
        w[4] = v1.x; w[5] = v1.y; w[6] = v1.z; w[7] = v1.w;
    }
    template <int W> __device__ static void store_nt(void* p, const uint32_t (&w)[W]) {
        u32x4 v0 = {w[0], w[1], w[2], w[3]};
        u32x4 v1 = {w[4], w[5], w[6], w[7]};
        __builtin_nontemporal_store(v0, (u32x4*)p);
        __builtin_nontemporal_store(v1, (u32x4*)p + 1);
    }
};

template <Kind K, int VEC>
__device__ __forceinline__ void raw_load(RawVec<K, VEC>& r, const void* p) {
    WideAccess<RawVec<K, VEC>::BYTES>::load(r.w, p);
}

template <Kind K, int VEC>
__device__ __forceinline__ void raw_store_nt(void* p, const RawVec<K, VEC>& r) {
    WideAccess<RawVec<K, VEC>::BYTES>::store_nt(p, r.w);
}

template <Kind K, int VEC>
__device__ __forceinline__ void raw_bload(RawVec<K, VEC>& r, Rsrc rs, uint32_t off) {
    WideAccess<RawVec<K, VEC>::BYTES>::bload(r.w, rs, off);
}

template <Kind K, int VEC>
__device__ __forceinline__ void raw_bstore_nt(Rsrc rs, uint32_t off, const RawVec<K, VEC>& r) {
    WideAccess<RawVec<K, VEC>::BYTES>::bstore_nt(rs, off, r.w);
}

// decode element i of a raw vector into its state type
template <Kind K, int VEC> struct Codec;

template <int VEC> struct Codec<K_F32, VEC> {
    __device__ static float get(const RawVec<K_F32, VEC>& r, int i) { return __uint_as_float(r.w[i]); }
    __device__ static void put(RawVec<K_F32, VEC>& r, int i, float v) { r.w[i] = __float_as_uint(v); }
    __device__ static void put_all(RawVec<K_F32, VEC>& r, const float (&v)[VEC]) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) r.w[i] = __float_as_uint(v[i]);
    }
};
template <int VEC> struct Codec<K_BF16, VEC> {
    __device__ static float get(const RawVec<K_BF16, VEC>& r, int i) {
        return (i & 1) ? bf16_hi(r.w[i >> 1]) : bf16_lo(r.w[i >> 1]);
    }
    __device__ static void put(RawVec<K_BF16, VEC>& r, int i, float v) {
        const uint32_t b = f32_to_bf16(v);
        if (i & 1) r.w[i >> 1] = (r.w[i >> 1] & 0x0000FFFFu) | (b << 16);
        else r.w[i >> 1] = (r.w[i >> 1] & 0xFFFF0000u) | b;
    }
    __device__ static void put_all(RawVec<K_BF16, VEC>& r, const float (&v)[VEC]) {
        if constexpr (VEC == 1) {
            r.w[0] = f32_to_bf16(v[0]);
        } else {
#pragma unroll
            for (int i = 0; i < VEC / 2; ++i) r.w[i] = f32x2_to_bf16x2(v[2 * i], v[2 * i + 1]);
        }
    }
};
template <int VEC> struct Codec<K_C64, VEC> {
    __device__ static cf get(const RawVec<K_C64, VEC>& r, int i) {
        return cf{__uint_as_float(r.w[2 * i]), __uint_as_float(r.w[2 * i + 1])};
    }
    __device__ static void put(RawVec<K_C64, VEC>& r, int i, cf v) {
        r.w[2 * i] = __float_as_uint(v.re);
        r.w[2 * i + 1] = __float_as_uint(v.im);
    }
    __device__ static void put_all(RawVec<K_C64, VEC>& r, const cf (&v)[VEC]) {
#pragma unroll
        for (int i = 0; i < VEC; ++i) put(r, i, v[i]);
    }
};

// ------------------------------------------------------ cross-lane moves
// The value held by the lane whose index differs from this lane's in bit m
// (m a power of two from 1 to 32, the same in every lane; every lane
// active).  Where the hardware allows it the move is a modifier of a VALU
// instruction rather than a trip through the LDS crossbar: DPP quad
// permutations for m = 1 and 2, the 16-lane row rotation by 8 for m = 8
// (within a row of 16 lanes, i + 8 mod 16 = i xor 8), and v_permlane32_swap
// (gfx950) for m = 32, which exchanges the wavefront's two halves; m = 4 and
// 16 use ds_swizzle's xor mode (lanes within 32, no LDS memory).
__device__ __forceinline__ uint32_t lanes_xor(uint32_t v, int m) {
    switch (m) {
        case 1: return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0xB1, 0xF, 0xF, false);  // quad_perm [1,0,3,2]
        case 2: return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x4E, 0xF, 0xF, false);  // quad_perm [2,3,0,1]
        case 4: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x101F);                         // xor mask 4
        case 8: return (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x128, 0xF, 0xF, false); // row_ror:8
        case 16: return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, 0x401F);                        // xor mask 16
        default: {
            // new vdst: the low half copied to the high half; new vsrc: the
            // high half copied to the low half
            const auto pr = __builtin_amdgcn_permlane32_swap(v, v, false, false);
            return (threadIdx.x & 32) ? pr[0] : pr[1];
        }
    }
}
__device__ __forceinline__ float lanes_xor(float v, int m) { return __uint_as_float(lanes_xor(__float_as_uint(v), m)); }
// the value of lane `src` (ds_bpermute)
__device__ __forceinline__ float lanes_read(float v, int src) { return __shfl(v, src, 64); }
__device__ __forceinline__ cf lanes_read(cf v, int src) { return cf{__shfl(v.re, src, 64), __shfl(v.im, src, 64)}; }
__device__ __forceinline__ cf lanes_xor(cf v, int m) { return cf{lanes_xor(v.re, m), lanes_xor(v.im, m)}; }
__device__ __forceinline__ uint64_t lanes_xor(uint64_t v, int m) {
    return (uint64_t)lanes_xor((uint32_t)v, m) | ((uint64_t)lanes_xor((uint32_t)(v >> 32), m) << 32);
}
__device__ __forceinline__ int64_t lanes_xor(int64_t v, int m) { return (int64_t)lanes_xor((uint64_t)v, m); }

// ds_swizzle in bitmask mode: lane l (of each group of 32) reads lane
// (l & AND) | OR of its group; no LDS memory is touched.
template <int AND, int OR>
__device__ __forceinline__ uint32_t swz(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_ds_swizzle((int)v, AND | (OR << 5));
}
// every lane reads the same lane index in the other half of the wavefront
__device__ __forceinline__ uint32_t half_swap(uint32_t v) {
    const auto pr = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return (threadIdx.x & 32) ? pr[0] : pr[1];
}

// Moves of a Sklansky scan over lane groups (lane = j * QP + q, QP a power
// of two).  At step M (a multiple of QP below 64) the lanes form blocks of
// 2M; sk_move<false> gives every lane the value of the LAST group of the
// lower half of its block, (l & ~(2M - 1)) | (M - QP) | q, which is what the
// upper half needs for a forward scan; sk_move<true> gives the FIRST group
// of the upper half, (l & ~(2M - 1)) | M | q, for a reverse scan.  The row
// shifts by 8 are DPP modifiers, the others ds_swizzle patterns within 32
// lanes (source (l & AND) | OR), followed by a half swap when the block is
// the whole wavefront; M = 32 with QP = 1 is a scalar lane read.
template <bool UP, int M, int QP>
__device__ __forceinline__ uint32_t sk_move(uint32_t v) {
    static_assert(QP >= 1 && QP <= M && M <= 32 && (QP & (QP - 1)) == 0 && (M & (M - 1)) == 0, "Sklansky step");
    constexpr int Q = QP - 1;
    if constexpr (M == 8 && QP == 8) {
        return UP ? (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x108, 0xF, 0xF, false)   // row_shl:8
                  : (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x118, 0xF, 0xF, false);  // row_shr:8
    } else if constexpr (M == 32 && QP == 1) {
        return (uint32_t)__builtin_amdgcn_readlane((int)v, UP ? 32 : 31);
    } else if constexpr (M == 32) {
        return half_swap(swz<Q, UP ? 0 : 32 - QP>(v));
    } else {
        return swz<(0x1F & ~(2 * M - 1)) | Q, UP ? M : M - QP>(v);
    }
}
template <bool UP, int M, int QP>
__device__ __forceinline__ float sk_move(float v) {
    return __uint_as_float(sk_move<UP, M, QP>(__float_as_uint(v)));
}
template <bool UP, int M, int QP>
__device__ __forceinline__ cf sk_move(cf v) {
    return cf{sk_move<UP, M, QP>(v.re), sk_move<UP, M, QP>(v.im)};
}

// Inclusive prefix sum over the lanes of a wavefront in strides of `stride`
// lanes (lane = j * stride + q; the groups j = 0, 1, ... are summed in
// order, separately for each q): an xor butterfly, log2(64 / stride) moves.
template <class V>
__device__ __forceinline__ V lanes_prefix_sum(V v, int stride) {
    const int lane = threadIdx.x & 63;
    V tot = v;
    for (int m = stride; m < 64; m <<= 1) {
        const V o = lanes_xor(tot, m);
        if (lane & m) v += o;
        tot += o;
    }
    return v;
}

// ------------------------------------------------------- descriptor words
// Cross-tile communication of the single-pass scan.  Every word is written
// once per call with a relaxed agent-scope atomic store and read with relaxed
// agent-scope atomic loads, and validates itself: an unpublished word holds
// all-ones bytes, and a published value never has that bit pattern because
// every float is canonicalised (any NaN becomes 0x7FC00000) before it is
// stored.  No fence is needed: a reader that sees a valid word sees the whole
// value, and no other memory is ordered against it.
//
// The words live in two banks.  A call publishes into the bank of its epoch's
// parity and every tile resets its own words of the other bank to all ones,
// so the next call (epoch + 1) finds its bank clean without any fill pass:
// a prepared workspace (all ones) stays ready from call to call.  The epoch
// comes from the tile counters, which are never reset: a call takes exactly
// n tickets from a counter that hands out n per call, so ticket / n is the
// number of calls before it.

constexpr uint32_t kEmpty32 = 0xFFFFFFFFu;
constexpr uint64_t kEmpty64 = 0xFFFFFFFFFFFFFFFFull;

__device__ __forceinline__ float canon(float v) { return v != v ? __uint_as_float(0x7FC00000u) : v; }

__device__ __forceinline__ uint64_t pack2(float lo, float hi) {
    return (uint64_t)__float_as_uint(canon(lo)) | ((uint64_t)__float_as_uint(canon(hi)) << 32);
}
__device__ __forceinline__ float unpack_lo(uint64_t w) { return __uint_as_float((uint32_t)w); }
__device__ __forceinline__ float unpack_hi(uint64_t w) { return __uint_as_float((uint32_t)(w >> 32)); }

__device__ __forceinline__ void publish64(uint64_t* p, uint64_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t peek64(const uint64_t* p) {
    return __hip_atomic_load(const_cast<uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void publish32(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint32_t peek32(const uint32_t* p) {
    return __hip_atomic_load(const_cast<uint32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// A state value as one self-validating 64-bit word (real: (v, 0); complex:
// (re, im)), and back.
__device__ __forceinline__ uint64_t pack_state(float v) { return pack2(v, 0.0f); }
__device__ __forceinline__ uint64_t pack_state(cf v) { return pack2(v.re, v.im); }
template <class S> __device__ __forceinline__ S unpack_state(uint64_t w);
template <> __device__ __forceinline__ float unpack_state<float>(uint64_t w) { return unpack_lo(w); }
template <> __device__ __forceinline__ cf unpack_state<cf>(uint64_t w) { return cf{unpack_lo(w), unpack_hi(w)}; }

// Per-feature tile summary of the scan state, in the two forms a successor
// can use.  AGG: (A, H) of a tile without a begin step, i.e. h_end =
// A * h_before + H.  INCL: h_end itself (the tile's inclusive prefix).
//   real:    AGG = one 64-bit word (A, H);      INCL = one 32-bit word H
//   complex: AGG = two 64-bit words A, H;       INCL = one 64-bit word H
template <class S> struct Desc;

template <> struct Desc<float> {
    static constexpr int agg_bytes = 8;
    static constexpr int incl_bytes = 4;
    __device__ static void put_agg(void* base, int64_t i, float A, float H) {
        publish64((uint64_t*)base + i, pack2(A, H));
    }
    __device__ static void put_incl(void* base, int64_t i, float H) {
        publish32((uint32_t*)base + i, __float_as_uint(canon(H)));
    }
    __device__ static bool get_agg(const void* base, int64_t i, float& A, float& H) {
        const uint64_t w = peek64((const uint64_t*)base + i);
        A = unpack_lo(w);
        H = unpack_hi(w);
        return w != kEmpty64;
    }
    __device__ static bool get_incl(const void* base, int64_t i, float& H) {
        const uint32_t w = peek32((const uint32_t*)base + i);
        H = __uint_as_float(w);
        return w != kEmpty32;
    }
    // back to unpublished (words of the idle bank; plain stores, read only
    // after the kernel has ended)
    __device__ static void clear(void* agg, void* incl, int64_t i) {
        ((uint64_t*)agg)[i] = kEmpty64;
        ((uint32_t*)incl)[i] = kEmpty32;
    }
};

template <> struct Desc<cf> {
    static constexpr int agg_bytes = 16;
    static constexpr int incl_bytes = 8;
    __device__ static void put_agg(void* base, int64_t i, cf A, cf H) {
        publish64((uint64_t*)base + 2 * i, pack2(A.re, A.im));
        publish64((uint64_t*)base + 2 * i + 1, pack2(H.re, H.im));
    }
    __device__ static void put_incl(void* base, int64_t i, cf H) {
        publish64((uint64_t*)base + i, pack2(H.re, H.im));
    }
    __device__ static bool get_agg(const void* base, int64_t i, cf& A, cf& H) {
        const uint64_t wa = peek64((const uint64_t*)base + 2 * i);
        const uint64_t wh = peek64((const uint64_t*)base + 2 * i + 1);
        A = cf{unpack_lo(wa), unpack_hi(wa)};
        H = cf{unpack_lo(wh), unpack_hi(wh)};
        return wa != kEmpty64 && wh != kEmpty64;
    }
    __device__ static bool get_incl(const void* base, int64_t i, cf& H) {
        const uint64_t w = peek64((const uint64_t*)base + i);
        H = cf{unpack_lo(w), unpack_hi(w)};
        return w != kEmpty64;
    }
    __device__ static void clear(void* agg, void* incl, int64_t i) {
        ((uint64_t*)agg)[2 * i] = kEmpty64;
        ((uint64_t*)agg)[2 * i + 1] = kEmpty64;
        ((uint64_t*)incl)[i] = kEmpty64;
    }
};

// FFM transition of a chain's Dp features, a_jk = exp(-|alpha_j|) (cos omega_k
// + i sin omega_k) for feature f = j * c + k, evaluated once per tile: lane
// l < Dp (Dp <= 64, so wavefront 0 alone) takes feature f_base + l, in double
// and rounded once to float (with |a| near 1 the error of a is amplified by up
// to the episode length), into tab[l].  conj_a stores conj(a) (the reverse
// scan's coefficient).  Features past d get a valid, unused value.  The caller
// synchronises the workgroup before reading tab.  Two steps, so that a
// kernel can load the parameters first and evaluate the table while its
// other loads are in flight.
struct FfmParam {
    float alpha, omega;
};
__device__ __forceinline__ FfmParam ffm_param_load(const float* alpha, const float* omega, int64_t d, int64_t c,
                                                   int64_t f_base, int Dp) {
    FfmParam r{0.f, 0.f};
    const int l = threadIdx.x;
    if (l < Dp) {
        const int64_t f = f_base + l < d ? f_base + l : 0;
        const int64_t jj = f / c, kk = f - jj * c;
        r.alpha = alpha[jj];
        r.omega = omega[kk];
    }
    return r;
}
__device__ __forceinline__ void ffm_table_store(cf* tab, FfmParam pr, int Dp, bool conj_a) {
    const int l = threadIdx.x;
    if (l < Dp) {
        const double mag = exp(-fabs((double)pr.alpha));
        double sn, cs;
        sincos((double)pr.omega, &sn, &cs);
        const float im = (float)(mag * sn);
        tab[l] = cf{(float)(mag * cs), conj_a ? -im : im};
    }
}

// Descriptor slot of feature v of lane q inside tile `ticket`'s block of Dp
// features: lanes are contiguous for a fixed v, so the accesses of a
// wavefront coalesce.
__device__ __forceinline__ int64_t desc_slot(int64_t ticket, int Dp, int Qp, int q, int v) {
    return ticket * Dp + (int64_t)v * Qp + q;
}



// Bound on polls of one predecessor descriptor before a wait gives up and
// flags MEMOROID_ETIMEOUT in the workspace (about a second of polling).  The
// ticketed tile order guarantees every awaited tile is running or done, so
// the bound only matters if that guarantee were broken.
constexpr uint32_t kMaxPolls = 1u << 22;

// The header's timeout word reads all ones until a wait gives up.
constexpr uint32_t kTimedOut = 0u;
__device__ __forceinline__ void flag_timeout(uint32_t* timeout) {
    __hip_atomic_store(timeout, kTimedOut, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------- look-back
// Carry-in of a tile: the chain's state just before the tile, found by
// walking back over predecessor tiles (tickets pred, pred - nchains, ...):
// aggregates are folded until an inclusive prefix closes the walk.  One whole
// wavefront runs it.  Its lanes form 64 / Qp groups of Qp lanes; lane (j, q)
// polls predecessor base - j * nchains for the features of lane position q,
// so each round trip to memory examines a window of 64 / Qp predecessors.
// The window's entries go through LDS, and every lane then walks the window
// in order for its q (lanes sharing q compute identical results).  A round
// ends by resolving, by consuming the ready prefix of the window, or, if the
// nearest predecessor is not yet published, by sleeping and polling again.
// `need` false (no carry needed, or features past d) yields zeros.
template <class S, int VEC>
struct LookbackLds {
    uint32_t st[64];
    S a[64 * VEC];
    S h[64 * VEC];
};

template <class S, int VEC>
__device__ __forceinline__ void lookback(const void* agg, const void* incl, int64_t first_pred, int nchains,
                                         int Dp, int Qp, bool need, S (&carry)[VEC], LookbackLds<S, VEC>& lds,
                                         uint32_t* timeout) {
    const int lane = threadIdx.x & 63;
    const int qsh = __builtin_ctz((unsigned)Qp);   // Qp is a power of two
    const int q = lane & (Qp - 1);
    const int j = lane >> qsh;
    const int Gw = 64 >> qsh;
    S accA[VEC], accH[VEC];
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        accA[v] = s_one<S>();
        accH[v] = s_zero<S>();
        carry[v] = s_zero<S>();
    }
    int64_t base = first_pred;
    bool done = !need;
    uint32_t polls = 0;
    while (!__all(done)) {
        const int64_t pj = base - (int64_t)j * nchains;
        uint32_t stt = 0;
        S va[VEC], vh[VEC];
        if (!done && pj >= 0) {
            S ih[VEC], ga[VEC], gh[VEC];
            bool inc_ok = true, agg_ok = true;
#pragma unroll
            for (int v = 0; v < VEC; ++v)
                inc_ok = Desc<S>::get_incl(incl, desc_slot(pj, Dp, Qp, q, v), ih[v]) && inc_ok;
#pragma unroll
            for (int v = 0; v < VEC; ++v)
                agg_ok = Desc<S>::get_agg(agg, desc_slot(pj, Dp, Qp, q, v), ga[v], gh[v]) && agg_ok;
            stt = inc_ok ? 2u : (agg_ok ? 1u : 0u);
#pragma unroll
            for (int v = 0; v < VEC; ++v) {
                va[v] = ga[v];
                vh[v] = inc_ok ? ih[v] : gh[v];
            }
        }
        lds.st[lane] = stt;
#pragma unroll
        for (int v = 0; v < VEC; ++v) {
            lds.a[lane * VEC + v] = va[v];
            lds.h[lane * VEC + v] = vh[v];
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (!done) {
            int consumed = 0;
            bool resolved = false;
            for (int jj = 0; jj < Gw; ++jj) {
                const int e = jj * Qp + q;
                const uint32_t se = lds.st[e];
                if (se == 2u) {
#pragma unroll
                    for (int v = 0; v < VEC; ++v) carry[v] = mad(accA[v], lds.h[e * VEC + v], accH[v]);
                    resolved = true;
                    break;
                }
                if (se != 1u) break;
#pragma unroll
                for (int v = 0; v < VEC; ++v) {
                    accH[v] = mad(accA[v], lds.h[e * VEC + v], accH[v]);
                    accA[v] = accA[v] * lds.a[e * VEC + v];
                }
                ++consumed;
            }
            base -= (int64_t)consumed * nchains;
            if (resolved) {
                done = true;
            } else if (consumed == 0) {
                if (++polls > kMaxPolls) {
                    flag_timeout(timeout);
                    done = true;
                } else {
                    __builtin_amdgcn_s_sleep(1);
                }
            }
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
}

// A workgroup barrier that orders LDS only.  __syncthreads also waits until
// the wavefront's global stores are acknowledged (one completion counter
// covers loads and stores here), which puts a store round trip on the path of
// every barrier that follows a publication; these barriers hand on LDS values
// only.
__device__ __forceinline__ void barrier_lds() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// The nearest predecessor's inclusive words for lane position q, read ahead
// of the look-back (a speculative first poll): a tile usually starts well
// after the previous tile of its chain was handed out, so these words are
// often published already, and reading them before the tile's data loads
// hides the round trip behind those loads.  Returns whether all were there.
template <class S, int VEC>
__device__ __forceinline__ bool peek_incl_ahead(const void* incl, int64_t pred, int Dp, int Qp, int q,
                                                S (&h)[VEC]) {
    bool ok = true;
#pragma unroll
    for (int v = 0; v < VEC; ++v) ok = Desc<S>::get_incl(incl, desc_slot(pred, Dp, Qp, q, v), h[v]) && ok;
    return ok;
}

// ------------------------------------------------------------ segments
// Summary of a run of consecutive steps (in scan order) of one feature: the
// state after the run is  f ? H : A * (state before) + H,  f meaning "the run
// holds an episode boundary".  This is the resettable monoid of the Section 4
// theorem specialised to the diagonal recurrence, carried as a select.
template <class S, int VEC>
struct Seg {
    S A[VEC], H[VEC];
    bool f;
};

template <class S, int VEC>
__device__ __forceinline__ Seg<S, VEC> seg_identity() {
    Seg<S, VEC> r;
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        r.A[v] = s_one<S>();
        r.H[v] = s_zero<S>();
    }
    r.f = false;
    return r;
}

// the run `first` followed by the run `second`
template <class S, int VEC>
__device__ __forceinline__ Seg<S, VEC> seg_then(const Seg<S, VEC>& first, const Seg<S, VEC>& second) {
    if (second.f) return second;
    Seg<S, VEC> r;
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        r.H[v] = mad(second.A[v], first.H[v], second.H[v]);
        r.A[v] = second.A[v] * first.A[v];
    }
    r.f = first.f;
    return r;
}

// state after the run, given the state before it
template <class S, int VEC>
__device__ __forceinline__ S seg_apply(const Seg<S, VEC>& sg, int v, S before) {
    return sg.f ? sg.H[v] : mad(sg.A[v], before, sg.H[v]);
}


template <class S, int VEC>
__device__ __forceinline__ Seg<S, VEC> seg_select(bool c, const Seg<S, VEC>& x, const Seg<S, VEC>& y) {
    Seg<S, VEC> r;
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        r.A[v] = c ? x.A[v] : y.A[v];
        r.H[v] = c ? x.H[v] : y.H[v];
    }
    r.f = c ? x.f : y.f;
    return r;
}

template <class S, int VEC, bool UP, int M, int QP>
__device__ __forceinline__ Seg<S, VEC> seg_sk_move(const Seg<S, VEC>& x) {
    Seg<S, VEC> r;
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        r.A[v] = sk_move<UP, M, QP>(x.A[v]);
        r.H[v] = sk_move<UP, M, QP>(x.H[v]);
    }
    r.f = sk_move<UP, M, QP>((uint32_t)x.f) != 0u;
    return r;
}

// the Sklansky steps M, 2 M, ... 32 of wave_group_scan (groups of QP lanes)
template <class S, int VEC, bool REV, int M, int QP>
__device__ __forceinline__ void sk_steps(Seg<S, VEC>& inc) {
    if constexpr (M < 64) {
        const int lane = threadIdx.x & 63;
        const Seg<S, VEC> o = seg_sk_move<S, VEC, REV, M, QP>(inc);
        const bool takes = REV ? (lane & M) == 0 : (lane & M) != 0;
        inc = seg_select<S, VEC>(takes, seg_then<S, VEC>(o, inc), inc);
        sk_steps<S, VEC, REV, 2 * M, QP>(inc);
    }
}

template <class S, int VEC>
__device__ __forceinline__ Seg<S, VEC> seg_shfl(const Seg<S, VEC>& x, int src) {
    Seg<S, VEC> r;
#pragma unroll
    for (int v = 0; v < VEC; ++v) {
        r.A[v] = lanes_read(x.A[v], src);
        r.H[v] = lanes_read(x.H[v], src);
    }
    r.f = __shfl((int)x.f, src, 64) != 0;
    return r;
}

// Scan across the Gw = 64 / Qp lane groups of a wavefront (lane = j * Qp + q;
// Qp <= QMAX;
// group j holds consecutive steps, group j + 1 the ones after).  Forward
// (REV = false): groups earlier in time come first; reverse: later ones.  On
// return `inc` is the run from the wavefront's first group (in scan order)
// through this lane's group, and `exc` the run before this lane's group.
// Sklansky: at step M (M = Qp, 2 Qp, ... 32) the half of each block of 2M
// lanes that comes second in scan order puts the other half's total (the
// inclusive run of that half's last group in scan order) in front of its
// own run -- one partner move (DPP row shift, ds_swizzle, permlane half
// swap: sk_move) and one combine per step, no LDS memory and no barrier.
// The exclusive run is the inclusive run of the previous group, one
// ds_bpermute.
template <class S, int VEC, bool REV, int QMAX = 64>
__device__ __forceinline__ void wave_group_scan(Seg<S, VEC>& inc, Seg<S, VEC>& exc, int Qp) {
    const int lane = threadIdx.x & 63;
    const int qsh = __builtin_ctz((unsigned)Qp);   // Qp is a power of two
    const int j = lane >> qsh;
    const int Gw = 64 >> qsh;
    // one uniform dispatch on the group width; every step's moves are then
    // fixed at compile time
    // (QMAX: the largest group width the kernel's plans use)
    switch (Qp) {
        case 1: sk_steps<S, VEC, REV, 1, 1>(inc); break;
        case 2: if constexpr (QMAX >= 2) sk_steps<S, VEC, REV, 2, 2>(inc); break;
        case 4: if constexpr (QMAX >= 4) sk_steps<S, VEC, REV, 4, 4>(inc); break;
        case 8: if constexpr (QMAX >= 8) sk_steps<S, VEC, REV, 8, 8>(inc); break;
        case 16: if constexpr (QMAX >= 16) sk_steps<S, VEC, REV, 16, 16>(inc); break;
        case 32: if constexpr (QMAX >= 32) sk_steps<S, VEC, REV, 32, 32>(inc); break;
        default: break;                                  // one group: nothing to scan
    }
    const bool has = REV ? (j + 1 < Gw) : (j >= 1);
    const Seg<S, VEC> o = seg_shfl<S, VEC>(inc, has ? (REV ? lane + Qp : lane - Qp) : lane);
    exc = seg_select<S, VEC>(has, o, seg_identity<S, VEC>());
}

// ------------------------------------------------------- count look-back
// Running count of begin steps before a tile (the episode index is that count
// minus one), carried by one 64-bit word per tile: all ones = not yet
// published, bit 62 = the tile's own count, bit 63 = the count through the
// end of the tile; the low 62 bits hold the value (under 2^32 for a count
// of begin steps, under 2^48 for the row sums of batch sampling).  A count
// never resets, so the walk always goes back to an inclusive word; one
// wavefront polls a window of 256 predecessors per round trip (position
// o = 64 k + lane is predecessor base - o * stride) and the ready prefix of
// the window is summed with cross-lane reductions.  The wide window matters
// when a thousand tiles run at once: a running count then crosses them in a
// few round trips.
constexpr uint64_t kCountOwn = 1ull << 62;
constexpr uint64_t kCountIncl = 2ull << 62;
constexpr uint64_t kCountValue = kCountOwn - 1;

__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v) {
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) v += lanes_xor(v, m);
    return v;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
    for (int m = 1; m < 64; m <<= 1) v += lanes_xor(v, m);
    return v;
}
__device__ __forceinline__ uint32_t wave_sum(uint32_t v) { return wave_sum_u32(v); }
__device__ __forceinline__ uint64_t wave_sum(uint64_t v) { return wave_sum_u64(v); }

constexpr int kCountWin = 4;      // blocks of 64 predecessors per round trip

// One round trip of a count look-back from predecessor `base`: `sum` gets the
// counts of the window's ready prefix (through the nearest inclusive word, or
// up to the nearest unpublished one) and `used` the positions consumed;
// returns true when an inclusive word closed the walk.  Positions before the
// first tile of the tape read as an inclusive zero.
template <typename V, int WIN = kCountWin>
__device__ __forceinline__ bool count_window(const uint64_t* desc, int64_t base, int64_t stride, V& sum, int& used) {
    const int lane = threadIdx.x & 63;
    uint64_t w[WIN];
#pragma unroll
    for (int k = 0; k < WIN; ++k) {
        const int64_t i = base - (int64_t)(64 * k + lane) * stride;
        w[k] = i >= 0 ? peek64(desc + i) : kCountIncl;
    }
    int fi = 64 * WIN, fe = 64 * WIN;                   // first inclusive / unpublished position
#pragma unroll
    for (int k = WIN - 1; k >= 0; --k) {                // the nearest block wins
        const bool empty = w[k] == kEmpty64;
        const uint64_t me = __ballot(empty);
        const uint64_t mi = __ballot(!empty && (w[k] & kCountIncl) != 0);
        if (me) fe = 64 * k + __builtin_ctzll(me);
        if (mi) fi = 64 * k + __builtin_ctzll(mi);
    }
    const bool stop = fi < fe;
    used = stop ? fi + 1 : fe;
    V mine = 0;
#pragma unroll
    for (int k = 0; k < WIN; ++k) mine += 64 * k + lane < used ? (V)(w[k] & kCountValue) : (V)0;
    sum = wave_sum(mine);
    return stop;
}

__device__ __forceinline__ uint32_t count_lookback(const uint64_t* desc, int64_t first_pred, int64_t stride,
                                                   uint32_t* timeout) {
    uint32_t acc = 0;
    int64_t base = first_pred;
    uint32_t polls = 0;
    while (true) {
        uint32_t s;
        int used;
        if (count_window(desc, base, stride, s, used)) return acc + s;
        acc += s;
        base -= (int64_t)used * stride;
        if (used == 0) {
            if (++polls > kMaxPolls) {
                flag_timeout(timeout);
                return acc;
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
}

// Workspace header shared by the scan kernels (first 256 bytes).  Prepared
// state: all ones.
struct WsHeader {
    uint32_t reserved;
    uint32_t timeout;    // kTimedOut: some wait gave up
    uint64_t sig;        // signature of the call the workspace is bound to
    uint32_t pad[60];
};

// Signature word: all ones = not bound yet; kSigPoisoned = a call with
// another signature found the workspace (it must be prepared again).
constexpr uint64_t kSigPoisoned = 0ull;

// The signature word as a tile reads it: a cacheable load (workgroup
// scope), so that thousands of tiles reading the one word are served by the
// caches instead of queueing at one memory channel.  Within a call the word
// only changes from all ones to the call's own signature, or to
// kSigPoisoned in a call that finds a foreign signature (whose tiles all
// stand down whichever of the values they see); between calls the kernel
// boundary makes the last value visible.
__device__ __forceinline__ uint64_t peek_sig(const WsHeader* hdr) {
    // one aligned 8-byte raw buffer load (never torn): an ordinary cached
    // load, which the compiler need not order after the counter atomic
    // issued just before it
    typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
    const Rsrc r = make_rsrc(hdr, sizeof(WsHeader));
    const u32x2 w = __builtin_amdgcn_raw_buffer_load_b64(r, (int)offsetof(WsHeader, sig), 0, 0);
    return (uint64_t)w.x | ((uint64_t)w.y << 32);
}

// Binding check of a tile (one thread), given the signature word it read
// (`w`, loaded beside the tile's counter atomic so that the check costs no
// extra round trip): a fresh workspace is bound to the first call's
// signature (written by one designated tile of that call); a call with
// another signature poisons it and all of its tiles stand down (every tile
// of that call sees a foreign or poisoned signature, so they agree).
__device__ __forceinline__ bool ws_bound_to(WsHeader* hdr, uint64_t sig, uint64_t w, bool designated) {
    if (w == sig) return true;
    if (w == kEmpty64) {
        if (designated) publish64(&hdr->sig, sig);
        return true;
    }
    publish64(&hdr->sig, kSigPoisoned);
    return false;
}

// Ticket of a tile from a counter that is never reset: a wrapping atomic
// increment (new = old >= 2n - 1 ? 0 : old + 1, n tickets per call) cycles
// the counter through 0 .. 2n - 1, two calls per cycle, starting from the
// prepared value (all ones wraps to 0).  new < n: position new in an
// even-epoch call (bank 0); otherwise position new - n in an odd one
// (bank 1).  No division and no reset.
struct Claim {
    uint32_t pos;
    uint32_t bank;
};
__device__ __forceinline__ uint32_t take_ticket(uint32_t* ctr, uint32_t per_call) {
    const uint32_t top = 2u * per_call - 1u;
    const uint32_t old = __builtin_amdgcn_atomic_inc32(ctr, top, __ATOMIC_RELAXED, "agent");
    return old >= top ? 0u : old + 1u;
}
__device__ __forceinline__ Claim claim_of(uint32_t t, uint32_t per_call) {
    return t < per_call ? Claim{t, 0u} : Claim{t - per_call, 1u};
}

// Epoch of a tile that is ordered by its workgroup index: every tile owns
// one 32-bit epoch word, reads it (plus one: this call's epoch, the prepared
// value all ones reading as epoch 0) and stores the new value back at its
// end, where no later wait of the storing wavefront covers the store.  Only
// the owner touches the word and calls are ordered by the stream, so plain
// accesses suffice and nothing is contended.
__device__ __forceinline__ uint32_t read_epoch(const uint32_t* word) { return *word + 1u; }
__device__ __forceinline__ void write_epoch(uint32_t* word, uint32_t e) { *word = e; }

}  // namespace memoroid
