/*
 * memoroid_testing.h -- test-only controls of libmemoroid.so.  Not part of
 * the computation's interface (include/memoroid.h); meant for the library's
 * own tests, which use it to drive rarely taken code paths on purpose.
 */
#ifndef MEMOROID_TESTING_H
#define MEMOROID_TESTING_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------------------
 * Look-back fallback threshold of the kernels ordered by workgroup index
 * (discounted return, GAE, TBB begin indices and sampling).  A tile that
 * polls an awaited predecessor this many times without progress computes
 * that predecessor's summary from the predecessor's inputs instead of
 * waiting; 0 makes every wait take the fallback at once, so a test can
 * check its results.  The value applies to calls enqueued after this one
 * returns, process-wide; polls below 0 restore the default (4096).
 * Returns the previous value.
 * ------------------------------------------------------------------------ */
int64_t memoroid_testing_set_fallback_polls(int64_t polls);

/* ------------------------------------------------------------------------
 * Steps per tile of a diagonal scan's plan: the forward scan
 * (reverse == 0) or the reverse scan (reverse != 0) of B tapes of T steps
 * and d features of `dtype` (a memoroid_dtype; the forward scan's input
 * dtype), with a per-step (a_stride_t == d) or time-invariant
 * (a_stride_t == 0) a, on the vectorised kernels (vectorised != 0; they run
 * when d is a multiple of the vector width and the pointers are 16-byte
 * aligned) or the scalar ones.  Tests use it to place tapes exactly at tile
 * boundaries.  Returns 0 for arguments the entry point would reject.
 * ------------------------------------------------------------------------ */
int64_t memoroid_testing_tile_steps(int reverse, int64_t B, int64_t T, int64_t d, int dtype,
                                    int64_t a_stride_t, int vectorised);

#ifdef __cplusplus
}
#endif

#endif /* MEMOROID_TESTING_H */
