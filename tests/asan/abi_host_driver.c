/* abi_host_driver.c -- drives the host side of libmemoroid's C ABI without a
 * GPU: every workspace query over a grid of sizes (including extents whose
 * products overflow), and every entry point with arguments it must reject
 * before any HIP call (fake, aligned device addresses that are never
 * dereferenced).  Built by tests/test_abi_asan.py with AddressSanitizer and
 * UndefinedBehaviorSanitizer on the host code; any report aborts the run.
 * TEST INFRASTRUCTURE. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "memoroid.h"
#include "memoroid_testing.h"

#define CHECK(cond)                                                              \
    do {                                                                         \
        if (!(cond)) {                                                           \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #cond);   \
            return 1;                                                            \
        }                                                                        \
    } while (0)

static void* P(uintptr_t a) { return (void*)a; }

int main(void) {
    const int64_t ext[] = {-1, 0, 1, 3, 63, 64, 65, 511, 512, 513, 4097, 65536, 1 << 20,
                           (int64_t)1 << 31, (int64_t)1 << 40, INT64_MAX / 3, INT64_MAX};
    const int n = (int)(sizeof ext / sizeof ext[0]);
    size_t sink = 0;
    for (int i = 0; i < n; ++i)
        for (int j = 0; j < n; ++j)
            for (int k = 0; k < n; ++k) {
                const int64_t B = ext[i], T = ext[j], d = ext[k];
                for (int a = 0; a < 3; ++a)
                    for (int b = 0; b < 3; ++b) sink += memoroid_scan_diag_workspace_bytes(B, T, d, a, b);
                sink += memoroid_scan_diag_bwd_workspace_bytes(B, T, d, MEMOROID_F32, d);
                sink += memoroid_scan_diag_bwd_workspace_bytes(B, T, d, MEMOROID_C64, 0);
                sink += memoroid_scan_ffm_workspace_bytes(B, T, d, 8);
                sink += memoroid_scan_ffm_bwd_workspace_bytes(B, T, d, 4);
                sink += memoroid_scan_linattn_workspace_bytes(T, d, 64, 64, 64);
                sink += memoroid_scan_linattn_bwd_workspace_bytes(T, d, 64, 64, 64);
                sink += memoroid_discount_workspace_bytes(B, T);
                sink += memoroid_tbb_begin_indices_workspace_bytes(T);
                sink += memoroid_tbb_sample_workspace_bytes(B, T);
                for (int op = -1; op <= 10; ++op) sink += memoroid_workspace_bytes((memoroid_op)op, B, T, d, 64, 64, 64);
                for (int rev = 0; rev < 2; ++rev)
                    for (int vec = 0; vec < 2; ++vec)
                        sink += (size_t)memoroid_testing_tile_steps(rev, B, T, d, MEMOROID_F32, 0, vec);
            }
    printf("queries done (%zu)\n", sink);

    const uintptr_t A = 0x10000, X = 0x20000, S = 0x30000, H = 0x40000, W = 0x50000, I = 0x60000;
    /* diagonal scans: each call fails validation or is empty */
    CHECK(memoroid_scan_diag(P(A), 8, P(X), P(S), P(H), NULL, -1, 100, 8, 0, 0, P(W), 1 << 30, NULL) == MEMOROID_EINVAL);
    CHECK(memoroid_scan_diag(P(A), 8, P(X), P(S), P(H), NULL, 2, 0, 8, 0, 0, P(W), 1 << 30, NULL) == MEMOROID_OK);
    CHECK(memoroid_scan_diag(P(A), 8, P(X), P(S), P(X), NULL, 2, 100, 8, 0, 0, P(W), 1 << 30, NULL) == MEMOROID_EINVAL);
    CHECK(memoroid_scan_diag(P(A), 8, P(X), P(S), P(H), NULL, 2, 100, 8, 0, 0, NULL, 0, NULL) == MEMOROID_EWORKSPACE);
    CHECK(memoroid_scan_diag(P(A), 8, P(X), P(S), P(H), NULL, (int64_t)1 << 40, (int64_t)1 << 40, 8, 0, 0, P(W),
                             1 << 30, NULL) == MEMOROID_EINVAL);
    CHECK(memoroid_scan_diag_prepared(P(A), 3, P(X), P(S), P(H), NULL, 2, 100, 8, 0, 0, P(W), 1 << 30, NULL) ==
          MEMOROID_EINVAL);
    CHECK(memoroid_scan_diag_noalloc(P(A), 512, P(X), P(S), P(H), NULL, 64, 65536, 512, MEMOROID_BF16, MEMOROID_BF16,
                                     NULL) == MEMOROID_EWORKSPACE);
    CHECK(memoroid_scan_diag_noalloc(P(A), 8, P(X), P(S), P(H), NULL, INT64_MAX, 2, 8, 0, 0, NULL) == MEMOROID_EINVAL);
    CHECK(memoroid_scan_diag_bwd(P(A), 8, P(S), P(H), P(X), P(X), NULL, 1, 50, 8, 0, P(W), 1 << 30, NULL) ==
          MEMOROID_EINVAL);
    CHECK(memoroid_scan_diag_bwd_prepared(P(A), 8, P(S), P(H), P(X), P(I), NULL, 1, 50, 8, MEMOROID_BF16, P(W),
                                          1 << 30, NULL) == MEMOROID_EUNSUPPORTED);
    /* FFM */
    CHECK(memoroid_scan_ffm(P(A), P(X), P(S), P(H), P(I + 4), NULL, 2, 100, 4, 3, P(W), 1 << 30, NULL) ==
          MEMOROID_EINVAL);
    CHECK(memoroid_scan_ffm_prepared(P(A), P(X), P(S), P(H), P(I), NULL, 2, 100, (int64_t)1 << 32,
                                     (int64_t)1 << 32, P(W), 1 << 30, NULL) == MEMOROID_EINVAL);
    CHECK(memoroid_scan_ffm_bwd(P(A), P(X), P(S), P(H), P(I), P(0x90000), NULL, NULL, 1, 100, 4, 3, P(W), 1 << 30,
                                NULL) == MEMOROID_EUNSUPPORTED);
    CHECK(memoroid_scan_ffm_bwd_prepared(P(A), P(X), P(S), NULL, P(I), P(0x90000), P(0xA0000), NULL, 1, 100, 4, 4,
                                         P(W), 1 << 30, NULL) == MEMOROID_EINVAL);
    /* linear attention */
    CHECK(memoroid_scan_linattn(P(A), P(X), P(S), P(H), P(I), NULL, 1000, 4, 32, 64, 64, P(W), 1 << 30, NULL) ==
          MEMOROID_EUNSUPPORTED);
    CHECK(memoroid_scan_linattn(P(A), P(X), P(S), P(H), P(A), NULL, 1000, 4, 64, 64, 64, P(W), 1 << 30, NULL) ==
          MEMOROID_EINVAL);
    CHECK(memoroid_scan_linattn_bwd(P(A), P(X), P(S), P(H), P(I), P(W), P(A), P(0xA0000), P(0xB0000), 1000, 4, 64,
                                    64, 64, P(0xC0000), 1 << 30, NULL) == MEMOROID_EINVAL);
    /* return, GAE */
    CHECK(memoroid_discounted_return(P(A), P(S), 1.5f, P(H), 2, 100, P(W), 1 << 30, NULL) == MEMOROID_EINVAL);
    CHECK(memoroid_discounted_return_prepared(P(A), P(S), 0.9f, P(A), 2, 100, P(W), 1 << 30, NULL) == MEMOROID_EINVAL);
    CHECK(memoroid_gae(P(A), P(X), NULL, NULL, P(S), 0.99f, 2.0f, P(H), NULL, 2, 100, P(W), 1 << 30, NULL) ==
          MEMOROID_EINVAL);
    CHECK(memoroid_gae_prepared(P(A), P(X), NULL, NULL, P(S), 0.99f, 0.95f, P(H), P(H), 2, 100, P(W), 1 << 30,
                                NULL) == MEMOROID_EINVAL);
    /* TBB */
    CHECK(memoroid_tbb_begin_indices(P(S), (int64_t)1 << 31, 0, P(I), P(A), P(W), 1 << 30, NULL) ==
          MEMOROID_EUNSUPPORTED);
    CHECK(memoroid_tbb_begin_indices_prepared(P(S), 1000, INT64_MAX, P(I), P(A), P(W), 1 << 30, NULL) ==
          MEMOROID_EINVAL);
    CHECK(memoroid_tbb_sample(P(A), 1000, 64, P(X), 10, P(S), 100, (int64_t)1 << 62, P(H), P(I), NULL, NULL, P(W),
                              1 << 30, NULL) == MEMOROID_EINVAL);
    CHECK(memoroid_tbb_sample_prepared(P(A), 1000, 64, P(X), 10, P(S), ((int64_t)1 << 24) + 1, 500, P(H), P(I), NULL,
                                       NULL, P(W), 1 << 30, NULL) == MEMOROID_EUNSUPPORTED);
    /* workspace helpers and strings */
    CHECK(memoroid_workspace_prepare(NULL, 4096, NULL) == MEMOROID_EINVAL);
    CHECK(memoroid_workspace_status(NULL, 4096, NULL) == MEMOROID_EINVAL);
    for (int s = -10; s <= 3; ++s) CHECK(memoroid_status_string(s) != NULL && strlen(memoroid_status_string(s)) > 0);
    CHECK(memoroid_abi_version() == MEMOROID_ABI_VERSION);
    CHECK(memoroid_testing_set_fallback_polls(7) == 4096 && memoroid_testing_set_fallback_polls(-1) == 7);
    printf("validation done\n");
    return 0;
}
