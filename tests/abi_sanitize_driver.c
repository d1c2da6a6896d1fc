/*
 * Test driver: calls the library's host-side entry points that need no GPU (workspace sizes,
 * status strings, every argument check that returns before a launch) with valid and invalid
 * arguments.  The test that builds it compiles the library's host code and this driver under
 * AddressSanitizer and UndefinedBehaviorSanitizer; device pointers passed here are never
 * dereferenced.  Prints "done" on success.
 */
#include <stddef.h>
#include <stdint.h>
#include <stdio.h>

#include "tt.h"

#define EXPECT(cond)                                          \
    do {                                                      \
        if (!(cond)) {                                        \
            printf("failed: %s (line %d)\n", #cond, __LINE__); \
            return 1;                                         \
        }                                                     \
    } while (0)

int main(void) {
    int32_t *const D = (int32_t *)0x1000; /* never dereferenced */
    float *const F = (float *)0x1000;
    void *const W = (void *)0x1000;
    size_t n = 0;
    for (int s = -6; s <= 2; ++s) EXPECT(tt_status_string(s) != NULL);
    EXPECT(tt_version() >= 100);
    EXPECT(tt_verify_workspace_size(256, 151936, &n) == TT_OK && n > 0);
    EXPECT(tt_verify_workspace_size(-1, 10, &n) == TT_EINVAL);
    EXPECT(tt_align_workspace_size(1024, 512, 512, 8, 8, &n) == TT_OK && n > 0);
    EXPECT(tt_align_workspace_size(8, 4096, 4096, -1, 16, &n) == TT_EUNSUPPORTED);
    EXPECT(tt_step_workspace_size(256, 151936, 8, 30, 8, 8, &n) == TT_OK);
    EXPECT(tt_token_index_size(151936, &n) == TT_OK && n == 16u * (1u << 20) + (1u << 20) / 4u);
    EXPECT(tt_retokenize_workspace_size(4, 0, &n) == TT_EINVAL);

    tt_vocab v = {(const uint8_t *)0x1000, D, 10, 8};
    tt_vocab big = {(const uint8_t *)0x1000, D, 10, 65};
    EXPECT(tt_align(NULL, &v, 1, D, D, D, D, 4, 4, 8, D, D, D, D, NULL, 0, NULL) == TT_EINVAL);
    EXPECT(tt_align(&big, &v, 1, D, D, D, D, 4, 4, 8, D, D, D, D, NULL, 0, NULL) == TT_EUNSUPPORTED);
    EXPECT(tt_align(&v, &v, 0, NULL, NULL, NULL, NULL, 4, 4, 8, NULL, NULL, NULL, NULL, NULL, 0, NULL) == TT_OK);
    EXPECT(tt_transfer(1, 10, D, D, D, D, F, 5, F, NULL) == TT_EINVAL);
    EXPECT(tt_verify(1, 10, D, D, F, F, 9, F, F, 4, D, D, NULL, W, 1 << 20, NULL) == TT_EINVAL);
    EXPECT(tt_verify(1, 10, D, D, F, F, 10, F, F, 4, D, D, NULL, W, 0, NULL) == TT_EWORKSPACE);
    EXPECT(tt_verify_dense(1, 10, D, D, F, 9, F, 10, F, F, 4, D, D, NULL, W, 1 << 20, NULL) == TT_EINVAL);
    EXPECT(tt_verify_dense(1, 10, D, D, F, 10, F, 10, F, F, 4, D, D, NULL, W, 0, NULL) == TT_EWORKSPACE);
    EXPECT(tt_step(&v, &v, 1, 10, 10, D, D, D, D, 4, 0, 8, F, 10, F, 10, F, F, D, D, D, D, F, D, D, NULL, W,
                   1 << 30, NULL) == TT_EINVAL);
    EXPECT(tt_step(&v, &v, 1, 10, 10, D, D, D, D, 4, 4, 8, F, 10, F, 10, F, F, D, D, D, D, F, D, D, NULL, W, 16,
                   NULL) == TT_EWORKSPACE);
    EXPECT(tt_delta_histogram(1, D, D, D, D, 0, D, NULL) == TT_EINVAL);
    EXPECT(tt_delta_quantile(D, 0, 9, 10, D, NULL) == TT_EINVAL);
    EXPECT(tt_delta_quantile(D, 8, 11, 10, D, NULL) == TT_EINVAL);
    EXPECT(tt_token_index_build(&big, W, 1 << 30, NULL) == TT_EUNSUPPORTED);
    EXPECT(tt_token_index_build(&v, (void *)0x1004, 1 << 30, NULL) == TT_EINVAL);
    EXPECT(tt_retokenize(&v, &v, W, 1 << 20, 1, D, D, 0, 16, D, D, W, 1 << 20, NULL) == TT_EINVAL);
    EXPECT(tt_retokenize(&v, &v, W, 1 << 20, 1, D, D, 64, 16, D, D, W, 4, NULL) == TT_EWORKSPACE);
    EXPECT(tt_vocab_intersection(&v, W, 1 << 20, &v, W, 16, D, D, NULL) == TT_EINVAL);
    EXPECT(tt_vocab_intersection(&big, W, 1 << 20, &v, W, 1 << 20, D, D, NULL) == TT_EUNSUPPORTED);
    EXPECT(tt_tli_proposal(1, 10, 10, D, D, F, 9, F, 10, NULL) == TT_EINVAL);
    EXPECT(tt_tli_proposal(0, 10, 10, NULL, NULL, NULL, 10, NULL, 10, NULL) == TT_OK);
    EXPECT(tt_verify_logits(1, 10, D, D, F, (const uint16_t *)W, 9, F, NULL, F, F, 4, D, D, NULL) == TT_EINVAL);
    EXPECT(tt_verify_logits(0, 10, NULL, NULL, NULL, NULL, 10, NULL, NULL, NULL, NULL, 4, NULL, NULL, NULL) ==
           TT_OK);
    EXPECT(tt_verify_tli(1, 10, 12, D, D, D, D, F, 9, NULL, F, 12, F, F, 4, D, D, NULL) == TT_EINVAL);
    EXPECT(tt_verify_tli(0, 10, 12, NULL, NULL, NULL, NULL, NULL, 10, NULL, NULL, 12, NULL, NULL, 4, NULL, NULL,
                         NULL) == TT_OK);
    printf("done\n");
    return 0;
}
