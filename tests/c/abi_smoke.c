/* A C99 client of libreshard.so using only include/reshard.h: plans the
 * fp16 (2, 64, 1024) reshard from mesh (4,8) "R R S^{01}" to mesh (4,8)
 * "R S^1 R", checks the plan totals, runs it through the host interpreter
 * on host buffers filled with each element's linear index, checks every
 * destination element, and checks the error paths.  No GPU is used.
 * Prints "ok" and exits 0 on success. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "reshard.h"

#define CHECK(c)                                                                  \
    do {                                                                          \
        if (!(c)) {                                                               \
            fprintf(stderr, "failed: %s (%s)\n", #c, reshard_last_error());       \
            return 1;                                                             \
        }                                                                         \
    } while (0)

int main(void) {
    const int64_t shape[3] = {2, 64, 1024}, mesh[2] = {4, 8};
    reshard_plan_t *plan = NULL;
    CHECK(reshard_plan(3, shape, RESHARD_F16, 2, mesh, "R R S^{01}", 2, mesh, "R S^1 R", 0, &plan) == RESHARD_OK);
    int64_t rd = 0, wr = 0, tasks = 0, descs = 0, fan = 0;
    CHECK(reshard_plan_stats(plan, &rd, &wr, &tasks, &descs, &fan) == RESHARD_OK);
    CHECK(rd == 2 * 64 * 1024 * 2 && wr == 4 * rd && tasks == 256 && fan == 4 && descs > 0);
    CHECK(reshard_plan_alignment(plan) == 16);

    /* source device k = (c0, c1) holds columns [32 * (8 c0 + c1), +32) of every row */
    uint16_t *src[32], *dst[32];
    void *sp[32], *dp[32];
    for (int k = 0; k < 32; ++k) {
        int64_t ls[3], ld[3];
        CHECK(reshard_plan_local_shape(plan, 0, k, ls) == RESHARD_OK);
        CHECK(reshard_plan_local_shape(plan, 1, k, ld) == RESHARD_OK);
        CHECK(ls[0] == 2 && ls[1] == 64 && ls[2] == 32 && ld[0] == 2 && ld[1] == 8 && ld[2] == 1024);
        src[k] = aligned_alloc(16, 2 * 64 * 32 * 2);
        dst[k] = aligned_alloc(16, 2 * 8 * 1024 * 2);
        CHECK(src[k] && dst[k]);
        for (int b = 0; b < 2; ++b)
            for (int s = 0; s < 64; ++s)
                for (int c = 0; c < 32; ++c)
                    src[k][(b * 64 + s) * 32 + c] = (uint16_t)((b * 64 + s) * 1024 + 32 * k + c);
        memset(dst[k], 0xFF, 2 * 8 * 1024 * 2);
        sp[k] = src[k];
        dp[k] = dst[k];
    }
    CHECK(reshard_debug_execute_host(plan, sp, dp) == RESHARD_OK);
    /* destination device k = (c0, c1) holds sequence rows [8 c1, 8 c1 + 8) */
    for (int k = 0; k < 32; ++k)
        for (int b = 0; b < 2; ++b)
            for (int s = 0; s < 8; ++s)
                for (int c = 0; c < 1024; ++c)
                    CHECK(dst[k][(b * 8 + s) * 1024 + c] == (uint16_t)((b * 64 + 8 * (k % 8) + s) * 1024 + c));

    /* errors: a malformed spec, a NULL out pointer, a NULL plan */
    reshard_plan_t *bad = NULL;
    CHECK(reshard_plan(3, shape, RESHARD_F16, 2, mesh, "R Q R", 2, mesh, "R R R", 0, &bad) == RESHARD_EINVAL);
    CHECK(bad == NULL && strlen(reshard_last_error()) > 0);
    CHECK(reshard_plan(3, shape, RESHARD_F16, 2, mesh, "R R R", 2, mesh, "R R R", 0, NULL) == RESHARD_EINVAL);
    CHECK(reshard_execute(NULL, sp, dp, NULL) == RESHARD_EINVAL);
    CHECK(reshard_version() != NULL);
    reshard_plan_destroy(plan);
    reshard_plan_destroy(NULL);
    for (int k = 0; k < 32; ++k) {
        free(src[k]);
        free(dst[k]);
    }
    printf("ok\n");
    return 0;
}
