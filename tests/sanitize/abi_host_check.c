/*
 * abi_host_check.c -- host-side checks of the C ABI (include/pardnn.h) for a
 * build of the library's HOST code with AddressSanitizer and
 * UndefinedBehaviorSanitizer (no device code is built), run where no GPU is
 * visible: every entry point with a NULL handle, argument checks that come
 * before any device call, the status strings and the per-thread error text,
 * the allocation-failure hook (PARDNN_FAULT_ALLOC) and the no-device path.
 * Exit status 0 when every check holds; a sanitizer finding aborts.
 */
#define _POSIX_C_SOURCE 200112L   /* setenv, unsetenv */

#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "pardnn.h"

static int n_failed = 0;

#define EXPECT(cond)                                                         \
    do {                                                                     \
        if (!(cond)) {                                                       \
            fprintf(stderr, "check failed (line %d): %s\n", __LINE__, #cond); \
            n_failed++;                                                      \
        }                                                                    \
    } while (0)

int main(void)
{
    pardnn_graph *h = NULL;
    int32_t src[2] = {0, 1}, dst[2] = {1, 2};
    int64_t w[3] = {1, 1, 1};

    /* status strings: static text for every code, "unknown status" beyond */
    EXPECT(strcmp(pardnn_status_string(PARDNN_OK), "ok") == 0);
    for (int s = -8; s <= 3; s++) EXPECT(pardnn_status_string(s) != NULL);
    EXPECT(strcmp(pardnn_status_string(12345), "unknown status") == 0);

    /* create: argument checks come before any device call */
    EXPECT(pardnn_graph_create(3, 2, NULL, dst, w, w, w, NULL, &h) == PARDNN_E_INVAL);
    EXPECT(h == NULL);
    EXPECT(pardnn_graph_create(3, 2, src, NULL, w, w, w, NULL, &h) == PARDNN_E_INVAL);
    EXPECT(pardnn_graph_create(3, 2, src, dst, w, NULL, w, NULL, &h) == PARDNN_E_INVAL);
    EXPECT(pardnn_graph_create(3, 2, src, dst, NULL, w, w, NULL, &h) == PARDNN_E_INVAL);
    EXPECT(pardnn_graph_create(3, 2, src, dst, w, w, NULL, NULL, &h) == PARDNN_E_INVAL);
    EXPECT(pardnn_graph_create(-1, 0, NULL, NULL, NULL, NULL, NULL, NULL, &h) == PARDNN_E_INVAL);
    EXPECT(pardnn_graph_create(0, -1, NULL, NULL, NULL, NULL, NULL, NULL, &h) == PARDNN_E_INVAL);
    EXPECT(pardnn_graph_create(0, 0, NULL, NULL, NULL, NULL, NULL, NULL, NULL) == PARDNN_E_INVAL);
    EXPECT(pardnn_graph_create(PARDNN_MAX_NODES + 1, 0, NULL, NULL, NULL, NULL, NULL, NULL, &h) ==
           PARDNN_E_INVAL);
    EXPECT(strstr(pardnn_last_error(), "2^26") != NULL);
    EXPECT(pardnn_graph_create(4, (int64_t)PARDNN_MAX_EDGES + 1, src, dst, w, w, w, NULL, &h) ==
           PARDNN_E_INVAL);

    /* the allocation-failure hook: the handle is the first allocation */
    setenv("PARDNN_FAULT_ALLOC", "1", 1);
    EXPECT(pardnn_graph_create(3, 2, src, dst, w, w, w, NULL, &h) == PARDNN_E_NOMEM);
    EXPECT(h == NULL);
    EXPECT(strstr(pardnn_last_error(), "host allocation") != NULL);
    unsetenv("PARDNN_FAULT_ALLOC");

    /* no GPU visible: E_DEVICE, no handle, nothing leaked */
    EXPECT(pardnn_graph_create(3, 2, src, dst, w, w, w, NULL, &h) == PARDNN_E_DEVICE);
    EXPECT(h == NULL);
    EXPECT(strlen(pardnn_last_error()) > 0);

    /* every entry point refuses a NULL handle (destroy: a no-op) */
    int32_t i32[4] = {0, 0, 0, 0};
    int64_t i64[4] = {0, 0, 0, 0};
    uint8_t u8[4] = {0, 0, 0, 0};
    const char *name = NULL;
    float ms = 0.f;
    pardnn_info info;
    EXPECT(pardnn_graph_destroy(NULL) == PARDNN_OK);
    EXPECT(pardnn_set_stream(NULL, NULL) == PARDNN_E_INVAL);
    EXPECT(pardnn_get_info(NULL, &info) == PARDNN_E_INVAL);
    EXPECT(pardnn_levelize(NULL, i32, i32, i32, i32) == PARDNN_E_INVAL);
    EXPECT(pardnn_tb_levels(NULL, i32, i64, i64, i64) == PARDNN_E_INVAL);
    EXPECT(pardnn_critical_path(NULL, i32, i64, i64, i64, u8, i32, i32) == PARDNN_E_INVAL);
    EXPECT(pardnn_label_memory(NULL, i32, 1, i64, i64, i64) == PARDNN_E_INVAL);
    EXPECT(pardnn_apply_moves(NULL, i32, 1, i32, i32) == PARDNN_E_INVAL);
    EXPECT(pardnn_build_placements(NULL, i32, 1, i64, 1, i32, i32, i32) == PARDNN_E_INVAL);
    EXPECT(pardnn_evaluate_batch(NULL, 1, i32, 1, i64, i64, i64, i64, u8, i32, 1, i32, i64,
                                 i64) == PARDNN_E_INVAL);
    EXPECT(pardnn_evaluate_batch_fixed(NULL, 1, i32, 1, i64, i64, i64, i64, u8, i32, 1, i32,
                                       i64, i64) == PARDNN_E_INVAL);
    EXPECT(pardnn_evaluate_moves(NULL, i32, 1, i64, 1, i32, i32, 1, i64, i64, i64, i64, u8, i32,
                                 1, i32, i64, i64) == PARDNN_E_INVAL);
    EXPECT(pardnn_memory_balance(NULL, 1, i32, i32, i32, 1, i64, i64, u8, i64) ==
           PARDNN_E_INVAL);
    EXPECT(pardnn_cluster_criticality(NULL, i32, 1, i64, i32) == PARDNN_E_INVAL);
    EXPECT(pardnn_span_work(NULL, i32, 1, i32, 1, i64, i64, i64, i64, i64, i32) ==
           PARDNN_E_INVAL);
    EXPECT(pardnn_slice_primaries(NULL, 1, i32, i32, 1, i32, i64) == PARDNN_E_INVAL);
    EXPECT(pardnn_slice_graph(NULL, 1, i32, i32, i32, i32, i64) == PARDNN_E_INVAL);
    EXPECT(pardnn_tb_levels_batch(NULL, 1, i32, i64, i64, i64) == PARDNN_E_INVAL);
    EXPECT(pardnn_set_timing(NULL, 1) == PARDNN_E_INVAL);
    EXPECT(pardnn_get_timing(NULL, &name, &ms) == PARDNN_E_INVAL);
    EXPECT(pardnn_set_deferred_errors(NULL, 1) == PARDNN_E_INVAL);
    EXPECT(pardnn_take_errors(NULL) == PARDNN_E_INVAL);
    EXPECT(strstr(pardnn_last_error(), "null") != NULL);

    /* many failing calls: the error text is replaced, never accumulated */
    for (int k = 0; k < 10000; k++) (void)pardnn_tb_levels(NULL, NULL, NULL, NULL, NULL);
    EXPECT(strlen(pardnn_last_error()) < 256);

    if (n_failed) fprintf(stderr, "%d check(s) failed\n", n_failed);
    else printf("abi host checks: all passed\n");
    return n_failed ? 1 : 0;
}
