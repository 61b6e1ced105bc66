/* Host-side checks of every libxred entry point, built against a copy of
 * the library whose host code is compiled with AddressSanitizer: argument
 * arrays are heap blocks of exactly the size the call may read, so a read
 * past one (srcs[nsrc], items[nitems], ...) is reported.  Every call here
 * either fails validation or, with valid-looking arguments, fails at its
 * first HIP runtime call because no GPU is visible; the program refuses to
 * run when a GPU is visible, since its pointers are not real device memory. */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "xred.h"

static int failures = 0;

#define EXPECT(call, want)                                                                \
    do {                                                                                  \
        xred_status got_ = (call);                                                        \
        if (got_ != (want)) {                                                             \
            fprintf(stderr, "line %d: %s returned %d (%s), expected %d: %s\n", __LINE__, #call, \
                    (int)got_, xred_status_string(got_), (int)(want), xred_last_error());  \
            ++failures;                                                                   \
        }                                                                                 \
    } while (0)

/* a fake, suitably aligned device address: never dereferenced on the host */
static void *fake(uintptr_t k) { return (void *)(uintptr_t)(0x7f0000000000ull + k * 0x1000000ull); }

static const void **ptrs(int n, uintptr_t first)
{
    const void **p = malloc(sizeof(void *) * (size_t)(n > 0 ? n : 1));
    for (int i = 0; i < n; ++i) p[i] = fake(first + (uintptr_t)i);
    return p;
}

int main(void)
{
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) == hipSuccess && ndev > 0) {
        printf("skipped: a GPU is visible\n");
        return 0;
    }
    const xred_status NODEV = XRED_HIP_ERROR;

    /* xred_allreduce_local */
    const void **s8 = ptrs(8, 1), **s64 = ptrs(64, 1);
    EXPECT(xred_allreduce_local(s8, 0, fake(0), 16, XRED_FLOAT32, XRED_SUM, NULL), XRED_INVALID_ARGUMENT);
    EXPECT(xred_allreduce_local(s64, 65, fake(0), 16, XRED_FLOAT32, XRED_SUM, NULL), XRED_INVALID_ARGUMENT);
    EXPECT(xred_allreduce_local(NULL, 8, fake(0), 16, XRED_FLOAT32, XRED_SUM, NULL), XRED_INVALID_ARGUMENT);
    EXPECT(xred_allreduce_local(NULL, 8, fake(0), 0, XRED_FLOAT32, XRED_SUM, NULL), XRED_SUCCESS);
    EXPECT(xred_allreduce_local(s8, 8, NULL, 16, XRED_FLOAT32, XRED_SUM, NULL), XRED_INVALID_ARGUMENT);
    EXPECT(xred_allreduce_local(s8, 8, (char *)fake(0) + 2, 16, XRED_FLOAT32, XRED_SUM, NULL),
           XRED_INVALID_ARGUMENT);
    EXPECT(xred_allreduce_local(s8, 8, fake(0), 16, (xred_dtype)99, XRED_SUM, NULL), XRED_INVALID_ARGUMENT);
    EXPECT(xred_allreduce_local(s8, 8, fake(0), 16, XRED_FLOAT32, (xred_op)99, NULL), XRED_INVALID_ARGUMENT);
    EXPECT(xred_allreduce_local(s8, 8, fake(0), 16, XRED_INT32, XRED_AVG, NULL), XRED_UNSUPPORTED);
    EXPECT(xred_allreduce_local(s8, 8, fake(0), SIZE_MAX / 2, XRED_FLOAT32, XRED_SUM, NULL),
           XRED_INVALID_ARGUMENT);
    EXPECT(xred_allreduce_local(s8, 8, (char *)s8[3] + 16, 16, XRED_FLOAT32, XRED_SUM, NULL), XRED_ALIAS);
    EXPECT(xred_allreduce_local(s8, 8, fake(0), 16, XRED_BFLOAT16, XRED_SUM, NULL), NODEV);
    EXPECT(xred_allreduce_local(s64, 64, fake(0), 1000, XRED_INT64, XRED_MAX, NULL), NODEV);

    /* xred_reduce_scatter_local */
    EXPECT(xred_reduce_scatter_local(s8, 8, 8, fake(0), 16, XRED_FLOAT32, XRED_SUM, NULL),
           XRED_INVALID_ARGUMENT);
    EXPECT(xred_reduce_scatter_local(s8, 8, -1, fake(0), 16, XRED_FLOAT32, XRED_SUM, NULL),
           XRED_INVALID_ARGUMENT);
    EXPECT(xred_reduce_scatter_local(s8, 8, 0, fake(0), SIZE_MAX / 16, XRED_FLOAT32, XRED_SUM, NULL),
           XRED_INVALID_ARGUMENT);
    EXPECT(xred_reduce_scatter_local(s8, 8, 2, (char *)s8[1] + 2 * 64 + 4, 16, XRED_FLOAT32,
                                     XRED_SUM, NULL), XRED_ALIAS);
    EXPECT(xred_reduce_scatter_local(s8, 8, 2, fake(0), 16, XRED_FLOAT32, XRED_SUM, NULL), NODEV);

    /* xred_reduce_copy_step and xred_acc_cast */
    EXPECT(xred_reduce_copy_step(fake(1), fake(2), fake(3), 16, XRED_BFLOAT16, XRED_SUM, 4u, NULL),
           XRED_INVALID_ARGUMENT);
    EXPECT(xred_reduce_copy_step(fake(1), fake(2), fake(3), 16, XRED_BFLOAT16, XRED_AVG, 0u, NULL),
           XRED_UNSUPPORTED);
    EXPECT(xred_reduce_copy_step(fake(1), (char *)fake(1) + 16, fake(3), 16, XRED_BFLOAT16, XRED_SUM,
                                 0u, NULL), XRED_ALIAS);
    EXPECT(xred_reduce_copy_step(fake(1), fake(2), fake(3), 16, XRED_BFLOAT16, XRED_SUM,
                                 XRED_STEP_INIT | XRED_STEP_FINAL, NULL), NODEV);
    EXPECT(xred_acc_cast(fake(2), (char *)fake(2) + 8, 16, XRED_BFLOAT16, NULL), XRED_ALIAS);
    EXPECT(xred_acc_cast(fake(2), fake(3), 16, XRED_BFLOAT16, NULL), NODEV);

    /* xred_batched_reduce with host descriptors: exact-size arrays */
    enum { K = 3000 };
    xred_item *items = malloc(sizeof(xred_item) * K);
    const void ***rows = malloc(sizeof(void *) * K);
    for (int k = 0; k < K; ++k) {
        const int P = 1 + k % 9;
        rows[k] = ptrs(P, 100 + (uintptr_t)k * 10);
        items[k].srcs = rows[k];
        items[k].dst = fake(50000 + (uintptr_t)k);
        items[k].count = 1 + (uint64_t)(k * 977) % 300000;
        items[k].nsrc = (uint32_t)P;
        items[k].reserved = 0;
    }
    EXPECT(xred_batched_reduce(items, K, XRED_BFLOAT16, XRED_SUM, 0u, NULL), NODEV);
    EXPECT(xred_batched_reduce(items, -1, XRED_BFLOAT16, XRED_SUM, 0u, NULL), XRED_INVALID_ARGUMENT);
    EXPECT(xred_batched_reduce(items, K, XRED_BFLOAT16, XRED_SUM, 8u, NULL), XRED_INVALID_ARGUMENT);
    EXPECT(xred_batched_reduce(NULL, K, XRED_BFLOAT16, XRED_SUM, 0u, NULL), XRED_INVALID_ARGUMENT);
    EXPECT(xred_batched_reduce(items, 0, XRED_BFLOAT16, XRED_SUM, 0u, NULL), XRED_SUCCESS);
    items[K - 1].reserved = 1;
    EXPECT(xred_batched_reduce(items, K, XRED_BFLOAT16, XRED_SUM, 0u, NULL), XRED_INVALID_ARGUMENT);
    items[K - 1].reserved = 0;
    items[17].nsrc = 0;
    EXPECT(xred_batched_reduce(items, K, XRED_BFLOAT16, XRED_SUM, 0u, NULL), XRED_INVALID_ARGUMENT);
    items[17].nsrc = 1 + 17 % 9;
    items[18].srcs = NULL;
    EXPECT(xred_batched_reduce(items, K, XRED_BFLOAT16, XRED_SUM, 0u, NULL), XRED_INVALID_ARGUMENT);
    items[18].srcs = rows[18];
    items[19].dst = (char *)rows[19][0] + 2;
    EXPECT(xred_batched_reduce(items, K, XRED_BFLOAT16, XRED_SUM, 0u, NULL), XRED_ALIAS);
    items[19].dst = fake(50000 + 19);
    items[20].count = SIZE_MAX / 2;
    EXPECT(xred_batched_reduce(items, K, XRED_BFLOAT16, XRED_SUM, 0u, NULL), XRED_INVALID_ARGUMENT);
    items[20].count = 5;
    EXPECT(xred_batched_reduce((const xred_item *)((char *)items + 4), 2, XRED_BFLOAT16, XRED_SUM,
                               XRED_ITEMS_ON_DEVICE, NULL), XRED_INVALID_ARGUMENT);

    /* xred_batched_reduce_noalloc (device descriptors: never read on the host) */
    EXPECT(xred_batched_reduce_noalloc((const xred_item *)fake(9), 16385, XRED_BFLOAT16, XRED_SUM,
                                       NULL), XRED_UNSUPPORTED);
    EXPECT(xred_batched_reduce_noalloc((const xred_item *)fake(9), -1, XRED_BFLOAT16, XRED_SUM, NULL),
           XRED_INVALID_ARGUMENT);
    EXPECT(xred_batched_reduce_noalloc((const xred_item *)((char *)fake(9) + 4), 5, XRED_BFLOAT16,
                                       XRED_SUM, NULL), XRED_INVALID_ARGUMENT);

    /* xred_ring_reduce */
    const void **c16 = ptrs(16, 200);
    EXPECT(xred_ring_reduce(c16, 0, fake(0), 1024, XRED_BFLOAT16, XRED_SUM, NULL, 0, 0, NULL, NULL),
           XRED_INVALID_ARGUMENT);
    const void **c16b = ptrs(16, 200);
    c16b[5] = (const char *)c16b[5] + 2;   /* one chunk at another offset within 16 bytes */
    EXPECT(xred_ring_reduce(c16b, 16, fake(0), 1024, XRED_BFLOAT16, XRED_SUM, NULL, 0, 0, NULL,
                            NULL), XRED_UNSUPPORTED);
    EXPECT(xred_ring_reduce(c16, 16, fake(0), 1024, XRED_BFLOAT16, XRED_SUM,
                            (const uint32_t *)((char *)fake(7) + 2), 0, 0, NULL, NULL),
           XRED_INVALID_ARGUMENT);
    EXPECT(xred_ring_reduce(c16, 16, fake(0), 1024, XRED_BFLOAT16, XRED_AVG, NULL, 0, 0, NULL, NULL),
           XRED_UNSUPPORTED);
    {
        /* valid arguments: capacity is unknown without a device */
        const xred_status st =
            xred_ring_reduce(c16, 16, fake(0), 1024, XRED_BFLOAT16, XRED_SUM, NULL, 0, 0, NULL, NULL);
        if (st != NODEV && st != XRED_UNSUPPORTED) {
            fprintf(stderr, "ring with valid arguments returned %d\n", (int)st);
            ++failures;
        }
    }

    /* xred_allreduce_sim */
    const void **send = ptrs(8, 300);
    void **recv = (void **)ptrs(8, 400);
    EXPECT(xred_allreduce_sim(send, recv, 3, 1024, XRED_BFLOAT16, XRED_SUM, XRED_SCHEDULE_RHD, NULL),
           XRED_INVALID_ARGUMENT);
    EXPECT(xred_allreduce_sim(send, recv, 8, 1024, XRED_BFLOAT16, XRED_SUM, (xred_schedule)9, NULL),
           XRED_INVALID_ARGUMENT);
    recv[5] = (char *)send[2] + 64;
    EXPECT(xred_allreduce_sim(send, recv, 8, 1024, XRED_BFLOAT16, XRED_SUM, XRED_SCHEDULE_RING, NULL),
           XRED_ALIAS);
    recv[5] = fake(405);
    EXPECT(xred_allreduce_sim(send, recv, 8, 1024, XRED_BFLOAT16, XRED_SUM, XRED_SCHEDULE_RING, NULL),
           NODEV);

    /* the rest of the interface */
    for (int s = -1; s <= 6; ++s)
        if (xred_status_string((xred_status)s) == NULL) ++failures;
    if (xred_version() <= 0) ++failures;
    if (xred_acc_elem_size(XRED_INT64) != 8 || xred_acc_elem_size((xred_dtype)99) != 0) ++failures;
    if (xred_sim_chunk(1000, 8) == 0 || xred_sim_chunk(1000, 0) != 0) ++failures;
    /* CU partition: slot checks first, then the device query fails */
    void *ps = (void *)1, *pr = (void *)1;
    EXPECT(xred_stream_create_partition(16, NULL, &pr), XRED_INVALID_ARGUMENT);
    EXPECT(xred_stream_create_partition(0, &ps, &pr), XRED_INVALID_ARGUMENT);
    if (ps != NULL || pr != NULL) ++failures;
    ps = (void *)1;
    EXPECT(xred_stream_create_partition(16, &ps, NULL), NODEV);
    if (ps != NULL) ++failures;
    EXPECT(xred_stream_destroy(NULL), XRED_INVALID_ARGUMENT);
    const unsigned prev = xred_set_max_workgroups(7);
    if (xred_set_max_workgroups(prev) != 7) ++failures;
    xred_release();

    for (int k = 0; k < K; ++k) free((void *)rows[k]);
    free(rows);
    free(items);
    free((void *)s8);
    free((void *)s64);
    free((void *)c16);
    free((void *)send);
    free(recv);
    if (failures) {
        fprintf(stderr, "%d checks failed\n", failures);
        return 1;
    }
    printf("all host checks passed\n");
    return 0;
}
