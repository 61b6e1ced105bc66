/* A plain C caller of libxred: four fp32 sources of small integers (so every
 * binary32 sum is exact) reduced with xred_allreduce_local through the HIP C
 * runtime API, checked element by element; then one rejected call (a
 * partially overlapping output) that must leave the stream untouched. */
#include <stdio.h>
#include <stdlib.h>

#include <hip/hip_runtime_api.h>

#include "xred.h"

#define P 4
#define N 100003

static int fail_hip(hipError_t e, const char *what)
{
    fprintf(stderr, "%s: %s\n", what, hipGetErrorString(e));
    return 1;
}

int main(void)
{
    float *host = malloc(sizeof(float) * (size_t)N * P);
    float *res = malloc(sizeof(float) * N);
    void *dev[P];
    void *out = NULL;
    hipError_t e;
    if (!host || !res) return 1;
    for (int p = 0; p < P; ++p)
        for (int i = 0; i < N; ++i) host[(size_t)p * N + i] = (float)((i * 7 + p * 13) % 101 - 50);
    for (int p = 0; p < P; ++p) {
        if ((e = hipMalloc(&dev[p], sizeof(float) * N)) != hipSuccess) return fail_hip(e, "hipMalloc");
        if ((e = hipMemcpy(dev[p], host + (size_t)p * N, sizeof(float) * N, hipMemcpyHostToDevice)) !=
            hipSuccess)
            return fail_hip(e, "hipMemcpy");
    }
    if ((e = hipMalloc(&out, sizeof(float) * N)) != hipSuccess) return fail_hip(e, "hipMalloc");

    xred_status st = xred_allreduce_local((const void *const *)dev, P, out, N, XRED_FLOAT32,
                                          XRED_SUM, NULL);
    if (st != XRED_SUCCESS) {
        fprintf(stderr, "xred_allreduce_local: %s (%s)\n", xred_status_string(st), xred_last_error());
        return 1;
    }
    if ((e = hipMemcpy(res, out, sizeof(float) * N, hipMemcpyDeviceToHost)) != hipSuccess)
        return fail_hip(e, "hipMemcpy");
    for (int i = 0; i < N; ++i) {
        float want = 0.0f;
        for (int p = 0; p < P; ++p) want += host[(size_t)p * N + i];
        if (res[i] != want) {
            fprintf(stderr, "element %d: got %g, expected %g\n", i, res[i], want);
            return 1;
        }
    }

    st = xred_allreduce_local((const void *const *)dev, P, (char *)dev[0] + 4, N - 1,
                              XRED_FLOAT32, XRED_SUM, NULL);
    if (st != XRED_ALIAS) {
        fprintf(stderr, "overlapping output: got status %d, expected XRED_ALIAS\n", (int)st);
        return 1;
    }
    printf("libxred %d: %d x %d fp32 sum exact; overlap rejected: %s\n", xred_version(), P, N,
           xred_last_error());
    for (int p = 0; p < P; ++p) (void)hipFree(dev[p]);
    (void)hipFree(out);
    free(host);
    free(res);
    return 0;
}
