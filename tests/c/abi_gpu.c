/* End-to-end use of the C ABI from plain C on the GPU (HIP runtime API for memory, no Python):
 * int32 AllReduces on a ring (latency- and bandwidth-optimal), a torus and a ring of 8, and two
 * with the message-contiguous block placement, are checked against exact column sums; congestion
 * loads against 3^k. Exit status 0 on success. */
#include <hip/hip_runtime_api.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "trivance.h"

static int failures = 0;
#define CHECK(cond)                                                                      \
    do {                                                                                 \
        if (!(cond)) {                                                                   \
            fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond);    \
            ++failures;                                                                  \
        }                                                                                \
    } while (0)

static void run_case(int n, const int* dims, int ndims, int variant, unsigned flags,
                     int64_t elems) {
    trivance_plan_t* plan = NULL;
    if (trivance_plan_ex(n, dims, ndims, variant, flags, &plan) != TRIVANCE_OK) {
        CHECK(0);
        return;
    }
    const size_t count = (size_t)n * (size_t)elems;
    int32_t* host = (int32_t*)malloc(count * sizeof(int32_t));
    int64_t* want = (int64_t*)calloc((size_t)elems, sizeof(int64_t));
    uint64_t x = 0x243F6A8885A308D3ull;
    for (size_t i = 0; i < count; ++i) {
        x ^= x << 13;
        x ^= x >> 7;
        x ^= x << 17;
        host[i] = (int32_t)(x % 2001) - 1000;
        want[i % (size_t)elems] += host[i];
    }
    void* dev = NULL;
    CHECK(hipMalloc(&dev, count * sizeof(int32_t)) == hipSuccess);
    CHECK(hipMemcpy(dev, host, count * sizeof(int32_t), hipMemcpyHostToDevice) == hipSuccess);
    CHECK(trivance_allreduce_emulated(dev, n, elems, TRIVANCE_I32, plan, NULL) == TRIVANCE_OK);
    CHECK(hipDeviceSynchronize() == hipSuccess);
    CHECK(hipMemcpy(host, dev, count * sizeof(int32_t), hipMemcpyDeviceToHost) == hipSuccess);
    size_t bad = 0;
    for (size_t i = 0; i < count; ++i)
        if ((int64_t)host[i] != want[i % (size_t)elems]) ++bad;
    if (bad) fprintf(stderr, "n=%d variant=%d: %zu wrong elements\n", n, variant, bad);
    CHECK(bad == 0);
    CHECK(hipFree(dev) == hipSuccess);
    free(host);
    free(want);
    trivance_plan_destroy(plan);
}

int main(void) {
    int ring27[1] = {27}, torus[2] = {9, 9}, ring8[1] = {8};
    run_case(27, ring27, 1, TRIVANCE_LATENCY_OPT, 0u, 64 * 27 * 2 + 4);
    run_case(27, ring27, 1, TRIVANCE_BANDWIDTH_OPT, 0u, 64 * 27 * 3 + 7);
    run_case(81, torus, 2, TRIVANCE_BANDWIDTH_OPT, 0u, 64 * 81 * 2 * 2 + 12);
    run_case(8, ring8, 1, TRIVANCE_BANDWIDTH_OPT, 0u, 64 * 8 * 4 + 3);
    /* the message-contiguous block placement */
    run_case(27, ring27, 1, TRIVANCE_BANDWIDTH_OPT, TRIVANCE_PLACE_BY_SCHEDULE, 64 * 27 * 3 + 7);
    run_case(81, torus, 2, TRIVANCE_BANDWIDTH_OPT, TRIVANCE_PLACE_BY_SCHEDULE, 64 * 81 * 4 + 12);

    /* congestion of the 27-ring, latency-optimal: every directed link carries 3^k in pass k */
    trivance_plan_t* plan = NULL;
    CHECK(trivance_plan(27, ring27, 1, TRIVANCE_LATENCY_OPT, &plan) == TRIVANCE_OK);
    const int64_t need = trivance_congestion(plan, NULL, NULL, 0);
    CHECK(need == 3 * 27 * 2);
    int64_t loads[3 * 27 * 2];
    CHECK(trivance_congestion(plan, NULL, loads, need) == TRIVANCE_OK);
    for (int k = 0, pw = 1; k < 3; ++k, pw *= 3)
        for (int i = 0; i < 27 * 2; ++i) CHECK(loads[k * 27 * 2 + i] == pw);
    trivance_plan_destroy(plan);

    if (failures == 0) printf("abi_gpu ok\n");
    return failures == 0 ? 0 : 1;
}
