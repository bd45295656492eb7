/* Host-only use of the C ABI from plain C (no GPU calls): plans, introspection, partition,
 * byte accounting, the congestion length query and error codes. Exit status 0 on success. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "trivance.h"

static int failures = 0;
#define CHECK(cond)                                                        \
    do {                                                                   \
        if (!(cond)) {                                                     \
            fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                    \
        }                                                                  \
    } while (0)

int main(void) {
    trivance_plan_t* p = NULL;
    int dims[2] = {27, 27};
    CHECK(trivance_plan(729, dims, 2, TRIVANCE_BANDWIDTH_OPT, &p) == TRIVANCE_OK && p != NULL);
    CHECK(trivance_plan_num_steps(p) == 6);
    CHECK(trivance_plan_num_passes(p) == 12);
    int phase, dim, distance;
    CHECK(trivance_plan_step(p, 0, 1, &phase, &dim, &distance) == TRIVANCE_OK);
    CHECK(phase == TRIVANCE_PHASE_REDUCE_SCATTER && dim == 1 && distance == 1);
    CHECK(trivance_plan_step_index(p, 0) == 0);
    CHECK(trivance_plan_step(p, 4, 0, &phase, &dim, &distance) == TRIVANCE_OK);
    CHECK(phase == TRIVANCE_PHASE_REDUCE_SCATTER && dim == 0 && distance == 9);
    CHECK(trivance_plan_step(p, 11, 0, &phase, &dim, &distance) == TRIVANCE_OK);
    CHECK(phase == TRIVANCE_PHASE_ALLGATHER && dim == 0 && distance == 1);
    CHECK(trivance_plan_step_index(p, 11) == 0 && trivance_plan_step_index(p, 6) == 5);
    CHECK(trivance_plan_step_index(p, 12) == TRIVANCE_EINVAL);
    /* 3.5 w E (n - 1) for the bandwidth-optimal variant */
    const int64_t E = 1048576;
    CHECK(2 * trivance_algorithmic_bytes(p, E, TRIVANCE_F32) == 7 * 4 * E * 728);
    int64_t b = -1, e = -1;
    CHECK(trivance_block_range(p, E, 1, -1, &b, &e) == TRIVANCE_OK && b == E / 2 && e == E);
    CHECK(trivance_block_range(p, E, 0, 0, &b, &e) == TRIVANCE_OK && b == 0 && e == 704);
    CHECK(trivance_congestion(p, NULL, NULL, 0) == (int64_t)12 * 729 * 4);
    CHECK(trivance_plan_step(p, 12, 0, &phase, &dim, &distance) == TRIVANCE_EINVAL);
    /* the Sec. 2.1 cost model: Table 2's 104/81 for 27 x 27, 12 alphas, per-pass link bytes */
    {
        trivance_cost_result cr;
        double peaks[12];
        CHECK(trivance_cost_model(p, 729.0 * 2.0, 1.5e-6, 1e-11, peaks, 12, &cr) == TRIVANCE_OK);
        CHECK(cr.passes == 12 && cr.theta > 104.0 / 81.0 - 1e-12 && cr.theta < 104.0 / 81.0 + 1e-12);
        CHECK(cr.latency > 12 * 1.5e-6 - 1e-18 && cr.latency < 12 * 1.5e-6 + 1e-18);
        CHECK(peaks[0] > 243.0 - 1e-9 && peaks[0] < 243.0 + 1e-9); /* m / (D 3) */
        CHECK(trivance_cost_model(p, 1.0, 0.0, 0.0, peaks, 11, &cr) == TRIVANCE_ESIZE);
    }
    trivance_plan_destroy(p);

    /* a ring whose size is not a power of three (Sec. 4.4): two steps at distances 1 and 3 */
    trivance_plan_t* q = NULL;
    CHECK(trivance_plan(8, NULL, 0, TRIVANCE_BANDWIDTH_OPT, &q) == TRIVANCE_OK);
    CHECK(trivance_plan_num_steps(q) == 2);
    CHECK(trivance_plan_step(q, 1, 0, NULL, NULL, &distance) == TRIVANCE_OK && distance == 3);
    trivance_plan_destroy(q);

    /* message-contiguous placement: on a 27-ring block 1 lies at position 9 (digits reversed) */
    trivance_plan_t* pl = NULL;
    CHECK(trivance_plan_ex(27, NULL, 0, TRIVANCE_BANDWIDTH_OPT, TRIVANCE_PLACE_BY_SCHEDULE, &pl) ==
          TRIVANCE_OK);
    CHECK(trivance_block_range(pl, 27 * 64, 0, 1, &b, &e) == TRIVANCE_OK && b == 576 && e == 640);
    trivance_plan_destroy(pl);
    CHECK(trivance_plan_ex(27, NULL, 0, TRIVANCE_LATENCY_OPT, TRIVANCE_PLACE_BY_SCHEDULE, &pl) ==
          TRIVANCE_EUNSUPPORTED);
    CHECK(trivance_plan_ex(27, NULL, 0, TRIVANCE_BANDWIDTH_OPT, 4u, &pl) == TRIVANCE_EINVAL);

    /* errors */
    trivance_plan_t* r = NULL;
    CHECK(trivance_plan(8, NULL, 0, TRIVANCE_BRUCK_REF, &r) == TRIVANCE_EUNSUPPORTED && r == NULL);
    /* the latency-optimal variant on a ring of 8 keeps partials in a workspace (Sec. 4.4) */
    CHECK(trivance_plan(8, NULL, 0, TRIVANCE_LATENCY_OPT, &r) == TRIVANCE_OK && r != NULL);
    CHECK(trivance_plan_num_passes(r) == 2);
    CHECK(trivance_workspace_bytes(r, 100, TRIVANCE_F32) == 2 * 8 * 100 * 4);
    trivance_plan_destroy(r);
    r = NULL;
    CHECK(trivance_plan(80, dims, 2, TRIVANCE_LATENCY_OPT, &r) == TRIVANCE_EINVAL);
    CHECK(trivance_allreduce_emulated(NULL, 9, 0, TRIVANCE_F32, NULL, NULL) == TRIVANCE_EINVAL);
    CHECK(strcmp(trivance_strerror(TRIVANCE_ESIZE), "output buffer too small") == 0);
    /* a derived plan with a lower dispatch limit: range [1024, 2^31], the original untouched */
    trivance_plan_t* lim = NULL;
    CHECK(trivance_plan(9, NULL, 0, TRIVANCE_LATENCY_OPT, &r) == TRIVANCE_OK);
    CHECK(trivance_plan_with_dispatch_limit(r, 1 << 20, &lim) == TRIVANCE_OK && lim != NULL);
    CHECK(trivance_plan_num_passes(lim) == 2 && trivance_plan_num_passes(r) == 2);
    trivance_plan_destroy(lim);
    CHECK(trivance_plan_with_dispatch_limit(r, 100, &lim) == TRIVANCE_EINVAL && lim == NULL);
    trivance_plan_destroy(r);
    /* the copy helper checks its arguments before any launch; a zero-byte copy does nothing */
    CHECK(trivance_copy_device(NULL, NULL, 0, NULL) == TRIVANCE_OK);
    CHECK(trivance_copy_device((void*)4096, (const void*)8192, 24, NULL) == TRIVANCE_EINVAL);
    CHECK(trivance_copy_device((void*)4104, (const void*)8192, 16, NULL) == TRIVANCE_EINVAL);
    CHECK(trivance_copy_device((void*)4096, (const void*)4128, 64, NULL) == TRIVANCE_EINVAL);
    trivance_plan_destroy(NULL);

    if (failures == 0) printf("abi_host ok\n");
    return failures == 0 ? 0 : 1;
}
