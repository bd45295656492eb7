// Host-only test of the dispatch split (for_each_dispatch): every workgroup of a grid is covered
// exactly once, in order, by dispatches of whole workgroups that stay within the work-item limit,
// for grids beyond 2^32 work-items, and an early failure ends the loop. Built with g++ against
// the schedule code (plan.cpp); no GPU. Exit status 0 on success.
#include <cstdint>
#include <cstdio>
#include <vector>

#include "plan.h"

static int failures = 0;
#define CHECK(cond)                                                                  \
    do {                                                                             \
        if (!(cond)) {                                                               \
            std::fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond); \
            ++failures;                                                              \
        }                                                                            \
    } while (0)

static void covers(uint64_t grid, int threads, int64_t limit) {
    CHECK(trivance_set_dispatch_limit(limit) > 0);
    uint64_t next = 0, pieces = 0;
    bool whole = true;
    const bool ok = trivance::for_each_dispatch(grid, threads, [&](uint32_t first, uint32_t count) {
        whole = whole && first == next && count >= 1 &&
                (uint64_t)count * (uint64_t)threads <= (uint64_t)limit;
        next = (uint64_t)first + count;
        ++pieces;
        return true;
    });
    CHECK(ok);
    CHECK(whole);
    CHECK(next == grid);
    const uint64_t per = (uint64_t)limit / (uint64_t)threads;
    CHECK(pieces == (grid + per - 1) / per);
}

int main() {
    const int64_t def = (int64_t)1 << 31;
    CHECK(trivance_set_dispatch_limit(4096) == def);  // the default
    CHECK(trivance::dispatch_work_items() == 4096);
    CHECK(trivance_set_dispatch_limit(1023) == TRIVANCE_EINVAL);
    CHECK(trivance_set_dispatch_limit(def + 1) == TRIVANCE_EINVAL);
    CHECK(trivance_set_dispatch_limit(0) == TRIVANCE_EINVAL);
    CHECK(trivance::dispatch_work_items() == 4096);

    // a 3^18-wave grid of 256-thread workgroups (2.5e10 work-items) at the default limit
    covers(96855123, 256, def);
    covers(1, 256, def);
    covers(0, 256, def);
    covers(8388608, 256, def);   // exactly one full dispatch of 2^31 work-items
    covers(8388609, 256, def);   // one workgroup more
    covers(1000, 576, 1024);     // one 576-thread workgroup per dispatch
    covers(1000, 64, 1024);      // 16 per dispatch, the last one short
    covers(12345, 256, 4096);

    // a failing dispatch ends the loop
    CHECK(trivance_set_dispatch_limit(1024) > 0);
    int calls = 0;
    const bool ok = trivance::for_each_dispatch(100, 256, [&](uint32_t, uint32_t) {
        return ++calls < 3;
    });
    CHECK(!ok && calls == 3);
    CHECK(trivance_set_dispatch_limit(def) == 1024);

    if (failures == 0) std::printf("dispatch_split ok\n");
    return failures == 0 ? 0 : 1;
}
