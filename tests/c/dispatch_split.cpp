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
    uint64_t next = 0, pieces = 0;
    bool whole = true;
    const bool ok = trivance::for_each_dispatch(grid, threads, limit,
                                                [&](uint32_t first, uint32_t count) {
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
    const int64_t def = trivance::kMaxDispatchItems;
    CHECK(def == ((int64_t)1 << 31));

    // a plan carries its limit; a derived plan has its own and leaves the original untouched
    trivance_plan_t* p = nullptr;
    CHECK(trivance_plan(27, nullptr, 0, TRIVANCE_BANDWIDTH_OPT, &p) == TRIVANCE_OK);
    CHECK(p->dispatch_items == def);
    trivance_plan_t* q = nullptr;
    CHECK(trivance_plan_with_dispatch_limit(p, 4096, &q) == TRIVANCE_OK && q != nullptr);
    CHECK(q->dispatch_items == 4096 && p->dispatch_items == def);
    CHECK(q->passes.size() == p->passes.size() && q->n == p->n && q->S == p->S);
    trivance_plan_t* r = reinterpret_cast<trivance_plan_t*>(1);
    CHECK(trivance_plan_with_dispatch_limit(p, 1023, &r) == TRIVANCE_EINVAL && r == nullptr);
    CHECK(trivance_plan_with_dispatch_limit(p, def + 1, &r) == TRIVANCE_EINVAL);
    CHECK(trivance_plan_with_dispatch_limit(nullptr, 4096, &r) == TRIVANCE_EINVAL);
    CHECK(trivance_plan_with_dispatch_limit(p, 4096, nullptr) == TRIVANCE_EINVAL);
    trivance_plan_destroy(p);
    CHECK(q->dispatch_items == 4096);  // still valid after the original is gone
    trivance_plan_destroy(q);

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
    int calls = 0;
    const bool ok = trivance::for_each_dispatch(100, 256, 1024, [&](uint32_t, uint32_t) {
        return ++calls < 3;
    });
    CHECK(!ok && calls == 3);

    if (failures == 0) std::printf("dispatch_split ok\n");
    return failures == 0 ? 0 : 1;
}
