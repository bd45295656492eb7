// Host-only sweep of the schedule generator and the cost model, built with g++ under
// AddressSanitizer and UndefinedBehaviorSanitizer by tests/test_host_sanitizers.py (plan.cpp and
// cost.cpp are plain C++; no GPU). For many rings and tori in both variants and both block
// placements it builds the plan and calls every host entry point on every pass, collective and
// block at several element counts, checking the invariants each one states: distances within the
// side, blocks that tile their segment, per-pass bytes that add up to the algorithmic bytes, a cost
// made of passes x alpha plus the per-pass link bytes. Then the documented error paths. Exit status
// 0 on success; a sanitizer report aborts the run.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <vector>

#include "trivance.h"

static int failures = 0;
#define CHECK(cond)                                                                          \
    do {                                                                                     \
        if (!(cond)) {                                                                       \
            std::fprintf(stderr, "%s:%d: check failed: %s\n", __FILE__, __LINE__, #cond);  \
            ++failures;                                                                      \
        }                                                                                    \
    } while (0)

static void sweep_plan(const std::vector<int>& dims, int variant, unsigned flags) {
    const int D = (int)dims.size();
    int n = 1;
    for (int s : dims) n *= s;
    trivance_plan_t* p = nullptr;
    const int rc = trivance_plan_ex(n, dims.data(), D, variant, flags, &p);
    if (rc != TRIVANCE_OK) {
        CHECK(rc == TRIVANCE_EUNSUPPORTED && p == nullptr);
        return;
    }
    const int S = trivance_plan_num_steps(p), P = trivance_plan_num_passes(p);
    CHECK(S >= 0 && P >= S);
    for (int pass = 0; pass < P; ++pass) {
        CHECK(trivance_plan_step_index(p, pass) >= 0);
        for (int c = 0; c < D; ++c) {
            int phase = -1, dim = -1, dist = -1;
            CHECK(trivance_plan_step(p, pass, c, &phase, &dim, &dist) == TRIVANCE_OK);
            CHECK(phase >= 0 && phase <= 2 && dim >= 0 && dim < D && dist >= 1);
            CHECK(dist == 1 || dist < dims[dim]);
        }
    }
    const int64_t counts[] = {0, 1, 63, 64 * (int64_t)D * n + 5, 1 << 20};
    for (int64_t E : counts) {
        for (int dt = 0; dt < 2; ++dt) {
            const int64_t alg = trivance_algorithmic_bytes(p, E, dt);
            int64_t sum = 0;
            for (int pass = 0; pass < P; ++pass) sum += trivance_pass_bytes(p, E, dt, pass);
            CHECK(alg >= 0 && sum == alg);
        }
        for (int c = 0; c < D; ++c) {
            int64_t b0 = -1, e0 = -1;
            CHECK(trivance_block_range(p, E, c, -1, &b0, &e0) == TRIVANCE_OK);
            CHECK(0 <= b0 && b0 <= e0 && e0 <= E);
            // blocks tile the segment (in position order, which is block order without placement)
            int64_t covered = 0;
            for (int j = 0; j < n; ++j) {
                int64_t b = -1, e = -1;
                CHECK(trivance_block_range(p, E, c, j, &b, &e) == TRIVANCE_OK);
                CHECK(b0 <= b && b <= e && e <= e0);
                covered += e - b;
            }
            CHECK(covered == e0 - b0);
        }
    }
    std::vector<double> link((size_t)P, -1.0);
    trivance_cost_result res{};
    const int cr = trivance_cost_model(p, 8.0 * (1 << 20), 1.5e-6, 1e-11, link.data(), P, &res);
    if (variant == TRIVANCE_BRUCK_REF) {
        CHECK(cr == TRIVANCE_EUNSUPPORTED);
    } else {
        CHECK(cr == TRIVANCE_OK);
        double trans = 0.0;
        for (double v : link) {
            CHECK(v >= 0.0);
            trans += v;
        }
        CHECK(res.passes == P);
        CHECK(std::fabs(res.latency - P * 1.5e-6) <= 1e-12 * P);
        CHECK(std::fabs(res.transmission - 1e-11 * trans) <= 1e-9 * res.transmission + 1e-30);
        CHECK(std::fabs(res.total - res.latency - res.transmission) <= 1e-9 * res.total + 1e-30);
    }
    trivance_plan_t* q = nullptr;
    CHECK(trivance_plan_with_dispatch_limit(p, 1024, &q) == TRIVANCE_OK && q != nullptr);
    CHECK(trivance_plan_num_passes(q) == P);
    trivance_plan_destroy(q);
    trivance_plan_destroy(p);
}

int main() {
    std::vector<std::vector<int>> shapes;
    for (int s = 1; s <= 120; ++s) shapes.push_back({s});
    for (int s : {243, 728, 729, 2187, 2200}) shapes.push_back({s});
    const std::vector<std::vector<int>> tori = {
        {3, 3}, {9, 9}, {27, 27}, {3, 9}, {9, 27}, {3, 3, 3}, {9, 9, 9}, {3, 3, 9}, {3, 3, 3, 3},
        {3, 3, 3, 3, 3, 3}, {1, 9}, {9, 1}, {1, 1, 27}, {4, 4}, {2, 3}, {5, 7}, {8, 64}, {32, 32},
        {16, 16, 16}, {2, 3, 4}, {9, 8}, {10, 3, 3}, {5, 5, 5, 5}, {2, 2, 2, 2}, {100, 100},
        {2000, 20}, {7, 1, 5}, {3, 2200}};
    for (const auto& t : tori) shapes.push_back(t);
    int plans = 0;
    for (const auto& dims : shapes) {
        for (int variant : {TRIVANCE_LATENCY_OPT, TRIVANCE_BANDWIDTH_OPT, TRIVANCE_BRUCK_REF}) {
            for (unsigned flags : {0u, (unsigned)TRIVANCE_PLACE_BY_SCHEDULE}) {
                sweep_plan(dims, variant, flags);
                ++plans;
            }
        }
    }
    // error paths
    trivance_plan_t* p = nullptr;
    const int d9[1] = {9};
    // NULL sides mean the ring of n
    CHECK(trivance_plan(9, nullptr, 1, TRIVANCE_LATENCY_OPT, &p) == TRIVANCE_OK && p != nullptr);
    CHECK(trivance_plan_num_steps(p) == 2);
    trivance_plan_destroy(p);
    p = nullptr;
    CHECK(trivance_plan(0, d9, 1, TRIVANCE_LATENCY_OPT, &p) == TRIVANCE_EINVAL && p == nullptr);
    CHECK(trivance_plan(8, d9, 1, TRIVANCE_LATENCY_OPT, &p) == TRIVANCE_EINVAL);
    CHECK(trivance_plan(9, d9, 1, 7, &p) == TRIVANCE_EINVAL);
    CHECK(trivance_plan(9, d9, 1, TRIVANCE_LATENCY_OPT, nullptr) == TRIVANCE_EINVAL);
    CHECK(trivance_plan(9, d9, 1, TRIVANCE_LATENCY_OPT, &p) == TRIVANCE_OK);
    int a = 0, b = 0, c = 0;
    CHECK(trivance_plan_step(p, -1, 0, &a, &b, &c) == TRIVANCE_EINVAL);
    CHECK(trivance_plan_step(p, 99, 0, &a, &b, &c) == TRIVANCE_EINVAL);
    CHECK(trivance_plan_step(p, 0, 5, &a, &b, &c) == TRIVANCE_EINVAL);
    CHECK(trivance_plan_step(nullptr, 0, 0, &a, &b, &c) == TRIVANCE_EINVAL);
    int64_t lo = 0, hi = 0;
    CHECK(trivance_block_range(p, -1, 0, 0, &lo, &hi) == TRIVANCE_EINVAL);
    CHECK(trivance_block_range(p, 100, 0, 9, &lo, &hi) == TRIVANCE_EINVAL);
    CHECK(trivance_pass_bytes(p, 100, 0, 99) < 0);
    CHECK(trivance_algorithmic_bytes(nullptr, 100, 0) < 0);
    trivance_plan_t* q = nullptr;
    CHECK(trivance_plan_with_dispatch_limit(p, 10, &q) == TRIVANCE_EINVAL);
    trivance_plan_destroy(p);
    trivance_plan_destroy(nullptr);
    CHECK(trivance_strerror(TRIVANCE_EUNSUPPORTED) != nullptr);
    std::printf("%d plan requests, %d failures\n", plans, failures);
    return failures == 0 ? 0 : 1;
}
