// Host-only dump of the plan's per-side reduction trees (Sec. 4.4), for the brute-force checks in
// tests/test_nonpow3_trees.py. For every side given on the command line it builds a bandwidth-
// optimal plan of a ring of that side, or of a torus side x 2 when the side is a power of three
// (so that it still gets a tree), and prints
//   tree <side> <steps> <distance of step 0> ...
//   recv <step> <offset>:<L|R|LR> ...     receivers of the step and the sides their children send from
//   alive <m> <offset> ...                offsets not forwarded before step m
// Built with g++ against plan.cpp; no GPU. Exit status 0 on success.
#include <cstdio>
#include <cstdlib>

#include "plan.h"

int main(int argc, char** argv) {
    for (int i = 1; i < argc; ++i) {
        const int side = std::atoi(argv[i]);
        int pw = 1;
        while (pw < side) pw *= 3;
        const int dims[2] = {side, 2};
        const int D = pw == side ? 2 : 1;
        trivance_plan_t* p = nullptr;
        if (trivance_plan(D * side, dims, D, TRIVANCE_BANDWIDTH_OPT, &p) != TRIVANCE_OK || !p->tree) {
            std::fprintf(stderr, "no tree plan for side %d\n", side);
            return 1;
        }
        const trivance::DimTree& t = p->trees[0];
        std::printf("tree %d %d", t.side, t.S);
        for (int k = 0; k < t.S; ++k) std::printf(" %d", t.dist[k]);
        std::printf("\n");
        for (int k = 0; k < t.S; ++k) {
            std::printf("recv %d", k);
            for (uint32_t e : t.recv[k]) {
                const bool l = (e & trivance::kFromLeft) != 0, r = (e & trivance::kFromRight) != 0;
                std::printf(" %u:%s%s", e & 0x3FFFFFFFu, l ? "L" : "", r ? "R" : "");
            }
            std::printf("\n");
        }
        for (size_t m = 0; m < t.alive.size(); ++m) {
            std::printf("alive %zu", m);
            for (uint32_t o : t.alive[m]) std::printf(" %u", o);
            std::printf("\n");
        }
        trivance_plan_destroy(p);
    }
    return 0;
}
