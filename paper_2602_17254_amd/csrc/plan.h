// Internal schedule representation shared by the host plan code and the HIP launchers.
#pragma once

#include <cstdint>
#include <vector>

#include "../../include/trivance.h"

namespace trivance {

constexpr int kMaxDims = TRIVANCE_MAX_DIMS;
constexpr int kGranule = 64;  // elements per partition granule (256 B of fp32 / int32)

// One kernel-materialised step.
struct Pass {
    int phase;           // trivance_phase
    int step;                 // global step index t
    int distance[kMaxDims];   // peer distance of each collective: 3^(steps it took before in dim)
    int dim[kMaxDims];        // active dimension of each collective
    // modulus[c][d] = 3^(number of steps <= t that collective c has taken in dimension d).
    // Rank r keeps block j after reduce-scatter step t iff j_d == r_d (mod modulus[c][d]) for
    // every d; the same pairs (r, j) are the senders of all-gather step t.
    int modulus[kMaxDims][kMaxDims];
    int64_t kept_per_rank;  // n / 3^(t+1): blocks kept by a rank after the step
};

}  // namespace trivance

struct trivance_plan {
    int n = 0;
    int D = 0;
    int variant = 0;
    int S = 0;
    int dims[trivance::kMaxDims] = {};
    int strides[trivance::kMaxDims] = {};
    std::vector<trivance::Pass> passes;
};

namespace trivance {

// Element range [begin, end) of block `block` (or the whole segment for block < 0) of segment c.
void block_bounds(const trivance_plan_t* p, int64_t elems, int c, int block, int64_t* begin,
                  int64_t* end);

// Largest number of granules in any block, over all segments.
int64_t max_block_granules(const trivance_plan_t* p, int64_t elems);

}  // namespace trivance
