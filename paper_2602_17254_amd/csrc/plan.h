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

namespace trivance {
constexpr int kMaxRecv = 768;     // receivers per step of a tree plan (kernel-argument table)
constexpr int kMaxTreeRanks = 2200;
// Tree-plan receiver entry: bits 0..29 offset of the receiving rank from the block's owner
// (0 <= offset < n), bit 30: a child at offset - distance sends (from the left), bit 31: a
// child at offset + distance sends (from the right).
constexpr uint32_t kFromLeft = 1u << 30;
constexpr uint32_t kFromRight = 1u << 31;
}  // namespace trivance

struct trivance_plan {
    int n = 0;
    int D = 0;
    int variant = 0;
    int S = 0;
    int dims[trivance::kMaxDims] = {};
    int strides[trivance::kMaxDims] = {};
    std::vector<trivance::Pass> passes;
    // Rings whose size is not a power of three (bandwidth-optimal only): every block is reduced
    // along one tree; per step, the receivers and the sides their children send from.
    bool tree = false;
    std::vector<int> tree_dist;                  // distance of step k
    std::vector<std::vector<uint32_t>> tree_recv;  // receivers of step k
    std::vector<int> tree_dirs;                  // step k: bit 0 a child sends towards +, bit 1 towards -
};

namespace trivance {

// Element range [begin, end) of block `block` (or the whole segment for block < 0) of segment c.
void block_bounds(const trivance_plan_t* p, int64_t elems, int c, int block, int64_t* begin,
                  int64_t* end);

// Largest number of granules in any block, over all segments.
int64_t max_block_granules(const trivance_plan_t* p, int64_t elems);

}  // namespace trivance
