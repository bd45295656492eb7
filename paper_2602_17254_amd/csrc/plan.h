// Internal schedule representation shared by the host plan code and the HIP launchers.
#pragma once

#include <algorithm>
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
    // Tree plans only: the step index inside the active dimension's tree, and the number of
    // steps collective c took in dimension d before this one.
    int dim_step[kMaxDims];
    int taken[kMaxDims][kMaxDims];
};

// Latency-optimal plans with a side that is not a power of three: every rank keeps several partial
// sums ("slots") per collective between passes. Output slot i of a pass is the joint reduction
// (own + left) + right of the input slots own[i] of the rank itself, left[i] of its peer at
// -distance and right[i] of its peer at +distance (-1: that term is absent).
constexpr int kMaxSlots = 64;
struct SlotPass {
    int nin[kMaxDims];   // slots per rank before the pass, per collective
    int nout[kMaxDims];  // after it
    int8_t own[kMaxDims][kMaxSlots], left[kMaxDims][kMaxSlots], right[kMaxDims][kMaxSlots];
};

}  // namespace trivance

namespace trivance {
constexpr int kMaxTab = 768;       // offset-table entries of one tree step (kernel arguments)
constexpr int kMaxTreeSide = 2200;  // longest side of a tree plan
constexpr int kMaxTreeDims = 4;
// Tree-plan table entry: bits 0..29 offset of a rank from the block's owner along one dimension
// (0 <= offset < side); on the active dimension's receivers, bit 30: a child at offset - distance
// sends (from the left), bit 31: a child at offset + distance sends (from the right).
constexpr uint32_t kFromLeft = 1u << 30;
constexpr uint32_t kFromRight = 1u << 31;

// The reduction tree of one dimension (Sec. 4.4 for sides that are not powers of three; the
// ordinary balanced-ternary tree otherwise; no steps for a side of 1).
struct DimTree {
    int side = 1;
    int S = 0;
    std::vector<int> dist;                     // distance of step k
    std::vector<std::vector<uint32_t>> recv;   // step k: receivers with the sides of their children
    std::vector<std::vector<uint32_t>> alive;  // alive[m]: offsets not forwarded in steps < m
    std::vector<int> dirs;                     // step k: bit 0 a child sends towards +, bit 1 towards -
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
    // Rings and tori with a side that is not a power of three (bandwidth-optimal only): every
    // block is reduced along one tree per dimension (trees[d]); a rank holds a partial of block j
    // while its offset from j, in every dimension, has not yet been forwarded.
    bool tree = false;
    std::vector<trivance::DimTree> trees;
    // TRIVANCE_PLACE_BY_SCHEDULE (equal power-of-three sides, bandwidth-optimal): block j of
    // segment c lies at position trivance::placed_position(p, c, j).
    bool placed = false;
    // Most work-items one kernel dispatch may hold (trivance_plan_with_dispatch_limit).
    int64_t dispatch_items = (int64_t)1 << 31;
    // Latency-optimal plans with a side that is not a power of three: the slot program of every
    // pass (same length as `passes`), and the most slots any state between passes holds.
    std::vector<trivance::SlotPass> slots;
    int max_slots = 0;
};

namespace trivance {

// Element range [begin, end) of block `block` (or the whole segment for block < 0) of segment c.
void block_bounds(const trivance_plan_t* p, int64_t elems, int c, int block, int64_t* begin,
                  int64_t* end);

// Position of block `block` of segment c under TRIVANCE_PLACE_BY_SCHEDULE: the base-3 digits of
// its coordinates in the order collective c's steps fix them, most significant first.
int placed_position(const trivance_plan_t* p, int c, int block);

// Largest number of granules in any block, over all segments.
int64_t max_block_granules(const trivance_plan_t* p, int64_t elems);

// Division by an invariant d >= 1 of dividends below 2^31 with one 32-bit multiply-high:
// x / d == mulhi(2 x, mul) >> shift, shift = ceil(log2 d), mul = floor(2^(31 + shift) / d) + 1
// (Granlund and Montgomery, "Division by invariant integers using multiplication", PLDI 1994,
// with N = 31; mul < 2^32 because d > 2^(shift - 1)). The doubled dividend turns their shift by
// 31 + shift into the high word's shift by `shift`.
struct FastDiv32 {
    uint32_t mul;
    uint32_t shift;
};

inline FastDiv32 make_fastdiv32(uint32_t d) {
    uint32_t l = 0;
    while (((uint64_t)1 << l) < d) ++l;
    return FastDiv32{(uint32_t)((((uint64_t)1 << (31 + l)) / d) + 1), l};
}

// Host form of the device division (for tests): x < 2^31.
inline uint32_t fastdiv32_host(uint32_t x, FastDiv32 f) {
    return (uint32_t)((((uint64_t)(x << 1) * f.mul) >> 32) >> f.shift);
}

// Most work-items of one kernel dispatch (also the default of every plan).
constexpr int64_t kMaxDispatchItems = (int64_t)1 << 31;

// A dispatch packet holds its grid size as a 32-bit count of work-items, and a larger grid is not
// rejected: it runs only part of the workgroups. Launches therefore go through this loop, which
// splits a grid of `grid` workgroups of `threads` work-items into consecutive dispatches of at
// most `items` work-items; one(first, count) enqueues workgroups [first, first + count) and
// returns false on failure, which ends the loop.
template <typename F>
inline bool for_each_dispatch(uint64_t grid, int threads, int64_t items, F&& one) {
    const uint64_t per = std::max<uint64_t>(1, (uint64_t)items / (uint64_t)threads);
    for (uint64_t first = 0; first < grid; first += per)
        if (!one((uint32_t)first, (uint32_t)std::min(per, grid - first))) return false;
    return true;
}

}  // namespace trivance
