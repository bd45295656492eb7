// Step executor of the emulated Trivance AllReduce for gfx950 (MI355X).
//
// n virtual ranks keep their vectors as rows of one rank-major device array. One kernel launch
// materialises one step of the schedule in place; the kernel boundary is the per-step barrier
// of Sec. 4.3 (both incoming messages are reduced before the next step starts).
//
// Latency-optimal step (Sec. 4.2): every rank r of collective c computes
//     x_r <- (x_r + x_{r - d e}) + x_{r + d e}     over its segment,
// with the pre-step values of all three rows. Along the active dimension the ranks split into
// cycles {r0, r0 + d, r0 + 2d, ...} of length L = side / d (a power of three >= 3); a thread owns
// one column vector of one cycle and walks the cycle with a sliding window held in registers, so
// every location is read once and written once although three ranks consume it. The rows of the
// cycle's first and last position stay in registers, which makes the in-place update safe.
//
// Bandwidth-optimal reduce-scatter step t (Sec. 4.1, block sets of Sec. 4.3): for every collective
// c, rank r and block j with j_d == r_d (mod modulus[c][d]) for all d (the blocks r keeps after
// step t),
//     x_r[blk j] <- (x_r[blk j] + x_{r - d e}[blk j]) + x_{r + d e}[blk j].
// Within one pass every input location is read by exactly one such pair and the locations read
// from a neighbour are never written, so the update is in place.
// All-gather step t (Sec. 4.1 reverse order; Appendix D: no reduction): the same (r, j) pairs are
// the senders; x_{r -/+ d e}[blk j] <- x_r[blk j] (one load feeds two stores).
//
// Work unit of the block steps: one wavefront handles one chunk (64 lanes x VEC x U elements) of
// one (collective, rank, block) pair. The pair is decoded from the unit index once per wavefront
// with wave-uniform integer arithmetic; lanes then issue 16-byte loads and stores.
//
// Rings and tori with a side that is not a power of three (Sec. 4.4) run the same reduce-scatter
// and all-gather steps along one reduction tree per dimension (tree_step_kernel below).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>

#include "device.h"
#include "plan.h"

namespace trivance {
namespace {

constexpr int kBlockThreads = 256;
constexpr int kWavesPerBlock = kBlockThreads / 64;

// Division by a per-pass constant d of dividends below 2^31 (FastDiv32 in plan.h: one 32-bit
// multiply-high and a shift), with the divisor kept for remainders.
struct FastDiv {
    uint32_t mul;
    uint32_t shift;
    uint32_t d;
};

inline FastDiv make_fastdiv(uint32_t d) {
    const FastDiv32 f = make_fastdiv32(d);
    return FastDiv{f.mul, f.shift, d};
}

__device__ __forceinline__ uint32_t fdiv(uint32_t x, const FastDiv& f) {
    return __umulhi(x << 1, f.mul) >> f.shift;
}

// Base-3 digits of a block index of a power-of-three plan (n < 2^31, so at most 19).
constexpr int kMaxPlacedDigits = 20;

struct StepArgs {
    int64_t elems;                 // elements per rank row
    int64_t seg_g[kMaxDims + 1];   // segment granule starts, seg_g[D] = total granules
    int n;
    int D;
    int dims[kMaxDims];
    int strides[kMaxDims];
    int act_dim[kMaxDims];         // active dimension per collective
    int modulus[kMaxDims][kMaxDims];
    int dist[kMaxDims];            // peer distance per collective
    // latency step (one launch covers collectives c_first .. c_first + ncoll - 1, which share
    // the cycle length)
    int c_first;
    int ncycles;                   // cycles per collective
    int colblocks;                 // thread blocks per (collective, cycle)
    // block steps
    int kept;                      // blocks kept per rank: n / 3^(t+1)
    int cpb;                       // chunks per block
    uint32_t units_per_coll;       // n * kept * cpb
    uint32_t total_units;          // D * units_per_coll
    int narrow;                    // 1 if n * (granules per segment + 1) < 2^31
    FastDiv f_upc, f_cpb, f_kept, f_n;
    FastDiv f_side[kMaxDims];
    FastDiv f_mod[kMaxDims][kMaxDims];   // modulus[c][d]
    FastDiv f_nq[kMaxDims][kMaxDims];    // dims[d] / modulus[c][d]
    uint32_t wg_base;              // first workgroup of this dispatch (for_each_dispatch)
    int keep;                      // store policy of the pass (st_out)
    // block steps of plans placed by schedule digits (TRIVANCE_PLACE_BY_SCHEDULE)
    // (32-bit words: the scalar unit loads them directly; bytes would go through vector loads)
    int placed;
    uint32_t pdig[kMaxDims][kMaxDims];    // digits of dimension d that collective c has fixed
    uint32_t pexp_off[kMaxDims];          // first entry of dimension d in pexp[c]
    uint32_t pexp[kMaxDims][kMaxPlacedDigits / 4];  // entry i of collective c: byte i % 4 of
                                                     // word i / 4; entry pexp_off[d] + k is the
                                                     // position exponent of digit k of dimension d
};

// ---------------------------------------------------------------------------------------------
// Latency-optimal step: sliding window over one rank cycle.
// Grid: D * ncycles * colblocks thread blocks; each thread owns VPT column vectors. Non-temporal
// loads; stores with the pass's policy (st_out_as), a template argument as in the tiles below.
template <typename T, int VEC, int VPT, int KEEP>
__global__ __launch_bounds__(kBlockThreads) void latency_step_kernel(T* __restrict__ buf,
                                                                     StepArgs a) {
    using V = Vec<T, VEC>;
    const uint32_t wg = a.wg_base + blockIdx.x;
    const uint32_t cb = wg % (uint32_t)a.colblocks;
    const uint32_t rest = wg / (uint32_t)a.colblocks;
    const int cyc = (int)(rest % (uint32_t)a.ncycles);
    const int c = a.c_first + (int)(rest / (uint32_t)a.ncycles);

    const int dim = a.act_dim[c];
    const int side = a.dims[dim];
    const int stride = a.strides[dim];
    const int dist = a.dist[c];
    const int len = side / dist;  // cycle length, a power of three >= 3
    const int res = cyc % dist;
    const int other = cyc / dist;
    const int first_rank = (other % stride) + (other / stride) * stride * side + res * stride;

    const int64_t E = a.elems;
    const int64_t seg_b = imin64(a.seg_g[c] * kGranule, E);
    const int64_t seg_e = imin64(a.seg_g[c + 1] * kGranule, E);
    const int64_t nvec = (seg_e - seg_b) / VEC;
    const int64_t rowstep = (int64_t)dist * stride * E;
    T* const base = buf + (int64_t)first_rank * E + seg_b;

    T* col[VPT];
    bool ok[VPT];
    // stores: the wave's 64 column vectors of row i start at wcol[u] + i rowstep
    const uint32_t wave = (uint32_t)__builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t off = (threadIdx.x & 63) * VEC * (uint32_t)sizeof(T);
    T* wcol[VPT];
    uint32_t nb[VPT];
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
        const int64_t v = ((int64_t)cb * VPT + u) * kBlockThreads + threadIdx.x;
        ok[u] = v < nvec;
        col[u] = base + v * VEC;
        const int64_t w = ((int64_t)cb * VPT + u) * kBlockThreads + (int64_t)wave * 64;
        wcol[u] = base + w * VEC;
        nb[u] = nvec > w ? (uint32_t)(imin64(nvec - w, 64) * VEC * (int64_t)sizeof(T)) : 0u;
    }

    V first[VPT], last[VPT], prev[VPT], a0[VPT], a1[VPT], a2[VPT];
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
        if (ok[u]) {
            last[u] = ld<T, VEC, true>(col[u] + (int64_t)(len - 1) * rowstep);
            first[u] = ld<T, VEC, true>(col[u]);
            a1[u] = ld<T, VEC, true>(col[u] + rowstep);
            a2[u] = len == 3 ? last[u] : ld<T, VEC, true>(col[u] + 2 * rowstep);
            prev[u] = last[u];
            a0[u] = first[u];
        }
    }
    for (int i = 0; i < len; i += 3) {
        const bool more = i + 3 < len;
        V b0[VPT], b1[VPT], b2[VPT];
        // fetch the next group of three rows before overwriting the current one
#pragma unroll
        for (int u = 0; u < VPT; ++u) {
            if (ok[u]) {
                if (more) {
                    b0[u] = ld<T, VEC, true>(col[u] + (int64_t)(i + 3) * rowstep);
                    b1[u] = ld<T, VEC, true>(col[u] + (int64_t)(i + 4) * rowstep);
                    b2[u] = (i + 5 == len - 1)
                                ? last[u]
                                : ld<T, VEC, true>(col[u] + (int64_t)(i + 5) * rowstep);
                } else {
                    b0[u] = first[u];
                    b1[u] = first[u];
                    b2[u] = first[u];
                }
            }
        }
#pragma unroll
        for (int u = 0; u < VPT; ++u) {
            if (ok[u]) {
                T* p = wcol[u] + (int64_t)i * rowstep;
                st_out_as<KEEP>(buffer_rsrc(p, nb[u]), off, joint(a0[u], prev[u], a1[u]));
                st_out_as<KEEP>(buffer_rsrc(p + rowstep, nb[u]), off, joint(a1[u], a0[u], a2[u]));
                st_out_as<KEEP>(buffer_rsrc(p + 2 * rowstep, nb[u]), off,
                                joint(a2[u], a1[u], b0[u]));
                prev[u] = a2[u];
                a0[u] = b0[u];
                a1[u] = b1[u];
                a2[u] = b2[u];
            }
        }
    }
}

// ---------------------------------------------------------------------------------------------
// Latency-optimal step, cycle of LEN = P * SUB ranks split over the P wavefronts of a workgroup.
// Wave w walks rows [w SUB, (w+1) SUB) of the cycle for 64 column vectors. The only values a
// wave needs from outside its rows are the pre-step rows just before and after its range; every
// wave publishes its own first and last row in LDS and reads its neighbours' after one barrier,
// before any store, so the in-place update stays correct. Splitting gives P times more, P times
// shorter wavefronts than walking the whole cycle in one wavefront.
template <typename T, int VEC, int SUB, int P, int PD, bool NT, int KEEP>
__global__ __launch_bounds__(64 * P) void latency_split_kernel(T* __restrict__ buf, StepArgs a) {
    static_assert(SUB % 3 == 0, "rows are processed in groups of three");
    using V = Vec<T, VEC>;
    constexpr int G = SUB / 3;
    __shared__ V halo[P][2][64];

    const uint32_t wg = a.wg_base + blockIdx.x;
    const uint32_t cb = wg % (uint32_t)a.colblocks;
    const uint32_t rest = wg / (uint32_t)a.colblocks;
    const int cyc = (int)(rest % (uint32_t)a.ncycles);
    const int c = a.c_first + (int)(rest / (uint32_t)a.ncycles);
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;

    const int dim = a.act_dim[c];
    const int side = a.dims[dim];
    const int stride = a.strides[dim];
    const int dist = a.dist[c];
    const int res = cyc % dist;
    const int other = cyc / dist;
    const int first_rank = (other % stride) + (other / stride) * stride * side + res * stride;

    const int64_t E = a.elems;
    const int64_t seg_b = imin64(a.seg_g[c] * kGranule, E);
    const int64_t seg_e = imin64(a.seg_g[c + 1] * kGranule, E);
    const int64_t nvec = (seg_e - seg_b) / VEC;
    const int64_t v_idx = (int64_t)cb * 64 + lane;
    const bool ok = v_idx < nvec;
    const int64_t rowstep = (int64_t)dist * stride * E;
    T* const col = buf + (int64_t)first_rank * E + seg_b + (ok ? v_idx : 0) * VEC +
                   (int64_t)(w * SUB) * rowstep;
    // stores: st_out_as with the pass's policy; the wave's 64 columns of row i start at wcol +
    // i rowstep
    T* const wcol = buf + (int64_t)first_rank * E + seg_b + (int64_t)cb * 64 * VEC +
                    (int64_t)(w * SUB) * rowstep;
    const int64_t wvec = nvec - (int64_t)cb * 64;  // column vectors of this block that exist
    const uint32_t nbytes =
        wvec > 0 ? (uint32_t)(imin64(wvec, 64) * VEC * (int64_t)sizeof(T)) : 0u;
    const uint32_t off = (uint32_t)lane * VEC * (uint32_t)sizeof(T);

    V v[SUB];
    if (ok) {
        v[0] = ld<T, VEC, NT>(col);
        v[SUB - 1] = ld<T, VEC, NT>(col + (int64_t)(SUB - 1) * rowstep);
#pragma unroll
        for (int i = 1; i < 3 * (PD + 1); ++i)
            if (i < SUB - 1) v[i] = ld<T, VEC, NT>(col + (int64_t)i * rowstep);
        halo[w][0][lane] = v[0];
        halo[w][1][lane] = v[SUB - 1];
    }
    __syncthreads();
    if (!ok) return;
    const V before = halo[(w + P - 1) % P][1][lane];  // pre-step row w SUB - 1
    const V after = halo[(w + 1) % P][0][lane];       // pre-step row (w + 1) SUB
#pragma unroll
    for (int g = 0; g < G; ++g) {
#pragma unroll
        for (int i = 3 * (g + PD + 1); i < 3 * (g + PD + 2); ++i)
            if (i < SUB - 1) v[i] = ld<T, VEC, NT>(col + (int64_t)i * rowstep);
#pragma unroll
        for (int i = 3 * g; i < 3 * g + 3; ++i) {
            const V& left = i == 0 ? before : v[i > 0 ? i - 1 : 0];
            const V& right = i == SUB - 1 ? after : v[i + 1 < SUB ? i + 1 : i];
            st_out_as<KEEP>(buffer_rsrc(wcol + (int64_t)i * rowstep, nbytes), off,
                            joint(v[i], left, right));
        }
    }
}

// ---------------------------------------------------------------------------------------------
// Decode of a block-step work unit (all values wave-uniform).

// 3^e for the digit weights of placed plans (n < 2^31, so e <= 19).
__constant__ uint32_t kPow3[20] = {1u,        3u,         9u,         27u,        81u,
                                   243u,      729u,       2187u,      6561u,      19683u,
                                   59049u,    177147u,    531441u,    1594323u,   4782969u,
                                   14348907u, 43046721u,  129140163u, 387420489u, 1162261467u};
struct Unit {
    int64_t begin, end;  // element range of this unit's chunk (begin < end when active)
    int rank, left, right;
};

__device__ __forceinline__ bool decode_unit(const StepArgs& a, uint32_t unit, int chunk_elems,
                                            Unit* out) {
    const uint32_t c = fdiv(unit, a.f_upc);
    const uint32_t rem = unit - c * a.units_per_coll;
    const uint32_t pair = fdiv(rem, a.f_cpb);
    const uint32_t chunk = rem - pair * (uint32_t)a.cpb;
    const uint32_t r = fdiv(pair, a.f_kept);
    uint32_t q = pair - r * (uint32_t)a.kept;
    const int act = a.act_dim[c];

    // j: the block (default partition) or its position (placed plans)
    uint32_t j = 0, rr = r, r_act = 0;
    if (a.placed) {
        // the centre keeps the blocks that agree with it in the digits fixed so far, which sit
        // at one run of positions: the centre's own fixed digits, each at the weight 3^(S - 1 -
        // the step that fixed it), then q
        const uint32_t q0 = q;
#pragma unroll
        for (int d = 0; d < kMaxDims; ++d) {
            if (d < a.D) {
                const uint32_t rr_next = fdiv(rr, a.f_side[d]);
                uint32_t x = rr - rr_next * (uint32_t)a.dims[d];
                rr = rr_next;
                if (d == act) r_act = x;
                const uint32_t base = a.pexp_off[d];
                for (uint32_t k = 0; k < a.pdig[c][d]; ++k) {
                    const uint32_t x3 = __umulhi(x, 0xAAAAAAABu) >> 1;  // x / 3
                    const uint32_t i = base + k;
                    const uint32_t e = (a.pexp[c][i >> 2] >> (8 * (i & 3))) & 0xFFu;
                    j += (x - 3u * x3) * kPow3[e];
                    x = x3;
                }
            }
        }
        j += q0;
    } else {
#pragma unroll
        for (int d = 0; d < kMaxDims; ++d) {
            if (d < a.D) {
                const uint32_t rr_next = fdiv(rr, a.f_side[d]);
                const uint32_t rd = rr - rr_next * (uint32_t)a.dims[d];
                rr = rr_next;
                const FastDiv& fk = a.f_mod[c][d];
                const FastDiv& fq = a.f_nq[c][d];
                const uint32_t q_next = fdiv(q, fq);
                const uint32_t qd = q - q_next * fq.d;
                q = q_next;
                const uint32_t rd_mod = rd - fdiv(rd, fk) * fk.d;
                j += (rd_mod + fk.d * qd) * (uint32_t)a.strides[d];
                if (d == act) r_act = rd;
            }
        }
    }
    const int side = a.dims[act];
    const int st = a.strides[act];
    const int dist = a.dist[c];
    out->rank = (int)r;
    out->left = (int)r_act >= dist ? (int)r - dist * st : (int)r + (side - dist) * st;
    out->right = (int)r_act + dist < side ? (int)r + dist * st : (int)r - (side - dist) * st;

    const int64_t g0 = a.seg_g[c];
    const int64_t Gc = a.seg_g[c + 1] - g0;
    int64_t gb, ge;
    if (a.narrow) {
        gb = g0 + fdiv(j * (uint32_t)Gc, a.f_n);
        ge = g0 + fdiv((j + 1) * (uint32_t)Gc, a.f_n);
    } else {
        gb = g0 + (int64_t)j * Gc / a.n;
        ge = g0 + (int64_t)(j + 1) * Gc / a.n;
    }
    const int64_t E = a.elems;
    const int64_t b = imin64(gb * kGranule, E);
    const int64_t e = imin64(ge * kGranule, E);
    out->begin = b + (int64_t)chunk * chunk_elems;
    out->end = e;
    return out->begin < e;
}

// WPB wavefronts per workgroup, one unit each.
template <typename T, int VEC, int U, bool REDUCE, bool NT, bool XCD, int WPB>
__global__ __launch_bounds__(64 * WPB) void block_step_kernel(T* __restrict__ buf, StepArgs a) {
    using V = Vec<T, VEC>;
    constexpr int kChunk = 64 * VEC * U;
    const int lane = threadIdx.x & 63;
    const uint32_t wave = (uint32_t)__builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t wg = a.wg_base + (XCD ? xcd_contiguous(blockIdx.x, gridDim.x) : blockIdx.x);
    const uint32_t unit = wg * (uint32_t)WPB + wave;
    if (unit >= a.total_units) return;
    Unit w;
    if (!decode_unit(a, unit, kChunk, &w)) return;

    const int64_t E = a.elems;
    T* const own = buf + (int64_t)w.rank * E;
    T* const pl = buf + (int64_t)w.left * E;
    T* const pr = buf + (int64_t)w.right * E;
    int64_t idx[U];
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
        idx[u] = w.begin + (int64_t)(u * 64 + lane) * VEC;
        ok[u] = idx[u] < w.end;
    }
    // stores: buffer stores (st_out) over this wave's chunk (the descriptor ends at the block)
    const uint32_t nbytes = (uint32_t)(imin64(w.end - w.begin, kChunk) * (int64_t)sizeof(T));
    if constexpr (REDUCE) {
        V x[U], y[U], z[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (ok[u]) {
                x[u] = ld<T, VEC, NT>(own + idx[u]);
                y[u] = ld<T, VEC, NT>(pl + idx[u]);
                z[u] = ld<T, VEC, NT>(pr + idx[u]);
            }
        }
        const BufI4 ro = buffer_rsrc(own + w.begin, nbytes);
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (ok[u])
                st_out<T, VEC>(ro, (uint32_t)(u * 64 + lane) * VEC * sizeof(T),
                               joint(x[u], y[u], z[u]), a.keep);
    } else {
        V x[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (ok[u]) x[u] = ld<T, VEC, NT>(own + idx[u]);
        const BufI4 rl = buffer_rsrc(pl + w.begin, nbytes), rr = buffer_rsrc(pr + w.begin, nbytes);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (ok[u]) {
                const uint32_t off = (uint32_t)(u * 64 + lane) * VEC * sizeof(T);
                st_out<T, VEC>(rl, off, x[u], a.keep);
                st_out<T, VEC>(rr, off, x[u], a.keep);
            }
        }
    }
}

// ---------------------------------------------------------------------------------------------
// Sides that are not powers of three (Sec. 4.4): every block is reduced along one tree per
// dimension (see plan.cpp). A rank holds a partial of block j while its offset from j has not
// been forwarded in any dimension, so the ranks working on block j in one step of collective c
// are j + o, with o_a a receiver of the active dimension a's tree at that step (flagged with the
// sides its children send from) and o_d, for every other d, an offset not yet forwarded in d.
// The reduce-scatter computes x <- (x + from_left) + from_right with absent terms skipped, the
// all-gather copies x to the children. Each rank forwards each block once, so within a step no
// location is both read by a neighbour and written: the update is in place.
//
// One wave handles one chunk of 64 * VEC elements of one (collective, block, offset tuple).
// Units are numbered collective by collective; inside a collective: chunk fastest, then the
// offset list of dimension 0, 1, ..., then, on a ring, the block's coordinate, and on a torus the
// receiving rank's coordinates (dimension 0 first; the block is the rank minus the offsets).
// Waves in flight together thus share rows on a torus and blocks on a ring, the order measured
// faster for each (tori 4-9%, rings 1-5%).
// DM: the number of dimensions (the decode is compiled for it); CAP: capacity of the offset table,
// which sizes the kernel arguments, copied at every launch.
//
// The decode is wave-uniform (scalar unit). With blocks of a few granules the units are small
// and the scalar unit, not HBM, bounds the step, so the host precomputes everything a unit needs
// per collective, divisions take one 32-bit multiply-high, and the U consecutive units of a wave
// are decoded incrementally: the next chunk of the same block, or the next offset of list 0
// (same ranks on a torus, same block on a ring), reuse the previous unit's state.
constexpr uint32_t kOffsetMask = 0x3FFFFFFFu;
constexpr uint32_t kFlagBits = kFromLeft | kFromRight;

// Per collective of one pass.
template <int DM>
struct TreeColl {
    int64_t dE;           // elements from a rank's row to its neighbour's at +distance
    int64_t spanE;        // elements spanned by the ring of the active dimension
    int64_t g0, gc;       // first granule and number of granules of the segment
    uint32_t begin;       // first unit of the collective
    int act;              // active dimension
    uint32_t dist;        // its distance
    uint32_t side_act;    // its side
    uint32_t len[DM];     // length of the offset list of dimension d
    FastDiv32 f_len[DM];
    uint32_t lstart[DM];  // first table entry of that list
};

template <int DM, int CAP>
struct TreeArgs {
    int64_t elems;
    uint32_t total;       // units of the pass
    int n;
    int D;
    int narrow;           // 1 if n * (granules of a segment + 1) < 2^31
    int cpb;              // chunks per block (of the largest block)
    uint32_t unit_end[DM];  // collective c owns units [unit_end[c-1], unit_end[c])
    uint32_t side[DM];
    uint32_t stride[DM];
    FastDiv32 f_cpb, f_n;
    FastDiv32 f_side[DM];
    TreeColl<DM> coll[DM];
    uint32_t wg_base;     // first workgroup of this dispatch (for_each_dispatch)
    int keep;             // store policy of the pass (st_out)
    uint32_t tab[CAP];
};
static_assert(sizeof(TreeArgs<kMaxTreeDims, kMaxTab>) <= 4096,
              "tree-step kernel arguments above 4 KiB");


// One decoded unit (wave-uniform) and the state its successors are derived from.
struct TreeUnit {
    int64_t row, rl, rr;  // element offsets of the own row and of its neighbours' rows
    int64_t b, e;         // element range of the block
    uint32_t chunk;
    uint32_t fl;          // the active dimension's children (kFromLeft / kFromRight)
    uint32_t i0;          // index in the offset list of dimension 0
    uint32_t x0;          // torus: the rank's coordinate 0; ring: the block
    uint32_t jrest;       // torus: the block minus its coordinate 0
    int c;
};

template <int DM, int CAP>
__device__ __forceinline__ void tree_rows(const TreeArgs<DM, CAP>& a, const TreeColl<DM>& k,
                                          uint32_t x, uint32_t xa, TreeUnit* w) {
    w->row = (int64_t)x * a.elems;
    w->rl = w->row - k.dE + (xa < k.dist ? k.spanE : 0);
    w->rr = w->row + k.dE - (xa + k.dist >= k.side_act ? k.spanE : 0);
}

template <int DM, int CAP>
__device__ __forceinline__ void tree_block(const TreeArgs<DM, CAP>& a, const TreeColl<DM>& k,
                                           uint32_t j, TreeUnit* w) {
    int64_t gb, ge;
    if (a.narrow) {
        const uint32_t p = j * (uint32_t)k.gc;
        gb = k.g0 + fdiv32(p, a.f_n);
        ge = k.g0 + fdiv32(p + (uint32_t)k.gc, a.f_n);
    } else {
        gb = k.g0 + (int64_t)j * k.gc / a.n;
        ge = k.g0 + (int64_t)(j + 1) * k.gc / a.n;
    }
    w->b = imin64(gb * kGranule, a.elems);
    w->e = imin64(ge * kGranule, a.elems);
}

// Full decode of `unit`; false past the pass's last unit.
template <int DM, int CAP>
__device__ __forceinline__ bool tree_decode(const TreeArgs<DM, CAP>& a, uint32_t unit,
                                            TreeUnit* w) {
    if (unit >= a.total) return false;
    int c = 0;
#pragma unroll
    for (int i = 0; i < DM - 1; ++i)
        if (unit >= a.unit_end[i]) c = i + 1;
    const TreeColl<DM>& k = a.coll[c];
    w->c = c;
    uint32_t rest = unit - k.begin;
    uint32_t q = fdiv32(rest, a.f_cpb);
    w->chunk = rest - q * (uint32_t)a.cpb;
    rest = q;
    uint32_t e[DM];
#pragma unroll
    for (int d = 0; d < DM; ++d) {
        q = fdiv32(rest, k.f_len[d]);
        const uint32_t i = rest - q * k.len[d];
        rest = q;
        if (d == 0) w->i0 = i;
        e[d] = a.tab[k.lstart[d] + i];
    }
    if (DM == 1) {
        // ring: the block is j = rest, its rank j + offset
        const uint32_t off = e[0] & kOffsetMask;
        uint32_t x = rest + off;
        if (x >= a.side[0]) x -= a.side[0];
        w->x0 = rest;
        w->fl = e[0] & kFlagBits;
        tree_rows(a, k, x, x, w);
        tree_block(a, k, rest, w);
        return true;
    }
    // torus: rest is the rank (dimension 0 fastest); the block is the rank minus the offsets
    const uint32_t x = rest;
    uint32_t j = 0, xa = 0, fl = 0, jd0 = 0;
#pragma unroll
    for (int d = 0; d < DM; ++d) {
        uint32_t xd = rest;
        if (d + 1 < DM) {
            q = fdiv32(rest, a.f_side[d]);
            xd = rest - q * a.side[d];
            rest = q;
        }
        const uint32_t off = e[d] & kOffsetMask;
        const uint32_t jd = xd >= off ? xd - off : xd + a.side[d] - off;
        j += jd * a.stride[d];
        if (d == k.act) {
            xa = xd;
            fl = e[d] & kFlagBits;
        }
        if (d == 0) {
            w->x0 = xd;
            jd0 = jd;
        }
    }
    w->fl = fl;
    w->jrest = j - jd0;
    tree_rows(a, k, x, xa, w);
    tree_block(a, k, j, w);
    return true;
}

// Moves a decoded unit to `unit` = its successor; full decode when more than the chunk and the
// offset of list 0 change.
template <int DM, int CAP>
__device__ __forceinline__ bool tree_next(const TreeArgs<DM, CAP>& a, uint32_t unit,
                                          TreeUnit* w) {
    if (w->chunk + 1 < (uint32_t)a.cpb) {
        ++w->chunk;
        return true;
    }
    const TreeColl<DM>& k = a.coll[w->c];
    if (w->i0 + 1 < k.len[0]) {
        w->chunk = 0;
        ++w->i0;
        const uint32_t e0 = a.tab[k.lstart[0] + w->i0];
        const uint32_t off = e0 & kOffsetMask;
        if (DM == 1) {
            uint32_t x = w->x0 + off;
            if (x >= a.side[0]) x -= a.side[0];
            w->fl = e0 & kFlagBits;
            tree_rows(a, k, x, x, w);
        } else {
            const uint32_t xd = w->x0;
            const uint32_t jd = xd >= off ? xd - off : xd + a.side[0] - off;
            if (k.act == 0) w->fl = e0 & kFlagBits;
            tree_block(a, k, w->jrest + jd, w);
        }
        return true;
    }
    return tree_decode(a, unit, w);
}

// One-wave workgroups (measured equal or up to 3% faster than four-wave ones on MI355X). A wave
// takes U consecutive units and issues all their loads before the first store, which keeps more
// bytes in flight per wave when blocks fill only part of a chunk.
template <typename T, int VEC, int U, bool REDUCE, int DM, int CAP>
__global__ __launch_bounds__(64) void tree_step_kernel(T* __restrict__ buf, TreeArgs<DM, CAP> a) {
    using V = Vec<T, VEC>;
    constexpr int kChunk = 64 * VEC;
    const int lane = threadIdx.x;
    const uint32_t wg = a.wg_base + xcd_contiguous(blockIdx.x, gridDim.x);
    const uint32_t first = wg * (uint32_t)U;
    int64_t po[U], pl[U], pr[U];
    int64_t co[U], cl[U], cr[U];  // wave-uniform element offsets of the unit's chunk in the rows
    uint32_t nb[U];               // bytes of the chunk that belong to the block
    uint32_t fl[U];
    bool ok[U];
    V vo[U], vl[U], vr[U];
    TreeUnit w;
    bool live = tree_decode(a, first, &w);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        if (u > 0 && live) live = tree_next(a, first + u, &w);
        const int64_t cs = w.b + (int64_t)w.chunk * kChunk;
        const int64_t idx = cs + (int64_t)lane * VEC;
        ok[u] = live && idx < w.e;
        nb[u] = live && cs < w.e ? (uint32_t)(imin64(w.e - cs, kChunk) * (int64_t)sizeof(T)) : 0u;
        co[u] = w.row + cs;
        cl[u] = w.rl + cs;
        cr[u] = w.rr + cs;
        po[u] = w.row + idx;
        pl[u] = w.rl + idx;
        pr[u] = w.rr + idx;
        fl[u] = w.fl;
        if (ok[u]) {
            vo[u] = ld<T, VEC, true>(buf + po[u]);
            if (REDUCE) {
                if (fl[u] & kFromLeft) vl[u] = ld<T, VEC, true>(buf + pl[u]);
                if (fl[u] & kFromRight) vr[u] = ld<T, VEC, true>(buf + pr[u]);
            }
        }
    }
    // stores: buffer stores (st_out) over each unit's chunk (the descriptor ends at the block)
    const uint32_t off = (uint32_t)lane * VEC * (uint32_t)sizeof(T);
#pragma unroll
    for (int u = 0; u < U; ++u) {
        if (!ok[u]) continue;
        if constexpr (REDUCE) {
            V acc = vo[u];
            if (fl[u] & kFromLeft) acc = vadd(acc, vl[u]);
            if (fl[u] & kFromRight) acc = vadd(acc, vr[u]);
            st_out<T, VEC>(buffer_rsrc(buf + co[u], nb[u]), off, acc, a.keep);
        } else {
            if (fl[u] & kFromLeft)
                st_out<T, VEC>(buffer_rsrc(buf + cl[u], nb[u]), off, vo[u], a.keep);
            if (fl[u] & kFromRight)
                st_out<T, VEC>(buffer_rsrc(buf + cr[u], nb[u]), off, vo[u], a.keep);
        }
    }
}

// ---------------------------------------------------------------------------------------------
// Host side.

// Enqueues `kernel` over `grid` workgroups of `threads` work-items as consecutive dispatches of
// whole workgroups (for_each_dispatch), each with its first workgroup in the argument block.
template <typename T, typename Args>
hipError_t dispatch(void (*kernel)(T*, Args), uint64_t grid, int threads, const Exec& x,
                    T* buf, Args a, size_t dynamic_lds = 0) {
    hipError_t err = hipSuccess;
    for_each_dispatch(grid, threads, x.items, [&](uint32_t first, uint32_t count) {
        a.wg_base = first;
        hipLaunchKernelGGL(kernel, dim3(count), dim3(threads), dynamic_lds, x.stream, buf, a);
        err = hipGetLastError();
        return err == hipSuccess;
    });
    return err;
}

// Launch geometry of one pass.
struct Launch {
    uint32_t grid = 0;
    int U = 0;            // block steps: 16-byte vectors per lane per chunk
    int64_t max_vec = 0;  // latency steps: column vectors of the longest segment
    int ncoll = 0;        // latency steps: collectives in this launch group
};

// Arguments common to every pass of one call.
inline int base_args(const trivance_plan_t* p, int64_t elems, StepArgs* out, int64_t* max_blk) {
    StepArgs a{};
    a.elems = elems;
    a.n = p->n;
    a.D = p->D;
    const int64_t G = (elems + kGranule - 1) / kGranule;
    for (int c = 0; c <= p->D; ++c) a.seg_g[c] = (int64_t)c * G / p->D;
    for (int d = 0; d < kMaxDims; ++d) {
        a.dims[d] = d < p->D ? p->dims[d] : 1;
        a.strides[d] = d < p->D ? p->strides[d] : 1;
    }
    int64_t max_gc = 0;
    for (int c = 0; c < p->D; ++c) max_gc = std::max<int64_t>(max_gc, a.seg_g[c + 1] - a.seg_g[c]);
    a.narrow = (int64_t)p->n * (max_gc + 1) < ((int64_t)1 << 31) ? 1 : 0;
    a.f_n = make_fastdiv((uint32_t)p->n);
    a.placed = p->placed ? 1 : 0;
    if (p->placed) {
        // position exponent S - 1 - t of the digit that reduce-scatter step t fixes
        int off = 0;
        for (int d = 0; d < p->D; ++d) {
            a.pexp_off[d] = (uint32_t)off;
            for (int v = p->dims[d]; v > 1; v /= 3) ++off;
        }
        if (off > kMaxPlacedDigits || p->S != off) return TRIVANCE_EUNSUPPORTED;
        for (int c = 0; c < p->D; ++c) {
            int taken[kMaxDims] = {};
            for (int t = 0; t < p->S; ++t) {
                const int d = p->passes[t].dim[c];
                const uint32_t i = a.pexp_off[d] + (uint32_t)taken[d]++;
                a.pexp[c][i >> 2] |= (uint32_t)(p->S - 1 - t) << (8 * (i & 3));
            }
        }
    }
    for (int d = 0; d < kMaxDims; ++d) a.f_side[d] = make_fastdiv((uint32_t)a.dims[d]);
    *max_blk = max_block_granules(p, elems) * kGranule;
    if (*max_blk >= ((int64_t)1 << 31)) return TRIVANCE_EUNSUPPORTED;
    *out = a;
    return TRIVANCE_OK;
}

// Per-pass fields: active dimensions, distance, moduli and the launch geometry.
template <int VEC>
inline int pass_args(const trivance_plan_t* p, const Pass& ps, int64_t max_blk, int chunk_vecs,
                     StepArgs* a, Launch* L) {
    for (int c = 0; c < kMaxDims; ++c) {
        a->act_dim[c] = ps.dim[c];
        a->dist[c] = ps.distance[c];
        for (int d = 0; d < kMaxDims; ++d) {
            const int m = c < p->D && d < p->D ? ps.modulus[c][d] : 1;
            a->modulus[c][d] = m;
            a->f_mod[c][d] = make_fastdiv((uint32_t)m);
            a->f_nq[c][d] = make_fastdiv((uint32_t)(a->dims[d] / m));
            int digits = 0;
            for (int v = m; v > 1; v /= 3) ++digits;
            a->pdig[c][d] = (uint32_t)digits;
        }
    }
    a->kept = (int)ps.kept_per_rank;
    if (ps.phase == TRIVANCE_PHASE_LATENCY) {
        int64_t max_seg = 0;
        for (int c = 0; c < a->D; ++c) {
            const int64_t b = std::min(a->seg_g[c] * kGranule, a->elems);
            const int64_t e = std::min(a->seg_g[c + 1] * kGranule, a->elems);
            max_seg = std::max(max_seg, e - b);
        }
        L->max_vec = (max_seg + VEC - 1) / VEC;
        // the grid is set per launch group (set_columns); check the largest one fits
        const int64_t cols = std::max<int64_t>(1, (L->max_vec + 63) / 64);
        if ((int64_t)a->D * p->n * cols >= ((int64_t)1 << 31)) return TRIVANCE_EUNSUPPORTED;
        return TRIVANCE_OK;
    }
    // chunk: U 16-byte vectors per lane. One (1 KiB of fp32 per row and wavefront) measured
    // best on MI355X for every workload shape; larger chunks over-subscribe the memory system.
    const int U = chunk_vecs;
    const int64_t chunk = 64 * VEC * U;
    a->cpb = (int)std::max<int64_t>(1, (max_blk + chunk - 1) / chunk);
    const int64_t upc = (int64_t)a->n * a->kept * a->cpb;
    const int64_t total = upc * a->D;
    if (total >= ((int64_t)1 << 31)) return TRIVANCE_EUNSUPPORTED;
    a->units_per_coll = (uint32_t)upc;
    a->total_units = (uint32_t)total;
    a->f_upc = make_fastdiv((uint32_t)upc);
    a->f_cpb = make_fastdiv((uint32_t)a->cpb);
    a->f_kept = make_fastdiv((uint32_t)a->kept);
    L->U = U;
    return TRIVANCE_OK;
}

// Grid for workgroups covering `cols` column vectors each, over the a->ncoll collectives of
// the launch group.
inline void set_columns(StepArgs* a, Launch* L, int cols) {
    a->colblocks = (int)std::max<int64_t>(1, (L->max_vec + cols - 1) / cols);
    L->grid = (uint32_t)((int64_t)L->ncoll * a->ncycles * a->colblocks);
}

// LDS of one MI355X compute unit. A workgroup that asks for 1/k of it, less kLdsSlack bytes
// (so that allocation rounding never leaves room for fewer than k), fits k times at most; the
// latency tiles and the block reduce-scatter use this to cap how many workgroups a CU runs.
constexpr size_t kLdsPerCu = 160 * 1024;
constexpr size_t kLdsSlack = 256;

// Resident workgroups per CU for each latency tile (0: no cap), measured best on MI355X over
// rings of 81 to 2187 ranks and 2D to 4D tori. Fewer concurrent cycles keep fewer rows
// streaming at once; tiles whose waves walk many rows keep enough bytes in flight with one
// workgroup per CU, while the 27-row tile (3 rows per wave) needs the full occupancy.
template <int SUB, int P>
constexpr int latency_wg_per_cu() {
    return (SUB == 3 && P == 1) ? 16
         : (SUB == 3 && P == 3) ? 4
         : (SUB == 9 && P == 1) ? 4
         : (SUB == 3 && P == 9) ? 0
                                : 1;
}

template <typename T, int VEC, int SUB, int P>
hipError_t launch_split(T* buf, StepArgs a, Launch L, const Exec& x) {
    set_columns(&a, &L, 64);
    constexpr int cap = latency_wg_per_cu<SUB, P>();
    constexpr size_t halo = (size_t)P * 2 * 64 * sizeof(Vec<T, VEC>);  // the kernel's own LDS
    constexpr size_t extra = cap ? kLdsPerCu / cap - halo - kLdsSlack : 0;  // unused: the cap
    static_assert(extra + halo <= kLdsPerCu, "a workgroup must fit in one CU's LDS");
    // the store policy (st_out_as) as a template argument: a branch per store measured 6% slower
    // on the 9x9x9 torus at 8 MiB per rank, and one branch around the walk doubled the registers
    // of the 81-row walks
    if (a.keep)
        return dispatch(latency_split_kernel<T, VEC, SUB, P, 1, true, 1>, L.grid, 64 * P, x, buf,
                        a, extra);
    return dispatch(latency_split_kernel<T, VEC, SUB, P, 1, true, 0>, L.grid, 64 * P, x, buf, a,
                    extra);
}

template <typename T, int VEC>
hipError_t launch_latency(T* buf, const StepArgs& a, const Launch& L, int len, const Exec& x) {
    switch (len) {
        // rows per wavefront x wavefronts per workgroup, measured best on MI355X
        case 3: return launch_split<T, VEC, 3, 1>(buf, a, L, x);
        case 9:
            // one wave per cycle measured 5-10% faster on tori of three or more dimensions, and
            // up to 2% slower on rings
            if (a.D >= 3) return launch_split<T, VEC, 9, 1>(buf, a, L, x);
            return launch_split<T, VEC, 3, 3>(buf, a, L, x);
        case 27: return launch_split<T, VEC, 3, 9>(buf, a, L, x);
        case 81: return launch_split<T, VEC, 9, 9>(buf, a, L, x);
        case 243: return launch_split<T, VEC, 81, 3>(buf, a, L, x);
        // 81 rows per wavefront keep the register window in registers (72 VGPRs); 243 would spill
        case 729: return launch_split<T, VEC, 81, 9>(buf, a, L, x);
        default: {
            StepArgs b = a;
            Launch M = L;
            set_columns(&b, &M, kBlockThreads);
            if (b.keep)
                return dispatch(latency_step_kernel<T, VEC, 1, 1>, M.grid, kBlockThreads, x, buf,
                                b);
            return dispatch(latency_step_kernel<T, VEC, 1, 0>, M.grid, kBlockThreads, x, buf, b);
        }
    }
}

// Reduce-scatter: one-wave workgroups, at most 20 per CU (unused dynamic LDS); all-gather: four-wave
// workgroups, no cap. Measured best on MI355X over the 243-ring, 27x27 and 9x9x9 (both block
// placements, 4 to 32 MiB per rank): the reduce-scatter gained 1.5-3.8% over four-wave
// workgroups without a cap, while every cap cost the all-gather 5-30%.
constexpr int kBlockRsWgPerCu = 20;

template <typename T, int VEC>
hipError_t launch_block(T* buf, const StepArgs& a, const Launch& L, bool reduce, const Exec& x) {
    if (L.U != 1) return hipErrorInvalidValue;
    if (reduce)
        return dispatch(block_step_kernel<T, VEC, 1, true, true, true, 1>, a.total_units, 64, x,
                        buf, a, kLdsPerCu / kBlockRsWgPerCu - kLdsSlack);
    return dispatch(block_step_kernel<T, VEC, 1, false, true, true, kWavesPerBlock>,
                    ((uint64_t)a.total_units + kWavesPerBlock - 1) / kWavesPerBlock, kBlockThreads,
                    x, buf, a);
}

template <typename T, int VEC>
int run_passes_vec(T* buf, int64_t elems, const trivance_plan_t* p, hipStream_t stream, int pb,
                   int pe) {
    const Exec x{stream, p->dispatch_items};
    StepArgs a;
    int64_t max_blk;
    int rc = base_args(p, elems, &a, &max_blk);
    if (rc != TRIVANCE_OK) return rc;
    for (int pi = pb; pi < pe; ++pi) {
        const Pass& ps = p->passes[pi];
        Launch L;
        rc = pass_args<VEC>(p, ps, max_blk, 1, &a, &L);
        if (rc != TRIVANCE_OK) return rc;
        a.keep = keep_stores(p, elems, pi);
        hipError_t err = hipSuccess;
        if (ps.phase == TRIVANCE_PHASE_LATENCY) {
            // collectives that share a cycle length run in one launch; with equal sides that is
            // all of them, otherwise one launch per collective
            bool same = true;
            for (int c = 1; c < p->D; ++c)
                same = same && p->dims[ps.dim[c]] == p->dims[ps.dim[0]] &&
                       ps.distance[c] == ps.distance[0];
            for (int c0 = 0; c0 < p->D && err == hipSuccess; c0 += same ? p->D : 1) {
                const int side = p->dims[ps.dim[c0]];
                a.c_first = c0;
                a.ncycles = (p->n / side) * ps.distance[c0];
                L.ncoll = same ? p->D : 1;
                err = launch_latency<T, VEC>(buf, a, L, side / ps.distance[c0], x);
            }
            a.c_first = 0;
        } else {
            err = launch_block<T, VEC>(buf, a, L, ps.phase == TRIVANCE_PHASE_REDUCE_SCATTER, x);
        }
        if (err != hipSuccess) return TRIVANCE_EHIP;
    }
    return TRIVANCE_OK;
}

template <typename T, int VEC, int U, int DM, int CAP>
hipError_t launch_tree(T* buf, const TreeArgs<DM, CAP>& a, bool rs, int64_t total, const Exec& x) {
    const uint64_t waves = (uint64_t)((total + U - 1) / U);  // one wave per workgroup
    if (rs) return dispatch(tree_step_kernel<T, VEC, U, true, DM, CAP>, waves, 64, x, buf, a);
    return dispatch(tree_step_kernel<T, VEC, U, false, DM, CAP>, waves, 64, x, buf, a);
}

// Offset-table entries of pass `pi` (all collectives).
size_t tree_entries(const trivance_plan_t* p, int pi) {
    const Pass& ps = p->passes[pi];
    size_t used = 0;
    for (int c = 0; c < p->D; ++c)
        for (int d = 0; d < p->D; ++d)
            used += d == ps.dim[c] ? p->trees[d].recv[ps.dim_step[c]].size()
                                   : p->trees[d].alive[ps.taken[c][d]].size();
    return used;
}

template <typename T, int VEC, int DM, int CAP>
int run_tree_impl(T* buf, int64_t elems, const trivance_plan_t* p, hipStream_t stream, int pb,
                  int pe) {
    const Exec x{stream, p->dispatch_items};
    TreeArgs<DM, CAP> a;
    std::memset(&a, 0, sizeof(a));
    a.elems = elems;
    a.n = p->n;
    a.D = p->D;
    int64_t max_gc = 0, seg_g0[kMaxTreeDims] = {}, seg_gc[kMaxTreeDims] = {};
    const int64_t G = (elems + kGranule - 1) / kGranule;
    for (int c = 0; c < p->D; ++c) {
        seg_g0[c] = (int64_t)c * G / p->D;
        seg_gc[c] = (int64_t)(c + 1) * G / p->D - seg_g0[c];
        max_gc = std::max(max_gc, seg_gc[c]);
    }
    a.narrow = (int64_t)p->n * (max_gc + 1) < ((int64_t)1 << 31) ? 1 : 0;
    a.f_n = make_fastdiv32((uint32_t)p->n);
    for (int d = 0; d < p->D; ++d) {
        a.side[d] = (uint32_t)p->dims[d];
        a.stride[d] = (uint32_t)p->strides[d];
        a.f_side[d] = make_fastdiv32((uint32_t)p->dims[d]);
    }
    const int64_t max_blk = max_block_granules(p, elems) * kGranule;
    const int64_t chunk = 64 * VEC;
    a.cpb = (int)std::max<int64_t>(1, (max_blk + chunk - 1) / chunk);
    a.f_cpb = make_fastdiv32((uint32_t)a.cpb);
    // Units per wave, measured on MI355X over rings and 2- to 4-dimensional tori. When blocks
    // fill less than 80% of their chunks on average (blocks of a few granules, e.g. 16 x 16 x 16
    // ranks at 8 and 16 MiB, 32 x 32 at 1 MiB) the all-gather (one load per unit) takes eight on
    // rings and 2D tori and two on tori of three or more dimensions, and the reduce-scatter two
    // on rings and 2D tori; everything else takes one.
    const double fill = (double)elems / ((double)p->D * p->n * a.cpb * chunk);
    const int u_rs = fill < 0.8 && p->D <= 2 ? 2 : 1;
    const int u_ag = fill < 0.8 ? (p->D <= 2 ? 8 : 2) : 1;
    for (int pi = pb; pi < pe; ++pi) {
        const Pass& ps = p->passes[pi];
        int used = 0;
        int64_t total = 0;
        for (int c = 0; c < p->D; ++c) {
            TreeColl<DM>& k = a.coll[c];
            const int ad = ps.dim[c];
            k.act = ad;
            k.dist = (uint32_t)ps.distance[c];
            k.side_act = (uint32_t)p->dims[ad];
            k.dE = (int64_t)ps.distance[c] * p->strides[ad] * elems;
            k.spanE = (int64_t)p->dims[ad] * p->strides[ad] * elems;
            k.g0 = seg_g0[c];
            k.gc = seg_gc[c];
            k.begin = (uint32_t)total;
            int64_t units = (int64_t)p->n * a.cpb;
            for (int d = 0; d < p->D; ++d) {
                const std::vector<uint32_t>& list =
                    d == ad ? p->trees[d].recv[ps.dim_step[c]] : p->trees[d].alive[ps.taken[c][d]];
                if (used + (int)list.size() > CAP) return TRIVANCE_EUNSUPPORTED;
                k.lstart[d] = (uint32_t)used;
                for (uint32_t v : list) a.tab[used++] = v;
                k.len[d] = (uint32_t)list.size();
                k.f_len[d] = make_fastdiv32((uint32_t)std::max<size_t>(1, list.size()));
                units *= (int64_t)list.size();
            }
            total += units;
            if (total >= ((int64_t)1 << 31) - 4096) return TRIVANCE_EUNSUPPORTED;
            a.unit_end[c] = (uint32_t)total;
        }
        a.total = (uint32_t)total;
        if (total == 0) continue;
        a.keep = keep_stores(p, elems, pi);
        const bool rs = ps.phase == TRIVANCE_PHASE_REDUCE_SCATTER;
        hipError_t err;
        switch (rs ? u_rs : u_ag) {
            case 8: err = launch_tree<T, VEC, 8>(buf, a, rs, total, x); break;
            case 2: err = launch_tree<T, VEC, 2>(buf, a, rs, total, x); break;
            default: err = launch_tree<T, VEC, 1>(buf, a, rs, total, x); break;
        }
        if (err != hipSuccess) return TRIVANCE_EHIP;
    }
    return TRIVANCE_OK;
}

// The decode is compiled per number of dimensions (1 to 4); plans whose passes need at most 64
// table entries take the short argument block.
template <typename T, int VEC>
int run_tree_passes(T* buf, int64_t elems, const trivance_plan_t* p, hipStream_t stream, int pb,
                    int pe) {
    size_t need = 0;
    for (int pi = pb; pi < pe; ++pi) need = std::max(need, tree_entries(p, pi));
    if (need > (size_t)kMaxTab) return TRIVANCE_EUNSUPPORTED;
    const bool small = need <= 64;
    if (p->D == 1)
        return small ? run_tree_impl<T, VEC, 1, 64>(buf, elems, p, stream, pb, pe)
                     : run_tree_impl<T, VEC, 1, kMaxTab>(buf, elems, p, stream, pb, pe);
    switch (p->D) {
        case 2: return small ? run_tree_impl<T, VEC, 2, 64>(buf, elems, p, stream, pb, pe)
                             : run_tree_impl<T, VEC, 2, kMaxTab>(buf, elems, p, stream, pb, pe);
        case 3: return small ? run_tree_impl<T, VEC, 3, 64>(buf, elems, p, stream, pb, pe)
                             : run_tree_impl<T, VEC, 3, kMaxTab>(buf, elems, p, stream, pb, pe);
        case 4: return small ? run_tree_impl<T, VEC, 4, 64>(buf, elems, p, stream, pb, pe)
                             : run_tree_impl<T, VEC, 4, kMaxTab>(buf, elems, p, stream, pb, pe);
        default: return TRIVANCE_EUNSUPPORTED;
    }
}

template <typename T>
int run_passes(T* buf, int64_t elems, const trivance_plan_t* p, T* ws, hipStream_t stream, int pb,
               int pe) {
    if (!p->slots.empty()) return run_slot_passes(buf, elems, p, ws, stream, pb, pe);
    if (p->tree) {
        if (elems % 4 == 0 && (uintptr_t)buf % 16 == 0)
            return run_tree_passes<T, 4>(buf, elems, p, stream, pb, pe);
        return run_tree_passes<T, 1>(buf, elems, p, stream, pb, pe);
    }
    // 16-byte vectors need 16-byte aligned rows: an aligned base and elems % 4 == 0
    if (elems % 4 == 0 && (uintptr_t)buf % 16 == 0)
        return run_passes_vec<T, 4>(buf, elems, p, stream, pb, pe);
    return run_passes_vec<T, 1>(buf, elems, p, stream, pb, pe);
}

}  // namespace
}  // namespace trivance

extern "C" {

int64_t trivance_workspace_bytes(const trivance_plan_t* plan, int64_t elems, int dtype) {
    if (!plan || elems < 0) return TRIVANCE_EINVAL;
    if (dtype != TRIVANCE_F32 && dtype != TRIVANCE_I32) return TRIVANCE_EINVAL;
    if (plan->slots.empty()) return 0;
    return (int64_t)trivance::slot_halves(plan) * plan->max_slots * plan->n * elems * 4;
}

int trivance_allreduce_emulated_steps_ws(void* buffers, int n, int64_t elems, int dtype,
                                         const trivance_plan_t* plan, void* workspace,
                                         int64_t workspace_bytes, void* stream, int pass_begin,
                                         int pass_end) {
    if (!plan || n != plan->n || elems < 0) return TRIVANCE_EINVAL;
    if (dtype != TRIVANCE_F32 && dtype != TRIVANCE_I32) return TRIVANCE_EINVAL;
    const int np = (int)plan->passes.size();
    if (pass_begin < 0 || pass_end < pass_begin || pass_end > np) return TRIVANCE_EINVAL;
    if (plan->variant == TRIVANCE_BRUCK_REF) return TRIVANCE_EUNSUPPORTED;
    if (elems == 0 || pass_begin == pass_end) return TRIVANCE_OK;
    if (!buffers) return TRIVANCE_EINVAL;
    const int64_t need = trivance_workspace_bytes(plan, elems, dtype);
    if (workspace_bytes < need || (need > 0 && !workspace)) return TRIVANCE_ESIZE;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (dtype == TRIVANCE_F32)
        return trivance::run_passes<float>(static_cast<float*>(buffers), elems, plan,
                                           static_cast<float*>(workspace), s, pass_begin, pass_end);
    return trivance::run_passes<int>(static_cast<int*>(buffers), elems, plan,
                                     static_cast<int*>(workspace), s, pass_begin, pass_end);
}

int trivance_allreduce_emulated_ws(void* buffers, int n, int64_t elems, int dtype,
                                   const trivance_plan_t* plan, void* workspace,
                                   int64_t workspace_bytes, void* stream) {
    if (!plan) return TRIVANCE_EINVAL;
    return trivance_allreduce_emulated_steps_ws(buffers, n, elems, dtype, plan, workspace,
                                                workspace_bytes, stream, 0,
                                                (int)plan->passes.size());
}

int trivance_allreduce_emulated_steps(void* buffers, int n, int64_t elems, int dtype,
                                      const trivance_plan_t* plan, void* stream, int pass_begin,
                                      int pass_end) {
    return trivance_allreduce_emulated_steps_ws(buffers, n, elems, dtype, plan, nullptr, 0, stream,
                                                pass_begin, pass_end);
}

int trivance_allreduce_emulated(void* buffers, int n, int64_t elems, int dtype,
                                const trivance_plan_t* plan, void* stream) {
    if (!plan) return TRIVANCE_EINVAL;
    return trivance_allreduce_emulated_steps(buffers, n, elems, dtype, plan, stream, 0,
                                             (int)plan->passes.size());
}

}  // extern "C"
