// Latency-optimal passes on sides that are not powers of three (Sec. 4.2 with Sec. 4.4), for
// gfx950: the slot-step kernel and its launcher. The slot programs come from plan.cpp.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <cstring>

#include "device.h"
#include "plan.h"

namespace trivance {
namespace {

// ---------------------------------------------------------------------------------------------
// Latency-optimal step on sides that are not powers of three (Sec. 4.2 with Sec. 4.4): every rank
// keeps a few partial sums ("slots", see plan.cpp) per collective. Output slot i of rank x is the
// joint reduction (own + left) + right of input slot own[i] of x, left[i] of the peer at -distance
// and right[i] of the peer at +distance along the collective's active dimension (absent terms
// skipped). Inputs and outputs are different state arrays (slot s of a state is an [n][elems]
// array at s * n * elems), so the pass has no in-place hazard.
//
// One wave handles 64 column vectors of one rank of one collective and computes all its output
// slots. Along the active dimension the ranks x, x + d, x + 2d, ... form cycles; units are
// numbered so that consecutive ones are consecutive ranks of one cycle at the same columns, and
// each XCD takes one contiguous range of units: the partials a wave reads from its peers at -d
// and +d were just read by its neighbours in the schedule, so they come from the XCD's L2 rather
// than HBM (rocprofv3 FETCH_SIZE equals the bytes of one read per partial). Consecutive units
// first take kSlotGroup consecutive column blocks of one rank, so that the waves in flight also
// stream contiguous kilobytes of each row instead of single kilobytes of many rows: 64 KiB runs
// measured 5-11% faster than 16 KiB ones on the 64-ring and the 32x32 torus at 8 MiB per rank
// (32 KiB in between, 128 and 512 KiB no better).
struct SlotArgs {
    int64_t elems;
    int64_t seg_g[kMaxDims + 1];
    int64_t slot_stride;  // elements from one slot array to the next: n * elems
    int n;
    int D;
    uint32_t colblocks;   // groups of kSlotGroup column blocks (kSlotChunks x 64 vectors) per rank
    uint32_t per_coll;    // units of one collective: n * colblocks
    uint32_t units;       // D * per_coll
    FastDiv32 f_per_coll, f_colblocks;
    // per collective: active dimension, distance, its side and stride, cycle length
    // L = side / gcd(side, distance) and the g = side / L cycles of one line
    int act[kMaxDims], dist[kMaxDims], side[kMaxDims], stride[kMaxDims], nout[kMaxDims];
    int cycle[kMaxDims], gcyc[kMaxDims];
    FastDiv32 f_cycle[kMaxDims], f_gcyc[kMaxDims], f_side[kMaxDims], f_stride[kMaxDims];
    int8_t own[kMaxDims][kMaxSlots], left[kMaxDims][kMaxSlots], right[kMaxDims][kMaxSlots];
    uint32_t wg_base;
    int keep;  // store policy of the pass (st_out)
};
static_assert(sizeof(SlotArgs) <= 4096, "slot-step kernel arguments above 4 KiB");

constexpr int kSlotWaves = 4;   // waves per workgroup
constexpr int kSlotChunks = 1;  // 64-vector chunks of one partial per wave
constexpr int kSlotGroup = 64;  // consecutive column blocks of one rank in consecutive units
constexpr int kSlotBatch = 4;   // output partials whose loads are issued together
// A pass after the first whose bytes fit in the 256 MB last-level cache (MALL) and that writes at
// most two partials per collective takes batches of two: 40 instead of 63 VGPRs, so 12 waves per
// SIMD instead of 8. It reads the partials the previous pass has just written (kept in the cache
// by the SC1 store policy), and on the rings of 4 and 8 at 96-288 MiB per pass it measured 8-15%
// faster. A first pass reads the caller's rows from HBM: there, and on passes with two outputs
// above 256 MiB, batches of two measured 4-16% slower (over-subscribed, like the block steps'
// larger chunks), and 14-20% on 32x32's first pass.
constexpr int kSlotBatchSmall = 2;
constexpr int64_t kSmallSlotPassBytes = (int64_t)256 << 20;

template <typename T, int VEC, int BATCH>
__global__ __launch_bounds__(64 * kSlotWaves) void slot_step_kernel(T* __restrict__ out,
                                                                   const T* __restrict__ in,
                                                                   SlotArgs a) {
    using V = Vec<T, VEC>;
    const uint32_t wave = (uint32_t)__builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t unit =
        (a.wg_base + xcd_contiguous(blockIdx.x, gridDim.x)) * kSlotWaves + wave;
    if (unit >= a.units) return;
    // unit = (((c * cycles + cycle) * groups + grp) * L + i) * kSlotGroup + j: column block
    // cb = grp * kSlotGroup + j of the rank at position i of the cycle; every divisor is a
    // per-pass constant (one multiply-high each)
    const int c = (int)fdiv32(unit, a.f_per_coll);
    uint32_t r = unit - (uint32_t)c * a.per_coll;
    const int dim = a.act[c];
    const uint32_t side = (uint32_t)a.side[dim], stride = (uint32_t)a.stride[dim];
    const uint32_t dist = (uint32_t)a.dist[c], L = (uint32_t)a.cycle[c];
    const uint32_t j = r % kSlotGroup;
    r /= kSlotGroup;
    uint32_t q = fdiv32(r, a.f_cycle[c]);
    const uint32_t i = r - q * L;
    r = q;
    q = fdiv32(r, a.f_colblocks);  // colblocks counts groups here
    const uint32_t cb = (r - q * a.colblocks) * kSlotGroup + j;
    const uint32_t cyc = q;
    const uint32_t line = fdiv32(cyc, a.f_gcyc[c]);
    const uint32_t res = cyc - line * (uint32_t)a.gcyc[c];
    const uint32_t id = i * dist;  // < side^2 < 2^31
    uint32_t xa = res + (id - fdiv32(id, a.f_side[dim]) * side);
    if (xa >= side) xa -= side;    // the coordinate along the active dimension
    const uint32_t lq = fdiv32(line, a.f_stride[dim]);
    const int x = (int)((line - lq * stride) + lq * stride * side + xa * stride);
    const int xl = x + (int)((xa >= dist ? -(int)dist : (int)(side - dist)) * (int)stride);
    const int xr = x + (int)((xa + dist < side ? (int)dist : (int)dist - (int)side) * (int)stride);
    const int64_t E = a.elems;
    const int64_t seg_b = imin64(a.seg_g[c] * kGranule, E);
    const int64_t seg_e = imin64(a.seg_g[c + 1] * kGranule, E);
    const int64_t col0 = seg_b + ((int64_t)cb * kSlotChunks * 64 + (threadIdx.x & 63)) * VEC;
    if (col0 >= seg_e) return;
    bool ok[kSlotChunks];
#pragma unroll
    for (int u = 0; u < kSlotChunks; ++u) ok[u] = col0 + (int64_t)u * 64 * VEC < seg_e;
    const T* const own_row = in + (int64_t)x * E + col0;
    const T* const left_row = in + (int64_t)xl * E + col0;
    const T* const right_row = in + (int64_t)xr * E + col0;
    // stores: buffer stores (st_out) over the wave's 64 column vectors of each output partial
    T* const out_wave = out + (int64_t)x * E + seg_b + (int64_t)cb * kSlotChunks * 64 * VEC;
    const uint32_t nbytes = (uint32_t)(imin64(seg_e - (seg_b + (int64_t)cb * kSlotChunks * 64 * VEC),
                                              (int64_t)kSlotChunks * 64 * VEC) *
                                       (int64_t)sizeof(T));
    const uint32_t off = (uint32_t)(threadIdx.x & 63) * VEC * (uint32_t)sizeof(T);
    // outputs in batches of BATCH: all loads of a batch are issued before its stores
    for (int k0 = 0; k0 < a.nout[c]; k0 += BATCH) {
        V vo[BATCH][kSlotChunks], vl[BATCH][kSlotChunks], vr[BATCH][kSlotChunks];
        int so[BATCH], sl[BATCH], sr[BATCH];
#pragma unroll
        for (int b = 0; b < BATCH; ++b) {
            const bool live = k0 + b < a.nout[c];
            so[b] = live ? a.own[c][k0 + b] : -1;
            sl[b] = live ? a.left[c][k0 + b] : -1;
            sr[b] = live ? a.right[c][k0 + b] : -1;
#pragma unroll
            for (int u = 0; u < kSlotChunks; ++u) {
                if (!ok[u]) continue;
                const int64_t off = (int64_t)u * 64 * VEC;
                if (so[b] >= 0) vo[b][u] = ld<T, VEC>(own_row + so[b] * a.slot_stride + off);
                if (sl[b] >= 0) vl[b][u] = ld<T, VEC>(left_row + sl[b] * a.slot_stride + off);
                if (sr[b] >= 0) vr[b][u] = ld<T, VEC>(right_row + sr[b] * a.slot_stride + off);
            }
        }
#pragma unroll
        for (int b = 0; b < BATCH; ++b) {
            if (k0 + b >= a.nout[c]) break;
#pragma unroll
            for (int u = 0; u < kSlotChunks; ++u) {
                if (!ok[u]) continue;
                // (own + left) + right, absent terms skipped
                V acc = so[b] >= 0 ? vo[b][u] : (sl[b] >= 0 ? vl[b][u] : vr[b][u]);
                if (so[b] >= 0 && sl[b] >= 0) acc = vadd(acc, vl[b][u]);
                if (sr[b] >= 0 && (so[b] >= 0 || sl[b] >= 0)) acc = vadd(acc, vr[b][u]);
                st_out<T, VEC>(buffer_rsrc(out_wave + (int64_t)(k0 + b) * a.slot_stride, nbytes),
                               off + (uint32_t)(u * 64 * VEC * sizeof(T)), acc, a.keep);
            }
        }
    }}

// dst[i] = src[i] for `vecs` vectors of VEC elements (workgroups from `wg0` on).
template <typename T, int VEC>
__global__ __launch_bounds__(256) void copy_rows_kernel(T* __restrict__ dst,
                                                        const T* __restrict__ src, int64_t vecs,
                                                        uint64_t wg0) {
    const int64_t i = (int64_t)((wg0 + blockIdx.x) * 256 + threadIdx.x);
    if (i < vecs) st<T, VEC, true>(dst + i * VEC, ld<T, VEC, true>(src + i * VEC));
}

template <typename T, int VEC>
int run_slot_passes_vec(T* buf, int64_t elems, const trivance_plan_t* p, T* ws, hipStream_t stream,
                    int pb, int pe) {
    const Exec x{stream, p->dispatch_items};
    SlotArgs a;
    std::memset(&a, 0, sizeof(a));
    a.elems = elems;
    a.n = p->n;
    a.D = p->D;
    a.slot_stride = (int64_t)p->n * elems;
    const int64_t G = (elems + kGranule - 1) / kGranule;
    int64_t max_seg = 0;
    for (int c = 0; c <= p->D; ++c) a.seg_g[c] = (int64_t)c * G / p->D;
    for (int c = 0; c < p->D; ++c)
        max_seg = std::max(max_seg, std::min(a.seg_g[c + 1] * kGranule, elems) -
                                        std::min(a.seg_g[c] * kGranule, elems));
    const int64_t vecs = (max_seg + VEC - 1) / VEC;
    const int64_t blocks = std::max<int64_t>(1, (vecs + 64 * kSlotChunks - 1) / (64 * kSlotChunks));
    a.colblocks = (uint32_t)((blocks + kSlotGroup - 1) / kSlotGroup);  // groups of column blocks
    const int64_t units = (int64_t)p->D * p->n * a.colblocks * kSlotGroup;
    if (units >= ((int64_t)1 << 31) - 64 * kSlotWaves) return TRIVANCE_EUNSUPPORTED;
    a.units = (uint32_t)units;
    a.per_coll = (uint32_t)((int64_t)p->n * a.colblocks * kSlotGroup);
    a.f_per_coll = make_fastdiv32(a.per_coll);
    a.f_colblocks = make_fastdiv32(a.colblocks);
    const int64_t half = (int64_t)p->max_slots * a.slot_stride;
    const int S = p->S;
    for (int pi = pb; pi < pe; ++pi) {
        const Pass& ps = p->passes[pi];
        const SlotPass& sp = p->slots[pi];
        a.keep = keep_stores(p, elems, pi);
        for (int c = 0; c < p->D; ++c) {
            a.act[c] = ps.dim[c];
            a.dist[c] = ps.distance[c];
            a.nout[c] = sp.nout[c];
            int g = p->dims[ps.dim[c]], h = ps.distance[c];  // gcd(side, distance)
            while (h) {
                const int t = g % h;
                g = h;
                h = t;
            }
            a.cycle[c] = p->dims[ps.dim[c]] / g;
            a.gcyc[c] = g;
            a.f_cycle[c] = make_fastdiv32((uint32_t)a.cycle[c]);
            a.f_gcyc[c] = make_fastdiv32((uint32_t)g);
            for (int i = 0; i < kMaxSlots; ++i) {
                a.own[c][i] = sp.own[c][i];
                a.left[c][i] = sp.left[c][i];
                a.right[c][i] = sp.right[c][i];
            }
        }
        for (int d = 0; d < kMaxDims; ++d) {
            a.side[d] = d < p->D ? p->dims[d] : 1;
            a.stride[d] = d < p->D ? p->strides[d] : 1;
            a.f_side[d] = make_fastdiv32((uint32_t)a.side[d]);
            a.f_stride[d] = make_fastdiv32((uint32_t)a.stride[d]);
        }
        int most = 0;  // output partials of the pass, most over the collectives
        for (int c = 0; c < p->D; ++c) most = std::max(most, a.nout[c]);
        const bool small = pi > 0 && most <= kSlotBatchSmall &&
                           trivance_pass_bytes(p, elems, TRIVANCE_F32, pi) <= kSmallSlotPassBytes;
        const T* in = pi == 0 ? buf : ws + ((pi - 1) % 2) * half;
        T* out = (pi == S - 1 && S > 1) ? buf : ws + (pi % 2) * half;
        hipError_t err = hipSuccess;
        const uint64_t wgs = ((uint64_t)a.units + kSlotWaves - 1) / kSlotWaves;
        for_each_dispatch(wgs, 64 * kSlotWaves, x.items, [&](uint32_t first, uint32_t count) {
            a.wg_base = first;
            if (small)
                hipLaunchKernelGGL((slot_step_kernel<T, VEC, kSlotBatchSmall>), dim3(count),
                                   dim3(64 * kSlotWaves), 0, x.stream, out, in, a);
            else
                hipLaunchKernelGGL((slot_step_kernel<T, VEC, kSlotBatch>), dim3(count),
                                   dim3(64 * kSlotWaves), 0, x.stream, out, in, a);
            err = hipGetLastError();
            return err == hipSuccess;
        });
        if (err != hipSuccess) return TRIVANCE_EHIP;
        if (S == 1) {
            // the one pass wrote its result to half 0: copy it back with a kernel (no runtime
            // copy, so that the whole call is kernel launches, also under stream capture)
            const int64_t vecs = a.slot_stride / VEC;  // slot_stride = n * elems, VEC | elems
            for_each_dispatch(((uint64_t)vecs + 255) / 256, 256, x.items,
                              [&](uint32_t first, uint32_t count) {
                hipLaunchKernelGGL((copy_rows_kernel<T, VEC>), dim3(count), dim3(256), 0,
                                   x.stream, buf, ws, vecs, (uint64_t)first);
                err = hipGetLastError();
                return err == hipSuccess;
            });
            if (err != hipSuccess) return TRIVANCE_EHIP;
        }
    }
    return TRIVANCE_OK;
}

}  // namespace

// Workspace halves of a slot plan: state t (0 < t < S) lives in half (t - 1) % 2; a one-pass plan
// writes its result to half 0 and copies it back (input and output must not alias).
int slot_halves(const trivance_plan_t* p) { return p->S >= 3 ? 2 : (p->S >= 1 ? 1 : 0); }

template <typename T>
static int run_slot(T* buf, int64_t elems, const trivance_plan_t* p, T* ws, hipStream_t stream,
                    int pb, int pe) {
    if (elems % 4 == 0 && (uintptr_t)buf % 16 == 0 && (uintptr_t)ws % 16 == 0)
        return run_slot_passes_vec<T, 4>(buf, elems, p, ws, stream, pb, pe);
    return run_slot_passes_vec<T, 1>(buf, elems, p, ws, stream, pb, pe);
}

int run_slot_passes(float* buf, int64_t elems, const trivance_plan_t* p, float* ws,
                    hipStream_t stream, int pb, int pe) {
    return run_slot(buf, elems, p, ws, stream, pb, pe);
}

int run_slot_passes(int* buf, int64_t elems, const trivance_plan_t* p, int* ws, hipStream_t stream,
                    int pb, int pe) {
    return run_slot(buf, elems, p, ws, stream, pb, pe);
}

}  // namespace trivance
