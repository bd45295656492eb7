// Per-link congestion counter of a Trivance (or Bruck comparison) schedule, on the GPU.
//
// Sec. 2.1: the congestion of a step is the number of chunks (messages) sharing a link. The
// network is a ring or torus with one port per direction and dimension; every transmission stays
// inside one dimension (Appendix E). In each pass every rank sends, for every collective, one
// message per offset along that collective's active dimension: offsets -3^k and +3^k for
// Trivance (Sec. 4.1), +3^k and +2*3^k for the Bruck comparison pattern (Sec. 2.4, Fig. 1).
// With a side that is not a power of three (Sec. 4.4) a step's distance is the tree's, and a
// rank sends towards a side only when some child of the active dimension's tree does so at that
// step (every rank then does, the trees being the same relative to every block).
//
// One 64-thread workgroup handles one (pass, dimension, line) triple, a line being the ring of
// ranks that differ only in that dimension's coordinate (dimensions with longer sides have fewer
// lines; their surplus workgroups exit at once). Each message adds +1 over a cyclic range
// of directed links; the workgroup records the range ends in an LDS difference array (plus a
// count of ranges that wrap past position 0) and turns it into per-link loads with a wavefront
// inclusive scan. Every output entry is written, so no clearing pass is needed.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "plan.h"

// Device scratch of the allocation-free form, trivance_congestion_noalloc: the loads are computed
// into it and copied to the caller's host array. Every GPU the library runs on holds its own copy
// until the process ends. In host code `scratch` names a host-side stand-in, not device memory:
// its device address is taken per device with hipGetSymbolAddress (scratch_address below) and only
// that address is used.
constexpr int64_t kScratchEntries = (int64_t)1 << 20;  // 8 MiB of int64 loads
static __device__ __align__(256) int64_t scratch[kScratchEntries];

namespace trivance {
namespace {

constexpr int kMaxPasses = 40;
constexpr int kMaxSide = 6561;  // LDS: two difference arrays of side + 1 ints

struct CongArgs {
    int n;
    int D;
    int npasses;
    int bruck;
    int shortest;
    int max_lines;  // lines of the dimension with the smallest side: n / min side
    int dims[kMaxDims];
    int strides[kMaxDims];
    int16_t distance[kMaxPasses][kMaxDims];  // per pass and collective (at most kMaxSide / 2)
    uint8_t dirs[kMaxPasses][kMaxDims];     // per pass and collective: bit 0 messages towards +, bit 1 towards -
    uint8_t act_dim[kMaxPasses][kMaxDims];
    uint32_t wg_base;  // first workgroup of this dispatch (for_each_dispatch)
};

// Direction (+1 / -1) and hop count of a message over `offset` on a ring of `side` nodes.
__device__ __forceinline__ void route(int offset, int side, bool shortest, int* dir, int* hops) {
    int fwd = offset % side;
    if (fwd < 0) fwd += side;
    if (fwd == 0) {
        *dir = 1;
        *hops = 0;
        return;
    }
    const int back = side - fwd;
    if (!shortest) {
        *dir = offset > 0 ? 1 : -1;
        *hops = offset > 0 ? offset : -offset;
        return;
    }
    if (fwd < back) {
        *dir = 1;
        *hops = fwd;
    } else if (back < fwd) {
        *dir = -1;
        *hops = back;
    } else {
        *dir = offset > 0 ? 1 : -1;
        *hops = fwd;
    }
}

// +1 on the cyclic link range [s, s + len) of a line with `side` positions.
__device__ __forceinline__ void add_range(int* diff, int* wraps, int s, int len, int side) {
    const int e = s + len;
    atomicAdd(&diff[s], 1);
    if (e <= side) {
        atomicAdd(&diff[e], -1);  // diff[side] is a sentinel, never read back
    } else {
        atomicAdd(wraps, 1);
        atomicAdd(&diff[e - side], -1);
    }
}

__global__ __launch_bounds__(64) void congestion_kernel(int64_t* __restrict__ loads, CongArgs a) {
    extern __shared__ int lds[];
    const int lane = threadIdx.x;
    const uint32_t wg = a.wg_base + blockIdx.x;
    const int line = (int)(wg % (uint32_t)a.max_lines);
    const uint32_t rest = wg / (uint32_t)a.max_lines;
    const int dim = (int)(rest % (uint32_t)a.D);
    const int pass = (int)(rest / (uint32_t)a.D);

    const int side = a.dims[dim];
    const int stride = a.strides[dim];
    if (line >= a.n / side) return;  // this dimension has fewer lines (unequal sides)
    const int line_base = (line % stride) + (line / stride) * stride * side;
    int* plus = lds;               // side + 1 entries
    int* minus = lds + side + 1;   // side + 1 entries
    int* wraps = lds + 2 * side + 2;  // [0] plus, [1] minus

    for (int x = lane; x < 2 * side + 4; x += 64) lds[x] = 0;
    __syncthreads();

    for (int x = lane; x < side; x += 64) {
        for (int c = 0; c < a.D; ++c) {
            if (a.act_dim[pass][c] != dim) continue;
            const int dist = a.distance[pass][c];
            const int off0 = a.bruck ? dist : -dist;
            const int off1 = a.bruck ? 2 * dist : dist;
            for (int m = 0; m < 2; ++m) {
                if (!a.bruck && !(a.dirs[pass][c] & (m == 0 ? 2 : 1))) continue;
                int dir, hops;
                route(m == 0 ? off0 : off1, side, a.shortest != 0, &dir, &hops);
                if (hops == 0) continue;
                if (dir > 0) {
                    add_range(plus, &wraps[0], x, hops, side);
                } else {
                    // links leaving x, x-1, ..., x-hops+1 towards -dim
                    int s = x - hops + 1;
                    if (s < 0) s += side;
                    add_range(minus, &wraps[1], s, hops, side);
                }
            }
        }
    }
    __syncthreads();

    const int port_plus = 2 * dim;
    const int64_t row = (int64_t)pass * a.n;
    for (int sgn = 0; sgn < 2; ++sgn) {
        const int* diff = sgn == 0 ? plus : minus;
        int carry = wraps[sgn];
        for (int x0 = 0; x0 < side; x0 += 64) {
            const int x = x0 + lane;
            int v = x < side ? diff[x] : 0;
#pragma unroll
            for (int off = 1; off < 64; off <<= 1) {
                const int t = __shfl_up(v, off, 64);
                if (lane >= off) v += t;
            }
            if (x < side) {
                const int rank = line_base + x * stride;
                loads[(row + rank) * (2 * a.D) + port_plus + sgn] = (int64_t)(carry + v);
            }
            carry += __shfl(v, 63, 64);
        }
    }
}

}  // namespace
}  // namespace trivance

using trivance::CongArgs;

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
int64_t* g_scratch[kMaxDevices] = {};

// Device address of `scratch` on the current device, looked up once per device with that device
// current.
int scratch_address(int64_t** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return TRIVANCE_EHIP;
    if (dev < 0 || dev >= kMaxDevices) return TRIVANCE_EUNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch[dev]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr)
            return TRIVANCE_EHIP;
        g_scratch[dev] = static_cast<int64_t*>(ptr);
    }
    *out = g_scratch[dev];
    return TRIVANCE_OK;
}

}  // namespace

extern "C" {

int trivance_congestion_device(const trivance_plan_t* plan, const trivance_topology* topo,
                               int64_t* loads_dev, int64_t loads_len, void* stream) {
    if (!plan) return TRIVANCE_EINVAL;
    int routing = TRIVANCE_ROUTE_SCHEDULED;
    if (topo) {
        if (topo->ndims != plan->D) return TRIVANCE_EINVAL;
        for (int d = 0; d < plan->D; ++d)
            if (topo->dims[d] != plan->dims[d]) return TRIVANCE_EINVAL;
        if (topo->routing != TRIVANCE_ROUTE_SCHEDULED && topo->routing != TRIVANCE_ROUTE_SHORTEST)
            return TRIVANCE_EINVAL;
        routing = topo->routing;
    }
    const int P = (int)plan->passes.size();
    const int64_t need = (int64_t)P * plan->n * 2 * plan->D;
    if (loads_len < need) return TRIVANCE_ESIZE;
    if (need == 0) return TRIVANCE_OK;
    if (!loads_dev) return TRIVANCE_EINVAL;
    if (P > trivance::kMaxPasses) return TRIVANCE_EUNSUPPORTED;
    for (int d = 0; d < plan->D; ++d)
        if (plan->dims[d] > trivance::kMaxSide) return TRIVANCE_EUNSUPPORTED;

    CongArgs a{};
    a.n = plan->n;
    a.D = plan->D;
    a.npasses = P;
    a.bruck = plan->variant == TRIVANCE_BRUCK_REF ? 1 : 0;
    a.shortest = routing == TRIVANCE_ROUTE_SHORTEST ? 1 : 0;
    int min_side = plan->dims[0];
    for (int d = 1; d < plan->D; ++d) min_side = plan->dims[d] < min_side ? plan->dims[d] : min_side;
    a.max_lines = plan->n / min_side;
    for (int d = 0; d < trivance::kMaxDims; ++d) {
        a.dims[d] = d < plan->D ? plan->dims[d] : 1;
        a.strides[d] = d < plan->D ? plan->strides[d] : 1;
    }
    int max_side = 1;
    for (int d = 0; d < plan->D; ++d) max_side = plan->dims[d] > max_side ? plan->dims[d] : max_side;
    for (int p = 0; p < P; ++p) {
        for (int c = 0; c < trivance::kMaxDims; ++c) {
            a.act_dim[p][c] = (uint8_t)plan->passes[p].dim[c];
            a.distance[p][c] = (int16_t)plan->passes[p].distance[c];
        }
        for (int c = 0; c < trivance::kMaxDims; ++c) {
            a.dirs[p][c] = 3;
            if (!plan->slots.empty() && c < plan->D) {
                // latency-optimal slot programs: a rank sends towards + when some slot takes a
                // part from the peer at -distance, towards - when some slot takes one from +
                const trivance::SlotPass& sp = plan->slots[p];
                int m = 0;
                for (int i = 0; i < sp.nout[c]; ++i) {
                    if (sp.left[c][i] >= 0) m |= 1;
                    if (sp.right[c][i] >= 0) m |= 2;
                }
                a.dirs[p][c] = (uint8_t)m;
            }
            if (plan->tree && c < plan->D) {
                // a reduce-scatter step sends child -> parent (every rank sends towards a side
                // when any offset of the active dimension's tree does); its all-gather step
                // retraces the messages, so the directions swap
                const trivance::Pass& ps = plan->passes[p];
                const int m = plan->trees[ps.dim[c]].dirs[ps.dim_step[c]];
                a.dirs[p][c] = (uint8_t)(ps.phase == TRIVANCE_PHASE_REDUCE_SCATTER
                                             ? m : (((m & 1) << 1) | ((m & 2) >> 1)));
            }
        }
    }
    const int64_t grid = (int64_t)P * plan->D * a.max_lines;
    if (grid >= ((int64_t)1 << 31)) return TRIVANCE_EUNSUPPORTED;
    const size_t lds = (size_t)(2 * max_side + 4) * sizeof(int);
    const bool ok = trivance::for_each_dispatch((uint64_t)grid, 64, plan->dispatch_items,
                                                [&](uint32_t first, uint32_t count) {
        a.wg_base = first;
        hipLaunchKernelGGL(trivance::congestion_kernel, dim3(count), dim3(64), lds,
                           reinterpret_cast<hipStream_t>(stream), loads_dev, a);
        return hipGetLastError() == hipSuccess;
    });
    return ok ? TRIVANCE_OK : TRIVANCE_EHIP;
}

int64_t trivance_congestion(const trivance_plan_t* plan, const trivance_topology* topo,
                            int64_t* loads, int64_t loads_len) {
    if (!plan) return TRIVANCE_EINVAL;
    const int64_t need = (int64_t)plan->passes.size() * plan->n * 2 * plan->D;
    if (!loads) return need;
    if (loads_len < need) return TRIVANCE_ESIZE;
    if (need == 0) return TRIVANCE_OK;
    int64_t* dev = nullptr;
    if (hipMalloc(reinterpret_cast<void**>(&dev), need * sizeof(int64_t)) != hipSuccess)
        return TRIVANCE_EHIP;
    int rc = trivance_congestion_device(plan, topo, dev, need, nullptr);
    if (rc == TRIVANCE_OK) {
        if (hipMemcpy(loads, dev, need * sizeof(int64_t), hipMemcpyDeviceToHost) != hipSuccess)
            rc = TRIVANCE_EHIP;
    }
    if (hipFree(dev) != hipSuccess && rc == TRIVANCE_OK) rc = TRIVANCE_EHIP;
    return rc;
}

int64_t trivance_congestion_noalloc(const trivance_plan_t* plan, const trivance_topology* topo,
                                    int64_t* loads, int64_t loads_len) {
    if (!plan) return TRIVANCE_EINVAL;
    const int64_t need = (int64_t)plan->passes.size() * plan->n * 2 * plan->D;
    if (!loads) return need;
    if (loads_len < need) return TRIVANCE_ESIZE;
    if (need == 0) return TRIVANCE_OK;
    if (need > kScratchEntries) return TRIVANCE_ESCRATCH;
    int64_t* dev = nullptr;
    int rc = scratch_address(&dev);
    if (rc != TRIVANCE_OK) return rc;
    // the kernel writes every entry of [0, need), so the scratch needs no clearing
    rc = trivance_congestion_device(plan, topo, dev, need, nullptr);
    if (rc != TRIVANCE_OK) return rc;
    if (hipMemcpy(loads, dev, need * sizeof(int64_t), hipMemcpyDeviceToHost) != hipSuccess)
        return TRIVANCE_EHIP;
    return TRIVANCE_OK;
}

}  // extern "C"
