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
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "plan.h"

namespace trivance {
namespace {

constexpr int kBlockThreads = 256;
constexpr int kWavesPerBlock = kBlockThreads / 64;

struct StepArgs {
    int64_t elems;                 // elements per rank row
    int64_t seg_g[kMaxDims + 1];   // segment granule starts, seg_g[D] = total granules
    int n;
    int D;
    int dims[kMaxDims];
    int strides[kMaxDims];
    int act_dim[kMaxDims];         // active dimension per collective
    int modulus[kMaxDims][kMaxDims];
    int distance;
    // latency step
    int ncycles;                   // cycles per collective
    int colblocks;                 // thread blocks per (collective, cycle)
    // block steps
    int kept;                      // blocks kept per rank: n / 3^(t+1)
    int cpb;                       // chunks per block
    uint32_t units_per_coll;       // n * kept * cpb
    uint32_t total_units;          // D * units_per_coll
    int narrow;                    // 1 if n * (granules per segment) < 2^32
};

template <typename T, int N>
struct alignas(sizeof(T) * N) Vec {
    T v[N];
};

__device__ __forceinline__ float add1(float a, float b) { return a + b; }
__device__ __forceinline__ int add1(int a, int b) {
    return (int)((unsigned)a + (unsigned)b);  // two's-complement wrap
}

template <typename T, int N>
__device__ __forceinline__ Vec<T, N> vadd(const Vec<T, N>& a, const Vec<T, N>& b) {
    Vec<T, N> r;
#pragma unroll
    for (int i = 0; i < N; ++i) r.v[i] = add1(a.v[i], b.v[i]);
    return r;
}

// Joint reduction of Sec. 4.3 in the fixed order (own + left) + right.
template <typename T, int N>
__device__ __forceinline__ Vec<T, N> joint(const Vec<T, N>& own, const Vec<T, N>& left,
                                           const Vec<T, N>& right) {
    return vadd(vadd(own, left), right);
}

template <typename T, int N>
__device__ __forceinline__ Vec<T, N> ld(const T* p) {
    return *reinterpret_cast<const Vec<T, N>*>(p);
}

template <typename T, int N>
__device__ __forceinline__ void st(T* p, const Vec<T, N>& v) {
    *reinterpret_cast<Vec<T, N>*>(p) = v;
}

__device__ __forceinline__ int64_t imin64(int64_t a, int64_t b) { return a < b ? a : b; }

// ---------------------------------------------------------------------------------------------
// Latency-optimal step: sliding window over one rank cycle.
// Grid: D * ncycles * colblocks thread blocks; each thread owns VPT column vectors.
template <typename T, int VEC, int VPT>
__global__ __launch_bounds__(kBlockThreads) void latency_step_kernel(T* __restrict__ buf,
                                                                     StepArgs a) {
    using V = Vec<T, VEC>;
    const uint32_t wg = blockIdx.x;
    const uint32_t cb = wg % (uint32_t)a.colblocks;
    const uint32_t rest = wg / (uint32_t)a.colblocks;
    const int cyc = (int)(rest % (uint32_t)a.ncycles);
    const int c = (int)(rest / (uint32_t)a.ncycles);

    const int dim = a.act_dim[c];
    const int side = a.dims[dim];
    const int stride = a.strides[dim];
    const int dist = a.distance;
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
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
        const int64_t v = ((int64_t)cb * VPT + u) * kBlockThreads + threadIdx.x;
        ok[u] = v < nvec;
        col[u] = base + v * VEC;
    }

    V first[VPT], last[VPT], prev[VPT], a0[VPT], a1[VPT], a2[VPT];
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
        if (ok[u]) {
            last[u] = ld<T, VEC>(col[u] + (int64_t)(len - 1) * rowstep);
            first[u] = ld<T, VEC>(col[u]);
            a1[u] = ld<T, VEC>(col[u] + rowstep);
            a2[u] = len == 3 ? last[u] : ld<T, VEC>(col[u] + 2 * rowstep);
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
                    b0[u] = ld<T, VEC>(col[u] + (int64_t)(i + 3) * rowstep);
                    b1[u] = ld<T, VEC>(col[u] + (int64_t)(i + 4) * rowstep);
                    b2[u] = (i + 5 == len - 1) ? last[u]
                                               : ld<T, VEC>(col[u] + (int64_t)(i + 5) * rowstep);
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
                T* p = col[u] + (int64_t)i * rowstep;
                st<T, VEC>(p, joint(a0[u], prev[u], a1[u]));
                st<T, VEC>(p + rowstep, joint(a1[u], a0[u], a2[u]));
                st<T, VEC>(p + 2 * rowstep, joint(a2[u], a1[u], b0[u]));
                prev[u] = a2[u];
                a0[u] = b0[u];
                a1[u] = b1[u];
                a2[u] = b2[u];
            }
        }
    }
}

// ---------------------------------------------------------------------------------------------
// Decode of a block-step work unit (all values wave-uniform).
struct Unit {
    int64_t begin, end;  // element range of this unit's chunk (begin < end when active)
    int rank, left, right;
};

__device__ __forceinline__ bool decode_unit(const StepArgs& a, uint32_t unit, int chunk_elems,
                                            Unit* out) {
    const uint32_t c = unit / a.units_per_coll;
    const uint32_t rem = unit - c * a.units_per_coll;
    const uint32_t pair = rem / (uint32_t)a.cpb;
    const int chunk = (int)(rem - pair * (uint32_t)a.cpb);
    const int r = (int)(pair / (uint32_t)a.kept);
    int q = (int)(pair - (uint32_t)r * (uint32_t)a.kept);
    const int act = a.act_dim[c];

    int j = 0, rr = r, r_act = 0;
#pragma unroll
    for (int d = 0; d < kMaxDims; ++d) {
        if (d < a.D) {
            const int side = a.dims[d];
            const int rd = rr % side;
            rr /= side;
            const int K = a.modulus[c][d];
            const int nq = side / K;
            const int qd = q % nq;
            q /= nq;
            j += (rd % K + K * qd) * a.strides[d];
            if (d == act) r_act = rd;
        }
    }
    const int side = a.dims[act];
    const int st = a.strides[act];
    const int dist = a.distance;
    out->rank = r;
    out->left = r_act >= dist ? r - dist * st : r + (side - dist) * st;
    out->right = r_act + dist < side ? r + dist * st : r - (side - dist) * st;

    const int64_t g0 = a.seg_g[c];
    const int64_t Gc = a.seg_g[c + 1] - g0;
    int64_t gb, ge;
    if (a.narrow) {
        gb = g0 + (int64_t)((uint32_t)j * (uint32_t)Gc / (uint32_t)a.n);
        ge = g0 + (int64_t)((uint32_t)(j + 1) * (uint32_t)Gc / (uint32_t)a.n);
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

template <typename T, int VEC, int U, bool REDUCE>
__global__ __launch_bounds__(kBlockThreads) void block_step_kernel(T* __restrict__ buf,
                                                                   StepArgs a) {
    using V = Vec<T, VEC>;
    constexpr int kChunk = 64 * VEC * U;
    const int lane = threadIdx.x & 63;
    const uint32_t wave = (uint32_t)__builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const uint32_t unit = blockIdx.x * (uint32_t)kWavesPerBlock + wave;
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
    if constexpr (REDUCE) {
        V x[U], y[U], z[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (ok[u]) {
                x[u] = ld<T, VEC>(own + idx[u]);
                y[u] = ld<T, VEC>(pl + idx[u]);
                z[u] = ld<T, VEC>(pr + idx[u]);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (ok[u]) st<T, VEC>(own + idx[u], joint(x[u], y[u], z[u]));
    } else {
        V x[U];
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (ok[u]) x[u] = ld<T, VEC>(own + idx[u]);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (ok[u]) {
                st<T, VEC>(pl + idx[u], x[u]);
                st<T, VEC>(pr + idx[u], x[u]);
            }
        }
    }
}

// ---------------------------------------------------------------------------------------------
// Host side.

constexpr int kLatencyVPT = 1;

template <typename T, int VEC>
hipError_t launch_pass(T* buf, const StepArgs& a0, int phase, int max_blk_elems,
                       hipStream_t stream) {
    StepArgs a = a0;
    if (phase == TRIVANCE_PHASE_LATENCY) {
        int64_t max_seg = 0;
        for (int c = 0; c < a.D; ++c) {
            const int64_t b = std::min(a.seg_g[c] * kGranule, a.elems);
            const int64_t e = std::min(a.seg_g[c + 1] * kGranule, a.elems);
            max_seg = std::max(max_seg, e - b);
        }
        const int64_t max_vec = (max_seg + VEC - 1) / VEC;
        const int64_t per_block = (int64_t)kBlockThreads * kLatencyVPT;
        a.colblocks = (int)((max_vec + per_block - 1) / per_block);
        if (a.colblocks < 1) a.colblocks = 1;
        const int64_t grid = (int64_t)a.D * a.ncycles * a.colblocks;
        if (grid >= (int64_t)1 << 31) return hipErrorInvalidConfiguration;
        hipLaunchKernelGGL((latency_step_kernel<T, VEC, kLatencyVPT>), dim3((uint32_t)grid),
                           dim3(kBlockThreads), 0, stream, buf, a);
        return hipGetLastError();
    }
    // chunk size: four 16-byte vectors per lane for large blocks, fewer for small ones
    int U = 4;
    if (max_blk_elems <= 64 * VEC) U = 1;
    else if (max_blk_elems <= 2 * 64 * VEC) U = 2;
    const int chunk = 64 * VEC * U;
    a.cpb = (max_blk_elems + chunk - 1) / chunk;
    if (a.cpb < 1) a.cpb = 1;
    const int64_t upc = (int64_t)a.n * a.kept * a.cpb;
    const int64_t total = upc * a.D;
    if (total >= ((int64_t)1 << 32) - kWavesPerBlock) return hipErrorInvalidConfiguration;
    a.units_per_coll = (uint32_t)upc;
    a.total_units = (uint32_t)total;
    const uint32_t grid = (uint32_t)((total + kWavesPerBlock - 1) / kWavesPerBlock);
    const bool rs = phase == TRIVANCE_PHASE_REDUCE_SCATTER;
#define TRIVANCE_LAUNCH_BLOCK(UU)                                                              \
    if (rs)                                                                                    \
        hipLaunchKernelGGL((block_step_kernel<T, VEC, UU, true>), dim3(grid),                  \
                           dim3(kBlockThreads), 0, stream, buf, a);                            \
    else                                                                                       \
        hipLaunchKernelGGL((block_step_kernel<T, VEC, UU, false>), dim3(grid),                 \
                           dim3(kBlockThreads), 0, stream, buf, a);
    if (U == 4) {
        TRIVANCE_LAUNCH_BLOCK(4)
    } else if (U == 2) {
        TRIVANCE_LAUNCH_BLOCK(2)
    } else {
        TRIVANCE_LAUNCH_BLOCK(1)
    }
#undef TRIVANCE_LAUNCH_BLOCK
    return hipGetLastError();
}

template <typename T>
int run_passes(T* buf, int64_t elems, const trivance_plan_t* p, hipStream_t stream, int pb,
               int pe) {
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
    a.narrow = (int64_t)p->n * (max_gc + 1) < ((int64_t)1 << 32) ? 1 : 0;
    const int64_t max_blk = max_block_granules(p, elems) * kGranule;
    if (max_blk >= ((int64_t)1 << 31)) return TRIVANCE_EUNSUPPORTED;

    const bool vec4 = (elems % 4 == 0) && ((uintptr_t)buf % 16 == 0);
    for (int pi = pb; pi < pe; ++pi) {
        const Pass& ps = p->passes[pi];
        a.distance = ps.distance;
        for (int c = 0; c < kMaxDims; ++c) {
            a.act_dim[c] = ps.dim[c];
            for (int d = 0; d < kMaxDims; ++d) a.modulus[c][d] = ps.modulus[c][d];
        }
        const int side = p->dims[ps.dim[0]];
        a.ncycles = (p->n / side) * ps.distance;
        a.kept = (int)ps.kept_per_rank;
        const hipError_t err = vec4 ? launch_pass<T, 4>(buf, a, ps.phase, (int)max_blk, stream)
                                    : launch_pass<T, 1>(buf, a, ps.phase, (int)max_blk, stream);
        if (err == hipErrorInvalidConfiguration) return TRIVANCE_EUNSUPPORTED;
        if (err != hipSuccess) return TRIVANCE_EHIP;
    }
    return TRIVANCE_OK;
}

}  // namespace
}  // namespace trivance

extern "C" {

int trivance_allreduce_emulated_steps(void* buffers, int n, int64_t elems, int dtype,
                                      const trivance_plan_t* plan, void* stream, int pass_begin,
                                      int pass_end) {
    if (!plan || n != plan->n || elems < 0) return TRIVANCE_EINVAL;
    if (dtype != TRIVANCE_F32 && dtype != TRIVANCE_I32) return TRIVANCE_EINVAL;
    const int np = (int)plan->passes.size();
    if (pass_begin < 0 || pass_end < pass_begin || pass_end > np) return TRIVANCE_EINVAL;
    if (plan->variant == TRIVANCE_BRUCK_REF) return TRIVANCE_EUNSUPPORTED;
    if (elems == 0 || pass_begin == pass_end) return TRIVANCE_OK;
    if (!buffers) return TRIVANCE_EINVAL;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    if (dtype == TRIVANCE_F32)
        return trivance::run_passes<float>(static_cast<float*>(buffers), elems, plan, s,
                                           pass_begin, pass_end);
    return trivance::run_passes<int>(static_cast<int*>(buffers), elems, plan, s, pass_begin,
                                     pass_end);
}

int trivance_allreduce_emulated(void* buffers, int n, int64_t elems, int dtype,
                                const trivance_plan_t* plan, void* stream) {
    if (!plan) return TRIVANCE_EINVAL;
    return trivance_allreduce_emulated_steps(buffers, n, elems, dtype, plan, stream, 0,
                                             (int)plan->passes.size());
}

}  // extern "C"
