// Device-side building blocks shared by the step kernels (executor.hip, slot.hip): vectors of
// elements, 16-byte loads and stores, the joint reduction in its fixed order, and the XCD-aware
// workgroup order.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "plan.h"

namespace trivance {

// x / d for x < 2^31 with the multiplier of make_fastdiv32 (plan.h).
__device__ __forceinline__ uint32_t fdiv32(uint32_t x, FastDiv32 f) {
    return __umulhi(x << 1, f.mul) >> f.shift;
}

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
using Native = T __attribute__((ext_vector_type(N)));

// 16-byte (or element) load/store; NT selects the non-temporal (streaming) cache policy.
template <typename T, int N, bool NT = false>
__device__ __forceinline__ Vec<T, N> ld(const T* p) {
    Vec<T, N> r;
    if constexpr (N == 1) {
        r.v[0] = NT ? __builtin_nontemporal_load(p) : *p;
    } else {
        const Native<T, N>* q = reinterpret_cast<const Native<T, N>*>(p);
        const Native<T, N> x = NT ? __builtin_nontemporal_load(q) : *q;
#pragma unroll
        for (int i = 0; i < N; ++i) r.v[i] = x[i];
    }
    return r;
}

template <typename T, int N, bool NT = false>
__device__ __forceinline__ void st(T* p, const Vec<T, N>& v) {
    if constexpr (N == 1) {
        if (NT) __builtin_nontemporal_store(v.v[0], p);
        else *p = v.v[0];
    } else {
        Native<T, N> x;
#pragma unroll
        for (int i = 0; i < N; ++i) x[i] = v.v[i];
        Native<T, N>* q = reinterpret_cast<Native<T, N>*>(p);
        if (NT) __builtin_nontemporal_store(x, q);
        else *q = x;
    }
}

// Store of a write-once output through a raw buffer descriptor, with one of two instruction
// cache policies chosen per pass by the host (`keep`, wave-uniform):
//  * keep = 0: NT | SC1 (streaming). Passes over gigabytes measured 1-3.5% faster this way than
//    with NT alone (global_store ... nt) on the 243-ring, the 27x27 and the 9x9x9 tori, both
//    phases, and 6-17% faster than with the default policy.
//  * keep = 1: SC1 alone. A pass whose algorithmic bytes stay within kKeepPassBytes writes about
//    the size of the 256 MB last-level (MALL) cache or less, and the next pass reads what it
//    wrote: with NT those lines leave the cache; without it the ring of 8 at 32 MiB per rank and
//    the ring of 64 at 8 MiB (bandwidth-optimal) measured 9-10% faster, and their small late
//    passes up to 20%.
typedef int BufI4 __attribute__((ext_vector_type(4)));
__device__ void raw_buffer_store_v4i32(BufI4 data, BufI4 rsrc, int voffset, int soffset,
                                       int cpol) __asm("llvm.amdgcn.raw.buffer.store.v4i32");
__device__ void raw_buffer_store_i32(int data, BufI4 rsrc, int voffset, int soffset,
                                     int cpol) __asm("llvm.amdgcn.raw.buffer.store.i32");
constexpr int kCpolStream = 2 | 16;  // NT | SC1
constexpr int kCpolKeep = 16;        // SC1
constexpr int64_t kKeepPassBytes = (int64_t)1 << 30;

// The store policy of pass `pass` of plan p over rows of `elems` elements (1: SC1 alone). Both
// element types are 4 bytes wide, so the pass's bytes do not depend on which one a call moves.
inline int keep_stores(const trivance_plan_t* p, int64_t elems, int pass) {
    return trivance_pass_bytes(p, elems, TRIVANCE_F32, pass) <= kKeepPassBytes ? 1 : 0;
}

// Raw buffer descriptor of the `bytes` bytes from the wave-uniform `base`: a lane whose byte
// offset lies beyond writes nothing (the descriptor's range check), so a ragged tail needs no
// predicate.
__device__ __forceinline__ BufI4 buffer_rsrc(const void* base, uint32_t bytes) {
    const uint64_t a = reinterpret_cast<uint64_t>(base);
    BufI4 r;
    r.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    r.y = __builtin_amdgcn_readfirstlane((int)((uint32_t)(a >> 32) & 0xFFFFu));  // stride 0
    r.z = __builtin_amdgcn_readfirstlane((int)bytes);                           // num_records
    r.w = 0x00020000;  // raw 32-bit data format (gfx9 family)
    return r;
}

// The value goes to the intrinsic as one reinterpreted vector: assembled component by component,
// the operand was compiled into one dword repeated four times by this toolchain.
template <int KEEP, typename T, int N>
__device__ __forceinline__ void st_out_as(BufI4 rsrc, uint32_t byte_offset, const Vec<T, N>& v) {
    static_assert(sizeof(T) == 4 && (N == 1 || N == 4), "32-bit elements, 4- or 16-byte stores");
    constexpr int cpol = KEEP ? kCpolKeep : kCpolStream;
    if constexpr (N == 4) {
        raw_buffer_store_v4i32(__builtin_bit_cast(BufI4, v), rsrc, (int)byte_offset, 0, cpol);
    } else {
        raw_buffer_store_i32(__builtin_bit_cast(int, v), rsrc, (int)byte_offset, 0, cpol);
    }
}

// The policy as a wave-uniform run-time flag: one scalar branch per store.
template <typename T, int N>
__device__ __forceinline__ void st_out(BufI4 rsrc, uint32_t byte_offset, const Vec<T, N>& v,
                                       int keep) {
    if (keep) st_out_as<1>(rsrc, byte_offset, v);
    else st_out_as<0>(rsrc, byte_offset, v);
}

__device__ __forceinline__ int64_t imin64(int64_t a, int64_t b) { return a < b ? a : b; }

// Workgroup index remapped so that each of the 8 XCDs (which receive workgroups round-robin)
// works on one contiguous range of units.
__device__ __forceinline__ uint32_t xcd_contiguous(uint32_t wg, uint32_t nwg) {
    constexpr uint32_t kXcds = 8;
    const uint32_t per = nwg / kXcds, rem = nwg % kXcds;
    const uint32_t xcd = wg % kXcds, idx = wg / kXcds;
    return xcd < rem ? xcd * (per + 1) + idx : rem * (per + 1) + (xcd - rem) * per + idx;
}



// Where and how a call's launches go: the stream, and the most work-items of one dispatch (the
// plan's limit).
struct Exec {
    hipStream_t stream;
    int64_t items;
};


// Latency-optimal passes on sides that are not powers of three (slot.hip): the workspace halves a
// slot plan uses, and the launcher of passes [pb, pe).
int slot_halves(const trivance_plan_t* p);
int run_slot_passes(float* buf, int64_t elems, const trivance_plan_t* p, float* ws,
                    hipStream_t stream, int pb, int pe);
int run_slot_passes(int* buf, int64_t elems, const trivance_plan_t* p, int* ws, hipStream_t stream,
                    int pb, int pe);

}  // namespace trivance
