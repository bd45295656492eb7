// Device-side helpers that are not part of the AllReduce: the benchmark's streaming copy, and
// the input generator below.
//
// Input generator: counter-based U(-1, 1) fp32 values
// from SplitMix64 (Steele, Lea, Flood, "Fast splittable pseudorandom number generators",
// OOPSLA 2014). Value i of the rank-major array (i = r * elems + e) is the k-th output of a
// SplitMix64 generator started at state 0, k = seed * 2^40 + i + 1: h = mix(k * golden_gamma);
// the top 24 bits give u = (h >> 40) * 2^-23 - 1, exactly representable in fp32.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "device.h"
#include "plan.h"

namespace trivance {
namespace {

__device__ __forceinline__ uint64_t splitmix64_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__global__ __launch_bounds__(256) void fill_hash_uniform_kernel(float* __restrict__ out,
                                                                uint64_t total, uint64_t key0) {
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
        const uint64_t h = splitmix64_mix((key0 + i + 1) * 0x9E3779B97F4A7C15ull);
        out[i] = (float)(uint32_t)(h >> 40) * 0x1p-23f - 1.0f;
    }
}

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Plain streaming copy, one 16-byte vector per lane, one-wave workgroups: the simplest kernel
// with the step kernels' access granularity, timed as the practical ceiling. Non-temporal loads,
// and the streaming store of the step kernels' large passes (st_out_as, NT | SC1), which copies
// 1 GiB 1.2% faster than a non-temporal global store.
__global__ __launch_bounds__(64) void copy_stream_kernel(const u32x4* __restrict__ src,
                                                         u32x4* __restrict__ dst, uint64_t nvec,
                                                         uint64_t wg_base) {
    const uint64_t w0 = (wg_base + blockIdx.x) * 64;  // this wave's first vector
    if (w0 >= nvec) return;
    const uint64_t i = w0 + threadIdx.x;
    const uint64_t here = nvec - w0 < 64 ? nvec - w0 : 64;
    const BufI4 r = buffer_rsrc(dst + w0, (uint32_t)(here * sizeof(u32x4)));
    if (i < nvec) {
        const u32x4 x = __builtin_nontemporal_load(src + i);
        st_out_as<0>(r, threadIdx.x * (uint32_t)sizeof(u32x4),
                     __builtin_bit_cast(Vec<uint32_t, 4>, x));
    }
}

}  // namespace
}  // namespace trivance

extern "C" int trivance_copy_device(void* dst, const void* src, int64_t bytes, void* stream) {
    if (bytes < 0 || bytes % 16 != 0) return TRIVANCE_EINVAL;
    if (bytes == 0) return TRIVANCE_OK;
    if (!dst || !src || reinterpret_cast<uintptr_t>(dst) % 16 != 0 ||
        reinterpret_cast<uintptr_t>(src) % 16 != 0)
        return TRIVANCE_EINVAL;
    const uint64_t nvec = (uint64_t)bytes / 16;
    const char* s = static_cast<const char*>(src);
    char* d = static_cast<char*>(dst);
    if (s < d + bytes && d < s + bytes) return TRIVANCE_EINVAL;  // overlapping ranges
    hipError_t err = hipSuccess;
    trivance::for_each_dispatch((nvec + 63) / 64, 64, trivance::kMaxDispatchItems,
                                [&](uint32_t first, uint32_t count) {
        hipLaunchKernelGGL(trivance::copy_stream_kernel, dim3(count), dim3(64), 0,
                           reinterpret_cast<hipStream_t>(stream),
                           static_cast<const trivance::u32x4*>(src),
                           static_cast<trivance::u32x4*>(dst), nvec, (uint64_t)first);
        err = hipGetLastError();
        return err == hipSuccess;
    });
    return err == hipSuccess ? TRIVANCE_OK : TRIVANCE_EHIP;
}

extern "C" int trivance_fill_hash_uniform(void* buffers, int n, int64_t elems, uint64_t seed,
                                          void* stream) {
    if (n < 0 || elems < 0) return TRIVANCE_EINVAL;
    const uint64_t total = (uint64_t)n * (uint64_t)elems;
    if (total == 0) return TRIVANCE_OK;
    if (!buffers) return TRIVANCE_EINVAL;
    uint64_t blocks = (total + 255) / 256;
    if (blocks > 65536ull * 8) blocks = 65536ull * 8;
    hipLaunchKernelGGL(trivance::fill_hash_uniform_kernel, dim3((uint32_t)blocks), dim3(256), 0,
                       reinterpret_cast<hipStream_t>(stream), static_cast<float*>(buffers), total,
                       seed << 40);
    return hipGetLastError() == hipSuccess ? TRIVANCE_OK : TRIVANCE_EHIP;
}
