// f2probe.hip -- ceiling probes for the roofline figures (gfx950): a streaming
// non-temporal copy (achievable HBM bandwidth), a run of independent 32-bit bitwise VALU
// instructions (achievable integer issue rate), and scattered reads and writes at
// random positions of a buffer (achievable rate of the random accesses that a
// context-grouped encode makes).  Nothing here is part of the fit or the encode.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/f2probe.h"

namespace {

constexpr int kThreads = 256;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// non-temporal 16-byte loads and stores (the streamed data is not kept in the
// caches), four in flight per thread, a grid-stride loop
__global__ __launch_bounds__(kThreads) void k_probe_copy(const u32x4* __restrict__ src, u32x4* __restrict__ dst,
                                                         int64_t n16) {
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
    int64_t i = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const u32x4 a = __builtin_nontemporal_load(src + i), b = __builtin_nontemporal_load(src + i + stride);
        const u32x4 c = __builtin_nontemporal_load(src + i + 2 * stride), d = __builtin_nontemporal_load(src + i + 3 * stride);
        __builtin_nontemporal_store(a, dst + i);
        __builtin_nontemporal_store(b, dst + i + stride);
        __builtin_nontemporal_store(c, dst + i + 2 * stride);
        __builtin_nontemporal_store(d, dst + i + 3 * stride);
    }
    for (; i < n16; i += stride) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

constexpr int kVals = 16;

template <int OP>
__global__ __launch_bounds__(kThreads) void k_probe_bitops(uint32_t* out, int iters) {
    const uint32_t t = blockIdx.x * kThreads + threadIdx.x;
    uint32_t v[kVals];
#pragma unroll
    for (int k = 0; k < kVals; ++k) v[k] = t * 0x9e3779b9u + static_cast<uint32_t>(k) * 0x85ebca6bu;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int k = 0; k < kVals; ++k) {
            if constexpr (OP == 0)
                v[k] ^= v[(k + 1) & (kVals - 1)];
            else
                v[k] = __builtin_amdgcn_bitop3_b32(v[k], v[(k + 1) & (kVals - 1)], v[(k + 5) & (kVals - 1)], 0x96);
        }
    }
    uint32_t r = 0;
#pragma unroll
    for (int k = 0; k < kVals; ++k) r += v[k];
    out[t] = r;
}

// splitmix64's output function (Steele, Lea and Flood, 2014) as a position hash
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
    z += 0x9e3779b97f4a7c15ull;
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

// op 0: each thread reads 32 bytes at `per` random 32-byte slots (XOR-folded, one
// word stored per thread); op 1: each thread writes 16 bytes at `per` random
// 16-byte slots
template <int OP>
__global__ __launch_bounds__(kThreads) void k_probe_scatter(uint64_t* __restrict__ buf, int64_t slots, int per,
                                                            uint64_t* __restrict__ out) {
    const uint64_t t = static_cast<uint64_t>(blockIdx.x) * kThreads + threadIdx.x;
    uint64_t acc = 0;
    for (int r = 0; r < per; ++r) {
        const uint64_t sl = mix64(t * 64 + static_cast<uint64_t>(r)) % static_cast<uint64_t>(slots);
        if constexpr (OP == 0) {
            const u32x4* p = reinterpret_cast<const u32x4*>(buf + 4 * sl);
            const u32x4 a = p[0], b = p[1];
            acc ^= (static_cast<uint64_t>(a.x ^ b.x) << 32) | (a.y ^ a.z ^ a.w ^ b.y ^ b.z ^ b.w);
        } else {
            u32x4 v;
            v.x = static_cast<uint32_t>(t);
            v.y = static_cast<uint32_t>(r);
            v.z = v.w = 0u;
            *reinterpret_cast<u32x4*>(buf + 2 * sl) = v;
        }
    }
    if constexpr (OP == 0) out[t] = acc;
}

}  // namespace

extern "C" {

int f2probe_scatter(uint64_t* buf, int64_t bytes, int32_t blocks, int32_t per, int32_t op, uint64_t* out,
                    void* stream) {
    if (!buf || bytes < 32 || blocks < 1 || per < 1 || (op != 0 && op != 1) || (op == 0 && !out) ||
        (reinterpret_cast<uintptr_t>(buf) & 15u))
        return -1;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (op == 0)
        hipLaunchKernelGGL(k_probe_scatter<0>, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, s, buf, bytes / 32,
                           per, out);
    else
        hipLaunchKernelGGL(k_probe_scatter<1>, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, s, buf, bytes / 16,
                           per, out);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

int f2probe_copy(const uint64_t* src, uint64_t* dst, int64_t words, void* stream) {
    if (words < 0 || (words > 0 && (!src || !dst)) || (words & 1) ||
        (reinterpret_cast<uintptr_t>(src) & 15u) || (reinterpret_cast<uintptr_t>(dst) & 15u))
        return -1;
    if (words == 0) return 0;
    const int64_t n16 = words / 2;
    int64_t blocks = (n16 + kThreads - 1) / kThreads;
    if (blocks > 131072) blocks = 131072;  // then the loop (fastest of 2k-128k workgroups on 2 GiB)
    hipLaunchKernelGGL(k_probe_copy, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0,
                       static_cast<hipStream_t>(stream), reinterpret_cast<const u32x4*>(src),
                       reinterpret_cast<u32x4*>(dst), n16);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

int f2probe_bitops(uint32_t* out, int32_t blocks, int32_t iters, int32_t op, void* stream) {
    if (!out || blocks < 1 || iters < 0 || (op != 0 && op != 1)) return -1;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (op == 0)
        hipLaunchKernelGGL(k_probe_bitops<0>, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, s, out, iters);
    else
        hipLaunchKernelGGL(k_probe_bitops<1>, dim3(static_cast<unsigned>(blocks)), dim3(kThreads), 0, s, out, iters);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

}  // extern "C"
