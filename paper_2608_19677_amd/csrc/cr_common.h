// Internal device/host helpers of libcr (gfx950, wave64). Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/cr.h"

namespace cr {

constexpr int kWave = 64;

__device__ __forceinline__ uint32_t lane_id()
{
    return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
}

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

__device__ __forceinline__ uint64_t lanemask_lt()
{
    const uint32_t l = lane_id();
    return l == 0 ? 0ull : (~0ull >> (64 - l));
}

__device__ __forceinline__ uint32_t rdlane(uint32_t v, uint32_t l)
{
    return (uint32_t)__builtin_amdgcn_readlane((int)v, (int)l);
}

__device__ __forceinline__ uint64_t rdlane64(uint64_t v, uint32_t l)
{
    return (uint64_t)rdlane((uint32_t)v, l) | ((uint64_t)rdlane((uint32_t)(v >> 32), l) << 32);
}

__device__ __forceinline__ double rdlane_f64(double v, uint32_t l)
{
    return __longlong_as_double((long long)rdlane64((uint64_t)__double_as_longlong(v), l));
}

__device__ __forceinline__ uint32_t first_lane(uint64_t mask) { return (uint32_t)__builtin_ctzll(mask); }

// MurmurHash3's 32-bit finalizer.
__host__ __device__ __forceinline__ uint32_t fmix32(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x85EBCA6Bu;
    x ^= x >> 13;
    x *= 0xC2B2AE35u;
    x ^= x >> 16;
    return x;
}

// Per-call seed mix; the per-request hash is fmix32(lo(i) ^ fmix32(hi(i) ^ s)).
__host__ __device__ __forceinline__ uint32_t seed_mix(uint64_t seed)
{
    return fmix32((uint32_t)seed ^ (uint32_t)(seed >> 32) ^ 0x9E3779B9u);
}

__device__ __forceinline__ uint32_t req_hash(uint32_t s, uint64_t i)
{
    return fmix32((uint32_t)i ^ fmix32((uint32_t)(i >> 32) ^ s));
}

// Largest j in [0, J) with off[j] <= i (off[J] = n > i). Malformed offsets still give
// an index in range.
__device__ __forceinline__ uint32_t find_interval(const uint64_t* __restrict__ off, uint32_t J, uint64_t i)
{
    uint32_t lo = 0, hi = J;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (off[mid] <= i) lo = mid;
        else hi = mid;
    }
    return lo;
}

// Block-wide exclusive scan of 32-bit values (blockDim.x a multiple of 64, <= 1024).
// `sh` needs 16 words. Returns the exclusive prefix; *total gets the block sum.
__device__ __forceinline__ uint32_t block_exscan_u32(uint32_t v, uint32_t* sh, uint32_t* total)
{
    const uint32_t lane = lane_id(), wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
    uint32_t x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(x, o, 64);
        if (lane >= (uint32_t)o) x += y;
    }
    if (lane == 63) sh[wv] = x;
    __syncthreads();
    uint32_t base = 0, tot = 0;
    for (uint32_t w = 0; w < nw; ++w) {
        const uint32_t t = sh[w];
        base += (w < wv) ? t : 0u;
        tot += t;
    }
    __syncthreads();
    *total = tot;
    return base + x - v;
}

inline hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

inline int device_max_lds()
{
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 65536;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess) return 65536;
    return v;
}

inline int device_cus()
{
    int dev = 0, v = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 256;
    return v;
}

}  // namespace cr
