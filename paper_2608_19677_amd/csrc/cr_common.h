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

// Raises the calling wavefront's instruction-issue priority on its SIMD (s_setprio 3). The
// placement, routing and partition kernels are chains of dependent latency-bound steps; when
// they share SIMDs with the vector-bound replay launched on another stream, this keeps the
// replay's wavefronts from taking every issue slot ahead of them. Results are unaffected.
__device__ __forceinline__ void issue_priority_high() { __builtin_amdgcn_s_setprio(3); }

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

// v_writelane_b32: returns `old` with lane `lane` replaced by the uniform value `val`.
__device__ int cr_amdgcn_writelane(int val, int lane, int old) __asm("llvm.amdgcn.writelane.i32");

__device__ __forceinline__ uint32_t wrlane(uint32_t old, uint32_t val, uint32_t lane)
{
    return (uint32_t)cr_amdgcn_writelane((int)val, (int)lane, (int)old);
}

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

template <int kCtrl, int kRowMask>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, kCtrl, kRowMask, 0xF, false);
}

// Inclusive wave64 prefix sum with DPP row shifts and row broadcasts (no LDS traffic).
__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v)
{
    v += dpp_u32<0x111, 0xF>(v);  // row_shr:1
    v += dpp_u32<0x112, 0xF>(v);  // row_shr:2
    v += dpp_u32<0x114, 0xF>(v);  // row_shr:4
    v += dpp_u32<0x118, 0xF>(v);  // row_shr:8
    v += dpp_u32<0x142, 0xA>(v);  // row_bcast:15 into rows 1 and 3
    v += dpp_u32<0x143, 0xC>(v);  // row_bcast:31 into rows 2 and 3
    return v;
}

// Block-wide exclusive scan of 32-bit values (blockDim.x a multiple of 64, <= 1024).
// `sh` needs 16 words. Returns the exclusive prefix; *total gets the block sum.
__device__ __forceinline__ uint32_t block_exscan_u32(uint32_t v, uint32_t* sh, uint32_t* total)
{
    const uint32_t wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const uint32_t x = wave_incl_scan_u32(v);
    if (lane_id() == 63) sh[wv] = x;
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

// Block-wide exclusive count of a predicate (ballot + popcount per wave).
__device__ __forceinline__ uint32_t block_exscan_flag(bool f, uint32_t* sh, uint32_t* total)
{
    const uint32_t wv = threadIdx.x >> 6, nw = blockDim.x >> 6;
    const uint64_t m = ballot(f);
    if (lane_id() == 0) sh[wv] = (uint32_t)__popcll(m);
    __syncthreads();
    uint32_t base = 0, tot = 0;
    for (uint32_t w = 0; w < nw; ++w) {
        const uint32_t t = sh[w];
        base += (w < wv) ? t : 0u;
        tot += t;
    }
    __syncthreads();
    *total = tot;
    return base + (uint32_t)__popcll(m & lanemask_lt());
}

// Index of this wavefront in its block, as a value the compiler knows is uniform.
__device__ __forceinline__ uint32_t wave_in_block()
{
    return (uint32_t)__builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
}

// Workgroups are dealt to the 8 XCDs round-robin (block b runs on XCD b % 8). A grid
// rounded up to a multiple of 8 and remapped this way hands every XCD one contiguous
// eighth of the tiles, so neighbouring tiles share that XCD's L2.
constexpr uint32_t kXcds = 8;

__host__ __device__ __forceinline__ uint32_t xcd_grid(uint32_t tiles) { return (tiles + kXcds - 1) / kXcds * kXcds; }

__device__ __forceinline__ uint32_t xcd_tile(uint32_t b, uint32_t grid)
{
    return (b % kXcds) * (grid / kXcds) + b / kXcds;
}

// Buffer resource over [p, p + bytes) for raw buffer loads: reads outside the range return
// 0 instead of touching memory (gfx9 buffer addressing; word 3 = 0x00020000 on this family).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), 0, (int)bytes, 0x00020000);
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
