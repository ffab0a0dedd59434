// Rate counting per control interval (Algorithm 1 input "rates").
//
// HBM-bound stream: every request's key is read once (4 B per request) and every
// counts row is written once. Three launch shapes, chosen on the host:
//   owner  many intervals, key space fits LDS: one block owns whole intervals, counts
//          them in an LDS histogram and writes each row with plain coalesced stores
//          (no zeroing pass, no global atomics);
//   tiled  few long intervals: rows are zeroed, blocks count tiles of requests into
//          LDS-private bins (u32, or two u16 per word for up to 2x more keys with tiles
//          of at most 65,535 requests) and merge nonzero bins with one atomic each;
//   global key spaces beyond LDS: rows are zeroed and each request adds one atomic.
#include "cr_common.h"

namespace cr {
namespace {

constexpr int kCountThreads = 1024;

enum Bins { kBinsNone = 0, kBinsU32 = 1, kBinsU16 = 2 };

__global__ void k_zero(uint32_t* __restrict__ p, uint64_t n)
{
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0u;
}

template <int kBins>
__device__ __forceinline__ void add_key(uint32_t b, uint32_t K, uint32_t* hist, uint32_t* row, bool& bad)
{
    if (b < K) {
        if (kBins == kBinsU32) atomicAdd(&hist[b], 1u);
        else if (kBins == kBinsU16) atomicAdd(&hist[b >> 1], 1u << ((b & 1u) << 4));
        else atomicAdd(&row[b], 1u);
    } else {
        bad = true;
    }
}

// Count keys[s, e) into hist (or row); head to a 16-byte boundary, uint4 body, tail.
template <int kBins>
__device__ __forceinline__ void count_range(const uint32_t* __restrict__ keys, uint64_t s, uint64_t e, uint32_t K,
                                            uint32_t* hist, uint32_t* row, bool& bad)
{
    const uint32_t tid = threadIdx.x, bd = blockDim.x;
    const uint64_t mis = (((uintptr_t)keys >> 2) + s) & 3u;  // keys is 4-byte aligned
    uint64_t a = s + ((4u - mis) & 3u);
    if (a > e) a = e;
    for (uint64_t i = s + tid; i < a; i += bd) add_key<kBins>(keys[i], K, hist, row, bad);
    const uint64_t nv = (e - a) >> 2;
    const uint4* __restrict__ k4 = reinterpret_cast<const uint4*>(keys + a);
    uint64_t v = tid;
    for (; v + 3 * bd < nv; v += 4 * bd) {  // four independent 16-byte loads in flight
        const uint4 q0 = k4[v], q1 = k4[v + bd], q2 = k4[v + 2 * bd], q3 = k4[v + 3 * bd];
        const uint32_t bs[16] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w,
                                 q2.x, q2.y, q2.z, q2.w, q3.x, q3.y, q3.z, q3.w};
#pragma unroll
        for (int t = 0; t < 16; ++t) add_key<kBins>(bs[t], K, hist, row, bad);
    }
    for (; v < nv; v += bd) {
        const uint4 q = k4[v];
        add_key<kBins>(q.x, K, hist, row, bad);
        add_key<kBins>(q.y, K, hist, row, bad);
        add_key<kBins>(q.z, K, hist, row, bad);
        add_key<kBins>(q.w, K, hist, row, bad);
    }
    for (uint64_t i = a + (nv << 2) + tid; i < e; i += bd) add_key<kBins>(keys[i], K, hist, row, bad);
}

__global__ __launch_bounds__(kCountThreads) void k_count_owner(const uint32_t* __restrict__ keys, uint64_t n,
                                                               const uint64_t* __restrict__ off, uint32_t J,
                                                               uint32_t K, uint32_t* __restrict__ counts,
                                                               uint32_t* __restrict__ err)
{
    extern __shared__ uint32_t hist[];
    const uint32_t tid = threadIdx.x, bd = blockDim.x;
    bool bad = false;
    for (uint32_t j = blockIdx.x; j < J; j += gridDim.x) {
        for (uint32_t b = tid; b < K; b += bd) hist[b] = 0;
        __syncthreads();
        uint64_t e = off[j + 1], s = off[j];
        e = e < n ? e : n;
        s = s < e ? s : e;
        count_range<kBinsU32>(keys, s, e, K, hist, nullptr, bad);
        __syncthreads();
        uint32_t* __restrict__ row = counts + (uint64_t)j * K;
        for (uint32_t b = tid; b < K; b += bd) row[b] = hist[b];
        __syncthreads();
    }
    if (bad) atomicOr(err, CR_ERR_KEY_RANGE);
}

template <int kBins>
__global__ __launch_bounds__(kCountThreads) void k_count_tiled(const uint32_t* __restrict__ keys, uint64_t n,
                                                               const uint64_t* __restrict__ off, uint32_t J,
                                                               uint32_t K, uint32_t* __restrict__ counts,
                                                               uint32_t* __restrict__ err, uint64_t tile)
{
    extern __shared__ uint32_t hist[];
    __shared__ uint32_t s_j;
    __shared__ uint64_t s_end;
    const uint64_t t0 = (uint64_t)blockIdx.x * tile;
    if (t0 >= n) return;
    const uint64_t t1 = t0 + tile < n ? t0 + tile : n;
    const uint32_t tid = threadIdx.x, bd = blockDim.x;
    const uint32_t words = kBins == kBinsU16 ? (K + 1) >> 1 : K;
    bool bad = false;
    uint64_t i0 = t0;
    while (i0 < t1) {
        if (tid == 0) {
            const uint32_t j = find_interval(off, J, i0);
            const uint64_t e = off[j + 1];
            s_j = j;
            s_end = (e > i0 && e < t1) ? e : t1;
        }
        if (kBins != kBinsNone)
            for (uint32_t b = tid; b < words; b += bd) hist[b] = 0;
        __syncthreads();
        const uint32_t j = s_j;
        const uint64_t e = s_end;
        uint32_t* __restrict__ row = counts + (uint64_t)j * K;
        count_range<kBins>(keys, i0, e, K, hist, row, bad);
        if (kBins != kBinsNone) {
            __syncthreads();
            for (uint32_t q = tid; q < words; q += bd) {
                const uint32_t v = hist[q];
                if (!v) continue;
                if (kBins == kBinsU32) {
                    atomicAdd(&row[q], v);
                } else {
                    if (v & 0xFFFFu) atomicAdd(&row[2 * q], v & 0xFFFFu);
                    if (v >> 16) atomicAdd(&row[2 * q + 1], v >> 16);
                }
            }
        }
        __syncthreads();
        i0 = e;
    }
    if (bad) atomicOr(err, CR_ERR_KEY_RANGE);
}

}  // namespace
}  // namespace cr

extern "C" cr_status cr_count_rates(const uint32_t* keys, uint64_t n, const uint64_t* off, uint32_t J,
                                    uint32_t num_keys, uint32_t* counts, uint32_t* err, void* stream)
{
    using namespace cr;
    if (J == 0 || num_keys == 0 || num_keys == 0xFFFFFFFFu || !off || !counts || !err) return CR_EINVAL;
    if (n > 0 && (!keys || ((uintptr_t)keys & 3u))) return CR_EINVAL;
    const hipStream_t st = as_stream(stream);
    const int max_lds = device_max_lds() - 512;
    const int cus = device_cus();
    const uint64_t rows = (uint64_t)J * num_keys;
    const bool fits32 = (uint64_t)num_keys * 4u <= (uint64_t)max_lds;
    const bool fits16 = (uint64_t)((num_keys + 1) / 2) * 4u <= (uint64_t)max_lds;
    (void)hipGetLastError();
    if (fits32 && J >= (uint32_t)cus) {
        const uint32_t lds = num_keys * 4u;
        if (hipFuncSetAttribute((const void*)k_count_owner, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
            hipSuccess)
            return CR_EHIP;
        const uint32_t grid = J < 65535u ? J : 65535u;
        hipLaunchKernelGGL(k_count_owner, dim3(grid), dim3(kCountThreads), (size_t)lds, st, keys, n, off, J, num_keys,
                           counts, err);
        return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
    }
    hipLaunchKernelGGL(k_zero, dim3(2048), dim3(256), 0, st, counts, rows);
    if (n == 0) return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
    const int bins = fits32 ? kBinsU32 : (fits16 ? kBinsU16 : kBinsNone);
    const uint64_t target_blocks = (uint64_t)cus * (bins != kBinsNone ? 2u : 8u);
    uint64_t tile = (n + target_blocks - 1) / target_blocks;
    const uint64_t min_tile = bins != kBinsNone ? (uint64_t)(num_keys > 16384 ? num_keys : 16384) : 8192u;
    if (tile < min_tile) tile = min_tile;
    tile = (tile + 1023) & ~1023ull;
    if (bins == kBinsU16 && tile > 65535u) tile = 64512u;  // a u16 bin never overflows
    const uint64_t blocks = (n + tile - 1) / tile;
    if (blocks > 0x7FFFFFFFull) return CR_EINVAL;
    const uint32_t lds = bins == kBinsU32 ? num_keys * 4u : (bins == kBinsU16 ? ((num_keys + 1) / 2) * 4u : 0u);
    if (bins == kBinsU32) {
        if (hipFuncSetAttribute((const void*)k_count_tiled<kBinsU32>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)lds) != hipSuccess)
            return CR_EHIP;
        hipLaunchKernelGGL(k_count_tiled<kBinsU32>, dim3((uint32_t)blocks), dim3(kCountThreads), (size_t)lds, st, keys,
                           n, off, J, num_keys, counts, err, tile);
    } else if (bins == kBinsU16) {
        if (hipFuncSetAttribute((const void*)k_count_tiled<kBinsU16>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)lds) != hipSuccess)
            return CR_EHIP;
        hipLaunchKernelGGL(k_count_tiled<kBinsU16>, dim3((uint32_t)blocks), dim3(kCountThreads), (size_t)lds, st, keys,
                           n, off, J, num_keys, counts, err, tile);
    } else {
        hipLaunchKernelGGL(k_count_tiled<kBinsNone>, dim3((uint32_t)blocks), dim3(kCountThreads), 0, st, keys, n, off,
                           J, num_keys, counts, err, tile);
    }
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}

extern "C" const char* cr_version(void) { return "cr 0.2 gfx950"; }
