// Rate counting per control interval (Algorithm 1 input "rates").
//
// HBM-bound stream: every request's key is read once (4 B per request). Each block
// owns a contiguous tile of requests; within a tile, each interval segment is counted
// into an LDS-privatised histogram (when num_keys bins fit in LDS) and the nonzero
// bins are merged into counts[j][*] with one global atomic per bin, so hot keys never
// contend in L2. Larger key spaces fall back to one global atomic per request.
#include "cr_common.h"

namespace cr {
namespace {

constexpr int kCountThreads = 1024;

template <bool kLds>
__global__ __launch_bounds__(kCountThreads) void k_count(const uint32_t* __restrict__ keys, uint64_t n,
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
    bool bad = false;
    uint64_t i0 = t0;
    while (i0 < t1) {
        if (tid == 0) {
            const uint32_t j = find_interval(off, J, i0);
            const uint64_t e = off[j + 1];
            s_j = j;
            s_end = (e > i0 && e < t1) ? e : t1;
        }
        if (kLds)
            for (uint32_t b = tid; b < K; b += bd) hist[b] = 0;
        __syncthreads();
        const uint32_t j = s_j;
        const uint64_t e = s_end;
        uint32_t* __restrict__ row = counts + (uint64_t)j * K;
        // Head up to a 16-byte boundary, then uint4 body, then tail.
        const uint64_t mis = (((uintptr_t)keys >> 2) + i0) & 3u;  // keys is 4-byte aligned
        uint64_t a = i0 + ((4u - mis) & 3u);
        if (a > e) a = e;
        for (uint64_t i = i0 + tid; i < a; i += bd) {
            const uint32_t b = keys[i];
            if (b < K) {
                if (kLds) atomicAdd(&hist[b], 1u);
                else atomicAdd(&row[b], 1u);
            } else {
                bad = true;
            }
        }
        const uint64_t nv = (e - a) >> 2;
        const uint4* __restrict__ k4 = reinterpret_cast<const uint4*>(keys + a);
        for (uint64_t v = tid; v < nv; v += bd) {
            const uint4 q = k4[v];
            const uint32_t bs[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                if (bs[t] < K) {
                    if (kLds) atomicAdd(&hist[bs[t]], 1u);
                    else atomicAdd(&row[bs[t]], 1u);
                } else {
                    bad = true;
                }
            }
        }
        for (uint64_t i = a + (nv << 2) + tid; i < e; i += bd) {
            const uint32_t b = keys[i];
            if (b < K) {
                if (kLds) atomicAdd(&hist[b], 1u);
                else atomicAdd(&row[b], 1u);
            } else {
                bad = true;
            }
        }
        if (kLds) {
            __syncthreads();
            for (uint32_t b = tid; b < K; b += bd) {
                const uint32_t c = hist[b];
                if (c) atomicAdd(&row[b], c);
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
    if (n == 0) return CR_OK;
    const hipStream_t st = as_stream(stream);
    const int max_lds = device_max_lds();
    const uint64_t lds_bytes = (uint64_t)num_keys * 4u;
    const bool use_lds = lds_bytes + 256u <= (uint64_t)max_lds;
    // Enough tiles to give every CU a few blocks; LDS tiles are larger so the bin
    // clear/merge amortises over many requests.
    const int cus = device_cus();
    uint64_t target_blocks = (uint64_t)cus * (use_lds ? 2u : 8u);
    uint64_t tile = (n + target_blocks - 1) / target_blocks;
    uint64_t min_tile = use_lds ? (uint64_t)(num_keys > 16384 ? num_keys : 16384) : 8192u;
    if (tile < min_tile) tile = min_tile;
    tile = (tile + 1023) & ~1023ull;
    const uint64_t blocks = (n + tile - 1) / tile;
    if (blocks > 0x7FFFFFFFull) return CR_EINVAL;
    (void)hipGetLastError();
    if (use_lds) {
        if (hipFuncSetAttribute((const void*)k_count<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)lds_bytes) != hipSuccess)
            return CR_EHIP;
        hipLaunchKernelGGL(k_count<true>, dim3((uint32_t)blocks), dim3(kCountThreads), (size_t)lds_bytes, st, keys,
                           n, off, J, num_keys, counts, err, tile);
    } else {
        hipLaunchKernelGGL(k_count<false>, dim3((uint32_t)blocks), dim3(kCountThreads), 0, st, keys, n, off, J,
                           num_keys, counts, err, tile);
    }
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}

extern "C" const char* cr_version(void) { return "cr 0.1 gfx950"; }
