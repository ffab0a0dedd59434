// Request dispatch through fixed plans (Section 3.1 "Placement and dispatch"; Fig. 1),
// in the order-independent form: admitted keys pick a member of T(b) by the request
// hash, cold keys use power of two choices on the plan's interval-start loads.
//
// HBM-bound stream: 4 B key read + 2 B destination written per request and candidate.
// Each thread owns 4 consecutive requests: one 16-byte key load, then per candidate 4
// independent lookups in the plan's compact table (a 16-byte key-index entry: admitted
// bits of 64 keys and the key rank of the first; an admitted key reads its route word by
// rank) and one 8-byte store of 4 destinations. A plan's table is a few KB for tens of
// thousands of keys, so the lookups stay in cache.
#include "cr_common.h"

namespace cr {
namespace {

constexpr int kRouteThreads = 256;
constexpr int kPer = 4;

__device__ __forceinline__ uint32_t route_one(bool admitted, uint32_t word, uint32_t h, uint32_t R,
                                              const double* __restrict__ L, const uint32_t* __restrict__ mo,
                                              const uint16_t* __restrict__ mem)
{
    if (!admitted) {
        const uint32_t d1 = ((h & 0xFFFFu) * R) >> 16;
        const uint32_t d2 = ((h >> 16) * R) >> 16;
        return L[d2] < L[d1] ? d2 : d1;
    }
    if (word & CR_ROUTE_SINGLE) return word & 0xFFFFu;
    const uint32_t o = mo[word], k = mo[word + 1] - o;
    return mem[o + (((h >> 16) * k) >> 16)];
}

template <bool kVec>
__global__ __launch_bounds__(kRouteThreads) void k_route(
    const uint32_t* __restrict__ keys, uint64_t n, uint64_t first_index, uint32_t smix,
    const uint64_t* __restrict__ off, const uint32_t* __restrict__ gmap, uint32_t J, uint32_t K, uint32_t R,
    uint32_t cands, uint32_t NG, uint32_t KW, const uint64_t* __restrict__ key_index,
    const uint32_t* __restrict__ route, const uint32_t* __restrict__ member_off, uint32_t cmax,
    const uint16_t* __restrict__ members, const double* __restrict__ load, uint16_t* __restrict__ dest,
    uint32_t* __restrict__ err)
{
    __shared__ uint32_t s_j0;
    __shared__ uint64_t s_bnd[4];  // starts of the next four intervals (~0 past the last)
    const uint64_t bstart = (uint64_t)xcd_tile(blockIdx.x, gridDim.x) * kRouteThreads * kPer;
    if (bstart >= n) return;
    if (threadIdx.x < 64) {
        const uint32_t j0 = find_interval(off, J, bstart);
        if (threadIdx.x == 0) s_j0 = j0;
        if (threadIdx.x < 4) s_bnd[threadIdx.x] = j0 + 1 + threadIdx.x < J ? off[j0 + 1 + threadIdx.x] : ~0ull;
    }
    __syncthreads();
    const uint64_t base = bstart + (uint64_t)threadIdx.x * kPer;
    if (base >= n) return;
    const bool full = kVec && base + kPer <= n;
    uint32_t b[kPer], g[kPer], h[kPer];
    if (full) {
        const uint4 q = *reinterpret_cast<const uint4*>(keys + base);
        b[0] = q.x;
        b[1] = q.y;
        b[2] = q.z;
        b[3] = q.w;
    } else {
#pragma unroll
        for (int t = 0; t < kPer; ++t) b[t] = base + t < n ? keys[base + t] : 0u;
    }
    const uint32_t j0 = s_j0;
    const uint64_t e0 = s_bnd[0], e1 = s_bnd[1], e2 = s_bnd[2], e3 = s_bnd[3];
    bool bad = false;
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
        const uint64_t i = base + t;
        uint32_t j = j0 + (i >= e0) + (i >= e1) + (i >= e2) + (i >= e3);
        if (i >= e3)
            while (j + 1 < J && off[j + 1] <= i) ++j;
        const uint32_t gg = gmap[j];
        g[t] = gg < NG ? gg : NG - 1;
        h[t] = req_hash(smix, first_index + i);
        const bool valid = i >= n || b[t] < K;
        bad |= !valid;
        if (!valid) b[t] = 0xFFFFFFFFu;
    }
    for (uint32_t c = 0; c < cands; ++c) {
        ulonglong2 e[kPer];
        uint32_t d[kPer];
#pragma unroll
        for (int t = 0; t < kPer; ++t) {
            const uint64_t p = (uint64_t)g[t] * cands + c;
            e[t] = b[t] < K ? *reinterpret_cast<const ulonglong2*>(key_index + (p * KW + (b[t] >> 6)) * 2u)
                            : make_ulonglong2(0ull, 0ull);
        }
#pragma unroll
        for (int t = 0; t < kPer; ++t) {
            const uint64_t p = (uint64_t)g[t] * cands + c;
            const uint64_t below = e[t].x & ((1ull << (b[t] & 63u)) - 1ull);
            const bool adm = (e[t].x >> (b[t] & 63u)) & 1ull;
            const uint32_t word = adm ? route[p * cmax + (uint32_t)e[t].y + (uint32_t)__popcll(below)] : 0u;
            d[t] = route_one(adm, word, h[t], R, load + p * R, member_off + p * (cmax + 1u), members + p * cmax);
        }
        uint16_t* __restrict__ dc = dest + (uint64_t)c * n + base;
        if (full) {
            const uint2 v = make_uint2(d[0] | (d[1] << 16), d[2] | (d[3] << 16));
            *reinterpret_cast<uint2*>(dc) = v;
        } else {
#pragma unroll
            for (int t = 0; t < kPer; ++t)
                if (base + t < n) dc[t] = (uint16_t)d[t];
        }
    }
    if (bad) atomicOr(err, CR_ERR_KEY_RANGE);
}

}  // namespace
}  // namespace cr

extern "C" cr_status cr_route(const uint32_t* keys, uint64_t n, uint64_t first_index, uint64_t seed,
                              const uint64_t* off, const uint32_t* gmap, uint32_t J, const cr_plan_set* plans,
                              uint16_t* dest, uint32_t* err, void* stream)
{
    using namespace cr;
    if (!plans || !off || !gmap || J == 0 || !err) return CR_EINVAL;
    if (plans->cands == 0 || plans->num_plans == 0 || plans->num_plans % plans->cands || plans->R == 0 ||
        plans->R > CR_MAX_R || plans->num_keys == 0 || plans->num_keys == 0xFFFFFFFFu || plans->max_W == 0 ||
        !plans->key_index || !plans->route || !plans->member_off || !plans->members || !plans->load)
        return CR_EINVAL;
    if (n == 0) return CR_OK;
    if (!keys || !dest || ((uintptr_t)keys & 3u) || ((uintptr_t)dest & 1u)) return CR_EINVAL;
    const uint32_t cmax = plans->R * plans->max_W;
    const uint64_t per_block = (uint64_t)kRouteThreads * kPer;
    const uint64_t blocks = (n + per_block - 1) / per_block;
    if (blocks > 0x7FFFFFF0ull) return CR_EINVAL;
    // 16-byte key loads and 8-byte destination stores need aligned rows.
    const bool vec = ((uintptr_t)keys & 15u) == 0 && ((uintptr_t)dest & 7u) == 0 && (n & 3u) == 0;
    (void)hipGetLastError();
#define CR_ROUTE_LAUNCH(V)                                                                                         \
    hipLaunchKernelGGL(k_route<V>, dim3(xcd_grid((uint32_t)blocks)), dim3(kRouteThreads), 0, as_stream(stream), keys, n, \
                       first_index, seed_mix(seed), off, gmap, J, plans->num_keys, plans->R, plans->cands,        \
                       plans->num_plans / plans->cands, (plans->num_keys + 63u) / 64u, plans->key_index, plans->route, \
                       plans->member_off, cmax, plans->members, plans->load, dest, err)
    if (vec) CR_ROUTE_LAUNCH(true);
    else CR_ROUTE_LAUNCH(false);
#undef CR_ROUTE_LAUNCH
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}
