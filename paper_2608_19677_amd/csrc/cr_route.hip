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
constexpr uint32_t kBlockReq = kRouteThreads * kPer;
constexpr int kBnd = 4;  // interval starts cached per block; more boundaries take a slow path

// Every gather below is unconditional (indices are clamped into range and the results
// selected afterwards) so the four requests of a thread keep their loads in flight
// together instead of waiting on each other behind branches.
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
    __shared__ uint32_t s_rel[kBnd];     // next interval starts relative to the block (clamped)
    __shared__ uint32_t s_g[kBnd + 1];   // plan groups of intervals j0 .. j0 + kBnd
    const uint64_t bstart = (uint64_t)xcd_tile(blockIdx.x, gridDim.x) * kBlockReq;
    if (bstart >= n) return;
    if (threadIdx.x < 64) {
        const uint32_t j0 = find_interval(off, J, bstart);
        if (threadIdx.x == 0) s_j0 = j0;
        if (threadIdx.x < kBnd) {
            const uint32_t jb = j0 + 1 + threadIdx.x;
            const uint64_t e = jb < J ? off[jb] : ~0ull;
            s_rel[threadIdx.x] = e - bstart < kBlockReq ? (uint32_t)(e - bstart) : kBlockReq;
        }
        if (threadIdx.x <= kBnd) {
            const uint32_t jj = j0 + threadIdx.x < J ? j0 + threadIdx.x : J - 1;
            const uint32_t gg = gmap[jj];
            s_g[threadIdx.x] = gg < NG ? gg : NG - 1;
        }
    }
    __syncthreads();
    const uint32_t rel0 = threadIdx.x * kPer;
    const uint64_t base = bstart + rel0;
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
    const uint32_t r0 = s_rel[0], r1 = s_rel[1], r2 = s_rel[2], r3 = s_rel[3];
    // request hash: the inner mix depends only on the high word of the global index
    const uint64_t gi0 = first_index + base;
    const uint32_t inner0 = fmix32((uint32_t)(gi0 >> 32) ^ smix);
    bool bad = false;
#pragma unroll
    for (int t = 0; t < kPer; ++t) {
        const uint32_t rel = rel0 + t;
        const uint32_t q = (rel >= r0) + (rel >= r1) + (rel >= r2) + (rel >= r3);
        if (rel >= r3 && r3 < kBlockReq) {  // more than kBnd boundaries in this block
            uint32_t j = j0 + kBnd;
            while (j + 1 < J && off[j + 1] <= base + t) ++j;
            const uint32_t gg = gmap[j];
            g[t] = gg < NG ? gg : NG - 1;
        } else {
            g[t] = s_g[q];
        }
        const uint64_t gi = gi0 + t;
        const uint32_t inner = (uint32_t)(gi >> 32) == (uint32_t)(gi0 >> 32) ? inner0 : fmix32((uint32_t)(gi >> 32) ^ smix);
        h[t] = fmix32((uint32_t)gi ^ inner);
        const bool valid = base + t >= n || b[t] < K;
        bad |= !valid;
    }
    for (uint32_t c = 0; c < cands; ++c) {
        ulonglong2 e[kPer];
        double l1[kPer], l2[kPer];
        uint32_t d1[kPer], d2[kPer], pl[kPer];
#pragma unroll
        for (int t = 0; t < kPer; ++t) {
            const uint32_t p = g[t] * cands + c;
            pl[t] = p;
            const uint32_t bb = b[t] < K ? b[t] : 0u;
            e[t] = *reinterpret_cast<const ulonglong2*>(key_index + ((uint64_t)p * KW + (bb >> 6)) * 2u);
            d1[t] = ((h[t] & 0xFFFFu) * R) >> 16;
            d2[t] = ((h[t] >> 16) * R) >> 16;
            l1[t] = load[(uint64_t)p * R + d1[t]];
            l2[t] = load[(uint64_t)p * R + d2[t]];
        }
        uint32_t word[kPer];
        bool adm[kPer];
#pragma unroll
        for (int t = 0; t < kPer; ++t) {
            const uint32_t sh = b[t] & 63u;
            adm[t] = b[t] < K && ((e[t].x >> sh) & 1ull);
            const uint32_t rank = (uint32_t)e[t].y + (uint32_t)__popcll(e[t].x & ((1ull << sh) - 1ull));
            word[t] = route[(uint64_t)pl[t] * cmax + (adm[t] ? rank : 0u)];
        }
        uint32_t d[kPer];
        bool multi = false;
#pragma unroll
        for (int t = 0; t < kPer; ++t) {
            d[t] = adm[t] ? (word[t] & 0xFFFFu) : (l2[t] < l1[t] ? d2[t] : d1[t]);
            multi |= adm[t] && !(word[t] & CR_ROUTE_SINGLE);
        }
        if (ballot(multi)) {  // some admitted key of this wave has k > 1
#pragma unroll
            for (int t = 0; t < kPer; ++t) {
                const bool m = adm[t] && !(word[t] & CR_ROUTE_SINGLE);
                const uint32_t a = m ? word[t] : 0u;
                const uint32_t* __restrict__ mo = member_off + (uint64_t)pl[t] * (cmax + 1u);
                const uint32_t o = mo[a], k = mo[a + 1] - o;
                const uint32_t pick = m ? o + (((h[t] >> 16) * k) >> 16) : 0u;
                const uint32_t dm = members[(uint64_t)pl[t] * cmax + pick];
                d[t] = m ? dm : d[t];
            }
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
    const uint64_t per_block = kBlockReq;
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
