// Request dispatch through fixed plans (Section 3.1 "Placement and dispatch"; Fig. 1).
// k_route is the order-independent form: admitted keys pick a member of T(b) by the
// request hash, cold keys use power of two choices on the plan's interval-start loads.
// k_route_live is the live-load form, one serial chain per interval (see below).
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
    issue_priority_high();
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

// Live-load dispatch (Section 3.1 "Placement and dispatch"; Fig. 1): during an interval,
// admitted keys take the least-loaded member of T(b) and the rest power of two choices,
// on the running count of requests each destination has received in the interval. Every
// decision depends on the earlier ones, so an interval is one serial chain; the chains of
// different intervals and candidates are independent, one wavefront each. With R <= 64,
// lane r holds destination r's count and a decision reads it with v_readlane; otherwise the
// counts sit in LDS. For each batch of 64 requests the lanes look their requests up in
// parallel (table entry, hash, both draws; a single-copy key is a choice between its
// member and itself), then the wavefront walks the 64 decisions in order.
template <bool kLds>
__global__ __launch_bounds__(64) void k_route_live(
    const uint32_t* __restrict__ keys, uint64_t n, uint64_t first_index, uint32_t smix,
    const uint64_t* __restrict__ off, const uint32_t* __restrict__ gmap, uint32_t K, uint32_t R, uint32_t cands,
    uint32_t NG, uint32_t KW, const uint64_t* __restrict__ key_index, const uint32_t* __restrict__ route,
    const uint32_t* __restrict__ member_off, uint32_t cmax, const uint16_t* __restrict__ members,
    uint16_t* __restrict__ dest, uint32_t* __restrict__ err)
{
    __shared__ uint32_t s_live[kLds ? CR_MAX_R : 1];
    const uint32_t lane = threadIdx.x;
    const uint32_t j = blockIdx.x / cands, c = blockIdx.x % cands;
    const uint64_t i0 = off[j];
    uint64_t i1 = off[j + 1];
    i1 = i1 < n ? i1 : n;
    if (i1 <= i0) return;
    const uint32_t g = gmap[j] < NG ? gmap[j] : NG - 1u;
    const uint32_t p = g * cands + c;
    const uint64_t* __restrict__ kx = key_index + (uint64_t)p * 2u * KW;
    const uint32_t* __restrict__ rw = route + (uint64_t)p * cmax;
    const uint32_t* __restrict__ mo = member_off + (uint64_t)p * (cmax + 1u);
    const uint16_t* __restrict__ mem = members + (uint64_t)p * cmax;
    uint16_t* __restrict__ dc = dest + (uint64_t)c * n;
    uint32_t live = 0;  // lane r: requests of this interval sent to destination r (R <= 64)
    if (kLds)
        for (uint32_t r = lane; r < R; r += 64u) s_live[r] = 0;
    auto load_of = [&](uint32_t d) -> uint32_t {
        if (kLds) return (uint32_t)__builtin_amdgcn_readfirstlane((int)s_live[d]);
        return rdlane(live, d);
    };
    auto charge = [&](uint32_t d) {
        if (kLds) {
            if (lane == 0) s_live[d] = s_live[d] + 1u;
        } else {
            live += lane == d ? 1u : 0u;
        }
    };
    bool bad = false;
    for (uint64_t base = i0; base < i1; base += 64u) {
        const uint64_t i = base + lane;
        const bool in = i < i1;
        const uint32_t b = in ? keys[i] : 0u;
        const bool valid = in && b < K;
        bad |= in && b >= K;
        const ulonglong2 e = valid ? *reinterpret_cast<const ulonglong2*>(kx + 2u * (b >> 6))
                                   : make_ulonglong2(0ull, 0ull);
        const bool adm = valid && ((e.x >> (b & 63u)) & 1ull);
        const uint32_t w =
            adm ? rw[(uint32_t)e.y + (uint32_t)__popcll(e.x & ((1ull << (b & 63u)) - 1ull))] : 0u;
        const uint32_t h = req_hash(smix, first_index + i);
        uint32_t d1 = (uint32_t)(((uint64_t)(h & 0xFFFFu) * R) >> 16);
        uint32_t d2 = (uint32_t)(((uint64_t)(h >> 16) * R) >> 16);
        if (adm && (w & CR_ROUTE_SINGLE)) d1 = d2 = w & 0xFFFFu;
        const uint64_t multi = ballot(adm && !(w & CR_ROUTE_SINGLE));
        const uint32_t nb = i1 - base < 64u ? (uint32_t)(i1 - base) : 64u;
        uint32_t out = 0;
        if (!kLds && multi == 0 && nb == 64u) {
            // Full batch without multi-copy keys: 64 branch-free decisions, draws read 16 ahead.
#pragma unroll
            for (uint32_t gq = 0; gq < 4; ++gq) {
                uint32_t e1[16], e2[16];
#pragma unroll
                for (uint32_t t = 0; t < 16; ++t) {
                    e1[t] = rdlane(d1, 16u * gq + t);
                    e2[t] = rdlane(d2, 16u * gq + t);
                }
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (uint32_t t = 0; t < 16; ++t) {
                    const uint32_t d = rdlane(live, e2[t]) < rdlane(live, e1[t]) ? e2[t] : e1[t];
                    live += lane == d ? 1u : 0u;
                    out = wrlane(out, d, 16u * gq + t);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            dc[i] = (uint16_t)out;
            continue;
        }
        for (uint32_t t = 0; t < nb; ++t) {
            uint32_t d;
            if ((multi >> t) & 1ull) {
                // least (load, destination) among the members of T(b)
                const uint32_t a = rdlane(w, t);
                const uint32_t o0 = (uint32_t)__builtin_amdgcn_readfirstlane((int)mo[a]);
                const uint32_t o1 = (uint32_t)__builtin_amdgcn_readfirstlane((int)mo[a + 1u]);
                d = (uint32_t)__builtin_amdgcn_readfirstlane((int)mem[o0]);
                uint32_t ld = load_of(d);
                for (uint32_t o = o0 + 1u; o < o1; ++o) {
                    const uint32_t m = (uint32_t)__builtin_amdgcn_readfirstlane((int)mem[o]);
                    const uint32_t lm = load_of(m);
                    if (lm < ld || (lm == ld && m < d)) {
                        d = m;
                        ld = lm;
                    }
                }
            } else {
                const uint32_t e1 = rdlane(d1, t), e2 = rdlane(d2, t);
                d = load_of(e2) < load_of(e1) ? e2 : e1;
            }
            charge(d);
            out = wrlane(out, d, t);
        }
        if (in) dc[i] = (uint16_t)out;
    }
    if (ballot(bad) && lane == 0) atomicOr(err, CR_ERR_KEY_RANGE);
}

}  // namespace
}  // namespace cr

extern "C" cr_status cr_route_live(const uint32_t* keys, uint64_t n, uint64_t first_index, uint64_t seed,
                                   const uint64_t* off, const uint32_t* gmap, uint32_t J, const cr_plan_set* plans,
                                   uint16_t* dest, uint32_t* err, void* stream)
{
    using namespace cr;
    if (!plans || !off || !gmap || J == 0 || !err) return CR_EINVAL;
    if (plans->cands == 0 || plans->num_plans == 0 || plans->num_plans % plans->cands || plans->R == 0 ||
        plans->R > CR_MAX_R || plans->num_keys == 0 || plans->num_keys == 0xFFFFFFFFu || plans->max_W == 0 ||
        !plans->key_index || !plans->route || !plans->member_off || !plans->members)
        return CR_EINVAL;
    if (n == 0) return CR_OK;
    if (!keys || !dest || ((uintptr_t)keys & 3u) || ((uintptr_t)dest & 1u)) return CR_EINVAL;
    const uint64_t blocks = (uint64_t)J * plans->cands;
    if (blocks > 0x7FFFFFF0ull) return CR_EINVAL;
    const uint32_t cmax = plans->R * plans->max_W;
    (void)hipGetLastError();
#define CR_LIVE_LAUNCH(L)                                                                                          \
    hipLaunchKernelGGL(k_route_live<L>, dim3((uint32_t)blocks), dim3(64), 0, as_stream(stream), keys, n, first_index, \
                       seed_mix(seed), off, gmap, plans->num_keys, plans->R, plans->cands,                          \
                       plans->num_plans / plans->cands, (plans->num_keys + 63u) / 64u, plans->key_index, plans->route, \
                       plans->member_off, cmax, plans->members, dest, err)
    if (plans->R <= 64) CR_LIVE_LAUNCH(false);
    else CR_LIVE_LAUNCH(true);
#undef CR_LIVE_LAUNCH
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}

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
