// Request dispatch through fixed plans (Section 3.1 "Placement and dispatch"; Fig. 1),
// in the order-independent form: admitted keys pick a member of T(b) by the request
// hash, cold keys use power of two choices on the plan's interval-start loads.
//
// HBM-bound stream: 4 B key read + 2 B destination written per request and candidate.
// The route table of a group is key-major ([key][candidate]) so one request reads one
// contiguous row; rows of hot keys and the R loads stay in L2.
#include "cr_common.h"

namespace cr {
namespace {

constexpr int kRouteThreads = 256;
constexpr int kRouteItems = 8;

__device__ __forceinline__ uint16_t route_one(uint32_t word, uint32_t h, uint32_t R, const double* __restrict__ L,
                                              const uint32_t* __restrict__ mo, const uint16_t* __restrict__ mem)
{
    if (word == CR_ROUTE_COLD) {
        const uint32_t d1 = ((h & 0xFFFFu) * R) >> 16;
        const uint32_t d2 = ((h >> 16) * R) >> 16;
        return (uint16_t)(L[d2] < L[d1] ? d2 : d1);
    }
    if (word & CR_ROUTE_SINGLE) return (uint16_t)(word & 0xFFFFu);
    const uint32_t o = mo[word], k = mo[word + 1] - o;
    return mem[o + (((h >> 16) * k) >> 16)];
}

__global__ __launch_bounds__(kRouteThreads) void k_route(
    const uint32_t* __restrict__ keys, uint64_t n, uint64_t first_index, uint32_t smix,
    const uint64_t* __restrict__ off, const uint32_t* __restrict__ gmap, uint32_t J, uint32_t K, uint32_t R,
    uint32_t cands, uint32_t NG, const uint32_t* __restrict__ route, const uint32_t* __restrict__ member_off,
    uint32_t mo_stride, const uint16_t* __restrict__ members, uint32_t mem_stride, const double* __restrict__ load,
    uint16_t* __restrict__ dest, uint32_t* __restrict__ err)
{
    __shared__ uint32_t s_j0;
    const uint64_t tile0 = (uint64_t)blockIdx.x * kRouteThreads * kRouteItems;
    if (tile0 >= n) return;
    if (threadIdx.x == 0) s_j0 = find_interval(off, J, tile0);
    __syncthreads();
    uint32_t j = s_j0;
    bool bad = false;
#pragma unroll
    for (int it = 0; it < kRouteItems; ++it) {
        const uint64_t i = tile0 + (uint64_t)it * kRouteThreads + threadIdx.x;
        if (i >= n) break;
        while (j + 1 < J && off[j + 1] <= i) ++j;
        uint32_t g = gmap[j];
        g = g < NG ? g : NG - 1;
        const uint32_t b = keys[i];
        const bool valid = b < K;
        bad |= !valid;
        const uint32_t h = req_hash(smix, first_index + i);
        const uint32_t* __restrict__ rw = route + ((uint64_t)g * K + (valid ? b : 0u)) * cands;
        for (uint32_t c = 0; c < cands; ++c) {
            const uint64_t p = (uint64_t)g * cands + c;
            const uint32_t word = valid ? rw[c] : CR_ROUTE_COLD;
            dest[(uint64_t)c * n + i] =
                route_one(word, h, R, load + p * R, member_off + p * mo_stride, members + p * mem_stride);
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
        !plans->route || !plans->member_off || !plans->members || !plans->load)
        return CR_EINVAL;
    if (n == 0) return CR_OK;
    if (!keys || !dest) return CR_EINVAL;
    const uint32_t cmax = plans->R * plans->max_W;
    const uint64_t per_block = (uint64_t)kRouteThreads * kRouteItems;
    const uint64_t blocks = (n + per_block - 1) / per_block;
    if (blocks > 0x7FFFFFFFull) return CR_EINVAL;
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_route, dim3((uint32_t)blocks), dim3(kRouteThreads), 0, as_stream(stream), keys, n,
                       first_index, seed_mix(seed), off, gmap, J, plans->num_keys, plans->R, plans->cands,
                       plans->num_plans / plans->cands, plans->route, plans->member_off, cmax + 1u, plans->members,
                       cmax, plans->load, dest, err);
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}
