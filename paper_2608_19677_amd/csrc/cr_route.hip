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

// ---------------------------------------------------------------------------------------
// Group dispatch tables. Candidates of one group built from the same window admit prefixes
// of that window's order, so one row per order position holds every candidate's dispatch of
// a key, and one row per destination holds every candidate's load rank, which decides the
// power-of-two-choices fallback. A request then reads its key's position, one row of CS
// u16 entries and the rank rows of its two draws (a table of R x CS u16 that stays in
// cache) instead of a handful of gathers per candidate into per-plan tables.
// ---------------------------------------------------------------------------------------
constexpr uint32_t kGrpRows = 64;      // order positions per k_group_dest block
constexpr uint32_t kGrpThreads = 256;

__global__ void k_fill_u32(uint32_t* __restrict__ p, uint64_t n, uint32_t v)
{
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

// window_rank[w][order[w][a]] = a for a < n_order[w]
__global__ __launch_bounds__(256) void k_win_rank_set(const uint32_t* __restrict__ order,
                                                      const uint32_t* __restrict__ n_order, uint32_t cmax, uint32_t K,
                                                      uint32_t* __restrict__ wr)
{
    const uint32_t w = blockIdx.y, a = blockIdx.x * 256u + threadIdx.x;
    const uint32_t no = n_order[w] < cmax ? n_order[w] : cmax;
    if (a >= no) return;
    const uint32_t b = order[(uint64_t)w * cmax + a];
    if (b < K) wr[(uint64_t)w * K + b] = a;
}

// Rows a0 .. a0+63 of group g: entry c = candidate c's dispatch of the key at order position a.
__global__ __launch_bounds__(kGrpThreads) void k_group_dest(uint32_t cands, uint32_t CS, uint32_t cmax,
                                                            const cr_plan_spec* __restrict__ specs,
                                                            const uint32_t* __restrict__ num_admitted,
                                                            const uint32_t* __restrict__ member_off,
                                                            const uint16_t* __restrict__ members,
                                                            uint16_t* __restrict__ gdest, uint32_t* __restrict__ gmulti,
                                                            uint32_t* __restrict__ err)
{
    __shared__ uint16_t tile[kGrpRows * (CR_MAX_CANDS + 8)];
    const uint32_t g = blockIdx.y, a0 = blockIdx.x * kGrpRows;
    const uint32_t row = threadIdx.x % kGrpRows, a = a0 + row;
    const uint32_t w0 = specs[(uint64_t)g * cands].window;
    bool mismatch = false;
    for (uint32_t c = threadIdx.x / kGrpRows; c < CS; c += kGrpThreads / kGrpRows) {
        uint16_t e = (uint16_t)CR_GROUP_COLD;
        if (c < cands) {
            const uint64_t p = (uint64_t)g * cands + c;
            mismatch |= specs[p].window != w0;
            if (a < num_admitted[p] && a < cmax) {
                const uint32_t* __restrict__ mo = member_off + p * (cmax + 1u);
                const uint32_t o = mo[a], k = mo[a + 1] - o;
                e = k == 1 ? members[p * cmax + o] : (uint16_t)CR_GROUP_MULTI;
                if (k != 1) gmulti[((uint64_t)g * cmax + a) * CS + c] = o | (k << 20);
            }
        }
        tile[row * CS + c] = e;
    }
    if (mismatch && row == 0) atomicOr(err, CR_ERR_SPEC);
    __syncthreads();
    const uint32_t per = CS / 8u;  // 16-byte pieces per row
    for (uint32_t q = threadIdx.x; q < kGrpRows * per; q += kGrpThreads) {
        const uint32_t r = q / per, part = q % per;
        if (a0 + r >= cmax) continue;
        const uint16_t* src = tile + r * CS + part * 8u;
        uint4 v;
        v.x = (uint32_t)src[0] | ((uint32_t)src[1] << 16);
        v.y = (uint32_t)src[2] | ((uint32_t)src[3] << 16);
        v.z = (uint32_t)src[4] | ((uint32_t)src[5] << 16);
        v.w = (uint32_t)src[6] | ((uint32_t)src[7] << 16);
        *reinterpret_cast<uint4*>(gdest + ((uint64_t)g * cmax + a0 + r) * CS + part * 8u) = v;
    }
}

// Load ranks of group g: entry c of row d = #{d' : L_c[d'] < L_c[d]}, so that
// L_c[d2] < L_c[d1] exactly when rank_c[d2] < rank_c[d1] (equal loads share a rank).
// One block per (candidate slot, group); slots past cands get 0 and are never used.
__global__ __launch_bounds__(256) void k_group_rank(uint32_t R, uint32_t cands, uint32_t CS,
                                                    const double* __restrict__ load, uint16_t* __restrict__ grank)
{
    __shared__ double s_l[CR_MAX_R];
    const uint32_t c = blockIdx.x, g = blockIdx.y;
    uint16_t* __restrict__ out = grank + (uint64_t)g * R * CS + c;
    if (c >= cands) {
        for (uint32_t d = threadIdx.x; d < R; d += blockDim.x) out[(uint64_t)d * CS] = 0;
        return;
    }
    const double* __restrict__ l = load + ((uint64_t)g * cands + c) * R;
    for (uint32_t d = threadIdx.x; d < R; d += blockDim.x) s_l[d] = l[d];
    __syncthreads();
    for (uint32_t d = threadIdx.x; d < R; d += blockDim.x) {
        const double x = s_l[d];
        uint32_t r = 0;
        for (uint32_t e = 0; e < R; ++e) r += s_l[e] < x ? 1u : 0u;  // same address across lanes: broadcast
        out[(uint64_t)d * CS] = (uint16_t)r;
    }
}

// Requests per k_route_group block: the destination tile holds CS x T entries in LDS
// (kGrpTileWords 32-bit words at most); T is a multiple of 64 in 64 .. 1024.
constexpr uint32_t kGrpTileWords = 8192;

__host__ __device__ __forceinline__ uint32_t group_tile(uint32_t CS)
{
    const uint32_t t = (2u * kGrpTileWords / CS) & ~63u;
    return t > 1024u ? 1024u : (t < 64u ? 64u : t);
}

// Row stride of the LDS tile in 32-bit words: T/2 + 2 puts the eight candidate rows that a
// wavefront's lanes write at once 16 banks apart.
__host__ __device__ __forceinline__ uint32_t group_tile_stride(uint32_t T) { return T / 2u + 2u; }

__host__ __device__ __forceinline__ size_t group_route_lds(uint32_t CS)
{
    const uint32_t T = group_tile(CS);
    return ((size_t)CS * group_tile_stride(T) + (size_t)T * 4u) * 4u;
}

// Load of a T at a 32-bit byte offset from a kernel-argument base (every group table is
// below 4 GiB), so the address is a scalar base plus one 32-bit register.
template <typename V, typename B>
__device__ __forceinline__ V ld_at(const B* base, uint32_t byte_off)
{
    return *reinterpret_cast<const V*>(reinterpret_cast<const char*>(base) + byte_off);
}

__device__ __forceinline__ uint32_t u4_at(const uint4& v, int i)
{
    return i == 0 ? v.x : (i == 1 ? v.y : (i == 2 ? v.z : v.w));
}

// Dispatch of every candidate of the request's plan group from the group tables; results
// equal k_route's. A block takes T consecutive requests in three phases:
//  1. per request: key, plan group, window position a, hash and both fallback draws into LDS;
//  2. one task per (4 consecutive requests, 8-candidate piece): the requests' 16-byte row
//     pieces (consecutive lanes read consecutive pieces of a row, so a row is one 128-byte
//     line per 8 lanes) and the 16-byte load-rank pieces of their draws, resolved to
//     destinations (a key with k > 1: its member list from the multi table, then the member
//     the request hash picks) and written to an LDS tile [candidate][request pair];
//  3. each candidate's T destinations leave as one contiguous run of 32-bit stores, marked
//     non-temporal so that they do not push the tables out of the L2.
// Gathers are issued unconditionally (clamped indices, results selected afterwards) so that
// a lane keeps all of them in flight together.
template <bool kVec>
__global__ __launch_bounds__(kRouteThreads) void k_route_group(
    const uint32_t* __restrict__ keys, uint64_t n, uint64_t first_index, uint32_t smix,
    const uint64_t* __restrict__ off, const uint32_t* __restrict__ gmap, uint32_t J, uint32_t K, uint32_t R,
    uint32_t cands, uint32_t CS, uint32_t NG, uint32_t NW, uint32_t cmax, const cr_plan_spec* __restrict__ specs,
    const uint32_t* __restrict__ wrank, const uint16_t* __restrict__ gdest, const uint16_t* __restrict__ grank,
    const uint32_t* __restrict__ gmulti, const uint16_t* __restrict__ members, uint16_t* __restrict__ dest,
    uint32_t* __restrict__ err)
{
    extern __shared__ __align__(16) uint32_t s_dyn[];
    __shared__ uint32_t s_j0;
    __shared__ uint32_t s_rel[kBnd];
    __shared__ uint32_t s_g[kBnd + 1];
    __shared__ uint32_t s_w[kBnd + 1];
    const uint32_t T = group_tile(CS), TS2 = group_tile_stride(T), NP = CS / 8u;
    uint32_t* __restrict__ m_a = s_dyn;                 // window position, 0xFFFFFFFF = none
    uint32_t* __restrict__ m_d = m_a + T;               // d1 | d2 << 16
    uint32_t* __restrict__ m_g = m_d + T;               // plan group
    uint32_t* __restrict__ m_h = m_g + T;               // request hash
    uint32_t* __restrict__ tile = m_h + T;              // [CS][TS2]: destinations of requests 2i, 2i+1
    const uint64_t bstart = (uint64_t)xcd_tile(blockIdx.x, gridDim.x) * T;
    if (bstart >= n) return;
    const uint32_t nb = n - bstart < T ? (uint32_t)(n - bstart) : T;
    if (threadIdx.x < 64) {
        const uint32_t j0 = find_interval(off, J, bstart);
        if (threadIdx.x == 0) s_j0 = j0;
        if (threadIdx.x < kBnd) {
            const uint32_t jb = j0 + 1 + threadIdx.x;
            const uint64_t e = jb < J ? off[jb] : ~0ull;
            s_rel[threadIdx.x] = e - bstart < T ? (uint32_t)(e - bstart) : T;
        }
        if (threadIdx.x <= kBnd) {
            const uint32_t jj = j0 + threadIdx.x < J ? j0 + threadIdx.x : J - 1;
            const uint32_t gg = gmap[jj] < NG ? gmap[jj] : NG - 1;
            const uint32_t ww = specs[(uint64_t)gg * cands].window;
            s_g[threadIdx.x] = gg;
            s_w[threadIdx.x] = ww < NW ? ww : 0u;
        }
    }
    __syncthreads();
    // phase 1: up to four requests per thread, keys first, then positions
    const uint32_t j0 = s_j0;
    const uint32_t r0 = s_rel[0], r1 = s_rel[1], r2 = s_rel[2], r3 = s_rel[3];
    bool bad = false;
    {
        constexpr int kP1 = 1024 / kRouteThreads;
        uint32_t b[kP1], w[kP1], g[kP1];
#pragma unroll
        for (int t = 0; t < kP1; ++t) {
            const uint32_t r = threadIdx.x + (uint32_t)t * kRouteThreads;
            b[t] = r < nb ? keys[bstart + r] : 0u;
        }
#pragma unroll
        for (int t = 0; t < kP1; ++t) {
            const uint32_t r = threadIdx.x + (uint32_t)t * kRouteThreads;
            const uint32_t q = (r >= r0) + (r >= r1) + (r >= r2) + (r >= r3);
            g[t] = s_g[q < kBnd ? q : kBnd];
            w[t] = s_w[q < kBnd ? q : kBnd];
            if (r < nb && r >= r3 && r3 < T) {  // more than kBnd boundaries in this block
                uint32_t j = j0 + kBnd;
                while (j + 1 < J && off[j + 1] <= bstart + r) ++j;
                g[t] = gmap[j] < NG ? gmap[j] : NG - 1;
                const uint32_t ww = specs[(uint64_t)g[t] * cands].window;
                w[t] = ww < NW ? ww : 0u;
            }
        }
        uint32_t ar[kP1];
#pragma unroll
        for (int t = 0; t < kP1; ++t) {
            const uint32_t r = threadIdx.x + (uint32_t)t * kRouteThreads;
            const bool ok = r < nb && b[t] < K;
            bad |= r < nb && b[t] >= K;
            ar[t] = ld_at<uint32_t>(wrank, (w[t] * K + (ok ? b[t] : 0u)) * 4u);
            ar[t] = ok && ar[t] < cmax ? ar[t] : 0xFFFFFFFFu;
        }
#pragma unroll
        for (int t = 0; t < kP1; ++t) {
            const uint32_t r = threadIdx.x + (uint32_t)t * kRouteThreads;
            if (r >= T) break;
            const uint64_t gi = first_index + bstart + r;
            const uint32_t h = fmix32((uint32_t)gi ^ fmix32((uint32_t)(gi >> 32) ^ smix));
            m_a[r] = ar[t];
            m_d[r] = (((h & 0xFFFFu) * R) >> 16) | ((((h >> 16) * R) >> 16) << 16);
            m_g[r] = g[t];
            m_h[r] = h;
        }
    }
    __syncthreads();
    // phase 2
    const uint32_t tasks = (T / 4u) * NP;
    for (uint32_t q = threadIdx.x; q < tasks; q += kRouteThreads) {
        const uint32_t rq = q / NP, pc = q % NP, ra = 4u * rq;
        const uint4 va = *reinterpret_cast<const uint4*>(m_a + ra);
        const uint4 vd = *reinterpret_cast<const uint4*>(m_d + ra);
        const uint4 vg = *reinterpret_cast<const uint4*>(m_g + ra);
        uint32_t roff[4];  // element index of the 8-entry piece in group_dest and group_multi
        uint4 row[4], x1[4], x2[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const uint32_t A = u4_at(va, s), D = u4_at(vd, s), G = u4_at(vg, s);
            roff[s] = (G * cmax + (A != 0xFFFFFFFFu ? A : 0u)) * CS + 8u * pc;
            row[s] = ld_at<uint4>(gdest, roff[s] * 2u);
            const uint32_t rb = G * R * CS + 8u * pc;
            x1[s] = ld_at<uint4>(grank, (rb + (D & 0xFFFFu) * CS) * 2u);
            x2[s] = ld_at<uint4>(grank, (rb + (D >> 16) * CS) * 2u);
        }
        uint32_t ent[4][8];
        bool multi = false;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const uint32_t A = u4_at(va, s), D = u4_at(vd, s);
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const uint32_t sh = (u & 1) * 16;
                const uint32_t ev = A == 0xFFFFFFFFu ? CR_GROUP_COLD : (u4_at(row[s], u >> 1) >> sh) & 0xFFFFu;
                const uint32_t q1 = (u4_at(x1[s], u >> 1) >> sh) & 0xFFFFu, q2 = (u4_at(x2[s], u >> 1) >> sh) & 0xFFFFu;
                const uint32_t cold = q2 < q1 ? (D >> 16) : (D & 0xFFFFu);
                ent[s][u] = ev == CR_GROUP_COLD ? cold : ev;
                multi |= ev == CR_GROUP_MULTI;
            }
        }
        if (multi) {  // k > 1: the member picked by the request hash
            uint4 mv[4][2];
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                mv[s][0] = ld_at<uint4>(gmulti, roff[s] * 4u);
                mv[s][1] = ld_at<uint4>(gmulti, roff[s] * 4u + 16u);
            }
            const uint4 vh = *reinterpret_cast<const uint4*>(m_h + ra);
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                const uint32_t G = u4_at(vg, s), H = u4_at(vh, s);
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const bool m = ent[s][u] == CR_GROUP_MULTI;
                    const uint32_t ok = u4_at(mv[s][u >> 2], u & 3);
                    const uint32_t pick = (ok & 0xFFFFFu) + (((H >> 16) * (ok >> 20)) >> 16);
                    const uint32_t idx = m ? (G * cands + 8u * pc + (uint32_t)u) * cmax + pick : 0u;
                    const uint32_t dm = ld_at<uint16_t>(members, idx * 2u);
                    ent[s][u] = m ? dm : ent[s][u];
                }
            }
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            uint32_t* __restrict__ tr = tile + (8u * pc + u) * TS2 + 2u * rq;
            tr[0] = ent[0][u] | (ent[1][u] << 16);
            tr[1] = ent[2][u] | (ent[3][u] << 16);
        }
    }
    __syncthreads();
    // phase 3
    const uint32_t nw = (nb + 1u) / 2u;  // words holding at least one request of the block
    for (uint32_t c = 0; c < cands; ++c) {
        const uint32_t* __restrict__ tr = tile + c * TS2;
        uint16_t* __restrict__ dc = dest + (uint64_t)c * n + bstart;
        for (uint32_t wdx = threadIdx.x; wdx < nw; wdx += kRouteThreads) {
            const uint32_t v = tr[wdx];
            if (kVec) {
                __builtin_nontemporal_store(v, reinterpret_cast<uint32_t*>(dc) + wdx);  // n even: both halves used
            } else {
                dc[2u * wdx] = (uint16_t)v;
                if (2u * wdx + 1u < nb) dc[2u * wdx + 1u] = (uint16_t)(v >> 16);
            }
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
    const bool grouped = plans->window_rank || plans->group_dest || plans->group_rank || plans->group_multi;
    if (grouped) {
        if (!plans->window_rank || !plans->group_dest || !plans->group_rank || !plans->group_multi ||
            ((uintptr_t)plans->group_dest & 15u) || ((uintptr_t)plans->group_rank & 15u) ||
            ((uintptr_t)plans->group_multi & 15u) || ((uintptr_t)plans->window_rank & 3u) || !plans->specs ||
            !plans->order || !plans->n_order || !plans->num_admitted)
            return CR_EINVAL;
        if (plans->num_windows > 65535u || plans->num_plans / plans->cands > 65535u) return CR_EINVAL;  // grid y
        // the kernels address every table with 32-bit byte offsets
        const uint64_t NG = plans->num_plans / plans->cands, CS = (plans->cands + 7u) & ~7u;
        if ((uint64_t)plans->num_windows * plans->num_keys * 4u > 0xFFFFFFFFull ||
            NG * cmax * CS * 4u > 0xFFFFFFFFull || (uint64_t)plans->num_plans * cmax * 2u > 0xFFFFFFFFull)
            return CR_EINVAL;
    }
    (void)hipGetLastError();
    if (grouped) {
        const hipStream_t st = as_stream(stream);
        const uint32_t NG = plans->num_plans / plans->cands, cands = plans->cands;
        const uint32_t CS = (cands + 7u) & ~7u;
        const uint64_t wr_n = (uint64_t)plans->num_windows * plans->num_keys;
        const uint32_t T = group_tile(CS);
        const uint64_t gblocks = (n + T - 1) / T;
        if (gblocks > 0x7FFFFFF0ull) return CR_EINVAL;
        const size_t lds = group_route_lds(CS);
        hipLaunchKernelGGL(k_fill_u32, dim3(2048), dim3(256), 0, st, plans->window_rank, wr_n, 0xFFFFFFFFu);
        hipLaunchKernelGGL(k_win_rank_set, dim3((cmax + 255u) / 256u, plans->num_windows), dim3(256), 0, st,
                           plans->order, plans->n_order, cmax, plans->num_keys, plans->window_rank);
        hipLaunchKernelGGL(k_group_dest, dim3((cmax + kGrpRows - 1u) / kGrpRows, NG), dim3(kGrpThreads), 0, st, cands,
                           CS, cmax, plans->specs, plans->num_admitted, plans->member_off, plans->members,
                           plans->group_dest, plans->group_multi, err);
        hipLaunchKernelGGL(k_group_rank, dim3(CS, NG), dim3(256), 0, st, plans->R, cands, CS, plans->load,
                           plans->group_rank);
        // 32-bit destination stores need an even n and a 4-byte aligned dest
        const bool v32 = ((uintptr_t)dest & 3u) == 0 && (n & 1u) == 0;
#define CR_ROUTE_GROUP(V)                                                                                          \
    do {                                                                                                           \
        if (hipFuncSetAttribute((const void*)k_route_group<V>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) \
            != hipSuccess)                                                                                         \
            return CR_EHIP;                                                                                        \
        hipLaunchKernelGGL((k_route_group<V>), dim3(xcd_grid((uint32_t)gblocks)), dim3(kRouteThreads), lds, st, keys, \
                           n, first_index, seed_mix(seed), off, gmap, J, plans->num_keys, plans->R, cands, CS, NG,   \
                           plans->num_windows, cmax, plans->specs, plans->window_rank, plans->group_dest,            \
                           plans->group_rank, plans->group_multi, plans->members, dest, err);                       \
    } while (0)
        if (v32) CR_ROUTE_GROUP(true);
        else CR_ROUTE_GROUP(false);
#undef CR_ROUTE_GROUP
        return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
    }
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
