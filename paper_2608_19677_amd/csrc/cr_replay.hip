// Shadow replay of P candidate routings against per-destination LRU prefix caches
// (Section 3.2: admitted and cold prefixes share one cache per destination; Section 3.1
// equal-slot model: W whole-prefix slots per destination).
//
// Pipeline (all on the caller's stream, workspace from the caller):
//   k_part_hist / k_scan_dest / k_seg_items / k_part_scatter
//        stable partition of every candidate's requests by destination, preserving
//        arrival order; each record packs (key, suffix, interval) into 8 bytes;
//        k_seg_items also splits every (candidate, destination) stream into segments of
//        S records;
//   k_replay<SL>
//        one wavefront per segment. The LRU state before a segment is exactly the most
//        recent W distinct keys seen at that destination (carried state appended), so a
//        wavefront rebuilds it by scanning backwards, then replays its segment. This
//        turns R*P sequential streams into thousands of independent wavefronts with
//        results identical to one sequential pass;
//   k_replay_grp<G>
//        lists of at most 16 slots in calls with one interval: G = 4 or 8 segments per
//        wavefront, one per lane group (below).
// The LRU lives in registers. Up to 64 slots it is a move-to-front list across the lanes:
// lane i holds the i-th most recent key. A lookup is one compare and a ballot; the first
// set bit p is the hit depth, and the update shifts lanes 0..p (all lanes on a miss) up
// by one and writes the key into lane 0, a single select between a lane and its left
// neighbour under a scalar mask. Above 64 slots the list takes SL = ceil(W / 64)
// registers. Up to 128 slots it is interleaved over them (position SL * lane + s in
// register s), so that moving a position back by one is a copy from register s-1 in the
// same lane, and only the last register wraps into register 0 of the next lane through a
// one-lane DPP shift; an access is SL compares and SL selects under scalar masks, without
// branches. Above 128 slots it is two-level: the 64 most recent keys in a front register
// that every access updates like the one-register list, the rest interleaved behind it and
// touched only when the front misses. No form needs a per-request search or reduction.
#include "cr_common.h"

#include <mutex>

namespace cr {
namespace {

constexpr int kReplayThreads = 256;

struct WArg {
    uint16_t W[CR_MAX_CANDS];
    uint8_t grp[CR_MAX_CANDS];  // lists per wavefront: G > 1 for k_replay_grp<G>, else 1
    uint32_t seg_min;  // shortest segment for this call's record count
};

// The candidates one k_replay launch serves and the first wavefront of each: wavefront v
// takes work item v - wv0[i] of candidate cand[i] for wv0[i] <= v < wv0[i + 1]. Each
// candidate gets as many wavefronts as it can have work items (one per stream plus one per
// full segment), so a launch runs no wavefront for another list size's candidates. n = 0
// when the launch serves every candidate of the call: wavefront v then takes work item v.
struct CandMap {
    uint32_t n;
    uint16_t cand[CR_MAX_CANDS];
    uint32_t wv0[CR_MAX_CANDS + 1];
};

// Segment i of a stream of cnt records cut into nseg = ceil(cnt / S) segments (at least one):
// records [seg_start(i), seg_start(i + 1)). The stream's ceil(cnt / 64) batches of 64 records
// are dealt evenly, so segments differ by at most one batch and only the last one ends in a
// partial batch (the replay takes a full batch in one unrolled pass, a partial one record by
// record); the wavefronts of a launch thus run for about as long as each other (with
// segments of exactly S, a stream's last one was its remainder, and those short wavefronts
// left the chip part empty near each launch's end). One 32-bit division per bound.
__host__ __device__ __forceinline__ uint32_t seg_start(uint32_t i, uint32_t nseg, uint32_t cnt)
{
    const uint32_t nb = (cnt + 63u) / 64u, L = nb / nseg, r = nb - L * nseg;
    const uint32_t b = i * L + (i < r ? i : r);
    return b < nb ? 64u * b : cnt;
}

// Segments the whole replay is cut into, a few rounds of wavefronts over the chip: a
// wavefront's LRU chain is serial, so several per SIMD hide its latency, and beyond that
// longer segments only save the backward rebuild of the initial state.
constexpr uint64_t kSegTarget = 16384;

// Shortest segment; the launch sizes its grid for segments of this length.
constexpr uint32_t kSegFloor = 1024;
constexpr uint32_t kSegPerSlot = 16;

// Records per segment: at least kSegPerSlot W (the rebuild scans back to W distinct keys)
// and at least the share that keeps the number of segments near kSegTarget. A candidate
// whose wavefronts hold G lists (k_replay_grp) takes segments G times shorter, so that it
// still has as many wavefronts.
__host__ __device__ __forceinline__ uint32_t seg_len(uint32_t W, uint32_t seg_min, uint32_t G)
{
    uint32_t s = kSegPerSlot * W;
    s = s > seg_min ? s : seg_min;
    s = s < kSegFloor ? kSegFloor : (s > 65536u ? 65536u : s);
    if (G > 1u) s = s / G < kSegFloor ? kSegFloor : s / G;
    return s;
}

// Lists per wavefront of a W-slot list in k_replay_grp (lane groups of 64 / G lanes), or 1
// for the one-wavefront-per-list kernels. Only calls with one interval: the grouped kernel
// keeps one set of statistics per segment. Two lists per wavefront (W <= 32) measured
// slower than one on the 1e8-request sweep (10.2 against 7.2 ms for its W = 26 plans).
__host__ __device__ __forceinline__ uint32_t grp_of(uint32_t W, uint32_t J)
{
    if (J != 1u || W > 16u) return 1u;
    return W <= 8u ? 8u : 4u;
}

// Registers per lane of a W-slot list: ceil(W / 64), 1 .. 8. An access costs about one
// compare and one select per register, so each W gets the fewest that hold it.
__host__ __device__ __forceinline__ uint32_t slot_class(uint32_t W)
{
    const uint32_t sl = (W + 63u) / 64u;
    return sl < 1u ? 1u : (sl > 8u ? 8u : sl);
}

// Lists of 3 registers and more are two-level (a 64-key front and the rest behind it). On
// the 1e8-request sweep: W = 156 19.8 ms two-level against 21.6 interleaved, W = 283 26.6
// against 32.7; at W = 86 (two registers) interleaved was faster, 16.1 against 16.5 ms.
constexpr uint32_t kTwoLevelFrom = 3;

struct PartGeom {
    uint64_t tile;
    uint64_t ntiles;
};

inline PartGeom part_geom(uint64_t n, uint32_t P)
{
    const uint64_t target = 16384u / P > 0 ? 16384u / P : 1u;
    uint64_t tile = (n + target - 1) / target;
    tile = (tile + 1023) & ~1023ull;  // whole sub-tiles of the scatter
    if (tile < 1024) tile = 1024;
    return PartGeom{tile, n ? (n + tile - 1) / tile : 0};
}

// Per-tile destination counts; with aligned rows (kVec) every thread reads four
// destinations with one 8-byte load.
constexpr uint32_t kHistThreads = 256;

template <bool kVec>
__global__ __launch_bounds__(kHistThreads) void k_part_hist(const uint16_t* __restrict__ dest, uint64_t n, uint32_t R,
                                                            uint64_t tile, uint64_t ntiles, uint32_t* __restrict__ tcnt,
                                                            uint32_t* __restrict__ err)
{
    issue_priority_high();
    extern __shared__ uint32_t h[];
    const uint32_t c = blockIdx.y;
    const uint64_t t = blockIdx.x;
    const uint64_t t0 = t * tile, t1 = t0 + tile < n ? t0 + tile : n;
    for (uint32_t d = threadIdx.x; d < R; d += blockDim.x) h[d] = 0;
    __syncthreads();
    const uint16_t* __restrict__ dc = dest + (uint64_t)c * n;
    bool bad = false;
    auto add = [&](uint32_t d) {
        if (d < R) atomicAdd(&h[d], 1u);
        else bad = true;
    };
    uint64_t a = t0;
    if (kVec) {
        for (; a + 4u * kHistThreads <= t1; a += 4u * kHistThreads) {
            const uint2 q = *reinterpret_cast<const uint2*>(dc + a + 4u * threadIdx.x);
            add(q.x & 0xFFFFu);
            add(q.x >> 16);
            add(q.y & 0xFFFFu);
            add(q.y >> 16);
        }
    }
    for (uint64_t i = a + threadIdx.x; i < t1; i += blockDim.x) add(dc[i]);
    __syncthreads();
    for (uint32_t d = threadIdx.x; d < R; d += blockDim.x) tcnt[((uint64_t)c * R + d) * ntiles + t] = h[d];
    if (bad) atomicOr(err, CR_ERR_DEST_RANGE);
}

// One block per (destination, candidate): exclusive scan of that destination's per-tile
// counts, which are contiguous in tcnt[c][d][tile], in place; the destination's total goes
// to dtot[c][d]. Destination bases within a candidate are added later (k_seg_items).
constexpr uint32_t kScanThreads = 1024;

__global__ __launch_bounds__(kScanThreads) void k_scan_dest(uint32_t* __restrict__ tcnt, uint64_t ntiles, uint32_t R,
                                                            uint32_t* __restrict__ dtot)
{
    issue_priority_high();
    __shared__ uint32_t s_scan[16];
    const uint32_t d = blockIdx.x, c = blockIdx.y;
    uint32_t* __restrict__ t = tcnt + ((uint64_t)c * R + d) * ntiles;
    uint32_t carry = 0;
    for (uint64_t e0 = 0; e0 < ntiles; e0 += 4u * kScanThreads) {
        const uint64_t e = e0 + 4u * threadIdx.x;
        uint32_t v[4], sum = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            v[q] = e + q < ntiles ? t[e + q] : 0u;
            sum += v[q];
        }
        uint32_t tot;
        uint32_t ex = block_exscan_u32(sum, s_scan, &tot) + carry;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (e + q < ntiles) t[e + q] = ex;
            ex += v[q];
        }
        carry += tot;
    }
    if (threadIdx.x == 0) dtot[(uint64_t)c * R + d] = carry;
}

// One wavefront per (tile, candidate): stable scatter into packed records, kSub requests
// at a time. Pass one ranks every request among the earlier ones of its destination in
// the sub-tile (ballots over the destination bits, plus a per-destination counter in
// LDS); the records are then staged in LDS in destination order and written out so that
// consecutive lanes store consecutive addresses of one destination's run: whole cache
// lines instead of a few bytes in each of R streams per instruction.
constexpr uint32_t kSub = 1024;
constexpr uint32_t kSubChunks = kSub / 64;
static_assert(kSub == 1024, "part_geom rounds tiles to 1024 requests");

inline size_t scatter_lds_bytes(uint32_t R) { return (size_t)kSub * 12u + (size_t)R * 12u; }

__global__ __launch_bounds__(64) void k_part_scatter(const uint32_t* __restrict__ keys,
                                                     const uint16_t* __restrict__ suffix,
                                                     const uint16_t* __restrict__ dest, uint64_t n,
                                                     const uint64_t* __restrict__ off, uint32_t J, uint32_t R,
                                                     uint32_t nbits, uint64_t tile, uint64_t ntiles,
                                                     const uint32_t* __restrict__ tcnt,
                                                     const uint32_t* __restrict__ grp_off, uint64_t* __restrict__ rec)
{
    issue_priority_high();
    extern __shared__ uint64_t lds[];
    uint64_t* srec = lds;                                        // [kSub] staged records
    uint32_t* spos = reinterpret_cast<uint32_t*>(srec + kSub);  // [kSub] their output positions
    uint32_t* run = spos + kSub;                                 // [R] next output position
    uint32_t* lcnt = run + R;                                    // [R] sub-tile count
    uint32_t* loff = lcnt + R;                                   // [R] sub-tile offset
    const uint32_t c = blockIdx.y, lane = lane_id();
    const uint64_t t = xcd_tile(blockIdx.x, gridDim.x);
    if (t >= ntiles) return;
    const uint64_t t0 = t * tile, t1 = t0 + tile < n ? t0 + tile : n;
    for (uint32_t d = lane; d < R; d += 64) {
        run[d] = grp_off[(uint64_t)c * (R + 1u) + d] + tcnt[((uint64_t)c * R + d) * ntiles + t];
        lcnt[d] = 0;
    }
    __syncthreads();
    const uint16_t* __restrict__ dc = dest + (uint64_t)c * n;
    uint64_t* __restrict__ rc = rec + (uint64_t)c * n;
    const uint32_t per = (R + 63u) >> 6;  // destinations per lane in the offset scan
    uint32_t j = find_interval(off, J, t0);
    uint64_t jend = j + 1 < J ? off[j + 1] : ~0ull;  // first request of the next interval
    for (uint64_t sb = t0; sb < t1; sb += kSub) {
        const uint64_t se = sb + kSub < t1 ? sb + kSub : t1;
        uint32_t dk[kSubChunks], kv[kSubChunks], mv[kSubChunks];
#pragma unroll
        for (uint32_t m = 0; m < kSubChunks; ++m) {
            const uint64_t i = sb + m * 64u + lane;
            const bool in = i < se;
            dk[m] = in ? dc[i] : 0xFFFFu;
            kv[m] = in ? keys[i] : 0u;
            mv[m] = in ? suffix[i] : 0u;
        }
#pragma unroll
        for (uint32_t m = 0; m < kSubChunks; ++m) {
            const uint64_t base = sb + m * 64u;
            if (base >= se) {  // past the end of the tile: nothing to stage
                dk[m] = 0xFFFFFFFFu;
                continue;
            }
            const uint64_t i = base + lane;
            const uint32_t d = dk[m];
            const bool valid = i < se && d < R;
            uint32_t jl = j;
            if (base + 63 >= jend) {  // an interval boundary falls inside these 64 requests
                while (jl + 1 < J && off[jl + 1] <= i) ++jl;
                j = rdlane(jl, 63);
                jend = j + 1 < J ? off[j + 1] : ~0ull;
            }
            uint64_t peers = ballot(valid);
            for (uint32_t bit = 0; bit < nbits; ++bit) {
                const bool on = (d >> bit) & 1u;
                const uint64_t bb = ballot(on);
                peers &= on ? bb : ~bb;
            }
            const uint32_t rk = (uint32_t)__popcll(peers & lanemask_lt());
            const uint32_t lr = valid ? lcnt[d] + rk : 0u;
            __syncthreads();
            if (valid && rk == 0) lcnt[d] += (uint32_t)__popcll(peers);
            __syncthreads();
            dk[m] = valid ? (d << 16) | lr : 0xFFFFFFFFu;
            mv[m] |= jl << 16;
        }
        // exclusive offsets of the destinations within the sub-tile
        uint32_t own = 0;
        for (uint32_t q = 0; q < per; ++q) {
            const uint32_t d = lane * per + q;
            own += d < R ? lcnt[d] : 0u;
        }
        uint32_t acc = wave_incl_scan_u32(own) - own;
        const uint32_t total = rdlane(acc + own, 63);
        for (uint32_t q = 0; q < per; ++q) {
            const uint32_t d = lane * per + q;
            if (d < R) {
                loff[d] = acc;
                acc += lcnt[d];
            }
        }
        __syncthreads();
#pragma unroll
        for (uint32_t m = 0; m < kSubChunks; ++m) {
            if (dk[m] != 0xFFFFFFFFu) {
                const uint32_t d = dk[m] >> 16, lr = dk[m] & 0xFFFFu;
                const uint32_t slot = loff[d] + lr;
                srec[slot] = (uint64_t)kv[m] | ((uint64_t)mv[m] << 32);
                spos[slot] = run[d] + lr;
            }
        }
        __syncthreads();
        for (uint32_t q = lane; q < total; q += 64) rc[spos[q]] = srec[q];
        __syncthreads();
        for (uint32_t d = lane; d < R; d += 64) {
            run[d] += lcnt[d];
            lcnt[d] = 0;
        }
        __syncthreads();
    }
}

// R <= 64: the same scatter with each lane owning a run of kRun consecutive requests of
// the sub-tile. A lane counts its run's destinations in a private row of 16-bit counters in
// LDS, in request order, which ranks every request within its run; a prefix sum of the rows
// across the lanes (packed pairs of counters, one wave scan per pair of destinations) gives
// each lane's offset per destination. A request's rank within the sub-tile is then its lane's
// offset plus its rank within the run: no cross-lane matching of destinations at all. With
// aligned rows (kVec) a lane reads its run with 16-byte loads.
constexpr uint32_t kRun = kSub / 64;

// Row stride in counters: R rounded up to 8 (16-byte pieces).
__host__ __device__ __forceinline__ uint32_t scat64_row(uint32_t R) { return (R + 7u) & ~7u; }

inline size_t scatter64_lds_bytes(uint32_t R) { return (size_t)kSub * 12u + 64u * 8u + 64u * scat64_row(R) * 2u; }

template <bool kVec>
__global__ __launch_bounds__(64) void k_part_scatter64(const uint32_t* __restrict__ keys,
                                                       const uint16_t* __restrict__ suffix,
                                                       const uint16_t* __restrict__ dest, uint64_t n,
                                                       const uint64_t* __restrict__ off, uint32_t J, uint32_t R,
                                                       uint64_t tile, uint64_t ntiles, const uint32_t* __restrict__ tcnt,
                                                       const uint32_t* __restrict__ grp_off,
                                                       uint64_t* __restrict__ rec)
{
    issue_priority_high();
    extern __shared__ uint64_t lds[];
    uint64_t* srec = lds;                                            // [kSub] staged records
    uint32_t* spos = reinterpret_cast<uint32_t*>(srec + kSub);      // [kSub] their output positions
    uint64_t* sbase = reinterpret_cast<uint64_t*>(spos + kSub);     // [64] {sub-tile offset, output position}
    uint16_t* rows = reinterpret_cast<uint16_t*>(sbase + 64);       // [64][RW] counters per lane
    uint32_t* stot = spos;  // [64] sub-tile count per destination (spos is free until staging)
    const uint32_t RW = scat64_row(R);
    const uint32_t c = blockIdx.y, lane = lane_id();
    const uint64_t t = xcd_tile(blockIdx.x, gridDim.x);
    if (t >= ntiles) return;
    const uint64_t t0 = t * tile, t1 = t0 + tile < n ? t0 + tile : n;
    // lane d: next output position of destination d
    uint32_t run = lane < R ? grp_off[(uint64_t)c * (R + 1u) + lane] + tcnt[((uint64_t)c * R + lane) * ntiles + t] : 0u;
    const uint16_t* __restrict__ dc = dest + (uint64_t)c * n;
    uint64_t* __restrict__ rc = rec + (uint64_t)c * n;
    uint16_t* row = rows + lane * RW;
    uint32_t jw = find_interval(off, J, t0);  // interval of the sub-tile's first request
    for (uint64_t sb = t0; sb < t1; sb += kSub) {
        const uint64_t se = sb + kSub < t1 ? sb + kSub : t1;
        const uint64_t i0 = sb + (uint64_t)lane * kRun;
        uint32_t kv[kRun], dv[kRun], mv[kRun];
        if (kVec && se - sb == kSub) {
            const uint4* k4 = reinterpret_cast<const uint4*>(keys + i0);
            const uint4* d4 = reinterpret_cast<const uint4*>(dc + i0);
            const uint4* m4 = reinterpret_cast<const uint4*>(suffix + i0);
            uint4 qk[4], qd[2], qm[2];
#pragma unroll
            for (uint32_t v = 0; v < 4; ++v) qk[v] = k4[v];
#pragma unroll
            for (uint32_t v = 0; v < 2; ++v) {
                qd[v] = d4[v];
                qm[v] = m4[v];
            }
#pragma unroll
            for (uint32_t v = 0; v < 4; ++v) {
                kv[4 * v + 0] = qk[v].x;
                kv[4 * v + 1] = qk[v].y;
                kv[4 * v + 2] = qk[v].z;
                kv[4 * v + 3] = qk[v].w;
            }
#pragma unroll
            for (uint32_t v = 0; v < 2; ++v) {
                const uint32_t dw[4] = {qd[v].x, qd[v].y, qd[v].z, qd[v].w};
                const uint32_t mw[4] = {qm[v].x, qm[v].y, qm[v].z, qm[v].w};
#pragma unroll
                for (uint32_t h = 0; h < 4; ++h) {
                    dv[8 * v + 2 * h] = dw[h] & 0xFFFFu;
                    dv[8 * v + 2 * h + 1] = dw[h] >> 16;
                    mv[8 * v + 2 * h] = mw[h] & 0xFFFFu;
                    mv[8 * v + 2 * h + 1] = mw[h] >> 16;
                }
            }
        } else {
#pragma unroll
            for (uint32_t v = 0; v < kRun; ++v) {
                const uint64_t i = i0 + v;
                const bool in = i < se;
                dv[v] = in ? dc[i] : 0xFFFFu;
                kv[v] = in ? keys[i] : 0u;
                mv[v] = in ? suffix[i] : 0u;
            }
        }
        for (uint32_t w = 0; w < RW; w += 8) *reinterpret_cast<uint4*>(row + w) = make_uint4(0u, 0u, 0u, 0u);
        // interval of each request: from the sub-tile's, past the boundaries up to it
        uint32_t jl = jw;
        uint64_t nb = jl + 1 < J ? off[jl + 1] : ~0ull;  // first request of the next interval
        // rank of each request within the run: the run's earlier requests to its destination
#pragma unroll
        for (uint32_t v = 0; v < kRun; ++v) {
            const uint64_t i = i0 + v;
            const bool in = i < se;
            while (in && i >= nb) {
                ++jl;
                nb = jl + 1 < J ? off[jl + 1] : ~0ull;
            }
            mv[v] |= jl << 16;
            const uint32_t d = dv[v];
            if (in && d < R) {
                const uint32_t r = row[d];
                row[d] = (uint16_t)(r + 1u);
                dv[v] = d | (r << 16);
            } else {
                dv[v] = 0xFFFFFFFFu;
            }
        }
        // exclusive prefix of the rows across the lanes; lane 63's inclusive sums are the
        // sub-tile's counts per destination
        for (uint32_t w = 0; w < RW; w += 8) {
            uint4* q = reinterpret_cast<uint4*>(row + w);
            const uint4 own = *q;
            const uint4 inc = make_uint4(wave_incl_scan_u32(own.x), wave_incl_scan_u32(own.y),
                                         wave_incl_scan_u32(own.z), wave_incl_scan_u32(own.w));
            *q = make_uint4(inc.x - own.x, inc.y - own.y, inc.z - own.z, inc.w - own.w);
            if (lane == 63) {
                const uint32_t iw[4] = {inc.x, inc.y, inc.z, inc.w};
#pragma unroll
                for (uint32_t h = 0; h < 4; ++h) {
                    stot[w + 2 * h] = iw[h] & 0xFFFFu;
                    stot[w + 2 * h + 1] = iw[h] >> 16;
                }
            }
        }
        __syncthreads();
        // destination offsets within the sub-tile (lane d)
        const uint32_t tl = lane < R ? stot[lane] : 0u;
        const uint32_t ex = wave_incl_scan_u32(tl) - tl;
        const uint32_t total = rdlane(ex + tl, 63);
        sbase[lane] = (uint64_t)ex | ((uint64_t)run << 32);
        __syncthreads();
#pragma unroll
        for (uint32_t v = 0; v < kRun; ++v) {
            if (dv[v] != 0xFFFFFFFFu) {
                const uint32_t d = dv[v] & 0xFFFFu;
                const uint32_t lr = row[d] + (dv[v] >> 16);
                const uint64_t bs = sbase[d];
                const uint32_t slot = (uint32_t)bs + lr;
                srec[slot] = (uint64_t)kv[v] | ((uint64_t)mv[v] << 32);
                spos[slot] = (uint32_t)(bs >> 32) + lr;
            }
        }
        __syncthreads();
        for (uint32_t q = lane; q < total; q += 64) rc[spos[q]] = srec[q];
        run += tl;
        while (jw + 1 < J && off[jw + 1] <= se) ++jw;  // interval of the next sub-tile's first request
        __syncthreads();
    }
}

// R > 64, several wavefronts per block: sub-tiles of kWideSub requests, wavefront w taking
// the sub-tile's requests 1024 w .. 1024 w + 1023 as 16 chunks of 64 in order. A chunk ranks
// each request among its chunk's requests to the same destination by ballots over the
// destination bits; the chunk's leader adds the chunk's count to the wavefront's counter of
// that destination in LDS and hands the old value to its peers, which ranks the request
// within the wavefront's requests. Per destination, a block scan over the totals gives the
// destination's run in the sub-tile and each wavefront's base in it; the records are staged
// in LDS in destination order and written out run by run (about kWideSub / R consecutive
// records per destination, against one in k_part_scatter's 1,024-request sub-tiles).
// Blocks are dealt to the XCDs round-robin; block b takes candidate (b / 8) mod P of tile
// ((b / 8) / P) * 8 + b mod 8, so that an XCD runs the P candidates of one tile together
// and fetches the tile's keys and suffixes into its L2 once for all of them (with the
// candidates fastest over the whole grid, each XCD held eight tiles' keys at a time, more
// than its L2, and read them about once per candidate).
constexpr uint32_t kWideWaves = 4;
constexpr uint32_t kWideThreads = 64 * kWideWaves;
constexpr uint32_t kWideSub = 1024 * kWideWaves;
constexpr uint32_t kWideChunks = 16;  // chunks of 64 per wavefront and sub-tile

__host__ __device__ __forceinline__ uint32_t wide_row(uint32_t R) { return (R + 3u) & ~3u; }  // padded to 4 per thread

// LDS: staged records and their destinations, per-wavefront counters and the runs' bases,
// and per wavefront two matching scratch areas (64 peer masks, then one byte per
// destination), one for even and one for odd chunks.
inline size_t scatter_wide_lds_bytes(uint32_t R)
{
    return (size_t)kWideSub * 10u + (size_t)wide_row(R) * 4u * (kWideWaves + 1u) +
           (size_t)kWideWaves * 2u * (512u + ((wide_row(R) + 7u) & ~7u));
}

__global__ __launch_bounds__(kWideThreads) void k_part_scatter_wide(
    const uint32_t* __restrict__ keys, const uint16_t* __restrict__ suffix, const uint16_t* __restrict__ dest,
    uint64_t n, const uint64_t* __restrict__ off, uint32_t J, uint32_t P, uint32_t R, uint32_t nbits,
    uint64_t tile, uint64_t ntiles, const uint32_t* __restrict__ tcnt, const uint32_t* __restrict__ grp_off,
    uint64_t* __restrict__ rec)
{
    issue_priority_high();
    extern __shared__ uint64_t lds[];
    const uint32_t R4 = wide_row(R);
    uint64_t* srec = lds;                                           // [kWideSub] staged records
    uint16_t* sdst = reinterpret_cast<uint16_t*>(srec + kWideSub);  // [kWideSub] their destinations
    uint32_t* cnt = reinterpret_cast<uint32_t*>(sdst + kWideSub);  // [kWideWaves][R4] counts per wavefront, then its slot bases
    uint32_t* gbase = cnt + kWideWaves * R4;  // [R4] output position of the destination's run minus its start
    __shared__ uint32_t s_scan[16];
    const uint32_t bi = blockIdx.x / kXcds;
    const uint32_t c = bi % P, lane = lane_id(), wv = wave_in_block(), tid = threadIdx.x;
    // this wavefront's matching scratch, two areas (even and odd chunks): peer masks by
    // representative lane, and a tag byte per destination naming the representative
    const uint32_t area = 64u + (R4 + 7u) / 8u;  // 8-byte words
    unsigned long long* pm0 = reinterpret_cast<unsigned long long*>(gbase + R4) + wv * 2u * area;
    unsigned long long* pm1 = pm0 + area;
    uint8_t* tag0 = reinterpret_cast<uint8_t*>(pm0 + 64);
    uint8_t* tag1 = reinterpret_cast<uint8_t*>(pm1 + 64);
    const uint64_t t = (uint64_t)(bi / P) * kXcds + blockIdx.x % kXcds;
    if (t >= ntiles) return;
    const uint64_t t0 = t * tile, t1 = t0 + tile < n ? t0 + tile : n;
    // thread tid owns destinations 4 tid .. 4 tid + 3 in the scans: their next output positions
    const bool owner = 4u * tid < R4;
    uint32_t run[4];
#pragma unroll
    for (uint32_t q = 0; q < 4; ++q) {
        const uint32_t d = 4u * tid + q;
        run[q] = d < R ? grp_off[(uint64_t)c * (R + 1u) + d] + tcnt[((uint64_t)c * R + d) * ntiles + t] : 0u;
    }
    const uint16_t* __restrict__ dc = dest + (uint64_t)c * n;
    uint64_t* __restrict__ rc = rec + (uint64_t)c * n;
    uint32_t* __restrict__ wc = cnt + wv * R4;
    for (uint64_t sb = t0; sb < t1; sb += kWideSub) {
        const uint64_t se = sb + kWideSub < t1 ? sb + kWideSub : t1;
        if (owner)
#pragma unroll
            for (uint32_t w = 0; w < kWideWaves; ++w)
                *reinterpret_cast<uint4*>(cnt + w * R4 + 4u * tid) = make_uint4(0u, 0u, 0u, 0u);
        __syncthreads();
        // this wavefront's requests: ws .. ws + 1023 of the sub-tile
        const uint64_t ws = sb + 1024u * wv;
        uint32_t jl = ws < se ? find_interval(off, J, ws) : 0u;
        uint64_t jend = jl + 1 < J ? off[jl + 1] : ~0ull;
        uint32_t dk[kWideChunks], kv[kWideChunks], mv[kWideChunks];
#pragma unroll
        for (uint32_t m = 0; m < kWideChunks; ++m) {
            const uint64_t i = ws + 64u * m + lane;
            const bool in = i < se;
            dk[m] = in ? dc[i] : 0xFFFFu;
            kv[m] = in ? keys[i] : 0u;
            mv[m] = in ? suffix[i] : 0u;
        }
        // Chunks in pairs, each with its own matching area, so that the LDS round trips of
        // the two chunks overlap. Lanes with the same destination: every lane writes its id
        // into the destination's tag byte and reads it back, so the lanes of one destination
        // read one common representative (whichever write landed last); each lane then sets
        // its bit in the representative's peer mask and reads the mask. LDS operations of a
        // wavefront complete in order, so no barrier is needed, and the counter updates of
        // chunk m precede those of chunk m + 1.
#pragma unroll
        for (uint32_t m = 0; m < kWideChunks; m += 2) {
            uint32_t dd[2], jj[2];
            bool vv[2];
#pragma unroll
            for (uint32_t h = 0; h < 2; ++h) {
                const uint64_t base = ws + 64u * (m + h);
                const uint64_t i = base + lane;
                dd[h] = dk[m + h];
                vv[h] = i < se && dd[h] < R;
                uint32_t j = jl;
                if (base < se && base + 63 >= jend) {  // an interval boundary falls inside these 64
                    while (j + 1 < J && off[j + 1] <= i) ++j;
                    jl = rdlane(j, 63);
                    jend = jl + 1 < J ? off[jl + 1] : ~0ull;
                }
                jj[h] = j;
            }
            pm0[lane] = 0ull;
            pm1[lane] = 0ull;
            if (vv[0]) tag0[dd[0]] = (uint8_t)lane;
            if (vv[1]) tag1[dd[1]] = (uint8_t)lane;
            const uint32_t rep0 = vv[0] ? (uint32_t)tag0[dd[0]] : lane;
            const uint32_t rep1 = vv[1] ? (uint32_t)tag1[dd[1]] : lane;
            if (vv[0]) atomicOr(&pm0[rep0], 1ull << lane);
            if (vv[1]) atomicOr(&pm1[rep1], 1ull << lane);
            const uint64_t peers0 = vv[0] ? (uint64_t)pm0[rep0] : 0ull;
            const uint64_t peers1 = vv[1] ? (uint64_t)pm1[rep1] : 0ull;
            const uint32_t rk0 = (uint32_t)__popcll(peers0 & lanemask_lt());
            const uint32_t rk1 = (uint32_t)__popcll(peers1 & lanemask_lt());
            const uint32_t ld0 = vv[0] ? (uint32_t)__builtin_ctzll(peers0) : lane;
            const uint32_t ld1 = vv[1] ? (uint32_t)__builtin_ctzll(peers1) : lane;
            uint32_t old0 = 0, old1 = 0;
            if (vv[0] && rk0 == 0) old0 = atomicAdd(&wc[dd[0]], (uint32_t)__popcll(peers0));
            if (vv[1] && rk1 == 0) old1 = atomicAdd(&wc[dd[1]], (uint32_t)__popcll(peers1));
            old0 = (uint32_t)__builtin_amdgcn_ds_bpermute((int)(ld0 << 2), (int)old0);
            old1 = (uint32_t)__builtin_amdgcn_ds_bpermute((int)(ld1 << 2), (int)old1);
            dk[m] = vv[0] ? (dd[0] << 16) | (old0 + rk0) : 0xFFFFFFFFu;  // destination, rank in the wavefront
            dk[m + 1] = vv[1] ? (dd[1] << 16) | (old1 + rk1) : 0xFFFFFFFFu;
            mv[m] |= jj[0] << 16;
            mv[m + 1] |= jj[1] << 16;
        }
        __syncthreads();
        // destination runs in the sub-tile: each wavefront's slot base within its destination's
        // run, and the run's output position minus its start (16-byte accesses, one thread per
        // four destinations)
        uint4 cw[kWideWaves];
        uint32_t tq[4] = {0u, 0u, 0u, 0u};
        if (owner) {
#pragma unroll
            for (uint32_t w = 0; w < kWideWaves; ++w) {
                cw[w] = *reinterpret_cast<const uint4*>(cnt + w * R4 + 4u * tid);
                tq[0] += cw[w].x, tq[1] += cw[w].y, tq[2] += cw[w].z, tq[3] += cw[w].w;
            }
        }
        uint32_t total;
        uint32_t acc = block_exscan_u32(tq[0] + tq[1] + tq[2] + tq[3], s_scan, &total);
        if (owner) {
            uint32_t st[4];
#pragma unroll
            for (uint32_t q = 0; q < 4; ++q) {
                st[q] = acc;
                acc += tq[q];
            }
            uint32_t b[4] = {st[0], st[1], st[2], st[3]};
#pragma unroll
            for (uint32_t w = 0; w < kWideWaves; ++w) {
                const uint4 x = cw[w];
                *reinterpret_cast<uint4*>(cnt + w * R4 + 4u * tid) = make_uint4(b[0], b[1], b[2], b[3]);
                b[0] += x.x, b[1] += x.y, b[2] += x.z, b[3] += x.w;
            }
            *reinterpret_cast<uint4*>(gbase + 4u * tid) =
                make_uint4(run[0] - st[0], run[1] - st[1], run[2] - st[2], run[3] - st[3]);
#pragma unroll
            for (uint32_t q = 0; q < 4; ++q) run[q] += tq[q];
        }
        __syncthreads();
#pragma unroll
        for (uint32_t m = 0; m < kWideChunks; ++m) {
            if (dk[m] != 0xFFFFFFFFu) {
                const uint32_t d = dk[m] >> 16, lr = dk[m] & 0xFFFFu;
                const uint32_t slot = wc[d] + lr;
                srec[slot] = (uint64_t)kv[m] | ((uint64_t)mv[m] << 32);
                sdst[slot] = (uint16_t)d;
            }
        }
        __syncthreads();
        for (uint32_t q = tid; q < total; q += kWideThreads) rc[gbase[sdst[q]] + q] = srec[q];
        __syncthreads();
    }
}

// Destination bases and work items, from the destination totals dtot[c][d]:
//   grp_off[c][d] = records of candidate c routed to destinations < d (grp_off[c][R] = all),
//   item_off[e]   = first work item of stream e = c * R + d, one item per segment of S
//                   records (at least one per stream).
// Pass one scans over all (c, d) in one block; pass two rebases grp_off per candidate.
__global__ __launch_bounds__(1024) void k_seg_items(const uint32_t* __restrict__ dtot, uint32_t P, uint32_t R,
                                                    WArg wa, uint32_t* __restrict__ grp_off,
                                                    uint32_t* __restrict__ item_off, uint32_t* __restrict__ gwave_off)
{
    issue_priority_high();
    __shared__ uint32_t s_scan[16];
    __shared__ uint32_t s_cstart[CR_MAX_CANDS + 1];
    const uint32_t total = P * R;
    uint32_t carry = 0, icarry = 0;
    for (uint32_t e0 = 0; e0 < total; e0 += blockDim.x) {
        const uint32_t e = e0 + threadIdx.x;
        uint32_t cnt = 0, nseg = 0;
        if (e < total) {
            cnt = dtot[e];
            const uint32_t S = seg_len(wa.W[e / R], wa.seg_min, wa.grp[e / R]);
            nseg = cnt ? (cnt + S - 1) / S : 1u;
        }
        uint32_t tot, itot;
        const uint32_t ex = block_exscan_u32(cnt, s_scan, &tot);
        const uint32_t iex = block_exscan_u32(nseg, s_scan, &itot);
        if (e < total) {
            const uint32_t c = e / R, d = e % R;
            grp_off[(uint64_t)c * (R + 1u) + d] = carry + ex;
            item_off[e] = icarry + iex;
            if (d == 0) s_cstart[c] = carry + ex;
        }
        carry += tot;
        icarry += itot;
    }
    if (threadIdx.x == 0) {
        item_off[total] = icarry;
        s_cstart[P] = carry;
    }
    __syncthreads();
    for (uint32_t e = threadIdx.x; e < total; e += blockDim.x) {
        const uint32_t c = e / R, d = e % R;
        grp_off[(uint64_t)c * (R + 1u) + d] -= s_cstart[c];
    }
    for (uint32_t c = threadIdx.x; c < P; c += blockDim.x)
        grp_off[(uint64_t)c * (R + 1u) + R] = s_cstart[c + 1] - s_cstart[c];
    // gwave_off[c]: first k_replay_grp wavefront of candidate c (G work items per wavefront;
    // none for candidates replayed one list per wavefront)
    __syncthreads();
    const uint32_t c = threadIdx.x;
    const uint32_t G = c < P ? wa.grp[c] : 1u;
    const uint32_t nw = G > 1u ? (item_off[(c + 1u) * R] - item_off[c * R] + G - 1u) / G : 0u;
    uint32_t wtot;
    const uint32_t wex = block_exscan_u32(nw, s_scan, &wtot);  // P <= CR_MAX_CANDS <= blockDim.x
    if (c < P) gwave_off[c] = wex;
    if (c == 0) gwave_off[P] = wtot;
}

template <int SL>
__device__ __forceinline__ bool lru_contains(const uint32_t (&skey)[SL], uint32_t kk)
{
    uint64_t m = 0;
#pragma unroll
    for (int s = 0; s < SL; ++s) m |= ballot(skey[s] == kk);
    return m != 0;
}

// List positions in registers. Interleaved (kTwo false): position SL lane + s in register s.
// Two-level (kTwo, SL >= 2): register 0 is the front, position lane (the 64 most recent
// keys), and registers 1..SL-1 the back, position 64 + (SL-1) lane + (s-1) in register s.
template <int SL, bool kTwo>
__device__ __forceinline__ uint32_t list_pos(uint32_t s, uint32_t lane)
{
    if (kTwo) return s == 0 ? lane : 64u + (uint32_t)(SL - 1) * lane + (s - 1u);
    return (uint32_t)SL * lane + s;
}

template <int SL, bool kTwo>
__device__ __forceinline__ void lru_put_slot(uint32_t (&skey)[SL], uint32_t q, uint32_t kk, uint32_t lane)
{
    (void)lane;
    uint32_t rs, rl;  // register and lane of position q
    if (kTwo) {
        const uint32_t b = q - 64u;
        rs = q < 64u ? 0u : 1u + b % (uint32_t)(SL - 1);
        rl = q < 64u ? q : b / (uint32_t)(SL - 1);
    } else {
        rs = q % (uint32_t)SL;
        rl = q / (uint32_t)SL;
    }
#pragma unroll
    for (int s = 0; s < SL; ++s)
        if ((uint32_t)s == rs) skey[s] = wrlane(skey[s], kk, rl);
}

// Move-to-front update after a lookup whose hit mask is m: p = first set bit of m
// (0xFFFFFFFF when none); lanes 1..p (every lane on a miss) take their left neighbour's
// key and deeper lanes keep theirs, by one v_cndmask with a wave_shr:1 DPP source under
// VCC = ~1 << p. Lane 0 is left undefined for the caller to overwrite with the key. The
// scalar steps sit in the same block as the select so that no wait states are inserted
// between them; the DPP read of sk comes at least three instructions after sk's last
// VALU write (the compare that produced m, s_ff1 and s_lshl), which covers the two wait
// states such a read needs.
__device__ __forceinline__ uint32_t mtf_core(uint32_t& sk, uint64_t m)
{
    uint32_t p, out;
    asm("s_ff1_i32_b64 %1, %3\n\t"
        "s_lshl_b64 vcc, -2, %1\n\t"
        "v_cndmask_b32_dpp %0, %2, %2, vcc wave_shr:1 row_mask:0xf bank_mask:0xf"
        : "=v"(out), "=&s"(p)
        : "v"(sk), "s"(m)
        : "vcc", "scc");  // s_lshl_b64 sets SCC
    sk = out;
    return p;
}

// mtf_core with the lane mask made by the vector unit (VCC = lanes above p, one compare of
// the lane id with p) instead of s_lshl: for lists whose scalar unit is the busier one. A
// miss (p = 0xFFFFFFFF) leaves VCC empty, so every lane shifts, as in mtf_core.
__device__ __forceinline__ uint32_t mtf_core_v(uint32_t& sk, uint64_t m, uint32_t lane)
{
    uint32_t p, out;
    asm("s_ff1_i32_b64 %1, %3\n\t"
        "v_cmp_lt_u32 vcc, %1, %4\n\t"
        "v_cndmask_b32_dpp %0, %2, %2, vcc wave_shr:1 row_mask:0xf bank_mask:0xf"
        : "=v"(out), "=&s"(p)
        : "v"(sk), "s"(m), "v"(lane)
        : "vcc");
    sk = out;
    return p;
}

// Move-to-front access of key kk (lane i = i-th most recent key; lanes outside `wmask`
// are ignored). Returns the hit depth, or 0xFFFFFFFF on a miss. On a miss the shift runs
// over every lane, which drops the least recent key of a full list.
__device__ __forceinline__ uint32_t mtf_step(uint32_t& sk, uint32_t kk, uint64_t wmask)
{
    const uint32_t p = mtf_core(sk, ballot(sk == kk) & wmask);
    sk = wrlane(sk, kk, 0u);
    return p;
}

// Rebuild step over one full batch of 64 valid records (lane t = record t), newest first:
// every key not yet collected is appended at position q (SL lane + s in register s). Each
// record is branch-free: the put is a select on lane position == target, with target = q
// for a new key and no position otherwise. q is compared with W once per 8 records, so up
// to 7 keys may land past W; positions >= W are ignored everywhere (and positions past
// the registers are never written). Returns the new q.
template <int SL, bool kTwo>
__device__ __forceinline__ uint32_t rebuild_batch(uint32_t (&sk)[SL], const uint64_t* __restrict__ rb, uint32_t q,
                                                  uint32_t W, uint32_t lane)
{
    // keys by scalar loads from the batch's records (rb is uniform), 8 per load
    for (int g = 7; g >= 0 && q < W; --g) {
        uint64_t rk[8];
#pragma unroll
        for (uint32_t t = 0; t < 8; ++t) rk[t] = rb[8u * (uint32_t)g + t];
        uint32_t key[8];
#pragma unroll
        for (uint32_t t = 0; t < 8; ++t) key[t] = (uint32_t)rk[7u - t];  // newest first
        if (SL == 1 && q + 8u <= W) {
            // Positions q and up are free while the list is rebuilt, so every key is written
            // into lane q and q advances only past a new one; a repeated key left in lane q
            // duplicates an entry at a smaller position, which every later lookup finds
            // first, and the next new key overwrites it. Lanes past the final q are cleared
            // once the rebuild ends. q + 8 <= W <= 64 keeps every write inside the wave.
#pragma unroll
            for (uint32_t t = 0; t < 8; ++t) {
                const uint64_t m = ballot(sk[0] == key[t]);
                sk[0] = wrlane(sk[0], key[t], q);
                asm("s_cmp_eq_u64 %1, 0\n\ts_addc_u32 %0, %0, 0" : "+s"(q) : "s"(m) : "scc");  // q += (m == 0)
            }
            continue;
        }
#pragma unroll
        for (uint32_t t = 0; t < 8; ++t) {
            uint64_t m = 0;
#pragma unroll
            for (int s = 0; s < SL; ++s) m |= ballot(sk[s] == key[t]);
            const bool fresh = m == 0;
            const uint32_t target = fresh ? q : 0xFFFFFFFFu;
#pragma unroll
            for (int s = 0; s < SL; ++s) sk[s] = list_pos<SL, kTwo>((uint32_t)s, lane) == target ? key[t] : sk[s];
            q += fresh ? 1u : 0u;
        }
    }
    return q;
}

// Register 0 of the interleaved list after an access whose combined hit mask is m: with
// l = first set bit of m (0xFFFFFFFF when none, which shifts by 63 and keeps no lane),
// keep = ~1 << l and lanes outside keep take the last register's key from the lane before
// (one v_cndmask with a wave_shr:1 DPP source); lane 0 is left for the caller. The scalar
// steps precede the select in the same block, which gives the DPP read of `last` the two
// wait states it needs after that register's last VALU write.
__device__ __forceinline__ uint32_t il_core(uint32_t first, uint32_t last, uint64_t m, uint64_t& keep, uint32_t& l)
{
    asm("s_ff1_i32_b64 %1, %4\n\t"
        "s_lshl_b64 %2, -2, %1\n\t"
        "s_mov_b64 vcc, %2\n\t"
        "v_cndmask_b32_dpp %0, %3, %0, vcc wave_shr:1 row_mask:0xf bank_mask:0xf"
        : "+v"(first), "=&s"(l), "=&s"(keep)
        : "v"(last), "s"(m)
        : "vcc", "scc");  // s_lshl_b64 sets SCC
    return first;
}

// Move-to-front access of key kk over the interleaved list (position SL lane + s in
// register s; with kMasked, vm[s] masks the positions < W). Returns the hit position's
// lane, or 0xFFFFFFFF on a miss. With the hit in lane l of register h, positions up to the
// hit move back by one: register s > 0 takes register s-1 in lanes <= l (lanes < l when
// s > h), register 0 takes the last register of the lane before in lanes 1..l, and lane 0
// of register 0 takes the key. A miss moves every position, dropping the least recent key
// of a full list.
template <int SL, bool kMasked>
__device__ __forceinline__ uint32_t mtf_step_il(uint32_t (&sk)[SL], uint32_t kk, const uint64_t (&vm)[SL])
{
    uint64_t mh[SL];
    uint64_t m = 0;
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        mh[s] = ballot(sk[s] == kk);
        if (kMasked) mh[s] &= vm[s];
        m |= mh[s];
    }
    uint64_t keep;
    uint32_t l;
    const uint32_t r0 = il_core(sk[0], sk[SL - 1], m, keep, l);
    uint64_t before[SL];  // hit bits of registers before s
    before[0] = 0;
#pragma unroll
    for (int s = 1; s < SL; ++s) before[s] = before[s - 1] | mh[s - 1];
#pragma unroll
    for (int s = SL - 1; s >= 1; --s) sk[s] = __builtin_amdgcn_inverse_ballot_w64(keep | before[s]) ? sk[s] : sk[s - 1];
    sk[0] = wrlane(r0, kk, 0u);
    return l;
}

// 64 records (lane t of kl = key of record t, all valid) through the interleaved list;
// returns lane t = hit lane of record t (0xFFFFFFFF on a miss). Keys are read 16 at a
// time ahead of use.
template <int SL, bool kMasked>
__device__ __forceinline__ uint32_t mtf_batch_il(uint32_t (&sk)[SL], const uint64_t* __restrict__ rb,
                                                 const uint64_t (&vm)[SL])
{
    uint32_t depth = 0xFFFFFFFFu;  // keys by scalar loads, 8 records per load (rb is uniform)
#pragma unroll
    for (uint32_t g = 0; g < 8; ++g) {
        uint64_t rk[8];
#pragma unroll
        for (uint32_t t = 0; t < 8; ++t) rk[t] = rb[8u * g + t];
#pragma unroll
        for (uint32_t t = 0; t < 8; ++t)
            depth = wrlane(depth, mtf_step_il<SL, kMasked>(sk, (uint32_t)rk[t], vm), 8u * g + t);
    }
    return depth;
}

// Two-level list, back operation for an access that missed the front: kk is the accessed
// key and ins the key the front pushed out (its old position 63). If kk is in the back, the
// back positions before it move back by one; otherwise every back position does, dropping
// the least recent key of a full list. ins takes back position 0. The interleaved move-to-
// front of mtf_step_il over registers 1..SL-1, inserting ins instead of kk. Returns the hit
// mask of kk over the back (0 when kk was not there).
template <int SL, bool kMasked>
__device__ __forceinline__ uint64_t back_step(uint32_t (&sk)[SL], uint32_t kk, uint32_t ins, const uint64_t (&vm)[SL])
{
    uint64_t mh[SL];
    uint64_t m = 0;
#pragma unroll
    for (int s = 1; s < SL; ++s) {
        mh[s] = ballot(sk[s] == kk);
        if (kMasked) mh[s] &= vm[s];
        m |= mh[s];
    }
    if constexpr (SL == 2) {
        mtf_core(sk[1], m);
        sk[1] = wrlane(sk[1], ins, 0u);
    } else {
        uint64_t keep;
        uint32_t l;
        const uint32_t r1 = il_core(sk[1], sk[SL - 1], m, keep, l);
        uint64_t before[SL];  // hit bits of back registers before s
        before[1] = 0;
#pragma unroll
        for (int s = 2; s < SL; ++s) before[s] = before[s - 1] | mh[s - 1];
#pragma unroll
        for (int s = SL - 1; s >= 2; --s)
            sk[s] = __builtin_amdgcn_inverse_ballot_w64(keep | before[s]) ? sk[s] : sk[s - 1];
        sk[1] = wrlane(r1, ins, 0u);
    }
    return m;
}

// Two-level list, 64 records (all valid). Every access changes the front alone until it
// misses there, and the back changes only on those misses (its operation takes the key and
// the key the front pushed out of position 63). Each record's front access is branch-free;
// a front miss runs its back operation first, behind a branch the whole wavefront takes
// together, so nothing is logged per record. The keys come by scalar loads, 8 records
// per load, and the 8 records of a load are unrolled with one copy of the back operation
// each. Each front miss writes its lane of a vector register with whether the back held the
// key (one writelane). Returns lane t = 1 if record t hit (front or back).
template <int SL, bool kMasked>
__device__ __forceinline__ uint32_t mtf_batch_two(uint32_t (&sk)[SL], const uint64_t* __restrict__ rb,
                                                  const uint64_t (&vm)[SL], uint32_t lane)
{
    uint32_t missed = 0;  // lane t: 1 if record t was in neither part of the list
#pragma unroll 1
    for (uint32_t g = 0; g < 8; ++g) {
        uint64_t rk[8];
#pragma unroll
        for (uint32_t t = 0; t < 8; ++t) rk[t] = rb[8u * g + t];
#pragma unroll
        for (uint32_t t = 0; t < 8; ++t) {
            const uint32_t key = (uint32_t)rk[t];
            const uint64_t m = ballot(sk[0] == key);
            if (m == 0) {  // the back operation first, while front position 63 still holds the key it pushes out
                const uint64_t mb = back_step<SL, kMasked>(sk, key, rdlane(sk[0], 63u), vm);
                uint32_t miss;  // 1 when the back did not hold the key either, chosen by the scalar unit
                asm("s_cmp_eq_u64 %1, 0\n\ts_cselect_b32 %0, 1, 0" : "=s"(miss) : "s"(mb) : "scc");
                missed = wrlane(missed, miss, 8u * g + t);
            }
            mtf_core_v(sk[0], m, lane);  // with m = 0 every front position moves
            sk[0] = wrlane(sk[0], key, 0u);
        }
    }
    return missed ^ 1u;
}

// 64 records (lane t of kl = key of record t, all valid) through the move-to-front list;
// returns lane t = hit depth of record t. Keys are read 16 at a time ahead of their use.
template <bool kMasked>
__device__ __forceinline__ uint32_t mtf_batch(uint32_t& sk, const uint64_t* __restrict__ rb, uint64_t wmask)
{
    // The keys come from the batch's records (rb is uniform) by scalar loads, 8 records per
    // load: no vector instruction moves a key into a scalar register. A wavefront waits for
    // each load; the other wavefronts of its SIMD cover the wait.
    uint32_t depth = 0xFFFFFFFFu;
#pragma unroll
    for (uint32_t g = 0; g < 8; ++g) {
        uint64_t rk[8];
#pragma unroll
        for (uint32_t t = 0; t < 8; ++t) rk[t] = rb[8u * g + t];
#pragma unroll
        for (uint32_t t = 0; t < 8; ++t) {
            const uint32_t key = (uint32_t)rk[t];
            uint64_t m = ballot(sk == key);
            if (kMasked) m &= wmask;
            const uint32_t p = mtf_core(sk, m);
            sk = wrlane(sk, key, 0u);
            depth = wrlane(depth, p, 8u * g + t);
        }
    }
    return depth;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += (uint64_t)__shfl_xor((unsigned long long)v, o, 64);
    return v;
}

// One work item per segment (kSeq false), or per run of consecutive segments whose
// rebuild ran out of budget (kSeq true).
//
// A segment rebuilds its initial state by scanning back for W distinct keys; a stream with
// fewer distinct keys than W would make every segment scan to the stream's start, which is
// quadratic in its length. The scan therefore stops after kRebuildBudget segment lengths:
// a segment that has neither found W keys nor reached the start writes nothing and marks
// itself in `aborted`. In the kSeq launch that follows, the wavefront of the first segment
// of each run of marked segments starts at the run's predecessor (which is never marked:
// the first segment of a stream has nothing to rebuild), rebuilds the predecessor's state
// as that segment did, replays it without counting, and then replays the run in order,
// counting it and writing the final state if the run ends the stream. Each marked record
// is thus replayed once more, and every record is scanned at most kRebuildBudget + 1 times,
// whatever the keys. The kSeq launch rebuilds without a budget: a run's predecessor is an
// unmarked segment, whose rebuild ended within its budget. Eight segment lengths: with two,
// the whale-dominated destinations of the component ablation (8 keys at 6 % each) sent most
// of their segments to the serial kSeq pass (1.8 ms per step against 0.01 ms with eight).
constexpr uint32_t kRebuildBudget = 8;

// Budget of k_replay_grp's forward rebuild, in its own (G times shorter) segment lengths.
// Its rebuild windows run in lockstep with the other lists of the wavefront, so a deep one
// holds up G - 1 others: with eight, the 1e8-request sweep's W = 8 and 14 plans took 15.6 ms
// against 12.7 ms with two (kSeq pass included).
constexpr uint32_t kGrpRebuildBudget = 2;

__device__ __forceinline__ bool item_marked(const uint32_t* __restrict__ aborted, uint64_t it)
{
    return (aborted[it >> 5] >> (it & 31u)) & 1u;
}

// At most 96 scalar registers, so that eight wavefronts fit on a SIMD (the W = 512 list took
// 104 and seven); the one- and two-register lists spill three of theirs to vector-register
// lanes. The sweep's replay measured 117.6 -> 116.2 ms alone with the cap.
template <int SL, bool kTwo, bool kSeq>
__global__ __launch_bounds__(kReplayThreads) __attribute__((amdgpu_num_sgpr(96))) void k_replay(
    const uint64_t* __restrict__ rec, uint64_t n, const uint32_t* __restrict__ grp_off,
    const uint32_t* __restrict__ item_off, uint32_t P, uint32_t R, uint32_t K, uint32_t J,
    const uint32_t* __restrict__ prefix_len, WArg wa, CandMap cm, uint32_t max_W,
    const uint32_t* __restrict__ lru_in, uint32_t* __restrict__ lru_out, uint64_t* __restrict__ stats,
    uint32_t* __restrict__ aborted, uint32_t* __restrict__ err)
{
    const uint32_t lane = lane_id();
    const uint32_t v = blockIdx.x * (kReplayThreads / 64u) + wave_in_block();
    uint64_t item;
    uint32_t lo, hi;  // the item's stream is searched for in [lo, hi)
    if (cm.n == 0) {  // every candidate of the call: wavefront v takes work item v
        item = v;
        if (item >= item_off[P * R]) return;
        lo = 0;
        hi = P * R;
    } else {
        if (v >= cm.wv0[cm.n]) return;
        uint32_t ci = 0;  // the last i with wv0[i] <= v
        {
            uint32_t h = cm.n;
            while (h - ci > 1) {
                const uint32_t mid = (ci + h) >> 1;
                if (cm.wv0[mid] <= v) ci = mid;
                else h = mid;
            }
        }
        const uint32_t cc = cm.cand[ci];
        item = (uint64_t)item_off[cc * R] + (v - cm.wv0[ci]);
        if (item >= item_off[(cc + 1) * R]) return;
        lo = cc * R;
        hi = (cc + 1) * R;
    }
    if (kSeq && !item_marked(aborted, item)) return;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (item_off[mid] <= item) lo = mid;
        else hi = mid;
    }
    const uint32_t c = lo / R;
    // kSeq: only the first marked segment of a run, which is never a stream's first item
    if (kSeq && (item == item_off[lo] || item_marked(aborted, item - 1))) return;
    const uint32_t d = lo - c * R;
    const uint32_t W = wa.W[c];
    if (slot_class(W) != (uint32_t)SL) return;
    if (!kSeq && wa.grp[c] > 1u) return;  // k_replay_grp's segments (its marked ones come here in kSeq)
    const uint32_t* go = grp_off + (uint64_t)c * (R + 1u);
    const uint32_t gs = go[d], cnt = go[d + 1] - gs;
    const uint32_t S = seg_len(W, wa.seg_min, wa.grp[c]);
    const uint32_t nseg = item_off[lo + 1] - item_off[lo];
    // [s0, s1): the records this wavefront replays; [s0, sc) of them are replayed only to
    // reach the state at sc (the run's predecessor in the kSeq pass)
    uint64_t i0 = item, i1 = item + 1;
    if (kSeq) {
        i0 = item - 1;
        while (i1 < item_off[lo + 1] && item_marked(aborted, i1)) ++i1;
    }
    const uint32_t s0 = seg_start((uint32_t)(i0 - item_off[lo]), nseg, cnt);
    const uint32_t sc = kSeq ? seg_start((uint32_t)(item - item_off[lo]), nseg, cnt) : s0;
    const uint32_t s1 = seg_start((uint32_t)(i1 - item_off[lo]), nseg, cnt);
    const uint64_t* __restrict__ rl = rec + (uint64_t)c * n + gs;

    // Slot q of the rebuilt state is the q-th most recent key, which is already the
    // move-to-front order.
    uint32_t skey[SL];
    uint64_t vm[SL];  // lanes of register s whose position is < W
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        skey[s] = CR_EMPTY_SLOT;
        uint32_t nl;  // lanes l with list_pos(s, l) < W
        if (kTwo && s == 0) nl = W < 64u ? W : 64u;
        else if (kTwo) nl = W > 63u + (uint32_t)s ? (W - 63u - (uint32_t)s + SL - 2u) / (uint32_t)(SL - 1) : 0u;
        else nl = W > (uint32_t)s ? (W - (uint32_t)s + SL - 1u) / (uint32_t)SL : 0u;
        vm[s] = nl >= 64u ? ~0ull : (1ull << nl) - 1ull;
    }
    const uint64_t wmask = vm[0];
    uint32_t q = 0;
    {
        // State before record s0: the most recent W distinct keys, newest first. Records
        // are read backwards 64 at a time, the next (older) batch in flight while one is
        // scanned. (A kSeq wavefront rebuilds an unmarked segment, which stays in budget.)
        uint32_t pos = s0, scanned = 0;
        const uint32_t budget = kRebuildBudget * S;
        uint32_t nb = pos < 64u ? pos : 64u;
        uint32_t kl_next = lane < nb ? (uint32_t)rl[pos - nb + lane] : CR_EMPTY_SLOT;
        while (q < W && pos > 0) {
            if (!kSeq && scanned >= budget) {  // too few distinct keys: left to the kSeq pass
                if (lane == 0) atomicOr(&aborted[item >> 5], 1u << (item & 31u));
                return;
            }
            const uint32_t kl = kl_next;
            const uint32_t cnb = nb;
            pos -= cnb;
            scanned += cnb;
            nb = pos < 64u ? pos : 64u;
            kl_next = lane < nb ? (uint32_t)rl[pos - nb + lane] : CR_EMPTY_SLOT;
            if (cnb == 64u && ballot(kl < K) == ~0ull) {
                q = rebuild_batch<SL, kTwo>(skey, rl + pos, q, W, lane);
                continue;
            }
            for (int t = (int)cnb - 1; t >= 0 && q < W; --t) {
                const uint32_t kk = rdlane(kl, (uint32_t)t);
                if (kk >= K) continue;
                if (!lru_contains<SL>(skey, kk)) {
                    lru_put_slot<SL, kTwo>(skey, q, kk, lane);
                    ++q;
                }
            }
        }
    }
    if (q < W && lru_in) {
        const uint32_t* __restrict__ li = lru_in + ((uint64_t)c * R + d) * max_W;
        bool done = false;
        for (uint32_t s = 0; s < W && q < W && !done; s += 64) {
            const uint32_t nb = W - s < 64u ? W - s : 64u;
            const uint32_t v = lane < nb ? li[s + lane] : CR_EMPTY_SLOT;
            for (uint32_t t = 0; t < nb && q < W; ++t) {
                const uint32_t kk = rdlane(v, t);
                if (kk == CR_EMPTY_SLOT) {
                    done = true;
                    break;
                }
                if (kk >= K) continue;
                if (!lru_contains<SL>(skey, kk)) {
                    lru_put_slot<SL, kTwo>(skey, q, kk, lane);
                    ++q;
                }
            }
        }
    }

    if constexpr (SL == 1) {
        if (q < W) skey[0] = lane >= q ? CR_EMPTY_SLOT : skey[0];  // drop what the rebuild left past q
    }

    // Per-lane sums for the current interval; flushed (one atomic per statistic) when the
    // interval changes and at the end of a range.
    uint64_t a_req = 0, a_hit = 0, a_pre = 0, a_hp = 0;
    uint32_t cur = 0xFFFFFFFFu;
    bool bad = false;
    auto flush = [&]() {
        if (cur >= J) return;
        const uint64_t r0 = wave_sum_u64(a_req), r1 = wave_sum_u64(a_hit), r2 = wave_sum_u64(a_pre),
                       r3 = wave_sum_u64(a_hp);
        if (lane == 0) {
            unsigned long long* st = (unsigned long long*)(stats + (((uint64_t)cur * P + c) * R + d) * 4u);
            atomicAdd(st + 0, (unsigned long long)r0);
            if (r1) atomicAdd(st + 1, (unsigned long long)r1);
            atomicAdd(st + 2, (unsigned long long)r2);
            if (r3) atomicAdd(st + 3, (unsigned long long)r3);
        }
        a_req = a_hit = a_pre = a_hp = 0;
    };
    // Forward replay of records [r0, r1); the next batch of records is in flight while one
    // is replayed. With `on` false the list advances but nothing is counted.
    auto run = [&](uint32_t r0, uint32_t r1, bool on) {
        uint64_t rv_next = r0 + lane < r1 ? rl[r0 + lane] : 0ull;
        for (uint32_t b0 = r0; b0 < r1; b0 += 64) {
            const uint32_t nb = r1 - b0 < 64u ? r1 - b0 : 64u;
            const uint64_t rv = rv_next;
            rv_next = b0 + 64u + lane < r1 ? rl[b0 + 64u + lane] : 0ull;
            const uint32_t kl = lane < nb ? (uint32_t)rv : CR_EMPTY_SLOT;
            const bool vl = lane < nb && kl < K;
            bad |= lane < nb && kl >= K;
            const uint32_t pl = vl && on ? prefix_len[kl] : 0u;  // consumed after the batch
            bool hl;
            if constexpr (SL == 1) {
                uint32_t depth = 0xFFFFFFFFu;  // lane t: hit depth of record t
                if (ballot(vl) == ~0ull) {
                    depth = W == 64u ? mtf_batch<false>(skey[0], rl + b0, wmask)
                                     : mtf_batch<true>(skey[0], rl + b0, wmask);
                } else {
                    for (uint32_t t = 0; t < nb; ++t) {
                        const uint32_t kk = rdlane(kl, t);
                        if (kk < K) depth = wrlane(depth, mtf_step(skey[0], kk, wmask), t);
                    }
                }
                hl = depth != 0xFFFFFFFFu;
            } else if constexpr (kTwo) {
                uint32_t hit = 0;  // lane t: 1 if record t hit
                if (ballot(vl) == ~0ull) {
                    hit = W == 64u * SL ? mtf_batch_two<SL, false>(skey, rl + b0, vm, lane)
                                        : mtf_batch_two<SL, true>(skey, rl + b0, vm, lane);
                } else {
                    for (uint32_t t = 0; t < nb; ++t) {
                        const uint32_t kk = rdlane(kl, t);
                        if (kk >= K) continue;
                        const uint64_t m = ballot(skey[0] == kk);
                        const uint32_t ev = rdlane(skey[0], 63u);
                        mtf_core(skey[0], m);
                        skey[0] = wrlane(skey[0], kk, 0u);
                        if (m || back_step<SL, true>(skey, kk, ev, vm) != 0) hit = wrlane(hit, 1u, t);
                    }
                }
                hl = hit != 0u;
            } else {
                uint32_t depth = 0xFFFFFFFFu;  // lane t: hit lane of record t
                if (ballot(vl) == ~0ull) {
                    depth = W == 64u * SL ? mtf_batch_il<SL, false>(skey, rl + b0, vm)
                                          : mtf_batch_il<SL, true>(skey, rl + b0, vm);
                } else {
                    for (uint32_t t = 0; t < nb; ++t) {
                        const uint32_t kk = rdlane(kl, t);
                        if (kk < K) depth = wrlane(depth, mtf_step_il<SL, true>(skey, kk, vm), t);
                    }
                }
                hl = depth != 0xFFFFFFFFu;
            }
            if (!on) continue;
            const uint32_t sfx = (uint32_t)(rv >> 32) & 0xFFFFu;
            const uint32_t ivl = (uint32_t)(rv >> 48);
            uint64_t rem = ballot(vl);
            while (rem) {
                const uint32_t iv = rdlane(ivl, first_lane(rem));
                if (iv != cur) {
                    flush();
                    cur = iv;
                }
                const uint64_t sel = rem & ballot(ivl == iv);
                if ((sel >> lane) & 1ull) {
                    a_req += 1;
                    a_hit += hl ? 1u : 0u;
                    a_pre += sfx + (hl ? 0u : pl);
                    a_hp += hl ? pl : 0u;
                }
                rem &= ~sel;
            }
        }
        flush();
    };
    if (sc > s0) run(s0, sc < s1 ? sc : s1, false);
    run(sc, s1, true);
    if (ballot(bad) && lane == 0) atomicOr(err, CR_ERR_KEY_RANGE);
    if (s1 == cnt) {
        uint32_t* __restrict__ lo_ = lru_out + ((uint64_t)c * R + d) * max_W;
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            const uint32_t idx = list_pos<SL, kTwo>((uint32_t)s, lane);
            if (idx < W) lo_[idx] = skey[s];
        }
        for (uint32_t idx = W + lane; idx < max_W; idx += 64) lo_[idx] = CR_EMPTY_SLOT;
    }
}

// ---------------------------------------------------------------------------------------
// Small lists, several segments per wavefront (calls with one interval). A list of
// W <= 64 / G slots needs W lanes, so a wavefront keeps G lists side by side in lane groups
// of w = 64 / G lanes (group g: lanes g w .. g w + w - 1, position j in lane g w + j), each
// replaying its own segment, and one instruction advances all G of them. Per step, group g
// reads its record's key from LDS into all of its lanes; one compare gives the hit mask m
// (at most one lane per group). With END the lanes of position W - 1 and START those of
// position 0, M = m | END has a set bit in every group and its lowest one at or above the
// group's START is the hit (or position W - 1 on a miss), so the borrow of M - START runs
// exactly over positions 0 .. hit of each group: M ^ (M - START) is the set of lanes that
// move back by one, in every group at once. The move is one select with a wave_shr:1 DPP
// source, and the key goes into each group's position 0 by a second select. Groups without
// a record at a step (segment ended, key out of range) read a marker key that matches no
// slot and are masked out of both selects.
//
// The state before a segment is rebuilt forward: the D records before it are replayed from
// an empty list (from the carried state where the window reaches the stream start). When
// the window holds W distinct keys the list is exactly the W most recent ones, so it is full
// when it is right; otherwise D grows, up to kGrpRebuildBudget S rounded up to whole
// 64-record batches. A segment whose window still holds fewer than W distinct keys there is
// marked in `aborted`, and the kSeq pass of k_replay<1> replays it from its predecessor.
//
// Statistics: a step's hit is the bit of the lane that held its key; each lane shifts its
// bits into a register, and after a round of 64 steps the group's registers, OR-ed, give the
// round's hits. Every lane then adds the count, suffix + prefix lengths and the prefix
// lengths of the hits over the records it staged; the group's lanes are summed at the end.
constexpr uint32_t kGrpSent = 0xFFFFFFFEu;  // staged key of a skipped step: never a key (K <= 0xFFFFFFFE), never empty

// Positions 0 .. hit of every group move back by one: lanes with `keep` set hold their key,
// the others take their left neighbour's (a wave_shr:1 DPP source). The destination is the
// source, so lane 0, which has no left neighbour, keeps its key.
__device__ __forceinline__ void grp_move(uint32_t& sk, uint64_t movebits, uint64_t act)
{
    asm("s_nand_b64 vcc, %1, %2\n\t"
        "v_cndmask_b32_dpp %0, %0, %0, vcc wave_shr:1 row_mask:0xf bank_mask:0xf"
        : "+v"(sk)
        : "s"(movebits), "s"(act)
        : "vcc");
}

// h = 2 h + (this lane's bit of m): one add with carry-in
__device__ __forceinline__ void shift_in_lane_bit(uint32_t& h, uint64_t m)
{
    uint64_t dummy;
    asm("v_addc_co_u32 %0, %1, %0, %0, %2" : "+v"(h), "=s"(dummy) : "s"(m));
}

template <int G>
__global__ __launch_bounds__(kReplayThreads) void k_replay_grp(
    const uint64_t* __restrict__ rec, uint64_t n, const uint32_t* __restrict__ grp_off,
    const uint32_t* __restrict__ item_off, const uint32_t* __restrict__ gwave_off, uint32_t P, uint32_t R, uint32_t K,
    const uint32_t* __restrict__ prefix_len, WArg wa, uint32_t max_W, const uint32_t* __restrict__ lru_in,
    uint32_t* __restrict__ lru_out, uint64_t* __restrict__ stats, uint32_t* __restrict__ aborted,
    uint32_t* __restrict__ err)
{
    constexpr uint32_t w = 64u / G;
    constexpr uint32_t kStride = 65u;  // keys per group in the stage (padded: groups on other banks)
    __shared__ uint32_t s_stage[kReplayThreads / 64][G * kStride];
    const uint32_t lane = lane_id(), wv = wave_in_block();
    const uint32_t g = lane / w, j = lane % w;
    const uint32_t wid = blockIdx.x * (kReplayThreads / 64u) + wv;
    if (wid >= gwave_off[P]) return;
    uint32_t c = 0;  // the candidate: the last c with gwave_off[c] <= wid
    {
        uint32_t hi = P;
        while (hi - c > 1) {
            const uint32_t mid = (c + hi) >> 1;
            if (gwave_off[mid] <= wid) c = mid;
            else hi = mid;
        }
    }
    if (wa.grp[c] != (uint32_t)G) return;
    const uint32_t W = wa.W[c];
    const uint64_t it1 = item_off[(uint64_t)(c + 1) * R];
    const uint64_t item = item_off[(uint64_t)c * R] + (uint64_t)G * (wid - gwave_off[c]) + g;
    bool live = item < it1;
    uint32_t lo = c * R;  // the item's stream
    if (live) {
        uint32_t hi = (c + 1) * R;
        while (hi - lo > 1) {
            const uint32_t mid = (lo + hi) >> 1;
            if (item_off[mid] <= item) lo = mid;
            else hi = mid;
        }
    }
    const uint32_t d = lo - c * R;
    const uint32_t S = seg_len(W, wa.seg_min, G);
    const uint32_t* go = grp_off + (uint64_t)c * (R + 1u);
    const uint32_t gs = live ? go[d] : 0u, cnt = live ? go[d + 1] - gs : 0u;
    const uint32_t nseg = live ? item_off[lo + 1] - item_off[lo] : 1u;
    const uint32_t s0 = live ? seg_start((uint32_t)(item - item_off[lo]), nseg, cnt) : 0u;
    const uint32_t s1 = live ? seg_start((uint32_t)(item - item_off[lo]) + 1u, nseg, cnt) : 0u;
    const uint64_t* __restrict__ rl = rec + (uint64_t)c * n + gs;
    uint32_t* __restrict__ stage = s_stage[wv] + g * kStride;

    uint64_t START = 0, END = 0;
#pragma unroll
    for (uint32_t q = 0; q < G; ++q) {
        START |= 1ull << (q * w);
        END |= 1ull << (q * w + W - 1u);
    }
    uint32_t sk = CR_EMPTY_SLOT;
    bool bad = false;
    uint32_t a_hit = 0, a_req = 0;
    uint64_t a_hp = 0, a_all = 0;

    // One step of every group: key kv (kGrpSent: none). With hb, each lane shifts its hit
    // bit of the step into hb (hb = 2 hb + hit: after 32 steps, step t is bit 31 - t).
    auto step = [&](uint32_t kv, uint32_t* hb) {
        const uint64_t m = ballot(sk == kv);
        const uint64_t act = ballot(kv != kGrpSent);
        const uint64_t M = m | END;
        grp_move(sk, M ^ (M - START), act);
        sk = __builtin_amdgcn_inverse_ballot_w64(START & act) ? kv : sk;
        if (hb) shift_in_lane_bit(*hb, m);
    };
    // Records [a, a + len) of each group's stream through its list, in rounds of 64 steps:
    // lane j of a group stages the keys of steps j, j + w, ... of its group in LDS. The next
    // round's records are loaded while a round runs. With statistics, the prefix lengths of
    // a round's records are gathered as it starts and used once it has run: every round is
    // 64 steps (idle ones at the end of a group's range), and the hit bits of the group's
    // lanes, OR-ed together, say which of its steps hit.
    auto run = [&](uint32_t a, uint32_t len, bool with_stats) {
        uint32_t most = len;
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            const uint32_t x = __shfl_xor(most, o, 64);
            most = x > most ? x : most;
        }
        most = __builtin_amdgcn_readfirstlane(most);
        uint64_t rv[G];
#pragma unroll
        for (uint32_t i = 0; i < G; ++i) {
            const uint32_t t = j + w * i;
            rv[i] = t < len ? rl[a + t] : 0ull;
        }
        for (uint32_t t0 = 0; t0 < most; t0 += 64u) {
            uint32_t key[G], sfx[G];
            bool ok[G];
#pragma unroll
            for (uint32_t i = 0; i < G; ++i) {
                const uint32_t t = t0 + j + w * i;
                key[i] = (uint32_t)rv[i];
                sfx[i] = (uint32_t)(rv[i] >> 32) & 0xFFFFu;
                ok[i] = t < len && key[i] < K;
                bad |= t < len && key[i] >= K;
                stage[j + w * i] = ok[i] ? key[i] : kGrpSent;
            }
            uint32_t pl[G];
            if (with_stats) {
#pragma unroll
                for (uint32_t i = 0; i < G; ++i) pl[i] = prefix_len[ok[i] ? key[i] : 0u];
            }
#pragma unroll
            for (uint32_t i = 0; i < G; ++i) {  // the next round's records
                const uint32_t t = t0 + 64u + j + w * i;
                rv[i] = t < len ? rl[a + t] : 0ull;
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            if (with_stats) {
                uint32_t h0 = 0, h1 = 0;
#pragma unroll
                for (uint32_t t = 0; t < 32u; ++t) step(stage[t], &h0);
#pragma unroll
                for (uint32_t t = 32; t < 64u; ++t) step(stage[t], &h1);
#pragma unroll
                for (uint32_t o = w / 2; o >= 1; o >>= 1) {
                    h0 |= __shfl_xor(h0, o, 64);
                    h1 |= __shfl_xor(h1, o, 64);
                }
                if (j == 0) a_hit += __builtin_popcount(h0) + __builtin_popcount(h1);
#pragma unroll
                for (uint32_t i = 0; i < G; ++i) {
                    const uint32_t t = j + w * i;
                    const bool hit = ((t < 32u ? h0 >> (31u - t) : h1 >> (63u - t)) & 1u) != 0u;
                    a_req += ok[i] ? 1u : 0u;
                    a_all += ok[i] ? (uint64_t)sfx[i] + pl[i] : 0ull;
                    a_hp += ok[i] && hit ? (uint64_t)pl[i] : 0ull;
                }
            } else {
                const uint32_t nt = most - t0 < 64u ? most - t0 : 64u;
                if (nt == 64u) {
#pragma unroll 16
                    for (uint32_t t = 0; t < 64u; ++t) step(stage[t], nullptr);
                } else {
                    for (uint32_t t = 0; t < nt; ++t) step(stage[t], nullptr);
                }
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        }
    };
    // The carried state of the groups in `on`, oldest entry first, through their lists: the
    // entries before the row's first empty slot, keys >= K skipped, as the backward rebuild
    // appends them.
    auto carried = [&](bool on) {
        const uint32_t* __restrict__ li = lru_in + ((uint64_t)c * R + d) * max_W;
        const uint32_t v = on && j < W ? li[j] : CR_EMPTY_SLOT;
        uint32_t fe = W;  // the row's first empty slot
        for (uint32_t i = 0; i < W; ++i) {
            const uint32_t x = __shfl(v, g * w + i, 64);
            fe = x == CR_EMPTY_SLOT && fe == W ? i : fe;
        }
        for (uint32_t i = W; i-- > 0;) {
            const uint32_t x = __shfl(v, g * w + i, 64);
            step(on && i < fe && x < K ? x : kGrpSent, nullptr);
        }
    };

    // rebuild the state at s0
    const uint32_t budget = (kGrpRebuildBudget * S + 63u) & ~63u;
    const uint32_t dmax = s0 < budget ? s0 : budget;
    bool ready = !live || s0 == 0;
    if (lru_in && ballot(live && s0 == 0)) carried(live && s0 == 0);
    for (uint32_t D = 4u * W; ballot(!ready) != 0; D *= 8u) {
        const bool part = !ready;
        const uint32_t dg = D < dmax ? D : dmax;
        sk = part ? CR_EMPTY_SLOT : sk;
        if (lru_in && ballot(part && dg == s0)) carried(part && dg == s0);
        run(s0 - dg, part ? dg : 0u, false);
        const uint64_t F = ballot(j == W - 1u && sk != CR_EMPTY_SLOT);
        const bool full = (F >> (g * w + W - 1u)) & 1ull;
        const bool ok = part && (full || dg == s0);
        if (part && !ok && dg == dmax) {  // too few distinct keys in reach: left to the kSeq pass
            if (j == 0) atomicOr(&aborted[item >> 5], 1u << (item & 31u));
            live = false;
        }
        ready = ready || ok || (part && dg == dmax);
    }
    run(s0, live ? s1 - s0 : 0u, true);
    if (ballot(bad) && lane == 0) atomicOr(err, CR_ERR_KEY_RANGE);
    // the group's sums in its lane 0
#pragma unroll
    for (uint32_t o = w / 2; o >= 1; o >>= 1) {
        a_hit += __shfl_xor(a_hit, o, 64);
        a_req += __shfl_xor(a_req, o, 64);
        a_hp += (uint64_t)__shfl_xor((unsigned long long)a_hp, o, 64);
        a_all += (uint64_t)__shfl_xor((unsigned long long)a_all, o, 64);
    }
    if (live && j == 0) {
        unsigned long long* st = (unsigned long long*)(stats + ((uint64_t)c * R + d) * 4u);  // interval 0
        atomicAdd(st + 0, (unsigned long long)a_req);
        if (a_hit) atomicAdd(st + 1, (unsigned long long)a_hit);
        atomicAdd(st + 2, (unsigned long long)(a_all - a_hp));
        if (a_hp) atomicAdd(st + 3, (unsigned long long)a_hp);
    }
    if (live && s1 == cnt) {
        uint32_t* __restrict__ lo_ = lru_out + ((uint64_t)c * R + d) * max_W;
        if (j < W) lo_[j] = sk;
        for (uint32_t idx = W + j; idx < max_W; idx += w) lo_[idx] = CR_EMPTY_SLOT;
    }
}

__global__ void k_zero_u32(uint32_t* __restrict__ p, uint64_t n)
{
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = 0u;
}

struct ReplayWs {
    uint64_t* rec;
    uint32_t* tcnt;
    uint32_t* dtot;
    uint32_t* grp_off;
    uint32_t* item_off;
    uint32_t* gwave_off;  // [P + 1] first k_replay_grp wavefront of each candidate
    uint32_t* aborted;  // bit per work item: its rebuild ran out of budget
    uint64_t flag_words;
    size_t bytes;
};

// Upper bound on replay work items: one per (c, d) plus one per full shortest segment.
inline uint64_t max_items(uint64_t n, uint32_t P, uint32_t R) { return (uint64_t)P * R + (uint64_t)P * n / kSegFloor + 1u; }

inline ReplayWs replay_layout(void* base, uint64_t n, uint32_t P, uint32_t R)
{
    const PartGeom g = part_geom(n, P);
    auto up = [](uint64_t x) { return (x + 255) & ~255ull; };
    uint8_t* b = reinterpret_cast<uint8_t*>(base);
    uint64_t o = 0;
    ReplayWs w{};
    w.rec = reinterpret_cast<uint64_t*>(b + o);
    o = up(o + (uint64_t)P * n * 8u);
    w.tcnt = reinterpret_cast<uint32_t*>(b + o);
    o = up(o + (uint64_t)P * R * g.ntiles * 4u);
    w.dtot = reinterpret_cast<uint32_t*>(b + o);
    o = up(o + (uint64_t)P * R * 4u);
    w.grp_off = reinterpret_cast<uint32_t*>(b + o);
    o = up(o + (uint64_t)P * (R + 1u) * 4u);
    w.item_off = reinterpret_cast<uint32_t*>(b + o);
    o = up(o + ((uint64_t)P * R + 1u) * 4u);
    w.gwave_off = reinterpret_cast<uint32_t*>(b + o);
    o = up(o + ((uint64_t)P + 1u) * 4u);
    w.aborted = reinterpret_cast<uint32_t*>(b + o);
    w.flag_words = (max_items(n, P, R) + 31u) / 32u;
    o = up(o + w.flag_words * 4u);
    w.bytes = (size_t)o + 256u;
    return w;
}

struct ReplayArgs {
    WArg wa;
    uint32_t classes;    // bit SL - 1: some candidate's list has SL registers
    uint32_t wclasses;   // the same, candidates replayed one list per wavefront only
    uint32_t groups;     // bit G: some candidate is replayed by k_replay_grp<G>
    uint64_t grp_waves;  // bound on k_replay_grp wavefronts
};

// Records (n times the number of candidates with W <= 16) from which a one-interval call
// replays those candidates by k_replay_grp; below it there are too few segments to fill the
// chip with a G-th of the wavefronts.
uint64_t g_grp_min_records = 1ull << 25;

inline cr_status replay_args(uint64_t n, uint32_t J, uint32_t P, uint32_t R, const uint32_t* W, uint32_t max_W,
                             size_t ws_bytes, void* ws, ReplayArgs* ra)
{
    if (P == 0 || P > CR_MAX_CANDS || R == 0 || R > CR_MAX_R || J == 0 || J > CR_MAX_J || !W || max_W == 0 ||
        max_W > CR_MAX_W || !ws || n >= 0xFFFFFFFFull)
        return CR_EINVAL;
    ra->wa = WArg{};
    ra->wa.seg_min = (uint32_t)(((uint64_t)n * P + kSegTarget - 1) / kSegTarget);
    ra->classes = 0;
    ra->wclasses = 0;
    ra->groups = 0;
    ra->grp_waves = 0;
    uint64_t small = 0;  // candidates k_replay_grp could take
    for (uint32_t c = 0; c < P; ++c) small += grp_of(W[c], J) > 1u ? 1u : 0u;
    const bool grouped = small > 0 && n * small >= g_grp_min_records;
    for (uint32_t c = 0; c < P; ++c) {
        if (W[c] == 0 || W[c] > max_W) return CR_EINVAL;
        ra->wa.W[c] = (uint16_t)W[c];
        const uint32_t G = grouped ? grp_of(W[c], J) : 1u;
        ra->wa.grp[c] = (uint8_t)G;
        ra->classes |= 1u << (slot_class(W[c]) - 1u);
        if (G == 1u) ra->wclasses |= 1u << (slot_class(W[c]) - 1u);
        const uint32_t S = seg_len(W[c], ra->wa.seg_min, G);
        if (G > 1u) {  // at most R + n / S work items, G per wavefront
            ra->groups |= 1u << G;
            ra->grp_waves += ((uint64_t)R + n / S) / G + 1u;
        }
    }
    if (ws_bytes < replay_layout(nullptr, n, P, R).bytes) return CR_ESIZE;
    return CR_OK;
}

inline void* ws_base(void* ws) { return reinterpret_cast<void*>(((uintptr_t)ws + 255) & ~(uintptr_t)255); }

}  // namespace
}  // namespace cr

extern "C" void cr_replay_set_group_min_records(uint64_t min_records) { cr::g_grp_min_records = min_records; }

extern "C" size_t cr_replay_workspace_bytes(uint64_t n, uint32_t P, uint32_t R)
{
    return cr::replay_layout(nullptr, n, P, R).bytes;
}

extern "C" size_t cr_workspace_bytes(uint32_t num_keys, uint32_t R, uint32_t P, uint64_t max_n)
{
    const size_t a = cr_count_slice_workspace_bytes(max_n, num_keys), b = cr_replay_workspace_bytes(max_n, P, R);
    return a > b ? a : b;
}

extern "C" size_t cr_lru_state_bytes(uint32_t P, uint32_t R, uint32_t max_W)
{
    return (size_t)P * R * max_W * sizeof(uint32_t);
}

namespace cr {
namespace {
__global__ void k_lru_fill(uint32_t* __restrict__ p, uint64_t n)
{
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = CR_EMPTY_SLOT;
}
}  // namespace
}  // namespace cr

extern "C" cr_status cr_lru_reset(uint32_t* lru_state, uint32_t P, uint32_t R, uint32_t max_W, void* stream)
{
    using namespace cr;
    if (!lru_state || P == 0 || P > CR_MAX_CANDS || R == 0 || R > CR_MAX_R || max_W == 0 || max_W > CR_MAX_W)
        return CR_EINVAL;
    const uint64_t n = (uint64_t)P * R * max_W;
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_lru_fill, dim3((uint32_t)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096)), dim3(256), 0,
                       as_stream(stream), lru_state, n);
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}

extern "C" cr_status cr_replay_partition(const uint32_t* keys, const uint16_t* suffix, const uint16_t* dest,
                                         uint64_t n, const uint64_t* off, uint32_t J, uint32_t P, uint32_t R,
                                         const uint32_t* W, void* ws, size_t ws_bytes, uint32_t* err, void* stream)
{
    using namespace cr;
    ReplayArgs ra;
    uint32_t mw = 0;
    for (uint32_t c = 0; W && c < P && c < CR_MAX_CANDS; ++c) mw = W[c] > mw ? W[c] : mw;
    const cr_status v = replay_args(n, J, P, R, W, mw ? mw : 1u, ws_bytes, ws, &ra);
    if (v != CR_OK) return v;
    if (!off || !err || (n > 0 && (!keys || !suffix || !dest))) return CR_EINVAL;
    const ReplayWs w = replay_layout(ws_base(ws), n, P, R);
    const PartGeom g = part_geom(n, P);
    const hipStream_t st = as_stream(stream);
    uint32_t nbits = 0;
    while ((1u << nbits) < R) ++nbits;
    (void)hipGetLastError();
    // 16-byte loads of keys, destinations and suffixes need 16-byte aligned rows
    const bool vec = ((uintptr_t)keys & 15u) == 0 && ((uintptr_t)suffix & 15u) == 0 && ((uintptr_t)dest & 15u) == 0 &&
                     (n & 7u) == 0;
    if (g.ntiles && vec)
        hipLaunchKernelGGL(k_part_hist<true>, dim3((uint32_t)g.ntiles, P), dim3(kHistThreads), (size_t)R * 4u, st, dest,
                           n, R, g.tile, g.ntiles, w.tcnt, err);
    else if (g.ntiles)
        hipLaunchKernelGGL(k_part_hist<false>, dim3((uint32_t)g.ntiles, P), dim3(kHistThreads), (size_t)R * 4u, st, dest,
                           n, R, g.tile, g.ntiles, w.tcnt, err);
    hipLaunchKernelGGL(k_scan_dest, dim3(R, P), dim3(kScanThreads), 0, st, w.tcnt, g.ntiles, R, w.dtot);
    hipLaunchKernelGGL(k_seg_items, dim3(1), dim3(1024), 0, st, w.dtot, P, R, ra.wa, w.grp_off, w.item_off,
                       w.gwave_off);
    if (g.ntiles && R <= 64 && vec)
        hipLaunchKernelGGL(k_part_scatter64<true>, dim3(xcd_grid((uint32_t)g.ntiles), P), dim3(64),
                           scatter64_lds_bytes(R), st, keys, suffix, dest, n, off, J, R, g.tile, g.ntiles, w.tcnt,
                           w.grp_off, w.rec);
    else if (g.ntiles && R <= 64)
        hipLaunchKernelGGL(k_part_scatter64<false>, dim3(xcd_grid((uint32_t)g.ntiles), P), dim3(64),
                           scatter64_lds_bytes(R), st, keys, suffix, dest, n, off, J, R, g.tile, g.ntiles, w.tcnt,
                           w.grp_off, w.rec);
    else if (g.ntiles && g.ntiles <= 65535u) {
        const size_t lds = scatter_wide_lds_bytes(R);
        if (hipFuncSetAttribute((const void*)k_part_scatter_wide, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)lds) != hipSuccess)
            return CR_EHIP;
        hipLaunchKernelGGL(k_part_scatter_wide, dim3(P * xcd_grid((uint32_t)g.ntiles)), dim3(kWideThreads), lds, st,
                           keys, suffix, dest, n, off, J, P, R, nbits, g.tile, g.ntiles, w.tcnt, w.grp_off, w.rec);
    } else if (g.ntiles)
        hipLaunchKernelGGL(k_part_scatter, dim3(xcd_grid((uint32_t)g.ntiles), P), dim3(64), scatter_lds_bytes(R), st, keys,
                           suffix, dest, n, off, J, R, nbits, g.tile, g.ntiles, w.tcnt, w.grp_off, w.rec);
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}

namespace cr {
namespace {
// Two side streams per device (default priority) for the list-size launches of a replay
// call, created on a device's first call and kept until the process ends. A launch runs as
// many wavefronts as its segments, and near its end the chip empties while its last
// segments finish; on two streams one list size's launch fills the room another's leaves.
// The calls that share them are serialised by a host mutex (fork, launches and join).
#ifndef CR_REPLAY_SIDE_STREAMS
#define CR_REPLAY_SIDE_STREAMS 1
#endif
constexpr int kSideDevices = 64;
struct SideStreams {
    bool ready = false, failed = false;
    hipStream_t s[2] = {nullptr, nullptr};
    hipEvent_t fork = nullptr, join[2] = {nullptr, nullptr};
};
std::mutex g_side_mu;
SideStreams g_side[kSideDevices];

// The current device's side streams (caller holds g_side_mu), or nullptr: then the launches
// stay on the caller's stream. A device whose streams or events could not all be created
// releases what was made and is not tried again.
SideStreams* side_streams()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kSideDevices) return nullptr;
    SideStreams& q = g_side[dev];
    if (!q.ready && !q.failed) {
        bool ok = hipEventCreateWithFlags(&q.fork, hipEventDisableTiming) == hipSuccess;
        for (int i = 0; i < 2 && ok; ++i)
            ok = hipStreamCreateWithFlags(&q.s[i], hipStreamNonBlocking) == hipSuccess &&
                 hipEventCreateWithFlags(&q.join[i], hipEventDisableTiming) == hipSuccess;
        if (!ok) {
            for (int i = 0; i < 2; ++i) {
                if (q.join[i]) (void)hipEventDestroy(q.join[i]);
                if (q.s[i]) (void)hipStreamDestroy(q.s[i]);
                q.join[i] = nullptr;
                q.s[i] = nullptr;
            }
            if (q.fork) (void)hipEventDestroy(q.fork);
            q.fork = nullptr;
            (void)hipGetLastError();
            q.failed = true;
        }
        q.ready = ok;
    }
    return q.ready ? &q : nullptr;
}
}  // namespace
}  // namespace cr

extern "C" cr_status cr_replay_lru(const uint32_t* prefix_len, uint32_t num_keys, uint64_t n, uint32_t J,
                                   uint32_t P, uint32_t R, const uint32_t* W, uint32_t max_W, const uint32_t* lru_in,
                                   uint32_t* lru_out, uint64_t* stats, void* ws, size_t ws_bytes, uint32_t* err,
                                   void* stream)
{
    using namespace cr;
    ReplayArgs ra;
    const cr_status v = replay_args(n, J, P, R, W, max_W, ws_bytes, ws, &ra);
    if (v != CR_OK) return v;
    if (num_keys == 0 || num_keys == 0xFFFFFFFFu || !prefix_len || !lru_out || !stats || !err) return CR_EINVAL;
    if (lru_in && lru_in < lru_out + (uint64_t)P * R * max_W && lru_out < lru_in + (uint64_t)P * R * max_W)
        return CR_EINVAL;
    const ReplayWs w = replay_layout(ws_base(ws), n, P, R);
    const hipStream_t st = as_stream(stream);
    const uint64_t gblocks = (ra.grp_waves + (kReplayThreads / 64) - 1) / (kReplayThreads / 64);
    if (gblocks > 0x7FFFFFFFull) return CR_EINVAL;
    // One k_replay launch per list size, with wavefronts for its own candidates only: a
    // stream of cnt records has max(1, ceil(cnt / S)) work items, so a candidate has at most
    // R + n / S of them.
    CandMap cm;
    auto cand_map = [&](uint32_t SL, bool seq) -> uint64_t {
        uint64_t wv = 0;
        cm.n = 0;
        for (uint32_t c = 0; c < P; ++c) {
            if (slot_class(W[c]) != SL || (!seq && ra.wa.grp[c] > 1u)) continue;
            cm.cand[cm.n] = (uint16_t)c;
            cm.wv0[cm.n++] = (uint32_t)wv;
            wv += (uint64_t)R + n / seg_len(W[c], ra.wa.seg_min, ra.wa.grp[c]) + 1u;
        }
        cm.wv0[cm.n] = (uint32_t)wv;
        if (cm.n == P) cm.n = 0;  // every candidate, in order: work item v is wavefront v
        return wv;
    };
    for (uint32_t SL = 1; SL <= 8; ++SL)
        if (cand_map(SL, true) > 0x7FFFFFFFull) return CR_EINVAL;
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_zero_u32, dim3(256), dim3(256), 0, st, w.aborted, w.flag_words);
#define CR_REPLAY(SL, TWO, SEQ, NB)                                                                                 \
    hipLaunchKernelGGL((k_replay<SL, TWO, SEQ>), dim3((uint32_t)(NB)), dim3(kReplayThreads), 0, st, w.rec, n,        \
                       w.grp_off, w.item_off, P, R, num_keys, J, prefix_len, ra.wa, cm, max_W, lru_in, lru_out,       \
                       stats, w.aborted, err)
#define CR_CLASS(SL, SEQ)                                                                                           \
    if ((SEQ ? ra.classes : ra.wclasses) & (1u << ((SL) - 1))) {                                                   \
        const uint64_t nw = cand_map(SL, SEQ);                                                                      \
        if (nw) CR_REPLAY(SL, (SL) >= kTwoLevelFrom, SEQ, (nw + (kReplayThreads / 64) - 1) / (kReplayThreads / 64)); \
    }
    // The list sizes' launches and the grouped ones are independent of each other (other
    // candidates; the marked-segment bitmap takes atomic ORs); the kSeq passes read what all
    // of them marked, so they follow on the caller's stream after the join. A call under
    // stream capture keeps everything on the caller's stream.
    uint32_t nlaunch = __builtin_popcount(ra.wclasses) + __builtin_popcount(ra.groups);
    std::unique_lock<std::mutex> side_lock;
    SideStreams* side = nullptr;
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    if (CR_REPLAY_SIDE_STREAMS && nlaunch >= 2 && hipStreamIsCapturing(st, &cap) == hipSuccess &&
        cap == hipStreamCaptureStatusNone) {
        side_lock = std::unique_lock<std::mutex>(g_side_mu);
        side = side_streams();
    }
    hipStream_t lane_st[2] = {st, st};
    if (side) {
        if (hipEventRecord(side->fork, st) != hipSuccess || hipStreamWaitEvent(side->s[0], side->fork, 0) != hipSuccess ||
            hipStreamWaitEvent(side->s[1], side->fork, 0) != hipSuccess)
            return CR_EHIP;
        lane_st[0] = side->s[0];
        lane_st[1] = side->s[1];
    }
    // Launches in order of their work, each onto the stream with less work so far. A
    // launch's work is its candidates times a cost per candidate and request by list form,
    // in hundredths of the one-register list's (as measured alone on the 1e8-request sweep:
    // 0.98, 1.96, 2.2, 2.8 and 3.75 ms per candidate for 1, 2, 3, 5 and 8 registers, 0.55 and
    // 0.75 for the lists of 8 and 16 slots replayed 8 and 4 per wavefront).
    static constexpr uint32_t kCost[9] = {0u, 100u, 200u, 225u, 255u, 285u, 320u, 350u, 385u};
    struct Launch { uint32_t kind; uint64_t work; };  // kind 1..8: k_replay<kind>; 100 + G: k_replay_grp<G>
    Launch todo[10];
    uint32_t nt = 0;
    for (uint32_t SL = 1; SL <= 8; ++SL)
        if (ra.wclasses & (1u << (SL - 1))) {
            uint64_t wk = 0;
            for (uint32_t c = 0; c < P; ++c)
                if (slot_class(W[c]) == SL && ra.wa.grp[c] == 1u) wk += kCost[SL];
            todo[nt++] = Launch{SL, wk};
        }
    for (uint32_t G = 4; G <= 8; G += 4)
        if (ra.groups & (1u << G)) {
            uint64_t wk = 0;
            for (uint32_t c = 0; c < P; ++c)
                if (ra.wa.grp[c] == G) wk += G == 8u ? 56u : 77u;
            todo[nt++] = Launch{100u + G, wk};
        }
    for (uint32_t a = 1; a < nt; ++a)  // insertion sort, heaviest first
        for (uint32_t b = a; b > 0 && todo[b].work > todo[b - 1].work; --b) {
            const Launch t = todo[b];
            todo[b] = todo[b - 1];
            todo[b - 1] = t;
        }
    uint64_t load[2] = {0, 0};
    for (uint32_t t = 0; t < nt; ++t) {
        const int li = load[1] < load[0] ? 1 : 0;  // the less loaded stream
        load[li] += todo[t].work;
        const hipStream_t ls = lane_st[li];
        const uint32_t k = todo[t].kind;
#define CR_ON(SL)                                                                                                  \
        if (k == (SL)) {                                                                                          \
            const uint64_t nw = cand_map(SL, false);                                                              \
            if (nw)                                                                                               \
                hipLaunchKernelGGL((k_replay<SL, (SL) >= kTwoLevelFrom, false>),                                  \
                                   dim3((uint32_t)((nw + (kReplayThreads / 64) - 1) / (kReplayThreads / 64))),     \
                                   dim3(kReplayThreads), 0, ls, w.rec, n, w.grp_off, w.item_off, P, R, num_keys, J, \
                                   prefix_len, ra.wa, cm, max_W, lru_in, lru_out, stats, w.aborted, err);           \
        }
        CR_ON(1) CR_ON(2) CR_ON(3) CR_ON(4) CR_ON(5) CR_ON(6) CR_ON(7) CR_ON(8)
#undef CR_ON
        // several lists per wavefront; their marked segments join the kSeq pass of k_replay<1>
#define CR_GRP(G)                                                                                                  \
        if (k == 100u + (G))                                                                                       \
            hipLaunchKernelGGL((k_replay_grp<G>), dim3((uint32_t)gblocks), dim3(kReplayThreads), 0, ls, w.rec, n,   \
                               w.grp_off, w.item_off, w.gwave_off, P, R, num_keys, prefix_len, ra.wa, max_W, lru_in, \
                               lru_out, stats, w.aborted, err);
        CR_GRP(4) CR_GRP(8)
#undef CR_GRP
    }
    if (side) {
        for (int i = 0; i < 2; ++i)
            if (hipEventRecord(side->join[i], side->s[i]) != hipSuccess ||
                hipStreamWaitEvent(st, side->join[i], 0) != hipSuccess)
                return CR_EHIP;
        side_lock.unlock();
    }
    CR_CLASS(1, true); CR_CLASS(2, true); CR_CLASS(3, true); CR_CLASS(4, true);
    CR_CLASS(5, true); CR_CLASS(6, true); CR_CLASS(7, true); CR_CLASS(8, true);
#undef CR_CLASS
#undef CR_REPLAY
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}

extern "C" cr_status cr_replay(const uint32_t* keys, const uint16_t* suffix, const uint32_t* prefix_len,
                               uint32_t num_keys, const uint16_t* dest, uint64_t n, const uint64_t* off, uint32_t J,
                               uint32_t P, uint32_t R, const uint32_t* W, uint32_t max_W, const uint32_t* lru_in,
                               uint32_t* lru_out, uint64_t* stats, void* ws, size_t ws_bytes, uint32_t* err,
                               void* stream)
{
    using namespace cr;
    ReplayArgs ra;
    cr_status v = replay_args(n, J, P, R, W, max_W, ws_bytes, ws, &ra);
    if (v != CR_OK) return v;
    if (num_keys == 0 || num_keys == 0xFFFFFFFFu || !prefix_len || !lru_out || !stats || !err || !off ||
        (n > 0 && (!keys || !suffix || !dest)))
        return CR_EINVAL;
    if (lru_in && lru_in < lru_out + (uint64_t)P * R * max_W && lru_out < lru_in + (uint64_t)P * R * max_W)
        return CR_EINVAL;
    v = cr_replay_partition(keys, suffix, dest, n, off, J, P, R, W, ws, ws_bytes, err, stream);
    if (v != CR_OK) return v;
    return cr_replay_lru(prefix_len, num_keys, n, J, P, R, W, max_W, lru_in, lru_out, stats, ws, ws_bytes, err,
                         stream);
}
