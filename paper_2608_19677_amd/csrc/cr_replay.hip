// Shadow replay of P candidate routings against per-destination LRU prefix caches
// (Section 3.2: admitted and cold prefixes share one cache per destination; Section 3.1
// equal-slot model: W whole-prefix slots per destination).
//
// Pipeline (all on the caller's stream, workspace from the caller):
//   k_part_hist / k_part_scan / k_part_scatter
//        stable partition of every candidate's requests by destination, preserving
//        arrival order; each record packs (key, suffix, interval) into 8 bytes;
//   k_seg_items
//        splits every (candidate, destination) stream into segments of S records;
//   k_replay<SL>
//        one wavefront per segment. The LRU state before a segment is exactly the most
//        recent W distinct keys seen at that destination (carried state appended), so a
//        wavefront rebuilds it by scanning backwards, then replays its segment. This
//        turns R*P sequential streams into thousands of independent wavefronts with
//        results identical to one sequential pass.
// The LRU lives in registers: slot (s, lane) holds a key and its recency rank (0 = most
// recent). A lookup is one compare per slot plus a ballot; the update is a rank shift, so
// no per-request search or reduction is needed.
#include "cr_common.h"

namespace cr {
namespace {

constexpr int kReplayThreads = 256;

struct WArg {
    uint16_t W[CR_MAX_CANDS];
};

__host__ __device__ __forceinline__ uint32_t seg_len(uint32_t W)
{
    const uint32_t s = 16u * W;
    return s < 2048u ? 2048u : (s > 16384u ? 16384u : s);
}

__host__ __device__ __forceinline__ uint32_t slot_class(uint32_t W)
{
    return W <= 64 ? 1u : (W <= 128 ? 2u : (W <= 256 ? 4u : 8u));
}

struct PartGeom {
    uint64_t tile;
    uint64_t ntiles;
};

inline PartGeom part_geom(uint64_t n, uint32_t P)
{
    const uint64_t target = 8192u / P > 0 ? 8192u / P : 1u;
    uint64_t tile = (n + target - 1) / target;
    if (tile < 1024) tile = 1024;
    tile = (tile + 63) & ~63ull;
    return PartGeom{tile, n ? (n + tile - 1) / tile : 0};
}

__global__ __launch_bounds__(256) void k_part_hist(const uint16_t* __restrict__ dest, uint64_t n, uint32_t R,
                                                   uint64_t tile, uint64_t ntiles, uint32_t* __restrict__ tcnt,
                                                   uint32_t* __restrict__ err)
{
    extern __shared__ uint32_t h[];
    const uint32_t c = blockIdx.y;
    const uint64_t t = blockIdx.x;
    const uint64_t t0 = t * tile, t1 = t0 + tile < n ? t0 + tile : n;
    for (uint32_t d = threadIdx.x; d < R; d += blockDim.x) h[d] = 0;
    __syncthreads();
    const uint16_t* __restrict__ dc = dest + (uint64_t)c * n;
    bool bad = false;
    for (uint64_t i = t0 + threadIdx.x; i < t1; i += blockDim.x) {
        const uint32_t d = dc[i];
        if (d < R) atomicAdd(&h[d], 1u);
        else bad = true;
    }
    __syncthreads();
    for (uint32_t d = threadIdx.x; d < R; d += blockDim.x) tcnt[((uint64_t)c * R + d) * ntiles + t] = h[d];
    if (bad) atomicOr(err, CR_ERR_DEST_RANGE);
}

// One block per candidate: exclusive scan of tcnt[c][d][tile] in (d, tile) order.
__global__ __launch_bounds__(1024) void k_part_scan(uint32_t* __restrict__ tcnt, uint32_t R, uint64_t ntiles,
                                                    uint32_t* __restrict__ grp_off)
{
    __shared__ uint32_t s_scan[16];
    const uint32_t c = blockIdx.x;
    uint32_t* __restrict__ t = tcnt + (uint64_t)c * R * ntiles;
    const uint64_t len = (uint64_t)R * ntiles;
    uint32_t carry = 0;
    for (uint64_t e0 = 0; e0 < len; e0 += 4u * blockDim.x) {
        const uint64_t e = e0 + 4u * threadIdx.x;
        uint32_t v[4];
        uint32_t s = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            v[q] = e + q < len ? t[e + q] : 0u;
            s += v[q];
        }
        uint32_t tot;
        uint32_t ex = block_exscan_u32(s, s_scan, &tot) + carry;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (e + q < len) t[e + q] = ex;
            ex += v[q];
        }
        carry += tot;
    }
    __syncthreads();
    uint32_t* __restrict__ go = grp_off + (uint64_t)c * (R + 1u);
    for (uint32_t d = threadIdx.x; d < R; d += blockDim.x) go[d] = ntiles ? t[(uint64_t)d * ntiles] : 0u;
    if (threadIdx.x == 0) go[R] = carry;
}

// One wavefront per (tile, candidate): stable scatter into packed records.
__global__ __launch_bounds__(64) void k_part_scatter(const uint32_t* __restrict__ keys,
                                                     const uint16_t* __restrict__ suffix,
                                                     const uint16_t* __restrict__ dest, uint64_t n,
                                                     const uint64_t* __restrict__ off, uint32_t J, uint32_t R,
                                                     uint32_t nbits, uint64_t tile, uint64_t ntiles,
                                                     const uint32_t* __restrict__ tcnt, uint64_t* __restrict__ rec)
{
    extern __shared__ uint32_t run[];
    const uint32_t c = blockIdx.y, lane = lane_id();
    const uint64_t t = blockIdx.x;
    const uint64_t t0 = t * tile, t1 = t0 + tile < n ? t0 + tile : n;
    for (uint32_t d = lane; d < R; d += 64) run[d] = tcnt[((uint64_t)c * R + d) * ntiles + t];
    __syncthreads();
    const uint16_t* __restrict__ dc = dest + (uint64_t)c * n;
    uint64_t* __restrict__ rc = rec + (uint64_t)c * n;
    uint32_t j = find_interval(off, J, t0);
    for (uint64_t base = t0; base < t1; base += 64) {
        const uint64_t i = base + lane;
        const bool in = i < t1;
        const uint32_t d = in ? dc[i] : 0xFFFFu;
        const bool valid = in && d < R;
        uint32_t jl = j;
        while (jl + 1 < J && off[jl + 1] <= i) ++jl;
        uint64_t peers = ballot(valid);
        for (uint32_t bit = 0; bit < nbits; ++bit) {
            const bool on = (d >> bit) & 1u;
            const uint64_t bb = ballot(on);
            peers &= on ? bb : ~bb;
        }
        const uint32_t rk = (uint32_t)__popcll(peers & lanemask_lt());
        if (valid) {
            const uint32_t pos = run[d] + rk;
            rc[pos] = (uint64_t)keys[i] | ((uint64_t)suffix[i] << 32) | ((uint64_t)jl << 48);
        }
        __syncthreads();
        if (valid && rk == 0) run[d] += (uint32_t)__popcll(peers);
        __syncthreads();
        j = rdlane(jl, 63);
    }
}

// Work items: one per segment of every (candidate, destination) stream (at least one).
__global__ __launch_bounds__(1024) void k_seg_items(const uint32_t* __restrict__ grp_off, uint32_t P, uint32_t R,
                                                    WArg wa, uint32_t* __restrict__ item_off)
{
    __shared__ uint32_t s_scan[16];
    const uint32_t total = P * R;
    uint32_t carry = 0;
    for (uint32_t e0 = 0; e0 < total; e0 += blockDim.x) {
        const uint32_t e = e0 + threadIdx.x;
        uint32_t nseg = 0;
        if (e < total) {
            const uint32_t c = e / R, d = e % R;
            const uint32_t* go = grp_off + (uint64_t)c * (R + 1u);
            const uint32_t cnt = go[d + 1] - go[d];
            const uint32_t S = seg_len(wa.W[c]);
            nseg = cnt ? (cnt + S - 1) / S : 1u;
        }
        uint32_t tot;
        const uint32_t ex = block_exscan_u32(nseg, s_scan, &tot);
        if (e < total) item_off[e] = carry + ex;
        carry += tot;
    }
    if (threadIdx.x == 0) item_off[total] = carry;
}

template <int SL>
__device__ __forceinline__ bool lru_contains(const uint32_t (&skey)[SL], uint32_t kk)
{
    uint64_t m = 0;
#pragma unroll
    for (int s = 0; s < SL; ++s) m |= ballot(skey[s] == kk);
    return m != 0;
}

template <int SL>
__device__ __forceinline__ void lru_put_slot(uint32_t (&skey)[SL], uint32_t q, uint32_t kk, uint32_t lane)
{
#pragma unroll
    for (int s = 0; s < SL; ++s)
        if ((uint32_t)s == (q >> 6) && lane == (q & 63u)) skey[s] = kk;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += (uint64_t)__shfl_xor((unsigned long long)v, o, 64);
    return v;
}

template <int SL>
__global__ __launch_bounds__(kReplayThreads) void k_replay(
    const uint64_t* __restrict__ rec, uint64_t n, const uint32_t* __restrict__ grp_off,
    const uint32_t* __restrict__ item_off, uint32_t P, uint32_t R, uint32_t K, uint32_t J, const uint32_t* __restrict__ prefix_len,
    WArg wa, uint32_t max_W, const uint32_t* __restrict__ lru_in, uint32_t* __restrict__ lru_out,
    uint64_t* __restrict__ stats, uint32_t* __restrict__ err)
{
    const uint32_t lane = lane_id();
    const uint64_t item = (uint64_t)blockIdx.x * (kReplayThreads / 64) + (threadIdx.x >> 6);
    const uint32_t ncd = P * R;
    if (item >= item_off[ncd]) return;
    uint32_t lo = 0, hi = ncd;
    while (hi - lo > 1) {
        const uint32_t mid = (lo + hi) >> 1;
        if (item_off[mid] <= item) lo = mid;
        else hi = mid;
    }
    const uint32_t c = lo / R, d = lo % R;
    const uint32_t W = wa.W[c];
    if (slot_class(W) != (uint32_t)SL) return;
    const uint32_t seg = (uint32_t)(item - item_off[lo]);
    const uint32_t* go = grp_off + (uint64_t)c * (R + 1u);
    const uint32_t gs = go[d], cnt = go[d + 1] - gs;
    const uint32_t S = seg_len(W);
    const uint32_t s0 = seg * S;
    const uint32_t s1 = cnt - s0 < S ? cnt : s0 + S;
    const uint64_t* __restrict__ rl = rec + (uint64_t)c * n + gs;

    uint32_t skey[SL], srank[SL];
#pragma unroll
    for (int s = 0; s < SL; ++s) {
        const uint32_t idx = (uint32_t)s * 64u + lane;
        skey[s] = CR_EMPTY_SLOT;
        srank[s] = idx < W ? idx : 0xFFFFFFFFu;
    }
    // State before the segment: most recent W distinct keys, newest first.
    uint32_t q = 0;
    for (uint32_t pos = s0; q < W && pos > 0;) {
        const uint32_t nb = pos < 64u ? pos : 64u;
        const uint32_t kl = lane < nb ? (uint32_t)rl[pos - nb + lane] : CR_EMPTY_SLOT;
        for (int t = (int)nb - 1; t >= 0 && q < W; --t) {
            const uint32_t kk = rdlane(kl, (uint32_t)t);
            if (kk >= K) continue;
            if (!lru_contains<SL>(skey, kk)) {
                lru_put_slot<SL>(skey, q, kk, lane);
                ++q;
            }
        }
        pos -= nb;
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
                    lru_put_slot<SL>(skey, q, kk, lane);
                    ++q;
                }
            }
        }
    }

    uint64_t a_req = 0, a_hit = 0, a_pre = 0, a_hp = 0;
    uint32_t cur = 0xFFFFFFFFu;
    bool bad = false;
    auto flush = [&](uint32_t iv) {
        if (iv >= J) return;
        const uint64_t r0 = wave_sum_u64(a_req), r1 = wave_sum_u64(a_hit), r2 = wave_sum_u64(a_pre),
                       r3 = wave_sum_u64(a_hp);
        if (lane == 0) {
            unsigned long long* st = (unsigned long long*)(stats + (((uint64_t)iv * P + c) * R + d) * 4u);
            atomicAdd(st + 0, (unsigned long long)r0);
            if (r1) atomicAdd(st + 1, (unsigned long long)r1);
            atomicAdd(st + 2, (unsigned long long)r2);
            if (r3) atomicAdd(st + 3, (unsigned long long)r3);
        }
        a_req = a_hit = a_pre = a_hp = 0;
    };
    for (uint32_t b0 = s0; b0 < s1; b0 += 64) {
        const uint32_t nb = s1 - b0 < 64u ? s1 - b0 : 64u;
        const uint64_t rv = lane < nb ? rl[b0 + lane] : 0ull;
        const uint32_t kl = lane < nb ? (uint32_t)rv : CR_EMPTY_SLOT;
        const uint32_t sfx = (uint32_t)(rv >> 32) & 0xFFFFu;
        const uint32_t ivl = (uint32_t)(rv >> 48);
        const bool vl = lane < nb && kl < K;
        bad |= lane < nb && kl >= K;
        const uint32_t pl = vl ? prefix_len[kl] : 0u;
        uint64_t hm = 0;
        for (uint32_t t = 0; t < nb; ++t) {
            const uint32_t kk = rdlane(kl, t);
            if (kk >= K) continue;
            uint32_t rh = W - 1;
            bool hit = false;
#pragma unroll
            for (int s = 0; s < SL; ++s) {
                const uint64_t m = ballot(skey[s] == kk);
                if (m) {
                    hit = true;
                    rh = rdlane(srank[s], first_lane(m));
                }
            }
#pragma unroll
            for (int s = 0; s < SL; ++s) {
                const bool sel = srank[s] == rh;
                const bool up = srank[s] < rh;
                skey[s] = sel ? kk : skey[s];
                srank[s] = sel ? 0u : (up ? srank[s] + 1u : srank[s]);
            }
            hm |= (uint64_t)hit << t;
        }
        const bool hl = (hm >> lane) & 1ull;
        uint64_t rem = ballot(vl);
        while (rem) {
            const uint32_t iv = rdlane(ivl, first_lane(rem));
            if (iv != cur) {
                flush(cur);
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
    flush(cur);
    if (ballot(bad) && lane == 0) atomicOr(err, CR_ERR_KEY_RANGE);
    if (s1 == cnt) {
        uint32_t* __restrict__ lo_ = lru_out + ((uint64_t)c * R + d) * max_W;
#pragma unroll
        for (int s = 0; s < SL; ++s) {
            const uint32_t idx = (uint32_t)s * 64u + lane;
            if (idx < W && srank[s] < W) lo_[srank[s]] = skey[s];
        }
        for (uint32_t idx = W + lane; idx < max_W; idx += 64) lo_[idx] = CR_EMPTY_SLOT;
    }
}

struct ReplayWs {
    uint64_t* rec;
    uint32_t* tcnt;
    uint32_t* grp_off;
    uint32_t* item_off;
    size_t bytes;
};

inline ReplayWs replay_layout(void* base, uint64_t n, uint32_t P, uint32_t R)
{
    const PartGeom g = part_geom(n, P);
    auto up = [](uint64_t x) { return (x + 255) & ~255ull; };
    uint64_t o = 0;
    ReplayWs w{};
    uint8_t* b = reinterpret_cast<uint8_t*>(base);
    const uint64_t o_rec = o;
    o = up(o + (uint64_t)P * n * 8u);
    const uint64_t o_t = o;
    o = up(o + (uint64_t)P * R * g.ntiles * 4u);
    const uint64_t o_g = o;
    o = up(o + (uint64_t)P * (R + 1u) * 4u);
    const uint64_t o_i = o;
    o = up(o + ((uint64_t)P * R + 1u) * 4u);
    w.rec = reinterpret_cast<uint64_t*>(b + o_rec);
    w.tcnt = reinterpret_cast<uint32_t*>(b + o_t);
    w.grp_off = reinterpret_cast<uint32_t*>(b + o_g);
    w.item_off = reinterpret_cast<uint32_t*>(b + o_i);
    w.bytes = (size_t)o + 256u;
    return w;
}

}  // namespace
}  // namespace cr

extern "C" size_t cr_replay_workspace_bytes(uint64_t n, uint32_t P, uint32_t R)
{
    return cr::replay_layout(nullptr, n, P, R).bytes;
}

extern "C" cr_status cr_replay(const uint32_t* keys, const uint16_t* suffix, const uint32_t* prefix_len,
                               uint32_t num_keys, const uint16_t* dest, uint64_t n, const uint64_t* off, uint32_t J,
                               uint32_t P, uint32_t R, const uint32_t* W, uint32_t max_W, const uint32_t* lru_in,
                               uint32_t* lru_out, uint64_t* stats, void* ws, size_t ws_bytes, uint32_t* err,
                               void* stream)
{
    using namespace cr;
    if (P == 0 || P > CR_MAX_CANDS || R == 0 || R > CR_MAX_R || J == 0 || J > CR_MAX_J || !W || max_W == 0 ||
        max_W > CR_MAX_W || num_keys == 0 || num_keys == 0xFFFFFFFFu || !off || !lru_out || !stats || !ws || !err ||
        !prefix_len)
        return CR_EINVAL;
    if (n > 0 && (!keys || !suffix || !dest)) return CR_EINVAL;
    if (n >= 0xFFFFFFFFull) return CR_EINVAL;
    if (lru_in && lru_in < lru_out + (uint64_t)P * R * max_W && lru_out < lru_in + (uint64_t)P * R * max_W)
        return CR_EINVAL;
    WArg wa{};
    uint32_t classes = 0;
    for (uint32_t c = 0; c < P; ++c) {
        if (W[c] == 0 || W[c] > max_W) return CR_EINVAL;
        wa.W[c] = (uint16_t)W[c];
        classes |= slot_class(W[c]);
    }
    if (ws_bytes < cr_replay_workspace_bytes(n, P, R)) return CR_ESIZE;
    void* base = reinterpret_cast<void*>(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    const ReplayWs w = replay_layout(base, n, P, R);
    const PartGeom g = part_geom(n, P);
    const hipStream_t st = as_stream(stream);
    uint32_t nbits = 0;
    while ((1u << nbits) < R) ++nbits;
    (void)hipGetLastError();
    if (g.ntiles) {
        hipLaunchKernelGGL(k_part_hist, dim3((uint32_t)g.ntiles, P), dim3(256), (size_t)R * 4u, st, dest, n, R, g.tile,
                           g.ntiles, w.tcnt, err);
    }
    hipLaunchKernelGGL(k_part_scan, dim3(P), dim3(1024), 0, st, w.tcnt, R, g.ntiles, w.grp_off);
    if (g.ntiles) {
        hipLaunchKernelGGL(k_part_scatter, dim3((uint32_t)g.ntiles, P), dim3(64), (size_t)R * 4u, st, keys, suffix, dest,
                           n, off, J, R, nbits, g.tile, g.ntiles, w.tcnt, w.rec);
    }
    hipLaunchKernelGGL(k_seg_items, dim3(1), dim3(1024), 0, st, w.grp_off, P, R, wa, w.item_off);
    // Upper bound on work items: one per (c, d) plus one per full segment.
    const uint64_t items = (uint64_t)P * R + (uint64_t)P * n / 2048u + 1u;
    const uint64_t blocks = (items + (kReplayThreads / 64) - 1) / (kReplayThreads / 64);
    if (blocks > 0x7FFFFFFFull) return CR_EINVAL;
#define CR_REPLAY(SL)                                                                                               \
    hipLaunchKernelGGL(k_replay<SL>, dim3((uint32_t)blocks), dim3(kReplayThreads), 0, st, w.rec, n, w.grp_off,       \
                       w.item_off, P, R, num_keys, J, prefix_len, wa, max_W, lru_in, lru_out, stats, err)
    if (classes & 1u) CR_REPLAY(1);
    if (classes & 2u) CR_REPLAY(2);
    if (classes & 4u) CR_REPLAY(4);
    if (classes & 8u) CR_REPLAY(8);
#undef CR_REPLAY
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}
