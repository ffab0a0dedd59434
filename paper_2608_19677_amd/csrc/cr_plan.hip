// Plan build: top-rate admission (Eq. 1; Section 3.1 "Warm-set admission"; Algorithm 1)
// and LPT placement (Section 3.1 "Placement and dispatch"; Algorithm 1 placement loop).
//
// Admission is split in two so that every candidate plan built from the same window
// shares one sort:
//   k_sort_window  one block per window: radix-select the C_max-th largest count, compact
//                  the keys at or above it in key order, and stable-LSD-radix-sort them by
//                  count (descending), which yields (count desc, key asc) exactly;
//   k_admit_plan   one block per plan: k by Eq. 1 in exact integers, block prefix sum of
//                  k, and the longest prefix whose sum fits C = R * W.
// LPT is a dependency chain of sum(k) steps per plan, cut into exact batches of
// consecutive jobs: one wavefront per plan for R <= 64 (k_lpt_small), one block of up to
// 1,024 threads per plan above that (k_lpt_block).
// k_plan_churn compares pairs of built plans for the replanning study.
#include <math.h>

#include <mutex>
#include <utility>

#include "cr_common.h"

namespace cr {
namespace {

constexpr int kSortThreads = 1024;
constexpr int kSortWaves = kSortThreads / kWave;

__host__ __device__ __forceinline__ bool hash_placed(uint32_t variant)
{
    return variant == CR_PLAN_AFFINITY || variant == CR_PLAN_REPLICATED;
}

__device__ __forceinline__ uint32_t wave_sum_u32(uint32_t v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += (uint64_t)__shfl_xor((unsigned long long)v, o, 64);
    return v;
}

__device__ __forceinline__ uint32_t wave_max_u32(uint32_t v)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const uint32_t u = __shfl_xor(v, o, 64);
        v = u > v ? u : v;
    }
    return v;
}

__device__ __forceinline__ uint32_t wave_exscan_u32(uint32_t v, uint32_t* total)
{
    const uint32_t x = wave_incl_scan_u32(v);
    *total = rdlane(x, 63);
    return x - v;
}

constexpr uint32_t kSortBlock = 1024;                // 16 wavefronts per window
constexpr uint32_t kSortNW = kSortBlock / 64;
constexpr uint32_t kSortLdsRowBytes = 96u * 1024u;  // rows up to this size are staged in LDS

// Loads counts[b] for b = base + 4*tid + {0..3} (zero past K), 16 bytes per thread when
// the row allows it.
__device__ __forceinline__ uint4 load4(const uint32_t* __restrict__ row, uint32_t K, uint32_t b, bool vec)
{
    if (vec && b + 3 < K) return *reinterpret_cast<const uint4*>(row + b);
    return make_uint4(b < K ? row[b] : 0u, b + 1 < K ? row[b + 1] : 0u, b + 2 < K ? row[b + 2] : 0u,
                      b + 3 < K ? row[b + 3] : 0u);
}

// One 1024-thread block per window. The window's nonzero keys are ordered by (count desc,
// key asc) and cut at C_max in three steps, each with O(1) block barriers:
//  1. one pass over the row: nnz, max, sum and a histogram of min(count, 255); the
//     C_max-th largest count t is read off the histogram unless it is >= 255, in which
//     case an MSB radix select over the row finds it;
//  2. ordered compaction: every wavefront owns a contiguous slice of the row, counts
//     what it keeps, takes its offset from the other wavefronts' totals, and writes its
//     keys in key order (keys equal to t are kept up to the number still needed);
//  3. stable LSD radix sort by (max - count) over the kept entries, 8 bits per pass, each
//     wavefront scattering a contiguous slice with ballot-ranked digits.
// When the row fits, step 1 also stages it in LDS and the later passes read it there.
template <bool kRowLds>
__global__ __launch_bounds__(kSortBlock) void k_sort_window(const uint32_t* __restrict__ counts, uint32_t K,
                                                            uint32_t Cmax, uint32_t* __restrict__ order,
                                                            uint32_t* __restrict__ order_count,
                                                            uint32_t* __restrict__ n_order,
                                                            uint64_t* __restrict__ row_sum, uint2* __restrict__ buf)
{
    extern __shared__ uint32_t s_row[];  // [K] when kRowLds
    __shared__ uint32_t s_hist[kSortNW][256];
    __shared__ uint32_t s_h256[256];
    __shared__ uint32_t s_w[kSortNW][4];
    __shared__ uint32_t s_nnz, s_max, s_t, s_take;
    __shared__ unsigned long long s_sum;
    const uint32_t w = blockIdx.x, tid = threadIdx.x, lane = lane_id(), wv = wave_in_block();
    const uint32_t* __restrict__ grow = counts + (uint64_t)w * K;
    const bool vec = (((uintptr_t)grow) & 15u) == 0;
    const uint32_t* row = kRowLds ? s_row : grow;
    uint2* b0 = buf + (uint64_t)w * 2u * Cmax;
    uint2* b1 = b0 + Cmax;
    for (uint32_t d = tid; d < 256; d += kSortBlock) s_h256[d] = 0;
    if (tid == 0) {
        s_nnz = 0;
        s_max = 0;
        s_sum = 0;
    }
    __syncthreads();
    // 1. statistics and the clamped histogram
    {
        uint32_t nnz = 0, mx = 0;
        uint64_t sum = 0;
        for (uint32_t b = 4 * tid; b < K; b += 4 * kSortBlock * 2) {
            const uint4 q0 = load4(grow, K, b, vec), q1 = load4(grow, K, b + 4 * kSortBlock, vec);
            const uint32_t cs[8] = {q0.x, q0.y, q0.z, q0.w, q1.x, q1.y, q1.z, q1.w};
            if (kRowLds) {
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    if (b + u < K) s_row[b + u] = cs[u];
                    if (b + 4 * kSortBlock + u < K) s_row[b + 4 * kSortBlock + u] = cs[4 + u];
                }
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const uint32_t c = cs[u];
                if (c) {
                    ++nnz;
                    mx = c > mx ? c : mx;
                    sum += c;
                    atomicAdd(&s_h256[c < 255u ? c : 255u], 1u);
                }
            }
        }
        nnz = rdlane(wave_incl_scan_u32(nnz), 63);
        mx = wave_max_u32(mx);
        sum = wave_sum_u64(sum);
        if (lane == 0) {
            atomicAdd(&s_nnz, nnz);
            atomicMax(&s_max, mx);
            atomicAdd(&s_sum, (unsigned long long)sum);
        }
    }
    __syncthreads();
    const uint32_t nnz = s_nnz, mx = s_max;
    const uint32_t M = nnz < Cmax ? nnz : Cmax;
    if (tid == 0) {
        n_order[w] = M;
        row_sum[w] = s_sum;
    }
    if (M == 0) return;
    // threshold from the clamped histogram (wave 0, four bins per lane from 255 down)
    if (wv == 0) {
        uint32_t h[4], hs = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            h[q] = s_h256[255u - 4u * lane - q];
            hs += h[q];
        }
        uint32_t tot;
        uint32_t above = wave_exscan_u32(hs, &tot);
        uint32_t sel = 0, need = 0;
        bool found = false;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (!found && above < M && above + h[q] >= M) {
                sel = 255u - 4u * lane - q;
                need = M - above;
                found = true;
            }
            above += h[q];
        }
        const uint32_t fl = first_lane(ballot(found));
        if (lane == 0) {
            s_t = rdlane(sel, fl);
            s_take = rdlane(need, fl);
        }
    }
    __syncthreads();
    if (s_t == 255u) {
        // the threshold is at least 255: MSB radix select over the row (rare)
        uint32_t prefix = 0, pmask = 0, need = M;
        for (int shift = 24; shift >= 0; shift -= 8) {
            if ((mx >> shift) == 0) {
                pmask |= 0xFFu << shift;
                continue;
            }
            __syncthreads();
            for (uint32_t d = tid; d < 256; d += kSortBlock) s_h256[d] = 0;
            __syncthreads();
            for (uint32_t b = tid; b < K; b += kSortBlock) {
                const uint32_t c = row[b];
                if (c != 0 && (c & pmask) == prefix) atomicAdd(&s_h256[(c >> shift) & 255u], 1u);
            }
            __syncthreads();
            if (wv == 0) {
                uint32_t h[4], hs = 0;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    h[q] = s_h256[255u - 4u * lane - q];
                    hs += h[q];
                }
                uint32_t tot;
                uint32_t above = wave_exscan_u32(hs, &tot);
                uint32_t sel = 0, nn = 0;
                bool found = false;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (!found && above < need && above + h[q] >= need) {
                        sel = 255u - 4u * lane - q;
                        nn = need - above;
                        found = true;
                    }
                    above += h[q];
                }
                const uint32_t fl = first_lane(ballot(found));
                if (lane == 0) {
                    s_t = rdlane(sel, fl);
                    s_take = rdlane(nn, fl);
                }
            }
            __syncthreads();
            prefix |= s_t << shift;
            pmask |= 0xFFu << shift;
            need = s_take;
        }
        __syncthreads();
        if (tid == 0) {
            s_t = prefix;
            s_take = need;
        }
        __syncthreads();
    }
    const uint32_t t = s_t, take_eq = s_take;

    // 2. ordered compaction, one contiguous slice of the row per wavefront
    const uint32_t span = (((K + kSortNW - 1) / kSortNW) + 63u) & ~63u;
    const uint32_t lo = wv * span < K ? wv * span : K, hi = lo + span < K ? lo + span : K;
    {
        uint32_t gt = 0, eq = 0;
        for (uint32_t b = lo + lane; b < hi; b += 64) {
            const uint32_t c = row[b];
            gt += c > t;
            eq += c == t;
        }
        gt = rdlane(wave_incl_scan_u32(gt), 63);
        eq = rdlane(wave_incl_scan_u32(eq), 63);
        if (lane == 0) {
            s_w[wv][0] = gt;
            s_w[wv][1] = eq;
        }
    }
    __syncthreads();
    {
        uint32_t eq_before = 0, sel_before = 0;
        for (uint32_t q = 0; q < wv; ++q) {
            const uint32_t eqq = s_w[q][1];
            const uint32_t left = take_eq > eq_before ? take_eq - eq_before : 0u;
            sel_before += s_w[q][0] + (eqq < left ? eqq : left);
            eq_before += eqq;
        }
        uint32_t running = sel_before, eq_seen = eq_before;
        for (uint32_t base = lo; base < hi; base += 64) {
            const uint32_t b = base + lane;
            const uint32_t c = b < hi ? row[b] : 0u;
            const uint64_t meq = ballot(b < hi && c == t);
            const uint32_t eq_rank = (uint32_t)__popcll(meq & lanemask_lt());
            const bool sel = b < hi && (c > t || (c == t && eq_seen + eq_rank < take_eq));
            const uint64_t ms = ballot(sel);
            const uint32_t pos = running + (uint32_t)__popcll(ms & lanemask_lt());
            if (sel && pos < M) b0[pos] = make_uint2(c, b);
            running += (uint32_t)__popcll(ms);
            eq_seen += (uint32_t)__popcll(meq);
        }
    }
    __syncthreads();

    // 3. stable LSD radix sort by v = mx - count (ascending v = descending count)
    const uint32_t range = mx - t;
    const uint32_t bits = range ? 32u - (uint32_t)__clz(range) : 0u;
    const uint32_t passes = (bits + 7u) / 8u;
    const uint32_t espan = (((M + kSortNW - 1) / kSortNW) + 63u) & ~63u;
    const uint32_t elo = wv * espan < M ? wv * espan : M, ehi = elo + espan < M ? elo + espan : M;
    uint2* src = b0;
    uint2* dst = b1;
    for (uint32_t pass = 0; pass < passes; ++pass) {
        const uint32_t shift = 8u * pass;
        for (uint32_t d = lane; d < 256; d += 64) s_hist[wv][d] = 0;
        for (uint32_t e = elo + lane; e < ehi; e += 64) atomicAdd(&s_hist[wv][((mx - src[e].x) >> shift) & 255u], 1u);
        __syncthreads();
        if (wv == 0) {  // offsets in (digit, wavefront) order
            uint32_t h[4][kSortNW], hs = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (uint32_t x = 0; x < kSortNW; ++x) {
                    h[q][x] = s_hist[x][4u * lane + q];
                    hs += h[q][x];
                }
            uint32_t tot;
            uint32_t ex = wave_exscan_u32(hs, &tot);
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (uint32_t x = 0; x < kSortNW; ++x) {
                    s_hist[x][4u * lane + q] = ex;
                    ex += h[q][x];
                }
        }
        __syncthreads();
        for (uint32_t e0 = elo; e0 < ehi; e0 += 64) {
            const uint32_t e = e0 + lane;
            const bool valid = e < ehi;
            const uint2 kv = valid ? src[e] : make_uint2(0u, 0u);
            const uint32_t d = valid ? ((mx - kv.x) >> shift) & 255u : 0u;
            uint64_t peers = ballot(valid);
#pragma unroll
            for (int bit = 0; bit < 8; ++bit) {
                const bool on = (d >> bit) & 1u;
                const uint64_t bb = ballot(on);
                peers &= on ? bb : ~bb;
            }
            const uint32_t rk = (uint32_t)__popcll(peers & lanemask_lt());
            const uint32_t at = valid ? s_hist[wv][d] + rk : 0u;
            if (valid && at < M) dst[at] = kv;
            if (valid && rk == 0) atomicAdd(&s_hist[wv][d], (uint32_t)__popcll(peers));
        }
        __syncthreads();
        uint2* tmp = src;
        src = dst;
        dst = tmp;
    }
    uint32_t* __restrict__ ord = order + (uint64_t)w * Cmax;
    uint32_t* __restrict__ ocnt = order_count + (uint64_t)w * Cmax;
    for (uint32_t e = tid; e < M; e += kSortBlock) {
        const uint2 kv = src[e];
        ord[e] = kv.y;
        ocnt[e] = kv.x;
    }
}

// Register-resident variant for rows of up to 1024 * kNpl keys and C_max <= kRegCmax:
// wavefront wv keeps its contiguous slice of the row in registers (kNpl values per lane,
// all loads in flight together), so the row is read from memory once and no LDS row copy
// limits the blocks per CU; the kept entries and both radix buffers live in LDS. Counts
// 1..3, the bulk of a long-tailed row, are histogrammed by ballots instead of contended
// LDS atomics. Same three steps and results as k_sort_window.
constexpr uint32_t kRegCmax = 2048;

// Up to 20 counts per thread the kernel fits 64 VGPRs, which leaves room for two blocks
// per CU (8 wavefronts per SIMD); the windows are independent, so that halves the rounds.
template <int kNpl>
__global__ __launch_bounds__(kSortBlock, kNpl <= 20 ? 8 : 1) void k_sort_window_reg(const uint32_t* __restrict__ counts, uint32_t K,
                                                                uint32_t Cmax, uint32_t* __restrict__ order,
                                                                uint32_t* __restrict__ order_count,
                                                                uint32_t* __restrict__ n_order,
                                                                uint64_t* __restrict__ row_sum)
{
    __shared__ uint2 s_buf[2][kRegCmax];
    __shared__ uint32_t s_hist[kSortNW][256];
    __shared__ uint32_t s_h256[256];
    __shared__ uint32_t s_w[kSortNW][2];
    __shared__ uint32_t s_nnz, s_max, s_t, s_take;
    __shared__ unsigned long long s_sum;
    const uint32_t w = blockIdx.x, tid = threadIdx.x, lane = lane_id(), wv = wave_in_block();
    const uint32_t* __restrict__ grow = counts + (uint64_t)w * K;
    const uint32_t span = (((K + kSortNW - 1) / kSortNW) + 63u) & ~63u;  // <= 64 * kNpl
    const uint32_t lo = wv * span < K ? wv * span : K, hi = lo + span < K ? lo + span : K;
    uint32_t v[kNpl];
    {  // the slice through a buffer resource: entries at or past hi read as 0
        const __amdgpu_buffer_rsrc_t rs = make_rsrc(grow + lo, (hi - lo) * 4u);
#pragma unroll
        for (int i = 0; i < kNpl; ++i) v[i] = __builtin_amdgcn_raw_buffer_load_b32(rs, (64u * i + lane) * 4u, 0, 0);
    }
    for (uint32_t d = tid; d < 256; d += kSortBlock) s_h256[d] = 0;
    if (tid == 0) {
        s_nnz = 0;
        s_max = 0;
        s_sum = 0;
    }
    __syncthreads();
    // 1. statistics and the clamped histogram
    {
        uint32_t nnz = 0, mx = 0, n1 = 0, n2 = 0, n3 = 0;  // per lane
        uint64_t sum = 0;
#pragma unroll
        for (int i = 0; i < kNpl; ++i) {
            const uint32_t c = v[i];
            nnz += c != 0u;
            n1 += c == 1u;
            n2 += c == 2u;
            n3 += c == 3u;
            mx = c > mx ? c : mx;
            sum += c;
            if (c >= 4u) atomicAdd(&s_h256[c < 255u ? c : 255u], 1u);
            __builtin_amdgcn_sched_barrier(0);
        }
        nnz = wave_sum_u32(nnz);
        n1 = wave_sum_u32(n1);
        n2 = wave_sum_u32(n2);
        n3 = wave_sum_u32(n3);
        mx = wave_max_u32(mx);
        sum = wave_sum_u64(sum);
        if (lane == 0) {
            atomicAdd(&s_nnz, nnz);
            atomicMax(&s_max, mx);
            atomicAdd(&s_sum, (unsigned long long)sum);
            if (n1) atomicAdd(&s_h256[1], n1);
            if (n2) atomicAdd(&s_h256[2], n2);
            if (n3) atomicAdd(&s_h256[3], n3);
        }
    }
    __syncthreads();
    const uint32_t nnz = s_nnz, mx = s_max;
    const uint32_t M = nnz < Cmax ? nnz : Cmax;
    if (tid == 0) {
        n_order[w] = M;
        row_sum[w] = s_sum;
    }
    if (M == 0) return;
    if (wv == 0) {  // threshold from the clamped histogram, four bins per lane from 255 down
        uint32_t h[4], hs = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            h[q] = s_h256[255u - 4u * lane - q];
            hs += h[q];
        }
        uint32_t tot;
        uint32_t above = wave_exscan_u32(hs, &tot);
        uint32_t sel = 0, need = 0;
        bool found = false;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            if (!found && above < M && above + h[q] >= M) {
                sel = 255u - 4u * lane - q;
                need = M - above;
                found = true;
            }
            above += h[q];
        }
        const uint32_t fl = first_lane(ballot(found));
        if (lane == 0) {
            s_t = rdlane(sel, fl);
            s_take = rdlane(need, fl);
        }
    }
    __syncthreads();
    if (s_t == 255u) {  // the threshold is at least 255: MSB radix select over the registers
        uint32_t prefix = 0, pmask = 0, need = M;
        for (int shift = 24; shift >= 0; shift -= 8) {
            if ((mx >> shift) == 0) {
                pmask |= 0xFFu << shift;
                continue;
            }
            __syncthreads();
            for (uint32_t d = tid; d < 256; d += kSortBlock) s_h256[d] = 0;
            __syncthreads();
#pragma unroll
            for (int i = 0; i < kNpl; ++i) {
                const uint32_t c = v[i];
                if (c != 0 && (c & pmask) == prefix) atomicAdd(&s_h256[(c >> shift) & 255u], 1u);
            }
            __syncthreads();
            if (wv == 0) {
                uint32_t h[4], hs = 0;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    h[q] = s_h256[255u - 4u * lane - q];
                    hs += h[q];
                }
                uint32_t tot;
                uint32_t above = wave_exscan_u32(hs, &tot);
                uint32_t sel = 0, nn = 0;
                bool found = false;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    if (!found && above < need && above + h[q] >= need) {
                        sel = 255u - 4u * lane - q;
                        nn = need - above;
                        found = true;
                    }
                    above += h[q];
                }
                const uint32_t fl = first_lane(ballot(found));
                if (lane == 0) {
                    s_t = rdlane(sel, fl);
                    s_take = rdlane(nn, fl);
                }
            }
            __syncthreads();
            prefix |= s_t << shift;
            pmask |= 0xFFu << shift;
            need = s_take;
        }
        __syncthreads();
        if (tid == 0) {
            s_t = prefix;
            s_take = need;
        }
        __syncthreads();
    }
    const uint32_t t = s_t, take_eq = s_take;

    // 2. ordered compaction from the registers (entry lo + 64 i + lane is in key order)
    {
        uint32_t gt = 0, eq = 0;  // per lane
#pragma unroll
        for (int i = 0; i < kNpl; ++i) {
            gt += v[i] > t;
            eq += v[i] == t;
        }
        gt = wave_sum_u32(gt);
        eq = wave_sum_u32(eq);
        if (lane == 0) {
            s_w[wv][0] = gt;
            s_w[wv][1] = eq;
        }
    }
    __syncthreads();
    {
        uint32_t eq_before = 0, sel_before = 0;
        for (uint32_t q = 0; q < wv; ++q) {
            const uint32_t eqq = s_w[q][1];
            const uint32_t left = take_eq > eq_before ? take_eq - eq_before : 0u;
            sel_before += s_w[q][0] + (eqq < left ? eqq : left);
            eq_before += eqq;
        }
        uint32_t running = sel_before, eq_seen = eq_before;
        const uint64_t lt = lanemask_lt();
#pragma unroll
        for (int i = 0; i < kNpl; ++i) {
            const uint32_t c = v[i];
            const uint64_t meq = ballot(c == t);
            const uint32_t eq_rank = (uint32_t)__popcll(meq & lt);
            const bool sel = c > t || (c == t && eq_seen + eq_rank < take_eq);
            const uint64_t ms = ballot(sel);
            const uint32_t pos = running + (uint32_t)__popcll(ms & lt);
            if (sel && pos < M) s_buf[0][pos] = make_uint2(c, lo + 64u * i + lane);
            running += (uint32_t)__popcll(ms);
            eq_seen += (uint32_t)__popcll(meq);
            __builtin_amdgcn_sched_barrier(0);  // one element's masks live at a time
        }
    }
    __syncthreads();

    // 3. stable LSD radix sort by v = mx - count in LDS
    const uint32_t range = mx - t;
    const uint32_t bits = range ? 32u - (uint32_t)__clz(range) : 0u;
    const uint32_t passes = (bits + 7u) / 8u;
    const uint32_t espan = (((M + kSortNW - 1) / kSortNW) + 63u) & ~63u;
    const uint32_t elo = wv * espan < M ? wv * espan : M, ehi = elo + espan < M ? elo + espan : M;
    uint32_t sb = 0;
    for (uint32_t pass = 0; pass < passes; ++pass) {
        const uint2* src = s_buf[sb];
        uint2* dst = s_buf[sb ^ 1u];
        const uint32_t shift = 8u * pass;
        for (uint32_t d = lane; d < 256; d += 64) s_hist[wv][d] = 0;
        for (uint32_t e = elo + lane; e < ehi; e += 64) atomicAdd(&s_hist[wv][((mx - src[e].x) >> shift) & 255u], 1u);
        __syncthreads();
        {  // offsets in (digit, wavefront) order: thread tid owns digit tid / 4, waves 4 (tid % 4) ..
            const uint32_t d = tid >> 2, x0 = (tid & 3u) * 4u;
            uint32_t hv[4], hs = 0;
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                hv[q] = s_hist[x0 + q][d];
                hs += hv[q];
            }
            __shared__ uint32_t s_scan[16];
            uint32_t tot;
            uint32_t ex = block_exscan_u32(hs, s_scan, &tot);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                s_hist[x0 + q][d] = ex;
                ex += hv[q];
            }
        }
        __syncthreads();
        for (uint32_t e0 = elo; e0 < ehi; e0 += 64) {
            const uint32_t e = e0 + lane;
            const bool valid = e < ehi;
            const uint2 kv = valid ? src[e] : make_uint2(0u, 0u);
            const uint32_t d = valid ? ((mx - kv.x) >> shift) & 255u : 0u;
            uint64_t peers = ballot(valid);
#pragma unroll
            for (int bit = 0; bit < 8; ++bit) {
                const bool on = (d >> bit) & 1u;
                const uint64_t bb = ballot(on);
                peers &= on ? bb : ~bb;
            }
            const uint32_t rk = (uint32_t)__popcll(peers & lanemask_lt());
            const uint32_t at = valid ? s_hist[wv][d] + rk : 0u;
            if (valid && at < M) dst[at] = kv;
            if (valid && rk == 0) atomicAdd(&s_hist[wv][d], (uint32_t)__popcll(peers));
        }
        __syncthreads();
        sb ^= 1u;
    }
    uint32_t* __restrict__ ord = order + (uint64_t)w * Cmax;
    uint32_t* __restrict__ ocnt = order_count + (uint64_t)w * Cmax;
    for (uint32_t e = tid; e < M; e += kSortBlock) {
        const uint2 kv = s_buf[sb][e];
        ord[e] = kv.y;
        ocnt[e] = kv.x;
    }
}

// Key index of a plan: bit b % 64 of word b / 64 is set for every admitted key b, and
// each word carries the key rank of its first admitted key (an exclusive scan of the
// word popcounts). Built in LDS when the words fit, else with global atomics.
constexpr uint32_t kKxLdsWords = 4096;  // 32 KB of bits: up to 262,144 keys

__device__ void build_key_index(const uint32_t* __restrict__ ord, uint32_t A, uint32_t KW, uint64_t* __restrict__ kx,
                                uint64_t* s_bits, uint32_t* s_scan)
{
    const uint32_t tid = threadIdx.x, bd = blockDim.x;
    const bool in_lds = KW <= kKxLdsWords;
    if (in_lds) {
        for (uint32_t w = tid; w < KW; w += bd) s_bits[w] = 0ull;
        __syncthreads();
        for (uint32_t a = tid; a < A; a += bd) {
            const uint32_t b = ord[a];
            atomicOr(reinterpret_cast<unsigned long long*>(&s_bits[b >> 6]), 1ull << (b & 63u));
        }
        __syncthreads();
    } else {
        for (uint32_t w = tid; w < KW; w += bd) kx[2u * w] = 0ull;
        __threadfence();
        __syncthreads();
        for (uint32_t a = tid; a < A; a += bd) {
            const uint32_t b = ord[a];
            atomicOr(reinterpret_cast<unsigned long long*>(&kx[2u * (b >> 6)]), 1ull << (b & 63u));
        }
        __threadfence();
        __syncthreads();
    }
    uint32_t carry = 0;
    for (uint32_t w0 = 0; w0 < KW; w0 += bd) {
        const uint32_t w = w0 + tid;
        uint64_t bits = 0;
        if (w < KW)
            bits = in_lds ? s_bits[w] : __hip_atomic_load(&kx[2u * w], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        uint32_t tot;
        const uint32_t ex = block_exscan_u32((uint32_t)__popcll(bits), s_scan, &tot);
        if (w < KW) {
            if (in_lds) kx[2u * w] = bits;
            kx[2u * w + 1u] = carry + ex;
        }
        carry += tot;
    }
}

// One block per plan: Eq. 1, the prefix admission and the plan's key index. Blocks of 8
// wavefronts: four fit on a CU, so a step's plans run in one round.
constexpr int kAdmitThreads = 512;

__global__ __launch_bounds__(kAdmitThreads) void k_admit_plan(
    uint32_t R, uint32_t Cmax, uint32_t NW, uint32_t KW,
    const cr_plan_spec* __restrict__ specs, const uint32_t* __restrict__ order,
    const uint32_t* __restrict__ order_count, const uint32_t* __restrict__ n_order,
    const uint64_t* __restrict__ row_sum, uint32_t* __restrict__ num_admitted, uint64_t* __restrict__ cold,
    uint32_t* __restrict__ clamped, uint32_t* __restrict__ member_off, uint64_t* __restrict__ key_index,
    uint32_t* __restrict__ err)
{
    __shared__ uint32_t s_scan[16];
    __shared__ unsigned long long s_carried;
    __shared__ uint64_t s_bits[kKxLdsWords];
    const uint32_t p = blockIdx.x, tid = threadIdx.x, bd = blockDim.x, lane = lane_id();
    const cr_plan_spec spec = specs[p];
    uint32_t* __restrict__ moff = member_off + (uint64_t)p * (Cmax + 1u);
    uint64_t* __restrict__ kx = key_index + (uint64_t)p * 2u * KW;
    const bool eq1 = spec.variant == CR_PLAN_FULL || spec.variant == CR_PLAN_REPLICATED;
    bool ok = spec.window < NW && spec.W >= 1 && (uint64_t)R * spec.W <= Cmax && spec.variant <= CR_PLAN_FLAT;
    // the flat variant admits nothing: its whole window is cold
    const uint32_t M = ok && spec.variant != CR_PLAN_FLAT ? n_order[spec.window] : 0u;
    // N_w: given, or (CR_WINDOW_SUM) the row's sum with the target relative to the mean load,
    // q_cap = (q_num / q_den) N_w / R, i.e. Eq. 1 with q_num N_w and q_den R
    const uint64_t nw = ok ? row_sum[spec.window] : 0ull;
    const bool rel = spec.n_window == CR_WINDOW_SUM;
    if (ok && !rel && spec.n_window != nw) ok = false;
    uint64_t q_num = spec.q_num, q_den = spec.q_den;
    if (ok && rel) {
        if (nw && q_num > 0x7FFFFFFFFFFFFFFFull / nw) ok = false;
        q_num *= nw;
        q_den *= R;
    }
    const uint64_t n_window = nw;
    if (ok && eq1 && M > 0 && (q_num == 0 || q_den == 0 || q_den >= (1ull << 31))) ok = false;
    if (!ok) {
        if (tid == 0) {
            num_admitted[p] = 0;
            cold[p] = 0;
            clamped[p] = 0;
            moff[0] = 0;
            atomicOr(err, CR_ERR_SPEC);
        }
        build_key_index(order, 0u, KW, kx, s_bits, s_scan);
        return;
    }
    const uint64_t C = (uint64_t)R * spec.W;
    const uint32_t* __restrict__ ocnt = order_count + (uint64_t)spec.window * Cmax;
    if (tid == 0) s_carried = 0;
    uint64_t used = 0;
    uint32_t A = 0, ncl = 0;
    for (uint32_t base = 0; base < M; base += bd) {
        const uint32_t a = base + tid;
        const bool valid = a < M;
        const uint32_t c = valid ? ocnt[a] : 0u;
        uint32_t k = 0;
        bool cl = false;
        if (valid && !eq1) {
            k = 1;  // affinity: one copy per admitted key
        } else if (valid) {
            const uint64_t num = (uint64_t)c * q_den;
            uint64_t kk = num / q_num + (num % q_num != 0);
            if (kk < 1) kk = 1;
            if (kk > R) {
                kk = R;
                cl = true;
            }
            k = (uint32_t)kk;
        }
        uint32_t ktot, ntot, ctot;
        const uint32_t ex = block_exscan_u32(k, s_scan, &ktot);
        const bool adm = valid && used + ex + k <= C;
        if (adm) moff[a] = (uint32_t)(used + ex);
        (void)block_exscan_u32(adm ? k : 0u, s_scan, &ntot);
        uint32_t nadm;
        (void)block_exscan_flag(adm, s_scan, &nadm);
        (void)block_exscan_flag(adm && cl, s_scan, &ctot);
        const uint64_t cs = wave_sum_u64(adm ? (uint64_t)c : 0ull);
        if (lane == 0 && cs) atomicAdd(&s_carried, (unsigned long long)cs);
        used += ntot;
        A += nadm;
        ncl += ctot;
        const uint32_t nvalid = M - base < bd ? M - base : bd;
        if (nadm < nvalid) break;
    }
    __syncthreads();
    if (tid == 0) {
        moff[A] = (uint32_t)used;
        num_admitted[p] = A;
        const uint64_t carried = s_carried;
        cold[p] = n_window >= carried ? n_window - carried : 0ull;
        clamped[p] = ncl;
    }
    build_key_index(order + (uint64_t)spec.window * Cmax, A, KW, kx, s_bits, s_scan);
}

__device__ __forceinline__ uint32_t dpp_shl1(uint32_t old, uint32_t v)  // lane i <- lane i+1
{
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, 0x130, 0xF, 0xF, false);
}

__device__ __forceinline__ uint32_t dpp_shr1(uint32_t old, uint32_t v)  // lane i <- lane i-1
{
    return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, 0x138, 0xF, 0xF, false);
}

__device__ __forceinline__ double dpp_shl1_f64(double v)
{
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = dpp_shl1((uint32_t)u, (uint32_t)u), hi = dpp_shl1((uint32_t)(u >> 32), (uint32_t)(u >> 32));
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

__device__ __forceinline__ double dpp_shr1_f64(double v)
{
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = dpp_shr1((uint32_t)u, (uint32_t)u), hi = dpp_shr1((uint32_t)(u >> 32), (uint32_t)(u >> 32));
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

struct LptBatch {
    uint32_t key, cnt, off, end;
};

__device__ __forceinline__ LptBatch lpt_load(const uint32_t* __restrict__ ord, const uint32_t* __restrict__ ocnt,
                                             const uint32_t* __restrict__ moff, uint32_t a, uint32_t A)
{
    LptBatch b{0u, 0u, 0u, 0u};
    if (a < A) {
        b.key = ord[a];
        b.cnt = ocnt[a];
        b.off = moff[a];
        b.end = moff[a + 1];
    }
    return b;
}

// Key index entry of key b ({bits, rank of the word's first admitted key}); the key's
// rank is entry.y + popcount of the bits below b.
__device__ __forceinline__ ulonglong2 kx_entry(const uint64_t* __restrict__ kx, uint32_t b, bool valid)
{
    return valid ? *reinterpret_cast<const ulonglong2*>(kx + 2u * (b >> 6)) : make_ulonglong2(0ull, 0ull);
}

__device__ __forceinline__ uint32_t kx_rank(ulonglong2 e, uint32_t b)
{
    return (uint32_t)e.y + (uint32_t)__popcll(e.x & ((1ull << (b & 63u)) - 1ull));
}

// R <= 64: lane i holds the i-th smallest (L, r), so the least-loaded destinations are
// lanes 0..k-1.
// Consecutive single-copy jobs are placed in batches. Job t+q would take lane q exactly as
// the sequential picks do as long as, for every q, lane q's load is below every charged
// load L_q' + x_q' of the earlier lanes q' < q (lane q is then the least (L, r) pair when
// job t+q is placed); an exclusive prefix minimum across the lanes gives the longest such
// batch M in one pass, ties ending it. The M charged lanes are merged back by rank: every
// lane's new position is the number of lanes with a smaller (L, r), counted either by
// pairwise exchanges over all lanes (many charged lanes) or by one ballot pass per charged
// lane (few), and one forward lane permutation applies it. A full round (M = R, equal x,
// order kept) needs no permutation.
// A batch of one is a single pick: three compares give the insertion rank and a one-lane
// DPP shift opens the slot; a job with k > 1 pops k lanes and re-inserts each.
// Admitted keys sit in two 64-key batches so a batch of jobs may straddle the boundary;
// the member picked for job a is kept in LDS slot a mod 128 until its batch is retired.
struct LptRaw {
    uint32_t key, cnt, off, end;
};

// Unconditional loads (the index is clamped into the plan's rows; entries past A are
// garbage and every use is masked by a < A): a load under an exec mask merges with a zero
// default, and that merge makes the wavefront wait for the load on the spot.
__device__ __forceinline__ LptRaw lpt_raw(const uint32_t* __restrict__ ord, const uint32_t* __restrict__ ocnt,
                                          const uint32_t* __restrict__ moff, uint32_t a, uint32_t Cmax)
{
    const uint32_t i = a < Cmax ? a : Cmax - 1u;
    return LptRaw{ord[i], ocnt[i], moff[i], moff[i + 1u]};
}

// The key index entry of key b as {bits lo, bits hi, rank of the word's first admitted key}
// (12 bytes: a 16-byte load would leave a dead register that the compiler may reuse, and
// the reuse has to wait for the load). Word indices past KW read word 0.
__device__ __forceinline__ uint3 kx_entry3(const uint64_t* __restrict__ kx, uint32_t b, uint32_t KW)
{
    const uint32_t w = (b >> 6) < KW ? (b >> 6) : 0u;
    return *reinterpret_cast<const uint3*>(kx + 2u * w);
}

__device__ __forceinline__ uint32_t kx_rank3(uint3 e, uint32_t b)
{
    const uint64_t bits = ((uint64_t)e.y << 32) | e.x;
    return e.z + (uint32_t)__popcll(bits & ((1ull << (b & 63u)) - 1ull));
}

__device__ __forceinline__ uint32_t ds_permute_u32(uint32_t dst_lane, uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_ds_permute((int)(dst_lane << 2), (int)v);
}

__device__ __forceinline__ double ds_permute_f64(uint32_t dst_lane, double v)
{
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = ds_permute_u32(dst_lane, (uint32_t)u), hi = ds_permute_u32(dst_lane, (uint32_t)(u >> 32));
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

__device__ __forceinline__ uint32_t ds_bpermute_u32(uint32_t src_lane, uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_ds_bpermute((int)(src_lane << 2), (int)v);
}

__device__ __forceinline__ double ds_bpermute_f64(uint32_t src_lane, double v)
{
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = ds_bpermute_u32(src_lane, (uint32_t)u), hi = ds_bpermute_u32(src_lane, (uint32_t)(u >> 32));
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// (o, orv) < (a, r) as 0 or 1, without branches
__device__ __forceinline__ uint32_t lt_pair(double o, uint32_t orv, double a, uint32_t r)
{
    return (uint32_t)((o < a) | ((o == a) & (orv < r)));
}

// Lane i of a 16-lane row receives lane (i - kK) mod 16 of the same row (DPP row_ror:kK).
template <int kK>
__device__ __forceinline__ uint32_t row_ror_u32(uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x120 + kK, 0xF, 0xF, true);  // every source is in range
}

template <int kK>
__device__ __forceinline__ double row_ror_f64(double v)
{
    const uint64_t u = (uint64_t)__double_as_longlong(v);
    const uint32_t lo = row_ror_u32<kK>((uint32_t)u), hi = row_ror_u32<kK>((uint32_t)(u >> 32));
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// How many of the row rotations kKs of (ov, orv) are smaller than this lane's (a, r). One
// rotation at a time (a scheduling barrier after each): unrolled together, their compare
// masks outgrow the scalar registers.
template <int... kKs>
__device__ __forceinline__ uint32_t count_rotations(double a, uint32_t r, double ov, uint32_t orv,
                                                    std::integer_sequence<int, kKs...>)
{
    uint32_t c = 0;
    ((c += lt_pair(row_ror_f64<kKs>(ov), row_ror_u32<kKs>(orv), a, r), __builtin_amdgcn_sched_barrier(0)), ...);
    return c;
}

// DPP move of a double; lanes whose source is outside the pattern (or whose row is masked
// off) receive `fill`.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ double dpp_f64(double v, double fill)
{
    const uint64_t u = (uint64_t)__double_as_longlong(v), f = (uint64_t)__double_as_longlong(fill);
    const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)f, (int)(uint32_t)u, kCtrl, kRowMask, 0xF, false);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)(f >> 32), (int)(uint32_t)(u >> 32), kCtrl,
                                                              kRowMask, 0xF, false);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// min over lanes 0 .. lane-1 (+inf on lane 0)
__device__ __forceinline__ double wave_exclusive_min_f64(double v)
{
    const double inf = INFINITY;
    double s = dpp_f64<0x138, 0xF>(v, inf);  // wave_shr:1
    s = fmin(s, dpp_f64<0x111, 0xF>(s, inf));  // row_shr:1
    s = fmin(s, dpp_f64<0x112, 0xF>(s, inf));  // row_shr:2
    s = fmin(s, dpp_f64<0x114, 0xF>(s, inf));  // row_shr:4
    s = fmin(s, dpp_f64<0x118, 0xF>(s, inf));  // row_shr:8
    s = fmin(s, dpp_f64<0x142, 0xA>(s, inf));  // row_bcast:15 into rows 1 and 3
    s = fmin(s, dpp_f64<0x143, 0xC>(s, inf));  // row_bcast:31 into rows 2 and 3
    return s;
}

__global__ __launch_bounds__(64) void k_lpt_small(uint32_t KW, uint32_t R, uint32_t Cmax, uint32_t NW,
                                                  const cr_plan_spec* __restrict__ specs,
                                                  const uint32_t* __restrict__ order,
                                                  const uint32_t* __restrict__ order_count,
                                                  const uint32_t* __restrict__ num_admitted,
                                                  const uint64_t* __restrict__ cold,
                                                  const uint32_t* __restrict__ member_off,
                                                  const uint64_t* __restrict__ key_index,
                                                  uint16_t* __restrict__ members, double* __restrict__ load,
                                                  uint32_t* __restrict__ route)
{
    issue_priority_high();
    // member picked for single-copy job a in slot a mod 128; slots 128.. take the stores of
    // lanes >= R so that the round loop needs no divergent branch
    __shared__ uint32_t s_mem[192];
    const uint32_t p = blockIdx.x, lane = lane_id();
    const cr_plan_spec spec = specs[p];
    if (hash_placed(spec.variant)) return;  // placed by cr_place_hash
    const uint32_t A = (uint32_t)__builtin_amdgcn_readfirstlane((int)num_admitted[p]);
    const uint32_t w = spec.window < NW ? spec.window : 0u;
    const uint32_t* __restrict__ ord = order + (uint64_t)w * Cmax;
    const uint32_t* __restrict__ ocnt = order_count + (uint64_t)w * Cmax;
    const uint32_t* __restrict__ moff = member_off + (uint64_t)p * (Cmax + 1u);
    uint16_t* __restrict__ mem = members + (uint64_t)p * Cmax;
    const uint64_t* __restrict__ kx = key_index + (uint64_t)p * 2u * KW;
    uint32_t* __restrict__ rw = route + (uint64_t)p * Cmax;
    double Lv = lane < R ? (double)cold[p] / (double)R : INFINITY;
    uint32_t rv = lane < R ? lane : 0xFFFFu;
    // Three 64-job batches in registers: the one being placed (cur), the next (nxt: a batch of
    // jobs may reach into it) and the one after (nx2), loaded a whole batch before it is first
    // read. The three register sets take these roles in turn (the step below is inlined three
    // times), so a retired batch's registers are reloaded in place with no copy. What the
    // placement loop reads of the batches (kc, xc, mc, mn, coff) is derived when the previous
    // batch retires, before that retire issues its loads: every wait is then for loads issued
    // a batch earlier, and the loop reads no register a load wrote (a loop that stores and
    // reads such registers gets a wait for every outstanding load at its entry).
    LptRaw s0 = lpt_raw(ord, ocnt, moff, lane, Cmax);
    LptRaw s1 = lpt_raw(ord, ocnt, moff, 64 + lane, Cmax);
    LptRaw s2 = lpt_raw(ord, ocnt, moff, 128 + lane, Cmax);
    uint3 kxc = kx_entry3(kx, s0.key, KW);                  // needed when the batch retires
    uint32_t kc = lane < A ? s0.end - s0.off : 0u;         // k of the current batch's keys (0 past A)
    double xc = kc == 1 ? (double)s0.cnt : (double)s0.cnt / (double)(kc ? kc : 1u);
    // lane q: the count of job base+q (mc) or base+64+q (mn) if it is a single-copy job, else
    // ~0; the current batch's member offsets xor k (coff)
    uint32_t mc = kc == 1 ? s0.cnt : 0xFFFFFFFFu;
    uint32_t mn = s1.end - s1.off == 1 ? s1.cnt : 0xFFFFFFFFu;
    uint32_t coff = s0.off ^ kc;
    const uint64_t rmask = R >= 64 ? ~0ull : ((1ull << R) - 1ull);
    const uint32_t P2 = R <= 1u ? 1u : 1u << (32 - __builtin_clz(R - 1u));  // power of two >= R
    uint32_t base = 0, t = 0;
    // Places jobs until the current batch retires (true: cur now holds the batch after nx2,
    // nxt is current) or every job is placed (false, after the final retire).
    auto step = [&](LptRaw& cur, const LptRaw& nxt, const LptRaw& nx2) __attribute__((always_inline)) -> bool {
        while (base + t < A) {
            // the loop state is uniform; saying so keeps it (and the masks built from it) scalar
            t = (uint32_t)__builtin_amdgcn_readfirstlane((int)t);
            base = (uint32_t)__builtin_amdgcn_readfirstlane((int)base);
            if (t >= 64) {  // retire the current batch; its registers take the batch after nx2
                const uint32_t fm = s_mem[(base + lane) & 127u];
                const uint32_t rk = kx_rank3(kxc, cur.key);
                const bool one = kc == 1, live = base + lane < A;
                const uint32_t roff = coff ^ kc;
                kc = base + 64 + lane < A ? nxt.end - nxt.off : 0u;
                xc = (double)nxt.cnt;
                if (ballot(kc > 1)) xc = kc > 1 ? (double)nxt.cnt / (double)kc : xc;
                mc = kc == 1 ? nxt.cnt : 0xFFFFFFFFu;
                mn = nx2.end - nx2.off == 1 ? nx2.cnt : 0xFFFFFFFFu;
                coff = nxt.off ^ kc;
                kxc = kx_entry3(kx, nxt.key, KW);
                if (live) {
                    if (one) mem[roff] = (uint16_t)fm;
                    rw[rk] = one ? (CR_ROUTE_SINGLE | fm) : (base + lane);
                }
                base += 64;
                t -= 64;
                cur = lpt_raw(ord, ocnt, moff, base + 128 + lane, Cmax);
                return true;
            }
            const uint32_t k = rdlane(kc, t);
            if (k == 1) {
                // lane q looks at job t+q: its count if it is a single-copy job, else ~0
                const uint32_t src = (lane + t) & 63u;
                const uint32_t c1 = ds_bpermute_u32(src, mc), c2 = ds_bpermute_u32(src, mn);
                const uint32_t cq = lane + t < 64u ? c1 : c2;
                const bool jq = lane < R && cq != 0xFFFFFFFFu && base + t + lane < A;
                const double a = Lv + (double)cq;  // lane q's load once charged with job t+q
                const double pm = wave_exclusive_min_f64(jq ? a : INFINITY);
                const uint64_t okm = ballot(jq && (lane == 0 || Lv < pm));
                const uint32_t M = ~okm ? (uint32_t)__builtin_ctzll(~okm) : 64u;
                if (M >= 2) {
                    if (lane < M) s_mem[(base + t + lane) & 127u] = rv;
                    bool round = false;
                    const uint32_t c0 = rdlane(cq, 0);
                    if (M == R) {
                        const double an = dpp_shl1_f64(a);
                        const uint32_t rn = dpp_shl1(rv, rv);
                        round = ballot(lane < R && cq != c0) == 0 && ballot(lane + 1 < R && an == a && rn < rv) == 0;
                    }
                    if (round) {
                        Lv = lane < R ? a : Lv;
                        t += M;
                        // Further full rounds of the same run: the next R jobs have the same x, so
                        // the batch test reduces to every load being below min L + x, and the
                        // order test to the charged loads keeping their (L, r) order.
                        // (c0 is a single-copy job's count, never ~0)
                        const uint64_t same_c = ballot(mc == c0 && base + lane < A);
                        const uint64_t same_n = ballot(mn == c0 && base + 64 + lane < A);
                        const double x0 = (double)c0;
                        while (t < 64) {
                            // jobs t .. t+R-1 must all be single-copy jobs of count c0
                            const uint32_t e = t + R;  // one past the last job of the round (<= 128)
                            const uint64_t need_c = (e >= 64 ? ~0ull : ((1ull << e) - 1ull)) & ~((1ull << t) - 1ull);
                            const uint64_t need_n = e > 64 ? (e >= 128 ? ~0ull : ((1ull << (e - 64)) - 1ull)) : 0ull;
                            if ((same_c & need_c) != need_c || (same_n & need_n) != need_n) break;
                            const double an = Lv + x0;
                            const double v0 = rdlane_f64(an, 0);
                            const double ann = dpp_shl1_f64(an);
                            const uint32_t rn2 = dpp_shl1(rv, rv);
                            if (ballot(lane < R && !(Lv < v0)) != 0 || ballot(lane + 1 < R && ann == an && rn2 < rv) != 0)
                                break;
                            s_mem[lane < R ? ((base + t + lane) & 127u) : 128u + lane] = rv;
                            Lv = lane < R ? an : Lv;
                            t += R;
                            t = (uint32_t)__builtin_amdgcn_readfirstlane((int)t);
                        }
                        continue;
                    } else {
                        const bool charged = lane < M;
                        const double av = charged ? a : Lv;
                        uint32_t np = 0;
                        if (4u * M > P2) {
                            // All pairs: lane i counts the lanes with a smaller (L, r). The 15
                            // other lanes of its 16-lane row come by DPP row rotations; each other
                            // row of the power-of-two block that holds the R destinations is
                            // brought over once (lane i ^ x) and rotated the same way. Lanes >= R
                            // hold +inf and count for no one.
                            using Rot = std::integer_sequence<int, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15>;
                            np = count_rotations(av, rv, av, rv, Rot{});
                            for (uint32_t x = 16; x < P2; x += 16) {
                                const double sw = ds_bpermute_f64(lane ^ x, av);
                                const uint32_t sr = ds_bpermute_u32(lane ^ x, rv);
                                np += lt_pair(sw, sr, av, rv) + count_rotations(av, rv, sw, sr, Rot{});
                            }
                            np = lane < R ? np : lane;
                        } else {
                            // Few charged lanes: one pass per charged lane q. The lanes preceding
                            // lane q form a lane mask; uncharged lanes after q count it.
                            uint32_t cnt = 0;
                            const uint64_t unch = rmask & ~((M >= 64 ? ~0ull : (1ull << M) - 1ull));
                            auto pass = [&](uint32_t q) {
                                const double aq = rdlane_f64(av, q);
                                const uint32_t rq = rdlane(rv, q);
                                const uint64_t bm = ballot(av < aq) | (ballot(av == aq) & ballot(rv < rq));
                                cnt += __builtin_amdgcn_inverse_ballot_w64(unch & ~bm) ? 1u : 0u;
                                return (uint32_t)__popcll(bm & rmask);
                            };
                            uint32_t q = 0;
                            for (; q + 1 < M; q += 2) {
                                const uint32_t r0 = pass(q), r1 = pass(q + 1);
                                cnt = wrlane(wrlane(cnt, r0, q), r1, q + 1);
                            }
                            if (q < M) {
                                const uint32_t rl = pass(q);  // before cnt is read: pass() adds to it
                                cnt = wrlane(cnt, rl, q);
                            }
                            np = charged ? cnt : (lane < R ? lane - M + cnt : lane);
                        }
                        Lv = ds_permute_f64(np, av);
                        rv = ds_permute_u32(np, rv);
                    }
                    t += M;
                    continue;
                }
                const double x = rdlane_f64(xc, t);
                const double v0 = rdlane_f64(Lv, 0) + x;
                const uint32_t r0 = rdlane(rv, 0);
                if (lane == 0) s_mem[(base + t) & 127u] = r0;
                // rank of (v0, r0) among lanes 1..: three compares, each straight to a lane mask
                const uint64_t m_lt = ballot(Lv < v0), m_eq = ballot(Lv == v0), m_r = ballot(rv < r0);
                const uint32_t pos = (uint32_t)__popcll((m_lt | (m_eq & m_r)) & ~1ull);
                const double sl = dpp_shl1_f64(Lv);
                const uint32_t sr = dpp_shl1(rv, rv);
                const bool lt = lane < pos, eq = lane == pos;
                Lv = lt ? sl : (eq ? v0 : Lv);
                rv = lt ? sr : (eq ? r0 : rv);
            } else {
                const double x = rdlane_f64(xc, t);
                const uint32_t off = rdlane(coff, t) ^ k;
                if (lane < k) mem[off + lane] = (uint16_t)rv;
                const double vnew = Lv + x;  // meaningful on lanes < k
                const uint32_t rnew = rv;
                const double sL = __shfl(Lv, (int)((lane + k) & 63u), 64);
                const uint32_t sR = __shfl(rv, (int)((lane + k) & 63u), 64);
                Lv = lane + k < 64u ? sL : INFINITY;
                rv = lane + k < 64u ? sR : 0xFFFFu;
                for (uint32_t u = 0; u < k; ++u) {
                    const double v = rdlane_f64(vnew, u);
                    const uint32_t r = rdlane(rnew, u);
                    const uint64_t m_lt = ballot(Lv < v), m_eq = ballot(Lv == v), m_r = ballot(rv < r);
                    const uint32_t pos = (uint32_t)__popcll(m_lt | (m_eq & m_r));
                    const double up = dpp_shr1_f64(Lv);
                    const uint32_t upr = dpp_shr1(rv, rv);
                    const bool gt = lane > pos, eq = lane == pos;
                    Lv = gt ? up : (eq ? v : Lv);
                    rv = gt ? upr : (eq ? r : rv);
                }
            }
            ++t;
        }
        // retire what is left (the current batch, and the next one if a batch of jobs reached it)
        {
            const uint32_t fm = s_mem[(base + lane) & 127u];
            if (base + lane < A) {
                if (kc == 1) mem[cur.off] = (uint16_t)fm;
                rw[kx_rank3(kxc, cur.key)] = kc == 1 ? (CR_ROUTE_SINGLE | fm) : (base + lane);
            }
        }
        if (t > 64) {
            const uint32_t fm = s_mem[(base + 64 + lane) & 127u];
            if (lane < t - 64 && base + 64 + lane < A) {
                const uint32_t kn = nxt.end - nxt.off;
                if (kn == 1) mem[nxt.off] = (uint16_t)fm;
                rw[kx_rank3(kx_entry3(kx, nxt.key, KW), nxt.key)] = kn == 1 ? (CR_ROUTE_SINGLE | fm) : (base + 64 + lane);
            }
        }
        return false;
    };
    while (step(s0, s1, s2) && step(s1, s2, s0) && step(s2, s0, s1)) {
    }
    if (lane < R) load[(uint64_t)p * R + rv] = Lv;
}

// 64 < R <= 1024: one block of N threads (N = the power of two >= R) per plan; thread i
// holds the i-th smallest (L, r) pair in registers, and the sorted state is mirrored in LDS.
// Jobs are placed in batches, with the rule k_lpt_small uses: consecutive single-copy jobs
// t, t+1, ... take sorted positions 0, 1, ... while position q's load is below every load
// charged to the positions before it in the batch (position q is then the least (L, r) pair
// when job t+q is placed), found by a block-wide exclusive prefix minimum; ties end the
// batch. A job with k > 1 is a batch of its own that charges positions 0..k-1, its members in
// that order. After a batch the charged positions are merged back into the sorted state:
// when their new (L, r) pairs are still in order, by a merge path (each element's rank in the
// other sorted list by binary search in LDS); otherwise by a bitonic sort of all N pairs.
// On the large sweep (R = 1,024, up to 524,288 jobs per plan) a plan takes about 600
// batches. Route words are written afterwards by k_route_words, in parallel.
template <int N>
struct LptBlockLds {
    double v[2][N];        // sorted state (double-buffered for the merge)
    uint32_t r[2][N];
    double cv[N];          // the batch's charged pairs (positions 0..M-1)
    uint32_t cr[N];
    uint32_t jc[2 * N];    // job ring: counts, member offsets, k (0 past A)
    uint32_t jo[2 * N];
    uint16_t jk[2 * N];
    double wmin[N / 64];   // per-wavefront minimum of the charged loads
    double l0a[N / 64];    // per-wavefront lane 0: charged load, load, destination
    double l0v[N / 64];
    uint32_t l0r[N / 64];
    uint32_t wfail[N / 64];  // per-wavefront first position that fails the batch rule
    uint32_t wuns[N / 64];   // per-wavefront: the charged pairs are out of order
};

// Number of pairs among (v[lo .. lo+len)) smaller than (x, rx); the list is sorted.
__device__ __forceinline__ uint32_t lower_bound_pair(const double* __restrict__ v, const uint32_t* __restrict__ r,
                                                     uint32_t lo, uint32_t len, double x, uint32_t rx)
{
    uint32_t n = len, b = lo;
    while (n > 0) {
        const uint32_t h = n >> 1;
        const uint32_t m = b + h;
        if (lt_pair(v[m], r[m], x, rx)) {
            b = m + 1;
            n -= h + 1;
        } else {
            n = h;
        }
    }
    return b - lo;
}

template <int N>
__global__ __launch_bounds__(N) void k_lpt_block(uint32_t R, uint32_t Cmax, const cr_plan_spec* __restrict__ specs,
                                                 const uint32_t* __restrict__ order_count,
                                                 const uint32_t* __restrict__ num_admitted,
                                                 const uint64_t* __restrict__ cold, uint32_t NW,
                                                 const uint32_t* __restrict__ member_off,
                                                 uint16_t* __restrict__ members, double* __restrict__ load)
{
    static_assert(N >= 128 && N <= 1024 && (N & (N - 1)) == 0, "block of 128..1024 threads");
    constexpr uint32_t NWV = N / 64;
    __shared__ LptBlockLds<N> sh;
    issue_priority_high();
    const uint32_t p = blockIdx.x, i = threadIdx.x, lane = lane_id(), wv = i >> 6;
    const cr_plan_spec spec = specs[p];
    if (hash_placed(spec.variant)) return;  // placed by cr_place_hash
    const uint32_t A = num_admitted[p];
    const uint32_t w = spec.window < NW ? spec.window : 0u;
    const uint32_t* __restrict__ ocnt = order_count + (uint64_t)w * Cmax;
    const uint32_t* __restrict__ moff = member_off + (uint64_t)p * (Cmax + 1u);
    uint16_t* __restrict__ mem = members + (uint64_t)p * Cmax;
    const double INF = INFINITY;
    double v = i < R ? (double)cold[p] / (double)R : INF;
    uint32_t r = i < R ? i : 0xFFFFFFFFu;
    sh.v[0][i] = v;
    sh.r[0][i] = r;
    // job a: (count, member offset, k); k = 0 marks a >= A
    auto job = [&](uint32_t a, uint32_t& c, uint32_t& o, uint32_t& k) {
        const uint32_t aa = a < A ? a : 0u;
        c = ocnt[aa];
        o = moff[aa];
        k = a < A ? moff[aa + 1] - o : 0u;
    };
    uint32_t pc, po, pk;  // job base + 2N + i, loaded one refill ahead
    {
        uint32_t c, o, k;
        job(i, c, o, k);
        sh.jc[i] = c, sh.jo[i] = o, sh.jk[i] = (uint16_t)k;
        job(N + i, c, o, k);
        sh.jc[N + i] = c, sh.jo[N + i] = o, sh.jk[N + i] = (uint16_t)k;
        job(2 * N + i, pc, po, pk);
    }
    uint32_t cur = 0, base = 0, t = 0;
    __syncthreads();
    while (t < A) {
        const uint32_t rj = (t + i) & (2u * N - 1u), r0 = t & (2u * N - 1u);
        const uint32_t c = sh.jc[rj], o = sh.jo[rj], k = sh.jk[rj];
        const uint32_t k0 = sh.jk[r0];
        double a;
        uint32_t M;
        if (k0 > 1) {
            // multi-copy job t: positions 0..k0-1, each charged count / k0
            const double x0 = (double)sh.jc[r0] / (double)k0;
            a = v + x0;
            if (lane == 0) {
                sh.l0a[wv] = a;
                sh.l0v[wv] = v;
                sh.l0r[wv] = r;
            }
            M = k0;
            if (i < M) mem[sh.jo[r0] + i] = (uint16_t)r;
            __syncthreads();
        } else {
            const bool single = k == 1 && i < R;
            a = single ? v + (double)c : INF;  // position i's load once charged with job t+i
            double pm = wave_exclusive_min_f64(a);
            const double wtot = __shfl(fmin(pm, a), 63, 64);
            if (lane == 0) {
                sh.wmin[wv] = wtot;
                sh.l0a[wv] = a;
                sh.l0v[wv] = v;
                sh.l0r[wv] = r;
            }
            __syncthreads();
            for (uint32_t u = 0; u < wv; ++u) pm = fmin(pm, sh.wmin[u]);
            const bool ok = single && (i == 0 || v < pm);
            const uint64_t bad = ballot(!ok);
            if (lane == 0) sh.wfail[wv] = bad ? wv * 64u + (uint32_t)__builtin_ctzll(bad) : N;
            __syncthreads();
            M = N;
            for (uint32_t u = 0; u < NWV; ++u) M = min(M, sh.wfail[u]);
            if (i < M) mem[o] = (uint16_t)r;
        }
        // charged pairs (positions < M) and whether they are still in (L, r) order
        const bool charged = i < M;
        const double wv_ = charged ? a : v;
        double nx = __shfl_down(wv_, 1, 64);
        uint32_t nr = __shfl_down(r, 1, 64);
        if (lane == 63 && wv + 1 < NWV) {
            nx = (wv + 1) * 64u < M ? sh.l0a[wv + 1] : sh.l0v[wv + 1];
            nr = sh.l0r[wv + 1];
        }
        const bool out_of_order = i + 1 < M && !lt_pair(wv_, r, nx, nr);
        const uint64_t uns = ballot(out_of_order);
        if (lane == 0) sh.wuns[wv] = uns != 0;
        if (charged) {
            sh.cv[i] = a;
            sh.cr[i] = r;
        }
        __syncthreads();
        uint32_t any_uns = 0;
        for (uint32_t u = 0; u < NWV; ++u) any_uns |= sh.wuns[u];
        const uint32_t nxt = cur ^ 1u;
        if (!any_uns) {
            // merge path: charged list cv[0..M) and the unchanged sorted positions M..R-1
            if (i < R) {
                const uint32_t pos = charged ? i + lower_bound_pair(sh.v[cur], sh.r[cur], M, R - M, a, r)
                                             : (i - M) + lower_bound_pair(sh.cv, sh.cr, 0, M, v, r);
                sh.v[nxt][pos] = charged ? a : v;
                sh.r[nxt][pos] = r;
            } else {
                sh.v[nxt][i] = INF;
                sh.r[nxt][i] = 0xFFFFFFFFu;
            }
            __syncthreads();
            v = sh.v[nxt][i];
            r = sh.r[nxt][i];
        } else {
            // bitonic sort of all N pairs (positions >= R hold (+inf, ~0) and stay last)
            v = wv_;
            for (uint32_t kk = 2; kk <= N; kk <<= 1) {
                for (uint32_t j = kk >> 1; j > 0; j >>= 1) {
                    double pv;
                    uint32_t pr;
                    if (j >= 64) {
                        sh.v[nxt][i] = v;
                        sh.r[nxt][i] = r;
                        __syncthreads();
                        pv = sh.v[nxt][i ^ j];
                        pr = sh.r[nxt][i ^ j];
                        __syncthreads();
                    } else {
                        pv = __shfl_xor(v, (int)j, 64);
                        pr = __shfl_xor(r, (int)j, 64);
                    }
                    const bool up = (i & kk) == 0, lower = (i & j) == 0;
                    const bool pless = lt_pair(pv, pr, v, r) != 0;
                    if (pless == (lower == up)) {
                        v = pv;
                        r = pr;
                    }
                }
            }
            sh.v[nxt][i] = v;
            sh.r[nxt][i] = r;
        }
        cur = nxt;
        t += k0 > 1 ? 1u : (M ? M : 1u);  // M = 0 only for a job with k = 0, which admission never makes
        if (t >= base + N) {  // the ring's older half is consumed: refill it one half ahead
            const uint32_t slot = (base + i) & (2u * N - 1u);
            sh.jc[slot] = pc, sh.jo[slot] = po, sh.jk[slot] = (uint16_t)pk;
            base += N;
            job(base + 2 * N + i, pc, po, pk);
        }
        __syncthreads();
    }
    if (i < R) load[(uint64_t)p * R + r] = v;
}

// Route words of plans placed by k_lpt_block: per admitted key a, CR_ROUTE_SINGLE | its
// member when k = 1, else a, stored at the key's rank in the plan's key index.
constexpr uint32_t kWordThreads = 256;

__global__ __launch_bounds__(kWordThreads) void k_route_words(uint32_t Cmax, uint32_t NW, uint32_t KW,
                                                              const cr_plan_spec* __restrict__ specs,
                                                              const uint32_t* __restrict__ order,
                                                              const uint32_t* __restrict__ num_admitted,
                                                              const uint32_t* __restrict__ member_off,
                                                              const uint16_t* __restrict__ members,
                                                              const uint64_t* __restrict__ key_index,
                                                              uint32_t* __restrict__ route)
{
    const uint32_t p = blockIdx.y;
    const uint32_t a = blockIdx.x * kWordThreads + threadIdx.x;
    const cr_plan_spec spec = specs[p];
    if (hash_placed(spec.variant) || a >= num_admitted[p]) return;
    const uint32_t w = spec.window < NW ? spec.window : 0u;
    const uint32_t b = order[(uint64_t)w * Cmax + a];
    const uint32_t* __restrict__ moff = member_off + (uint64_t)p * (Cmax + 1u);
    const uint32_t o = moff[a], k = moff[a + 1] - o;
    const uint32_t word = k == 1 ? (CR_ROUTE_SINGLE | members[(uint64_t)p * Cmax + o]) : a;
    const ulonglong2 e = kx_entry(key_index + (uint64_t)p * 2u * KW, b, (b >> 6) < KW);
    route[(uint64_t)p * Cmax + kx_rank(e, b)] = word;
}

// Hash placement of the ablation variants (Section 5.2, 8B component ablation table).
// Members do not depend on the loads, so they are found for every admitted key at once
// (k_hash_members, one thread per key: k passes over the R hashes, each taking the
// smallest u above the previous pick, since one key's u values are distinct); only the
// load sums are ordered, and one wavefront per plan adds them in admission order with
// the destinations spread over its lanes (k_hash_loads).
constexpr uint32_t kHashThreads = 256;
constexpr uint32_t kHashStage = 4096;  // largest Cmax whose lists k_hash_loads keeps in LDS

inline size_t hash_loads_lds_bytes(uint32_t Cmax) { return (size_t)Cmax * 14u + 2u + 512u; }

__device__ __forceinline__ uint32_t place_key_hash(uint32_t seed, uint32_t b)
{
    return fmix32(b ^ fmix32(seed ^ 0x7F4A7C15u));
}

__global__ void __launch_bounds__(kHashThreads)
    k_hash_members(uint32_t R, uint32_t Cmax, uint32_t NW, uint32_t KW, const cr_plan_spec* __restrict__ specs,
                   const uint32_t* __restrict__ order, const uint32_t* __restrict__ num_admitted,
                   const uint32_t* __restrict__ member_off, const uint64_t* __restrict__ key_index,
                   uint16_t* __restrict__ members, uint32_t* __restrict__ route)
{
    const uint32_t p = blockIdx.x;
    const uint32_t variant = specs[p].variant;
    if (!hash_placed(variant)) return;
    const uint32_t A = min(num_admitted[p], Cmax);
    const uint32_t a = blockIdx.y * kHashThreads + threadIdx.x;
    if (a >= A) return;
    const uint32_t w = min(specs[p].window, NW - 1u);  // A > 0 only for a valid window
    const uint32_t b = order[(uint64_t)w * Cmax + a];
    const uint32_t* __restrict__ moff = member_off + (uint64_t)p * (Cmax + 1u);
    const uint32_t o = moff[a], k = moff[a + 1u] - o;
    const uint32_t kb = place_key_hash(specs[p].place_seed, b);
    uint16_t* __restrict__ mem = members + (uint64_t)p * Cmax + o;
    uint32_t prev = 0, first = 0;
    for (uint32_t t = 0; t < k; ++t) {
        uint32_t best_u = 0, best_r = R;
        for (uint32_t r = 0; r < R; ++r) {
            const uint32_t u = fmix32(kb ^ r);
            if ((t == 0 || u > prev) && (best_r == R || u < best_u)) {
                best_u = u;
                best_r = r;
            }
        }
        mem[t] = (uint16_t)best_r;
        prev = best_u;
        if (t == 0) first = best_r;
    }
    const ulonglong2 e = kx_entry(key_index + (uint64_t)p * 2u * KW, b, true);
    route[(uint64_t)p * Cmax + kx_rank(e, b)] = k == 1u ? (CR_ROUTE_SINGLE | first) : a;
}

template <int kS>
__global__ void __launch_bounds__(64)
    k_hash_loads(uint32_t R, uint32_t Cmax, uint32_t NW, const cr_plan_spec* __restrict__ specs,
                 const uint32_t* __restrict__ order_count, const uint32_t* __restrict__ num_admitted,
                 const uint64_t* __restrict__ cold, const uint32_t* __restrict__ member_off,
                 const uint16_t* __restrict__ members, double* __restrict__ load, bool lds_ok)
{
    const uint32_t p = blockIdx.x, lane = lane_id();
    const cr_plan_spec spec = specs[p];
    if (!hash_placed(spec.variant)) return;
    const uint32_t A = min((uint32_t)__builtin_amdgcn_readfirstlane((int)num_admitted[p]), Cmax);
    const uint32_t w = min(spec.window, NW - 1u);
    const uint32_t* __restrict__ ocnt = order_count + (uint64_t)w * Cmax;
    const uint32_t* __restrict__ moff = member_off + (uint64_t)p * (Cmax + 1u);
    const uint16_t* __restrict__ mem = members + (uint64_t)p * Cmax;
    const double init = (double)cold[p] / (double)R;
    double Lr[kS];
#pragma unroll
    for (int s = 0; s < kS; ++s) Lr[s] = init;
    // R <= 64 with the plan's lists in LDS (the host gives kS == 1 launches Cmax-sized
    // dynamic LDS when Cmax <= kHashStage): a destination's load needs only its own jobs, in
    // job order. The member copies (job order, each job's members distinct) are sorted
    // stably by destination in LDS, 64 at a time (a copy's rank is its destination's count
    // in earlier chunks plus the earlier lanes of its chunk with the same destination, by
    // ballots over the destination bits); lane r then adds the charges of its own list in
    // order -- the same additions, in the same order per destination, as the job loop below.
    if (kS == 1 && lds_ok) {
        extern __shared__ double s_dyn[];
        double* s_x = s_dyn;                                                  // [Cmax] job charges
        uint16_t* s_mem = reinterpret_cast<uint16_t*>(s_x + Cmax);           // [Cmax] members
        uint16_t* s_job = s_mem + Cmax;                                       // [Cmax] job of a copy
        uint16_t* s_ord = s_job + Cmax;                                       // [Cmax] sorted copies
        uint32_t* s_cnt = reinterpret_cast<uint32_t*>(s_ord + Cmax + (Cmax & 1u));  // [64]
        uint32_t* s_run = s_cnt + 64;                                         // [64]
        const uint32_t total = A ? (uint32_t)__builtin_amdgcn_readfirstlane((int)moff[A]) : 0u;  // <= Cmax
        s_cnt[lane] = 0;
        for (uint32_t a = lane; a < A; a += 64u) {
            const uint32_t o = moff[a], k = moff[a + 1u] - o;
            s_x[a] = (double)ocnt[a] / (double)k;
            for (uint32_t t = 0; t < k; ++t) s_job[o + t] = (uint16_t)a;
        }
        for (uint32_t i0 = 0; i0 < total; i0 += 16u * 64u) {  // all loads in flight
            uint32_t v[16];
#pragma unroll
            for (uint32_t u = 0; u < 16; ++u) {
                const uint32_t i = i0 + u * 64u + lane;
                v[u] = i < total ? (uint32_t)mem[i] : 0xFFFFu;
            }
#pragma unroll
            for (uint32_t u = 0; u < 16; ++u) {
                const uint32_t i = i0 + u * 64u + lane;
                if (i < total) {
                    s_mem[i] = (uint16_t)v[u];
                    if (v[u] < R) atomicAdd(&s_cnt[v[u]], 1u);
                }
            }
        }
        __syncthreads();
        const uint32_t cnt = lane < R ? s_cnt[lane] : 0u;
        const uint32_t off = wave_incl_scan_u32(cnt) - cnt;
        s_run[lane] = off;
        __syncthreads();
        uint32_t nbits = 0;
        while ((1u << nbits) < R) ++nbits;
        for (uint32_t i0 = 0; i0 < total; i0 += 64u) {
            const uint32_t i = i0 + lane;
            const uint32_t m = i < total ? (uint32_t)s_mem[i] : 0xFFFFu;
            const bool valid = m < R;
            uint64_t peers = ballot(valid);
            for (uint32_t bit = 0; bit < nbits; ++bit) {
                const bool on = (m >> bit) & 1u;
                const uint64_t bb = ballot(on);
                peers &= on ? bb : ~bb;
            }
            const uint32_t rk = (uint32_t)__popcll(peers & lanemask_lt());
            const uint32_t at = valid ? s_run[m] + rk : 0u;
            if (valid) s_ord[at] = s_job[i];
            __syncthreads();
            if (valid && rk == 0) s_run[m] = at + (uint32_t)__popcll(peers);
            __syncthreads();
        }
        double L = Lr[0];
        for (uint32_t q = 0; q < cnt; ++q) L = L + s_x[s_ord[off + q]];
        if (lane < R) load[(uint64_t)p * R + lane] = L;
        return;
    }
    for (uint32_t base = 0; base < A; base += 64u) {
        // lane j holds job base + j: its charge, copy count, first member and offset
        const uint32_t a = base + lane;
        double x = 0.0;
        uint32_t k = 0, d = 0xFFFFu, o = 0;
        if (a < A) {
            o = moff[a];
            k = moff[a + 1u] - o;
            x = (double)ocnt[a] / (double)k;
            d = mem[o];
        }
        const uint32_t nb = A - base < 64u ? A - base : 64u;
        for (uint32_t j = 0; j < nb; ++j) {
            const double xj = rdlane_f64(x, j);
            const uint32_t kj = rdlane(k, j);
            if (kj == 1u) {
                const uint32_t dj = rdlane(d, j);
#pragma unroll
                for (int s = 0; s < kS; ++s)
                    if (s * 64u + lane == dj) Lr[s] = Lr[s] + xj;
            } else {
                const uint32_t oj = rdlane(o, j);
                for (uint32_t t = 0; t < kj; ++t) {
                    const uint32_t m = mem[oj + t];
#pragma unroll
                    for (int s = 0; s < kS; ++s)
                        if (s * 64u + lane == m) Lr[s] = Lr[s] + xj;
                }
            }
        }
    }
#pragma unroll
    for (int s = 0; s < kS; ++s) {
        const uint32_t r = s * 64u + lane;
        if (r < R) load[(uint64_t)p * R + r] = Lr[s];
    }
}

// Churn between two plans of a set (Section 5.4; Appendix E, table of replan measurements).
// One block per pair (p, q): its threads walk p's admitted keys in admission order, look
// each key up in q's compact dispatch table (one 16-byte key-index load and a popcount)
// and compare the two member lists; the work per key is k_p * k_q compares.
constexpr uint32_t kChurnThreads = 256;

__global__ void __launch_bounds__(kChurnThreads)
    k_plan_churn(uint32_t NP, uint32_t KW, uint32_t Cmax, uint32_t NW, const cr_plan_spec* __restrict__ specs,
                 const uint32_t* __restrict__ order, const uint32_t* __restrict__ num_admitted,
                 const uint32_t* __restrict__ member_off, const uint16_t* __restrict__ members,
                 const uint64_t* __restrict__ key_index, const uint32_t* __restrict__ route,
                 const uint32_t* __restrict__ pairs, uint64_t* __restrict__ out, uint32_t* __restrict__ err)
{
    __shared__ uint64_t s_acc[4][kChurnThreads / kWave];
    const uint32_t pr = blockIdx.x;
    const uint32_t p = pairs[2u * pr], q = pairs[2u * pr + 1u];
    uint64_t common_pairs = 0, both = 0, k_changed = 0, same_set = 0;
    if (p < NP && q < NP) {
        const uint32_t A = min(num_admitted[p], Cmax);
        const uint32_t w = specs[p].window;
        const uint32_t* ord = order + (uint64_t)min(w, NW - 1u) * Cmax;
        const uint32_t* mop = member_off + (uint64_t)p * (Cmax + 1u);
        const uint16_t* mep = members + (uint64_t)p * Cmax;
        const uint64_t* kxq = key_index + (uint64_t)q * KW * 2u;
        const uint32_t* rwq = route + (uint64_t)q * Cmax;
        const uint32_t* moq = member_off + (uint64_t)q * (Cmax + 1u);
        const uint16_t* meq = members + (uint64_t)q * Cmax;
        for (uint32_t a = w < NW ? threadIdx.x : A; a < A; a += kChurnThreads) {
            const uint32_t b = ord[a];
            const ulonglong2 e = kx_entry(kxq, b, true);
            if (!((e.x >> (b & 63u)) & 1ull)) continue;  // not admitted by q
            const uint32_t word = rwq[kx_rank(e, b)];
            const bool single = (word & CR_ROUTE_SINGLE) != 0u;
            const uint32_t q0 = single ? 0u : moq[word];
            const uint32_t kq = single ? 1u : moq[word + 1u] - q0;
            const uint32_t p0 = mop[a], kp = mop[a + 1u] - p0;
            uint32_t common = 0;
            for (uint32_t i = 0; i < kp; ++i) {
                const uint32_t m = mep[p0 + i];
                if (single) {
                    common += m == (word & 0xFFFFu);
                } else {
                    for (uint32_t t = 0; t < kq; ++t) common += m == (uint32_t)meq[q0 + t];
                }
            }
            common_pairs += common;
            both += 1u;
            k_changed += kp != kq;
            same_set += kp == kq && common == kp;
        }
    } else if (threadIdx.x == 0) {
        atomicOr(err, CR_ERR_SPEC);
    }
    const uint32_t wv = threadIdx.x / kWave;
    common_pairs = wave_sum_u64(common_pairs);
    both = wave_sum_u64(both);
    k_changed = wave_sum_u64(k_changed);
    same_set = wave_sum_u64(same_set);
    if ((threadIdx.x & (kWave - 1u)) == 0u) {
        s_acc[0][wv] = common_pairs;
        s_acc[1][wv] = both;
        s_acc[2][wv] = k_changed;
        s_acc[3][wv] = same_set;
    }
    __syncthreads();
    if (threadIdx.x < 4u) {
        uint64_t v = 0;
#pragma unroll
        for (uint32_t i = 0; i < kChurnThreads / kWave; ++i) v += s_acc[threadIdx.x][i];
        out[4ull * pr + threadIdx.x] = v;
    }
}

inline uint32_t key_words(uint32_t K) { return (K + 63u) / 64u; }

bool valid_set(const cr_plan_set* ps)
{
    if (!ps) return false;
    if (ps->num_plans == 0 || ps->cands == 0 || ps->cands > CR_MAX_CANDS || ps->num_plans % ps->cands) return false;
    if (ps->R == 0 || ps->R > CR_MAX_R || ps->max_W == 0 || ps->max_W > CR_MAX_W) return false;
    if (ps->num_keys == 0 || ps->num_keys == 0xFFFFFFFFu || ps->num_windows == 0) return false;
    if (!ps->specs || !ps->order || !ps->order_count || !ps->n_order || !ps->num_admitted || !ps->cold || !ps->clamped ||
        !ps->member_off || !ps->members || !ps->load || !ps->key_index || !ps->route)
        return false;
    return true;
}

}  // namespace
}  // namespace cr

extern "C" size_t cr_admit_workspace_bytes(uint32_t num_windows, uint32_t R, uint32_t max_W)
{
    const uint64_t cmax = (uint64_t)R * max_W;
    return (size_t)(num_windows * (2u * cmax * sizeof(uint2) + sizeof(uint64_t)) + 256u);
}

extern "C" void cr_plan_sizes(uint32_t num_plans, uint32_t cands, uint32_t R, uint32_t max_W, uint32_t num_keys,
                              uint32_t num_windows, size_t out_bytes[CR_PLAN_BUFFERS])
{
    if (!out_bytes) return;
    const uint64_t NP = num_plans, NW = num_windows, cmax = (uint64_t)R * max_W;
    const uint64_t NG = cands ? NP / cands : 0, CS = ((uint64_t)cands + 7) / 8 * 8;
    const uint64_t KW = ((uint64_t)num_keys + 63) / 64;
    const uint64_t b[CR_PLAN_BUFFERS] = {
        NP * sizeof(cr_plan_spec), NW * cmax * 4, NW * cmax * 4, NW * 4, NP * 4, NP * 8, NP * 4,
        NP * (cmax + 1) * 4, NP * cmax * 2, NP * R * 8, NP * KW * 16, NP * cmax * 4,
        NW * num_keys * 4, NG * cmax * CS * 2, NG * R * CS * 2, NG * cmax * CS * 4};
    for (int i = 0; i < CR_PLAN_BUFFERS; ++i) out_bytes[i] = (size_t)b[i];
}

extern "C" cr_status cr_admit(const uint32_t* counts, const cr_plan_set* plans, void* ws, size_t ws_bytes,
                              uint32_t* err, void* stream)
{
    using namespace cr;
    if (!counts || !valid_set(plans) || !ws || !err) return CR_EINVAL;
    const uint32_t cmax = plans->R * plans->max_W;
    if (ws_bytes < cr_admit_workspace_bytes(plans->num_windows, plans->R, plans->max_W)) return CR_ESIZE;
    uint8_t* base = reinterpret_cast<uint8_t*>(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    uint2* buf = reinterpret_cast<uint2*>(base);
    uint64_t* row_sum = reinterpret_cast<uint64_t*>(base + (uint64_t)plans->num_windows * 2u * cmax * sizeof(uint2));
    const hipStream_t st = as_stream(stream);
    (void)hipGetLastError();
    const uint32_t K = plans->num_keys;
    if (cmax <= kRegCmax && K <= 1024u * 32u) {
#define CR_SORT_REG(NPL)                                                                                            \
    hipLaunchKernelGGL(k_sort_window_reg<NPL>, dim3(plans->num_windows), dim3(kSortBlock), 0, st, counts, K, cmax,  \
                       plans->order, plans->order_count, plans->n_order, row_sum)
        if (K <= 1024u * 4u) CR_SORT_REG(4);
        else if (K <= 1024u * 8u) CR_SORT_REG(8);
        else if (K <= 1024u * 16u) CR_SORT_REG(16);
        else if (K <= 1024u * 20u) CR_SORT_REG(20);
        else CR_SORT_REG(32);
#undef CR_SORT_REG
    } else if ((uint64_t)plans->num_keys * 4u <= kSortLdsRowBytes) {
        const uint32_t lds = plans->num_keys * 4u;
        if (hipFuncSetAttribute((const void*)k_sort_window<true>, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)lds) != hipSuccess)
            return CR_EHIP;
        hipLaunchKernelGGL(k_sort_window<true>, dim3(plans->num_windows), dim3(kSortBlock), (size_t)lds, st, counts,
                           plans->num_keys, cmax, plans->order, plans->order_count, plans->n_order, row_sum, buf);
    } else {
        hipLaunchKernelGGL(k_sort_window<false>, dim3(plans->num_windows), dim3(kSortBlock), 0, st, counts,
                           plans->num_keys, cmax, plans->order, plans->order_count, plans->n_order, row_sum, buf);
    }
    hipLaunchKernelGGL(k_admit_plan, dim3(plans->num_plans), dim3(kAdmitThreads), 0, st, plans->R, cmax,
                       plans->num_windows, key_words(plans->num_keys), plans->specs, plans->order, plans->order_count,
                       plans->n_order, row_sum, plans->num_admitted, plans->cold, plans->clamped, plans->member_off,
                       plans->key_index, err);
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}

extern "C" cr_status cr_place_lpt(const uint32_t* counts, const cr_plan_set* plans, void* stream)
{
    using namespace cr;
    if (!counts || !valid_set(plans)) return CR_EINVAL;
    const uint32_t cmax = plans->R * plans->max_W;
    const hipStream_t st = as_stream(stream);
    (void)hipGetLastError();
    if (plans->R <= 64) {
        hipLaunchKernelGGL(k_lpt_small, dim3(plans->num_plans), dim3(64), 0, st, key_words(plans->num_keys), plans->R,
                           cmax, plans->num_windows, plans->specs, plans->order, plans->order_count,
                           plans->num_admitted, plans->cold, plans->member_off, plans->key_index, plans->members,
                           plans->load, plans->route);
        return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
    }
#define CR_LPT_BLOCK(NT)                                                                                          \
    hipLaunchKernelGGL(k_lpt_block<NT>, dim3(plans->num_plans), dim3(NT), 0, st, plans->R, cmax, plans->specs,     \
                       plans->order_count, plans->num_admitted, plans->cold, plans->num_windows, plans->member_off, \
                       plans->members, plans->load)
    if (plans->R <= 128) CR_LPT_BLOCK(128);
    else if (plans->R <= 256) CR_LPT_BLOCK(256);
    else if (plans->R <= 512) CR_LPT_BLOCK(512);
    else CR_LPT_BLOCK(1024);
#undef CR_LPT_BLOCK
    hipLaunchKernelGGL(k_route_words, dim3((cmax + kWordThreads - 1) / kWordThreads, plans->num_plans),
                       dim3(kWordThreads), 0, st, cmax, plans->num_windows, key_words(plans->num_keys), plans->specs,
                       plans->order, plans->num_admitted, plans->member_off, plans->members, plans->key_index,
                       plans->route);
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}

extern "C" cr_status cr_plan_churn(const cr_plan_set* plans, const uint32_t* pairs, uint32_t num_pairs, uint64_t* out,
                                   uint32_t* err, void* stream)
{
    using namespace cr;
    if (!valid_set(plans) || !err || (num_pairs > 0 && (!pairs || !out))) return CR_EINVAL;
    if (num_pairs > 0x7FFFFFFFu) return CR_EINVAL;
    if (num_pairs == 0) return CR_OK;
    const hipStream_t st = as_stream(stream);
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_plan_churn, dim3(num_pairs), dim3(kChurnThreads), 0, st, plans->num_plans,
                       key_words(plans->num_keys), plans->R * plans->max_W, plans->num_windows, plans->specs,
                       plans->order, plans->num_admitted, plans->member_off, plans->members, plans->key_index,
                       plans->route, pairs, out, err);
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}

extern "C" cr_status cr_place_hash(const uint32_t* counts, const cr_plan_set* plans, void* stream)
{
    using namespace cr;
    if (!counts || !valid_set(plans)) return CR_EINVAL;
    const uint32_t cmax = plans->R * plans->max_W;
    const hipStream_t st = as_stream(stream);
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_hash_members, dim3(plans->num_plans, (cmax + kHashThreads - 1) / kHashThreads),
                       dim3(kHashThreads), 0, st, plans->R, cmax, plans->num_windows, key_words(plans->num_keys),
                       plans->specs, plans->order, plans->num_admitted, plans->member_off, plans->key_index,
                       plans->members, plans->route);
#define CR_HASH_LOADS(S, LDS, OK)                                                                                   \
    hipLaunchKernelGGL(k_hash_loads<S>, dim3(plans->num_plans), dim3(64), (LDS), st, plans->R, cmax,                  \
                       plans->num_windows, plans->specs, plans->order_count, plans->num_admitted, plans->cold,        \
                       plans->member_off, plans->members, plans->load, (OK))
    const uint32_t s = (plans->R + 63) / 64;
    const bool lds_ok = s <= 1 && cmax <= kHashStage;  // R <= 64: the plan's lists fit in LDS
    if (s <= 1) CR_HASH_LOADS(1, lds_ok ? hash_loads_lds_bytes(cmax) : 0, lds_ok);
    else if (s <= 2) CR_HASH_LOADS(2, 0, false);
    else if (s <= 4) CR_HASH_LOADS(4, 0, false);
    else if (s <= 8) CR_HASH_LOADS(8, 0, false);
    else CR_HASH_LOADS(16, 0, false);
#undef CR_HASH_LOADS
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}

// ---------------------------------------------------------------------------------------
// cr_admit_noalloc: cr_admit with its workspace in a library-owned device array instead of
// the caller's. The array is a file-scope __device__ variable; its name in host code is a
// stand-in, so its device address is taken once per device with hipGetSymbolAddress (with
// that device current) and kept. Every call on a device shares that device's array.
// ---------------------------------------------------------------------------------------
namespace cr {
namespace {

constexpr size_t kAdmitScratchBytes = (size_t)CR_ADMIT_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) uint8_t scratch[kAdmitScratchBytes];

std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

cr_status admit_scratch(void** out)
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return CR_EHIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return CR_EHIP;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return CR_OK;
}

}  // namespace
}  // namespace cr

extern "C" cr_status cr_admit_noalloc(const uint32_t* counts, const cr_plan_set* plans, uint32_t* err, void* stream)
{
    using namespace cr;
    if (!counts || !valid_set(plans) || !err) return CR_EINVAL;
    if (cr_admit_workspace_bytes(plans->num_windows, plans->R, plans->max_W) > kAdmitScratchBytes) return CR_ESIZE;
    void* ws = nullptr;
    const cr_status st = admit_scratch(&ws);
    if (st != CR_OK) return st;
    return cr_admit(counts, plans, ws, kAdmitScratchBytes, err, stream);
}
