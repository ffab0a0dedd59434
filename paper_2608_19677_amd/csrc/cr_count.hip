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

// ---------------------------------------------------------------------------------------
// One slice with a key space beyond LDS (cr_count_slice): device-scope atomics on an
// MI355X travel to memory past the per-XCD L2, so a global atomic per request costs about
// 0.4 ns of the whole chip, and a Zipf head puts millions of them on one address. The slice
// is counted without global atomics instead:
//   k_slice_tiles   each block sorts a tile of kTile keys by bucket (key / KB) in LDS and
//                   writes them back contiguously with the tile's bucket offsets;
//   k_slice_bins    block (group g, bucket u) counts bucket u's segment of every tile of
//                   group g into KB LDS bins and writes them as the group's partial row;
//   k_slice_reduce  counts[b] += sum over groups of partial[g][b].
// Traffic: the keys are read twice and written once (12 B per request), plus G partial rows.
// ---------------------------------------------------------------------------------------
constexpr uint32_t kTile = 4096;        // keys per k_slice_tiles block
constexpr uint32_t kTileThreads = 256;  // 16 keys per thread
constexpr uint32_t kMaxBuckets = 256;
constexpr uint32_t kBinThreads = 1024;

struct SliceGeom {
    uint32_t kb_log;    // KB = 1 << kb_log keys per bucket
    uint32_t nb;        // buckets
    uint64_t ntiles;
    uint32_t groups;    // G
    uint64_t keys_off, toff_off, part_off, bytes;  // workspace layout
};

inline SliceGeom slice_geom(uint64_t n, uint32_t K, int max_lds, int cus)
{
    SliceGeom g{};
    g.kb_log = 15;
    while (g.kb_log > 10 && ((uint64_t)4u << g.kb_log) > (uint64_t)max_lds) --g.kb_log;
    g.nb = (uint32_t)(((uint64_t)K + (1ull << g.kb_log) - 1) >> g.kb_log);
    g.ntiles = (n + kTile - 1) / kTile;
    uint64_t G = ((uint64_t)2 * cus + g.nb - 1) / g.nb;
    G = G < 1 ? 1 : G;
    G = G > g.ntiles ? (g.ntiles ? g.ntiles : 1) : G;
    g.groups = (uint32_t)G;
    auto up = [](uint64_t x) { return (x + 255) & ~255ull; };
    g.keys_off = 0;
    g.toff_off = up(n * 4u);
    g.part_off = up(g.toff_off + g.ntiles * (g.nb + 1ull) * 4u);
    g.bytes = up(g.part_off + (uint64_t)g.groups * g.nb * (4ull << g.kb_log)) + 256u;
    return g;
}

__global__ __launch_bounds__(kTileThreads) void k_slice_tiles(const uint32_t* __restrict__ keys, uint64_t n,
                                                              uint32_t K, uint32_t kb_log, uint32_t nb,
                                                              uint32_t* __restrict__ skeys,
                                                              uint32_t* __restrict__ toff, uint32_t* __restrict__ err)
{
    __shared__ uint32_t s_keys[kTile];
    __shared__ uint32_t s_hist[kMaxBuckets + 1];
    __shared__ uint32_t s_scan[16];
    const uint64_t t = blockIdx.x;
    const uint64_t t0 = t * kTile;
    const uint32_t tn = n - t0 < kTile ? (uint32_t)(n - t0) : kTile;
    for (uint32_t u = threadIdx.x; u <= nb; u += kTileThreads) s_hist[u] = 0;
    __syncthreads();
    constexpr uint32_t kPerT = kTile / kTileThreads;
    uint32_t kv[kPerT], slot[kPerT];
    bool bad = false;
    const bool vec = tn == kTile && ((((uintptr_t)keys) >> 2) + t0) % 4u == 0;
    if (vec) {
        const uint4* k4 = reinterpret_cast<const uint4*>(keys + t0);
#pragma unroll
        for (uint32_t v = 0; v < kPerT / 4; ++v) {
            const uint4 q = k4[v * kTileThreads + threadIdx.x];  // coalesced; keys of one thread are spread
            kv[4 * v] = q.x, kv[4 * v + 1] = q.y, kv[4 * v + 2] = q.z, kv[4 * v + 3] = q.w;
        }
    } else {
#pragma unroll
        for (uint32_t v = 0; v < kPerT; ++v) {
            const uint32_t i = (v / 4) * (4 * kTileThreads) + threadIdx.x * 4 + (v % 4);
            kv[v] = i < tn ? keys[t0 + i] : 0xFFFFFFFFu;
        }
    }
#pragma unroll
    for (uint32_t v = 0; v < kPerT; ++v) {
        const uint32_t i = (v / 4) * (4 * kTileThreads) + threadIdx.x * 4 + (v % 4);
        const bool in = i < tn;
        const bool ok = in && kv[v] < K;
        bad |= in && !ok;
        slot[v] = ok ? atomicAdd(&s_hist[kv[v] >> kb_log], 1u) : 0xFFFFFFFFu;
    }
    __syncthreads();
    // exclusive scan of the bucket counts (nb <= 256: threads 0..255 hold one each)
    uint32_t tot;
    const uint32_t mine = threadIdx.x < nb ? s_hist[threadIdx.x] : 0u;
    const uint32_t ex = block_exscan_u32(mine, s_scan, &tot);
    __syncthreads();
    if (threadIdx.x < nb) s_hist[threadIdx.x] = ex;
    __syncthreads();
#pragma unroll
    for (uint32_t v = 0; v < kPerT; ++v)
        if (slot[v] != 0xFFFFFFFFu) s_keys[s_hist[kv[v] >> kb_log] + slot[v]] = kv[v];
    __syncthreads();
    uint32_t* __restrict__ out = skeys + t0;
    for (uint32_t i = threadIdx.x; i < tot; i += kTileThreads) out[i] = s_keys[i];
    uint32_t* __restrict__ to = toff + t * (nb + 1ull);
    for (uint32_t u = threadIdx.x; u < nb; u += kTileThreads) to[u] = s_hist[u];
    if (threadIdx.x == 0) to[nb] = tot;
    if (bad) atomicOr(err, CR_ERR_KEY_RANGE);
}

__global__ __launch_bounds__(kBinThreads) void k_slice_bins(const uint32_t* __restrict__ skeys,
                                                            const uint32_t* __restrict__ toff, uint64_t ntiles,
                                                            uint32_t K, uint32_t kb_log, uint32_t nb, uint32_t groups,
                                                            uint32_t* __restrict__ part)
{
    extern __shared__ uint32_t bins[];
    const uint32_t g = blockIdx.x, u = blockIdx.y;
    const uint32_t KB = 1u << kb_log;
    for (uint32_t i = threadIdx.x; i < KB; i += kBinThreads) bins[i] = 0;
    __syncthreads();
    const uint64_t tpg = (ntiles + groups - 1) / groups;
    const uint64_t ta = (uint64_t)g * tpg, tb = ta + tpg < ntiles ? ta + tpg : ntiles;
    const uint32_t wv = threadIdx.x >> 6, lane = lane_id();
    const uint32_t ubase = u << kb_log;
    for (uint64_t t = ta + wv; t < tb; t += kBinThreads / 64) {  // one tile's segment per wavefront
        const uint32_t s0 = toff[t * (nb + 1ull) + u], s1 = toff[t * (nb + 1ull) + u + 1];
        const uint32_t* __restrict__ seg = skeys + t * kTile;
        for (uint32_t i = s0 + lane; i < s1; i += 64) atomicAdd(&bins[seg[i] - ubase], 1u);
    }
    __syncthreads();
    const uint32_t lim = K - ubase < KB ? K - ubase : KB;
    uint32_t* __restrict__ pr = part + ((uint64_t)g * nb + u) * KB;
    for (uint32_t i = threadIdx.x; i < lim; i += kBinThreads) pr[i] = bins[i];
}

__global__ __launch_bounds__(256) void k_slice_reduce(const uint32_t* __restrict__ part, uint32_t K, uint32_t kb_log,
                                                      uint32_t nb, uint32_t groups, uint32_t* __restrict__ counts)
{
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    const uint64_t row = (uint64_t)nb << kb_log;  // one group's partial row
    for (uint64_t b = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; b < K; b += stride) {
        uint32_t s = counts[b];
        for (uint32_t g = 0; g < groups; ++g) s += part[g * row + b];
        counts[b] = s;
    }
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

extern "C" size_t cr_count_slice_workspace_bytes(uint64_t n, uint32_t num_keys)
{
    using namespace cr;
    if (num_keys == 0) return 256;
    return (size_t)slice_geom(n, num_keys, device_max_lds() - 512, device_cus()).bytes;
}

extern "C" cr_status cr_count_slice(const uint32_t* keys, uint64_t n, uint32_t num_keys, uint32_t* counts,
                                    uint32_t* err, void* ws, size_t ws_bytes, void* stream)
{
    using namespace cr;
    if (num_keys == 0 || num_keys == 0xFFFFFFFFu || !counts || !err) return CR_EINVAL;
    if (n == 0) return CR_OK;
    if (!keys || ((uintptr_t)keys & 3u) || !ws) return CR_EINVAL;
    const int max_lds = device_max_lds() - 512;
    const SliceGeom g = slice_geom(n, num_keys, max_lds, device_cus());
    if (g.nb > kMaxBuckets || g.ntiles > 0x7FFFFFFFull || n >= 0xFFFFFFFFull) return CR_EINVAL;
    if (ws_bytes < g.bytes) return CR_ESIZE;
    uint8_t* base = reinterpret_cast<uint8_t*>(((uintptr_t)ws + 255) & ~(uintptr_t)255);
    uint32_t* skeys = reinterpret_cast<uint32_t*>(base + g.keys_off);
    uint32_t* toff = reinterpret_cast<uint32_t*>(base + g.toff_off);
    uint32_t* part = reinterpret_cast<uint32_t*>(base + g.part_off);
    const hipStream_t st = as_stream(stream);
    const uint32_t lds = 4u << g.kb_log;
    (void)hipGetLastError();
    if (hipFuncSetAttribute((const void*)k_slice_bins, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
        hipSuccess)
        return CR_EHIP;
    hipLaunchKernelGGL(k_slice_tiles, dim3((uint32_t)g.ntiles), dim3(kTileThreads), 0, st, keys, n, num_keys, g.kb_log,
                       g.nb, skeys, toff, err);
    hipLaunchKernelGGL(k_slice_bins, dim3(g.groups, g.nb), dim3(kBinThreads), (size_t)lds, st, skeys, toff, g.ntiles,
                       num_keys, g.kb_log, g.nb, g.groups, part);
    hipLaunchKernelGGL(k_slice_reduce, dim3(1024), dim3(256), 0, st, part, num_keys, g.kb_log, g.nb, g.groups, counts);
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}
