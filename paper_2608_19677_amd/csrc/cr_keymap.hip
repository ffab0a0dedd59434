// Opaque-key directory (Appendix A.2 "Data handling": the planner needs only {(b, lambda_b)}
// and b may be salted or ephemeral; Section 2.1: the summaries carry opaque keys).
//
// Counting into dense per-key rows needs every opaque 32-bit id mapped to a dense index.
// The index of an id is the rank of its first occurrence among the distinct ids of the
// build stream, which no scheduling can change:
//   k_km_init    clears an open-addressing table of S = 2^s >= 2 * capacity slots and the
//                first-occurrence bitmap;
//   k_km_insert  inserts every request's id (linear probing, a compare-and-swap claims a
//                slot) and keeps the id's first request index with an atomic minimum, which
//                is skipped when the slot already holds a smaller index (the stream goes in
//                ranges of growing length so that frequent ids are settled early);
//   k_km_mark    sets bit `first` of the bitmap for every occupied slot;
//   k_km_sums / k_km_scan_sums / k_km_assign
//                exclusive prefix of the bitmap's popcounts (per block, then across blocks),
//                so an id's dense index is the number of first occurrences before its own.
// Lookups probe the same table; an id the table does not hold maps to CR_NO_KEY.
#include "cr_common.h"

namespace cr {
namespace {

constexpr uint32_t kKmThreads = 256;
constexpr uint32_t kKmWordsPerBlock = 4096;  // bitmap words summed per block
constexpr uint32_t kKmMaxSums = 1u << 20;     // blocks of bitmap words the scan handles

__host__ __device__ __forceinline__ uint32_t km_slots(uint32_t capacity)
{
    uint32_t s = 64;
    while (s < 2u * capacity) s <<= 1;
    return s;
}

__device__ __forceinline__ uint32_t km_hash(uint32_t id) { return fmix32(id ^ 0x2545F491u); }

// One slot per 16 bytes, {id, first request index, dense index, unused}, so that a probe
// is one cache-line access. CR_NO_KEY marks an empty slot.
struct KmTable {
    uint4* slot;  // [S]
};

inline KmTable km_table(void* t, uint32_t) { return KmTable{reinterpret_cast<uint4*>(t)}; }

__global__ __launch_bounds__(kKmThreads) void k_km_init(KmTable tab, uint32_t S, uint32_t* __restrict__ bitmap,
                                                        uint64_t words)
{
    const uint64_t stride = (uint64_t)gridDim.x * kKmThreads;
    for (uint64_t x = (uint64_t)blockIdx.x * kKmThreads + threadIdx.x; x < S; x += stride)
        tab.slot[x] = make_uint4(CR_NO_KEY, 0xFFFFFFFFu, CR_NO_KEY, 0u);
    for (uint64_t x = (uint64_t)blockIdx.x * kKmThreads + threadIdx.x; x < words; x += stride) bitmap[x] = 0;
}

// Slot of id in the table, or S when the id is absent (insert = false) or the table is full;
// *v receives the slot's contents as read (plain loads: a slot's id only ever goes from
// empty to one id and its first index only decreases, so a stale copy can only cost an
// extra compare-and-swap or atomic, never a wrong result).
template <bool kInsert>
__device__ __forceinline__ uint32_t km_probe(const KmTable& tab, uint32_t S, uint32_t id, uint4* v)
{
    uint32_t h = km_hash(id) & (S - 1u);
    for (uint32_t step = 0; step < S; ++step) {
        uint4 c = tab.slot[h];
        if (c.x == id) {
            *v = c;
            return h;
        }
        if (c.x == CR_NO_KEY) {
            if (!kInsert) return S;
            const uint32_t prev = atomicCAS(&tab.slot[h].x, CR_NO_KEY, id);
            if (prev == CR_NO_KEY || prev == id) {
                *v = make_uint4(id, prev == id ? c.y : 0xFFFFFFFFu, CR_NO_KEY, 0u);
                return h;
            }
        }
        h = (h + 1u) & (S - 1u);
    }
    return S;
}

// Requests [lo, hi), kKmPer consecutive ones per thread with their loads in flight
// together. The host runs the stream in ranges of geometrically growing length: a
// frequent id gets its first index from the first short range, so the many later
// requests for it see a smaller index already and issue no atomic (same-address atomics
// are serialised at the cache).
constexpr uint32_t kKmPer = 4;

__global__ __launch_bounds__(kKmThreads) void k_km_insert(const uint32_t* __restrict__ ids, uint64_t lo, uint64_t hi,
                                                          KmTable tab, uint32_t S, uint32_t* __restrict__ err)
{
    const uint64_t i0 = lo + ((uint64_t)blockIdx.x * kKmThreads + threadIdx.x) * kKmPer;
    if (i0 >= hi) return;
    uint32_t id[kKmPer];
#pragma unroll
    for (uint32_t t = 0; t < kKmPer; ++t) id[t] = i0 + t < hi ? ids[i0 + t] : CR_NO_KEY;
    uint32_t e = 0;
#pragma unroll
    for (uint32_t t = 0; t < kKmPer; ++t) {
        if (id[t] == CR_NO_KEY) {
            e |= i0 + t < hi ? CR_ERR_KEY_RANGE : 0u;
            continue;
        }
        uint4 v;
        const uint32_t h = km_probe<true>(tab, S, id[t], &v);
        if (h == S) {
            e |= CR_ERR_KEYMAP_FULL;
            continue;
        }
        if (v.y > (uint32_t)(i0 + t)) atomicMin(&tab.slot[h].y, (uint32_t)(i0 + t));
    }
    if (e) atomicOr(err, e);
}

__global__ __launch_bounds__(kKmThreads) void k_km_mark(KmTable tab, uint32_t S, uint32_t* __restrict__ bitmap)
{
    const uint32_t x = blockIdx.x * kKmThreads + threadIdx.x;
    if (x >= S) return;
    const uint4 c = tab.slot[x];
    if (c.x == CR_NO_KEY) return;
    atomicOr(bitmap + (c.y >> 5), 1u << (c.y & 31u));
}

__device__ __forceinline__ uint32_t block_sum_u32(uint32_t v, uint32_t* sh)
{
    uint32_t total;
    (void)block_exscan_u32(v, sh, &total);
    return total;
}

// Popcount of every block's share of bitmap words.
__global__ __launch_bounds__(kKmThreads) void k_km_sums(const uint32_t* __restrict__ bitmap, uint64_t words,
                                                        uint32_t* __restrict__ sums)
{
    __shared__ uint32_t sh[kKmThreads / 64];
    const uint64_t w0 = (uint64_t)blockIdx.x * kKmWordsPerBlock;
    uint32_t c = 0;
    for (uint32_t t = threadIdx.x; t < kKmWordsPerBlock; t += kKmThreads)
        if (w0 + t < words) c += __popc(bitmap[w0 + t]);
    const uint32_t total = block_sum_u32(c, sh);
    if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// Exclusive scan of the block sums in place (one block); total distinct ids to num_keys.
__global__ __launch_bounds__(1024) void k_km_scan_sums(uint32_t* __restrict__ sums, uint32_t nsums,
                                                       uint32_t capacity, uint32_t* __restrict__ num_keys,
                                                       uint32_t* __restrict__ err)
{
    __shared__ uint32_t sh[1024 / 64];
    uint32_t carry = 0;
    for (uint32_t b0 = 0; b0 < nsums; b0 += 1024) {
        const uint32_t x = b0 + threadIdx.x;
        const uint32_t v = x < nsums ? sums[x] : 0u;
        uint32_t total;
        const uint32_t ex = block_exscan_u32(v, sh, &total);
        if (x < nsums) sums[x] = carry + ex;
        carry += total;
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        num_keys[0] = carry;
        if (carry > capacity) atomicOr(err, CR_ERR_KEYMAP_FULL);
    }
}

// Exclusive prefix of popcounts per bitmap word (block offset + scan within the block).
__global__ __launch_bounds__(kKmThreads) void k_km_prefix(const uint32_t* __restrict__ bitmap, uint64_t words,
                                                          const uint32_t* __restrict__ sums,
                                                          uint32_t* __restrict__ prefix)
{
    __shared__ uint32_t sh[kKmThreads / 64];
    const uint64_t w0 = (uint64_t)blockIdx.x * kKmWordsPerBlock;
    uint32_t carry = sums[blockIdx.x];
    for (uint32_t t0 = 0; t0 < kKmWordsPerBlock; t0 += kKmThreads) {
        const uint64_t w = w0 + t0 + threadIdx.x;
        const uint32_t c = w < words ? __popc(bitmap[w]) : 0u;
        uint32_t total;
        const uint32_t ex = block_exscan_u32(c, sh, &total);
        if (w < words) prefix[w] = carry + ex;
        carry += total;
        __syncthreads();
    }
}

__global__ __launch_bounds__(kKmThreads) void k_km_assign(KmTable tab, uint32_t S, const uint32_t* __restrict__ bitmap,
                                                          const uint32_t* __restrict__ prefix)
{
    const uint32_t x = blockIdx.x * kKmThreads + threadIdx.x;
    if (x >= S) return;
    const uint4 c = tab.slot[x];
    if (c.x == CR_NO_KEY) return;
    const uint32_t f = c.y;
    tab.slot[x].z = prefix[f >> 5] + __popc(bitmap[f >> 5] & ((1u << (f & 31u)) - 1u));
}

__global__ __launch_bounds__(kKmThreads) void k_km_lookup(const uint32_t* __restrict__ ids, uint64_t n, KmTable tab,
                                                          uint32_t S, uint32_t* __restrict__ dense)
{
    const uint64_t i0 = ((uint64_t)blockIdx.x * kKmThreads + threadIdx.x) * kKmPer;
    if (i0 >= n) return;
    uint32_t id[kKmPer], d[kKmPer];
#pragma unroll
    for (uint32_t t = 0; t < kKmPer; ++t) id[t] = i0 + t < n ? ids[i0 + t] : CR_NO_KEY;
#pragma unroll
    for (uint32_t t = 0; t < kKmPer; ++t) {
        uint4 v;
        const uint32_t h = id[t] == CR_NO_KEY ? S : km_probe<false>(tab, S, id[t], &v);
        d[t] = h < S ? v.z : CR_NO_KEY;
    }
#pragma unroll
    for (uint32_t t = 0; t < kKmPer; ++t)
        if (i0 + t < n) dense[i0 + t] = d[t];
}

__global__ __launch_bounds__(kKmThreads) void k_km_scatter(KmTable tab, uint32_t S, const uint32_t* __restrict__ ids,
                                                           const uint32_t* __restrict__ values, uint64_t m,
                                                           uint32_t* __restrict__ out, uint32_t out_len)
{
    const uint64_t stride = (uint64_t)gridDim.x * kKmThreads;
    for (uint64_t x = (uint64_t)blockIdx.x * kKmThreads + threadIdx.x; x < m; x += stride) {
        const uint32_t id = ids[x];
        uint4 v;
        const uint32_t h = id == CR_NO_KEY ? S : km_probe<false>(tab, S, id, &v);
        if (h < S && v.z < out_len) out[v.z] = values[x];
    }
}

inline uint32_t km_grid(uint64_t items)
{
    const uint64_t b = (items + kKmThreads - 1) / kKmThreads;
    const uint64_t cap = (uint64_t)device_cus() * 16u;
    return (uint32_t)(b < 1 ? 1 : (b > cap ? cap : b));
}

inline uint64_t km_words(uint64_t n) { return (n + 31u) / 32u; }
inline uint64_t km_nsums(uint64_t n) { return (km_words(n) + kKmWordsPerBlock - 1) / kKmWordsPerBlock; }

}  // namespace
}  // namespace cr

extern "C" size_t cr_keymap_bytes(uint32_t capacity)
{
    return (size_t)cr::km_slots(capacity) * sizeof(uint4);
}

extern "C" size_t cr_keymap_workspace_bytes(uint64_t n)
{
    const uint64_t words = cr::km_words(n);
    return (size_t)((2u * words + cr::km_nsums(n) + 64u) * sizeof(uint32_t));
}

extern "C" cr_status cr_keymap_build(const uint32_t* ids, uint64_t n, uint32_t capacity, void* table,
                                     size_t table_bytes, void* ws, size_t ws_bytes, uint32_t* num_keys,
                                     uint32_t* err, void* stream)
{
    using namespace cr;
    if (capacity == 0 || capacity > CR_KEYMAP_MAX_CAPACITY || !table || !ws || !num_keys || !err ||
        (n > 0 && !ids) || n >= 0xFFFFFFFFull)
        return CR_EINVAL;
    if (table_bytes < cr_keymap_bytes(capacity) || ws_bytes < cr_keymap_workspace_bytes(n)) return CR_ESIZE;
    if (((uintptr_t)table & 15u) || ((uintptr_t)ws & 3u) || ((uintptr_t)ids & 3u)) return CR_EINVAL;
    const uint64_t words = km_words(n), nsums = km_nsums(n);
    if (nsums > kKmMaxSums) return CR_EINVAL;
    const uint32_t S = km_slots(capacity);
    const KmTable tab = km_table(table, S);
    uint32_t* bitmap = reinterpret_cast<uint32_t*>(ws);
    uint32_t* prefix = bitmap + words;
    uint32_t* sums = prefix + words;
    const hipStream_t st = as_stream(stream);
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_km_init, dim3(km_grid(words > S ? words : S)), dim3(kKmThreads), 0, st, tab, S, bitmap, words);
    for (uint64_t lo = 0, len = (n + 255) / 256; lo < n; lo += len, len *= 4) {
        const uint64_t hi = n - lo < len ? n : lo + len;
        const uint64_t threads = (hi - lo + kKmPer - 1) / kKmPer;
        hipLaunchKernelGGL(k_km_insert, dim3((uint32_t)((threads + kKmThreads - 1) / kKmThreads)), dim3(kKmThreads), 0,
                           st, ids, lo, hi, tab, S, err);
    }
    hipLaunchKernelGGL(k_km_mark, dim3((S + kKmThreads - 1) / kKmThreads), dim3(kKmThreads), 0, st, tab, S, bitmap);
    if (nsums) {
        hipLaunchKernelGGL(k_km_sums, dim3((uint32_t)nsums), dim3(kKmThreads), 0, st, bitmap, words, sums);
    }
    hipLaunchKernelGGL(k_km_scan_sums, dim3(1), dim3(1024), 0, st, sums, (uint32_t)nsums, capacity, num_keys, err);
    if (nsums) {
        hipLaunchKernelGGL(k_km_prefix, dim3((uint32_t)nsums), dim3(kKmThreads), 0, st, bitmap, words, sums, prefix);
    }
    hipLaunchKernelGGL(k_km_assign, dim3((S + kKmThreads - 1) / kKmThreads), dim3(kKmThreads), 0, st, tab, S, bitmap,
                       prefix);
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}

extern "C" cr_status cr_keymap_lookup(const void* table, size_t table_bytes, uint32_t capacity, const uint32_t* ids,
                                      uint64_t n, uint32_t* dense, void* stream)
{
    using namespace cr;
    if (capacity == 0 || capacity > CR_KEYMAP_MAX_CAPACITY || !table || (n > 0 && (!ids || !dense))) return CR_EINVAL;
    if (table_bytes < cr_keymap_bytes(capacity)) return CR_ESIZE;
    if (n == 0) return CR_OK;
    const uint32_t S = km_slots(capacity);
    const uint64_t threads = (n + kKmPer - 1) / kKmPer;
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_km_lookup, dim3((uint32_t)((threads + kKmThreads - 1) / kKmThreads)), dim3(kKmThreads), 0,
                       as_stream(stream), ids, n, km_table(const_cast<void*>(table), S), S, dense);
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}

extern "C" cr_status cr_keymap_scatter(const void* table, size_t table_bytes, uint32_t capacity, const uint32_t* ids,
                                       const uint32_t* values, uint64_t m, uint32_t* out, uint32_t out_len,
                                       void* stream)
{
    using namespace cr;
    if (capacity == 0 || capacity > CR_KEYMAP_MAX_CAPACITY || !table || (m > 0 && (!ids || !values || !out)))
        return CR_EINVAL;
    if (table_bytes < cr_keymap_bytes(capacity)) return CR_ESIZE;
    if (m == 0) return CR_OK;
    const uint32_t S = km_slots(capacity);
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_km_scatter, dim3(km_grid(m)), dim3(kKmThreads), 0, as_stream(stream),
                       km_table(const_cast<void*>(table), S), S, ids, values, m, out, out_len);
    return hipGetLastError() == hipSuccess ? CR_OK : CR_EHIP;
}
