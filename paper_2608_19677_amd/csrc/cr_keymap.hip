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
//                is skipped when the slot already holds a smaller index;
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

struct KmTable {
    uint32_t* ids;    // [S] CR_NO_KEY when empty
    uint32_t* first;  // [S] first request index of the slot's id
    uint32_t* dense;  // [S] dense index (valid after the build)
};

inline KmTable km_table(void* t, uint32_t S)
{
    uint32_t* p = reinterpret_cast<uint32_t*>(t);
    return KmTable{p, p + S, p + 2u * (uint64_t)S};
}

__global__ __launch_bounds__(kKmThreads) void k_km_init(KmTable tab, uint32_t S, uint32_t* __restrict__ bitmap,
                                                        uint64_t words)
{
    const uint64_t stride = (uint64_t)gridDim.x * kKmThreads;
    for (uint64_t x = (uint64_t)blockIdx.x * kKmThreads + threadIdx.x; x < S; x += stride) {
        tab.ids[x] = CR_NO_KEY;
        tab.first[x] = 0xFFFFFFFFu;
        tab.dense[x] = CR_NO_KEY;
    }
    for (uint64_t x = (uint64_t)blockIdx.x * kKmThreads + threadIdx.x; x < words; x += stride) bitmap[x] = 0;
}

// Slot of id in the table, or S when the id is absent (insert = false) or the table is full.
template <bool kInsert>
__device__ __forceinline__ uint32_t km_probe(const KmTable& tab, uint32_t S, uint32_t id)
{
    uint32_t h = km_hash(id) & (S - 1u);
    for (uint32_t step = 0; step < S; ++step) {
        uint32_t cur = tab.ids[h];
        if (cur == id) return h;
        if (cur == CR_NO_KEY) {
            if (!kInsert) return S;
            cur = atomicCAS(tab.ids + h, CR_NO_KEY, id);
            if (cur == CR_NO_KEY || cur == id) return h;
        }
        h = (h + 1u) & (S - 1u);
    }
    return S;
}

__global__ __launch_bounds__(kKmThreads) void k_km_insert(const uint32_t* __restrict__ ids, uint64_t n, KmTable tab,
                                                          uint32_t S, uint32_t* __restrict__ err)
{
    const uint64_t stride = (uint64_t)gridDim.x * kKmThreads;
    uint32_t e = 0;
    for (uint64_t i = (uint64_t)blockIdx.x * kKmThreads + threadIdx.x; i < n; i += stride) {
        const uint32_t id = ids[i];
        if (id == CR_NO_KEY) {
            e |= CR_ERR_KEY_RANGE;
            continue;
        }
        const uint32_t h = km_probe<true>(tab, S, id);
        if (h == S) {
            e |= CR_ERR_KEYMAP_FULL;
            continue;
        }
        if (__hip_atomic_load(tab.first + h, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) > (uint32_t)i)
            atomicMin(tab.first + h, (uint32_t)i);
    }
    if (e) atomicOr(err, e);
}

__global__ __launch_bounds__(kKmThreads) void k_km_mark(KmTable tab, uint32_t S, uint32_t* __restrict__ bitmap)
{
    const uint32_t x = blockIdx.x * kKmThreads + threadIdx.x;
    if (x >= S || tab.ids[x] == CR_NO_KEY) return;
    const uint32_t f = tab.first[x];
    atomicOr(bitmap + (f >> 5), 1u << (f & 31u));
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
    if (x >= S || tab.ids[x] == CR_NO_KEY) return;
    const uint32_t f = tab.first[x];
    tab.dense[x] = prefix[f >> 5] + __popc(bitmap[f >> 5] & ((1u << (f & 31u)) - 1u));
}

__global__ __launch_bounds__(kKmThreads) void k_km_lookup(const uint32_t* __restrict__ ids, uint64_t n, KmTable tab,
                                                          uint32_t S, uint32_t* __restrict__ dense)
{
    const uint64_t stride = (uint64_t)gridDim.x * kKmThreads;
    for (uint64_t i = (uint64_t)blockIdx.x * kKmThreads + threadIdx.x; i < n; i += stride) {
        const uint32_t id = ids[i];
        const uint32_t h = id == CR_NO_KEY ? S : km_probe<false>(tab, S, id);
        dense[i] = h < S ? tab.dense[h] : CR_NO_KEY;
    }
}

__global__ __launch_bounds__(kKmThreads) void k_km_scatter(KmTable tab, uint32_t S, const uint32_t* __restrict__ ids,
                                                           const uint32_t* __restrict__ values, uint64_t m,
                                                           uint32_t* __restrict__ out, uint32_t out_len)
{
    const uint64_t stride = (uint64_t)gridDim.x * kKmThreads;
    for (uint64_t x = (uint64_t)blockIdx.x * kKmThreads + threadIdx.x; x < m; x += stride) {
        const uint32_t id = ids[x];
        const uint32_t h = id == CR_NO_KEY ? S : km_probe<false>(tab, S, id);
        if (h < S) {
            const uint32_t k = tab.dense[h];
            if (k < out_len) out[k] = values[x];
        }
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
    return (size_t)3u * cr::km_slots(capacity) * sizeof(uint32_t);
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
    if (((uintptr_t)table & 3u) || ((uintptr_t)ws & 3u) || ((uintptr_t)ids & 3u)) return CR_EINVAL;
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
    if (n) hipLaunchKernelGGL(k_km_insert, dim3(km_grid(n)), dim3(kKmThreads), 0, st, ids, n, tab, S, err);
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
    (void)hipGetLastError();
    hipLaunchKernelGGL(k_km_lookup, dim3(km_grid(n)), dim3(kKmThreads), 0, as_stream(stream), ids, n,
                       km_table(const_cast<void*>(table), S), S, dense);
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
