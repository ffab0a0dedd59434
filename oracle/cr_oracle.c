/*
 * CacheRoute CPU oracle -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT PATH.
 *
 * A plain, slow, single-threaded C11 statement of what the periodic routing
 * planner and its shadow replay compute, written from the paper
 * ("CacheRoute: Planned Prefix-Affinity Routing for Large-Scale LLM Serving"):
 *   - per-key rates: the planner's only workload input is {(b, lambda_b)}
 *     (Section 3.1 Algorithm 1 inputs; Appendix A.2);
 *   - load-based assignment count k_b = max(1, ceil(lambda_b / q_cap)) (Eq. 1);
 *   - warm-set admission: keys in decreasing rate, admitted while the sum of
 *     k_b stays within C = R W slots (Section 3.1 "Warm-set admission",
 *     Algorithm 1);
 *   - LPT placement from the expected cold-tail share, k_b distinct
 *     least-loaded destinations per admitted key, each charged lambda_b / k_b
 *     (Section 3.1 "Placement and dispatch", Algorithm 1);
 *   - dispatch through the fixed table, cold tail by power-of-two choices
 *     (Section 3.1 "Placement and dispatch"; Fig. 1);
 *   - shadow replay of a plan against per-destination prefix caches shared by
 *     admitted and cold traffic (Section 3.2), modelled as an LRU of W
 *     whole-prefix slots per destination (the equal-slot model of Section 3.1).
 *
 * Readings where the paper is silent are listed in the design notes; the
 * ones that fix results are restated at each function below.
 *
 * Only tests/, __graft_entry__.smoke() and bench.py's CPU-baseline leg may load
 * this library. It shares no source, header or helper with the device library.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fPIC -shared cr_oracle.c
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define CRO_EMPTY 0xFFFFFFFFu

/* Offsets must start at 0, end at n and never decrease. */
static int cro_check_offsets(const uint64_t* off, uint32_t J, uint64_t n)
{
    if (J == 0 || off == NULL || off[0] != 0 || off[J] != n) return -1;
    for (uint32_t j = 0; j < J; ++j)
        if (off[j] > off[j + 1]) return -1;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Rates. The rate of key b over window j is its request count there; the    */
/* common factor 1/window-length never changes a decision, so the oracle     */
/* works in requests per window (Algorithm 1 inputs; Appendix A.2).          */
/* counts[j*K + b] += #{ i in [off[j], off[j+1]) : keys[i] == b }.           */
/* A key >= K is not counted; the number of such requests goes to *n_bad.    */
/* ------------------------------------------------------------------------ */
int cro_count_rates(const uint32_t* keys, uint64_t n, const uint64_t* offsets, uint32_t J,
                    uint32_t K, uint32_t* counts, uint64_t* n_bad)
{
    if (cro_check_offsets(offsets, J, n) || K == 0) return -1;
    uint64_t bad = 0;
    for (uint32_t j = 0; j < J; ++j) {
        uint32_t* row = counts + (uint64_t)j * K;
        for (uint64_t i = offsets[j]; i < offsets[j + 1]; ++i) {
            uint32_t b = keys[i];
            if (b < K) row[b] += 1;
            else bad += 1;
        }
    }
    if (n_bad) *n_bad += bad;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Eq. 1 with q_cap = q_num / q_den requests per window, in exact integers:  */
/* k = max(1, ceil(c * q_den / q_num)). A key cannot use more than R         */
/* distinct destinations, so k is clamped to R and the clamp is reported.    */
/* ------------------------------------------------------------------------ */
uint32_t cro_kb(uint32_t c, uint64_t q_num, uint64_t q_den, uint32_t R, uint32_t* clamped)
{
    uint64_t num = (uint64_t)c * q_den;          /* c < 2^32, q_den < 2^31 */
    uint64_t k = num / q_num + (num % q_num != 0);
    if (k < 1) k = 1;
    if (k > R) {
        k = R;
        if (clamped) *clamped += 1;
    }
    return (uint32_t)k;
}

typedef struct { uint32_t c, b; } cro_rate;

/* Decreasing rate; equal rates in increasing key id. */
static int cro_by_rate(const void* x, const void* y)
{
    const cro_rate* p = (const cro_rate*)x;
    const cro_rate* q = (const cro_rate*)y;
    if (p->c != q->c) return p->c > q->c ? -1 : 1;
    if (p->b != q->b) return p->b < q->b ? -1 : 1;
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Admission (Algorithm 1: compute k_b, sort keys by decreasing rate, admit  */
/* while the running sum of k_b is at most C = R W).                         */
/*  - keys with zero count in the window are absent from telemetry and are   */
/*    never admitted;                                                        */
/*  - "admit while" is a prefix: the first key that does not fit ends it;    */
/*  - cold = window requests not carried by an admitted key.                 */
/* adm_keys/adm_k have room for R*W entries.                                 */
/* ------------------------------------------------------------------------ */
int cro_admit(const uint32_t* counts_row, uint32_t K, uint32_t R, uint32_t W, uint64_t n_window,
              uint64_t q_num, uint64_t q_den, uint32_t* adm_keys, uint32_t* adm_k, uint32_t* A,
              uint64_t* cold, uint32_t* n_clamped)
{
    if (R == 0 || W == 0 || q_den == 0 || K == 0) return -1;
    uint64_t C = (uint64_t)R * W;
    cro_rate* v = (cro_rate*)malloc(sizeof(cro_rate) * (size_t)K);
    if (!v) return -2;
    uint32_t nnz = 0;
    uint64_t total = 0;
    for (uint32_t b = 0; b < K; ++b) {
        total += counts_row[b];
        if (counts_row[b] > 0) {
            v[nnz].c = counts_row[b];
            v[nnz].b = b;
            ++nnz;
        }
    }
    if (total != n_window || (nnz > 0 && q_num == 0)) {
        free(v);
        return -1;
    }
    qsort(v, nnz, sizeof(cro_rate), cro_by_rate);
    uint64_t used = 0, carried = 0;
    uint32_t a = 0, clamped = 0;
    for (uint32_t t = 0; t < nnz; ++t) {
        uint32_t k = cro_kb(v[t].c, q_num, q_den, R, &clamped);
        if (used + k > C) break;
        used += k;
        carried += v[t].c;
        adm_keys[a] = v[t].b;
        adm_k[a] = k;
        ++a;
    }
    *A = a;
    *cold = n_window - carried;
    if (n_clamped) *n_clamped = clamped;
    free(v);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* LPT placement (Algorithm 1 placement loop; Section 3.1).                  */
/*  - every destination starts at the expected cold-tail share cold / R      */
/*    (power-of-two choices spreads the cold tail evenly in expectation);    */
/*  - admitted keys are visited in admission order; key b with count c and   */
/*    k copies takes the k destinations with the smallest (L[r], r), listed  */
/*    in that order, and each of them is charged c / k;                      */
/*  - all arithmetic on L is IEEE double, one rounding per add/divide.       */
/* members[member_off[a] .. member_off[a+1]) is T(adm_keys[a]).             */
/* ------------------------------------------------------------------------ */
int cro_place_lpt(const uint32_t* adm_keys, const uint32_t* adm_k, uint32_t A,
                  const uint32_t* counts_row, uint32_t R, uint64_t cold, uint16_t* members,
                  uint32_t* member_off, double* L)
{
    if (R == 0 || R > 65535) return -1;
    unsigned char* taken = (unsigned char*)calloc(R, 1);
    if (!taken) return -2;
    double init = (double)cold / (double)R;
    for (uint32_t r = 0; r < R; ++r) L[r] = init;
    uint32_t off = 0;
    for (uint32_t a = 0; a < A; ++a) {
        uint32_t k = adm_k[a];
        if (k < 1 || k > R) {
            free(taken);
            return -1;
        }
        double x = (double)counts_row[adm_keys[a]] / (double)k;
        member_off[a] = off;
        for (uint32_t t = 0; t < k; ++t) {
            int64_t best = -1;
            for (uint32_t r = 0; r < R; ++r)
                if (!taken[r] && (best < 0 || L[r] < L[best])) best = r;
            members[off + t] = (uint16_t)best;
            taken[best] = 1;
        }
        for (uint32_t t = 0; t < k; ++t) {
            uint32_t r = members[off + t];
            L[r] = L[r] + x;
            taken[r] = 0;
        }
        off += k;
    }
    member_off[A] = off;
    free(taken);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Counter-based hash of (seed, global request index) feeding the per-      */
/* request random choices: the 32-bit finalizer of MurmurHash3 (Appleby,     */
/* public domain), applied twice.                                            */
/* ------------------------------------------------------------------------ */
uint32_t cro_fmix32(uint32_t x)
{
    x ^= x >> 16;
    x *= 0x85EBCA6Bu;
    x ^= x >> 13;
    x *= 0xC2B2AE35u;
    x ^= x >> 16;
    return x;
}

uint32_t cro_hash(uint64_t seed, uint64_t i)
{
    uint32_t s = cro_fmix32((uint32_t)seed ^ (uint32_t)(seed >> 32) ^ 0x9E3779B9u);
    return cro_fmix32((uint32_t)i ^ cro_fmix32((uint32_t)(i >> 32) ^ s));
}

/* ------------------------------------------------------------------------ */
/* Hash placement, the "random placement" stages of the component ablation */
/* (Section 5.2, 8B component ablation table). Key b's k members are a      */
/* uniformly random k-subset of the destinations: the k smallest (u, r) of  */
/* u(b, r) = fmix32(fmix32(b ^ t) ^ r), t = fmix32(seed ^ 0x7F4A7C15),      */
/* listed in that order. Loads start at cold / R and each member is charged */
/* c / k in admission order, as in LPT; only the choice of members differs. */
/* ------------------------------------------------------------------------ */
uint32_t cro_place_u(uint32_t seed, uint32_t b, uint32_t r)
{
    uint32_t t = cro_fmix32(seed ^ 0x7F4A7C15u);
    return cro_fmix32(cro_fmix32(b ^ t) ^ r);
}

int cro_place_hash(const uint32_t* adm_keys, const uint32_t* adm_k, uint32_t A,
                   const uint32_t* counts_row, uint32_t R, uint64_t cold, uint32_t seed,
                   uint16_t* members, uint32_t* member_off, double* L)
{
    if (R == 0 || R > 65535) return -1;
    unsigned char* taken = (unsigned char*)calloc(R, 1);
    if (!taken) return -2;
    double init = (double)cold / (double)R;
    for (uint32_t r = 0; r < R; ++r) L[r] = init;
    uint32_t off = 0;
    for (uint32_t a = 0; a < A; ++a) {
        uint32_t b = adm_keys[a], k = adm_k[a];
        if (k < 1 || k > R) {
            free(taken);
            return -1;
        }
        double x = (double)counts_row[b] / (double)k;
        member_off[a] = off;
        for (uint32_t t = 0; t < k; ++t) {
            int64_t best = -1;
            uint32_t ubest = 0;
            for (uint32_t r = 0; r < R; ++r) {
                if (taken[r]) continue;
                uint32_t u = cro_place_u(seed, b, r);
                if (best < 0 || u < ubest) {
                    best = r;
                    ubest = u;
                }
            }
            members[off + t] = (uint16_t)best;
            taken[best] = 1;
        }
        for (uint32_t t = 0; t < k; ++t) {
            uint32_t r = members[off + t];
            L[r] = L[r] + x;
            taken[r] = 0;
        }
        off += k;
    }
    member_off[A] = off;
    free(taken);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Dispatch through one fixed plan (Section 3.1 "Placement and dispatch";   */
/* Fig. 1). Request i has global index first_index + i and h = hash(seed,   */
/* that index). Order-independent reading:                                   */
/*  - admitted key with members M (k of them): M[((h >> 16) * k) >> 16];     */
/*  - otherwise power-of-two choices over all destinations with two draws    */
/*    d1 = ((h & 0xFFFF) * R) >> 16 and d2 = ((h >> 16) * R) >> 16, compared */
/*    on the plan's interval-start loads L: d2 if L[d2] < L[d1], else d1.    */
/* A key >= K is routed as cold and counted in *n_bad.                       */
/* ------------------------------------------------------------------------ */
int cro_route(const uint32_t* keys, uint64_t n, uint64_t first_index, uint64_t seed, uint32_t K,
              uint32_t R, const uint32_t* adm_keys, uint32_t A, const uint32_t* member_off,
              const uint16_t* members, const double* L, uint16_t* dest, uint64_t* n_bad)
{
    if (R == 0 || R > 65535 || K == 0) return -1;
    int64_t* rank = (int64_t*)malloc(sizeof(int64_t) * (size_t)K);
    if (!rank) return -2;
    for (uint32_t b = 0; b < K; ++b) rank[b] = -1;
    for (uint32_t a = 0; a < A; ++a) rank[adm_keys[a]] = a;
    uint64_t bad = 0;
    for (uint64_t i = 0; i < n; ++i) {
        uint32_t h = cro_hash(seed, first_index + i);
        uint32_t b = keys[i];
        if (b < K && rank[b] >= 0) {
            uint32_t a = (uint32_t)rank[b];
            uint32_t k = member_off[a + 1] - member_off[a];
            uint32_t pick = (uint32_t)(((uint64_t)(h >> 16) * k) >> 16);
            dest[i] = members[member_off[a] + pick];
        } else {
            if (b >= K) bad += 1;
            uint32_t d1 = (uint32_t)(((uint64_t)(h & 0xFFFFu) * R) >> 16);
            uint32_t d2 = (uint32_t)(((uint64_t)(h >> 16) * R) >> 16);
            dest[i] = (uint16_t)(L[d2] < L[d1] ? d2 : d1);
        }
    }
    if (n_bad) *n_bad += bad;
    free(rank);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Live-load dispatch through one fixed plan over ONE control interval      */
/* (Section 3.1 "Placement and dispatch": during the interval admitted      */
/* traffic takes the least-loaded member of its fixed T(b), other traffic   */
/* takes power of two choices; Fig. 1). The load of a destination is read   */
/* as the number of requests of this interval dispatched to it so far       */
/* (zero when the interval starts), so every decision depends on all        */
/* earlier ones:                                                            */
/*  - admitted key with members M: the member with the smallest            */
/*    (load, destination) pair (k = 1: the only member);                    */
/*  - otherwise d1, d2 from hash(seed, first_index + i) as in cro_route,    */
/*    and d2 only if load[d2] < load[d1];                                   */
/*  - load[dest] += 1.                                                      */
/* A key >= K is dispatched as cold and counted in *n_bad.                  */
/* ------------------------------------------------------------------------ */
int cro_route_live(const uint32_t* keys, uint64_t n, uint64_t first_index, uint64_t seed, uint32_t K,
                   uint32_t R, const uint32_t* adm_keys, uint32_t A, const uint32_t* member_off,
                   const uint16_t* members, uint16_t* dest, uint64_t* n_bad)
{
    if (R == 0 || R > 65535 || K == 0) return -1;
    int64_t* rank = (int64_t*)malloc(sizeof(int64_t) * (size_t)K);
    uint64_t* load = (uint64_t*)calloc(R, sizeof(uint64_t));
    if (!rank || !load) {
        free(rank);
        free(load);
        return -2;
    }
    for (uint32_t b = 0; b < K; ++b) rank[b] = -1;
    for (uint32_t a = 0; a < A; ++a) rank[adm_keys[a]] = a;
    uint64_t bad = 0;
    for (uint64_t i = 0; i < n; ++i) {
        uint32_t b = keys[i];
        uint32_t d;
        if (b < K && rank[b] >= 0) {
            uint32_t a = (uint32_t)rank[b];
            d = members[member_off[a]];
            for (uint32_t t = member_off[a] + 1; t < member_off[a + 1]; ++t) {
                uint32_t m = members[t];
                if (load[m] < load[d] || (load[m] == load[d] && m < d)) d = m;
            }
        } else {
            if (b >= K) bad += 1;
            uint32_t h = cro_hash(seed, first_index + i);
            uint32_t d1 = (uint32_t)(((uint64_t)(h & 0xFFFFu) * R) >> 16);
            uint32_t d2 = (uint32_t)(((uint64_t)(h >> 16) * R) >> 16);
            d = load[d2] < load[d1] ? d2 : d1;
        }
        dest[i] = (uint16_t)d;
        load[d] += 1;
    }
    if (n_bad) *n_bad += bad;
    free(rank);
    free(load);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Shadow replay of one plan's routing (Section 3.2: admitted and cold      */
/* prefixes share each destination's cache and eviction policy).            */
/* Model: destination d holds an LRU list of at most W whole prefixes       */
/* (the equal-slot model of Section 3.1), most recent first. The list is     */
/* carried in `lru` ([R][W], empty slots = 0xFFFFFFFF after the used ones)   */
/* and is never reset between intervals or plan changes.                     */
/* For request i (interval j, destination d, key b):                         */
/*   requests += 1; prefill += suffix[i];                                    */
/*   b cached: hits += 1; hit_prefix += prefix_len[b]; b becomes most recent */
/*   else:     prefill += prefix_len[b]; b inserted as most recent, the      */
/*             least recent entry dropped when W would be exceeded.          */
/* stats[(j*R + d)*4 + {0,1,2,3}] += {requests, hits, prefill, hit_prefix}.  */
/* Requests whose key is >= K are skipped and counted in *n_bad.             */
/* ------------------------------------------------------------------------ */
int cro_replay(const uint32_t* keys, const uint16_t* suffix, const uint32_t* prefix_len, uint32_t K,
               const uint16_t* dest, uint64_t n, const uint64_t* offsets, uint32_t J, uint32_t R,
               uint32_t W, uint32_t* lru, uint64_t* stats, uint64_t* n_bad)
{
    if (cro_check_offsets(offsets, J, n) || R == 0 || W == 0 || K == 0) return -1;
    uint32_t* used = (uint32_t*)calloc(R, sizeof(uint32_t));
    if (!used) return -2;
    for (uint32_t d = 0; d < R; ++d) {
        uint32_t* row = lru + (uint64_t)d * W;
        uint32_t u = 0;
        while (u < W && row[u] != CRO_EMPTY) ++u;
        for (uint32_t s = u; s < W; ++s) row[s] = CRO_EMPTY;
        used[d] = u;
    }
    uint64_t bad = 0;
    uint32_t j = 0;
    for (uint64_t i = 0; i < n; ++i) {
        while (i >= offsets[j + 1]) ++j;
        uint32_t d = dest[i];
        uint32_t b = keys[i];
        if (d >= R) {
            free(used);
            return -1;
        }
        if (b >= K) {
            bad += 1;
            continue;
        }
        uint64_t* s = stats + ((uint64_t)j * R + d) * 4;
        uint32_t* row = lru + (uint64_t)d * W;
        s[0] += 1;
        s[2] += suffix[i];
        uint32_t pos = 0;
        while (pos < used[d] && row[pos] != b) ++pos;
        if (pos < used[d]) {
            s[1] += 1;
            s[3] += prefix_len[b];
            memmove(row + 1, row, sizeof(uint32_t) * pos);
        } else {
            s[2] += prefix_len[b];
            uint32_t keep = used[d] < W ? used[d] : W - 1;
            memmove(row + 1, row, sizeof(uint32_t) * keep);
            if (used[d] < W) used[d] += 1;
        }
        row[0] = b;
    }
    if (n_bad) *n_bad += bad;
    free(used);
    return 0;
}
