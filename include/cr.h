/*
 * cr.h -- C ABI of the CacheRoute planner and shadow-replay library (libcr.so, gfx950).
 *
 * The library computes, on one MI355X GPU, the data-parallel core of the periodic
 * routing planner of "CacheRoute: Planned Prefix-Affinity Routing for Large-Scale
 * LLM Serving" (Section 3.1, Eq. 1, Algorithm 1; Section 3.2) and a shadow replay
 * of the resulting routing against per-destination prefix caches.
 *
 * Conventions for every entry point:
 *  - Buffers are DEVICE pointers owned by the caller unless marked "host".
 *  - A call validates its scalar arguments on the host, enqueues kernels on `stream`
 *    (a hipStream_t passed as void*; NULL = the default stream) and returns. It
 *    never allocates device memory, frees or synchronises, and keeps no state between
 *    calls, except where a call says otherwise (cr_replay_lru's side streams,
 *    cr_admit_noalloc's scratch array, cr_replay_set_group_min_records).
 *    Calls are thread-compatible: concurrent calls must not share output buffers.
 *  - Return value: CR_OK, or a negative cr_status. On CR_EINVAL or CR_ESIZE nothing
 *    has been enqueued; CR_EHIP reports a failed HIP call, and launches of the same
 *    call made before it may have been enqueued.
 *  - Data-dependent problems found on the device (a key >= num_keys, a destination
 *    >= R, an inconsistent plan spec) never abort a kernel: the offending item is
 *    skipped as documented per call, and a CR_ERR_* bit is OR-ed into the caller's
 *    device word `err` (which the caller clears).
 *  - Keys are dense ids in [0, num_keys); 0xFFFFFFFF is reserved (empty slot).
 *  - Request i of a stream has global index first_index + i; control intervals are
 *    given by device offsets off[0..J] with off[0] = 0, off[J] = n, non-decreasing.
 */
#ifndef CR_H
#define CR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t cr_status;
#define CR_OK 0
#define CR_EINVAL (-1) /* an argument is out of range or a pointer is NULL   */
#define CR_ESIZE (-2)  /* the workspace is smaller than the size query says   */
#define CR_EHIP (-3)   /* a HIP launch or runtime call failed                 */

#define CR_ERR_KEY_RANGE 1u   /* a key >= num_keys was seen                       */
#define CR_ERR_DEST_RANGE 2u  /* a destination >= R was seen by the replay        */
#define CR_ERR_SPEC 4u        /* a plan spec disagrees with its counts row         */
#define CR_ERR_KEYMAP_FULL 8u /* more distinct opaque ids than the directory holds  */

#define CR_EMPTY_SLOT 0xFFFFFFFFu /* unused LRU slot / unused key               */
#define CR_NO_KEY 0xFFFFFFFFu     /* not an opaque id; dense index of an unknown id */
#define CR_KEYMAP_MAX_CAPACITY (1u << 28) /* distinct opaque ids per directory      */
#define CR_ROUTE_SINGLE 0x80000000u /* route word flag: k = 1, low 16 bits = dest */

#define CR_MAX_R 1024      /* destinations per plan                            */
#define CR_MAX_W 512       /* warm slots per destination                       */
#define CR_MAX_CANDS 256   /* candidate plans per group                        */
#define CR_MAX_J 65535     /* control intervals per cr_replay call             */

/* Plan variants: the method and the stages of the paper's component ablation (Section 5.2,
 * 8B component ablation table), each a plan the same dispatch and replay can run.
 *   CR_PLAN_FULL        Eq. 1 replication and LPT placement (Algorithm 1)
 *   CR_PLAN_AFFINITY    k = 1 for every admitted key (top C keys), hash placement
 *   CR_PLAN_REPLICATED  Eq. 1 replication, hash placement
 *   CR_PLAN_FLAT        nothing admitted: every request takes the cold path, and with
 *                       uniform planned loads that is plain hashing (load balancing alone)
 * Hash placement gives key b the k destinations with the smallest (u(b, r), r), listed in
 * that order, where u(b, r) = fmix32(fmix32(b ^ t) ^ r), t = fmix32(place_seed ^ 0x7F4A7C15):
 * a uniformly random k-subset per key, independent of the loads. Every variant charges
 * count / k to each member after L[r] = cold / R, in admission order, as LPT does. */
#define CR_PLAN_FULL 0u
#define CR_PLAN_AFFINITY 1u
#define CR_PLAN_REPLICATED 2u
#define CR_PLAN_FLAT 3u

/* One plan problem (Algorithm 1 inputs: rates, R, q_cap, C). Arrays of these live in
 * DEVICE memory. q_cap = q_num / q_den requests per window, so Eq. 1 is evaluated as
 * k = max(1, ceil(c * q_den / q_num)) in exact integers; k is clamped to R.
 * With n_window = CR_WINDOW_SUM the device takes N_w = the counts row's sum and the target
 * is relative to the mean per-destination load: q_cap = (q_num / q_den) * N_w / R, i.e. the
 * rule above with q_num * N_w and q_den * R (q_num * N_w < 2^63, q_den * R < 2^31). */
#define CR_WINDOW_SUM 0xFFFFFFFFFFFFFFFFull
typedef struct {
    uint32_t window;     /* row of counts the plan is built from (< num_windows)      */
    uint32_t W;          /* warm slots per destination, 1..max_W; C = R * W           */
    uint64_t n_window;   /* requests in that row (its sum), or CR_WINDOW_SUM          */
    uint64_t q_num;      /* > 0 unless the window is empty (unused by AFFINITY, FLAT) */
    uint64_t q_den;      /* 1 .. 2^31 - 1 (likewise)                                  */
    uint32_t variant;    /* CR_PLAN_*                                                 */
    uint32_t place_seed; /* hash placement seed (AFFINITY, REPLICATED)                */
} cr_plan_spec;

/* A set of NP plans arranged as NG groups of `cands` candidates: plan p = g*cands + c.
 * Every plan of group g routes the same requests. A plan's dispatch table is compact:
 * key_index marks its admitted keys in a bit mask per 64 keys together with the key rank
 * (position in key order among the admitted keys) of the first admitted key of those 64,
 * and route holds one word per admitted key in key-rank order. A lookup is one 16-byte
 * load and a popcount; a cold key needs nothing more.
 * Host struct of device pointers; sizes follow from the fields (C_max = R * max_W,
 * KW = ceil(num_keys / 64)):
 *   order      u32 [num_windows][C_max]  nonzero keys by (count desc, key asc), cut at C_max
 *   order_count u32 [num_windows][C_max] their counts
 *   n_order    u32 [num_windows]         entries of order used
 *   num_admitted u32 [NP]                A
 *   cold       u64 [NP]                  window requests not carried by admitted keys
 *   clamped    u32 [NP]                  admitted keys whose k was clamped to R
 *   member_off u32 [NP][C_max + 1]       member list a = members[off[a] .. off[a+1])
 *   members    u16 [NP][C_max]           T(b) per admitted key, in selection order
 *   load       f64 [NP][R]               planned loads L after placement
 *   key_index  u64 [NP][KW][2]          {admitted-key bits of keys 64w..64w+63,
 *                                        key rank of the first admitted key among them}
 *   route      u32 [NP][C_max]           by key rank: CR_ROUTE_SINGLE | dest (k = 1)
 *                                        or the admission index a (k > 1)
 *
 * Optional group dispatch tables (all four NULL = per-plan tables only). When every
 * candidate of a group is built from the same counting window, a candidate admits a prefix
 * of that window's order, so cr_route can serve all candidates of a request from one row:
 * with these buffers present, cr_route first rebuilds them from the built plans and then
 * reads, per request, one position, one row of CS destinations and the load-rank rows of
 * the request's two fallback draws (CS = cands rounded up to a multiple of 8):
 *   window_rank u32 [num_windows][num_keys]  position of each key in its window's order
 *                                             (0xFFFFFFFF when absent)
 *   group_dest  u16 [NG][C_max][CS]          by position a: the member of candidate c when it
 *                                             admits the key with k = 1, CR_GROUP_MULTI when
 *                                             k > 1, CR_GROUP_COLD when it does not admit it
 *   group_rank  u16 [NG][R][CS]              by destination d: entry c = number of
 *                                             destinations whose L_c is strictly below L_c[d]
 *                                             (so L_c[d2] < L_c[d1] iff rank c of d2 < rank
 *                                             c of d1)
 *   group_multi u32 [NG][C_max][CS]          where group_dest holds CR_GROUP_MULTI:
 *                                             o | k << 20 with members[o .. o+k) the key's
 *                                             member list in candidate c (else unspecified)
 * A group whose candidates name different windows sets CR_ERR_SPEC, and its destinations
 * are then unspecified. group_dest, group_rank and group_multi must be 16-byte aligned, and
 * window_rank, group_multi and the members of all plans must each stay below 4 GiB
 * (CR_EINVAL otherwise). Sizes: cr_plan_sizes. */
#define CR_GROUP_MULTI 0xFFFEu
#define CR_GROUP_COLD 0xFFFFu
typedef struct {
    uint32_t num_plans;   /* NP = NG * cands                                       */
    uint32_t cands;       /* candidates per group, 1..CR_MAX_CANDS                 */
    uint32_t R;           /* destinations, 1..CR_MAX_R                             */
    uint32_t max_W;       /* >= every spec's W, <= CR_MAX_W                        */
    uint32_t num_keys;    /* K                                                     */
    uint32_t num_windows; /* rows of counts                                        */
    const cr_plan_spec* specs; /* [NP]                                             */
    uint32_t* order;
    uint32_t* order_count;
    uint32_t* n_order;
    uint32_t* num_admitted;
    uint64_t* cold;
    uint32_t* clamped;
    uint32_t* member_off;
    uint16_t* members;
    double* load;
    uint64_t* key_index;
    uint32_t* route;
    uint32_t* window_rank;  /* optional group dispatch tables (see above), or NULL      */
    uint16_t* group_dest;
    uint16_t* group_rank;
    uint32_t* group_multi;
} cr_plan_set;

/* Rates of one slice of the log, accumulated (Algorithm 1 input "rates"; Appendix A.2):
 *   counts[b] += #{ i < n : keys[i] == b }
 * keys u32 [n] (n < 2^32 - 1); counts u32 [num_keys] (accumulated: clear it for a fresh
 * window). Meant for key spaces beyond LDS (e.g. 10^6 keys): the slice is bucket-sorted by
 * key range in tiles and each bucket counted in LDS, with no global atomics, in a workspace
 * of cr_count_slice_workspace_bytes(n, num_keys) bytes (CR_ESIZE if smaller; buckets of up
 * to 32,768 keys and at most 256 buckets, CR_EINVAL beyond). A key >= num_keys is not
 * counted and sets CR_ERR_KEY_RANGE. */
size_t cr_count_slice_workspace_bytes(uint64_t n, uint32_t num_keys);
cr_status cr_count_slice(const uint32_t* keys, uint64_t n, uint32_t num_keys, uint32_t* counts, uint32_t* err,
                         void* ws, size_t ws_bytes, void* stream);

/* Rates per key per control interval (Algorithm 1 input "rates"; Appendix A.2: the
 * planner needs only {(b, lambda_b)}). Rates are kept in requests per window.
 *   counts[j * num_keys + b] = #{ i in [off[j], off[j+1]) : keys[i] == b }
 * keys u32 [n]; off u64 [J+1]; counts u32 [J][num_keys] (overwritten, every row).
 * A key >= num_keys is not counted and sets CR_ERR_KEY_RANGE. */
cr_status cr_count_rates(const uint32_t* keys, uint64_t n, const uint64_t* off, uint32_t J,
                         uint32_t num_keys, uint32_t* counts, uint32_t* err, void* stream);

/* Workspace for cr_admit, in bytes. */
size_t cr_admit_workspace_bytes(uint32_t num_windows, uint32_t R, uint32_t max_W);

/* Byte sizes of the buffers of a cr_plan_set with these fields, in struct order: specs, order,
 * order_count, n_order, num_admitted, cold, clamped, member_off, members, load, key_index,
 * route, window_rank, group_dest, group_rank, group_multi (the last four: the optional group
 * tables).
 * out_bytes has CR_PLAN_BUFFERS entries. */
#define CR_PLAN_BUFFERS 16
void cr_plan_sizes(uint32_t num_plans, uint32_t cands, uint32_t R, uint32_t max_W, uint32_t num_keys,
                   uint32_t num_windows, size_t out_bytes[CR_PLAN_BUFFERS]);

/* One workspace size that serves cr_count_slice for slices of up to max_n requests and
 * cr_replay / cr_replay_partition / cr_replay_lru for up to max_n requests, P candidates and
 * R destinations (cr_admit's depends on the windows and has its own query). */
size_t cr_workspace_bytes(uint32_t num_keys, uint32_t R, uint32_t P, uint64_t max_n);

/* Top-rate admission (Eq. 1; Section 3.1 "Warm-set admission"; Algorithm 1 sort/admit).
 * For every window: order its nonzero keys by (count desc, key asc), cut at C_max.
 * For every plan: k_b by Eq. 1 (exact integers, clamped to R), then admit the longest
 * prefix of that order whose k_b sum is <= C = R * W; cold = n_window - admitted counts.
 * counts u32 [num_windows][num_keys]. Writes order, order_count, n_order, num_admitted,
 * cold, clamped, member_off[0..A] (prefix sums of k) and the plan's whole key_index
 * (its admitted keys are order[window][0..A)). CR_PLAN_AFFINITY takes k = 1 for every key
 * and CR_PLAN_FLAT admits nothing. A spec with a window out of range, q_num == 0 on a
 * nonempty window (FULL, REPLICATED), n_window != row sum or an unknown variant sets
 * CR_ERR_SPEC (the plan then admits nothing). */
cr_status cr_admit(const uint32_t* counts, const cr_plan_set* plans, void* ws, size_t ws_bytes,
                   uint32_t* err, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): cr_admit with its workspace in a
 * library-owned device array of CR_ADMIT_SCRATCH_BYTES per GPU (held until the process
 * ends) instead of a caller workspace. The caller still owns counts, the plan set and err.
 * CR_ESIZE when cr_admit_workspace_bytes(num_windows, R, max_W) exceeds the array. The
 * call allocates nothing; every call on one GPU uses that GPU's array, so calls that
 * overlap on one GPU race (serialise them on one stream). Otherwise as cr_admit. */
#define CR_ADMIT_SCRATCH_BYTES (64u << 20)
cr_status cr_admit_noalloc(const uint32_t* counts, const cr_plan_set* plans, uint32_t* err, void* stream);

/* LPT placement (Section 3.1 "Placement and dispatch"; Algorithm 1 placement loop).
 * Per plan: L[r] = cold / R; admitted keys in admission order take the k smallest
 * (L[r], r) destinations, listed in that order, each charged count / k (IEEE double,
 * one rounding per operation, the same order as the definition). Writes members,
 * load and route[0..A) (it reads key_index as cr_admit left it). Plans of the hash-placed
 * variants (CR_PLAN_AFFINITY, CR_PLAN_REPLICATED) are left to cr_place_hash. */
cr_status cr_place_lpt(const uint32_t* counts, const cr_plan_set* plans, void* stream);

/* Hash placement of the ablation variants CR_PLAN_AFFINITY and CR_PLAN_REPLICATED (Section
 * 5.2): members are each key's k smallest (u(b, r), r) (see CR_PLAN_*), and the loads
 * L[r] = cold / R + the count / k of every admitted key placed on r, added in admission
 * order (IEEE double, as cr_place_lpt). Writes members, load and route[0..A) of those plans
 * and leaves the others untouched. Cost: R hashes per admitted key and k passes over them. */
cr_status cr_place_hash(const uint32_t* counts, const cr_plan_set* plans, void* stream);

/* Dispatch (Section 3.1 "Placement and dispatch"; Fig. 1), order-independent form.
 * Request i lies in interval j and uses plan group gmap[j]; for candidate c:
 *   h = fmix32((u32)g ^ fmix32((u32)(g >> 32) ^ s)), g = first_index + i,
 *   s = fmix32((u32)seed ^ (u32)(seed >> 32) ^ 0x9E3779B9) (fmix32 = MurmurHash3's finalizer);
 *   admitted key with members M (k of them): dest = M[((h >> 16) * k) >> 16];
 *   otherwise d1 = ((h & 0xFFFF) * R) >> 16, d2 = ((h >> 16) * R) >> 16 and
 *   dest = L[d2] < L[d1] ? d2 : d1 with L the plan's loads (power of two choices).
 * keys u32 [n]; off u64 [J+1]; gmap u32 [J] (< NG); dest u16 [cands][n].
 * A key >= num_keys is routed as cold and sets CR_ERR_KEY_RANGE. */
cr_status cr_route(const uint32_t* keys, uint64_t n, uint64_t first_index, uint64_t seed,
                   const uint64_t* off, const uint32_t* gmap, uint32_t J, const cr_plan_set* plans,
                   uint16_t* dest, uint32_t* err, void* stream);

/* Live-load dispatch (Section 3.1 "Placement and dispatch": during the interval admitted
 * traffic takes the least-loaded member of its fixed T(b), other traffic power of two
 * choices; Fig. 1). Load is the number of requests of the current interval already sent to
 * a destination (zero at every interval start), so each decision depends on all earlier
 * ones in its interval:
 *   admitted key: the member of T(b) with the smallest (load, destination);
 *   otherwise: d1, d2 drawn from the request hash exactly as in cr_route, and d2 only if
 *   load[d2] < load[d1].
 * Arguments, layouts and errors as for cr_route (the plans' loads are not read). Intervals
 * and candidates run in parallel, one serial chain each: the cost is the longest
 * interval's length, not n. */
cr_status cr_route_live(const uint32_t* keys, uint64_t n, uint64_t first_index, uint64_t seed,
                        const uint64_t* off, const uint32_t* gmap, uint32_t J, const cr_plan_set* plans,
                        uint16_t* dest, uint32_t* err, void* stream);

/* Churn between pairs of built plans of one set (Section 5.4 "Rate drift and remapping";
 * Appendix E, table of replan measurements). With S_x = {(b, r) : r in T_x(b)} over plan
 * x's admitted keys b, pair i = (p, q) = (pairs[2i], pairs[2i+1]) yields
 *   out[4i+0] = |S_p intersected with S_q|       (key-destination pairs in both plans)
 *   out[4i+1] = keys admitted by both plans
 *   out[4i+2] = of those, keys whose k differs
 *   out[4i+3] = of those, keys whose destination set T is the same.
 * Cache churn = 1 - out[4i] / (|S_p| + |S_q| - out[4i]) with |S_x| = member_off[x][A_x];
 * count churn = out[4i+2] / out[4i+1]. Cost per key admitted by both: k_p * k_q compares.
 * pairs u32 [num_pairs][2]; out u64 [num_pairs][4] (overwritten). The plans must have
 * been built by cr_admit and cr_place_lpt. A pair naming a plan >= num_plans sets
 * CR_ERR_SPEC and yields zeros. */
cr_status cr_plan_churn(const cr_plan_set* plans, const uint32_t* pairs, uint32_t num_pairs, uint64_t* out,
                        uint32_t* err, void* stream);

/* Workspace for cr_replay (and for its two phases), in bytes. */
size_t cr_replay_workspace_bytes(uint64_t n, uint32_t P, uint32_t R);

/* Carried LRU state of the replay, u32 [P][R][max_W] (most recent first, CR_EMPTY_SLOT after
 * the used entries): its size in bytes, and a reset of all of it to empty caches (a fill
 * kernel on `stream`; it records no memset, so it can be captured in a HIP graph). */
size_t cr_lru_state_bytes(uint32_t P, uint32_t R, uint32_t max_W);
cr_status cr_lru_reset(uint32_t* lru_state, uint32_t P, uint32_t R, uint32_t max_W, void* stream);

/* Shadow replay (Section 3.2: admitted and cold prefixes share each destination's
 * cache) against an LRU of W_c whole-prefix slots per destination (the equal-slot model
 * of Section 3.1), for P candidate routings of the same stream at once.
 * For candidate c, destination d, requests in arrival order:
 *   requests += 1; prefill += suffix[i];
 *   key cached: hits += 1; hit_prefix += prefix_len[key]; key becomes most recent;
 *   otherwise:  prefill += prefix_len[key]; key inserted as most recent, the least
 *               recent dropped once W_c would be exceeded.
 * keys u32 [n]; suffix u16 [n]; prefix_len u32 [num_keys]; dest u16 [P][n]; off u64 [J+1];
 * W host u32 [P] (1..CR_MAX_W); lru_in / lru_out u32 [P][R][max_W]: carried cache state,
 * most recent first, CR_EMPTY_SLOT after the used entries (lru_in NULL = all empty;
 * lru_in and lru_out must not overlap); stats u64 [J][P][R][4] (accumulated) =
 * {requests, hits, prefill_tokens, hit_prefix_tokens}. n < 2^32 - 1.
 * A destination >= R sets CR_ERR_DEST_RANGE and a key >= num_keys sets CR_ERR_KEY_RANGE;
 * such requests are skipped.
 * cr_replay = cr_replay_partition followed by cr_replay_lru on the same workspace. */
cr_status cr_replay(const uint32_t* keys, const uint16_t* suffix, const uint32_t* prefix_len,
                    uint32_t num_keys, const uint16_t* dest, uint64_t n, const uint64_t* off,
                    uint32_t J, uint32_t P, uint32_t R, const uint32_t* W, uint32_t max_W,
                    const uint32_t* lru_in, uint32_t* lru_out, uint64_t* stats, void* ws,
                    size_t ws_bytes, uint32_t* err, void* stream);

/* First phase of cr_replay: groups every candidate's requests by destination in arrival
 * order (records of key, suffix and interval in the workspace) and cuts each group into
 * independent segments. Arguments as for cr_replay. */
cr_status cr_replay_partition(const uint32_t* keys, const uint16_t* suffix, const uint16_t* dest,
                              uint64_t n, const uint64_t* off, uint32_t J, uint32_t P, uint32_t R,
                              const uint32_t* W, void* ws, size_t ws_bytes, uint32_t* err,
                              void* stream);

/* Second phase of cr_replay: replays the partitioned workspace (same n, J, P, R, W)
 * through the per-destination LRU caches and accumulates stats. Each segment rebuilds the
 * cache state it starts from by scanning its stream backwards for W distinct keys, at most
 * eight segment lengths; a segment whose scan runs out before that (a stretch with fewer than
 * W distinct keys) is left to a second launch, in which one wavefront per run of such
 * segments replays the segment before the run (without counting it) and then the run, in
 * order. Each request is thus replayed at most twice and scanned at most nine times,
 * whatever the key mix; the results do not depend on which launch counts them.
 * The launches of the first pass (one per list size, ceil(W/64) registers, and one per
 * grouped form) are independent of each other. When there are two or more and `stream`
 * is not capturing, they run on two side streams of the device, forked from `stream`
 * by an event and joined back to it before the second launch: the side streams and
 * their three events are created by the first such call on a device (hipStreamCreate,
 * default priority) and kept until the process ends, and calls from several host
 * threads take a host mutex while they enqueue. Ordering on `stream` is as if every
 * launch were on it. A failure to create them keeps the launches on `stream`. The HIP
 * runtime maps streams onto a few hardware queues (four per process by default); when
 * the process already holds streams of its own, both side streams can land on one
 * queue, and the launches then run one after another. */
cr_status cr_replay_lru(const uint32_t* prefix_len, uint32_t num_keys, uint64_t n, uint32_t J,
                        uint32_t P, uint32_t R, const uint32_t* W, uint32_t max_W,
                        const uint32_t* lru_in, uint32_t* lru_out, uint64_t* stats, void* ws,
                        size_t ws_bytes, uint32_t* err, void* stream);

/* Size rule of the replay of small caches (process-wide, not a result): in a call with one
 * interval (J == 1), the candidates with W <= 16 are replayed several per wavefront (4 or 8
 * caches side by side) when n times their number is at least min_records (default 2^25);
 * below that there are too few segments for the grouped form to fill the GPU. The results
 * are the same either way; 0 makes every such call use the grouped form (for tests). Takes
 * effect for calls issued after it returns; calls that overlap it in other threads may see
 * either value. */
void cr_replay_set_group_min_records(uint64_t min_records);

/* Opaque-key directory (Appendix A.2 "Data handling": the planner needs only the pairs
 * (b, lambda_b), and b may be salted or ephemeral; Section 2.1: the workload summaries
 * carry opaque keys). It maps 32-bit opaque ids to the dense indices the counting rows
 * need. The dense index of an id is the rank of its first occurrence among the distinct
 * ids of the build stream (order of first appearance), independent of scheduling.
 * CR_NO_KEY is not an id.
 *
 * Directory size in bytes for up to `capacity` distinct ids (an open-addressing table of
 * at least 2 * capacity slots, 16 bytes each); device memory owned by the caller, 16-byte
 * aligned. */
size_t cr_keymap_bytes(uint32_t capacity);
/* Workspace of cr_keymap_build for a stream of n ids, in bytes (a first-occurrence bitmap
 * of n bits, its per-word prefix and per-block sums). */
size_t cr_keymap_workspace_bytes(uint64_t n);
/* Builds the directory of ids u32 [n] (n < 2^32 - 1) into `table`, replacing its contents.
 * num_keys u32 [1] (device) receives the number of distinct ids. An id equal to CR_NO_KEY
 * sets CR_ERR_KEY_RANGE and is skipped. More than `capacity` distinct ids sets
 * CR_ERR_KEYMAP_FULL and the directory must not be used: once its table is full, ids
 * that found no slot are missing and the indices are ranks among the ids it holds. 1 <= capacity <=
 * CR_KEYMAP_MAX_CAPACITY. */
cr_status cr_keymap_build(const uint32_t* ids, uint64_t n, uint32_t capacity, void* table, size_t table_bytes,
                          void* ws, size_t ws_bytes, uint32_t* num_keys, uint32_t* err, void* stream);
/* dense[i] = dense index of ids[i], or CR_NO_KEY for an id the directory does not hold
 * (later stages skip such keys as out of range). ids, dense u32 [n]; `capacity` as built. */
cr_status cr_keymap_lookup(const void* table, size_t table_bytes, uint32_t capacity, const uint32_t* ids,
                           uint64_t n, uint32_t* dense, void* stream);
/* Per-key attributes given by opaque id, moved to dense order: out[dense(ids[x])] =
 * values[x] for every x < m whose id the directory holds and whose index is < out_len;
 * other entries of out are left as they are. ids, values u32 [m]; out u32 [out_len]. */
cr_status cr_keymap_scatter(const void* table, size_t table_bytes, uint32_t capacity, const uint32_t* ids,
                            const uint32_t* values, uint64_t m, uint32_t* out, uint32_t out_len, void* stream);

/* Library version string. */
const char* cr_version(void);

#ifdef __cplusplus
}
#endif
#endif /* CR_H */
