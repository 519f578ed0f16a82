/*
 * apc — approximate-cache prompt matching on MI355X (gfx950).
 *
 * C ABI of the per-batch step of prompt-aware scheduling for diffusion
 * serving with approximate caching (Approach section of the paper): for a
 * batch of prompt embeddings, find the nearest cached prompts, turn the best
 * closeness into an optimal skip level K, place every prompt on a model
 * instance under per-instance capacity (redirecting to other levels when the
 * optimal one is full), and gather the cached intermediate state (latent)
 * each placed prompt will start denoising from.
 *
 * Conventions shared by every call:
 *  - Pointers are DEVICE pointers unless marked (host).  All device buffers
 *    belong to the caller and must be 16-byte aligned.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Calls enqueue work on it and return without waiting, except
 *    apc_build_cache, which waits once to report data errors.
 *  - Calls keep no device state of their own between or across calls: calls
 *    on different streams may run concurrently when their output and
 *    workspace buffers are distinct (one cache handle may serve them all).
 *  - Arguments are checked on the host before anything is enqueued; on a
 *    non-OK status nothing was enqueued and no output was written, except
 *    APC_E_HIP (a launch failed; outputs are unspecified).
 *  - apc_last_error() gives a thread-local message for the last failing call.
 *  - Calls that take a cache handle must run with the handle's device
 *    current (the device that was current at apc_build_cache); on another
 *    device they return APC_E_ARG before enqueuing anything.
 *  - Calls on different streams may run concurrently when they write
 *    disjoint buffers (each match call needs its own workspace).
 */
#ifndef APC_H
#define APC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* storage type of embeddings and queries */
typedef enum {
    APC_F32 = 0,   /* IEEE binary32 */
    APC_F16 = 1,   /* IEEE binary16 */
    APC_BF16 = 2,  /* bfloat16 */
    APC_E4M3 = 3,  /* OCP e4m3fn codes with one float32 scale per row */
    APC_DTYPE_INT32 = 0x7fffffff  /* not a type: makes every int32 value a valid apc_dtype,
                                     so unknown types are reported as APC_E_DTYPE */
} apc_dtype;

typedef enum {
    APC_OK = 0,
    APC_E_ARG = 1,        /* bad size, pointer, alignment or count */
    APC_E_DTYPE = 2,      /* unknown storage type */
    APC_E_TABLE = 3,      /* bad threshold or instance table */
    APC_E_NONFINITE = 4,  /* a cache row holds Inf/NaN, or a row scale is not finite and > 0 */
    APC_E_ZERO_NORM = 5,  /* a cache row has zero norm */
    APC_E_WORKSPACE = 6,  /* workspace smaller than apc_match_workspace() asks */
    APC_E_NOMEM = 7,      /* device or host allocation failed */
    APC_E_HIP = 8,        /* a HIP runtime call or kernel launch failed */
    APC_STATUS_INT32 = 0x7fffffff  /* not a status: makes every int32 value a valid apc_status,
                                      so apc_status_str may be given any value */
} apc_status;

#define APC_MAX_K 64          /* largest neighbour count per query */
#define APC_MAX_LEVELS 32     /* largest number of skip levels L */
#define APC_MAX_INST 256      /* largest number of model instances */
#define APC_MAX_SHARDS 64     /* largest number of row shards apc_merge_shards merges */
#define APC_MAX_ROUTED_BATCH 16384  /* largest batch of apc_assign_routed / apc_assign_planned */

/* opaque, immutable after build */
typedef struct apc_cache apc_cache;

/*
 * Build a handle over a cache of n prompt embeddings (the approximate cache
 * of the Introduction: prior prompts whose intermediate states can be
 * reused).
 *
 * emb           n x d row-major elements of type dt; d * element size must be
 *               a multiple of 16 bytes.
 * row_scale     n float32 (APC_E4M3 only, else NULL): element value = code *
 *               scale.  Scales must be finite and > 0.  The cosine does not
 *               depend on them.
 * latents       n_slots x latent_bytes cached latents, or NULL with n_slots = 0
 *               (no gather).  latent_bytes must be a multiple of 16.
 * slot_of_entry n int32: the latent slot of each entry, -1 = not resident;
 *               NULL = entry i lives in slot i (then n_slots >= n).
 *
 * The handle BORROWS emb, row_scale, latents and slot_of_entry: they must
 * stay alive and unchanged until apc_destroy_cache.  The library owns only
 * the n float32 row factors (1 / norm; zero-padded past n to whole row
 * groups) on the current device.  Waits for the
 * stream once and returns APC_E_NONFINITE / APC_E_ZERO_NORM / APC_E_ARG
 * (slot out of range) for bad data, with *out left NULL.
 */
apc_status apc_build_cache(apc_dtype dt, int64_t n, int32_t d, const void* emb,
                           const float* row_scale, const void* latents, int64_t n_slots,
                           int64_t latent_bytes, const int32_t* slot_of_entry, void* stream,
                           apc_cache** out /* host */);

/* Frees the handle and its row factors (NULL is a no-op).  The caller must
   make sure no call using the handle is still running. */
void apc_destroy_cache(apc_cache* c);

/*
 * Row factors f = 1 / |x| of n rows of type dt (for APC_E4M3 the norm of
 * the codes; the scale cancels in the cosine), written to out (n float32).
 * Rows with a non-finite element or zero norm get NaN.  This is the
 * per-row preparation of both the cache build and the query batch.
 */
apc_status apc_row_factors(apc_dtype dt, int64_t n, int32_t d, const void* rows, float* out,
                           void* stream);

/*
 * Storage of float32 embeddings in a cache type (the step before
 * apc_build_cache or apc_match_batch for a caller that holds float32
 * vectors; the paper keeps prompt embeddings in its cache and fixes no
 * storage type, so this recipe is the library's):
 *   APC_F16, APC_BF16  each element rounded to nearest-even (overflow gives
 *                      +-Inf; NaN gives a quiet NaN of the same sign);
 *   APC_E4M3           per row the scale s = amax / 448 (amax = the largest
 *                      |x| of the row, float32 division; s = 1 when it is not
 *                      > 0, which includes a row holding NaN), then each
 *                      element's e4m3fn code of clamp(x / s, -448, 448)
 *                      rounded to nearest-even (NaN gives 0x7f with its sign).
 * x          n x d float32 rows (device, 16-byte aligned, caller-owned).
 * out        n x d elements of dt (device, 16-byte aligned; d * element
 *            size a multiple of 16 bytes).
 * row_scale  n float32 (device; APC_E4M3 only, else NULL): the scales s.
 * dt = APC_F32 is APC_E_DTYPE; a missing, extra or misaligned pointer or a
 * row size that is not a multiple of 16 bytes is APC_E_ARG, returned before
 * anything is enqueued.  n = 0 is a no-op.  Asynchronous on stream.
 */
apc_status apc_quantize_rows(apc_dtype dt, int64_t n, int32_t d, const float* x, void* out, float* row_scale,
                             void* stream);

/*
 * Checks n rows of type dt as apc_build_cache checks cache rows (the
 * per-row preparation of the Query Dispatcher's retrieval: a row whose
 * cosine is undefined cannot be matched), for example a batch of queries
 * before apc_match_batch.  Bits of a row's flag: 1 = a non-finite element,
 * or a float32 sum of squares that is not finite (elements whose squares
 * overflow); 2 = zero norm (the float32 sum of squares is 0: every element
 * is at most 2^-75 in magnitude); 4 = (APC_E4M3) the row scale is not
 * finite and > 0.
 * rows       n x d elements of dt (device, 16-byte aligned; d * element
 *            size a multiple of 16 bytes).
 * row_scale  n float32 (device; APC_E4M3 only, else NULL).
 * bad        n uint8 flags (device, may be NULL).
 * n_bad      (host) number of rows with a flag; first_bad (host, may be
 *            NULL) the lowest such row, or -1.
 * Argument errors (as apc_quantize_rows; n_bad NULL) return APC_E_ARG or
 * APC_E_DTYPE before anything is enqueued.  Allocates a few bytes of device
 * memory per call and waits for the stream.  n = 0 is a no-op.
 */
apc_status apc_validate_rows(apc_dtype dt, int64_t n, int32_t d, const void* rows, const float* row_scale,
                             uint8_t* bad, int64_t* n_bad /* host */, int64_t* first_bad /* host */, void* stream);

/* Copies the handle's n entry factors to out (n float32, device). */
apc_status apc_cache_row_factors(const apc_cache* c, float* out, void* stream);

/* Workspace bytes apc_match_batch needs for b queries and k neighbours. */
apc_status apc_match_workspace(const apc_cache* c, int32_t b, int32_t k, size_t* bytes /* host */);

/*
 * Nearest cached prompts (Query Dispatcher, "retrieves the nearest cache"):
 * for each of the b query rows, the k cache entries with the highest cosine
 * similarity of the stored vectors,
 *     s(q, e) = clamp(<q, e> * f_q * f_e, -1, 1),   f = 1 / |row|,
 * accumulated in float32 over all d elements (no split over d, so scores are
 * deterministic), in the order (score desc, entry index asc).
 *
 * q          b x d row-major queries in the cache's type.
 * q_scale    b float32 (APC_E4M3 only, else NULL).
 * top_score  b x k float32, top_idx b x k int32 (row q at q * k).
 * ws         workspace of at least apc_match_workspace() bytes.
 * 1 <= k <= min(n, APC_MAX_K).  b = 0 is a no-op.
 * A query row that is non-finite, has zero norm or (APC_E4M3) a scale that
 * is not finite and > 0 gets top_score = NaN and top_idx = -1.
 */
apc_status apc_match_batch(const apc_cache* c, const void* q, const float* q_scale, int32_t b,
                           int32_t k, float* top_score, int32_t* top_idx, void* ws,
                           size_t ws_bytes, void* stream);

/*
 * apc_match_batch without a caller workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation): the workspace is a static device array
 * of APC_STATIC_WS_BYTES that each device holds from the library's first
 * use on it until the process ends (looked up on the first call on a
 * device).  The call allocates nothing.  Same arguments, outputs and errors
 * as apc_match_batch, plus APC_E_WORKSPACE when apc_match_workspace(c, b, k)
 * exceeds APC_STATIC_WS_BYTES (every workload up to 16,384 queries x k = 32
 * fits).  Nothing in the array needs to start at zero.  All calls on one
 * device share the array: calls that overlap on one device (other streams,
 * other threads) race and give undefined results; serialise them.
 */
#define APC_STATIC_WS_BYTES (32u << 20)
apc_status apc_match_batch_static(const apc_cache* c, const void* q, const float* q_scale, int32_t b,
                                  int32_t k, float* top_score, int32_t* top_idx, void* stream);

/*
 * Optimal level and capacity-constrained placement (Approach: optimal-K,
 * redirection to K' < K or to the closest K' > K with Eq. 1 charging
 * degradation only upwards; greedy route-and-batch filling the longest
 * queue first).
 *
 * top_score   b rows of stride ld (>= 1) float32; column 0 is the best score.
 * theta, K    (host) L float32 thresholds and L skip counts, both strictly
 *             increasing, thresholds finite, K > 0; 0 <= L <= APC_MAX_LEVELS.
 *             Level lam = #{l : best >= theta[l]} (0 = no skip, K = 0).
 * inst_level, inst_cap, inst_queue (host) n_inst <= APC_MAX_INST instances:
 *             level in 0..L, capacity >= 0 (total <= INT32_MAX), queue
 *             length (NULL = all 0).
 * Outputs (device): opt_level[b] = lam; out_level/out_inst/out_slot[b] = the
 *             placement (-1 when no capacity is left anywhere); inst_fill[n_inst]
 *             = queries placed per instance.
 * Placement: rounds r = 0..L over the preference list
 *             [lam, lam-1, .., 0, lam+1, .., L]; in each round unassigned
 *             queries, in index order, take a place at their r-th preference
 *             while it has capacity.  Within a level, places are handed out
 *             over its instances ordered by (queue desc, index asc), each up
 *             to its capacity, slots from 0.
 */
apc_status apc_assign(const float* top_score, int32_t ld, int32_t b, int32_t L,
                      const float* theta /* host */, const int32_t* K /* host */, int32_t n_inst,
                      const int32_t* inst_level /* host */, const int32_t* inst_cap /* host */,
                      const int32_t* inst_queue /* host, nullable */, int32_t* opt_level,
                      int32_t* out_level, int32_t* out_inst, int32_t* out_slot,
                      int32_t* inst_fill, void* stream);

/*
 * Load-aware route-and-batch (Approach, Query Dispatcher: uniform routing at
 * batch size 1 under low load, greedy routing to the workers with the
 * longest queues at their optimal batch size under high load).  Levels and
 * redirections as for apc_assign; only the routing inside a level changes.
 *
 * load, load_threshold (host): the caller's load measure (for example
 *             queued prompts) and the switch point.  load >= load_threshold:
 *             greedy routing, exactly apc_assign.  Below it: uniform routing:
 *             each instance takes at most one query, and a level's admitted
 *             queries (admission rank t = 0, 1, ..) go to its instances
 *             ordered by (inst_rand asc, index asc).
 * inst_rand   (host, n_inst uint32; may be NULL under greedy routing) random
 *             keys drawn by the caller for this batch: drawn uniformly at
 *             random, they make each admitted query land on a uniformly
 *             random instance of its level, one query per instance.
 * routing     (host, out) 1 = greedy, 0 = uniform.
 * Other arguments, outputs and errors as for apc_assign; APC_E_ARG when
 * uniform routing is chosen without inst_rand or routing is NULL.
 */
apc_status apc_assign_load_aware(const float* top_score, int32_t ld, int32_t b, int32_t L,
                                 const float* theta /* host */, const int32_t* K /* host */, int32_t n_inst,
                                 const int32_t* inst_level /* host */, const int32_t* inst_cap /* host */,
                                 const int32_t* inst_queue /* host, nullable */,
                                 const uint32_t* inst_rand /* host, nullable under greedy routing */,
                                 int64_t load, int64_t load_threshold, int32_t* routing /* host, out */,
                                 int32_t* opt_level, int32_t* out_level, int32_t* out_inst, int32_t* out_slot,
                                 int32_t* inst_fill, void* stream);

/*
 * Route-Plan (Eq. 1; the K-to-K' Route Planner of the Resource Controller):
 * an optimal integer plan X for serving per-level demand H with per-level
 * places F.  Host only: no GPU, no stream.
 *
 * Reading of Eq. 1 (its constraints are not printed): X[i][j] >= 0 queries of
 * optimal level i are served at level j, sum_j X[i][j] <= H[i] and
 * sum_i X[i][j] <= F[j]; min(sum H, sum F) queries are served (an unserved
 * query costs more than any move), and among such plans the degradation
 *   D = sum_{j > i} X[i][j] * (K_j - K_i)      (K_0 = 0)
 * is minimal; moves to fewer skipped steps (j < i) cost nothing.  Excess
 * demand is left unserved from the lowest levels up.  Of the optimal plans
 * the one returned serves each level's own queries first and moves the rest
 * in first-in-first-out order along the levels; it is deterministic.
 *
 * L, K        0 <= L <= APC_MAX_LEVELS; K (host) L skip counts of levels
 *             1..L, > 0 and strictly increasing (NULL when L = 0).
 * H, F        (host) L+1 demands and places per level, >= 0, each sum <= 2^31-1.
 * X           (host, out) (L+1) x (L+1) int32, row-major: X[i * (L+1) + j].
 * degradation (host, out, nullable) D of X.
 * Errors: APC_E_TABLE for L or K out of range, APC_E_ARG for NULL or negative
 * inputs or sums past 2^31-1; X is not written then.
 */
apc_status apc_route_plan(int32_t L, const int32_t* K, const int32_t* H, const int32_t* F, int32_t* X,
                          int64_t* degradation);

/*
 * Placement that follows a route plan (the K-to-K' Router applying the
 * Route-Plan as per-(K, K') quotas instead of the rounds of apc_assign).
 * Arguments, outputs and errors as for apc_assign, plus:
 *
 * plan        (device, in) (L+1) x (L+1) int32 quotas X, row-major; negative
 *             entries count as 0.
 * b           <= APC_MAX_ROUTED_BATCH (else APC_E_ARG).
 * Placement: the queries of optimal level i, in index order, take the levels
 *             of their preference list [i, i-1, .., 0, i+1, .., L] in that
 *             order, X[i][j] of them for level j; queries past sum_j X[i][j]
 *             get out_level = -1.  A level admits the queries routed to it by
 *             (position of the level in the query's preference list, query
 *             index) while it has places (later ones get -1); admission rank
 *             t goes to the level's instances ordered by (queue desc, index
 *             asc), each up to its capacity, slots from 0.  Given the flow
 *             X[i][j] that apc_assign realises, the result equals apc_assign's.
 */
apc_status apc_assign_routed(const float* top_score, int32_t ld, int32_t b, int32_t L,
                             const float* theta /* host */, const int32_t* K /* host */, int32_t n_inst,
                             const int32_t* inst_level /* host */, const int32_t* inst_cap /* host */,
                             const int32_t* inst_queue /* host, nullable */, const int32_t* plan /* device */,
                             int32_t* opt_level, int32_t* out_level, int32_t* out_inst, int32_t* out_slot,
                             int32_t* inst_fill, void* stream);

/*
 * apc_assign_routed with the plan built on the device, in the same kernel,
 * from the batch's own level histogram H (H[l] = #{q : opt_level[q] = l}),
 * the places per level F (sum of inst_cap over the level's instances) and K:
 * the plan apc_route_plan returns for (L, K, H, F), written to plan (device,
 * out, (L+1) x (L+1) int32).  One launch, no host round trip.
 */
apc_status apc_assign_planned(const float* top_score, int32_t ld, int32_t b, int32_t L,
                              const float* theta /* host */, const int32_t* K /* host */, int32_t n_inst,
                              const int32_t* inst_level /* host */, const int32_t* inst_cap /* host */,
                              const int32_t* inst_queue /* host, nullable */, int32_t* plan /* device */,
                              int32_t* opt_level, int32_t* out_level, int32_t* out_inst, int32_t* out_slot,
                              int32_t* inst_fill, void* stream);

/*
 * Resident-aware fallback (a query starts from a cached state only if that
 * state is resident, Introduction and Approach): for each query, the first of
 * its k neighbours top_idx[q * ld + 0..k-1] (ordered best first, as
 * apc_match_batch writes them) whose entry has a resident latent in cache c
 * (slot_of_entry[e] in 0..n_slots-1; every entry e < n_slots when the cache
 * was built without slot_of_entry).  out_score[q] / out_idx[q] = that
 * neighbour's score and entry, NaN / -1 when none of the k is resident (or
 * the entries are -1).  Passing out_score, out_idx with ld = 1 to apc_assign
 * and apc_gather_latents places each query at the level its best reusable
 * neighbour supports (level 0 when none) and gathers that latent.
 *
 * 1 <= k <= min(ld, APC_MAX_K); the cache must hold latents (n_slots > 0).
 * Errors: APC_E_ARG for bad sizes, NULL buffers or a cache without latents.
 */
apc_status apc_resident_best(const apc_cache* c, const float* top_score, const int32_t* top_idx, int32_t ld,
                             int32_t k, int32_t b, float* out_score, int32_t* out_idx, void* stream);

/*
 * Level histogram of a batch (the demand H_K per optimal K that the
 * Optimal-K Predictor of the Resource Controller forecasts, and the Route-Plan
 * takes): hist[l] = #{q < b : level[q] == l}, l = 0..L; other values are not
 * counted.  level and hist are device buffers (b and L + 1 int32);
 * 0 <= L <= APC_MAX_LEVELS.  Errors: APC_E_ARG.
 */
apc_status apc_level_histogram(const int32_t* level, int32_t b, int32_t L, int32_t* hist, void* stream);

/*
 * Latent gather (the cached intermediate state a placed prompt starts from:
 * the Introduction's reuse of a prior prompt's intermediate state, which
 * skips K denoising steps, and the Query Dispatcher's route-and-batch, which
 * hands every worker its batch): for each query with out_level > 0 whose
 * top-1 entry top_idx[q * ld] has a resident latent, copy it to
 * batch_latents[(out_inst * slots_per_inst + out_slot) * latent_bytes] and
 * set hit[q] = 1; otherwise hit[q] = 0 and that batch slot is not written.
 * out_slot must be < slots_per_inst for every copied query (as apc_assign
 * produces with slots_per_inst >= max capacity).
 */
apc_status apc_gather_latents(const apc_cache* c, const int32_t* top_idx, int32_t ld, int32_t b,
                              const int32_t* out_level, const int32_t* out_inst,
                              const int32_t* out_slot, int32_t n_inst, int32_t slots_per_inst,
                              void* batch_latents, int32_t* hit, void* stream);

/*
 * Latent gather at the assigned level (the cached state after K skipped steps
 * depends on K, Introduction and Approach): as apc_gather_latents, with
 * levels_per_slot latents per resident slot of cache c, level-major inside the
 * slot: the latent of slot s at level l is latents row s * levels_per_slot +
 * l - 1.  A query placed at level l > 0 copies its entry's latent of level l
 * (no copy, hit = 0, when l > levels_per_slot).  levels_per_slot = 1 is
 * apc_gather_latents (one latent per entry, used at every level).  The
 * cache's n_slots counts latents, so it must be a multiple of levels_per_slot,
 * and slot_of_entry values index the n_slots / levels_per_slot entry slots
 * (larger ones are not resident).  1 <= levels_per_slot <= APC_MAX_LEVELS.
 */
apc_status apc_gather_latents_at_level(const apc_cache* c, const int32_t* top_idx, int32_t ld, int32_t b,
                                       const int32_t* out_level, const int32_t* out_inst, const int32_t* out_slot,
                                       int32_t n_inst, int32_t slots_per_inst, int32_t levels_per_slot,
                                       void* batch_latents, int32_t* hit, void* stream);

/*
 * Merge of the top-k lists of row shards of one cache (not a step of the
 * paper: the layout for a cache split by rows over g devices, where each runs
 * apc_match_batch on its shard, the lists are exchanged, and every device
 * merges them; the paper's nearest-cache retrieval is the whole cache's
 * top-k, which this reproduces).  scores / idx: g x b x k_in
 * lists as the shards' apc_match_batch calls wrote them (shard s's block at
 * s * b * k_in, best first, entries local to the shard), contiguous as an
 * all-gather leaves them.  offsets (host) g global entry numbers of the
 * shards' first rows.  out_score / out_idx: b x k, the best k of all shards'
 * candidates under (score desc, global entry asc); entries < 0, NaN scores
 * and global entry numbers (entry + offset, summed in 64 bits) of 2^31 - 1
 * or more are not candidates, and slots past the last candidate get NaN / -1.
 * Since every entry of the whole cache's top-k is in its shard's top-k, the
 * merge of the shards' top-k lists is the whole cache's top-k.
 * 1 <= g <= APC_MAX_SHARDS, 1 <= k, k_in <= APC_MAX_K, offsets >= 0.
 * Errors: APC_E_ARG.
 */
apc_status apc_merge_shards(const float* scores, const int32_t* idx, int32_t g, int32_t b, int32_t k_in,
                            const int32_t* offsets /* host */, int32_t k, float* out_score, int32_t* out_idx,
                            void* stream);

/*
 * Measurement hook (for benchmarks and profilers, not for the method):
 * the next apc_match_batch call on this thread records `start` (a
 * hipEvent_t) on its stream right before the similarity/top-k kernel and
 * `stop` right after it, then forgets both.  NULL, NULL clears the hook.
 */
apc_status apc_set_kernel_events(void* start, void* stop);

const char* apc_status_str(apc_status s);
const char* apc_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* APC_H */
