/*
 * finemoe_map.h - C ABI of the expert-map matching and prefetch-selection
 * library for AMD Instinct MI355X (gfx950).
 *
 * The library implements the per-iteration search of FineMoE (arXiv
 * 2502.05370): a batch of queries is scored by cosine similarity against a
 * GPU-resident store of historical iterations, the best stored iteration(s)
 * are kept per query, and the matched expert map is turned into per-layer
 * expert prefetch sets by probability thresholding.
 *
 *   expert map (Section 4.1)      L rows of E gate probabilities, one row per
 *                                 MoE layer (the paper's J experts are E here)
 *   semantic search (Eq. 4)       cosine of embedding-layer outputs
 *   trajectory search (Eq. 5)     cosine of the first p observed layers of
 *                                 gate probabilities, flattened
 *   threshold (Section 4.3)       fixed tau, or delta = Clip(1 - score, 0, 1)
 *   prefetch set (Eq. 6-8)        fewest experts, highest probability first,
 *                                 whose summed probability reaches the
 *                                 threshold, clamped to [k_min, k_max]
 *
 * Conventions shared by every call:
 *   - All pointers marked "device" are HIP device pointers owned by the
 *     caller; the library never allocates device memory and never frees a
 *     caller buffer.  A store handle only borrows its buffer.
 *   - Work is enqueued asynchronously on the given stream (a hipStream_t
 *     passed as void*; NULL means the null stream).  Outputs are valid once
 *     the caller has synchronised that stream.  No call synchronises the
 *     stream except fm_store_check.
 *   - Arguments are validated on the host before anything is enqueued; an
 *     invalid call returns a non-zero fm_status, enqueues nothing and leaves
 *     every output untouched.  fm_last_error() then describes the problem
 *     (thread-local, valid until the next call on the same thread).
 *   - Ranking order is (score descending, store index ascending); a NaN
 *     score ranks below every number.  Missing matches (an empty store, or
 *     k larger than the store) are returned as index -1 and score -inf, and
 *     select nothing.
 *   - bf16 values are IEEE-754 binary32 values truncated to their upper 16
 *     bits (as produced by round-to-nearest-even), stored as uint16.
 */
#ifndef FINEMOE_MAP_H
#define FINEMOE_MAP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FM_OK = 0,
    FM_ERR_INVALID = 1,      /* bad argument: NULL pointer, out-of-range size or parameter */
    FM_ERR_UNSUPPORTED = 2,  /* valid but not implemented (e.g. E > 64, d_emb not a multiple of 128) */
    FM_ERR_FULL = 3,         /* insert would exceed the store capacity */
    FM_ERR_HIP = 4,          /* a HIP runtime call failed (message from the runtime) */
    FM_ERR_DEVICE = 5        /* fm_store_check found a sticky device-side range error */
} fm_status;

/* The argument enums below end in a 32-bit sentinel so that any int a caller
 * passes is a value of the type, which the library then checks and rejects
 * if it is not one of the listed ones (FM_ERR_INVALID); the sentinels are not
 * valid arguments. */
typedef enum { FM_F32 = 0, FM_BF16 = 1, FM_DTYPE_ENUM_INT32_ = 0x7fffffff } fm_dtype;

/* Threshold of Section 4.3: FIXED uses params.tau for every layer; DYNAMIC
 * uses delta = Clip(1 - score, 0, 1) with the best match's score (a NaN score
 * gives delta = 1). */
typedef enum { FM_TAU_FIXED = 0, FM_TAU_DYNAMIC = 1, FM_TAU_ENUM_INT32_ = 0x7fffffff } fm_tau_mode;

/* Which probabilities guide a layer: NONE = the layer's row of the best match
 * (Sections 4.2.1 and 4.2.2 use the single highest-scoring map); SCORE = the
 * similarity-weighted mean of that row over the k kept matches, with weights
 * max(score, 0) (plain mean if every weight is 0). */
typedef enum { FM_BLEND_NONE = 0, FM_BLEND_SCORE = 1, FM_BLEND_ENUM_INT32_ = 0x7fffffff } fm_blend;

/* Which Section 4.5 priority fm_priority_order ranks by. */
typedef enum { FM_PRI_PREFETCH = 0, FM_PRI_EVICT = 1, FM_PRI_ENUM_INT32_ = 0x7fffffff } fm_pri_kind;

/* Sticky device-side flags reported by fm_store_check. */
#define FM_FLAG_DEPTH_CLAMPED 0x1u   /* a trajectory depth was outside [1, max_depth] and was clamped */
#define FM_FLAG_INDEX_RANGE   0x2u   /* fm_select_prefetch met an index >= the store size (row skipped) */
#define FM_FLAG_STATE_STALE   0x4u   /* fm_traj_step: the store size changed since layer 0, or layers out of order */
#define FM_FLAG_VALUE_RANGE   0x8u   /* a float32 map or trajectory-query value exceeds 8 in magnitude (gate
                                        probabilities lie in [0, 1]); float32 trajectory scores are then unspecified */

typedef struct fm_store fm_store;   /* opaque host-side handle */

typedef struct {
    int32_t cap;         /* capacity C in stored iterations, >= 1 */
    int32_t L;           /* MoE layers, 1..64 */
    int32_t E;           /* experts per layer, 1..64 (a prefetch set is a 64-bit mask) */
    int32_t d_emb;       /* semantic embedding size (hidden size h); 0 = no embeddings,
                            otherwise a positive multiple of 128 */
    fm_dtype map_dtype;  /* element type of stored maps and trajectory queries */
    void* buffer;        /* device, at least fm_store_bytes(...) bytes, 256-byte aligned */
    size_t buffer_bytes;
} fm_store_desc;

typedef struct {
    fm_tau_mode mode;
    float tau;           /* FIXED threshold; compared as the exact float value */
    int32_t k_min;       /* Eq. 8 floor (the model's K), 0 <= k_min <= k_max */
    int32_t k_max;       /* cap on the set size, k_max <= E */
    fm_blend blend;
} fm_select_params;

/* Bytes of the layer-major map planes alone: L planes of cap (rounded up to
 * 16) rows of E elements rounded up to a multiple of 4 (the padding is stored
 * as zeros), each plane padded to 256 bytes.  Inside a plane the maps are
 * stored in tiles of 16: for every quad of 4 consecutive experts, the tile's
 * 16 rows of that quad are contiguous.  For cap = 32768 maps of 24 x 60
 * float32 (Section 6.8's largest store, Qwen1.5-MoE shape) this is
 * 188,743,680 bytes. */
size_t fm_map_bytes(int32_t cap, int32_t L, int32_t E, fm_dtype map_dtype);

/* Bytes of the whole device buffer a store needs: map planes, the prefix
 * inverse norms 1/|x[y][0:l+1]| of every map at every depth (L x cap float32,
 * cap rounded up to 64, computed at insert time in float64), embeddings
 * (cap x d_emb bf16), their float32 norms and 256 bytes of device flags, each
 * part 256-byte aligned.  Returns 0 for invalid sizes. */
size_t fm_store_bytes(int32_t cap, int32_t L, int32_t E, int32_t d_emb, fm_dtype map_dtype);

/* Bytes of match workspace for a store of L layers of E experts (map_dtype)
 * and d_emb embedding dimensions (0 or a multiple of 128), serving batches of
 * up to B_max queries keeping up to k_max matches each (device memory,
 * 256-byte aligned, owned by the caller).  It holds the staged queries of one
 * launch (depth-sorted trajectory planes, or tiled semantic embeddings), the
 * query norms and the per-workgroup partial top-k lists.  Every match call
 * rewrites what it reads, so the contents need no initialisation.  Calls that
 * share a workspace must be ordered (same stream, or synchronised); concurrent
 * calls on one workspace race.  Returns 0 for invalid arguments. */
size_t fm_workspace_bytes(int32_t L, int32_t E, int32_t d_emb, fm_dtype map_dtype, int32_t B_max,
                          int32_t k_max);

/* Create a host handle over a caller-owned device buffer (Expert Map Store,
 * Section 4.4).  The store starts empty.  The buffer contents are not read;
 * the current HIP device at this call is the store's device.  Errors:
 * FM_ERR_INVALID for NULL pointers, out-of-range sizes or a short or
 * misaligned buffer; FM_ERR_UNSUPPORTED for E or L above 64, a d_emb that is
 * not a multiple of 128, or map planes so large that one group of layer
 * planes scanned together (32/E planes when E in {8, 16, 32}, else one)
 * exceeds 0xF0000000 bytes (e.g. cap above ~15.7 million maps of 64 float32
 * experts). */
fm_status fm_store_build(fm_store** out, const fm_store_desc* desc);

/* Append n iterations (Step 5 of Section 3.2: new expert maps enter the
 * store).  maps: device [n][L][E] of map_dtype, map-major; embs: device
 * [n][d_emb] bf16, 16-byte aligned, required when d_emb > 0 and ignored
 * otherwise.  The maps
 * are transposed into the layer-major planes, and their prefix norms and the
 * embedding norms are computed.  slots_out: device [n] int32 receiving the store index of each
 * inserted iteration, or NULL.  FM_ERR_FULL if size + n > cap (nothing is
 * inserted).  n == 0 is a no-op. */
fm_status fm_store_insert(fm_store* store, const void* maps, const void* embs, int32_t n,
                          int32_t* slots_out, void* stream);

/* Bytes of scratch (device memory owned by the caller, 256-byte aligned)
 * that fm_store_insert_dedup needs for batches of up to n_max new iterations
 * on a store of capacity cap: two dense float32 matrices of n_max x cap
 * scores plus 72 KB of index arrays.  Returns 0 unless cap >= 1 and
 * 1 <= n_max <= 1024. */
size_t fm_dedup_scratch_bytes(int32_t cap, int32_t n_max);

/* Insert with deduplication (Section 4.4, Expert map deduplication).  maps,
 * embs and slots_out as for fm_store_insert, 1 <= n <= 1024 (n == 0 is a
 * no-op).  While the store has room, new iterations are appended in batch
 * order.  The rest replace stored iterations: for each such new iteration x
 * the redundancy score against every iteration y stored before this call is
 *     RDY[x][y] = (d/L) score_sem[x][y] + ((L-d)/L) score_traj[x][y]
 * with d = prefetch_distance (0..L), score_sem the Eq. 4 cosine of the
 * embeddings and score_traj the Eq. 5 cosine over all L layers, both as the
 * match calls compute them (float32), weighted in float64 and rounded to
 * float32; a term with weight 0 is not computed.  In batch order, each x
 * overwrites the y with the highest RDY (lower index on equal values, NaN
 * last) that no earlier x of this call took; an x left without a candidate
 * (a store of fewer than n entries) is dropped and gets slot -1.  The
 * store size becomes min(size + n, cap).
 * workspace: as for the match calls, sized with B_max >= n.  scratch: at least
 * fm_dedup_scratch_bytes(cap, n) bytes, rewritten by the call.  Calls sharing
 * a workspace or scratch must be ordered.
 * Errors: FM_ERR_INVALID for NULL or misaligned pointers, n or d out of
 * range, d > 0 on a store without embeddings, or a short workspace or
 * scratch; nothing is enqueued then. */
fm_status fm_store_insert_dedup(fm_store* store, const void* maps, const void* embs, int32_t n,
                                int32_t prefetch_distance, int32_t* slots_out, void* workspace,
                                size_t workspace_bytes, void* scratch, size_t scratch_bytes, void* stream);

/* Current number of stored iterations (host-side count, no synchronisation). */
fm_status fm_store_size(const fm_store* store, int32_t* n_out);

/* Synchronise the stream, read and clear the sticky device flags
 * (FM_FLAG_*).  Returns FM_ERR_DEVICE when any flag was set; *flags_out (may
 * be NULL) receives them. */
fm_status fm_store_check(fm_store* store, void* stream, uint32_t* flags_out);

/* Release the host handle (the caller's buffer is untouched). */
fm_status fm_store_destroy(fm_store* store);

/* Semantic search, Eq. 4: for each query embedding q[b] (device [B][d_emb]
 * bf16, 16-byte aligned) the k stored iterations with the highest cosine
 * q[b].x[y] / (|q[b]| |x[y]|) over y < size, accumulated in float32.  A zero
 * norm gives score 0.  Outputs: idx_out device [B][k] int32, score_out device
 * [B][k] float32, in ranking order.  1 <= k <= 8, 1 <= B <= 65536.
 * FM_ERR_INVALID if the store has no embeddings, q is misaligned or the
 * workspace is too small. */
fm_status fm_match_semantic(const fm_store* store, const void* q, int32_t B, int32_t k,
                            int32_t* idx_out, float* score_out,
                            void* workspace, size_t workspace_bytes, void* stream);

/* Trajectory search, Eq. 5: query b observed its first p_b = depth[b] layers
 * (device [B] int32); q is device [B][L][E] of map_dtype, map-major, and rows
 * l >= p_b are never read.  Score = cosine between q[b][0:p_b] and
 * x[y][0:p_b], both flattened over (layer, expert), accumulated in float32.
 * max_depth (1..L) is a host-side bound on the depths that sizes the scan;
 * a depth outside [1, max_depth] is clamped and sets FM_FLAG_DEPTH_CLAMPED.
 * Outputs and limits as for fm_match_semantic. */
fm_status fm_match_trajectory(const fm_store* store, const void* q, const int32_t* depth,
                              int32_t max_depth, int32_t B, int32_t k,
                              int32_t* idx_out, float* score_out,
                              void* workspace, size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * fm_match_trajectory without a workspace argument.  Its workspace is a
 * device array of the library of FM_NOALLOC_SCRATCH_BYTES, one per GPU,
 * which every GPU the call runs on holds until the process ends; its address
 * is looked up on the first call on each device.  The call allocates and
 * frees nothing.  Arguments, results, limits and errors as for
 * fm_match_trajectory, plus FM_ERR_UNSUPPORTED when a trajectory search of
 * the store's L x E needs more workspace than the array holds (no shape with
 * L, E <= 64 does) and FM_ERR_HIP when the array's address cannot be
 * obtained.  All calls on one GPU share the array: calls that overlap in time
 * on one GPU (other streams, or host threads without ordering) race, and
 * their results are unspecified.  Nothing in it needs to start at zero
 * (every call rewrites what it reads). */
#define FM_NOALLOC_SCRATCH_BYTES (40u << 20)
fm_status fm_match_trajectory_noalloc(const fm_store* store, const void* q, const int32_t* depth,
                                      int32_t max_depth, int32_t B, int32_t k, int32_t* idx_out,
                                      float* score_out, void* stream);

/* Prefetch sets, Section 4.3 (Eq. 6-8): for query b and every layer l in
 * [layer_begin[b], layer_end[b]) (device [B] int32 each, clamped to [0, L]),
 * take the guiding probabilities (fm_blend), the threshold (fm_tau_mode) from
 * score[b][0], order the experts by probability (descending, lower expert
 * index first on equal values), find the smallest k* whose running float64
 * sum of the first k* reaches the threshold (k* = E if none does) and keep
 * the first min(max(k*, k_min), k_max).  idx/score: device [B][k] as written
 * by a match call.  mask_out: device [B][L] uint64, bit j = expert j;
 * count_out: device [B][L] uint8.  Layers outside the range, and queries whose
 * idx[b][0] is -1, get mask 0 and count 0. */
fm_status fm_select_prefetch(const fm_store* store, const int32_t* idx, const float* score,
                             int32_t B, int32_t k, const int32_t* layer_begin,
                             const int32_t* layer_end, const fm_select_params* params,
                             uint64_t* mask_out, uint8_t* count_out, void* stream);

/* A match call and the selection of its rows in one call: the semantic
 * search of Section 4.2.1 (Eq. 4) or the trajectory search of Section 4.2.2
 * (Eq. 5), then the prefetch sets of Section 4.3 (Eq. 6-8) of every row of
 * the batch, with the merge of the search's per-workgroup lists and the
 * selection in one launch.  Arguments, results and errors as for
 * fm_match_semantic / fm_match_trajectory followed by fm_select_prefetch on
 * the same B rows with the same k: idx_out/score_out receive the matches
 * (device [B][k]), mask_out/count_out the sets (device [B][L]); layer_begin,
 * layer_end and params as for fm_select_prefetch.  The results are those of
 * the two separate calls. */
fm_status fm_match_semantic_select(const fm_store* store, const void* q, int32_t B, int32_t k,
                                   const int32_t* layer_begin, const int32_t* layer_end,
                                   const fm_select_params* params, int32_t* idx_out, float* score_out,
                                   uint64_t* mask_out, uint8_t* count_out, void* workspace,
                                   size_t workspace_bytes, void* stream);
fm_status fm_match_trajectory_select(const fm_store* store, const void* q, const int32_t* depth,
                                     int32_t max_depth, int32_t B, int32_t k, const int32_t* layer_begin,
                                     const int32_t* layer_end, const fm_select_params* params,
                                     int32_t* idx_out, float* score_out, uint64_t* mask_out,
                                     uint8_t* count_out, void* workspace, size_t workspace_bytes,
                                     void* stream);

/* Misses of prefetch sets (Section 3: R_{l,j} = 1 iff expert j of layer l is
 * activated and not cached).  q: device [B][L][E] of map_dtype, each query's
 * own gate probabilities (the experts its layers actually route to); the
 * activated experts of a row are its K highest (lower expert index first on
 * equal values, NaN last), the cached ones its prefetch set (masks: device
 * [B][L] uint64 as written by fm_select_prefetch).  miss_out: device [B][L]
 * uint8, the number of activated experts outside the set for layers in
 * [layer_begin[b], layer_end[b]) (clamped to [0, L]), 0 elsewhere.
 * 1 <= K <= E, 1 <= B <= 65536.  Errors: FM_ERR_INVALID for NULL pointers or
 * out-of-range arguments; nothing is enqueued then. */
fm_status fm_miss_count(const fm_store* store, const void* q, int32_t B, int32_t K, const uint64_t* masks,
                        const int32_t* layer_begin, const int32_t* layer_end, uint8_t* miss_out, void* stream);

/* Expert priorities of Section 4.5, one ordered list per query.
 * FM_PRI_PREFETCH: the candidates are the experts of query b's prefetch set
 * (masks: device [B][L] uint64 as written by fm_select_prefetch) in the
 * layers after its current layer, l > l_now[b] (l_now: device [B] int32,
 * 0-based; -1 lists every layer); PRI = p_{l,j} / (l - l_now[b]).
 * FM_PRI_EVICT: the candidates are the cached experts (masks: device [L]
 * uint64, bit j of layer l = expert cached, one mask for all queries);
 * PRI = 1 / (p_{l,j} * freq[l][j]) with freq device [L][E] float32 visit
 * counts (p * freq = 0 gives +inf).  p_{l,j} is the query's guiding
 * probability, exactly as fm_select_prefetch computes it from idx/score/blend.
 * PRI is computed in float64 and rounded to float32.  Each query's
 * candidates are ordered by PRI descending, the lower l * E + j first on
 * equal values, NaN last; the first cap are written: order_out device
 * [B][cap] int32 (l * E + j, -1 past the candidates), pri_out device [B][cap]
 * float32 (-inf past the candidates); count_out device [B] int32 receives
 * the number of candidates.  A query whose idx[b][0] is -1 has none (an
 * index >= the store size also sets FM_FLAG_INDEX_RANGE).  1 <= k <= 8,
 * 1 <= B <= 65536, 1 <= cap <= 4096.  Errors: FM_ERR_INVALID for NULL
 * pointers (l_now for PREFETCH, freq for EVICT) or out-of-range arguments;
 * nothing is enqueued then. */
fm_status fm_priority_order(const fm_store* store, const int32_t* idx, const float* score, int32_t B, int32_t k,
                            fm_blend blend, fm_pri_kind kind, const uint64_t* masks, const int32_t* l_now,
                            const float* freq, int32_t cap, int32_t* order_out, float* pri_out,
                            int32_t* count_out, void* stream);

/* Bytes of state (device memory owned by the caller, 256-byte aligned) for
 * fm_traj_step passes of up to B_max queries (1..65536) on a store of
 * capacity cap: per group of 64 queries a 1,280-byte header (store size at
 * layer 0, last layer, float64 running query sums of squares in two slots)
 * and the running float32 dot products of each query with each stored map
 * (cap rounded up to 16, 4 query tiles of 16): 1,280 + 1,024 * ceil(cap / 16)
 * * 4 bytes per group, each group 256-byte aligned.
 * 0 for invalid arguments. */
size_t fm_traj_state_bytes(int32_t cap, int32_t B_max);

/* Incremental trajectory re-search (Section 4.2.2: after each newly observed
 * layer the trajectory search runs again with the prefix grown by one layer).
 * q_layer: device [B][E] of map_dtype, each query's gate probabilities at
 * layer `layer` (0-based).  layer == 0 starts a pass and overwrites the
 * state; every later call of the pass passes the next layer for the same B
 * queries, in the same order, on an unchanged store.  The state keeps the
 * running dot product of every (query, stored map) pair, so a step reads one
 * layer plane of the store instead of layer + 1.  Outputs as for
 * fm_match_trajectory with depth[b] = layer + 1 for every b (Eq. 5 over the
 * first layer + 1 layers, float32 accumulation, rows of the store beyond its
 * size at the call never ranked).  A step whose store size differs from the
 * size at layer 0, or whose layer does not follow the previous one, sets
 * FM_FLAG_STATE_STALE and its results are unspecified.  1 <= k <= 8,
 * 1 <= B <= 65536, 0 <= layer < L.  Errors: FM_ERR_INVALID for NULL or
 * misaligned pointers, out-of-range arguments, or a short state or
 * workspace; nothing is enqueued then. */
fm_status fm_traj_step(fm_store* store, void* state, size_t state_bytes, const void* q_layer, int32_t layer,
                       int32_t B, int32_t k, int32_t* idx_out, float* score_out, void* workspace,
                       size_t workspace_bytes, void* stream);

/* Test support: the dense float32 score matrix of a trajectory (q, depth
 * non-NULL) or semantic (q_sem non-NULL) search, written to scores_out device
 * [B][size] by the same kernels and arithmetic as the match calls.
 * Exactly one of q / q_sem must be non-NULL. */
fm_status fm_debug_scores(const fm_store* store, const void* q, const int32_t* depth,
                          int32_t max_depth, const void* q_sem, int32_t B, float* scores_out,
                          void* workspace, size_t workspace_bytes, void* stream);

/* Measurement support: start and stop are hipEvent_t handles (passed as
 * void*) created by the caller, or both NULL to switch this off.  While set,
 * every match call made on this thread records start on its stream right
 * before the launch of its scan kernel (k_traj_scan or k_sem_scan; k_traj_step
 * for fm_traj_step) and stop right after it, so the events bracket exactly
 * that kernel (for a batch of more than one launch, the last launch's).  The library does not own or
 * destroy the events.  FM_ERR_INVALID if exactly one of them is NULL. */
fm_status fm_debug_scan_events(void* start, void* stop);

/* Description of the last non-OK status on this thread ("" if none). */
const char* fm_last_error(void);

/* ABI version: (major << 16) | minor. */
int32_t fm_version(void);

#ifdef __cplusplus
}
#endif

#endif /* FINEMOE_MAP_H */
