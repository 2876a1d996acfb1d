/*
 * lodestar.h -- C ABI of the MI355X (gfx950) batched routing scorer.
 *
 * The library implements the data-parallel hot path of Lodestar's learned
 * router (arXiv 2606.00946): for every pending (request, instance) pair it
 * measures the prefix-cache overlap of the request's block-hashed prompt with
 * the instance's cached blocks, assembles the pair's feature row, runs the
 * shared reward model and picks, per request, the instance with the smallest
 * predicted TTFT (Section 4.1, Alg. 4).  It also applies one online SGD step to
 * that model from logged (features, observed TTFT) rows (Section 4.3.2).
 *
 * Conventions shared by every entry point
 *   - Every function returning int returns LS_OK (0) or a negative LS_ERR_*.
 *     No C++ exception crosses the ABI.  ls_last_error() describes the last
 *     failure on that context.
 *   - Arguments are validated on the host before anything is enqueued; an
 *     invalid call enqueues nothing and leaves the library state unchanged.
 *   - Device pointers are caller-owned HIP device memory (for example torch
 *     tensors on the current device); the caller keeps them alive and
 *     unmodified until the work enqueued on `stream` has finished.
 *   - `stream` is a hipStream_t (NULL: the legacy default stream).  Work is
 *     asynchronous and ordered on that stream; library state (model, cache
 *     state, workspace) is ordered by the stream of each call, so callers that
 *     use several streams must order them themselves.
 *   - A context is not thread-safe: use one per host thread, or serialise.
 *   - The library owns its tables, model copies and workspace (hipMalloc);
 *     workspace grows on demand, so a call that needs more than any earlier
 *     call may allocate.  Growth is ordered on the call's stream (the
 *     stream-ordered allocator: the old buffer is freed after the work already
 *     enqueued on that stream), so it neither waits for the device nor stalls
 *     other streams.
 */
#ifndef LODESTAR_H
#define LODESTAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LS_OK 0
#define LS_ERR_INVALID (-1)      /* bad argument, shape or null pointer */
#define LS_ERR_NOMEM (-2)        /* device or host allocation failed */
#define LS_ERR_DEVICE (-3)       /* a HIP runtime call or kernel launch failed */
#define LS_ERR_STATE (-4)        /* no model or cache state yet, or an instance-count mismatch */
#define LS_ERR_UNSUPPORTED (-5)  /* valid request this build does not implement */

#define LS_FP32 0   /* fp32 weights and activations */
#define LS_BF16 1   /* bf16 weights and layer inputs, fp32 accumulation, fp32 master weights */

#define LS_MAX_HIDDEN 3
#define LS_DERIVED_COLS 5

typedef struct ls_ctx ls_ctx;

/*
 * Reward-model shape (Section 4.1, Model architecture and Features).
 *   d          feature columns of a pair row, d > LS_DERIVED_COLS.  The row is
 *              [ instance state (d - 5 columns) | L, n | l, kappa, u ]:
 *              L = prompt tokens, n = hashed blocks, l = overlap in blocks,
 *              kappa = block_tokens * l / L (0 when L = 0), u = L - block_tokens * l.
 *   n_hidden   hidden layers, 1..3 (Section 4.1 uses 3 x 128; the evaluated
 *              configurations here use 2).  Two-layer models are scored by
 *              fused kernels (bf16 ones on the matrix cores); other depths by a
 *              layer-by-layer forward over chunks of pair rows, with the same
 *              arithmetic order (bias first, inputs ascending).
 *   hidden     widths, each 1..512.
 *   block_tokens tokens per hashed KV block (16 in the evaluated engines).
 *   dtype      LS_FP32 or LS_BF16.
 */
typedef struct ls_model_config {
    int32_t d;
    int32_t n_hidden;
    int32_t hidden[LS_MAX_HIDDEN];
    int32_t block_tokens;
    int32_t dtype;
} ls_model_config;

/* Parameters of the packed model: for each layer d -> hidden[0] -> ... -> 1,
 * W [out x in] row-major, then b [out].  Returns -1 for an invalid shape. */
int64_t ls_param_count(const ls_model_config* cfg);

/* Create a context on HIP device `device`.  *out is NULL on failure. */
int ls_create(const ls_model_config* cfg, int device, ls_ctx** out);

/* Wait for the context's outstanding work, free everything it owns.  NULL is a no-op. */
void ls_destroy(ls_ctx* ctx);

/* Message of the last failed call on ctx (never NULL; valid until the next call). */
const char* ls_last_error(const ls_ctx* ctx);

/*
 * Install a model (Section 4.3.1, P2: the new model replaces the old one
 * atomically with respect to scoring).  Host arrays, copied before return:
 *   params     [ls_param_count] fp32, the packing above;
 *   mu         [d] per-feature mean, inv_sigma [d] per-feature 1/sigma
 *              (Alg. 4, per-feature z-score: x~ = (x - mu) * inv_sigma).
 * Scoring and update calls enqueued on `stream` after this one see the new
 * model.  LS_BF16 contexts keep fp32 masters and derive bf16 copies.
 */
int ls_set_model(ls_ctx* ctx, const float* params, int64_t n_params,
                 const float* mu, const float* inv_sigma, void* stream);

/* Copy the current fp32 master model to host arrays (any may be NULL).
 * Synchronous: waits for the work enqueued on the context's streams. */
int ls_get_model(ls_ctx* ctx, float* params, int64_t n_params, float* mu, float* inv_sigma);

/*
 * Replace the whole prefix-cache state (Section 4.2, Prefix KV cache tracker:
 * the gateway's index of which prompt blocks each instance holds).
 *   n_instances  N >= 1
 *   inst_off     HOST   int64 [N+1], inst_off[0] = 0, non-decreasing: instance
 *                i's hashes are hashes[inst_off[i] .. inst_off[i+1]).
 *   hashes       DEVICE uint64 [inst_off[N]], any order, duplicates allowed,
 *                every uint64 value allowed.  Read only during this call's
 *                stream work.
 * The library builds one hash table per instance on the device.  Instance ids
 * are positions 0..N-1, shared with the rows of inst_feat in ls_score_batch.
 * LS_ERR_UNSUPPORTED for 2^32 or more hashes in all (or, with capacities set,
 * capacities summing to that).
 */
int ls_load_cache_state(ls_ctx* ctx, int32_t n_instances, const int64_t* inst_off,
                        const uint64_t* hashes, void* stream);

/*
 * Prefix-index maintenance (Section 2: after routing a request the gateway
 * records its prefix blocks on the chosen instance, and each engine evicts its
 * least recently used KV blocks; Section 4.2: the index follows the gateway's
 * own routing history).  Every cached block carries a recency stamp.
 *
 * ls_set_cache_capacity
 *   capacity  HOST int64 [n_instances], blocks each instance holds (>= 0).
 *   The next ls_load_cache_state with n_instances instances keeps each
 *   instance's block list with stamps -- entry j of its loaded hashes gets
 *   stamp j + 1 (list order = oldest first; a repeated hash keeps its newest
 *   entry) -- and sizes its table for max(loaded, capacity) blocks.  To change
 *   capacities, set them and load again.  capacity = NULL turns maintenance
 *   off (the default).  LS_ERR_INVALID for a negative capacity.
 *
 * ls_commit_routes
 *   DEVICE req_off int64 [R+1], req_hashes uint64 [n_hashes = req_off[R]],
 *   chosen int32 [R]: request r's blocks go to instance chosen[r]; a value
 *   outside [0, N) leaves the request out (e.g. -1).  Block k of request r is
 *   touched with stamp
 *       epoch * 2^44 + r * 2^20 + (2^20 - 1 - k),
 *   epoch = commits since the load, from 1: later commits, later requests of
 *   a batch and blocks nearer the prompt's start are more recent (engines free
 *   a sequence's tail first, so what stays cached of a request is a prefix of
 *   it).  A block keeps its largest stamp.  Then every instance above its
 *   capacity keeps its `capacity` most recent blocks (stamps are unique per
 *   instance, so the set is exact), and the tables are rebuilt: later calls on
 *   the stream see the new state.  R <= 2^24 (LS_ERR_INVALID); at most
 *   2^20 - 2 commits per load (LS_ERR_STATE); n_r <= 2^20 is the caller's
 *   (later blocks share the last rank).  LS_ERR_STATE unless the state was
 *   loaded under ls_set_cache_capacity.  Asynchronous; the library-owned
 *   workspace grows (stream-ordered) when a batch needs more.
 *
 * ls_read_cache_state
 *   Synchronous.  inst_off HOST int64 [n_instances + 1] out: the lists'
 *   offsets.  hashes / stamps DEVICE uint64 [max_entries] out (either may be
 *   NULL): each instance's blocks and stamps, in no particular order.
 *   LS_ERR_INVALID if an array is given and max_entries < inst_off[N].
 */
int ls_set_cache_capacity(ls_ctx* ctx, int32_t n_instances, const int64_t* capacity);
int ls_commit_routes(ls_ctx* ctx, int32_t R, int64_t n_hashes, const int64_t* req_off,
                     const uint64_t* req_hashes, const int32_t* chosen, void* stream);
int ls_read_cache_state(ls_ctx* ctx, int32_t n_instances, int64_t* inst_off, uint64_t* hashes,
                        uint64_t* stamps, int64_t max_entries, void* stream);

/*
 * Score a batch of R requests against the N loaded instances (Section 4.1
 * greedy routing; Alg. 4 normalise -> batched forward -> argmax of reward,
 * here argmin of predicted TTFT, ties to the lowest instance id).
 * DEVICE inputs:
 *   req_off     int64 [R+1], req_off[0] = 0, non-decreasing; request r's block
 *               hashes are req_hashes[req_off[r] .. req_off[r+1]), in prompt order.
 *   req_hashes  uint64 [req_off[R]]
 *   prompt_len  int32 [R] prompt tokens L (normally >= block_tokens * n_r)
 *   inst_feat   fp32 [N x (d-5)] row-major instance-state columns
 * DEVICE outputs (all but `chosen` may be NULL):
 *   chosen      int32 [R]      argmin instance
 *   min_ttft    fp32  [R]      its predicted TTFT (s); the reward is the negation
 *   scores      fp32  [R x N]  every predicted TTFT, request-major
 *   overlap     int32 [R x N]  leading cached blocks l (Section 2: prefix reuse
 *                              is strictly sequential)
 *   feat_out    fp32  [R x d]  raw feature row of the chosen pair (the training record)
 * R = 0 is a no-op.  N must equal the loaded instance count (LS_ERR_STATE).
 * Every returned value is the canonical one (the fp32 fma chains, or in bf16
 * mode bf16 operands with fp32 fma chains, bias first, inputs ascending).  On an
 * LS_BF16 context a call with scores == NULL scores on the matrix cores and
 * rescores the candidate band canonically (ls_set_exact_scores); a call that asks
 * for `scores` runs the canonical chain on every pair, so that the whole matrix
 * is canonical (much slower at large R x N).
 */
int ls_score_batch(ls_ctx* ctx, int32_t R, int32_t N,
                   const int64_t* req_off, const uint64_t* req_hashes, const int32_t* prompt_len,
                   const float* inst_feat,
                   int32_t* chosen, float* min_ttft, float* scores, int32_t* overlap, float* feat_out,
                   void* stream);

/*
 * ls_score_batch for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, hosts that forbid allocation during
 * serving.  Same arguments, results and errors as ls_score_batch, but the call
 * allocates nothing (no hipMalloc, hipFree or allocating library routine): its
 * scratch is one array of LS_NOALLOC_SCRATCH_BYTES per GPU, reserved while the
 * library is loaded and shared by every context on that GPU.  A batch whose
 * scratch would exceed it (about 29 bytes per pair plus 33 MiB at most;
 * passing `overlap` and `scores` saves 8 bytes per pair) gets LS_ERR_INVALID
 * before anything is enqueued.  Each call clears what it needs, but the array
 * keeps the last call's contents: calls that overlap on one GPU (different
 * streams, contexts or host threads) race on it, so the caller serialises them.
 * The context's cache state, model and caller buffers must already exist.
 * Per-kernel profiling records are not taken by this call.
 */
#define LS_NOALLOC_SCRATCH_BYTES (96u << 20)
int ls_score_batch_noalloc(ls_ctx* ctx, int32_t R, int32_t N,
                           const int64_t* req_off, const uint64_t* req_hashes, const int32_t* prompt_len,
                           const float* inst_feat,
                           int32_t* chosen, float* min_ttft, float* scores, int32_t* overlap, float* feat_out,
                           void* stream);

/*
 * Scoring precision of an LS_BF16 context.  By default a call that does not ask
 * for the score matrix runs the bf16 model on the matrix cores; every candidate
 * whose fast score lies within the error band of its request's best (see
 * ls_fast_scores) is then rescored with the canonical chain, and the decision
 * (`chosen`) and `min_ttft` come from those canonical scores.  enable != 0 runs
 * the canonical chain on every pair of every call instead.  fp32 contexts
 * always use the canonical chain.  Takes effect for later scoring calls.
 */
int ls_set_exact_scores(ls_ctx* ctx, int enable);

/*
 * Which kernels run the canonical fp32 chains of ls_update (the forward layers
 * and the hidden layers' backpropagated gradients, Section 4.3.2) and of the
 * layer-by-layer scorer of models other than two hidden layers (Section 4.1).
 * mode 0 (the default): on the matrix cores wherever a call's batch fills the
 * device.  There v_mfma_f32_32x32x1_2b_f32 takes one input k per instruction
 * and rounds each multiply-add once, as fmaf does, so every chain keeps its
 * order and its bits.  mode 1: on the vector ALUs only.  The two give
 * bit-identical results; the switch exists to compare them.  LS_ERR_INVALID
 * for another mode.  Takes effect for later calls.
 */
int ls_set_chain_kernels(ls_ctx* ctx, int mode);

/*
 * Validation aid for the matrix-core path of an LS_BF16 context (Section 4.1,
 * the batched forward of Alg. 4): for every pair of the batch, the fast score t
 * before any rescoring and its error scale err = 2^-7 (sum_j |w3_j| h2_j + |b3|)
 * -- w3, b3 the output layer, h2 the pair's last hidden activations on the
 * matrix cores.  band (nullable) gets 1 for the pairs a scoring call would
 * rescore (t - err <= min over the request of t + err, or a non-finite value),
 * else 0.  DEVICE arrays: t, err fp32 [R x N], band uint8 [R x N], inputs as in
 * ls_score_batch.  Decisions are exact whenever |t - t_canonical| <= err for
 * every pair outside the band.  LS_ERR_UNSUPPORTED if the context's model does
 * not run on the matrix cores (fp32, or a shape without a matrix-core kernel).
 */
int ls_fast_scores(ls_ctx* ctx, int32_t R, int32_t N, const int64_t* req_off, const uint64_t* req_hashes,
                   const int32_t* prompt_len, const float* inst_feat, float* t, float* err, uint8_t* band,
                   void* stream);

/*
 * Launch geometry: persistent and grid-stride kernels are sized for n compute
 * units (n = 0: all of the device's; a larger n is clamped to them), e.g. to
 * leave part of the GPU to other work.  Every result is independent of n: the
 * kernels fix their summation orders and partitions by the data, not by the
 * grid.  LS_ERR_INVALID for n < 0.  Takes effect for later calls.
 */
int ls_set_cu_limit(ls_ctx* ctx, int n);

/*
 * How ls_score_batch finds the overlap of followers -- requests whose first
 * block hash is shared with a longer request of the batch (Section 2: reuse is
 * strictly sequential, so a follower's overlap equals the longer request's up
 * to their common prefix).  Beyond that prefix, the follower's next block is
 * either probed in every instance's table (mode 2), or first looked up in one
 * pass over all cached keys, so that only followers whose next block is cached
 * somewhere are probed (mode 1).  Mode 0 (the default) picks per call from the
 * pair count and the total table size.  The overlaps are identical in every
 * mode.  Returns LS_ERR_INVALID for other modes; takes effect for later calls.
 */
int ls_set_prefix_join(ls_ctx* ctx, int mode);

/*
 * Declares that every instance's cached set is prefix-closed for every prompt
 * of later ls_score_batch / ls_route_batch calls: if block j of a prompt is
 * cached on an instance, its blocks 0..j-1 are too (the state an engine's
 * tail-first LRU keeps, Section 2).  Whether a block is cached is then
 * monotone along the prompt, and the library finds each run's end by a
 * multi-way search (O(log n) probe rounds) instead of walking it.  The
 * overlaps are exact under the invariant; without it they may be wrong (never
 * out of [0, n]).  enable = 0 (the default) restores the general walk.
 */
int ls_set_prefix_closed(ls_ctx* ctx, int enable);

/*
 * One SGD step on the installed model (Section 4.3.2, online learning; the
 * loss and optimiser are this library's reading: mean squared error of the
 * predicted TTFT, plain SGD).  L = (1/B) sum_b (t_b - y_b)^2, W <- W - lr dL/dW.
 * DEVICE inputs:  feats fp32 [B x d] raw rows (same layout as feat_out),
 *                 ttft  fp32 [B] observed TTFT in seconds.
 * DEVICE outputs (nullable): loss_out fp32 [1] pre-step loss;
 *                 grad_out fp32 [ls_param_count] dL/dW in the parameter packing.
 * LS_BF16 contexts use bf16 GEMM operands (weights, layer inputs and each
 * layer's output gradient), fp32 accumulation and fp32 master weights.
 */
int ls_update(ls_ctx* ctx, int32_t B, const float* feats, const float* ttft, float lr,
              float* loss_out, float* grad_out, void* stream);

/*
 * Dropout while training (Section 4.1: the predictor is trained with dropout
 * 0.1): from the next ls_update / ls_train_round on, inverted dropout on every
 * hidden layer's activations, rate p in [0, 1) (0 turns it off), scoring
 * unaffected.  Update calls are counted from 0 at this call (each minibatch of
 * ls_train_round is one call).  In call s, unit j of hidden layer l for row b
 * of that call's batch draws the splitmix64 output number c + 1 for `seed`,
 *     c = ((s * 4 + l) * 2^24 + b) * 2^10 + j,
 * and is dropped when the draw's top 53 bits are below floor(p * 2^53).  A kept
 * unit's activation is multiplied by the fp32 value of 1 / (1 - p) (after the
 * ReLU, before any bf16 rounding of the next layer's input); its gradient gets
 * the same factor, a dropped unit's is 0.  Requires batches below 2^24 rows
 * (LS_ERR_INVALID from ls_update) and hidden widths up to 1024.
 */
int ls_set_dropout(ls_ctx* ctx, float p, uint64_t seed);

/*
 * Routing policy around the reward model.
 *
 * The gateway pre-computes a heuristic choice for every request and uses it
 * whenever the routing service signals a fallback (Alg. 3); the service itself
 * (Alg. 4) returns a fallback status on a cold start (fewer than n_min logged
 * samples) or when a feature lies outside the bounds seen in training (the
 * out-of-range guard of Section 4.3.1), explores uniformly with probability
 * epsilon, and otherwise routes greedily on the model, with two refinements:
 * when the cluster's KV cache is saturated and the request's best prefix
 * benefit is large, the choice is restricted to K instances picked by
 * consistent hashing of its prefix group (Section 4.1, Consistent hashing
 * based filtering), and a near-best set within a relative margin delta is
 * broken uniformly at random (the reward tiebreak).
 *
 * Heuristics: LS_HEUR_PREFIX_LOAD is the prefix-cache-and-load policy (Alg. 1):
 * the least-loaded instance when request counts differ by more than
 * theta_imbal, else the best prefix match (ties: fewer requests, lower id)
 * among instances whose count is at most mean + overload_k * std (population
 * statistics), else the least loaded.  LS_HEUR_PREFIX_THRESHOLD (Alg. 2)
 * takes the best prefix match if it exceeds prefix_tau, else the least loaded.
 * The prefix match ratio is the pair's kappa = 16 l / L; the request count
 * c_i is the sum of the instance-feature columns count_cols (-1 skips one).
 *
 * Readings of points the paper leaves open:
 *   - bounds cover the request columns (L, n) and the instance columns; the
 *     pair columns (l, kappa, u) are not checked.  lo/hi are host arrays of
 *     d floats (copied); NULL disables the guard.  lo <= v <= hi is in range.
 *   - the prefix group is the request's first block hash; the K instances are
 *     its rendezvous top-K: instance i weighs output i + 1 of splitmix64
 *     (Steele, Lea and Flood, 2014) seeded with the hash, heaviest first.
 *   - the benefit is max_i kappa_i * L in tokens; saturation is the mean of
 *     instance column kv_col over all instances, compared with tau_sat.
 *   - the near-best set is {i : t_i <= t* + delta |t*|} on predicted TTFT t
 *     (the printed form on rewards is empty for negative rewards), taken within
 *     the K instances when the filter applies; delta < 0 disables the
 *     tie-break (lowest id wins ties then).
 *   - random draws come from the caller: rnd holds three uniform uint32 words
 *     per request (device, [R x 3]): exploration draw u0 (explore when
 *     u0 < floor(epsilon * 2^32)), exploration pick u1 and tie-break pick u2,
 *     a pick from n choices being (u * n) >> 32 over the choices in ascending
 *     instance order.  rnd may be NULL only when epsilon == 0 and delta < 0.
 * Decisions are exact: on the bf16 matrix-core path every pair that can be
 * the greedy choice, a member of the near-best set or one of the K filtered
 * instances is rescored with the canonical chain first.
 */
#define LS_HEUR_PREFIX_LOAD 1
#define LS_HEUR_PREFIX_THRESHOLD 2

#define LS_ROUTE_OK 0
#define LS_ROUTE_COLD_START 1     /* fallback: not enough samples yet (chosen = heuristic) */
#define LS_ROUTE_OOD 2            /* fallback: a feature outside the bounds (chosen = heuristic) */
#define LS_ROUTE_EXPLORED 0x100   /* flag on LS_ROUTE_OK: uniform exploration */
#define LS_ROUTE_KFILTER 0x200    /* flag on LS_ROUTE_OK: the choice was restricted to the K instances */
#define LS_ROUTE_TIEBREAK 0x400   /* flag on LS_ROUTE_OK: drawn from a near-best set of two or more */

#define LS_MAX_KFILTER 8

typedef struct {
    int32_t heuristic;        /* LS_HEUR_PREFIX_LOAD or LS_HEUR_PREFIX_THRESHOLD */
    int32_t count_cols[2];    /* instance-feature columns summed into the request count */
    float theta_imbal;        /* Alg. 1 imbalance threshold */
    float overload_k;         /* Alg. 1 overload factor */
    float prefix_tau;         /* Alg. 2 prefix-hit threshold */
    int64_t n_samples;        /* logged samples so far */
    int64_t n_min;            /* cold-start threshold */
    const float* lo;          /* host [d] or NULL */
    const float* hi;          /* host [d] or NULL */
    float epsilon;            /* exploration rate in [0, 1] */
    int32_t kv_col;           /* instance-feature column of KV-cache utilisation, -1: no K-filter */
    float tau_sat;            /* saturation threshold on the mean of kv_col */
    float tau_ben;            /* benefit threshold on max_i kappa_i * L (tokens) */
    int32_t k_filter;         /* K in [0, LS_MAX_KFILTER]; 0: no K-filter */
    float delta;              /* tie-break margin; < 0: no tie-break */
} ls_policy;

/*
 * Scores a batch like ls_score_batch and then routes every request with the
 * policy above.  Inputs as for ls_score_batch, plus rnd.  Outputs (device):
 *   chosen   int32 [R]      the instance the request is forwarded to
 *   status   int32 [R]      LS_ROUTE_* code and flags (nullable)
 *   heur     int32 [R]      the heuristic's choice (nullable)
 *   feat_out fp32  [R x d]  raw feature row of the chosen pair (nullable)
 * LS_ERR_INVALID for a bad policy (unknown heuristic, column out of range,
 * k_filter outside [0, LS_MAX_KFILTER], NaN parameters, missing rnd).
 */
int ls_route_batch(ls_ctx* ctx, const ls_policy* policy, int32_t R, int32_t N,
                   const int64_t* req_off, const uint64_t* req_hashes, const int32_t* prompt_len,
                   const float* inst_feat, const uint32_t* rnd,
                   int32_t* chosen, int32_t* status, int32_t* heur, float* feat_out, void* stream);

/*
 * Online-learning data path (Section 4.3.2, Training-data selection).
 *
 * The context keeps a FIFO of the newest fifo_cap logged samples and a replay
 * pool of up to replay_cap older ones on the device.  Samples the FIFO evicts
 * (oldest first) are offered to the pool by a gradient-coreset rule: a
 * sample's embedding is its prediction residual times its last-hidden-layer
 * activations, (t - y) a_L -- the output-weight gradient of the squared loss,
 * from the current model in kernel precision, with distances in double.  A
 * pool with room takes the sample; a full pool takes it in place of its most
 * redundant member (smallest nearest-neighbour distance, lowest slot on ties)
 * when the sample's distance to the pool is larger.  Embeddings are
 * re-evaluated with the current model at every push.  A retraining round runs
 * minibatch SGD (ls_update steps) over the FIFO and the pool.
 *
 *   ls_buffer_init   allocates empty pools (fifo_cap >= 1, 0 <= replay_cap <=
 *                    LS_MAX_REPLAY: the pool keeps its pairwise distances,
 *                    8 replay_cap^2 bytes); synchronous; discards any earlier
 *                    contents.
 *   ls_buffer_push   appends B raw rows feats [B x d] and ttft [B] (device);
 *                    admitted (device int32, nullable) gets the number of
 *                    samples the pool took.  Stream-ordered.
 *   ls_buffer_state  host counters: FIFO size, FIFO ring start, pool size.
 *   ls_buffer_read   copies the FIFO (oldest first, [fifo_count x d] and
 *                    [fifo_count]) and the pool (by slot) to device arrays
 *                    (each nullable).  Stream-ordered.
 *   ls_train_round   epochs passes over the n = FIFO + pool samples, sample k
 *                    being the k-th oldest FIFO entry for k < FIFO size and
 *                    pool slot k - FIFO size after it.  perm (host, nullable)
 *                    gives each epoch's visiting order as epochs rows of a
 *                    permutation of [0, n) (NULL: natural order); minibatches
 *                    of `batch` in that order, the last one possibly shorter,
 *                    one SGD step of learning rate lr each.  loss_out (device,
 *                    nullable) gets the mean pre-step minibatch loss of the
 *                    last epoch.  The model is updated in place, so scoring
 *                    calls ordered after the round see the new model.
 * Errors: LS_ERR_STATE before ls_buffer_init, without a model, or on an empty
 * buffer (train); LS_ERR_INVALID for bad sizes or a perm that is not a
 * permutation.
 */
#define LS_MAX_REPLAY 32768
int ls_buffer_init(ls_ctx* ctx, int32_t fifo_cap, int32_t replay_cap);
int ls_buffer_push(ls_ctx* ctx, int32_t B, const float* feats, const float* ttft, int32_t* admitted, void* stream);
int ls_buffer_state(ls_ctx* ctx, int32_t* fifo_count, int32_t* fifo_head, int32_t* replay_count);
int ls_buffer_read(ls_ctx* ctx, float* fifo_x, float* fifo_y, float* replay_x, float* replay_y, void* stream);
int ls_train_round(ls_ctx* ctx, int32_t epochs, int32_t batch, float lr, const int32_t* perm, float* loss_out,
                   void* stream);

/*
 * Double-buffered retraining (Section 4.3.1, the isolation of training from
 * inference: a newly trained model replaces the serving one at once, without
 * stopping routing; Section 4.3.2, retraining runs beside routing).
 *   ls_set_shadow_training  enable != 0 allocates (first time) a second copy of
 *                    the model, the shadow, and copies the live model into it
 *                    on `stream`; from then on ls_update, ls_train_round and
 *                    the embeddings of ls_buffer_push use the shadow, while
 *                    ls_score_batch and ls_route_batch keep using the live
 *                    model.  ls_set_model writes both; ls_get_model reads the
 *                    live one.  enable == 0 returns updates to the live model
 *                    (the shadow's contents are then dropped at the next
 *                    enable).  LS_ERR_STATE without a model.
 *   ls_swap_model    exchanges live and shadow, ordered on the device: the
 *                    serving stream waits for the work enqueued so far on the
 *                    training stream, the training stream waits for the work
 *                    enqueued so far on the serving stream, then (host side)
 *                    the two slots trade places and the new live model is
 *                    copied into the shadow on the training stream, so that
 *                    training continues from the model now serving.  Scoring
 *                    calls enqueued on serve_stream after the swap use the new
 *                    model; those enqueued before it, the old one.  The two
 *                    streams may be the same.  LS_ERR_STATE without a shadow.
 * Streams: ls_update, ls_buffer_push and ls_train_round use scratch memory of
 * their own, apart from the scoring calls', so with the shadow on they may run
 * on a training stream while ls_score_batch / ls_route_batch run on a serving
 * stream; the three training calls share their scratch and the buffer, so
 * they belong on one stream (or are ordered by the caller), as do the scoring
 * calls and ls_commit_routes among themselves.
 * Ownership: the shadow is freed by ls_destroy.  A context is still driven from
 * one host thread: the streams order device work, not host calls.
 */
int ls_set_shadow_training(ls_ctx* ctx, int enable, void* stream);
int ls_swap_model(ls_ctx* ctx, void* serve_stream, void* train_stream);

/*
 * Per-kernel timing (the library's own view of where the routing time goes;
 * Section 5.4 measures the router's overhead end to end).  While enabled, each
 * kernel launch group of the context is bracketed by HIP events on the stream
 * of its call (events without a system-scope fence: they order nothing and
 * cost no cache writeback).  Kinds: "table_build", "prefix_match", "instance_partial",
 * "score_pairs", "score_pairs_mfma", "band_select", "rescore", "argmin",
 * "update", "route", "buffer", "index" (prefix-index maintenance).
 *   ls_profile_enable  enable != 0 starts recording (and clears old records).
 *   ls_profile_read    synchronous; for up to max_kinds kinds writes the kind
 *                      name (static string), the number of launches and the
 *                      summed device time in milliseconds; *n_kinds gets the
 *                      number of kinds with at least one launch.
 */
int ls_profile_enable(ls_ctx* ctx, int enable);
int ls_profile_read(ls_ctx* ctx, int32_t max_kinds, const char** names, int64_t* launches, double* total_ms,
                    int32_t* n_kinds);

#ifdef __cplusplus
}
#endif

#endif /* LODESTAR_H */
