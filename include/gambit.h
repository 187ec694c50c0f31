/*
 * gambit.h - C ABI of the population-decode hot path of thought-level beam
 * search on MI355X (gfx950).
 *
 * A population of reasoning traces decodes in lock step.  Their KV caches
 * live in one pool of fixed-size blocks; a trace is a row of block ids.
 * Branching starts a child from its parent's prefix by sharing the parent's
 * KV blocks (Alg. 1 notation, Branch; Sec. 4.1 Case 2: the child reuses its
 * parent's cached KV, the prefix-caching mechanism), and pruning frees the
 * blocks nobody else references (Sec. 4.1 Case 2).  Every decode step
 * appends one token per trace and attends over the whole context; blocks
 * shared by several traces are read from HBM once per step for all of them.
 * At thought boundaries a probe scores every trace, the population is
 * ranked by score, the bottom is pruned and the top is branched (Alg. 1
 * Tournament; Eqs. 2-3).
 *
 * Memory ownership
 *   The caller owns ALL device memory: the K/V pools, the fp8 scales, the
 *   block table, the lengths, the refcounts, the workspace, and every input
 *   and output buffer.  The library owns only the host-side pool handle and
 *   its host mirror of the bookkeeping (lengths, block table, refcounts,
 *   free set, attention plan).  No entry point calls hipMalloc.
 *
 * Pointers
 *   "host" pointers are ordinary CPU memory, read before the call returns.
 *   "device" pointers are HIP device memory on the device that was current
 *   when the pool was created.  `stream` is a hipStream_t (NULL = the null
 *   stream).  A pool is used from one stream and one thread at a time.
 *
 * Errors
 *   Arguments are validated on the host against the host mirror before any
 *   work is enqueued; a call that returns an error has changed nothing.
 *   Out-of-blocks is detected the same way (the mirror knows every length
 *   and the free count).  Device-side invariant violations set an error word
 *   that gambit_pool_check() reports.  gambit_last_error() returns the text
 *   of the last error on a pool.
 *
 * Block allocation rule (all calls): a new block is the lowest free block
 * id; requests are served in the call's list order and, inside one trace,
 * in ascending logical block index.  The rule makes every block table a
 * deterministic function of the call sequence.
 */
#ifndef GAMBIT_H
#define GAMBIT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t gambit_status;

enum {
  GAMBIT_OK = 0,
  GAMBIT_ERR_INVALID = -1,        /* bad argument, id, length or state      */
  GAMBIT_ERR_OUT_OF_BLOCKS = -2,  /* the pool has too few free blocks       */
  GAMBIT_ERR_SHARED_WRITE = -3,   /* write into a block another trace holds */
  GAMBIT_ERR_UNSUPPORTED = -4,    /* shape the kernels do not implement     */
  GAMBIT_ERR_DEVICE = -5,         /* HIP error or device invariant violated */
  GAMBIT_ERR_WORKSPACE = -6       /* workspace smaller than required        */
};

enum { GAMBIT_KV_BF16 = 0, GAMBIT_KV_FP8_E4M3 = 1 };
enum { GAMBIT_OUT_BF16 = 0, GAMBIT_OUT_F32 = 1 };

typedef struct gambit_pool gambit_pool;

/*
 * Pool description.  Layouts (all device memory, caller-owned):
 *   k_cache, v_cache  per layer (num_layers of them, one after another; a
 *                     block id names the same slot in every layer)
 *                     num_blocks x num_kv_heads tiles of block_size x
 *                     head_dim elements, bf16 or OCP E4M3FN bytes for
 *                     GAMBIT_KV_FP8_E4M3 (tile bytes = 16 * 128 * element
 *                     size).  Inside a tile, with C = 16 / element size:
 *                       K element (token t, dim d) at element index
 *                         ((d / C) * 16 + p(t)) * C + d % C,
 *                         p(t) = t with its bits 2 and 3 swapped;
 *                       V element (t, d) at element index d * 16 + t.
 *                     Only the library's kernels write the caches.
 *   kv_scale          [num_layers][num_blocks][2] fp32 (K scale, V scale);
 *                     fp8 only, NULL for bf16.  A stored fp8 value means
 *                     code * scale.
 *   block_table       [max_traces][max_blocks_per_trace] int32, -1 = none
 *   seq_len           [max_traces] int32
 *   refcount          [num_blocks] int32
 *   workspace         >= gambit_workspace_size(desc) bytes, 256-B aligned
 * The pool initialises tables, lengths and refcounts itself.
 */
typedef struct {
  int32_t num_blocks;
  int32_t block_size;            /* must be 16                              */
  int32_t num_q_heads;           /* Hq                                      */
  int32_t num_kv_heads;          /* Hkv; Hq / Hkv in {1, 2, 4, 8, 16}       */
  int32_t head_dim;              /* must be 128                             */
  int32_t kv_dtype;              /* GAMBIT_KV_*                             */
  int32_t max_traces;            /* trace ids are 0 .. max_traces-1         */
  int32_t max_blocks_per_trace;
  int32_t max_splits;            /* attention partials per (trace, head), <= 64; 0 = 64 */
  float fp8_append_scale;        /* scale of blocks a decode step allocates; 0 = 2^-6 */
  int32_t num_layers;            /* layers sharing the block table; 0 = 1   */
  void* k_cache;
  void* v_cache;
  float* kv_scale;
  int32_t* block_table;
  int32_t* seq_len;
  int32_t* refcount;
  void* workspace;
  size_t workspace_bytes;
} gambit_pool_desc;

/* Plan statistics of a trace list under the pool's current state (host only). */
typedef struct {
  int64_t total_tokens;          /* sum of lengths over the listed traces        */
  int64_t unique_tokens;         /* valid tokens of the distinct blocks they use */
  int64_t unique_blocks;         /* distinct blocks they use                     */
  int64_t table_entries;         /* block-table entries they read (sum of blocks)*/
  int32_t n_units;               /* attention work units of the current plan     */
  int32_t max_splits_used;       /* largest number of partials of one trace      */
} gambit_stats;

/* Workspace bytes the description needs; 0 when the description is invalid. */
size_t gambit_workspace_size(const gambit_pool_desc* desc);

/* Create a pool over caller-owned memory; enqueues its initialisation on
 * `stream`.  *out receives the handle. */
gambit_status gambit_pool_create(const gambit_pool_desc* desc, void* stream, gambit_pool** out);
gambit_status gambit_pool_destroy(gambit_pool* pool);

/* Extend each listed trace by n_tokens[i] positions (allocation rule above).
 * trace_ids, n_tokens: host [n].  The new positions hold no data until
 * written.  fp8: new blocks get scale (1, 1).  A ghost's slot (see
 * gambit_evict) cannot be extended. */
gambit_status gambit_kv_alloc(gambit_pool* pool, int32_t n, const int32_t* trace_ids,
                              const int32_t* n_tokens, void* stream);

/* Write n tokens of K and V at positions pos0 .. pos0+n-1 of a trace, in
 * every layer.  k, v: device [num_layers][n][num_kv_heads][head_dim] in the
 * cache dtype.  Every touched block must be held by this trace alone (else
 * GAMBIT_ERR_SHARED_WRITE).  fp8: scales is host [num_layers][m][2] for the
 * m blocks whose first position lies in [pos0, pos0+n), ascending; the codes
 * of tokens in other blocks must already be quantised with those blocks'
 * scales.  bf16: scales is NULL. */
gambit_status gambit_kv_write(gambit_pool* pool, int32_t trace_id, int32_t pos0, int32_t n,
                              const void* k, const void* v, const float* scales, void* stream);

/* Branch (Alg. 1 notation; Sec. 4.1 Case 2): child_ids[i] starts from the
 * prefix of parent_ids[i].  The child row lists the parent's full blocks
 * (refcount + 1 each); a partial last block is copied into one new block
 * (with its fp8 scales); the child's length equals the parent's.  Children
 * must be empty (neither running nor a ghost), distinct, and not parents in
 * the same call; a child takes its parent's tournament scores (see below).
 * parent_ids, child_ids: host [n]. */
gambit_status gambit_kv_fork(gambit_pool* pool, int32_t n, const int32_t* parent_ids,
                             const int32_t* child_ids, void* stream);

/* Prune (Sec. 4.1 Case 2): every block of each listed trace loses one
 * reference and becomes free at zero; the row empties and the length
 * becomes 0.  trace_ids: host [n]; freeing an empty trace is an error. */
gambit_status gambit_kv_free(gambit_pool* pool, int32_t n, const int32_t* trace_ids, void* stream);

/* One decode step of a one-layer pool (num_layers 1) for the listed traces
 * (Alg. 1 Generate, attention part):
 * append k_new/v_new at position seq_len (taking a new block when seq_len is
 * a multiple of 16; fp8 blocks taken here get fp8_append_scale), then for
 * every trace t and query head h, with G = h / (Hq / Hkv),
 *     out[t][h] = softmax(q[t][h] . K_t[:, G]^T * sm_scale) V_t[:, G]
 * over all seq_len + 1 positions.  Blocks shared by several listed traces
 * are read once for all of them.
 *   trace_ids  host [n], distinct, each with seq_len > 0
 *   q          device [n][Hq][head_dim] bf16
 *   k_new,v_new device [n][Hkv][head_dim] cache dtype (fp8: codes for the
 *              scale of the block the token lands in)
 *   out        device [n][Hq][head_dim], bf16 or fp32 (out_dtype) */
gambit_status gambit_decode_attn(gambit_pool* pool, int32_t n, const int32_t* trace_ids,
                                 const void* q, const void* k_new, const void* v_new,
                                 void* out, int32_t out_dtype, float sm_scale, void* stream);

enum { GAMBIT_NEW_CACHE = 0, GAMBIT_NEW_BF16 = 1 };

/* One layer of a decode step: the operation of gambit_decode_attn on layer
 * `layer`'s caches.  A step is the calls for layers 0, 1, ..., num_layers - 1
 * in order, with the same trace list: the blocks the step opens are taken at
 * layer 0 (one allocation for all layers), the token lands at the same
 * position in every layer, and the lengths (and GenLen) advance after the
 * last layer.  While a step is open, calls that change or check the pool
 * (kv_*, evict, tournament, score_prune_branch, pool_check) fail with
 * GAMBIT_ERR_INVALID and change nothing.
 *   new_dtype  GAMBIT_NEW_CACHE: k_new/v_new in the cache dtype, as for
 *              gambit_decode_attn.  GAMBIT_NEW_BF16: bf16 [n][Hkv][head_dim];
 *              an fp8 pool quantises each element on append: code = the
 *              E4M3FN value nearest to x / s (the quotient rounded to fp32;
 *              ties to the even code; beyond 448 saturating, no NaN), s the
 *              landing block's K or V scale (fp8_append_scale for a block the
 *              step opens).  A bf16 pool stores them as they are.
 * The other arguments are those of gambit_decode_attn. */
gambit_status gambit_decode_attn_layer(gambit_pool* pool, int32_t layer, int32_t n, const int32_t* trace_ids,
                                       const void* q, const void* k_new, const void* v_new, int32_t new_dtype,
                                       void* out, int32_t out_dtype, float sm_scale, void* stream);

/* A thought boundary (Alg. 1 Tournament; Eqs. 2-3; Sec. 4.1):
 *   score[i] = 1 / (1 + exp(-(h[i] . w + b)))   (linear sigmoid probe, the
 *              head form of Eq. 6 applied to the boundary hidden state)
 *   rank the listed traces by (score descending, trace id ascending);
 *   keep_out = the first `keep` ids in rank order;
 *   prune the other n - keep traces (ascending id);
 *   branch: with c = (n - keep) / n_parents, freed slot j (ascending) becomes
 *   a child of keep_out[j / c]; the parent keeps running (App. A.5).
 * The paper's Case 2 is keep = C - K, n_parents = K (c = 1).
 *   trace_ids        host [n]
 *   h                device [n][Dh] bf16, in list order
 *   w                device [Dh] fp32;  b: bias
 *   scores_out       device [n] fp32, list order
 *   keep_out         device [keep] int32, rank order
 *   child_parent_out device [n - keep][2] int32 (child id, parent id)
 * Blocks until the ranking is known on the host (one device-to-host copy). */
gambit_status gambit_score_prune_branch(gambit_pool* pool, int32_t n, const int32_t* trace_ids,
                                        const void* h, int32_t Dh, const float* w, float b,
                                        int32_t keep, int32_t n_parents, float* scores_out,
                                        int32_t* keep_out, int32_t* child_parent_out,
                                        void* stream);

/* Stateless ranking (the selection step of Alg. 1 Tournament): keep_out[r]
 * = the id of rank r under (score descending, id ascending), r < keep.
 * trace_ids, scores: device [n]; keep_out: device [keep]; n <= 4096. */
gambit_status gambit_rank_topk(int32_t n, const int32_t* trace_ids, const float* scores,
                               int32_t keep, int32_t* keep_out, void* stream);

/*
 * The full tournament of Alg. 1.  Per trace slot the pool keeps the running
 * mean score s_bar over the trace's thoughts and their number n, the tokens
 * the trace has generated since its creation (GenLen: decode steps count,
 * kv_alloc/kv_write do not; a child starts at 0), and a ghost flag.  Two
 * views of the population (Sec. 4.2): the scheduler view is the running
 * traces (they hold KV blocks); the tree view adds the ghosts, traces the
 * scheduler evicted under memory pressure - no KV, no tokens, but they keep
 * their score and their place in the ranking, so capacity is counted on the
 * tree view.  A fork gives the child its parent's (s_bar, n); a trace that
 * ends (kv_free, pruning) clears its slot's state.
 */
typedef struct {
  int32_t case_taken;            /* 1: under capacity (Eq. 2), 2: swap (Eq. 3), 0: empty tree view */
  int32_t n_active;              /* N, the tree view's size before the round      */
  int32_t n_pruned;              /* entries written to pruned_out                 */
  int32_t n_children;            /* (child, parent) pairs written                 */
} gambit_round;

/* Alg. 1 Generate, scoring: each listed trace completed a thought; its score
 * is f = 1 / (1 + exp(-(h . w + b))) and its running mean becomes
 * s_bar + (f - s_bar) / (n + 1) over n + 1 thoughts (the mean of the thought
 * scores of Sec. 4.1).
 *   trace_ids   host [n], running traces, distinct
 *   h           device [n][Dh] bf16 (Dh a multiple of 8); w device [Dh] fp32
 *   scores_out  device [n] fp32: f in list order */
gambit_status gambit_score_update(gambit_pool* pool, int32_t n, const int32_t* trace_ids, const void* h,
                                  int32_t Dh, const float* w, float b, float* scores_out, void* stream);

/* Alg. 1 Schedule (Sec. 4.2): of the listed running traces, the one of
 * lowest s_bar (on equal scores the higher id) is evicted - its blocks are
 * released as by kv_free, but it becomes a ghost that keeps its score.
 *   trace_ids   host [n], running traces, n <= 4096;  victim_out host [1]
 * Blocks until the choice is known (one device-to-host copy). */
gambit_status gambit_evict(gambit_pool* pool, int32_t n, const int32_t* trace_ids, int32_t* victim_out,
                           void* stream);

/* Alg. 1 Tournament (Eqs. 2-3) over the tree view.  Rank it by s_bar
 * (descending; equal scores: lower id first).  Eligible parents: running
 * traces with GenLen >= warmup.  With N traces in the tree view:
 *   N < capacity (Case 1): branch the top min(capacity - N, |eligible|);
 *   N >= capacity (Case 2): prune the bottom min(swap_k, N) - running ones
 *     release their blocks, ghosts leave the tree view - then branch the top
 *     min(swap_k, |eligible not pruned|).
 * Children take the lowest vacant slots (neither running nor ghost, after
 * the pruning) in ascending order, one per parent in rank order; a branch is
 * a kv_fork (the parent continues, App. A.5).  Pruned slots are freed, in
 * ascending order, before any fork.
 *   capacity in 1 .. max_traces (<= 4096);  swap_k, warmup >= 0
 *   round_out         host: what the round did
 *   pruned_out        host [>= swap_k]: pruned ids, ascending
 *   child_parent_out  host [max_traces][2]: (child, parent) pairs
 *   ranked_out        device [max_traces] int32 or NULL: the tree view in
 *                     rank order (first n_active entries)
 * The plan is computed on the device, read back once, checked against the
 * host mirror (everything but the scores) and the out-of-blocks test, and
 * only then applied; on error nothing has changed. */
gambit_status gambit_tournament(gambit_pool* pool, int32_t capacity, int32_t swap_k, int32_t warmup,
                                gambit_round* round_out, int32_t* pruned_out, int32_t* child_parent_out,
                                int32_t* ranked_out, void* stream);

/* Running means from thought scores computed elsewhere (for instance by
 * gambit_mlp_score): as gambit_score_update with f given.
 *   trace_ids host [n], running traces, distinct;  f device [n] fp32 */
gambit_status gambit_record_scores(gambit_pool* pool, int32_t n, const int32_t* trace_ids, const float* f,
                                   void* stream);

/*
 * The 2-layer MLP scorer of the paper's main evaluation (STEP's off-the-shelf
 * probe on the thought-boundary hidden state, Sec. 4.1 and Sec. 5.1; the
 * paper gives no dimensions, activation or weights, so they are parameters):
 *     f(h) = 1 / (1 + exp(-(w2 . act(W1 h + b1) + b2)))
 * with act = ReLU or GELU (x * Phi(x), erf form).  W1 h runs on the bf16
 * matrix cores with fp32 accumulation, in 128 x 128 tiles whose k range is
 * split so that the chip has ~256 tiles of work (at most 16 MiB of fp32
 * partial sums); the partial sums are added in a fixed order before bias,
 * activation and w2, so a call's result depends only on its sizes and
 * inputs.  The ranking counts, for every score, the scores ahead of it.
 */
enum { GAMBIT_ACT_RELU = 0, GAMBIT_ACT_GELU = 1 };
typedef struct {
  int32_t dim;                   /* Dh, a multiple of 128                    */
  int32_t hidden;                /* H1, a multiple of 64                     */
  int32_t activation;            /* GAMBIT_ACT_*                             */
  const void* w1;                /* device [hidden][dim] bf16                */
  const float* b1;               /* device [hidden]                          */
  const float* w2;               /* device [hidden]                          */
  float b2;
} gambit_mlp;

/* Bytes of device workspace gambit_mlp_score needs (0: invalid sizes). */
size_t gambit_mlp_workspace_size(int32_t n, int32_t hidden);

/* Scores of n hidden states (n <= 4096).
 *   h           device [n][dim] bf16;  scores_out device [n] fp32
 *   keep > 0:   also rank (score descending, id ascending) and write the top
 *               `keep` ids to keep_out (device [keep]); trace_ids device [n]
 *   workspace   device, >= gambit_mlp_workspace_size(n, hidden) bytes
 * Stateless; enqueued on `stream`. */
gambit_status gambit_mlp_score(int32_t n, const void* h, const gambit_mlp* mlp, float* scores_out,
                               const int32_t* trace_ids, int32_t keep, int32_t* keep_out, void* workspace,
                               size_t workspace_bytes, void* stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops or harnesses that forbid allocation): the same
 * scoring as gambit_mlp_score, with its scratch (the tiles' partial sums)
 * in a buffer the library holds in device memory, one per device, for the
 * life of the process, instead of a caller workspace.  It calls no
 * allocator.  Sizes whose gambit_mlp_workspace_size(n, hidden) exceeds
 * GAMBIT_MLP_STATIC_SCRATCH_BYTES (16 MiB: any n <= 4096 with hidden up to 131072)
 * fail with GAMBIT_ERR_WORKSPACE.  Every call on one device shares that
 * device's buffer: calls that overlap on one device (other streams, other
 * threads) race and must be ordered by the caller.  Other arguments and
 * results as gambit_mlp_score. */
#define GAMBIT_MLP_STATIC_SCRATCH_BYTES ((size_t)16 << 20)
gambit_status gambit_mlp_score_static(int32_t n, const void* h, const gambit_mlp* mlp, float* scores_out,
                                      const int32_t* trace_ids, int32_t keep, int32_t* keep_out, void* stream);

/* Tournament state of the listed slots (host outputs, any may be NULL);
 * synchronises `stream`.  sbar fp32, nscore/gen int32, ghost 0/1. */
gambit_status gambit_trace_state(gambit_pool* pool, int32_t n, const int32_t* trace_ids, float* sbar_out,
                                 int32_t* nscore_out, int32_t* gen_out, int32_t* ghost_out, void* stream);

/* Synchronise `stream`, then compare the device block table, lengths,
 * refcounts, free set and tournament bookkeeping (scored thoughts, GenLen,
 * ghost flags) with the host mirror and read the device error word.
 * GAMBIT_OK when all agree. */
gambit_status gambit_pool_check(gambit_pool* pool, void* stream);

/* Statistics of the attention work for a trace list (host only, no sync). */
gambit_status gambit_plan_stats(gambit_pool* pool, int32_t n, const int32_t* trace_ids,
                                gambit_stats* out);

/* The kinds of attention work that cover each listed trace in the plan the
 * pool's decode steps of this exact trace list use (host only, no sync; the
 * plan is made by the first decode step after the list or the pool's block
 * sharing changed, so call this after such a step).  kinds_out host [n]:
 * an OR of GAMBIT_UNIT_* bits, one per kind of work unit whose rows include
 * the trace (narrow one-wave units of one row block, or - fp8, 17 to 32
 * rows - two; cooperative workgroup items with one or two row blocks per
 * wave);
 * GAMBIT_UNIT_TAIL_SLOT when one of them sits in the workgroup slots that
 * the launch claims at run time.  For test coverage of the kernel's paths.
 * GAMBIT_ERR_INVALID when the current plan is not for this list. */
enum {
  GAMBIT_UNIT_NARROW = 1,
  GAMBIT_UNIT_COOP_ONE = 2,
  GAMBIT_UNIT_COOP_TWO = 4,
  GAMBIT_UNIT_TAIL_SLOT = 16,
  GAMBIT_UNIT_NARROW_TWO = 32
};
gambit_status gambit_plan_kinds(gambit_pool* pool, int32_t n, const int32_t* trace_ids, int32_t* kinds_out);

/* Event timing of the split-K attention kernel, the dominant kernel of a
 * decode step.  Between gambit_profile_begin and gambit_profile_end every
 * gambit_decode_attn records a HIP event pair on its stream around that
 * kernel (at most max_launches pairs; later launches are not timed).
 * gambit_profile_end waits for the last event and returns the summed
 * kernel time in milliseconds and the number of timed launches. */
gambit_status gambit_profile_begin(gambit_pool* pool, int32_t max_launches);
gambit_status gambit_profile_end(gambit_pool* pool, double* attn_ms, int32_t* launches);

/*
 * The history-aware sequence scorer (App. A.1, Eqs. 4-6) with incremental
 * inference: each trace slot keeps the cached keys and values of its step
 * states; at a thought boundary a listed trace's new step state h_t is
 * scored in one pass against them,
 *     x = GELU(W_in LN_in(h_t))
 *     per layer:  x += W_o MHA(LN1(x))   causal over the trace's steps
 *                                        0..t, RoPE at the step index
 *                 x += W_2 (SiLU(W_1 LN2(x)) * W_3 LN2(x))
 *     y_t = 1 / (1 + exp(-(w_out . LN_out(x))))
 * which equals the whole-history forward at its last position.  LN is
 * LayerNorm with gain and bias, eps 1e-5; GELU the erf form; heads of 64
 * dims, scale 1/8; RoPE rotates (x_i, x_{i+32}) of each head by
 * t * 10000^(-i/32); no biases in the linear maps.  Weights (device fp32,
 * caller-owned, [out][in] row-major; 16-byte aligned):
 *   ln_in_g, ln_in_b [input_dim];  w_in [d_model][input_dim]
 *   ln1_g, ln1_b, ln2_g, ln2_b [n_layers][d_model]
 *   w_qkv [n_layers][3 d_model][d_model]   rows: W_q, then W_k, then W_v
 *   w_o   [n_layers][d_model][d_model]
 *   w_13  [n_layers][2 d_ff][d_model]      rows 32c .. 32c+15: W_1 rows
 *                                          16c .. 16c+15; rows 32c+16 ..
 *                                          32c+31: W_3 rows 16c .. 16c+15
 *   w_2   [n_layers][d_model][d_ff]
 *   ln_out_g, ln_out_b, w_out [d_model]
 * d_model = 64 n_heads; input_dim a multiple of 128, d_ff of 64; max_steps
 * <= 8192.  The workspace (>= gambit_scorer_workspace_size, 256-B aligned)
 * holds the per-slot caches (fp32, max_traces * n_layers * n_heads * 2 * 64
 * * max_steps floats), the step's activations and the input projection in
 * the library's own form: gambit_scorer_create reads ln_in_g, ln_in_b and
 * w_in once and keeps W_in scaled by ln_in_g as three bf16 planes whose sum
 * is that product exactly (the bf16 step states are multiplied with them on
 * the matrix cores, fp32 sums), its row sums and W_in ln_in_b; a change to
 * those three weights takes a new scorer.  The other weights are read at
 * every step.
 */
typedef struct gambit_scorer gambit_scorer;
typedef struct {
  int32_t input_dim, d_model, n_heads, n_layers, d_ff, max_steps, max_traces;
  const float *ln_in_g, *ln_in_b, *w_in;
  const float *ln1_g, *ln1_b, *w_qkv, *w_o, *ln2_g, *ln2_b, *w_13, *w_2;
  const float *ln_out_g, *ln_out_b, *w_out;
  void* workspace;
  size_t workspace_bytes;
} gambit_scorer_desc;

size_t gambit_scorer_workspace_size(const gambit_scorer_desc* desc);
/* Set-up work runs on `stream`; create returns after it has finished. */
gambit_status gambit_scorer_create(const gambit_scorer_desc* desc, void* stream, gambit_scorer** out);
gambit_status gambit_scorer_destroy(gambit_scorer* scorer);

/* One thought boundary: each listed slot appends its step state and gets
 * its score y_t.  trace_ids host [n], distinct, each holding < max_steps
 * steps; h device [n][input_dim] bf16 in list order; scores_out device [n]
 * fp32. */
gambit_status gambit_scorer_step(gambit_scorer* scorer, int32_t n, const int32_t* trace_ids, const void* h,
                                 float* scores_out, void* stream);

/* Branch: child_ids[i] takes the step history of parent_ids[i] (its cached
 * keys and values and its step count).  Children distinct and not parents
 * in the same call.  Host arrays [n]. */
gambit_status gambit_scorer_fork(gambit_scorer* scorer, int32_t n, const int32_t* parent_ids,
                                 const int32_t* child_ids, void* stream);

/* Prune / end: the listed slots forget their histories.  Host [n]. */
gambit_status gambit_scorer_free(gambit_scorer* scorer, int32_t n, const int32_t* trace_ids, void* stream);

/* Steps a slot holds (host mirror, no sync); -1 for a bad id. */
int32_t gambit_scorer_steps(const gambit_scorer* scorer, int32_t trace_id);

/* Compare the device step counts with the host mirror and read the device
 * error word (synchronises the stream).  GAMBIT_OK when they agree. */
gambit_status gambit_scorer_check(gambit_scorer* scorer, void* stream);
const char* gambit_scorer_last_error(const gambit_scorer* scorer);

/* Measurement, not a step of the method: the device's streaming-read rate,
 * the practical ceiling beside the published HBM peak for the attention
 * kernel's achieved bandwidth.  Reads `bytes` of device memory at `buf`
 * once (workgroup w a contiguous run of 64 KiB chunks; 16-byte loads, with
 * the non-temporal hint when nontemporal = 1) on `stream`; does not block.
 * sink: device [grid] uint32, caller-zeroed; each workgroup XORs the dwords
 * it read into sink[w], so the XOR of sink equals the XOR of the buffer's
 * dwords.  GAMBIT_ERR_INVALID unless buf is 16-byte aligned, bytes is a
 * positive multiple of 65536 and 1 <= grid <= min(65535, bytes / 65536);
 * GAMBIT_ERR_DEVICE if the launch fails. */
gambit_status gambit_stream_read(const void* buf, size_t bytes, int32_t nontemporal, int32_t grid,
                                 uint32_t* sink, void* stream);

/* Host mirror queries (no sync): length of a trace; free block count. */
int32_t gambit_seq_len(const gambit_pool* pool, int32_t trace_id);
int32_t gambit_free_blocks(const gambit_pool* pool);

const char* gambit_status_str(gambit_status s);
const char* gambit_last_error(const gambit_pool* pool);

#ifdef __cplusplus
}
#endif

#endif /* GAMBIT_H */
