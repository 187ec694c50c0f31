// Internal interface between the host library and the gfx950 kernels.
// Not part of the public ABI (include/gambit.h is).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace gambit {

constexpr int kBlock = 16;     // tokens per KV block
constexpr int kHeadDim = 128;  // head dimension the kernels implement
constexpr int kRowsPerUnit = 16;  // attention rows (trace x q-head) of one unit (one wavefront)
constexpr int kUnitsPerWG = 4;

// Layout of one (block, KV head) tile of 16 tokens x 128 d in the caches,
// chosen so that every matrix-core operand of the attention kernel is one
// 16-byte load per lane:
//  K: [d / C][k_phys(token)][C], C = 16 / element bytes (16-byte d-chunks;
//     within a chunk the token rows are stored with bits 2 and 3 of the
//     token index swapped).
//  V: [d][token] (transposed).
__host__ __device__ inline int k_phys(int t) { return (t & 3) | ((t >> 1) & 4) | ((t << 1) & 8); }

// One attention work entry: a chunk of a run of blocks that the same member
// traces share, for one KV head, and either one block of <= 16 rows (a
// narrow unit, one wavefront) or up to 64 rows (a cooperative item, one
// workgroup).
struct AttnUnit {
  int32_t owner;    // trace whose block-table row lists the run's blocks
  int32_t jb0;      // first logical block of the run
  int32_t nblk;     // blocks in the run; -1 = through the owner's last block (read at run time)
  int32_t kvh;      // KV head
  int32_t mem_off;  // first member (list position) in the member array
  int32_t mem_cnt;  // members in this tile; 0 = padding unit (does nothing)
  int32_t kidx;     // partial slot of this run for every member
  int32_t flags;    // kUnitCoop in the first entry of a cooperative workgroup slot
};

enum : int32_t { kUnitCoop = 1 };

// Rows of an fp8 narrow unit: one wave takes two row blocks (the widened K
// and V operands feed both); bf16 narrow units keep one.
constexpr int kRowsPerNarrowFp8 = 32;
constexpr int kRowsPerCoop = 128;  // rows of one cooperative item (4 waves x up to 2 row blocks)
constexpr int kTailSlots = 96;     // last workgroup slots of an XCD, claimed at run time

// Device view of a pool.
struct DevPool {
  uint8_t* k_cache;       // layer 0; layer l at + l * layer_bytes
  uint8_t* v_cache;
  float* kv_scale;        // [num_layers][num_blocks][2], fp8 only
  int32_t* table;         // [max_traces][max_blocks]
  int32_t* seq_len;       // [max_traces]
  int32_t* refcount;      // [num_blocks]
  uint32_t* freebits;     // [nwords], bit set = block free
  int32_t* alloc_list;    // [num_blocks] scratch of the allocator
  int32_t* err;           // device error word
  // tournament state per trace slot (Alg. 1): running mean score, scored
  // thoughts, tokens generated since creation, ghost flag (evicted by the
  // scheduler, still in the tree view)
  float* sbar;            // [max_traces]
  int32_t* nscore;        // [max_traces]
  int32_t* gen;           // [max_traces]
  int32_t* ghost;         // [max_traces]
  int32_t num_blocks, nwords, max_traces, max_blocks;
  int32_t Hq, Hkv, g;
  int32_t esize;          // bytes per cache element (2 bf16, 1 fp8)
  int32_t num_layers;
  size_t layer_bytes;     // bytes of one layer of k_cache (and of v_cache)

  // The same pool seen through layer l's caches.
  __host__ __device__ DevPool layer(int l) const {
    DevPool q = *this;
    q.k_cache += (size_t)l * layer_bytes;
    q.v_cache += (size_t)l * layer_bytes;
    if (q.kv_scale) q.kv_scale += (size_t)l * 2 * num_blocks;
    return q;
  }
};

enum : int32_t {
  kErrAllocShort = 1,       // allocator found fewer free blocks than requested
  kErrRefUnderflow = 2,     // a refcount dropped below zero
  kErrBadBlock = 4,         // a table entry outside [0, num_blocks)
};

constexpr int kMaxArgBlocks = 256;  // new blocks one decode step can hand to its launch

struct AttnLaunch {
  const uint16_t* q;        // [n][Hq][128] bf16
  const uint8_t* k_new;     // [n][Hkv][128] cache elements: this step's token, written by the
  const uint8_t* v_new;     //   unit that covers the trace's last block (end read at run time)
  const AttnUnit* units;    // workgroup slots of 4 entries, grouped by XCD
  int32_t xcd_off[9];       // XCD x's workgroup slots: entries [xcd_off[x], xcd_off[x+1])
  int32_t grid;             // one workgroup per slot, rounded up to a multiple of 8
  int32_t* queues;          // [8] tail claims per XCD (front | back << 16); zero at launch,
                            // reset by the merge kernel
  const int32_t* members;   // list positions
  const int32_t* nk;        // [n] partials per list position
  float* part_acc;          // [n][Hq][kmax][128]
  float2* part_ml;          // [n][Hq][kmax] (running max in log2 units, sum)
  int32_t kmax;
  int32_t n;
  float scale_log2;         // sm_scale * log2(e)
  void* out;
  int32_t out_f32;
  // The decode step's new blocks.  len_bias = 1: the lengths still exclude
  // this step's token; the blocks it opens (the lowest free ids, in list
  // order, as the host mirror took them) are listed here and claimed by the
  // appending units, and the merge kernel advances the lengths.  len_bias =
  // 0: the allocator kernel has already run.
  const int32_t* list;      // [n] trace ids in list order
  int32_t len_bias;
  int32_t n_new;            // entries of new_pos / new_blk, positions ascending
  float new_scale;          // fp8 scale of a block a decode step opens
  int32_t claim;            // enter the new blocks in table, refcounts and free set (the
                            //   step's first layer; every layer sets its own fp8 scales)
  int32_t advance;          // the merge advances lengths and GenLen (the step's last layer)
  int32_t new_bf16;         // fp8 pool: k_new / v_new are bf16, quantised on append
  int32_t new_pos[kMaxArgBlocks];
  int32_t new_blk[kMaxArgBlocks];
};

hipError_t launch_pool_init(const DevPool& P, hipStream_t s);
// m requests (trace ids, token counts) on the device; uniform_ntok >= 0
// overrides the counts.  fp8 pools give new blocks the scale `new_scale`.
// `generated`: the tokens are a decode step's (they count towards GenLen).
hipError_t launch_alloc(const DevPool& P, const int32_t* req_trace, const int32_t* req_ntok,
                        int32_t uniform_ntok, int32_t m, float new_scale, bool generated, hipStream_t s);
hipError_t launch_write(const DevPool& P, int32_t trace, int32_t pos0, int32_t n, const void* k,
                        const void* v, const float* started_scales, hipStream_t s);
// Free the listed traces' blocks.  kFreeEnd: the trace ends (its tournament
// state is cleared, a ghost leaves the tree view; rows may be empty);
// kFreeEvict: the scheduler evicts it (it becomes a ghost, its score stays).
enum : int32_t { kFreeEnd = 0, kFreeEvict = 1 };
hipError_t launch_free(const DevPool& P, const int32_t* ids, int32_t n, int32_t mode, hipStream_t s);
// pairs: device [n][2] (child, parent).  req_trace/req_ntok: scratch [n].
hipError_t launch_fork(const DevPool& P, const int32_t* pairs, int32_t n, int32_t* req_trace,
                       int32_t* req_ntok, hipStream_t s);

hipError_t launch_attention_units(const DevPool& P, const AttnLaunch& A, hipStream_t s);
hipError_t launch_attention_merge(const DevPool& P, const AttnLaunch& A, hipStream_t s);

// Probe + sigmoid + ranking + prune/branch plan in one launch.
struct ProbeLaunch {
  const int32_t* list;      // device [n] trace ids
  int32_t n;
  const uint16_t* h;        // [n][Dh] bf16
  int32_t Dh;
  const float* w;
  float b;
  int32_t keep, n_parents;
  float* scores_out;        // [n]
  int32_t* keep_out;        // [keep]
  int32_t* pairs_out;       // [n-keep][2]
  int32_t* free_list;       // [n-keep] scratch: pruned ids ascending
  uint32_t* ticket;         // zero before launch; the kernel leaves it zero
};
hipError_t launch_probe_rank(const ProbeLaunch& L, hipStream_t s);
hipError_t launch_rank_topk(int32_t n, const int32_t* ids, const float* scores, int32_t keep,
                            int32_t* keep_out, hipStream_t s);

// Thought scores of the listed traces and their running means (Alg. 1
// Generate): f = sigmoid(h . w + b), n += 1, s_bar += (f - s_bar) / n.
struct ScoreLaunch {
  const int32_t* list;      // device [n] trace ids
  int32_t n;
  const uint16_t* h;        // [n][Dh] bf16
  int32_t Dh;
  const float* w;
  float b;
  float* scores_out;        // [n]
};
hipError_t launch_score_update(const DevPool& P, const ScoreLaunch& L, hipStream_t s);

// The eviction choice (Alg. 1 Schedule): out[0] = the listed trace ranked
// last by (s_bar descending, id ascending).
hipError_t launch_evict_pick(const DevPool& P, const int32_t* list, int32_t n, int32_t* out,
                             hipStream_t s);

// The tournament plan over the tree view (Alg. 1 Tournament, Eqs. 2-3).
// out (device, kTournHeader + 3 * max_traces ints): header {case, N,
// pruned, children, vacant}, then the pruned ids ascending (max_traces
// entries), then (child, parent) pairs (2 * max_traces entries).
constexpr int kTournHeader = 8;
hipError_t launch_tournament(const DevPool& P, int32_t capacity, int32_t swap_k, int32_t warmup,
                             int32_t* out, int32_t* ranked_out, hipStream_t s);

constexpr int kMaxRank = 4096;  // largest population the in-LDS ranking handles

// The 2-layer MLP scorer f = sigmoid(w2 . act(W1 h + b1) + b2): W1 h in
// 128 x 128 tiles on the bf16 matrix cores with the k range split `splits`
// ways; with splits > 1 the tiles write fp32 pre-activation partial sums
// [splits][n][hidden] that a second launch adds in split order before bias,
// activation and w2; with splits = 1 the tiles apply them and write partial
// logits [tiles_u][n].  A third launch ranks when keep > 0.
struct MlpLaunch {
  int32_t n, dim, hidden, act;   // act: 0 ReLU, 1 GELU (erf)
  int32_t tiles_t, tiles_u;      // ceil(n / 128), ceil(hidden / 128)
  int32_t splits;                // k splits, <= dim / 128
  const uint16_t* h;             // [n][dim] bf16
  const uint16_t* w1;            // [hidden][dim] bf16
  const float* b1;               // [hidden]
  const float* w2;               // [hidden]
  float b2;
  float* parts;                  // scratch, mlp_workspace_bytes(n, hidden)
  float* scores_out;             // [n]
};
// k splits for n hidden states and `hidden` units: enough 128 x 128 tiles
// for ~256 workgroups, at most 32 and at most kMlpSplitBytes of partial sums
// (capped again by dim / 128 at launch).
constexpr size_t kMlpSplitBytes = (size_t)16 << 20;
inline int mlp_splits(int32_t n, int32_t hidden) {
  const long tiles = (long)((n + 127) / 128) * ((hidden + 127) / 128);
  long s = 256 / tiles;
  s = s < 1 ? 1 : (s > 32 ? 32 : s);
  while (s > 1 && (size_t)s * n * hidden * 4 > kMlpSplitBytes) --s;
  return (int)s;
}
inline size_t mlp_workspace_bytes(int32_t n, int32_t hidden) {
  const int s = mlp_splits(n, hidden);
  return s > 1 ? (size_t)s * n * hidden * 4 : (size_t)((hidden + 127) / 128) * n * 4;
}
// Running means from thought scores computed elsewhere (f device [n]).
hipError_t launch_record_scores(const DevPool& P, const int32_t* list, const float* f, int32_t n,
                                hipStream_t s);

}  // namespace gambit
