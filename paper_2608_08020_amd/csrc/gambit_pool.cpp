// Host side of libgambit: the pool handle, its host mirror of the block
// bookkeeping, argument validation, the shared-run attention planner and the
// C ABI entry points declared in include/gambit.h.
//
// The mirror applies exactly the allocation rule the device kernels apply
// (lowest free block id first, requests in list order, ascending logical
// index), so it always knows every length, every table row and the free
// count without reading the device.  That lets every call validate and
// detect out-of-blocks before it enqueues anything, and lets the planner
// find which traces share which blocks.  The one device-to-host read on the
// hot path is the ranking at a thought boundary.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <numeric>
#include <string>
#include <thread>
#include <vector>

#include "../../include/gambit.h"
#include "kernels.h"

using gambit::AttnUnit;

namespace {

constexpr size_t kAlign = 256;
constexpr int kDefaultSplits = 64;
constexpr int kMaxLayers = 1024;
constexpr int kDefaultChunkBlocks = 64;  // blocks per attention chunk before balancing

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
int cdiv(int a, int b) { return (a + b - 1) / b; }

// Per-token times of one attention unit on MI355X (microseconds), by kind and
// cache dtype: narrow units per wave, cooperative items per workgroup.  fp8:
// read from per-wave timelines of the 256-trace workload.  bf16: the figures
// the chunk caps were tuned with on the 256- and 512-trace workloads (per-
// wave timelines give 0.10 for narrow units and 0.033-0.053 for cooperative
// items, but caps from them cut the 512-trace launch's cooperative chunks
// shorter: 1.7% more HBM traffic, no gain).
constexpr double kUsNarrow16 = 0.16;     // bf16, <= 16 rows
constexpr double kUsNarrow8 = 0.045;     // fp8, <= 16 rows
constexpr double kUsNarrowTwo8 = 0.055;  // fp8, 17-32 rows (two row blocks)
constexpr double kUsCoop16 = 0.042;     // bf16, any row count
constexpr double kUsCoop64_8 = 0.037, kUsCoop128_8 = 0.051;  // fp8, 33-64 and 65-128 rows
// Chunk caps as fractions of the estimated launch length.
constexpr double kCapNarrow = 1.0, kCapCoop = 0.5;

// Workspace carve-up.  All offsets are kAlign-aligned.
struct Layout {
  size_t list, ids, req_trace, req_ntok, pairs, free_list, nk, ticket, queues, err, scales, freebits,
      alloc_list, units, members, part_ml, part_acc, sbar, nscore, gen, ghost, tourn, total;
  int kmax, max_units, max_members, nwords;
};

bool layout_of(const gambit_pool_desc* d, Layout* L) {
  if (!d) return false;
  if (d->num_blocks <= 0 || d->block_size != gambit::kBlock || d->head_dim != gambit::kHeadDim)
    return false;
  if (d->num_q_heads <= 0 || d->num_kv_heads <= 0 || d->num_q_heads % d->num_kv_heads) return false;
  const int g = d->num_q_heads / d->num_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8 && g != 16) return false;
  if (d->kv_dtype != GAMBIT_KV_BF16 && d->kv_dtype != GAMBIT_KV_FP8_E4M3) return false;
  if (d->max_traces <= 0 || d->max_blocks_per_trace <= 0 || d->max_splits < 0 || d->max_splits > 64) return false;
  if (d->num_layers < 0 || d->num_layers > kMaxLayers) return false;
  const size_t layers = d->num_layers ? d->num_layers : 1;
  const int T = d->max_traces;
  const int kmax = d->max_splits ? d->max_splits : kDefaultSplits;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  L->kmax = kmax;
  L->nwords = cdiv(d->num_blocks, 32);
  L->max_units = 2 * T * kmax * d->num_kv_heads + 64;
  L->max_members = T * kmax;
  L->list = take(4 * (size_t)T);
  L->ids = take(4 * (size_t)T);
  L->req_trace = take(4 * (size_t)T);
  L->req_ntok = take(4 * (size_t)T);
  L->pairs = take(8 * (size_t)T);
  L->free_list = take(4 * (size_t)T);
  L->nk = take(4 * (size_t)T);
  L->ticket = take(64);
  L->queues = take(64);
  L->err = take(64);
  L->scales = take(8 * ((size_t)d->max_blocks_per_trace + 1) * layers);
  L->freebits = take(4 * (size_t)L->nwords);
  L->alloc_list = take(4 * (size_t)d->num_blocks);
  L->units = take(sizeof(AttnUnit) * (size_t)L->max_units);
  L->members = take(4 * (size_t)L->max_members);
  L->part_ml = take(8 * (size_t)T * d->num_q_heads * kmax);
  L->part_acc = take(4 * (size_t)T * d->num_q_heads * kmax * gambit::kHeadDim);
  L->sbar = take(4 * (size_t)T);
  L->nscore = take(4 * (size_t)T);
  L->gen = take(4 * (size_t)T);
  L->ghost = take(4 * (size_t)T);
  L->tourn = take(4 * ((size_t)gambit::kTournHeader + 3 * (size_t)T));
  L->total = o;
  return true;
}

}  // namespace

struct gambit_pool {
  gambit_pool_desc d{};
  Layout L{};
  gambit::DevPool dev{};
  uint8_t* ws = nullptr;
  int g = 1;
  int n_cu = 256;  // compute units of the pool's device (two attention workgroups each)
  float append_scale = 1.f / 64.f;

  // host mirror
  std::vector<std::vector<int32_t>> table;
  std::vector<int32_t> seq_len, refcount;
  // tournament bookkeeping (Alg. 1): scored thoughts, tokens generated since
  // creation, ghost flag; the scores themselves live on the device only
  std::vector<int32_t> nscore, gen;
  std::vector<char> ghost;
  std::vector<uint64_t> freebits;  // bit set = free
  int32_t nfree = 0;
  size_t hint = 0;                 // no free bit below word `hint`

  // pinned staging for host-to-device copies, reused after an event fence
  int32_t* stage = nullptr;
  size_t stage_ints = 0;
  hipEvent_t stage_ev = nullptr;
  uint8_t* plan_stage = nullptr;
  size_t plan_stage_bytes = 0;
  hipEvent_t plan_ev = nullptr;

  // attention plan
  bool plan_valid = false;
  std::vector<int32_t> plan_list;
  int xcd_off[9] = {0};
  int grid = 0;
  int n_units = 0;
  bool queues_dirty = false;       // an attention launch was not followed by its merge
  int max_splits_used = 0;
  int step_next = 0;               // the layer the open decode step expects next (0: none open)
  gambit::AttnLaunch step{};       // the open step's launch arguments
  std::vector<int32_t> cnt, first;  // per-block planner scratch, zero / -1 between calls
  gambit_stats stats{};            // of plan_list, kept current by decode steps
  std::vector<int32_t> plan_kinds;  // per list position: GAMBIT_UNIT_* bits of the units covering it

  // attention-kernel event timing
  std::vector<hipEvent_t> prof_ev;
  int prof_used = 0;
  bool prof_on = false;

  std::string last_error;
};

namespace {

gambit_status fail(gambit_pool* p, gambit_status s, const char* fmt, ...) {
  if (p) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    p->last_error = buf;
  }
  return s;
}

gambit_status hip_fail(gambit_pool* p, hipError_t e, const char* where) {
  return fail(p, GAMBIT_ERR_DEVICE, "%s: %s", where, hipGetErrorString(e));
}

#define HIP_TRY(p, expr, where)                 \
  do {                                          \
    const hipError_t e_ = (expr);               \
    if (e_ != hipSuccess) return hip_fail(p, e_, where); \
  } while (0)

inline hipStream_t S(void* s) { return static_cast<hipStream_t>(s); }

template <class T>
T* ws_ptr(gambit_pool* p, size_t off) {
  return reinterpret_cast<T*>(p->ws + off);
}

// Runs f(0) .. f(n - 1) on up to 8 host threads (the calling one included),
// in chunks of 16 indices; serially for small n or if no thread can start.
template <class F>
void parallel_for(int n, F&& f) {
  const int nt = (int)std::min(8u, std::max(1u, std::thread::hardware_concurrency()));
  if (n < 128 || nt == 1) {
    for (int i = 0; i < n; ++i) f(i);
    return;
  }
  std::atomic<int> next{0};
  auto body = [&]() {
    for (int i; (i = next.fetch_add(16, std::memory_order_relaxed)) < n;)
      for (int k = i, e = std::min(n, i + 16); k < e; ++k) f(k);
  };
  std::vector<std::thread> th;
  for (int t = 1; t < nt; ++t) {
    try {
      th.emplace_back(body);
    } catch (...) {
      break;
    }
  }
  body();
  for (auto& x : th) x.join();
}

// ---- host mirror -----------------------------------------------------------
int take_lowest(gambit_pool* p) {
  for (size_t w = p->hint; w < p->freebits.size(); ++w) {
    if (p->freebits[w]) {
      const int bit = __builtin_ctzll(p->freebits[w]);
      p->freebits[w] &= p->freebits[w] - 1;
      p->hint = w;
      --p->nfree;
      return (int)(w * 64 + bit);
    }
  }
  return -1;
}

void release(gambit_pool* p, int b) {
  p->freebits[b >> 6] |= 1ull << (b & 63);
  p->hint = std::min(p->hint, (size_t)(b >> 6));
  ++p->nfree;
}

void mirror_grow(gambit_pool* p, int t, int ntok) {
  const int L = p->seq_len[t];
  for (int j = cdiv(L, 16); j < cdiv(L + ntok, 16); ++j) {
    const int b = take_lowest(p);
    p->refcount[b] = 1;
    p->table[t].push_back(b);
  }
  p->seq_len[t] = L + ntok;
}

// Forks of distinct children (none of them a parent of another), in pair
// order.  The children's rows copy the parents' full blocks; a parent that
// several consecutive pairs share adds all their references to each of its
// blocks in one pass.  The partial tails then follow in pair order, which
// decides the blocks they get.
void mirror_fork_many(gambit_pool* p, const int32_t* parents, const int32_t* children, int n) {
  for (int i = 0; i < n;) {
    const int par = parents[i];
    int e = i + 1;
    while (e < n && parents[e] == par) ++e;
    const int full = p->seq_len[par] / 16;
    const auto& prow = p->table[par];
    for (int k = i; k < e; ++k) p->table[children[k]].assign(prow.begin(), prow.begin() + full);
    for (int j = 0; j < full; ++j) p->refcount[prow[j]] += e - i;
    i = e;
  }
  for (int i = 0; i < n; ++i) {
    const int par = parents[i], ch = children[i];
    const int L = p->seq_len[par];
    p->seq_len[ch] = L / 16 * 16;
    mirror_grow(p, ch, L % 16);
    p->nscore[ch] = p->nscore[par];
    p->gen[ch] = 0;
    p->ghost[ch] = 0;
  }
}

void mirror_release_rows(gambit_pool* p, int t) {
  for (int b : p->table[t])
    if (--p->refcount[b] == 0) release(p, b);
  p->table[t].clear();
  p->seq_len[t] = 0;
  p->gen[t] = 0;
}

// Distinct traces end (pruned, completed, or ghosts leaving the tree view).
void mirror_free_many(gambit_pool* p, const int32_t* ids, int n) {
  for (int i = 0; i < n; ++i) {
    const int t = ids[i];
    mirror_release_rows(p, t);
    p->nscore[t] = 0;
    p->ghost[t] = 0;
  }
}

// The scheduler evicts the trace: no KV, but it stays in the tree view.
void mirror_evict(gambit_pool* p, int t) {
  mirror_release_rows(p, t);
  p->ghost[t] = 1;
}

// ---- staging ---------------------------------------------------------------
// Copies `n` ints from host memory into device memory `dst` on `stream`
// through the pinned staging buffer.
gambit_status upload_ints(gambit_pool* p, int32_t* dst, const int32_t* src, size_t n, hipStream_t s,
                          size_t stage_off = 0) {
  if (n == 0) return GAMBIT_OK;
  HIP_TRY(p, hipEventSynchronize(p->stage_ev), "staging fence");
  std::memcpy(p->stage + stage_off, src, n * 4);
  HIP_TRY(p, hipMemcpyAsync(dst, p->stage + stage_off, n * 4, hipMemcpyHostToDevice, s), "upload");
  HIP_TRY(p, hipEventRecord(p->stage_ev, s), "staging fence");
  return GAMBIT_OK;
}

gambit_status check_ids(gambit_pool* p, int32_t n, const int32_t* ids, const char* what,
                        std::vector<char>* seen_out = nullptr) {
  if (n < 0 || n > p->d.max_traces) return fail(p, GAMBIT_ERR_INVALID, "%s count %d out of range", what, n);
  if (n > 0 && !ids) return fail(p, GAMBIT_ERR_INVALID, "%s list is NULL", what);
  std::vector<char> seen(p->d.max_traces, 0);
  for (int i = 0; i < n; ++i) {
    const int t = ids[i];
    if (t < 0 || t >= p->d.max_traces) return fail(p, GAMBIT_ERR_INVALID, "%s id %d out of range", what, t);
    if (seen[t]) return fail(p, GAMBIT_ERR_INVALID, "duplicate %s id %d", what, t);
    seen[t] = 1;
  }
  if (seen_out) seen_out->swap(seen);
  return GAMBIT_OK;
}

// ---- planner ---------------------------------------------------------------
// Cuts every listed trace's context into runs of blocks referenced by the
// same set of listed traces.  Sharing only ever comes from forks, which hand
// the child the parent's whole full-block prefix, so along one trace the set
// of sharers can only shrink; two consecutive blocks with equal sharer
// counts therefore have equal sharer sets.  A shared run is emitted once, by
// its lowest list position, for all its sharers; the trailing private run
// ends at the trace's current last block (read by the kernel at run time),
// so the plan stays valid while decode steps append.
struct Group {
  double cost;
  int32_t first, count;  // its units in the plan's unit list
  bool coop;             // cooperative items (one workgroup each), else one narrow unit
};

gambit_status build_plan(gambit_pool* p, int n, const int32_t* ids, hipStream_t s) {
  const int Hkv = p->d.num_kv_heads;
  const int kmax = p->L.kmax;
  const int nb_total = p->d.num_blocks;
  const bool fp8 = p->d.kv_dtype == GAMBIT_KV_FP8_E4M3;
  // rows a narrow (one-wave) unit takes: 16, or two row blocks for fp8
  const int narrow_rows = fp8 ? gambit::kRowsPerNarrowFp8 : gambit::kRowsPerUnit;
  if ((int)p->first.size() != nb_total) p->first.assign(nb_total, -1);
  std::vector<int> nb(n);
  for (int pos = 0; pos < n; ++pos) nb[pos] = cdiv(p->seq_len[ids[pos]], 16);
  // Sharers per block among the listed traces.  When the list holds every
  // running trace that is the block's refcount (ghosts hold no blocks);
  // otherwise it is counted.
  int running = 0, listed_running = 0;
  for (int t = 0; t < p->d.max_traces; ++t) running += p->seq_len[t] > 0;
  for (int pos = 0; pos < n; ++pos) listed_running += p->seq_len[ids[pos]] > 0;
  const bool all = n == running && listed_running == n;  // ids are distinct
  const int32_t* cnt = all ? p->refcount.data() : p->cnt.data();
  std::vector<int32_t> touched;
  if (!all) {
    for (int pos = 0; pos < n; ++pos) {
      const auto& row = p->table[ids[pos]];
      for (int j = 0; j < nb[pos]; ++j)
        if (p->cnt[row[j]]++ == 0) touched.push_back(row[j]);
    }
  }
  {
    gambit_stats& st = p->stats;
    st = gambit_stats{};
    st.unique_blocks = all ? (int64_t)(nb_total - p->nfree) : (int64_t)touched.size();
    for (int pos = 0; pos < n; ++pos) {
      const int L = p->seq_len[ids[pos]];
      st.total_tokens += L;
      st.table_entries += nb[pos];
      // every block is full except a trace's partial last block, which only that trace holds
      st.unique_tokens += L % 16 ? L % 16 - 16 : 0;
    }
    st.unique_tokens += 16 * st.unique_blocks;
  }
  // The runs of every listed trace: [j0, j1) with c sharers; c == 1 is the
  // private rest of the trace.  A shared run starts at the same block in all
  // its sharers (they hold the same prefix blocks), so its member list is
  // keyed by that block; positions are visited in ascending order, so the
  // first one to reach it is the lowest (the run's owner) and the list is
  // ascending.  first[b] holds the run's index while the plan is built.
  struct Run {
    int32_t j0, j1, c, rid;
  };
  std::vector<int> run_off(n + 1, 0);
  std::vector<Run> runs;
  std::vector<std::vector<int32_t>> mem;
  std::vector<int32_t> starts;
  // the scan of every row for its runs, in parallel over positions
  std::vector<std::vector<Run>> pos_runs(n);
  parallel_for(n, [&](int pos) {
    const auto& row = p->table[ids[pos]];
    auto& out = pos_runs[pos];
    int j = 0;
    while (j < nb[pos]) {
      const int c = cnt[row[j]];
      if (c == 1) {
        out.push_back(Run{j, nb[pos], 1, -1});
        break;
      }
      int j1 = j + 1;
      while (j1 < nb[pos] && cnt[row[j1]] == c) ++j1;
      out.push_back(Run{j, j1, c, -1});
      j = j1;
    }
  });
  // member lists of the shared runs, in position order
  for (int pos = 0; pos < n; ++pos) {
    const auto& row = p->table[ids[pos]];
    run_off[pos] = (int)runs.size();
    for (Run R : pos_runs[pos]) {
      if (R.c > 1) {
        const int b0 = row[R.j0];
        if (p->first[b0] < 0) {
          p->first[b0] = (int)mem.size();
          mem.emplace_back();
          mem.back().reserve(R.c);
          starts.push_back(b0);
        }
        mem[p->first[b0]].push_back(pos);
        R.rid = p->first[b0];
      }
      runs.push_back(R);
    }
  }
  run_off[n] = (int)runs.size();
  for (int b : starts) p->first[b] = -1;
  for (int b : touched) p->cnt[b] = 0;

  // Chunk caps from the launch's own length.  A chunk is one unit's work, and
  // a unit that runs longer than the launch would take with its work spread
  // evenly sets the launch's length.  The estimate uses per-token times of
  // one unit by kind, read from per-wave timelines of MI355X launches: a
  // narrow unit on one wave (four to a workgroup slot), a cooperative item on
  // a whole slot, two slots per compute unit.  Narrow chunks are capped at a
  // fraction kCapNarrow of the estimated launch length, cooperative ones
  // (which start early) at kCapCoop.
  auto unit_us = [&](int rows) {  // us per token of the unit that takes `rows` rows
    if (rows <= narrow_rows) return fp8 ? (rows > gambit::kRowsPerUnit ? kUsNarrowTwo8 : kUsNarrow8) : kUsNarrow16;
    if (!fp8) return kUsCoop16;
    return rows <= 4 * gambit::kRowsPerUnit ? kUsCoop64_8 : kUsCoop128_8;
  };
  double launch_us = 0.0;
  {
    double slot_us = 0.0;
    for (int pos = 0; pos < n; ++pos)
      for (int r = run_off[pos]; r < run_off[pos + 1]; ++r) {
        const Run& R = runs[r];
        const double tok = 16.0 * (R.j1 - R.j0);
        const int rows = R.c * p->g;
        if (R.c == 1) {
          slot_us += tok * unit_us(rows) / 4;
        } else if (mem[R.rid][0] == pos) {
          slot_us += rows <= narrow_rows
                         ? tok * unit_us(rows) / 4
                         : tok * unit_us(std::min(rows, gambit::kRowsPerCoop)) * cdiv(rows, gambit::kRowsPerCoop);
        }
      }
    launch_us = slot_us * Hkv / (2.0 * p->n_cu);
  }
  // largest chunk (blocks) for a run of `rows` rows
  auto chunk_cap = [&](int rows) {
    const bool nar = rows <= narrow_rows;
    const double f = nar ? kCapNarrow : kCapCoop;
    return std::max(16.0, f * launch_us / unit_us(nar ? rows : std::min(rows, gambit::kRowsPerCoop)) / 16.0);
  };

  std::vector<Group> groups;
  std::vector<AttnUnit> gunits;  // the groups' units, contiguous per group
  std::vector<int32_t> members;
  std::vector<int32_t> nk(n, 0);
  gambit_status st = GAMBIT_OK;
  for (int chunk_blocks = kDefaultChunkBlocks;; chunk_blocks *= 2) {
    groups.clear();
    gunits.clear();
    members.clear();
    int worst = 0;
    // One group per (chunk, KV head): a chunk with <= narrow_rows rows is one
    // narrow unit; a wider chunk becomes cooperative items of up to 128 rows.
    auto emit = [&](int owner_pos, int jb0, int nblk, int ntok_est, const int32_t* mem_ids, int mcnt,
                    int kidx) {
      const int moff = (int)members.size();
      members.insert(members.end(), mem_ids, mem_ids + mcnt);
      const double tok = std::max(ntok_est, 1);
      if (mcnt * p->g <= narrow_rows) {
        for (int h = 0; h < Hkv; ++h) {
          groups.push_back(Group{tok, (int32_t)gunits.size(), 1, false});
          gunits.push_back(AttnUnit{ids[owner_pos], jb0, nblk, h, moff, mcnt, kidx, 0});
        }
        return;
      }
      const int item_members = gambit::kRowsPerCoop / p->g;
      for (int h = 0; h < Hkv; ++h) {
        Group gr{0.0, (int32_t)gunits.size(), 0, true};
        for (int m0 = 0; m0 < mcnt; m0 += item_members) {
          const int mc = std::min(item_members, mcnt - m0);
          gunits.push_back(AttnUnit{ids[owner_pos], jb0, nblk, h, moff + m0, mc, kidx, gambit::kUnitCoop});
          ++gr.count;
          gr.cost += tok * (2.0 + 4.0 * mc * p->g / 64.0);  // staging + compute per row
        }
        groups.push_back(gr);
      }
    };
    for (int pos = 0; pos < n; ++pos) {
      int kidx = 0;
      for (int r = run_off[pos]; r < run_off[pos + 1]; ++r) {
        const Run& R = runs[r];
        const int len = R.j1 - R.j0;
        // the caps apply to the first pass only: when the partial limit needs
        // longer chunks, the chunk lengths no longer depend on them
        const double grow = chunk_blocks == kDefaultChunkBlocks ? 1.0 : 1e9;
        if (R.c == 1) {  // private run: through the trace's last block, chunks of 4 chunk_blocks
          const int clen = (int)std::max(1.0, std::min(4.0 * chunk_blocks, chunk_cap(p->g) * grow));
          const int nch = std::max(1, cdiv(len, clen));
          for (int k = 0, jb = R.j0; k < nch; ++k) {
            const int sz = len / nch + (k < len % nch ? 1 : 0);
            const bool last = k == nch - 1;
            emit(pos, jb, last ? -1 : sz, sz * 16, &pos, 1, kidx++);
            jb += sz;
          }
          break;
        }
        // Chunk lengths (in units of chunk_blocks, 64 at first): 4 for runs
        // of narrow units, the row-block count up to 8 for wider runs
        // (cooperative items re-read their chunk per item, so longer chunks
        // mean fewer partials for the same bytes per row block).  Measured on
        // the 512-trace workload; shorter chunks lose more to per-unit
        // start-up and merging than they gain at the launch's tail.
        const bool nar = R.c * p->g <= narrow_rows;
        const int nrb = cdiv(R.c * p->g, gambit::kRowsPerUnit);
        const int clen = (int)std::max(1.0, std::min((double)chunk_blocks * (nar ? 4 : std::min(nrb, 8)),
                                                     chunk_cap(R.c * p->g) * grow));
        const int nch = cdiv(len, clen);
        const auto& ml = mem[R.rid];
        for (int k = 0, jb = R.j0; k < nch; ++k) {
          const int sz = len / nch + (k < len % nch ? 1 : 0);
          if (ml[0] == pos) emit(pos, jb, sz, sz * 16, ml.data(), R.c, kidx);
          ++kidx;
          jb += sz;
        }
        if (R.j1 == nb[pos]) emit(pos, R.j1, -1, 16, &pos, 1, kidx++);  // appends go past the shared prefix
      }
      nk[pos] = kidx;
      worst = std::max(worst, kidx);
    }
    if (worst <= kmax) {
      p->max_splits_used = worst;
      break;
    }
    if (chunk_blocks > p->d.max_blocks_per_trace) {
      st = fail(p, GAMBIT_ERR_UNSUPPORTED, "a trace needs %d attention partials, max_splits is %d",
                worst, kmax);
      break;
    }
  }
  if (st != GAMBIT_OK) return st;

  // Longest-processing-time assignment of groups to the 8 XCDs.
  std::vector<int> order(groups.size());
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return groups[a].cost > groups[b].cost; });
  double load[8] = {0};
  std::vector<std::vector<int>> per(8);
  for (int gi : order) {
    const int x = (int)(std::min_element(load, load + 8) - load);
    load[x] += groups[gi].cost;
    per[x].push_back(gi);
  }
  // Workgroup slots of four entries per XCD: a cooperative item (repeated
  // four times, flagged) or four narrow units.  The two kinds are interleaved
  // in proportion so compute-bound and HBM-bound workgroups share every CU,
  // the cooperative items over the first part of the narrow slots: they are
  // the long ones, and one that starts late ends the launch late.  bf16
  // (bound by HBM): over the first 85% (853 vs 858 us at 512 traces with all
  // of them; 50% starts too few narrow units early there: 947 vs 936-939 us,
  // though at 256 traces it gives 268 vs 273 us).
  // fp8 (bound by instruction issue, where the cooperative items' share of
  // the work starting early matters more than the overlap): over the first
  // 50% (217-220 vs 233-241 us at 256 traces; 45%: 226, 55%: 228, 70%: 224).
  const long spread_pct = p->d.kv_dtype == GAMBIT_KV_FP8_E4M3 ? 50 : 85;
  std::vector<AttnUnit> units;
  units.reserve(4 * gunits.size() + 8 * gambit::kUnitsPerWG);  // a cooperative item fills a 4-entry slot
  const AttnUnit empty{0, 0, 0, 0, 0, 0, 0, 0};
  std::vector<AttnUnit> C, N;
  for (int x = 0; x < 8; ++x) {
    p->xcd_off[x] = (int)units.size();
    C.clear();
    N.clear();
    for (int gi : per[x]) {
      const Group& g = groups[gi];
      (g.coop ? C : N).insert((g.coop ? C : N).end(), gunits.begin() + g.first, gunits.begin() + g.first + g.count);
    }
    const long nC = (long)C.size(), nN = cdiv((int)N.size(), gambit::kUnitsPerWG);
    long ci = 0, ni = 0;
    while (ci < nC || ni < nN) {
      if (ni >= nN || (ci < nC && ci * std::max(1L, nN * spread_pct / 100) <= ni * nC)) {
        for (int w = 0; w < gambit::kUnitsPerWG; ++w) units.push_back(C[ci]);
        ++ci;
      } else {
        for (int w = 0; w < gambit::kUnitsPerWG; ++w) {
          const size_t k = (size_t)ni * gambit::kUnitsPerWG + w;
          units.push_back(k < N.size() ? N[k] : empty);
        }
        ++ni;
      }
    }
  }
  p->xcd_off[8] = (int)units.size();
  // one workgroup per slot, and at least as many per XCD as that XCD has
  // slots outside its run-time claimed tail
  int per_xcd = cdiv((int)units.size() / gambit::kUnitsPerWG, 8);
  for (int x = 0; x < 8; ++x)
    per_xcd = std::max(per_xcd, (p->xcd_off[x + 1] - p->xcd_off[x]) / gambit::kUnitsPerWG - gambit::kTailSlots);
  p->grid = 8 * per_xcd;
  p->n_units = (int)units.size();
  if ((int)units.size() > p->L.max_units || (int)members.size() > p->L.max_members)
    return fail(p, GAMBIT_ERR_UNSUPPORTED, "plan exceeds workspace bounds");
  // The kinds of work covering each list position, as the kernel will pick
  // them (gambit_plan_kinds): a slot in an XCD's last kTailSlots is claimed
  // at run time.
  p->plan_kinds.assign(n, 0);
  for (int x = 0; x < 8; ++x) {
    const int nslots = (p->xcd_off[x + 1] - p->xcd_off[x]) / gambit::kUnitsPerWG;
    const int tail0 = std::max(nslots - gambit::kTailSlots, 0);
    for (int j = 0; j < nslots; ++j) {
      const int base = p->xcd_off[x] + gambit::kUnitsPerWG * j;
      const int32_t tail = j >= tail0 ? GAMBIT_UNIT_TAIL_SLOT : 0;
      auto mark = [&](const AttnUnit& u, int32_t kind) {
        for (int m = 0; m < u.mem_cnt; ++m) p->plan_kinds[members[u.mem_off + m]] |= kind | tail;
      };
      const AttnUnit& u0 = units[base];
      if (u0.flags & gambit::kUnitCoop) {
        const int rows = u0.mem_cnt * p->g;
        mark(u0, rows > 4 * gambit::kRowsPerUnit ? GAMBIT_UNIT_COOP_TWO : GAMBIT_UNIT_COOP_ONE);
      } else {
        for (int w = 0; w < gambit::kUnitsPerWG; ++w) {
          const AttnUnit& u = units[base + w];
          mark(u, u.mem_cnt * p->g > gambit::kRowsPerUnit ? GAMBIT_UNIT_NARROW_TWO : GAMBIT_UNIT_NARROW);
        }
      }
    }
  }

  // upload: list, nk, members, units through the pinned plan stage
  HIP_TRY(p, hipEventSynchronize(p->plan_ev), "plan fence");
  uint8_t* st8 = p->plan_stage;
  size_t o = 0;
  auto put = [&](const void* src, size_t bytes, void* dst) -> hipError_t {
    std::memcpy(st8 + o, src, bytes);
    const hipError_t e = hipMemcpyAsync(dst, st8 + o, bytes, hipMemcpyHostToDevice, s);
    o = align_up(o + bytes);
    return e;
  };
  HIP_TRY(p, put(ids, 4 * (size_t)n, ws_ptr<int32_t>(p, p->L.list)), "plan upload");
  HIP_TRY(p, put(nk.data(), 4 * (size_t)n, ws_ptr<int32_t>(p, p->L.nk)), "plan upload");
  if (!members.empty())
    HIP_TRY(p, put(members.data(), 4 * members.size(), ws_ptr<int32_t>(p, p->L.members)), "plan upload");
  if (!units.empty())
    HIP_TRY(p, put(units.data(), sizeof(AttnUnit) * units.size(), ws_ptr<AttnUnit>(p, p->L.units)),
            "plan upload");
  HIP_TRY(p, hipEventRecord(p->plan_ev, s), "plan fence");
  p->plan_list.assign(ids, ids + n);
  p->plan_valid = true;
  p->stats.n_units = p->n_units;
  p->stats.max_splits_used = p->max_splits_used;
  return GAMBIT_OK;
}

void invalidate_plan(gambit_pool* p) { p->plan_valid = false; }

}  // namespace

// =============================================================================
namespace {

// Calls that change or check the pool wait for an open decode step to end.
gambit_status step_open(gambit_pool* p) {
  return fail(p, GAMBIT_ERR_INVALID, "a decode step is open: layer %d of %d is next", p->step_next,
              p->dev.num_layers);
}

}  // namespace

extern "C" {

const char* gambit_status_str(gambit_status s) {
  switch (s) {
    case GAMBIT_OK: return "ok";
    case GAMBIT_ERR_INVALID: return "invalid argument";
    case GAMBIT_ERR_OUT_OF_BLOCKS: return "out of KV blocks";
    case GAMBIT_ERR_SHARED_WRITE: return "write into a shared block";
    case GAMBIT_ERR_UNSUPPORTED: return "unsupported";
    case GAMBIT_ERR_DEVICE: return "device error";
    case GAMBIT_ERR_WORKSPACE: return "workspace too small";
    default: return "unknown status";
  }
}

const char* gambit_last_error(const gambit_pool* pool) { return pool ? pool->last_error.c_str() : ""; }

size_t gambit_workspace_size(const gambit_pool_desc* desc) {
  Layout L;
  return layout_of(desc, &L) ? L.total : 0;
}

gambit_status gambit_pool_create(const gambit_pool_desc* desc, void* stream, gambit_pool** out) {
  if (!out) return GAMBIT_ERR_INVALID;
  *out = nullptr;
  Layout L;
  if (!layout_of(desc, &L)) return GAMBIT_ERR_INVALID;
  if (!desc->k_cache || !desc->v_cache || !desc->block_table || !desc->seq_len || !desc->refcount ||
      !desc->workspace)
    return GAMBIT_ERR_INVALID;
  if ((desc->kv_dtype == GAMBIT_KV_FP8_E4M3) != (desc->kv_scale != nullptr)) return GAMBIT_ERR_INVALID;
  if (desc->workspace_bytes < L.total) return GAMBIT_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(desc->workspace) % kAlign) return GAMBIT_ERR_INVALID;

  auto* p = new gambit_pool;
  p->d = *desc;
  p->L = L;
  p->ws = static_cast<uint8_t*>(desc->workspace);
  p->g = desc->num_q_heads / desc->num_kv_heads;
  if (desc->fp8_append_scale > 0.f) p->append_scale = desc->fp8_append_scale;

  gambit::DevPool& D = p->dev;
  D.k_cache = static_cast<uint8_t*>(desc->k_cache);
  D.v_cache = static_cast<uint8_t*>(desc->v_cache);
  D.kv_scale = desc->kv_scale;
  D.table = desc->block_table;
  D.seq_len = desc->seq_len;
  D.refcount = desc->refcount;
  D.freebits = ws_ptr<uint32_t>(p, L.freebits);
  D.alloc_list = ws_ptr<int32_t>(p, L.alloc_list);
  D.err = ws_ptr<int32_t>(p, L.err);
  D.sbar = ws_ptr<float>(p, L.sbar);
  D.nscore = ws_ptr<int32_t>(p, L.nscore);
  D.gen = ws_ptr<int32_t>(p, L.gen);
  D.ghost = ws_ptr<int32_t>(p, L.ghost);
  D.num_blocks = desc->num_blocks;
  D.nwords = L.nwords;
  D.max_traces = desc->max_traces;
  D.max_blocks = desc->max_blocks_per_trace;
  D.Hq = desc->num_q_heads;
  D.Hkv = desc->num_kv_heads;
  D.g = p->g;
  D.esize = desc->kv_dtype == GAMBIT_KV_FP8_E4M3 ? 1 : 2;
  D.num_layers = desc->num_layers ? desc->num_layers : 1;
  D.layer_bytes = (size_t)desc->num_blocks * desc->num_kv_heads * 16 * 128 * D.esize;

  p->table.assign(desc->max_traces, {});
  p->seq_len.assign(desc->max_traces, 0);
  p->refcount.assign(desc->num_blocks, 0);
  p->nscore.assign(desc->max_traces, 0);
  p->gen.assign(desc->max_traces, 0);
  p->ghost.assign(desc->max_traces, 0);
  p->cnt.assign(desc->num_blocks, 0);  // per-block counter of the planner and the round's out-of-blocks test
  p->freebits.assign(cdiv(desc->num_blocks, 64), ~0ull);
  if (desc->num_blocks % 64) p->freebits.back() = (1ull << (desc->num_blocks % 64)) - 1;
  p->nfree = desc->num_blocks;

  p->stage_ints = 8 * (size_t)desc->max_traces + 2 * ((size_t)desc->max_blocks_per_trace + 1) * D.num_layers;
  p->plan_stage_bytes = 4 * align_up(4 * (size_t)desc->max_traces) + sizeof(AttnUnit) * (size_t)L.max_units +
                        4 * (size_t)L.max_members + 4 * kAlign;
  hipError_t e = hipHostMalloc(reinterpret_cast<void**>(&p->stage), p->stage_ints * 4, hipHostMallocDefault);
  if (e == hipSuccess) e = hipHostMalloc(reinterpret_cast<void**>(&p->plan_stage), p->plan_stage_bytes, hipHostMallocDefault);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&p->stage_ev, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&p->plan_ev, hipEventDisableTiming);

  if (e == hipSuccess) {
    int dev = 0, ncu = 0;
    e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess && ncu > 0) p->n_cu = ncu;
  }
  if (e == hipSuccess) e = hipEventRecord(p->stage_ev, S(stream));
  if (e == hipSuccess) e = hipEventRecord(p->plan_ev, S(stream));
  if (e == hipSuccess) e = hipMemsetAsync(p->ws + L.ticket, 0, 64, S(stream));
  if (e == hipSuccess) e = hipMemsetAsync(p->ws + L.queues, 0, 64, S(stream));
  if (e == hipSuccess) e = gambit::launch_pool_init(D, S(stream));
  if (e != hipSuccess) {
    gambit_pool_destroy(p);
    return GAMBIT_ERR_DEVICE;
  }
  *out = p;
  return GAMBIT_OK;
}

gambit_status gambit_pool_destroy(gambit_pool* p) {
  if (!p) return GAMBIT_ERR_INVALID;
  if (p->stage_ev) (void)hipEventSynchronize(p->stage_ev);
  if (p->plan_ev) (void)hipEventSynchronize(p->plan_ev);
  if (p->stage) (void)hipHostFree(p->stage);
  if (p->plan_stage) (void)hipHostFree(p->plan_stage);
  for (hipEvent_t e : p->prof_ev) (void)hipEventDestroy(e);
  if (p->stage_ev) (void)hipEventDestroy(p->stage_ev);
  if (p->plan_ev) (void)hipEventDestroy(p->plan_ev);

  delete p;
  return GAMBIT_OK;
}

int32_t gambit_seq_len(const gambit_pool* p, int32_t t) {
  return (p && t >= 0 && t < p->d.max_traces) ? p->seq_len[t] : -1;
}

int32_t gambit_free_blocks(const gambit_pool* p) { return p ? p->nfree : -1; }

gambit_status gambit_kv_alloc(gambit_pool* p, int32_t n, const int32_t* ids, const int32_t* ntok,
                              void* stream) {
  if (!p) return GAMBIT_ERR_INVALID;
  if (p->step_next) return step_open(p);
  gambit_status st = check_ids(p, n, ids, "trace");
  if (st) return st;
  if (n > 0 && !ntok) return fail(p, GAMBIT_ERR_INVALID, "token counts are NULL");
  long need = 0;
  for (int i = 0; i < n; ++i) {
    if (ntok[i] < 0) return fail(p, GAMBIT_ERR_INVALID, "negative token count");
    if (p->ghost[ids[i]]) return fail(p, GAMBIT_ERR_INVALID, "slot %d holds a ghost trace", ids[i]);
    const long L = p->seq_len[ids[i]];
    if (cdiv((int)std::min<long>(L + ntok[i], 1L << 30), 16) > p->d.max_blocks_per_trace)
      return fail(p, GAMBIT_ERR_INVALID, "trace %d would exceed max_blocks_per_trace", ids[i]);
    need += cdiv((int)(L + ntok[i]), 16) - cdiv((int)L, 16);
  }
  if (need > p->nfree) return fail(p, GAMBIT_ERR_OUT_OF_BLOCKS, "need %ld blocks, %d free", need, p->nfree);
  if (n == 0) return GAMBIT_OK;
  int32_t* rt = ws_ptr<int32_t>(p, p->L.req_trace);
  int32_t* rn = ws_ptr<int32_t>(p, p->L.req_ntok);
  std::vector<int32_t> both(ids, ids + n);
  both.insert(both.end(), ntok, ntok + n);
  HIP_TRY(p, hipEventSynchronize(p->stage_ev), "staging fence");
  std::memcpy(p->stage, both.data(), 8 * (size_t)n);
  HIP_TRY(p, hipMemcpyAsync(rt, p->stage, 4 * (size_t)n, hipMemcpyHostToDevice, S(stream)), "upload");
  HIP_TRY(p, hipMemcpyAsync(rn, p->stage + n, 4 * (size_t)n, hipMemcpyHostToDevice, S(stream)), "upload");
  HIP_TRY(p, hipEventRecord(p->stage_ev, S(stream)), "staging fence");
  HIP_TRY(p, gambit::launch_alloc(p->dev, rt, rn, -1, n, 1.0f, false, S(stream)), "alloc kernel");
  for (int i = 0; i < n; ++i) mirror_grow(p, ids[i], ntok[i]);
  invalidate_plan(p);
  return GAMBIT_OK;
}

gambit_status gambit_kv_write(gambit_pool* p, int32_t t, int32_t pos0, int32_t n, const void* k,
                              const void* v, const float* scales, void* stream) {
  if (!p) return GAMBIT_ERR_INVALID;
  if (p->step_next) return step_open(p);
  if (t < 0 || t >= p->d.max_traces) return fail(p, GAMBIT_ERR_INVALID, "trace id %d out of range", t);
  if (pos0 < 0 || n < 0 || (long)pos0 + n > p->seq_len[t])
    return fail(p, GAMBIT_ERR_INVALID, "write [%d, %d) outside trace %d's %d positions", pos0, pos0 + n, t,
                p->seq_len[t]);
  if (n == 0) return GAMBIT_OK;
  if (!k || !v) return fail(p, GAMBIT_ERR_INVALID, "K or V is NULL");
  for (int j = pos0 / 16; j <= (pos0 + n - 1) / 16; ++j)
    if (p->refcount[p->table[t][j]] != 1)
      return fail(p, GAMBIT_ERR_SHARED_WRITE, "block %d of trace %d is shared", j, t);
  const int first = cdiv(pos0, 16), last = (pos0 + n - 1) / 16;
  const int started = std::max(0, last - first + 1);
  const bool fp8 = p->d.kv_dtype == GAMBIT_KV_FP8_E4M3;
  if (!fp8 && scales) return fail(p, GAMBIT_ERR_INVALID, "scales are only for fp8 pools");
  if (fp8 && started > 0 && !scales) return fail(p, GAMBIT_ERR_INVALID, "fp8 write needs block scales");
  float* dsc = nullptr;
  if (fp8 && started > 0) {
    dsc = ws_ptr<float>(p, p->L.scales);
    gambit_status st = upload_ints(p, reinterpret_cast<int32_t*>(dsc),
                                   reinterpret_cast<const int32_t*>(scales),
                                   2 * (size_t)started * p->dev.num_layers, S(stream));
    if (st) return st;
  }
  HIP_TRY(p, gambit::launch_write(p->dev, t, pos0, n, k, v, dsc, S(stream)), "write kernel");
  return GAMBIT_OK;
}

gambit_status gambit_kv_fork(gambit_pool* p, int32_t n, const int32_t* parents, const int32_t* children,
                             void* stream) {
  if (!p) return GAMBIT_ERR_INVALID;
  if (p->step_next) return step_open(p);
  std::vector<char> is_child;
  gambit_status st = check_ids(p, n, children, "child", &is_child);
  if (st) return st;
  if (n > 0 && !parents) return fail(p, GAMBIT_ERR_INVALID, "parent list is NULL");
  int tails = 0;
  for (int i = 0; i < n; ++i) {
    const int par = parents[i], ch = children[i];
    if (par < 0 || par >= p->d.max_traces) return fail(p, GAMBIT_ERR_INVALID, "parent id %d out of range", par);
    if (is_child[par]) return fail(p, GAMBIT_ERR_INVALID, "trace %d is both parent and child", par);
    if (p->seq_len[ch] != 0 || p->ghost[ch]) return fail(p, GAMBIT_ERR_INVALID, "child slot %d is not empty", ch);
    if (p->seq_len[par] == 0) return fail(p, GAMBIT_ERR_INVALID, "parent %d is empty", par);
    tails += p->seq_len[par] % 16 ? 1 : 0;
  }
  if (tails > p->nfree) return fail(p, GAMBIT_ERR_OUT_OF_BLOCKS, "need %d blocks, %d free", tails, p->nfree);
  if (n == 0) return GAMBIT_OK;
  std::vector<int32_t> pairs(2 * (size_t)n);
  for (int i = 0; i < n; ++i) {
    pairs[2 * i] = children[i];
    pairs[2 * i + 1] = parents[i];
  }
  int32_t* dp = ws_ptr<int32_t>(p, p->L.pairs);
  st = upload_ints(p, dp, pairs.data(), pairs.size(), S(stream));
  if (st) return st;
  HIP_TRY(p, gambit::launch_fork(p->dev, dp, n, ws_ptr<int32_t>(p, p->L.req_trace),
                                 ws_ptr<int32_t>(p, p->L.req_ntok), S(stream)),
          "fork kernels");
  mirror_fork_many(p, parents, children, n);
  invalidate_plan(p);
  return GAMBIT_OK;
}

gambit_status gambit_kv_free(gambit_pool* p, int32_t n, const int32_t* ids, void* stream) {
  if (!p) return GAMBIT_ERR_INVALID;
  if (p->step_next) return step_open(p);
  gambit_status st = check_ids(p, n, ids, "trace");
  if (st) return st;
  for (int i = 0; i < n; ++i)
    if (p->seq_len[ids[i]] == 0 && p->table[ids[i]].empty())
      return fail(p, GAMBIT_ERR_INVALID, "trace %d is already empty", ids[i]);
  if (n == 0) return GAMBIT_OK;
  int32_t* d = ws_ptr<int32_t>(p, p->L.ids);
  st = upload_ints(p, d, ids, n, S(stream));
  if (st) return st;
  HIP_TRY(p, gambit::launch_free(p->dev, d, n, gambit::kFreeEnd, S(stream)), "free kernel");
  mirror_free_many(p, ids, n);
  invalidate_plan(p);
  return GAMBIT_OK;
}

// One layer of a decode step.  Layer 0 opens the step: it validates the
// list, plans the launch, and takes the blocks the step opens.  The mirror
// takes them by the allocation rule (lowest free ids, in list order); when
// they fit in the launch arguments the layer-0 attention launch enters them
// and the last layer's merge advances the lengths, otherwise the allocator
// kernel enters them (and advances the lengths) before layer 0.
static gambit_status decode_layer(gambit_pool* p, int32_t layer, int32_t n, const int32_t* ids, const void* q,
                           const void* k_new, const void* v_new, int32_t new_dtype, void* out,
                           int32_t out_dtype, float sm_scale, void* stream) {
  if (!p) return GAMBIT_ERR_INVALID;
  const int nl = p->dev.num_layers;
  if (layer != p->step_next)
    return fail(p, GAMBIT_ERR_INVALID, "decode layer %d called, layer %d of %d is next", layer, p->step_next, nl);
  gambit_status st = check_ids(p, n, ids, "trace");
  if (st) return st;
  if (n == 0) return GAMBIT_OK;
  if (!q || !k_new || !v_new || !out) return fail(p, GAMBIT_ERR_INVALID, "NULL buffer");
  if (out_dtype != GAMBIT_OUT_BF16 && out_dtype != GAMBIT_OUT_F32)
    return fail(p, GAMBIT_ERR_INVALID, "bad output dtype");
  if (new_dtype != GAMBIT_NEW_CACHE && new_dtype != GAMBIT_NEW_BF16)
    return fail(p, GAMBIT_ERR_INVALID, "bad dtype of the new K/V");
  if (!std::isfinite(sm_scale)) return fail(p, GAMBIT_ERR_INVALID, "softmax scale is not finite");
  hipStream_t s = S(stream);
  gambit::AttnLaunch& A = p->step;
  if (layer == 0) {
    int need = 0;
    for (int i = 0; i < n; ++i) {
      const int L = p->seq_len[ids[i]];
      if (L == 0) return fail(p, GAMBIT_ERR_INVALID, "trace %d is empty", ids[i]);
      if (cdiv(L + 1, 16) > p->d.max_blocks_per_trace)
        return fail(p, GAMBIT_ERR_INVALID, "trace %d is full", ids[i]);
      need += L % 16 == 0;
    }
    if (need > p->nfree) return fail(p, GAMBIT_ERR_OUT_OF_BLOCKS, "need %d blocks, %d free", need, p->nfree);
    if (!p->plan_valid || (int)p->plan_list.size() != n ||
        !std::equal(p->plan_list.begin(), p->plan_list.end(), ids)) {
      st = build_plan(p, n, ids, s);
      if (st) return st;
    }
    const int32_t* dlist = ws_ptr<int32_t>(p, p->L.list);
    A = gambit::AttnLaunch{};
    const bool in_args = need <= gambit::kMaxArgBlocks;
    if (!in_args)
      HIP_TRY(p, gambit::launch_alloc(p->dev, dlist, nullptr, 1, n, p->append_scale, true, s), "append alloc");
    A.list = dlist;
    A.len_bias = in_args ? 1 : 0;
    A.new_scale = p->append_scale;
    for (int i = 0; i < n; ++i) {
      const bool opens = p->seq_len[ids[i]] % 16 == 0;
      mirror_grow(p, ids[i], 1);
      ++p->gen[ids[i]];
      if (opens && in_args) {
        A.new_pos[A.n_new] = i;
        A.new_blk[A.n_new++] = p->table[ids[i]].back();
      }
    }
    A.units = ws_ptr<AttnUnit>(p, p->L.units);
    std::memcpy(A.xcd_off, p->xcd_off, sizeof A.xcd_off);
    A.grid = p->grid;
    A.queues = ws_ptr<int32_t>(p, p->L.queues);
    A.members = ws_ptr<int32_t>(p, p->L.members);
    A.nk = ws_ptr<int32_t>(p, p->L.nk);
    A.part_acc = ws_ptr<float>(p, p->L.part_acc);
    A.part_ml = ws_ptr<float2>(p, p->L.part_ml);
    A.kmax = p->L.kmax;
    A.n = n;
    p->stats.total_tokens += n;
    p->stats.unique_tokens += n;
    p->stats.unique_blocks += need;
    p->stats.table_entries += need;
  } else if (n != A.n || !std::equal(p->plan_list.begin(), p->plan_list.end(), ids)) {
    return fail(p, GAMBIT_ERR_INVALID, "layer %d of a step lists other traces than layer 0", layer);
  }
  A.q = static_cast<const uint16_t*>(q);
  A.k_new = static_cast<const uint8_t*>(k_new);  // appended by the attention launch
  A.v_new = static_cast<const uint8_t*>(v_new);
  A.scale_log2 = sm_scale * 1.4426950408889634f;
  A.out = out;
  A.out_f32 = out_dtype == GAMBIT_OUT_F32;
  A.claim = layer == 0;
  A.advance = layer == nl - 1;
  A.new_bf16 = new_dtype == GAMBIT_NEW_BF16 && p->d.kv_dtype == GAMBIT_KV_FP8_E4M3;
  p->step_next = layer + 1 == nl ? 0 : layer + 1;
  const gambit::DevPool D = p->dev.layer(layer);
  // The merge kernel leaves the slot counters at zero for the next launch;
  // only after a launch that was not followed by its merge are they
  // cleared here.
  if (p->queues_dirty) HIP_TRY(p, hipMemsetAsync(A.queues, 0, 64, s), "slot counter reset");
  p->queues_dirty = true;
  const bool timed = p->prof_on && p->prof_used + 2 <= (int)p->prof_ev.size();
  if (timed) HIP_TRY(p, hipEventRecord(p->prof_ev[p->prof_used], s), "profile event");
  HIP_TRY(p, gambit::launch_attention_units(D, A, s), "attention");
  if (timed) {
    HIP_TRY(p, hipEventRecord(p->prof_ev[p->prof_used + 1], s), "profile event");
    p->prof_used += 2;
  }
  HIP_TRY(p, gambit::launch_attention_merge(D, A, s), "attention merge");
  p->queues_dirty = false;
  return GAMBIT_OK;
}

gambit_status gambit_decode_attn(gambit_pool* p, int32_t n, const int32_t* ids, const void* q,
                                 const void* k_new, const void* v_new, void* out, int32_t out_dtype,
                                 float sm_scale, void* stream) {
  if (!p) return GAMBIT_ERR_INVALID;
  if (p->dev.num_layers != 1)
    return fail(p, GAMBIT_ERR_INVALID, "the pool has %d layers: decode with gambit_decode_attn_layer",
                p->dev.num_layers);
  return decode_layer(p, 0, n, ids, q, k_new, v_new, GAMBIT_NEW_CACHE, out, out_dtype, sm_scale, stream);
}

gambit_status gambit_decode_attn_layer(gambit_pool* p, int32_t layer, int32_t n, const int32_t* ids,
                                       const void* q, const void* k_new, const void* v_new, int32_t new_dtype,
                                       void* out, int32_t out_dtype, float sm_scale, void* stream) {
  return decode_layer(p, layer, n, ids, q, k_new, v_new, new_dtype, out, out_dtype, sm_scale, stream);
}

gambit_status gambit_score_prune_branch(gambit_pool* p, int32_t n, const int32_t* ids, const void* h,
                                        int32_t Dh, const float* w, float b, int32_t keep,
                                        int32_t n_parents, float* scores_out, int32_t* keep_out,
                                        int32_t* child_parent_out, void* stream) {
  if (!p) return GAMBIT_ERR_INVALID;
  if (p->step_next) return step_open(p);
  gambit_status st = check_ids(p, n, ids, "trace");
  if (st) return st;
  if (n == 0 || n > gambit::kMaxRank) return fail(p, GAMBIT_ERR_UNSUPPORTED, "population size %d", n);
  if (!h || !w || !scores_out || !keep_out) return fail(p, GAMBIT_ERR_INVALID, "NULL buffer");
  if (Dh <= 0 || Dh % 8) return fail(p, GAMBIT_ERR_INVALID, "probe dimension %d is not a multiple of 8", Dh);
  if (keep < 1 || keep > n) return fail(p, GAMBIT_ERR_INVALID, "keep %d of %d", keep, n);
  const int nfree_traces = n - keep;
  if (nfree_traces > 0) {
    if (n_parents < 1 || n_parents > keep || nfree_traces % n_parents)
      return fail(p, GAMBIT_ERR_INVALID, "%d pruned traces do not split over %d parents", nfree_traces, n_parents);
    if (!child_parent_out) return fail(p, GAMBIT_ERR_INVALID, "NULL child/parent buffer");
  }
  for (int i = 0; i < n; ++i)
    if (p->seq_len[ids[i]] == 0) return fail(p, GAMBIT_ERR_INVALID, "trace %d is empty", ids[i]);
  hipStream_t s = S(stream);
  int32_t* dids = ws_ptr<int32_t>(p, p->L.ids);
  st = upload_ints(p, dids, ids, n, s);
  if (st) return st;
  gambit::ProbeLaunch PL{};
  PL.list = dids;
  PL.n = n;
  PL.h = static_cast<const uint16_t*>(h);
  PL.Dh = Dh;
  PL.w = w;
  PL.b = b;
  PL.keep = keep;
  PL.n_parents = nfree_traces > 0 ? n_parents : 0;
  PL.scores_out = scores_out;
  PL.keep_out = keep_out;
  PL.pairs_out = nfree_traces > 0 ? child_parent_out : ws_ptr<int32_t>(p, p->L.pairs);
  PL.free_list = ws_ptr<int32_t>(p, p->L.free_list);
  PL.ticket = ws_ptr<uint32_t>(p, p->L.ticket);
  HIP_TRY(p, gambit::launch_probe_rank(PL, s), "probe/rank kernel");
  // the one blocking readback: the ranking
  std::vector<int32_t> kept(keep), pairs(2 * (size_t)nfree_traces);
  HIP_TRY(p, hipMemcpyAsync(kept.data(), keep_out, 4 * (size_t)keep, hipMemcpyDeviceToHost, s), "readback");
  if (nfree_traces > 0)
    HIP_TRY(p, hipMemcpyAsync(pairs.data(), child_parent_out, 8 * (size_t)nfree_traces, hipMemcpyDeviceToHost, s),
            "readback");
  HIP_TRY(p, hipStreamSynchronize(s), "readback");
  // host check of the device plan, then the exact out-of-blocks test
  std::vector<char> in_list(p->d.max_traces, 0), is_kept(p->d.max_traces, 0);
  for (int i = 0; i < n; ++i) in_list[ids[i]] = 1;
  for (int t : kept) {
    if (t < 0 || t >= p->d.max_traces || !in_list[t] || is_kept[t])
      return fail(p, GAMBIT_ERR_DEVICE, "device ranking returned an invalid id %d", t);
    is_kept[t] = 1;
  }
  std::vector<int32_t> freed;
  for (int t = 0; t < p->d.max_traces; ++t)
    if (in_list[t] && !is_kept[t]) freed.push_back(t);
  const int c = nfree_traces > 0 ? nfree_traces / n_parents : 0;
  for (int j = 0; j < nfree_traces; ++j)
    if (pairs[2 * j] != freed[j] || pairs[2 * j + 1] != kept[j / c])
      return fail(p, GAMBIT_ERR_DEVICE, "device prune/branch plan disagrees with the ranking");
  if (nfree_traces == 0) return GAMBIT_OK;
  int tails = 0;
  for (int j = 0; j < nfree_traces; ++j) tails += p->seq_len[kept[j / c]] % 16 ? 1 : 0;
  if (tails > p->nfree) {
    // Only now count the blocks pruning releases: references the pruned
    // rows drop per block (the planner's per-block counter, left at zero).
    int released = 0;
    for (int t : freed)
      for (int blk : p->table[t]) released += ++p->cnt[blk] == p->refcount[blk];
    for (int t : freed)
      for (int blk : p->table[t]) p->cnt[blk] = 0;
    if (tails > p->nfree + released)
      return fail(p, GAMBIT_ERR_OUT_OF_BLOCKS, "branching needs %d blocks, %d free after pruning", tails,
                  p->nfree + released);
  }
  HIP_TRY(p, gambit::launch_free(p->dev, PL.free_list, nfree_traces, gambit::kFreeEnd, s), "free kernel");
  HIP_TRY(p, gambit::launch_fork(p->dev, child_parent_out, nfree_traces, ws_ptr<int32_t>(p, p->L.req_trace),
                                 ws_ptr<int32_t>(p, p->L.req_ntok), s),
          "fork kernels");
  std::vector<int32_t> par(nfree_traces);
  for (int j = 0; j < nfree_traces; ++j) par[j] = kept[j / c];
  mirror_free_many(p, freed.data(), nfree_traces);
  mirror_fork_many(p, par.data(), freed.data(), nfree_traces);
  invalidate_plan(p);
  return GAMBIT_OK;
}

gambit_status gambit_plan_kinds(gambit_pool* p, int32_t n, const int32_t* ids, int32_t* kinds_out) {
  if (!p) return GAMBIT_ERR_INVALID;
  if (n < 0 || (n > 0 && (!ids || !kinds_out))) return fail(p, GAMBIT_ERR_INVALID, "bad list or output");
  if (!p->plan_valid || (int)p->plan_list.size() != n || !std::equal(p->plan_list.begin(), p->plan_list.end(), ids))
    return fail(p, GAMBIT_ERR_INVALID, "no attention plan for this trace list (run a decode step first)");
  std::copy(p->plan_kinds.begin(), p->plan_kinds.end(), kinds_out);
  return GAMBIT_OK;
}

gambit_status gambit_rank_topk(int32_t n, const int32_t* ids, const float* scores, int32_t keep,
                               int32_t* keep_out, void* stream) {
  if (n <= 0 || n > gambit::kMaxRank || keep < 1 || keep > n || !ids || !scores || !keep_out)
    return GAMBIT_ERR_INVALID;
  return gambit::launch_rank_topk(n, ids, scores, keep, keep_out, S(stream)) == hipSuccess ? GAMBIT_OK
                                                                                             : GAMBIT_ERR_DEVICE;
}

namespace {

// Traces listed for scoring or eviction must be running.
gambit_status check_running(gambit_pool* p, int32_t n, const int32_t* ids) {
  gambit_status st = check_ids(p, n, ids, "trace");
  if (st) return st;
  for (int i = 0; i < n; ++i)
    if (p->seq_len[ids[i]] == 0) return fail(p, GAMBIT_ERR_INVALID, "trace %d is not running", ids[i]);
  return GAMBIT_OK;
}

}  // namespace

gambit_status gambit_score_update(gambit_pool* p, int32_t n, const int32_t* ids, const void* h, int32_t Dh,
                                  const float* w, float b, float* scores_out, void* stream) {
  if (!p) return GAMBIT_ERR_INVALID;
  gambit_status st = check_running(p, n, ids);
  if (st) return st;
  if (n == 0) return GAMBIT_OK;
  if (!h || !w || !scores_out) return fail(p, GAMBIT_ERR_INVALID, "NULL buffer");
  if (Dh <= 0 || Dh % 8) return fail(p, GAMBIT_ERR_INVALID, "probe dimension %d is not a multiple of 8", Dh);
  int32_t* d = ws_ptr<int32_t>(p, p->L.ids);
  st = upload_ints(p, d, ids, n, S(stream));
  if (st) return st;
  gambit::ScoreLaunch L{d, n, static_cast<const uint16_t*>(h), Dh, w, b, scores_out};
  HIP_TRY(p, gambit::launch_score_update(p->dev, L, S(stream)), "score kernel");
  for (int i = 0; i < n; ++i) ++p->nscore[ids[i]];
  return GAMBIT_OK;
}

gambit_status gambit_evict(gambit_pool* p, int32_t n, const int32_t* ids, int32_t* victim_out, void* stream) {
  if (!p) return GAMBIT_ERR_INVALID;
  if (p->step_next) return step_open(p);
  gambit_status st = check_running(p, n, ids);
  if (st) return st;
  if (n == 0 || !victim_out) return fail(p, GAMBIT_ERR_INVALID, "no eviction candidates");
  if (n > gambit::kMaxRank) return fail(p, GAMBIT_ERR_UNSUPPORTED, "%d candidates", n);
  hipStream_t s = S(stream);
  int32_t* d = ws_ptr<int32_t>(p, p->L.ids);
  int32_t* out = ws_ptr<int32_t>(p, p->L.tourn);
  st = upload_ints(p, d, ids, n, s);
  if (st) return st;
  HIP_TRY(p, gambit::launch_evict_pick(p->dev, d, n, out, s), "eviction kernel");
  int32_t v = -1;
  HIP_TRY(p, hipMemcpyAsync(&v, out, 4, hipMemcpyDeviceToHost, s), "readback");
  HIP_TRY(p, hipStreamSynchronize(s), "readback");
  if (std::find(ids, ids + n, v) == ids + n) return fail(p, GAMBIT_ERR_DEVICE, "device chose a non-candidate %d", v);
  HIP_TRY(p, gambit::launch_free(p->dev, out, 1, gambit::kFreeEvict, s), "free kernel");
  mirror_evict(p, v);
  invalidate_plan(p);
  *victim_out = v;
  return GAMBIT_OK;
}

gambit_status gambit_tournament(gambit_pool* p, int32_t capacity, int32_t swap_k, int32_t warmup,
                                gambit_round* round_out, int32_t* pruned_out, int32_t* child_parent_out,
                                int32_t* ranked_out, void* stream) {
  if (!p) return GAMBIT_ERR_INVALID;
  if (p->step_next) return step_open(p);
  const int T = p->d.max_traces;
  if (T > gambit::kMaxRank) return fail(p, GAMBIT_ERR_UNSUPPORTED, "%d trace slots", T);
  if (capacity < 1 || capacity > T || swap_k < 0 || warmup < 0)
    return fail(p, GAMBIT_ERR_INVALID, "capacity %d (slots %d), swap %d, warmup %d", capacity, T, swap_k, warmup);
  if (!round_out || !pruned_out || !child_parent_out) return fail(p, GAMBIT_ERR_INVALID, "NULL output");
  hipStream_t s = S(stream);
  int32_t* out = ws_ptr<int32_t>(p, p->L.tourn);
  HIP_TRY(p, gambit::launch_tournament(p->dev, capacity, swap_k, warmup, out, ranked_out, s), "tournament kernel");
  std::vector<int32_t> h((size_t)gambit::kTournHeader + 3 * (size_t)T);
  HIP_TRY(p, hipMemcpyAsync(h.data(), out, 4 * h.size(), hipMemcpyDeviceToHost, s), "readback");
  HIP_TRY(p, hipStreamSynchronize(s), "readback");
  // check the device plan against everything the mirror knows (all but the scores)
  const int kase = h[0], N = h[1], npr = h[2], m = h[3], nvac = h[4];
  const int32_t* pr = h.data() + gambit::kTournHeader;
  const int32_t* pairs = pr + T;
  int Nh = 0;
  for (int t = 0; t < T; ++t) Nh += p->seq_len[t] > 0 || p->ghost[t];
  const int kase_h = Nh == 0 ? 0 : (Nh < capacity ? 1 : 2);
  const int npr_h = kase_h == 2 ? std::min(swap_k, Nh) : 0;
  if (N != Nh || kase != kase_h || npr != npr_h)
    return fail(p, GAMBIT_ERR_DEVICE, "device tournament (case %d, N %d, pruned %d) disagrees with the mirror "
                "(case %d, N %d, pruned %d)", kase, N, npr, kase_h, Nh, npr_h);
  std::vector<char> gone(T, 0), par(T, 0);
  for (int i = 0; i < npr; ++i) {
    const int t = pr[i];
    if (t < 0 || t >= T || !(p->seq_len[t] > 0 || p->ghost[t]) || (i && pr[i - 1] >= t))
      return fail(p, GAMBIT_ERR_DEVICE, "device pruned an invalid trace %d", t);
    gone[t] = 1;
  }
  int nb = 0;
  for (int t = 0; t < T; ++t) nb += !gone[t] && p->seq_len[t] > 0 && !p->ghost[t] && p->gen[t] >= warmup;
  const int m_h = kase_h == 1 ? std::min(capacity - Nh, nb) : (kase_h == 2 ? std::min(swap_k, nb) : 0);
  std::vector<int32_t> vac;
  for (int t = 0; t < T; ++t)
    if ((p->seq_len[t] == 0 && !p->ghost[t]) || gone[t]) vac.push_back(t);
  if (m != m_h || nvac != (int)vac.size() || nvac < m)
    return fail(p, GAMBIT_ERR_DEVICE, "device tournament branches %d (mirror %d), vacant %d (mirror %d)", m, m_h,
                nvac, (int)vac.size());
  int tails = 0;
  for (int j = 0; j < m; ++j) {
    const int c = pairs[2 * j], q = pairs[2 * j + 1];
    if (c != vac[j] || q < 0 || q >= T || gone[q] || p->seq_len[q] == 0 || p->ghost[q] || p->gen[q] < warmup ||
        par[q])
      return fail(p, GAMBIT_ERR_DEVICE, "device branch %d -> %d is invalid", q, c);
    par[q] = 1;
    tails += p->seq_len[q] % 16 ? 1 : 0;
  }
  if (tails > p->nfree) {
    int released = 0;
    for (int i = 0; i < npr; ++i)
      for (int blk : p->table[pr[i]]) released += ++p->cnt[blk] == p->refcount[blk];
    for (int i = 0; i < npr; ++i)
      for (int blk : p->table[pr[i]]) p->cnt[blk] = 0;
    if (tails > p->nfree + released)
      return fail(p, GAMBIT_ERR_OUT_OF_BLOCKS, "branching needs %d blocks, %d free after pruning", tails,
                  p->nfree + released);
  }
  // apply: end the pruned traces (running and ghost), then branch
  HIP_TRY(p, gambit::launch_free(p->dev, out + gambit::kTournHeader, npr, gambit::kFreeEnd, s), "free kernel");
  HIP_TRY(p, gambit::launch_fork(p->dev, out + gambit::kTournHeader + T, m, ws_ptr<int32_t>(p, p->L.req_trace),
                                 ws_ptr<int32_t>(p, p->L.req_ntok), s),
          "fork kernels");
  mirror_free_many(p, pr, npr);
  std::vector<int32_t> fork_par(m), fork_ch(m);
  for (int j = 0; j < m; ++j) {
    fork_ch[j] = pairs[2 * j];
    fork_par[j] = pairs[2 * j + 1];
  }
  mirror_fork_many(p, fork_par.data(), fork_ch.data(), m);
  invalidate_plan(p);
  round_out->case_taken = kase;
  round_out->n_active = N;
  round_out->n_pruned = npr;
  round_out->n_children = m;
  std::copy(pr, pr + npr, pruned_out);
  std::copy(pairs, pairs + 2 * m, child_parent_out);
  return GAMBIT_OK;
}

gambit_status gambit_record_scores(gambit_pool* p, int32_t n, const int32_t* ids, const float* f, void* stream) {
  if (!p) return GAMBIT_ERR_INVALID;
  gambit_status st = check_running(p, n, ids);
  if (st) return st;
  if (n == 0) return GAMBIT_OK;
  if (!f) return fail(p, GAMBIT_ERR_INVALID, "NULL scores");
  int32_t* d = ws_ptr<int32_t>(p, p->L.ids);
  st = upload_ints(p, d, ids, n, S(stream));
  if (st) return st;
  HIP_TRY(p, gambit::launch_record_scores(p->dev, d, f, n, S(stream)), "record kernel");
  for (int i = 0; i < n; ++i) ++p->nscore[ids[i]];
  return GAMBIT_OK;
}

gambit_status gambit_trace_state(gambit_pool* p, int32_t n, const int32_t* ids, float* sbar_out,
                                 int32_t* nscore_out, int32_t* gen_out, int32_t* ghost_out, void* stream) {
  if (!p) return GAMBIT_ERR_INVALID;
  gambit_status st = check_ids(p, n, ids, "trace");
  if (st) return st;
  const int T = p->d.max_traces;
  std::vector<float> sb(T);
  std::vector<int32_t> ns(T), ge(T), gh(T);
  HIP_TRY(p, hipStreamSynchronize(S(stream)), "sync");
  HIP_TRY(p, hipMemcpy(sb.data(), p->ws + p->L.sbar, 4 * (size_t)T, hipMemcpyDeviceToHost), "state read");
  HIP_TRY(p, hipMemcpy(ns.data(), p->ws + p->L.nscore, 4 * (size_t)T, hipMemcpyDeviceToHost), "state read");
  HIP_TRY(p, hipMemcpy(ge.data(), p->ws + p->L.gen, 4 * (size_t)T, hipMemcpyDeviceToHost), "state read");
  HIP_TRY(p, hipMemcpy(gh.data(), p->ws + p->L.ghost, 4 * (size_t)T, hipMemcpyDeviceToHost), "state read");
  for (int i = 0; i < n; ++i) {
    const int t = ids[i];
    if (sbar_out) sbar_out[i] = sb[t];
    if (nscore_out) nscore_out[i] = ns[t];
    if (gen_out) gen_out[i] = ge[t];
    if (ghost_out) ghost_out[i] = gh[t];
  }
  return GAMBIT_OK;
}

gambit_status gambit_pool_check(gambit_pool* p, void* stream) {
  if (!p) return GAMBIT_ERR_INVALID;
  if (p->step_next) return step_open(p);
  hipStream_t s = S(stream);
  HIP_TRY(p, hipStreamSynchronize(s), "sync");
  const int T = p->d.max_traces, MB = p->d.max_blocks_per_trace, NB = p->d.num_blocks;
  std::vector<int32_t> tab((size_t)T * MB), len(T), ref(NB), err(1);
  std::vector<uint32_t> bits(p->L.nwords);
  HIP_TRY(p, hipMemcpy(tab.data(), p->d.block_table, 4 * tab.size(), hipMemcpyDeviceToHost), "check read");
  HIP_TRY(p, hipMemcpy(len.data(), p->d.seq_len, 4 * (size_t)T, hipMemcpyDeviceToHost), "check read");
  HIP_TRY(p, hipMemcpy(ref.data(), p->d.refcount, 4 * (size_t)NB, hipMemcpyDeviceToHost), "check read");
  HIP_TRY(p, hipMemcpy(err.data(), p->ws + p->L.err, 4, hipMemcpyDeviceToHost), "check read");
  HIP_TRY(p, hipMemcpy(bits.data(), p->ws + p->L.freebits, 4 * bits.size(), hipMemcpyDeviceToHost), "check read");
  std::vector<int32_t> nsc(T), gen(T), gh(T);
  HIP_TRY(p, hipMemcpy(nsc.data(), p->ws + p->L.nscore, 4 * (size_t)T, hipMemcpyDeviceToHost), "check read");
  HIP_TRY(p, hipMemcpy(gen.data(), p->ws + p->L.gen, 4 * (size_t)T, hipMemcpyDeviceToHost), "check read");
  HIP_TRY(p, hipMemcpy(gh.data(), p->ws + p->L.ghost, 4 * (size_t)T, hipMemcpyDeviceToHost), "check read");
  if (err[0]) return fail(p, GAMBIT_ERR_DEVICE, "device error word 0x%x", err[0]);
  for (int t = 0; t < T; ++t)
    if (nsc[t] != p->nscore[t] || gen[t] != p->gen[t] || (gh[t] != 0) != (p->ghost[t] != 0))
      return fail(p, GAMBIT_ERR_DEVICE, "tournament state of trace %d: device (%d, %d, %d), host (%d, %d, %d)", t,
                  nsc[t], gen[t], gh[t], p->nscore[t], p->gen[t], (int)p->ghost[t]);
  for (int t = 0; t < T; ++t) {
    if (len[t] != p->seq_len[t]) return fail(p, GAMBIT_ERR_DEVICE, "seq_len[%d]: device %d, host %d", t, len[t], p->seq_len[t]);
    const auto& row = p->table[t];
    for (int j = 0; j < MB; ++j) {
      const int want = j < (int)row.size() ? row[j] : -1;
      if (tab[(size_t)t * MB + j] != want)
        return fail(p, GAMBIT_ERR_DEVICE, "table[%d][%d]: device %d, host %d", t, j, tab[(size_t)t * MB + j], want);
    }
  }
  for (int b = 0; b < NB; ++b) {
    if (ref[b] != p->refcount[b]) return fail(p, GAMBIT_ERR_DEVICE, "refcount[%d]: device %d, host %d", b, ref[b], p->refcount[b]);
    const bool dfree = (bits[b >> 5] >> (b & 31)) & 1;
    const bool hfree = (p->freebits[b >> 6] >> (b & 63)) & 1;
    if (dfree != hfree) return fail(p, GAMBIT_ERR_DEVICE, "free bit of block %d: device %d, host %d", b, dfree, hfree);
  }
  return GAMBIT_OK;
}

gambit_status gambit_plan_stats(gambit_pool* p, int32_t n, const int32_t* ids, gambit_stats* out) {
  if (!p || !out) return GAMBIT_ERR_INVALID;
  gambit_status st = check_ids(p, n, ids, "trace");
  if (st) return st;
  if (p->plan_valid && (int)p->plan_list.size() == n && std::equal(p->plan_list.begin(), p->plan_list.end(), ids)) {
    *out = p->stats;
    return GAMBIT_OK;
  }
  std::vector<char> seen(p->d.num_blocks, 0);
  gambit_stats r{};
  for (int i = 0; i < n; ++i) {
    const int t = ids[i], L = p->seq_len[t];
    r.total_tokens += L;
    const auto& row = p->table[t];
    r.table_entries += (int64_t)row.size();
    for (size_t j = 0; j < row.size(); ++j) {
      if (seen[row[j]]) continue;
      seen[row[j]] = 1;
      ++r.unique_blocks;
      r.unique_tokens += std::min(16, L - 16 * (int)j);
    }
  }
  r.n_units = -1;
  r.max_splits_used = -1;
  *out = r;
  return GAMBIT_OK;
}

gambit_status gambit_profile_begin(gambit_pool* p, int32_t max_launches) {
  if (!p || max_launches < 0) return GAMBIT_ERR_INVALID;
  for (hipEvent_t e : p->prof_ev) (void)hipEventDestroy(e);
  p->prof_ev.assign(2 * (size_t)max_launches, nullptr);
  for (auto& e : p->prof_ev) HIP_TRY(p, hipEventCreate(&e), "profile events");
  p->prof_used = 0;
  p->prof_on = true;
  return GAMBIT_OK;
}

gambit_status gambit_profile_end(gambit_pool* p, double* attn_ms, int32_t* launches) {
  if (!p || !attn_ms || !launches) return GAMBIT_ERR_INVALID;
  double total = 0;
  if (p->prof_used > 0) HIP_TRY(p, hipEventSynchronize(p->prof_ev[p->prof_used - 1]), "profile sync");
  for (int i = 0; i + 1 < p->prof_used; i += 2) {
    float ms = 0;
    HIP_TRY(p, hipEventElapsedTime(&ms, p->prof_ev[i], p->prof_ev[i + 1]), "profile read");
    total += ms;
  }
  *attn_ms = total;
  *launches = p->prof_used / 2;
  for (hipEvent_t e : p->prof_ev) (void)hipEventDestroy(e);
  p->prof_ev.clear();
  p->prof_used = 0;
  p->prof_on = false;
  return GAMBIT_OK;
}

}  // extern "C"
