// Probe GEMV + sigmoid + ranking + prune/branch plan, fused in one launch.
//
// At a thought boundary each trace's hidden state h is scored by the linear
// sigmoid probe sigma(w.h + b) (the head form of Eq. 6 applied to h), the
// population is ranked by score (Alg. 1 Tournament: rank descending; ties go
// to the lower trace id), the traces outside the top `keep` are pruned and
// the freed slots are handed to children of the top `n_parents` (Eq. 3,
// generalised to (n - keep) / n_parents children per parent).
//
// One wave scores one trace (128-bit loads of h and w, shuffle reduction).
// The last workgroup to finish - found with an atomic ticket after a
// device-scope fence - sorts 64-bit keys (orderable score bits, inverted id)
// in LDS (a run-merge sort up to 1024 traces, a bitonic network beyond),
// writes the kept ids and the child -> parent pairs, and resets the ticket.
#include <cmath>

#include "kernels.h"

namespace gambit {
namespace {

constexpr int kProbeThreads = 256;

__device__ inline uint32_t orderable(float f) {
  const uint32_t u = __builtin_bit_cast(uint32_t, f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline float bf16_lo(uint32_t x) { return __builtin_bit_cast(float, x << 16); }
__device__ inline float bf16_hi(uint32_t x) { return __builtin_bit_cast(float, x & 0xFFFF0000u); }

// h . w over Dh (a multiple of 8) by one wave: each lane takes 8
// consecutive elements per 512-element step (128-bit loads); the loads of
// four steps are issued before their products, then a shuffle reduction;
// every lane returns the sum.
__device__ inline float probe_dot(const uint16_t* h, const float* w, int Dh, int lane) {
  float acc = 0.f;
  for (int d0 = lane * 8; d0 < Dh; d0 += 4 * 64 * 8) {
    uint4 hv[4];
    float4 w0[4], w1[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int d = d0 + u * 64 * 8;
      if (d < Dh) {
        hv[u] = *reinterpret_cast<const uint4*>(h + d);
        w0[u] = *reinterpret_cast<const float4*>(w + d);
        w1[u] = *reinterpret_cast<const float4*>(w + d + 4);
      } else {
        hv[u] = make_uint4(0u, 0u, 0u, 0u);
        w0[u] = w1[u] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      acc = fmaf(bf16_lo(hv[u].x), w0[u].x, acc);
      acc = fmaf(bf16_hi(hv[u].x), w0[u].y, acc);
      acc = fmaf(bf16_lo(hv[u].y), w0[u].z, acc);
      acc = fmaf(bf16_hi(hv[u].y), w0[u].w, acc);
      acc = fmaf(bf16_lo(hv[u].z), w1[u].x, acc);
      acc = fmaf(bf16_hi(hv[u].z), w1[u].y, acc);
      acc = fmaf(bf16_lo(hv[u].w), w1[u].z, acc);
      acc = fmaf(bf16_hi(hv[u].w), w1[u].w, acc);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  return acc;
}

// Sort keys[0..N) descending (N a power of two) with all threads of the block.
__device__ inline uint64_t shfl_xor64(uint64_t v, int m) {
  const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, m, 64);
  const uint32_t hi = (uint32_t)__shfl_xor((int)(uint32_t)(v >> 32), m, 64);
  return ((uint64_t)hi << 32) | lo;
}

// Bitonic sort, descending, of keys[0 .. N) (N a power of two) by the
// workgroup.  Compare-exchange stages whose partners are 128 or more apart
// go through LDS with a barrier each; the rest of a merge step stays inside
// 128-key blocks, which one wave holds in registers (keys base + lane and
// base + 64 + lane): distance 64 pairs a lane's two keys, shorter distances
// pair lanes by shuffles - one LDS round trip and one barrier for all of
// them.  Keys past N (when N < 128) pair only among themselves.
__device__ void bitonic_desc(uint64_t* keys, int N) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int k = 2; k <= N; k <<= 1) {
    int j = k >> 1;
    for (; j >= 128; j >>= 1) {
      for (int i = threadIdx.x; i < N; i += blockDim.x) {
        const int ixj = i ^ j;
        if (ixj > i) {
          const uint64_t a = keys[i], b = keys[ixj];
          const bool desc = (i & k) == 0;
          if (desc ? (a < b) : (a > b)) {
            keys[i] = b;
            keys[ixj] = a;
          }
        }
      }
      __syncthreads();
    }
    for (int base = 128 * wave; base < N; base += 128 * nw) {
      const int ia = base + lane, ib = ia + 64;
      uint64_t a = keys[ia], b = keys[ib];
      const bool desc_a = (ia & k) == 0, desc_b = (ib & k) == 0;
      for (int jj = j; jj > 0; jj >>= 1) {
        if (jj == 64) {  // a (index ia) is the lower of the pair (ia, ib); k >= 128 here
          if (desc_a ? (a < b) : (a > b)) {
            const uint64_t t = a;
            a = b;
            b = t;
          }
        } else {
          const uint64_t pa = shfl_xor64(a, jj), pb = shfl_xor64(b, jj);
          const bool lower = (lane & jj) == 0;
          a = (lower == desc_a) ? (a > pa ? a : pa) : (a < pa ? a : pa);
          b = (lower == desc_b) ? (b > pb ? b : pb) : (b < pb ? b : pb);
        }
      }
      keys[ia] = a;
      keys[ib] = b;
    }
    __syncthreads();
  }
}

// Sort of up to kMergeMax keys, descending, without a barrier per merge
// stage: every wave sorts runs of 128 keys in registers (two keys per lane;
// partners 64 apart are a lane's own pair, closer ones are exchanged by
// shuffles), then each key's final position is its place in its run plus,
// for every other run, the number of that run's keys ahead of it (a binary
// search; equal keys count as ahead when they come from an earlier run, so
// the positions are a permutation).  512 keys: 7.7 us for a ranking launch
// against 10.3 us with the bitonic network, whose stages each need a
// barrier; beyond 1024 keys the searches cost more than the network.
constexpr int kMergeMax = 1024;

__device__ __attribute__((always_inline)) inline void sort_runs128(const uint64_t* src, uint64_t* dst, int nruns) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
  for (int r = wave; r < nruns; r += nw) {
    uint64_t a = src[128 * r + lane], b = src[128 * r + 64 + lane];
    for (int k = 2; k <= 128; k <<= 1) {
      const bool desc_a = (lane & k) == 0, desc_b = ((64 + lane) & k) == 0;
      for (int j = k >> 1; j > 0; j >>= 1) {
        if (j == 64) {  // only for k == 128: a run-wide descending merge, a is the lower index
          if (a < b) {
            const uint64_t t = a;
            a = b;
            b = t;
          }
        } else {
          const uint64_t pa = shfl_xor64(a, j), pb = shfl_xor64(b, j);
          const bool lower = (lane & j) == 0;
          a = (lower == desc_a) ? (a > pa ? a : pa) : (a < pa ? a : pa);
          b = (lower == desc_b) ? (b > pb ? b : pb) : (b < pb ? b : pb);
        }
      }
    }
    dst[128 * r + lane] = a;
    dst[128 * r + 64 + lane] = b;
  }
}

// Number of keys of the descending run A[0..128) ahead of x: greater, or
// also equal when `ge`.
__device__ inline int ahead_in_run(const uint64_t* A, uint64_t x, bool ge) {
  int c = 0;
#pragma unroll
  for (int s = 64; s > 0; s >>= 1) {
    const uint64_t y = A[c + s - 1];
    c += (ge ? y >= x : y > x) ? s : 0;
  }
  const uint64_t y = A[c];  // c <= 127 here
  return c + ((ge ? y >= x : y > x) ? 1 : 0);
}

// Sorts keys[0 .. N) descending (N a power of two, N <= kMaxRank) with all
// threads of the workgroup; ends with a barrier.
__device__ __attribute__((always_inline)) inline void sort_desc(uint64_t* keys, int N) {
  if (N > kMergeMax) {
    bitonic_desc(keys, N);
    return;
  }
  __shared__ uint64_t runs[kMergeMax];
  const int M = N < 128 ? 128 : N;  // whole runs; the extra keys are below every real key
  for (int i = N + threadIdx.x; i < M; i += blockDim.x) keys[i] = 0;
  __syncthreads();
  const int nruns = M / 128;
  sort_runs128(keys, runs, nruns);
  __syncthreads();
  for (int p = threadIdx.x; p < M; p += blockDim.x) {
    const uint64_t x = runs[p];
    const int r = p >> 7;
    int g = p & 127;
    for (int q = 0; q < nruns; ++q)
      if (q != r) g += ahead_in_run(runs + 128 * q, x, q < r);
    keys[g] = x;
  }
  __syncthreads();
}

// keys from (score, id): higher score first, then lower id first.
__device__ inline uint64_t rank_key(float score, int id) {
  return ((uint64_t)orderable(score) << 32) | (uint64_t)(~(uint32_t)id);
}

__device__ __attribute__((always_inline)) inline void rank_and_plan(int n, const int32_t* ids, const float* scores, bool atomic_scores,
                              int keep, int n_parents, int32_t* keep_out, int32_t* pairs_out,
                              int32_t* free_list) {
  __shared__ uint64_t keys[kMaxRank];
  int N = 1;
  while (N < n) N <<= 1;
  for (int i = threadIdx.x; i < N; i += blockDim.x) {
    if (i < n) {
      const float s = atomic_scores ? __hip_atomic_load(scores + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)
                                    : scores[i];
      keys[i] = rank_key(s, ids[i]);
    } else {
      keys[i] = 0;  // below every real key
    }
  }
  __syncthreads();
  sort_desc(keys, N);
  for (int r = threadIdx.x; r < keep; r += blockDim.x) keep_out[r] = (int32_t)~(uint32_t)keys[r];
  if (!pairs_out) return;
  // pruned ids (ranks keep..n-1), sorted ascending: sort inverted ids descending
  __syncthreads();
  for (int i = threadIdx.x; i < N; i += blockDim.x) {
    const bool pruned = i >= keep && i < n;
    const uint32_t id = (uint32_t)~(uint32_t)keys[i];
    keys[i] = pruned ? (uint64_t)(~id) : 0;
  }
  __syncthreads();
  sort_desc(keys, N);
  const int nfree = n - keep;
  const int c = n_parents > 0 ? nfree / n_parents : 0;
  __syncthreads();
  // keep_out is read back from global memory written above by this block
  for (int j = threadIdx.x; j < nfree; j += blockDim.x) {
    const int child = (int)~(uint32_t)keys[j];
    free_list[j] = child;
    pairs_out[2 * j] = child;
    pairs_out[2 * j + 1] = c > 0 ? keep_out[j / c] : -1;
  }
}

__global__ __launch_bounds__(kProbeThreads) void probe_rank_kernel(ProbeLaunch L) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int i = blockIdx.x * (kProbeThreads / 64) + wave;
  if (i < L.n) {
    const float acc = probe_dot(L.h + (size_t)i * L.Dh, L.w, L.Dh, lane);
    if (lane == 0) {
      const float z = acc + L.b;
      L.scores_out[i] = 1.f / (1.f + expf(-z));
    }
  }
  // last workgroup ranks
  __shared__ bool last;
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) {
    const uint32_t t = atomicAdd(L.ticket, 1u);
    last = (t == gridDim.x - 1);
  }
  __syncthreads();
  if (!last) return;
  __threadfence();
  rank_and_plan(L.n, L.list, L.scores_out, true, L.keep, L.n_parents, L.keep_out, L.pairs_out,
                L.free_list);
  if (threadIdx.x == 0) *L.ticket = 0;
}

__global__ __launch_bounds__(kProbeThreads) void rank_topk_kernel(int n, const int32_t* ids,
                                                                  const float* scores, int keep,
                                                                  int32_t* keep_out) {
  rank_and_plan(n, ids, scores, false, keep, 0, keep_out, nullptr, nullptr);
}

// ------------------------------------------------------------- tournament --
// The full tournament of Alg. 1 keeps per trace slot a running mean score
// s_bar over its thoughts, the tokens it has generated since its creation
// (GenLen) and a ghost flag (Sec. 4.2: evicted by the scheduler, no KV, no
// tokens, still in the tree view).

constexpr int kTournThreads = 256;

// Exclusive scan of one int per thread over the 256 threads.
__device__ int scan256(int v, int* total) {
  __shared__ int wsum[kTournThreads / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int x = __shfl_up(incl, off);
    if (lane >= off) incl += x;
  }
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  int before = 0, all = 0;
#pragma unroll
  for (int k = 0; k < kTournThreads / 64; ++k) {
    before += k < w ? wsum[k] : 0;
    all += wsum[k];
  }
  __syncthreads();
  *total = all;
  return before + incl - v;
}

__device__ inline int key_id(uint64_t key) { return (int)~(uint32_t)key; }

// One wave per listed trace: the thought score f = sigmoid(h . w + b), then
// the running mean over the trace's thoughts (Alg. 1 Generate).
__global__ __launch_bounds__(kProbeThreads) void score_update_kernel(DevPool P, ScoreLaunch L) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int i = blockIdx.x * (kProbeThreads / 64) + wave;
  if (i >= L.n) return;
  const float acc = probe_dot(L.h + (size_t)i * L.Dh, L.w, L.Dh, lane);
  if (lane == 0) {
    const float f = 1.f / (1.f + expf(-(acc + L.b)));
    const int t = L.list[i];
    const int n = P.nscore[t] + 1;
    P.sbar[t] += (f - P.sbar[t]) / (float)n;
    P.nscore[t] = n;
    L.scores_out[i] = f;
  }
}

// The listed trace ranked last by (s_bar descending, id ascending): the
// smallest rank key.
__global__ __launch_bounds__(kTournThreads) void evict_pick_kernel(DevPool P, const int32_t* list, int n,
                                                                   int32_t* out) {
  __shared__ uint64_t wmin[kTournThreads / 64];
  uint64_t mn = ~0ull;
  for (int i = threadIdx.x; i < n; i += kTournThreads) {
    const int t = list[i];
    const uint64_t k = rank_key(P.sbar[t], t);
    mn = k < mn ? k : mn;
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const uint64_t o = __shfl_xor(mn, off);
    mn = o < mn ? o : mn;
  }
  if ((threadIdx.x & 63) == 0) wmin[threadIdx.x >> 6] = mn;
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int k = 1; k < kTournThreads / 64; ++k) mn = wmin[k] < mn ? wmin[k] : mn;
    out[0] = key_id(mn);
  }
}

// One workgroup plans a tournament round over the tree view (every slot
// that is running or a ghost): rank by (s_bar descending, id ascending);
// N < C: Case 1, branch the top min(C - N, |B|) eligible traces (Eq. 2);
// N >= C: Case 2, prune the bottom min(K, N), branch the top min(K, |B|)
// eligible traces that were not pruned (Eq. 3).  Eligible: running (not a
// ghost) with GenLen >= w.  Children take the lowest vacant slots
// (ascending) after the pruning, one per parent in rank order.  The plan is
// only written out; the host applies it after checking it.
__global__ __launch_bounds__(kTournThreads) void tournament_kernel(DevPool P, int C, int K, int w,
                                                                   int32_t* out, int32_t* ranked_out) {
  __shared__ uint64_t keys[kMaxRank];
  __shared__ uint8_t pruned[kMaxRank];
  const int T = P.max_traces;
  int Np2 = 1;
  while (Np2 < T) Np2 <<= 1;
  int nact = 0;
  for (int i = threadIdx.x; i < Np2; i += kTournThreads) {
    const bool act = i < T && (P.seq_len[i] > 0 || P.ghost[i] != 0);
    keys[i] = act ? rank_key(P.sbar[i], i) : 0;  // inactive slots sort last
    pruned[i] = 0;
    nact += act;
  }
  int N = 0;
  scan256(nact, &N);  // also a barrier
  sort_desc(keys, Np2);
  const int kase = N == 0 ? 0 : (N < C ? 1 : 2);
  const int npr = kase == 2 ? min(K, N) : 0;
  for (int r = N - npr + threadIdx.x; r < N; r += kTournThreads) pruned[key_id(keys[r])] = 1;
  __syncthreads();
  int32_t* out_pruned = out + kTournHeader;
  int32_t* out_pairs = out_pruned + T;
  const int per = (T + kTournThreads - 1) / kTournThreads;
  const int r0 = threadIdx.x * per, r1 = min(r0 + per, T);
  // parents: eligible ranks in order
  auto eligible = [&](int r) {
    if (r >= N) return false;
    const int t = key_id(keys[r]);
    return !pruned[t] && P.seq_len[t] > 0 && P.ghost[t] == 0 && P.gen[t] >= w;
  };
  int cnt = 0;
  for (int r = r0; r < r1; ++r) cnt += eligible(r);
  int nb = 0;
  int at = scan256(cnt, &nb);
  const int m = kase == 1 ? min(C - N, nb) : (kase == 2 ? min(K, nb) : 0);
  for (int r = r0; r < r1; ++r)
    if (eligible(r)) {
      if (at < m) out_pairs[2 * at + 1] = key_id(keys[r]);
      ++at;
    }
  // children: the lowest vacant slots after the pruning
  auto vacant = [&](int t) { return (P.seq_len[t] == 0 && P.ghost[t] == 0) || pruned[t]; };
  cnt = 0;
  for (int t = r0; t < r1; ++t) cnt += vacant(t);
  int nvac = 0;
  at = scan256(cnt, &nvac);
  for (int t = r0; t < r1; ++t)
    if (vacant(t)) {
      if (at < m) out_pairs[2 * at] = t;
      ++at;
    }
  // the pruned ids, ascending
  cnt = 0;
  for (int t = r0; t < r1; ++t) cnt += pruned[t];
  int np = 0;
  at = scan256(cnt, &np);
  for (int t = r0; t < r1; ++t)
    if (pruned[t]) out_pruned[at++] = t;
  if (ranked_out)
    for (int r = threadIdx.x; r < N; r += kTournThreads) ranked_out[r] = key_id(keys[r]);
  if (threadIdx.x == 0) {
    out[0] = kase;
    out[1] = N;
    out[2] = npr;
    out[3] = m;
    out[4] = nvac;
  }
}

__global__ void record_scores_kernel(DevPool P, const int32_t* list, const float* f, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n) return;
  const int t = list[i];
  const int c = P.nscore[t] + 1;
  P.sbar[t] += (f[i] - P.sbar[t]) / (float)c;
  P.nscore[t] = c;
}

}  // namespace

hipError_t launch_record_scores(const DevPool& P, const int32_t* list, const float* f, int32_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(record_scores_kernel, dim3((n + 255) / 256), dim3(256), 0, s, P, list, f, n);
  return hipGetLastError();
}

hipError_t launch_score_update(const DevPool& P, const ScoreLaunch& L, hipStream_t s) {
  if (L.n <= 0) return hipSuccess;
  const int wpb = kProbeThreads / 64;
  hipLaunchKernelGGL(score_update_kernel, dim3((L.n + wpb - 1) / wpb), dim3(kProbeThreads), 0, s, P, L);
  return hipGetLastError();
}

hipError_t launch_evict_pick(const DevPool& P, const int32_t* list, int32_t n, int32_t* out, hipStream_t s) {
  hipLaunchKernelGGL(evict_pick_kernel, dim3(1), dim3(kTournThreads), 0, s, P, list, n, out);
  return hipGetLastError();
}

hipError_t launch_tournament(const DevPool& P, int32_t capacity, int32_t swap_k, int32_t warmup,
                             int32_t* out, int32_t* ranked_out, hipStream_t s) {
  hipLaunchKernelGGL(tournament_kernel, dim3(1), dim3(kTournThreads), 0, s, P, capacity, swap_k, warmup,
                     out, ranked_out);
  return hipGetLastError();
}

hipError_t launch_probe_rank(const ProbeLaunch& L, hipStream_t s) {
  const int wpb = kProbeThreads / 64;
  hipLaunchKernelGGL(probe_rank_kernel, dim3((L.n + wpb - 1) / wpb), dim3(kProbeThreads), 0, s, L);
  return hipGetLastError();
}

hipError_t launch_rank_topk(int32_t n, const int32_t* ids, const float* scores, int32_t keep,
                            int32_t* keep_out, hipStream_t s) {
  hipLaunchKernelGGL(rank_topk_kernel, dim3(1), dim3(kProbeThreads), 0, s, n, ids, scores, keep,
                     keep_out);
  return hipGetLastError();
}

}  // namespace gambit
