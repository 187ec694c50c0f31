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
// device-scope fence - ranks all scores with a bitonic sort of 64-bit keys
// (orderable score bits, inverted id) in LDS, writes the kept ids and the
// child -> parent pairs, and resets the ticket.
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

// Sort keys[0..N) descending (N a power of two) with all threads of the block.
__device__ void bitonic_desc(uint64_t* keys, int N) {
  for (int k = 2; k <= N; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
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
  }
}

// keys from (score, id): higher score first, then lower id first.
__device__ inline uint64_t rank_key(float score, int id) {
  return ((uint64_t)orderable(score) << 32) | (uint64_t)(~(uint32_t)id);
}

__device__ void rank_and_plan(int n, const int32_t* ids, const float* scores, bool atomic_scores,
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
  bitonic_desc(keys, N);
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
  bitonic_desc(keys, N);
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
    const uint16_t* h = L.h + (size_t)i * L.Dh;
    float acc = 0.f;
    // Dh is a multiple of 8: each lane takes 8 consecutive elements per step
    for (int d = lane * 8; d < L.Dh; d += 64 * 8) {
      const uint4 hv = *reinterpret_cast<const uint4*>(h + d);
      const float4 w0 = *reinterpret_cast<const float4*>(L.w + d);
      const float4 w1 = *reinterpret_cast<const float4*>(L.w + d + 4);
      acc = fmaf(bf16_lo(hv.x), w0.x, acc);
      acc = fmaf(bf16_hi(hv.x), w0.y, acc);
      acc = fmaf(bf16_lo(hv.y), w0.z, acc);
      acc = fmaf(bf16_hi(hv.y), w0.w, acc);
      acc = fmaf(bf16_lo(hv.z), w1.x, acc);
      acc = fmaf(bf16_hi(hv.z), w1.y, acc);
      acc = fmaf(bf16_lo(hv.w), w1.z, acc);
      acc = fmaf(bf16_hi(hv.w), w1.w, acc);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
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

}  // namespace

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
