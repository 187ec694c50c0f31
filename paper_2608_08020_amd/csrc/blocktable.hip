// Block-table kernels: pool initialisation, lowest-free-first allocation,
// KV writes, prune (free) and branch (fork).
//
// Branch spawns a child from its parent's prefix by sharing the parent's KV
// blocks (Alg. 1 notation; Sec. 4.1 Case 2), so a fork copies block ids and
// bumps refcounts; only a partially filled last block is copied, because
// both traces keep appending into their own copy of it.  Prune frees the
// blocks nobody else references (Sec. 4.1 Case 2).
#include "kernels.h"

namespace gambit {
namespace {

constexpr int kAllocThreads = 1024;

__device__ inline int cdiv16(int x) { return (x + kBlock - 1) / kBlock; }

__global__ void pool_init_kernel(DevPool P) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  const size_t i0 = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t ntab = (size_t)P.max_traces * P.max_blocks;
  for (size_t i = i0; i < ntab; i += stride) P.table[i] = -1;
  for (size_t i = i0; i < (size_t)P.max_traces; i += stride) {
    P.seq_len[i] = 0;
    P.sbar[i] = 0.f;
    P.nscore[i] = 0;
    P.gen[i] = 0;
    P.ghost[i] = 0;
  }
  for (size_t i = i0; i < (size_t)P.num_blocks; i += stride) P.refcount[i] = 0;
  for (size_t w = i0; w < (size_t)P.nwords; w += stride) {
    const int lo = (int)w * 32;
    const int valid = min(32, P.num_blocks - lo);
    P.freebits[w] = valid >= 32 ? 0xFFFFFFFFu : ((1u << valid) - 1u);
  }
  if (i0 == 0) *P.err = 0;
}

// Exclusive scan of one int per thread across the workgroup (kAllocThreads
// = 16 waves): a shuffle scan inside each wave, then the wave totals.
__device__ int wg_exclusive_scan(int v, int* total) {
  __shared__ int wsum[kAllocThreads / 64];
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
  for (int k = 0; k < kAllocThreads / 64; ++k) {
    const int s = wsum[k];
    before += k < w ? s : 0;
    all += s;
  }
  __syncthreads();  // wsum may be reused
  *total = all;
  return before + incl - v;
}

// One workgroup.  Request i extends trace req_trace[i] by its token count;
// the blocks it needs are the next lowest free ids, in request order and
// ascending logical index.  The free bitmap is read in coalesced passes of
// one word per thread, only as far as the lowest `total` free blocks reach:
// a counting pass first (so a short pool is left untouched), then the
// assignment.
__global__ __launch_bounds__(kAllocThreads) void alloc_kernel(DevPool P, const int32_t* req_trace,
                                                             const int32_t* req_ntok, int32_t uniform,
                                                             int32_t m, float new_scale, int32_t generated) {
  const int t = threadIdx.x;
  const int rpt = (m + kAllocThreads - 1) / kAllocThreads;
  const int r0 = min(m, t * rpt), r1 = min(m, r0 + rpt);
  int need = 0;
  for (int i = r0; i < r1; ++i) {
    const int L = P.seq_len[req_trace[i]];
    const int nt = uniform >= 0 ? uniform : req_ntok[i];
    need += cdiv16(L + nt) - cdiv16(L);
  }
  int total = 0;
  const int base = wg_exclusive_scan(need, &total);
  if (total > 0) {  // uniform across the workgroup
    const int npass = (P.nwords + kAllocThreads - 1) / kAllocThreads;
    int last = -1, found = 0;  // passes that hold the lowest `total` free blocks
    for (int p = 0; p < npass && found < total; ++p) {
      const int w = p * kAllocThreads + t;
      int c = w < P.nwords ? __popc(P.freebits[w]) : 0, n = 0;
      wg_exclusive_scan(c, &n);
      found += n;
      last = p;
    }
    if (found < total) {  // the host mirror rules this out; leave the pool untouched
      if (t == 0) atomicOr(P.err, kErrAllocShort);
      return;
    }
    int acc = 0;
    for (int p = 0; p <= last; ++p) {
      const int w = p * kAllocThreads + t;
      uint32_t bits = w < P.nwords ? P.freebits[w] : 0u;
      int n = 0;
      int rank = acc + wg_exclusive_scan(__popc(bits), &n);
      if (rank < total && bits) {
        uint32_t taken = 0;
        while (bits && rank < total) {
          const int bit = __ffs(bits) - 1;
          bits &= bits - 1;
          taken |= 1u << bit;
          P.alloc_list[rank++] = w * 32 + bit;
        }
        P.freebits[w] &= ~taken;
      }
      acc += n;
    }
    __syncthreads();  // alloc_list is complete
  }
  int off = base;
  for (int i = r0; i < r1; ++i) {
    const int tr = req_trace[i];
    const int L = P.seq_len[tr];
    const int nt = uniform >= 0 ? uniform : req_ntok[i];
    const int j0 = cdiv16(L), j1 = cdiv16(L + nt);
    int32_t* row = P.table + (size_t)tr * P.max_blocks;
    for (int j = j0; j < j1; ++j) {
      const int b = P.alloc_list[off++];
      row[j] = b;
      P.refcount[b] = 1;
      if (P.kv_scale)
        for (int l = 0; l < P.num_layers; ++l) {
          float* sc = P.kv_scale + (size_t)l * 2 * P.num_blocks;
          sc[2 * b] = new_scale;
          sc[2 * b + 1] = new_scale;
        }
    }
    P.seq_len[tr] = L + nt;
    if (generated) P.gen[tr] += nt;
  }
}

// Copy one token's K and V (all KV heads) into its cache slot: K in 16-byte
// d-chunks at token row k_phys(row), V element-wise into the transposed tile.
__device__ inline void copy_token(const DevPool& P, int blk, int row, const uint8_t* ksrc,
                                  const uint8_t* vsrc) {
  const int es = P.esize;
  const int row_bytes = kHeadDim * es;  // one head, one token
  const int kchunks = row_bytes / 16;
  const size_t tile = (size_t)kBlock * row_bytes;
  const size_t blk0 = (size_t)blk * P.Hkv * tile;
  const int pr = k_phys(row);
  for (int c = threadIdx.x; c < P.Hkv * kchunks; c += blockDim.x) {
    const int head = c / kchunks, cc = c % kchunks;
    const size_t dst = blk0 + head * tile + ((size_t)cc * kBlock + pr) * 16;
    *reinterpret_cast<uint4*>(P.k_cache + dst) = *reinterpret_cast<const uint4*>(ksrc + (size_t)c * 16);
  }
  for (int e = threadIdx.x; e < P.Hkv * kHeadDim; e += blockDim.x) {
    const int head = e / kHeadDim, d = e % kHeadDim;
    const size_t dst = blk0 + head * tile + ((size_t)d * kBlock + row) * es;
    if (es == 2)
      *reinterpret_cast<uint16_t*>(P.v_cache + dst) = reinterpret_cast<const uint16_t*>(vsrc)[e];
    else
      P.v_cache[dst] = vsrc[e];
  }
}

// One workgroup per (token, layer); k, v: [layers][n][Hkv][128], started
// scales: [layers][started][2].
__global__ void write_kernel(DevPool P0, int32_t trace, int32_t pos0, int32_t n, const uint8_t* k,
                             const uint8_t* v, const float* started_scales, int32_t started) {
  const int i = blockIdx.x, l = blockIdx.y;
  const DevPool P = P0.layer(l);
  const int pos = pos0 + i;
  const int blk = P.table[(size_t)trace * P.max_blocks + pos / kBlock];
  if ((unsigned)blk >= (unsigned)P.num_blocks) {
    if (threadIdx.x == 0) atomicOr(P.err, kErrBadBlock);
    return;
  }
  const size_t tok_bytes = (size_t)P.Hkv * kHeadDim * P.esize;
  const size_t src = ((size_t)l * n + i) * tok_bytes;
  copy_token(P, blk, pos % kBlock, k + src, v + src);
  if (started_scales && threadIdx.x == 0 && pos % kBlock == 0) {
    const int first = (pos0 + kBlock - 1) / kBlock * kBlock;
    const int k2 = l * started + (pos - first) / kBlock;
    P.kv_scale[2 * blk] = started_scales[2 * k2];
    P.kv_scale[2 * blk + 1] = started_scales[2 * k2 + 1];
  }
}

// Prune (or evict): one workgroup per trace.  A row may be empty (a ghost
// leaving the tree view).
__global__ void free_kernel(DevPool P, const int32_t* ids, int32_t mode) {
  const int tr = ids[blockIdx.x];
  const int nb = cdiv16(P.seq_len[tr]);
  int32_t* row = P.table + (size_t)tr * P.max_blocks;
  for (int j = threadIdx.x; j < nb; j += blockDim.x) {
    const int b = row[j];
    row[j] = -1;
    if (b < 0 || b >= P.num_blocks) {
      atomicOr(P.err, kErrBadBlock);
      continue;
    }
    const int old = atomicSub(&P.refcount[b], 1);
    if (old == 1) atomicOr(&P.freebits[b >> 5], 1u << (b & 31));
    if (old < 1) atomicOr(P.err, kErrRefUnderflow);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    P.seq_len[tr] = 0;
    P.gen[tr] = 0;
    if (mode == kFreeEvict) {
      P.ghost[tr] = 1;  // keeps its score and its place in the tree view
    } else {
      P.ghost[tr] = 0;
      P.sbar[tr] = 0.f;
      P.nscore[tr] = 0;
    }
  }
}

// Branch, part 1: the child row takes the parent's full blocks (refcount + 1)
// and the child length is set to the full-block prefix; the partial tail is
// requested from the allocator (req_ntok = parent length mod 16).
__global__ void fork_share_kernel(DevPool P, const int32_t* pairs, int32_t* req_trace,
                                  int32_t* req_ntok) {
  const int child = pairs[2 * blockIdx.x], parent = pairs[2 * blockIdx.x + 1];
  const int L = P.seq_len[parent];
  const int full = L / kBlock;
  const int32_t* prow = P.table + (size_t)parent * P.max_blocks;
  int32_t* crow = P.table + (size_t)child * P.max_blocks;
  for (int j = threadIdx.x; j < full; j += blockDim.x) {
    const int b = prow[j];
    crow[j] = b;
    if ((unsigned)b < (unsigned)P.num_blocks)
      atomicAdd(&P.refcount[b], 1);
    else
      atomicOr(P.err, kErrBadBlock);
  }
  if (threadIdx.x == 0) {
    P.seq_len[child] = full * kBlock;
    req_trace[blockIdx.x] = child;
    req_ntok[blockIdx.x] = L % kBlock;
    // the child's trace is the parent's prefix: it inherits the parent's
    // thought scores, and has generated nothing of its own yet
    P.sbar[child] = P.sbar[parent];
    P.nscore[child] = P.nscore[parent];
    P.gen[child] = 0;
    P.ghost[child] = 0;
  }
}

// Branch, part 2: copy the partial tail block (every KV head; whole tiles,
// the slots past the tail are never read unmasked) and its fp8 scales into
// the child's new block; one workgroup per (pair, layer).
__global__ void fork_tail_kernel(DevPool P0, const int32_t* pairs) {
  const DevPool P = P0.layer(blockIdx.y);
  const int child = pairs[2 * blockIdx.x], parent = pairs[2 * blockIdx.x + 1];
  const int L = P.seq_len[parent];
  if (L % kBlock == 0) return;
  const int j = L / kBlock;
  const int src = P.table[(size_t)parent * P.max_blocks + j];
  const int dst = P.table[(size_t)child * P.max_blocks + j];
  if ((unsigned)src >= (unsigned)P.num_blocks || (unsigned)dst >= (unsigned)P.num_blocks) {
    if (threadIdx.x == 0) atomicOr(P.err, kErrBadBlock);
    return;
  }
  const size_t blk_bytes = (size_t)P.Hkv * kBlock * kHeadDim * P.esize;
  const uint4* ks = reinterpret_cast<const uint4*>(P.k_cache + (size_t)src * blk_bytes);
  const uint4* vs = reinterpret_cast<const uint4*>(P.v_cache + (size_t)src * blk_bytes);
  uint4* kd = reinterpret_cast<uint4*>(P.k_cache + (size_t)dst * blk_bytes);
  uint4* vd = reinterpret_cast<uint4*>(P.v_cache + (size_t)dst * blk_bytes);
  for (size_t c = threadIdx.x; c < blk_bytes / 16; c += blockDim.x) {
    kd[c] = ks[c];
    vd[c] = vs[c];
  }
  if (P.kv_scale && threadIdx.x == 0) {
    P.kv_scale[2 * dst] = P.kv_scale[2 * src];
    P.kv_scale[2 * dst + 1] = P.kv_scale[2 * src + 1];
  }
}

}  // namespace

hipError_t launch_pool_init(const DevPool& P, hipStream_t s) {
  hipLaunchKernelGGL(pool_init_kernel, dim3(1024), dim3(256), 0, s, P);
  return hipGetLastError();
}

hipError_t launch_alloc(const DevPool& P, const int32_t* req_trace, const int32_t* req_ntok,
                        int32_t uniform_ntok, int32_t m, float new_scale, bool generated, hipStream_t s) {
  if (m <= 0) return hipSuccess;
  hipLaunchKernelGGL(alloc_kernel, dim3(1), dim3(kAllocThreads), 0, s, P, req_trace, req_ntok,
                     uniform_ntok, m, new_scale, (int32_t)generated);
  return hipGetLastError();
}

hipError_t launch_write(const DevPool& P, int32_t trace, int32_t pos0, int32_t n, const void* k,
                        const void* v, const float* started_scales, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int first = (pos0 + kBlock - 1) / kBlock, last = (pos0 + n - 1) / kBlock;
  hipLaunchKernelGGL(write_kernel, dim3(n, P.num_layers), dim3(128), 0, s, P, trace, pos0, n,
                     static_cast<const uint8_t*>(k), static_cast<const uint8_t*>(v), started_scales,
                     last >= first ? last - first + 1 : 0);
  return hipGetLastError();
}

hipError_t launch_free(const DevPool& P, const int32_t* ids, int32_t n, int32_t mode, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(free_kernel, dim3(n), dim3(256), 0, s, P, ids, mode);
  return hipGetLastError();
}

hipError_t launch_fork(const DevPool& P, const int32_t* pairs, int32_t n, int32_t* req_trace,
                       int32_t* req_ntok, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fork_share_kernel, dim3(n), dim3(256), 0, s, P, pairs, req_trace, req_ntok);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = launch_alloc(P, req_trace, req_ntok, -1, n, 1.0f, false, s);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(fork_tail_kernel, dim3(n, P.num_layers), dim3(256), 0, s, P, pairs);
  return hipGetLastError();
}

}  // namespace gambit
