// The 2-layer MLP scorer (the paper's main-evaluation probe on the
// thought-boundary hidden state, Sec. 4.1 and Sec. 5.1):
//     f(h) = sigmoid(w2 . act(W1 h + b1) + b2)
// kernels and host entry points.
//
// Three launches:
//   1. mlp_gemm_kernel: W1 h on the bf16 matrix cores in 128 x 128 tiles
//      (hidden states x hidden units), the k range split S ways so that the
//      whole chip has work (512 x 4096 -> 1024: 32 tiles x 8 splits, one
//      eight-wave workgroup per CU).  With S > 1 each workgroup writes its
//      fp32 pre-activation partial sums; with S = 1 it applies bias,
//      activation and w2 itself and writes one partial logit per hidden state
//      and tile.
//   2. mlp_logit_kernel: per hidden state, the S partial sums in split order,
//      bias, activation, times w2, summed over the units (or the tiles'
//      partial logits in tile order), plus b2, sigmoid.
//   3. mlp_rank_kernel (keep > 0): every key's rank by counting the keys
//      ahead of it (score descending, id ascending), many workgroups at
//      once; ranks below `keep` write their id.
//
// Two entry points share those kernels: gambit_mlp_score takes its scratch
// from a caller workspace; gambit_mlp_score_static takes it from a buffer
// the library holds in device memory for the life of the process, so that
// callers that cannot allocate device memory at all (code under HIP graph
// capture, serving loops that forbid allocation) can score.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>

#include "../../include/gambit.h"
#include "kernels.h"
#include "seq_kernels.h"
#include "lds_dma.h"

namespace gambit {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kGT = 128;                 // hidden states per tile
constexpr int kGU = 128;                 // hidden units per tile
constexpr int kGK = 64;                  // k per LDS slab (128 B of each row)
constexpr int kGStages = 4;              // slabs in the LDS ring
constexpr int kGSlabA = kGT * kGK * 2;   // 16 KiB: one operand's slab
constexpr int kGSlab = 2 * kGSlabA;
constexpr int kGWaves = 8;               // two per SIMD
constexpr int kGThreads = 64 * kGWaves;
constexpr int kGLoads = kGT / 8 / kGWaves;       // 8-row loads per operand, wave and slab
constexpr int kGUB = kGU / 16 / (kGWaves / 2);   // 16-unit blocks per wave
static_assert(kGT == kGU, "both operands' slabs have the same shape");

__device__ inline float mlp_act(float x, int act) {
  return act == 0 ? fmaxf(x, 0.f) : 0.5f * x * (1.f + erff(x * 0.70710678118654752f));
}

__device__ inline uint32_t orderable(float f) {
  const uint32_t u = __builtin_bit_cast(uint32_t, f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// s_waitcnt lgkmcnt(0) (vmcnt, expcnt at their maxima): this wave's LDS
// reads are complete, so the stage they read may be refilled after the
// next barrier.
__device__ inline void wait_lds_reads() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// One workgroup, eight waves: tile (tt, tu) of split s, i.e. hidden states
// t0 .. t0 + 127 x units u0 .. u0 + 127 over k in [k0, k0 + 64 nslab).
//
// Operands go from global memory straight into an LDS ring of four 64-deep
// slabs (direct loads, three slabs in flight); wave w fills rows 16 w ..
// 16 w + 15 of both operands, eight rows of 128 B per load.  Row r's 16-byte
// chunk c sits at chunk position c ^ ((r >> 1) & 7) of its 128-byte row, so
// the sixteen rows that one matrix-core operand read touches (a 16 x 32
// block, 16 B per lane) fall on sixteen different 16-byte bank groups.
//
// Wave w computes hidden states 64 (w & 1) .. + 63 x units 32 (w >> 1) .. +
// 31: 4 x 2 blocks of v_mfma_f32_16x16x32_bf16, where lane (q, i) supplies
// row i's k values 8q .. 8q + 7 of both operands and holds, in block (a, b),
// hidden states 16 a + 4 q + e (e = 0..3) of unit 16 b + i.
__global__ __launch_bounds__(kGThreads) __attribute__((amdgpu_waves_per_eu(2, 2))) void mlp_gemm_kernel(MlpLaunch L) {
  __shared__ __attribute__((aligned(1024))) uint8_t ring[kGStages * kGSlab];
  __shared__ float red[kGWaves / 2][kGT];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  // Work items in (split, unit tile, state tile) order; when the grid is a
  // multiple of 8, consecutive items go to the same XCD (workgroup b runs on
  // XCD b % 8), so each XCD's L2 holds few operand rows (one split's k range
  // when there are 8 splits).
  const int G = gridDim.x;
  const int w = (G & 7) ? blockIdx.x : (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
  const int tiles = L.tiles_t * L.tiles_u;
  const int s = w / tiles, tile = w - s * tiles;
  const int tu = tile / L.tiles_t, tt = tile - tu * L.tiles_t;
  const int t0 = tt * kGT, u0 = tu * kGU;
  const int C = L.dim / 128;  // 128-wide k chunks, split as evenly as possible
  const int c0 = s * C / L.splits, c1 = (s + 1) * C / L.splits;
  const int k0 = c0 * 128, nslab = (c1 - c0) * 2;

  // this lane's load sources: rows 16 w + 8 d + lane / 8, chunk position
  // lane % 8 (rows past the end re-read the last row; never stored)
  const uint16_t* asrc[kGLoads];
  const uint16_t* bsrc[kGLoads];
#pragma unroll
  for (int d = 0; d < kGLoads; ++d) {
    const int r = 8 * kGLoads * wave + 8 * d + (lane >> 3);
    const int c = (lane & 7) ^ ((r >> 1) & 7);
    asrc[d] = L.h + (size_t)min(t0 + r, L.n - 1) * L.dim + k0 + 8 * c;
    bsrc[d] = L.w1 + (size_t)min(u0 + r, L.hidden - 1) * L.dim + k0 + 8 * c;
  }
  // Every workgroup takes its slabs in k order, so equal hidden states in
  // different tiles get bit-equal sums (and so equal scores, ranked by id).
  auto issue = [&](int sl) {
    uint8_t* st = ring + (sl % kGStages) * kGSlab;
    const int ko = sl * kGK;
#pragma unroll
    for (int d = 0; d < kGLoads; ++d) dma16(asrc[d] + ko, st + (8 * kGLoads * wave + 8 * d) * 128);
#pragma unroll
    for (int d = 0; d < kGLoads; ++d) dma16(bsrc[d] + ko, st + kGSlabA + (8 * kGLoads * wave + 8 * d) * 128);
  };

  // operand read offsets (bytes within a stage) for the two 32-deep halves
  const int i = lane & 15, q = lane >> 4, swz = (i >> 1) & 7;
  const int wt = wave & 1, wu = wave >> 1;
  const int offa = (64 * wt + i) * 128, offb = kGSlabA + (16 * kGUB * wu + i) * 128;
  const int pos0 = (q ^ swz) * 16, pos1 = ((q | 4) ^ swz) * 16;

  f32x4 acc[4][kGUB];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < kGUB; ++b) acc[a][b] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Per slab: wait for it (this wave's loads of the slabs after it stay in
  // flight), barrier, refill the stage of the slab before it (every wave has
  // read it), read both halves' operands, then their products.
  for (int sl = 0; sl < kGStages - 1 && sl < nslab; ++sl) issue(sl);
  for (int sl = 0; sl < nslab; ++sl) {
    switch (min(kGStages - 2, nslab - 1 - sl)) {  // slabs issued after this one
      case 2: wait_vmcnt<4 * kGLoads>(); break;
      case 1: wait_vmcnt<2 * kGLoads>(); break;
      default: wait_vmcnt<0>(); break;
    }
    wait_lds_reads();
    barrier_no_fence();  // slab sl is in LDS; every wave is done with slab sl - 1
    if (sl + kGStages - 1 < nslab) issue(sl + kGStages - 1);
    const uint8_t* st = ring + (sl % kGStages) * kGSlab;
    bf16x8 A0[4], B0[kGUB], A1[4], B1[kGUB];
#pragma unroll
    for (int a = 0; a < 4; ++a) A0[a] = *reinterpret_cast<const bf16x8*>(st + offa + a * 2048 + pos0);
#pragma unroll
    for (int b = 0; b < kGUB; ++b) B0[b] = *reinterpret_cast<const bf16x8*>(st + offb + b * 2048 + pos0);
#pragma unroll
    for (int a = 0; a < 4; ++a) A1[a] = *reinterpret_cast<const bf16x8*>(st + offa + a * 2048 + pos1);
#pragma unroll
    for (int b = 0; b < kGUB; ++b) B1[b] = *reinterpret_cast<const bf16x8*>(st + offb + b * 2048 + pos1);
    __builtin_amdgcn_sched_barrier(0);  // all sixteen reads are issued before the first product
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < kGUB; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A0[a], B0[b], acc[a][b], 0, 0, 0);
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < kGUB; ++b) acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A1[a], B1[b], acc[a][b], 0, 0, 0);
  }

  if (L.splits > 1 || !L.b1) {  // b1 == NULL: partial sums only (bf16_gemm_partials)
    // pre-activation partial sums of split s, through LDS so that each row
    // of the tile leaves as 512 contiguous bytes (rows padded by 16 B: the
    // four row groups of a write fall on different banks); non-temporal
    // stores, so the 16 MB of partial sums of a 512 x 1024 call stream out
    // instead of waiting dirty in L2 for the end of the launch
    constexpr int kRow = kGU * 4 + 16;
    static_assert(kGT * kRow <= kGStages * kGSlab, "epilogue staging fits the ring");
    wait_lds_reads();
    __syncthreads();  // every wave is done with the ring
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
      for (int b = 0; b < kGUB; ++b)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          *reinterpret_cast<float*>(ring + (64 * wt + 16 * a + 4 * q + e) * kRow + (16 * kGUB * wu + 16 * b + i) * 4) =
              acc[a][b][e];
    __syncthreads();
    float* out = L.parts + (size_t)s * L.n * L.hidden;
    for (int x = threadIdx.x; x < kGT * (kGU / 4); x += kGThreads) {
      const int r = x / (kGU / 4), c = 4 * (x % (kGU / 4));
      if (t0 + r < L.n && u0 + c < L.hidden)
        __builtin_nontemporal_store(*reinterpret_cast<const f32x4*>(ring + r * kRow + c * 4),
                                    reinterpret_cast<f32x4*>(out + (size_t)(t0 + r) * L.hidden + u0 + c));
    }
    return;
  }
  // S = 1: bias, activation, w2, summed over this wave's units (blocks b in
  // order, then the 16 lanes of a row group), then the unit groups in order
  float w2v[kGUB], b1v[kGUB];
#pragma unroll
  for (int b = 0; b < kGUB; ++b) {
    const int u = u0 + 16 * kGUB * wu + 16 * b + i;
    w2v[b] = u < L.hidden ? L.w2[u] : 0.f;
    b1v[b] = u < L.hidden ? L.b1[u] : 0.f;
  }
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      float v = 0.f;
#pragma unroll
      for (int b = 0; b < kGUB; ++b) v += w2v[b] * mlp_act(acc[a][b][e] + b1v[b], L.act);
#pragma unroll
      for (int off = 8; off > 0; off >>= 1) v += __shfl_xor(v, off);
      if (i == 0) red[wu][64 * wt + 16 * a + 4 * q + e] = v;
    }
  __syncthreads();
  if (threadIdx.x < kGT && t0 + (int)threadIdx.x < L.n) {
    float z = red[0][threadIdx.x];
#pragma unroll
    for (int g = 1; g < kGWaves / 2; ++g) z += red[g][threadIdx.x];
    L.parts[(size_t)tu * L.n + t0 + threadIdx.x] = z;
  }
}

// One workgroup per hidden state t.  S > 1: thread i takes units 4 i +
// 1024 m; the S partial sums of a unit are loaded eight splits at a time
// (indices clamped, so every load is in bounds and all eight are in flight
// together) and added in split order, then bias, activation and w2; the
// threads' sums are combined by a fixed shuffle tree per wave and the four
// waves in order.  S = 1: thread 0 adds the tiles' partial logits in tile
// order.
__global__ __launch_bounds__(256) void mlp_logit_kernel(MlpLaunch L) {
  __shared__ float wsum[4];
  const int t = blockIdx.x, lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  float z = 0.f;
  if (L.splits > 1) {
    const size_t split = (size_t)L.n * L.hidden;
    const float* p = L.parts + (size_t)t * L.hidden;
    for (int u = 4 * threadIdx.x; u < L.hidden; u += 1024) {
      float4 y = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int s0 = 0; s0 < L.splits; s0 += 8) {
        float4 v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = *reinterpret_cast<const float4*>(p + min(s0 + e, L.splits - 1) * split + u);
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (s0 + e < L.splits) {  // uniform; the loads above are already in flight
            y.x += v[e].x;
            y.y += v[e].y;
            y.z += v[e].z;
            y.w += v[e].w;
          }
      }
      const float4 bb = *reinterpret_cast<const float4*>(L.b1 + u);
      const float4 ww = *reinterpret_cast<const float4*>(L.w2 + u);
      z += ww.x * mlp_act(y.x + bb.x, L.act);
      z += ww.y * mlp_act(y.y + bb.y, L.act);
      z += ww.z * mlp_act(y.z + bb.z, L.act);
      z += ww.w * mlp_act(y.w + bb.w, L.act);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) z += __shfl_xor(z, off);
    if (lane == 0) wsum[wave] = z;
    __syncthreads();
    z = ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3];
  } else if (threadIdx.x == 0) {
    for (int k = 0; k < L.tiles_u; ++k) z += L.parts[(size_t)k * L.n + t];
  }
  if (threadIdx.x == 0) L.scores_out[t] = 1.f / (1.f + expf(-(L.b2 + z)));
}

// Ranks by counting: key k's rank is the number of keys ahead of it (higher
// score; equal score and lower id; equal both and lower index - a total
// order, so the ranks are a permutation).  A workgroup ranks 16 keys, each
// with 16 threads that split the others; all keys sit in LDS as (orderable
// score, id) pairs, padded with keys that are never ahead.  A part holds
// `per` keys, a multiple of 4 with per / 4 odd, so that the four parts a
// wave reads at once (16 bytes each) fall on different LDS banks.
constexpr int kRankKeys = 16;
constexpr int kRankSlots = kMaxRank + 64;
__host__ __device__ constexpr int rank_part(int n) {
  const int p = ((n + 15) / 16 + 3) / 4;
  return 4 * (p | 1);
}
static_assert(16 * rank_part(kMaxRank) <= kRankSlots, "rank LDS");
__global__ __launch_bounds__(256) void mlp_rank_kernel(int n, const float* scores, const int32_t* ids, int keep,
                                                       int32_t* keep_out) {
  __shared__ __attribute__((aligned(16))) uint2 kv[kRankSlots];
  __shared__ int cnt[4][kRankKeys];
  const int per = rank_part(n);
  for (int j = threadIdx.x; j < 16 * per; j += 256)
    kv[j] = j < n ? make_uint2(orderable(scores[j]), (uint32_t)ids[j]) : make_uint2(0u, ~0u);
  __syncthreads();
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int slot = lane & 15, part = 4 * wave + (lane >> 4);
  const int k = min(blockIdx.x * kRankKeys + slot, n - 1);
  const uint32_t sk = kv[k].x, ik = kv[k].y;
  const int j0 = part * per;
  int c = 0;
  for (int j = j0; j < j0 + per; j += 4) {
    const uint4 x = *reinterpret_cast<const uint4*>(&kv[j]);
    const uint4 y = *reinterpret_cast<const uint4*>(&kv[j + 2]);
    const uint32_t sj[4] = {x.x, x.z, y.x, y.z}, ij[4] = {x.y, x.w, y.y, y.w};
#pragma unroll
    for (int e = 0; e < 4; ++e)
      c += (sj[e] > sk) | ((sj[e] == sk) & ((ij[e] < ik) | ((ij[e] == ik) & (j + e < k))));
  }
  c += __shfl_xor(c, 16);
  c += __shfl_xor(c, 32);
  if (lane < kRankKeys) cnt[wave][lane] = c;
  __syncthreads();
  if (threadIdx.x < kRankKeys && blockIdx.x * kRankKeys + (int)threadIdx.x < n) {
    const int r = cnt[0][threadIdx.x] + cnt[1][threadIdx.x] + cnt[2][threadIdx.x] + cnt[3][threadIdx.x];
    if (r < keep) keep_out[r] = (int32_t)ik;
  }
}

// The static entry point's scratch.  In host code this name is only a
// stand-in for the symbol: its device address (one per device, each device
// holding its own copy) comes from hipGetSymbolAddress and is what the
// kernels receive.
constexpr size_t kStaticScratchBytes = GAMBIT_MLP_STATIC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch`, looked up once per device (with
// that device current) and kept.
hipError_t device_scratch(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

gambit_status check_mlp(int32_t n, const void* h, const gambit_mlp* mlp, const float* scores_out,
                        const int32_t* trace_ids, int32_t keep, const int32_t* keep_out) {
  if (!mlp || !h || !scores_out || n <= 0 || n > kMaxRank) return GAMBIT_ERR_INVALID;
  if (mlp->dim <= 0 || mlp->dim % 128 || mlp->hidden <= 0 || mlp->hidden % 64 ||
      (mlp->activation != GAMBIT_ACT_RELU && mlp->activation != GAMBIT_ACT_GELU) || !mlp->w1 || !mlp->b1 || !mlp->w2)
    return GAMBIT_ERR_INVALID;
  if (keep < 0 || keep > n || (keep > 0 && (!trace_ids || !keep_out))) return GAMBIT_ERR_INVALID;
  return GAMBIT_OK;
}

gambit_status launch(int32_t n, const void* h, const gambit_mlp* mlp, float* scores_out, const int32_t* trace_ids,
                     int32_t keep, int32_t* keep_out, float* parts, void* stream) {
  MlpLaunch L{};
  L.n = n;
  L.dim = mlp->dim;
  L.hidden = mlp->hidden;
  L.act = mlp->activation;
  L.tiles_t = (n + kGT - 1) / kGT;
  L.tiles_u = (mlp->hidden + kGU - 1) / kGU;
  L.splits = std::min(mlp_splits(n, mlp->hidden), mlp->dim / 128);
  L.h = static_cast<const uint16_t*>(h);
  L.w1 = static_cast<const uint16_t*>(mlp->w1);
  L.b1 = mlp->b1;
  L.w2 = mlp->w2;
  L.b2 = mlp->b2;
  L.parts = parts;
  L.scores_out = scores_out;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(mlp_gemm_kernel, dim3(L.tiles_t * L.tiles_u * L.splits), dim3(kGThreads), 0, s, L);
  if (hipGetLastError() != hipSuccess) return GAMBIT_ERR_DEVICE;
  hipLaunchKernelGGL(mlp_logit_kernel, dim3(n), dim3(256), 0, s, L);
  if (hipGetLastError() != hipSuccess) return GAMBIT_ERR_DEVICE;
  if (keep > 0) {
    hipLaunchKernelGGL(mlp_rank_kernel, dim3((n + kRankKeys - 1) / kRankKeys), dim3(256), 0, s, n,
                       (const float*)scores_out, trace_ids, keep, keep_out);
    if (hipGetLastError() != hipSuccess) return GAMBIT_ERR_DEVICE;
  }
  return GAMBIT_OK;
}

}  // namespace

// The split-k GEMM alone: parts[s][t][u] for every split, with no bias,
// activation or w2 (L.b1 stays NULL), also when there is one split.
hipError_t bf16_gemm_partials(const uint16_t* h, const uint16_t* w, int32_t n, int32_t dim, int32_t units,
                              int32_t splits, float* parts, hipStream_t s) {
  if (!h || !w || !parts || n <= 0 || dim <= 0 || dim % 128 || units <= 0 || units % 4 || splits < 1 ||
      splits > dim / 128)
    return hipErrorInvalidValue;
  MlpLaunch L{};
  L.n = n;
  L.dim = dim;
  L.hidden = units;
  L.tiles_t = (n + kGT - 1) / kGT;
  L.tiles_u = (units + kGU - 1) / kGU;
  L.splits = splits;
  L.h = h;
  L.w1 = w;
  L.parts = parts;
  hipLaunchKernelGGL(mlp_gemm_kernel, dim3(L.tiles_t * L.tiles_u * L.splits), dim3(kGThreads), 0, s, L);
  return hipGetLastError();
}

}  // namespace gambit

extern "C" {

size_t gambit_mlp_workspace_size(int32_t n, int32_t hidden) {
  if (n <= 0 || hidden <= 0 || hidden % 64) return 0;  // the documented unit multiple
  return gambit::mlp_workspace_bytes(n, hidden);
}

gambit_status gambit_mlp_score(int32_t n, const void* h, const gambit_mlp* mlp, float* scores_out,
                               const int32_t* trace_ids, int32_t keep, int32_t* keep_out, void* workspace,
                               size_t workspace_bytes, void* stream) {
  const gambit_status st = gambit::check_mlp(n, h, mlp, scores_out, trace_ids, keep, keep_out);
  if (st != GAMBIT_OK) return st;
  if (!workspace || workspace_bytes < gambit_mlp_workspace_size(n, mlp->hidden)) return GAMBIT_ERR_WORKSPACE;
  return gambit::launch(n, h, mlp, scores_out, trace_ids, keep, keep_out, static_cast<float*>(workspace), stream);
}

gambit_status gambit_mlp_score_static(int32_t n, const void* h, const gambit_mlp* mlp, float* scores_out,
                                      const int32_t* trace_ids, int32_t keep, int32_t* keep_out, void* stream) {
  const gambit_status st = gambit::check_mlp(n, h, mlp, scores_out, trace_ids, keep, keep_out);
  if (st != GAMBIT_OK) return st;
  if (gambit_mlp_workspace_size(n, mlp->hidden) > gambit::kStaticScratchBytes) return GAMBIT_ERR_WORKSPACE;
  void* parts = nullptr;
  if (gambit::device_scratch(&parts) != hipSuccess) return GAMBIT_ERR_DEVICE;
  return gambit::launch(n, h, mlp, scores_out, trace_ids, keep, keep_out, static_cast<float*>(parts), stream);
}

}  // extern "C"
