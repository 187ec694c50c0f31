// The history-aware sequence scorer (App. A.1, Eqs. 4-6), one new step per
// trace per thought boundary against cached keys and values of the trace's
// earlier steps.  fp32 weights, activations and caches; the step states
// arrive in bf16, and the input projection runs on the bf16 matrix cores
// with fp32 sums, its weights (scaled by the input LayerNorm's gain) split
// exactly into three bf16 planes when the scorer is created.
//
// Per boundary, for the n listed traces (rows):
//   x  = GELU(LN_in(h) W_in^T)             bf16_gemm_partials (h against the
//                                           planes, K split; mlp_scorer.hip);
//                                           reduce_in_kernel (the splits and
//                                           planes added, LN_in applied)
//   per layer: u = LN1(x); qkv = u Wqkv^T; o = attention step (RoPE, append
//   the step's key and value, attend over the trace's steps 0..t);
//   x += o Wo^T; u = LN2(x); a = u W13^T; g = SiLU(a1) * a3; x += g W2^T
//   y  = sigmoid(w_out . LN_out(x)), and the trace's step count advances.
// A K-split projection's partial sums are added, its epilogue applied and the
// LayerNorm that follows it (LN1, LN2, or LN_out and the head) taken in one
// launch (reduce_ln_kernel, reduce_in_kernel): 16 launches per boundary with
// two layers.
#include <hip/hip_runtime.h>

#include "seq_kernels.h"

namespace gambit {
namespace {

__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ inline float load_elem(const void* p, size_t i, bool bf16) {
  if (bf16) return __uint_as_float((uint32_t)reinterpret_cast<const uint16_t*>(p)[i] << 16);
  return reinterpret_cast<const float*>(p)[i];
}

__device__ inline float gelu_erf(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }

typedef float f32x4 __attribute__((ext_vector_type(4)));

// A 16-byte load with the non-temporal hint (the attention step's cached
// keys: each is read once per boundary, and the history of all traces is
// far larger than L2).  Measured at 512 traces, history 128: 23.5-23.9 vs
// 24.7-26.7 us per attention step; the same hint on the values as well
// made it slower (26.5-27.6 us).
__device__ inline float4 ld_stream4(const float* p) {
  const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}

// C[M][N] = A[M][K] . W[N][K]^T over K range [z * ks, (z + 1) * ks) of split
// z = blockIdx.z, on the fp32 matrix cores (v_mfma_f32_16x16x4f32).  TM x 64
// tiles (TM = 64 or 32); the K range is taken in chunks of 128 that are
// staged whole in LDS (rows padded to 132 floats, so the 16 rows of an
// operand read fall on 16 different 16-byte bank groups), the next chunk's
// global loads in flight in registers while the current one is multiplied.
// Each of the 4 waves computes a (TM / 2) x 32 quarter as 16 x 16 products.
// A lane reads 4 consecutive k of its row (one 16-byte read) and feeds them
// to 4 successive products: lane (q, i) contributes A[i][4q + kk] and
// W[i][4q + kk] to product kk, the same k for both operands, so each product
// sums over k = 4q + kk, q = 0..3; result element (4 (l / 16) + r, l % 16)
// sits in lane l, register r.
// part != NULL: the raw sums of split z go
// to part[z][M][N] for reduce_ln_kernel; else the epilogue is applied and C
// written (one split).
// kEpiSwiGLU: W holds W_1 and W_3 rows interleaved in groups of 16, so a
// wave's two column blocks are W_1 and W_3 of the same 16 outputs, and
// C[m][16 c + i] = SiLU(a1) * a3 with row stride N / 2.
constexpr int kKC = 128;       // k per staged chunk
constexpr int kKP = kKC + 4;   // padded LDS row, floats
template <int TM>
__global__ __launch_bounds__(256) void gemm_kernel(const float* A, const float* W, float* C, int M, int N, int K,
                                                   int ks, int epi, float* part) {
  constexpr int MB = TM / 32;                    // 16-row blocks per wave
  constexpr int AV = TM * (kKC / 4) / 256;       // float4 groups of A per thread and chunk
  constexpr int WV = 64 * (kKC / 4) / 256;       // of W
  __shared__ __attribute__((aligned(16))) float As[TM * kKP];
  __shared__ __attribute__((aligned(16))) float Ws[64 * kKP];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int m0 = blockIdx.y * TM, n0 = blockIdx.x * 64;
  const int k0 = blockIdx.z * ks;
  const int li = lane & 15, lq = lane >> 4;
  const int wm = (wave >> 1) * (TM / 2), wn = (wave & 1) * 32;
  // loader: group g = tid + 256 v is row g / 32, k offset 4 (g % 32); the k
  // offset is the same for every v
  const int lk = 4 * (tid & 31), lr = tid >> 5;
  float4 ar[AV], wr[WV];
  // chunk [kb, kb + kn): groups past kn (a shorter last chunk) stay zero and
  // read nothing
  auto fetch = [&](int kb, int kn) {
    const bool kin = lk < kn;
#pragma unroll
    for (int v = 0; v < AV; ++v) {
      const int m = m0 + lr + 8 * v;
      ar[v] = (m < M && kin) ? *reinterpret_cast<const float4*>(A + (size_t)m * K + kb + lk)
                             : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int v = 0; v < WV; ++v)
      wr[v] = kin ? *reinterpret_cast<const float4*>(W + (size_t)(n0 + lr + 8 * v) * K + kb + lk)
                  : make_float4(0.f, 0.f, 0.f, 0.f);
  };
  f32x4 acc[MB][2];
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  fetch(k0, min(kKC, ks));
  for (int kb = k0; kb < k0 + ks; kb += kKC) {
    const int kn = min(kKC, k0 + ks - kb);  // a multiple of 16
    __syncthreads();  // the previous chunk's reads are done
#pragma unroll
    for (int v = 0; v < AV; ++v) *reinterpret_cast<float4*>(&As[(lr + 8 * v) * kKP + lk]) = ar[v];
#pragma unroll
    for (int v = 0; v < WV; ++v) *reinterpret_cast<float4*>(&Ws[(lr + 8 * v) * kKP + lk]) = wr[v];
    __syncthreads();
    if (kb + kKC < k0 + ks) fetch(kb + kKC, min(kKC, k0 + ks - kb - kKC));
    for (int kc = 0; kc < kn; kc += 16) {
      float4 a[MB], b[2];
#pragma unroll
      for (int i = 0; i < MB; ++i) a[i] = *reinterpret_cast<const float4*>(&As[(wm + 16 * i + li) * kKP + kc + 4 * lq]);
#pragma unroll
      for (int j = 0; j < 2; ++j) b[j] = *reinterpret_cast<const float4*>(&Ws[(wn + 16 * j + li) * kKP + kc + 4 * lq]);
#pragma unroll
      for (int i = 0; i < MB; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].x, b[j].x, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].y, b[j].y, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].z, b[j].z, acc[i][j], 0, 0, 0);
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i].w, b[j].w, acc[i][j], 0, 0, 0);
        }
    }
  }
  if (epi == kEpiSwiGLU) {  // one split
    const int f = N / 2, c = (n0 + wn) / 32;
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm + 16 * i + 4 * lq + r;
        if (m >= M) continue;
        const float a = acc[i][0][r], b = acc[i][1][r];
        C[(size_t)m * f + 16 * c + li] = a / (1.f + expf(-a)) * b;
      }
    return;
  }
  const bool split = part != nullptr;
#pragma unroll
  for (int i = 0; i < MB; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int m = m0 + wm + 16 * i + 4 * lq + r, n = n0 + wn + 16 * j + li;
        if (m >= M) continue;
        const size_t o = (size_t)m * N + n;
        float v = acc[i][j][r];
        if (split)
          part[(size_t)blockIdx.z * M * N + o] = v;
        else
          C[o] = v;
      }
}

// One workgroup per row of a K-split projection (width d, a multiple of 64;
// thread c takes columns c + 256 k): the splits' partial sums added in split
// order (loaded eight splits at a time, indices clamped so all eight loads
// are in flight together), the residual R added, the row x written; then
// the LayerNorm of x (mean, then the mean squared deviation, each a fixed
// reduction over the workgroup): head == 0 writes u = LN(x) with gain g,
// bias b; head != 0 takes LN_out and the output head, scores[row] =
// sigmoid(w_out . LN_out(x)), and advances the trace's step count.  Each
// thread re-reads only the columns it wrote.
__device__ inline float block_sum(float v, float* red) {
  v = wave_sum(v);
  __syncthreads();  // red[] is free
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return ((red[0] + red[1]) + red[2]) + red[3];
}

// The LayerNorm of row x[base ..] (s: this thread's sum of the columns it
// wrote), then u = LN(x) or the output head.
__device__ inline void ln_tail(float s, const float* x, size_t base, int d, const float* g, const float* b, float* u,
                               int head, const SeqDev& S, float* scores, int row, float* red) {
  const float mean = block_sum(s, red) / d;
  float v = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    const float e = x[base + i] - mean;
    v += e * e;
  }
  const float rstd = 1.f / sqrtf(block_sum(v, red) / d + kSeqLnEps);
  if (!head) {
    for (int i = threadIdx.x; i < d; i += 256) u[base + i] = (x[base + i] - mean) * rstd * g[i] + b[i];
    return;
  }
  float z = 0.f;
  for (int i = threadIdx.x; i < d; i += 256)
    z += ((x[base + i] - mean) * rstd * S.ln_out_g[i] + S.ln_out_b[i]) * S.w_out[i];
  z = block_sum(z, red);
  if (threadIdx.x == 0) {
    scores[row] = 1.f / (1.f + expf(-z));
    S.lens[S.ids[row]] += 1;
  }
}

__global__ __launch_bounds__(256) void reduce_ln_kernel(const float* part, int splits, const float* R,
                                                        float* x, int d, const float* g, const float* b, float* u,
                                                        int head, SeqDev S, float* scores, int n) {
  __shared__ float red[4];
  const int row = blockIdx.x;
  const size_t MN = (size_t)n * d, base = (size_t)row * d;
  float s = 0.f;
  for (int i = threadIdx.x; i < d; i += 256) {
    float y = 0.f;
    for (int z0 = 0; z0 < splits; z0 += 8) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = part[(size_t)min(z0 + e, splits - 1) * MN + base + i];
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (z0 + e < splits) y += v[e];
    }
    y += R[base + i];
    x[base + i] = y;
    s += y;
  }
  ln_tail(s, x, base, d, g, b, u, head, S, scores, row, red);
}

// The input projection's reduce, one workgroup per row: the input
// LayerNorm's statistics of h[row] (mean, then the mean squared deviation),
// the split partial sums of h W'^T over the three planes (parts
// [splits][n][3 d]: plane p of column i at p d + i), added split by split in
// order, then x = GELU(rstd (y - mean c[i]) + dv[i]) (LN_in(h) W_in^T
// rearranged: c = the row sums of W', dv = W_in b), then ln_tail.  The
// state's first 4096 values (four 8-byte loads per thread, kept in
// registers for both statistics passes) and the first column's partial sums
// of up to kInBatch splits are all requested before any of them is used.
constexpr int kInBatch = 12;

__global__ __launch_bounds__(256) void reduce_in_kernel(const uint16_t* h, int dim, const float* part, int splits,
                                                        const float* c, const float* dv, float* x, int d,
                                                        const float* g, const float* b, float* u, int head, SeqDev S,
                                                        float* scores, int n) {
  __shared__ float red[4];
  const int row = blockIdx.x, tid = threadIdx.x;
  const uint2* h4 = reinterpret_cast<const uint2*>(h + (size_t)row * dim);  // four bf16 per load
  const int nh4 = dim / 4;
  const size_t units = (size_t)3 * d, MN = (size_t)n * units, pbase = (size_t)row * units, base = (size_t)row * d;
  // split partials of column i, splits z0 .. z0 + kInBatch - 1 (indices
  // clamped: every load is in bounds; only splits < `splits` are added)
  float v[kInBatch][3];
  auto load_parts = [&](int i, int z0) {
#pragma unroll
    for (int e = 0; e < kInBatch; ++e)
#pragma unroll
      for (int p = 0; p < 3; ++p) v[e][p] = part[(size_t)min(z0 + e, splits - 1) * MN + pbase + p * d + i];
  };
  uint2 hr[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) hr[j] = tid + 256 * j < nh4 ? h4[tid + 256 * j] : make_uint2(0u, 0u);
  if (tid < d) load_parts(tid, 0);
  auto f4 = [](uint2 w, float* o) {
    o[0] = __uint_as_float(w.x << 16), o[1] = __uint_as_float(w.x & 0xFFFF0000u);
    o[2] = __uint_as_float(w.y << 16), o[3] = __uint_as_float(w.y & 0xFFFF0000u);
  };
  float hs = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {  // zeros past the row add nothing
    float e[4];
    f4(hr[j], e);
    hs += (e[0] + e[1]) + (e[2] + e[3]);
  }
  for (int i = tid + 1024; i < nh4; i += 256) {
    float e[4];
    f4(h4[i], e);
    hs += (e[0] + e[1]) + (e[2] + e[3]);
  }
  const float hmean = block_sum(hs, red) / dim;
  float hv = 0.f;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (tid + 256 * j < nh4) {
      float e[4];
      f4(hr[j], e);
#pragma unroll
      for (int k = 0; k < 4; ++k) hv += (e[k] - hmean) * (e[k] - hmean);
    }
  }
  for (int i = tid + 1024; i < nh4; i += 256) {
    float e[4];
    f4(h4[i], e);
#pragma unroll
    for (int k = 0; k < 4; ++k) hv += (e[k] - hmean) * (e[k] - hmean);
  }
  const float hrstd = 1.f / sqrtf(block_sum(hv, red) / dim + kSeqLnEps);
  float s = 0.f;
  for (int i = tid; i < d; i += 256) {
    float y = 0.f;
    for (int z0 = 0; z0 < splits; z0 += kInBatch) {
      if (i != tid || z0 != 0) load_parts(i, z0);
#pragma unroll
      for (int e = 0; e < kInBatch; ++e)
        if (z0 + e < splits) y += (v[e][0] + v[e][1]) + v[e][2];
    }
    y = gelu_erf(hrstd * (y - hmean * c[i]) + dv[i]);
    x[base + i] = y;
    s += y;
  }
  ln_tail(s, x, base, d, g, b, u, head, S, scores, row, red);
}

// The input projection's weights for the bf16 matrix cores, one workgroup
// per output row n: W'[n][k] = W_in[n][k] g[k] (an fp32 product) split into
// three bf16 planes, hi = bf16(W'), mid = bf16(W' - hi), lo = W' - hi - mid
// (each difference exact in fp32; lo has at most 8 significant bits, so
// hi + mid + lo = W' exactly), planes [3][dm][dim]; c[n] = sum_k W'[n][k]
// and dv[n] = sum_k W_in[n][k] b[k], added in fp64 and rounded once.
__device__ inline uint16_t bf16_rne(float x) {
  const uint32_t u = __float_as_uint(x);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

__global__ __launch_bounds__(256) void prep_input_kernel(const float* w, const float* g, const float* b, int dim,
                                                         int dm, uint16_t* planes, float* c, float* dv) {
  __shared__ double red[2][4];
  const int n = blockIdx.x;
  double sc = 0.0, sd = 0.0;
  for (int k = threadIdx.x; k < dim; k += 256) {
    const float wv = w[(size_t)n * dim + k];
    const float x = wv * g[k];
    const uint16_t hi = bf16_rne(x);
    const float r1 = x - __uint_as_float((uint32_t)hi << 16);
    const uint16_t mid = bf16_rne(r1);
    const float r2 = r1 - __uint_as_float((uint32_t)mid << 16);
    planes[(size_t)n * dim + k] = hi;
    planes[((size_t)dm + n) * dim + k] = mid;
    planes[((size_t)2 * dm + n) * dim + k] = bf16_rne(r2);  // exact: r2 has at most 8 significant bits
    sc += (double)x;
    sd += (double)wv * (double)b[k];
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    sc += __shfl_xor(sc, o, 64);
    sd += __shfl_xor(sd, o, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    red[0][threadIdx.x >> 6] = sc;
    red[1][threadIdx.x >> 6] = sd;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    c[n] = (float)(((red[0][0] + red[0][1]) + red[0][2]) + red[0][3]);
    dv[n] = (float)(((red[1][0] + red[1][1]) + red[1][2]) + red[1][3]);
  }
}

// One attention step of one (trace row, head), head_dim 64, four waves.
// The trace's step index t is its count of earlier steps.  Wave 0 (one
// element per lane) applies RoPE - (x_i, x_{i+32}) rotated by
// t * 10000^(-i/32) - and appends the rotated key and the value at t in the
// trace's cache: keys in groups of four steps, [ks / 4][64][4] (ks =
// max_steps rounded up to a multiple of 4), so one group's 64 dimensions
// are 1 KB of consecutive memory and four consecutive steps of a dimension
// one 16-byte load; values [ks][64].  Scores of the earlier steps: thread
// (j4, eq) takes steps 4 j4 .. 4 j4 + 3 over dimensions eq + 8 e, e < 8
// (the eight threads of a group read 128 consecutive bytes per load, so a
// wave's load touches eight whole lines; the first group's loads are issued
// before wave 0 has finished the append, which they do not depend on), and the eight
// parts are added by shuffles; steps past t - 1 in the last group are
// masked (their slots are read but never used).  The softmax is taken over
// steps 0..t; for the values, thread (g, c) takes dimensions 4 c .. 4 c + 3
// of steps j = g mod 16, and the sixteen groups' sums and step t's own term
// (its key and value in wave 0's registers) are added.
__device__ inline float block_max(float v, float* red) {
  v = wave_max(v);
  __syncthreads();  // red[] is free
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}

__global__ __launch_bounds__(256) void seq_attn_kernel(SeqDev S, int layer, const float* qkv, float* o, int n) {
  extern __shared__ __attribute__((aligned(16))) float lds[];  // p[ks], q[64], partial outputs [4][64], red[4]
  const int ks = seq_kstride(S.max_steps);
  float* p = lds;
  float* qs = p + ks;
  float* op = qs + 64;
  float* red = op + 4 * 64;
  const int row = blockIdx.x / S.n_heads, h = blockIdx.x % S.n_heads;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (row >= n) return;  // uniform over the workgroup
  const int tr = S.ids[row];
  const int t = S.lens[tr];
  if (t >= S.max_steps) {  // the host bounds step counts; keep the cache in bounds regardless
    if (tid == 0) atomicOr(S.err, 1);
    return;
  }
  const int d = S.d_model;
  float* kq = S.cache + (((size_t)tr * S.n_layers + layer) * S.n_heads + h) * seq_region_floats(S.max_steps);
  float* vc = kq + (size_t)64 * ks;
  const int eq = tid & 7, jq = tid >> 3;
  // the first group of earlier steps' keys, before the append (disjoint slots)
  float4 kv[8];
  if (4 * jq < t) {
    const float* kr = kq + (size_t)jq * 256 + 4 * eq;
#pragma unroll
    for (int e = 0; e < 8; ++e) kv[e] = ld_stream4(kr + 32 * e);
  }
  float v = 0.f, st = 0.f;
  if (wave == 0) {
    const float* src = qkv + (size_t)row * 3 * d + h * 64;
    const float q = src[lane], k = src[d + lane];
    v = src[2 * d + lane];
    const int i = lane & 31;
    const float theta = exp2f(-(float)i * (13.287712379549449f / 32.f));  // 10000^(-i/32)
    float sn, cs;
    sincosf((float)t * theta, &sn, &cs);
    const float qp = __shfl_xor(q, 32, 64), kp = __shfl_xor(k, 32, 64);
    const float qr = lane < 32 ? q * cs - qp * sn : qp * sn + q * cs;
    const float kr = lane < 32 ? k * cs - kp * sn : kp * sn + k * cs;
    kq[(size_t)(t >> 2) * 256 + 4 * lane + (t & 3)] = kr;
    vc[(size_t)t * 64 + lane] = v;
    qs[lane] = qr;
    st = wave_sum(qr * kr) * 0.125f;  // scale 1 / sqrt(64)
  }
  __syncthreads();  // qs[] is visible
  float mx = -INFINITY;
  for (int j0 = 4 * jq; j0 < t; j0 += 128) {  // 32 groups of four steps per pass
    if (j0 != 4 * jq) {
      const float* kr = kq + (size_t)(j0 >> 2) * 256 + 4 * eq;
#pragma unroll
      for (int e = 0; e < 8; ++e) kv[e] = ld_stream4(kr + 32 * e);
    }
    float4 a = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float qe = qs[eq + 8 * e];
      a.x = fmaf(qe, kv[e].x, a.x);
      a.y = fmaf(qe, kv[e].y, a.y);
      a.z = fmaf(qe, kv[e].z, a.z);
      a.w = fmaf(qe, kv[e].w, a.w);
    }
#pragma unroll
    for (int m = 1; m <= 4; m <<= 1) {
      a.x += __shfl_xor(a.x, m, 64);
      a.y += __shfl_xor(a.y, m, 64);
      a.z += __shfl_xor(a.z, m, 64);
      a.w += __shfl_xor(a.w, m, 64);
    }
    a.x = j0 < t ? a.x * 0.125f : -INFINITY;
    a.y = j0 + 1 < t ? a.y * 0.125f : -INFINITY;
    a.z = j0 + 2 < t ? a.z * 0.125f : -INFINITY;
    a.w = j0 + 3 < t ? a.w * 0.125f : -INFINITY;
    if (eq == 0) *reinterpret_cast<float4*>(p + j0) = a;
    mx = fmaxf(mx, fmaxf(fmaxf(a.x, a.y), fmaxf(a.z, a.w)));
  }
  // the values of this thread's steps j0 + g + 16 i (i < 8) of a 128-step
  // chunk, all in flight at once; the first chunk's across the softmax
  const int c = tid & 15, g = tid >> 4;
  float4 vv[8];
  auto load_v = [&](int j0) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int j = j0 + g + 16 * i;
      vv[i] = j < t ? *reinterpret_cast<const float4*>(vc + (size_t)j * 64 + 4 * c) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  load_v(0);
  if (wave == 0 && lane == 0) mx = fmaxf(mx, st);
  mx = block_max(mx, red);  // also publishes p[]
  float sum = 0.f;
  for (int j = tid; j < t; j += 256) {
    const float e = expf(p[j] - mx);
    p[j] = e;
    sum += e;
  }
  sum = block_sum(sum, red);  // also publishes the exponentials
  // steps g + 32 k into a0, g + 16 + 32 k into a1 (independent sums)
  float4 a0 = make_float4(0.f, 0.f, 0.f, 0.f), a1 = a0;
  for (int j0 = 0; j0 < t; j0 += 128) {
    if (j0) load_v(j0);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int j = j0 + g + 16 * i;
      const float pj = j < t ? p[j] : 0.f;
      float4& a = (i & 1) ? a1 : a0;
      a.x = fmaf(pj, vv[i].x, a.x), a.y = fmaf(pj, vv[i].y, a.y), a.z = fmaf(pj, vv[i].z, a.z),
      a.w = fmaf(pj, vv[i].w, a.w);
    }
  }
  a0.x += a1.x, a0.y += a1.y, a0.z += a1.z, a0.w += a1.w;
#pragma unroll
  for (int m = 16; m <= 32; m <<= 1) {  // the wave's four step groups
    a0.x += __shfl_xor(a0.x, m, 64);
    a0.y += __shfl_xor(a0.y, m, 64);
    a0.z += __shfl_xor(a0.z, m, 64);
    a0.w += __shfl_xor(a0.w, m, 64);
  }
  if (lane < 16) *reinterpret_cast<float4*>(op + wave * 64 + 4 * lane) = a0;
  __syncthreads();
  if (wave == 0) {
    const float pt = expf(st - mx);
    const float total = sum + pt;
    o[(size_t)row * d + h * 64 + lane] =
        (((op[lane] + op[64 + lane]) + op[128 + lane]) + op[192 + lane] + pt * v) / total;
  }
}

// Branch: the child's history is the parent's (its whole cache region and
// its step count).  One workgroup per (pair, slice of the region).
__global__ __launch_bounds__(256) void seq_fork_kernel(SeqDev S, const int32_t* pairs, size_t region_f4) {
  const int child = pairs[2 * blockIdx.y], parent = pairs[2 * blockIdx.y + 1];
  const float4* src = reinterpret_cast<const float4*>(S.cache) + (size_t)parent * region_f4;
  float4* dst = reinterpret_cast<float4*>(S.cache) + (size_t)child * region_f4;
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < region_f4; i += (size_t)gridDim.x * 256)
    dst[i] = src[i];
  if (blockIdx.x == 0 && threadIdx.x == 0) S.lens[child] = S.lens[parent];
}

__global__ void seq_set_len_kernel(SeqDev S, const int32_t* ids, int n, int value) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) S.lens[ids[i]] = value;
}

}  // namespace

hipError_t seq_gemm(const float* A, const float* W, float* C, int M, int N, int K, int splits, int epi, float* part,
                    hipStream_t s) {
  const int ks = K / splits;
  // 64-row tiles when they alone give the GPU ~256 workgroups, else 32-row
  const bool wide = (long)(N / 64) * ((M + 63) / 64) * splits >= 256;
  const dim3 grid(N / 64, wide ? (M + 63) / 64 : (M + 31) / 32, splits);
  if (wide)
    hipLaunchKernelGGL((gemm_kernel<64>), grid, dim3(256), 0, s, A, W, C, M, N, K, ks, epi, part);
  else
    hipLaunchKernelGGL((gemm_kernel<32>), grid, dim3(256), 0, s, A, W, C, M, N, K, ks, epi, part);
  return hipGetLastError();
}

hipError_t seq_prep_input(const float* w_in, const float* ln_g, const float* ln_b, int dim, int dm, uint16_t* planes,
                          float* c, float* dv, hipStream_t s) {
  hipLaunchKernelGGL(prep_input_kernel, dim3(dm), dim3(256), 0, s, w_in, ln_g, ln_b, dim, dm, planes, c, dv);
  return hipGetLastError();
}

hipError_t seq_reduce_in(const uint16_t* h, int dim, const float* part, int splits, const float* c, const float* dv,
                         float* x, int d, const float* g, const float* b, float* u, bool head, const SeqDev& S,
                         float* scores, int n, hipStream_t s) {
  hipLaunchKernelGGL(reduce_in_kernel, dim3(n), dim3(256), 0, s, h, dim, part, splits, c, dv, x, d, g, b, u,
                     (int)head, S, scores, n);
  return hipGetLastError();
}

hipError_t seq_reduce_ln(const float* part, int splits, const float* R, float* x, int d, const float* g,
                         const float* b, float* u, bool head, const SeqDev& S, float* scores, int n, hipStream_t s) {
  hipLaunchKernelGGL(reduce_ln_kernel, dim3(n), dim3(256), 0, s, part, splits, R, x, d, g, b, u, (int)head, S,
                     scores, n);
  return hipGetLastError();
}

hipError_t seq_attention(const SeqDev& S, int layer, const float* qkv, float* o, int n, hipStream_t s) {
  const size_t lds = sizeof(float) * ((size_t)seq_kstride(S.max_steps) + 64 + 4 * 64 + 4);
  hipLaunchKernelGGL(seq_attn_kernel, dim3(n * S.n_heads), dim3(256), lds, s, S, layer, qkv, o, n);
  return hipGetLastError();
}

hipError_t seq_fork(const SeqDev& S, const int32_t* pairs, int n, hipStream_t s) {
  const size_t region_f4 = (size_t)S.n_layers * S.n_heads * seq_region_floats(S.max_steps) / 4;
  const unsigned slices = (unsigned)std::max<size_t>(1, std::min<size_t>(64, (region_f4 + 255) / 256));
  hipLaunchKernelGGL(seq_fork_kernel, dim3(slices, n), dim3(256), 0, s, S, pairs, region_f4);
  return hipGetLastError();
}

hipError_t seq_set_len(const SeqDev& S, const int32_t* ids, int n, int value, hipStream_t s) {
  hipLaunchKernelGGL(seq_set_len_kernel, dim3((n + 255) / 256), dim3(256), 0, s, S, ids, n, value);
  return hipGetLastError();
}

}  // namespace gambit
