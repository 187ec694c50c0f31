// The history-aware sequence scorer (App. A.1, Eqs. 4-6), one new step per
// trace per thought boundary against cached keys and values of the trace's
// earlier steps.  fp32 throughout (weights and activations); the step states
// arrive in bf16.
//
// Per boundary, for the n listed traces (rows):
//   u0 = LN_in(h)                          ln_rows_kernel (bf16 input)
//   x  = GELU(u0 W_in^T)                   gemm_kernel, split over K, reduce + GELU
//   per layer: u = LN1(x); qkv = u Wqkv^T; o = attention step (RoPE, append
//   the step's key and value, attend over the trace's steps 0..t);
//   x += o Wo^T; u = LN2(x); a = u W13^T; g = SiLU(a1) * a3; x += g W2^T
//   y  = sigmoid(w_out . LN_out(x)), and the trace's step count advances.
#include <hip/hip_runtime.h>

#include "seq_kernels.h"

namespace gambit {
namespace {

constexpr int kBM = 64, kBN = 64, kBK = 16;

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

// LayerNorm of each row (one wave per row): mean, then the mean squared
// deviation, both over the row; out = (x - mean) / sqrt(var + eps) * g + b.
__global__ __launch_bounds__(256) void ln_rows_kernel(const void* in, int in_bf16, float* out, int dim,
                                                      const float* g, const float* b, int n) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= n) return;
  const size_t base = (size_t)row * dim;
  float s = 0.f;
  for (int i = lane; i < dim; i += 64) s += load_elem(in, base + i, in_bf16);
  const float mean = wave_sum(s) / dim;
  float v = 0.f;
  for (int i = lane; i < dim; i += 64) {
    const float d = load_elem(in, base + i, in_bf16) - mean;
    v += d * d;
  }
  const float rstd = 1.f / sqrtf(wave_sum(v) / dim + kSeqLnEps);
  for (int i = lane; i < dim; i += 64)
    out[base + i] = (load_elem(in, base + i, in_bf16) - mean) * rstd * g[i] + b[i];
}

__device__ inline float gelu_erf(float x) { return 0.5f * x * (1.f + erff(x * 0.70710678118654752f)); }

// C[M][N] = A[M][K] . W[N][K]^T over K range [z * ks, (z + 1) * ks) of split
// z = blockIdx.z.  64 x 64 tiles, 16-deep K steps through LDS, 4 x 4 outputs
// per thread.  One split: the epilogue is applied and C written; several:
// the raw sums go to part[z][M][N] for seq_reduce_kernel.
__global__ __launch_bounds__(256) void gemm_kernel(const float* A, const float* W, float* C, int M, int N, int K,
                                                   int ks, int epi, const float* R, float* part) {
  __shared__ float As[kBK][kBM + 4];
  __shared__ float Ws[kBK][kBN + 4];
  const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
  const int m0 = blockIdx.y * kBM, n0 = blockIdx.x * kBN;
  const int k0 = blockIdx.z * ks, k1 = k0 + ks;
  const int lr = tid >> 2, lk = (tid & 3) * 4;  // loader: row lr of the tile, k offset lk
  float acc[4][4] = {};
  for (int kb = k0; kb < k1; kb += kBK) {
    float4 av = make_float4(0.f, 0.f, 0.f, 0.f);
    if (m0 + lr < M) av = *reinterpret_cast<const float4*>(A + (size_t)(m0 + lr) * K + kb + lk);
    const float4 wv = *reinterpret_cast<const float4*>(W + (size_t)(n0 + lr) * K + kb + lk);
    __syncthreads();  // the previous step's reads are done
    As[lk + 0][lr] = av.x;
    As[lk + 1][lr] = av.y;
    As[lk + 2][lr] = av.z;
    As[lk + 3][lr] = av.w;
    Ws[lk + 0][lr] = wv.x;
    Ws[lk + 1][lr] = wv.y;
    Ws[lk + 2][lr] = wv.z;
    Ws[lk + 3][lr] = wv.w;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kBK; ++k) {
      const float4 a = *reinterpret_cast<const float4*>(&As[k][ty * 4]);
      const float4 w = *reinterpret_cast<const float4*>(&Ws[k][tx * 4]);
      const float ar[4] = {a.x, a.y, a.z, a.w}, wr[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(ar[i], wr[j], acc[i][j]);
    }
  }
  const bool split = gridDim.z > 1;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = m0 + ty * 4 + i;
    if (m >= M) break;
    const size_t o = (size_t)m * N + n0 + tx * 4;
    float4 r = make_float4(acc[i][0], acc[i][1], acc[i][2], acc[i][3]);
    if (split) {
      *reinterpret_cast<float4*>(part + (size_t)blockIdx.z * M * N + o) = r;
      continue;
    }
    if (epi == kEpiGelu) {
      r.x = gelu_erf(r.x), r.y = gelu_erf(r.y), r.z = gelu_erf(r.z), r.w = gelu_erf(r.w);
    } else if (epi == kEpiResid) {
      const float4 q = *reinterpret_cast<const float4*>(R + o);
      r.x += q.x, r.y += q.y, r.z += q.z, r.w += q.w;
    }
    *reinterpret_cast<float4*>(C + o) = r;
  }
}

// Sum of the splits in split order, then the epilogue.
__global__ __launch_bounds__(256) void seq_reduce_kernel(const float* part, int splits, float* C, size_t MN, int epi,
                                                         const float* R) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= MN) return;
  float s = 0.f;
  for (int z = 0; z < splits; ++z) s += part[(size_t)z * MN + i];
  if (epi == kEpiGelu) s = gelu_erf(s);
  if (epi == kEpiResid) s += R[i];
  C[i] = s;
}

// g[m][j] = SiLU(a[m][j]) * a[m][f + j]   (a = u W13^T, W1 rows then W3 rows)
__global__ __launch_bounds__(256) void swiglu_kernel(const float* a, float* g, int n, int f) {
  const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= (size_t)n * f) return;
  const size_t m = i / f, j = i % f;
  const float x = a[m * 2 * f + j], y = a[m * 2 * f + f + j];
  g[i] = x / (1.f + expf(-x)) * y;
}

// One attention step of one (trace row, head), one wave, head_dim 64 (one
// element per lane).  The trace's step index t is its count of earlier
// steps.  RoPE rotates (x_i, x_{i+32}) by t * 10000^(-i/32); the rotated key
// and the value are appended at t in the trace's cache (keys transposed,
// [64][max_steps], so the score loop reads consecutive steps across lanes;
// values [max_steps][64]); then softmax over steps 0..t.  Step t's own score
// and value come from registers, the earlier ones from the cache.
__global__ __launch_bounds__(64) void seq_attn_kernel(SeqDev S, int layer, const float* qkv, float* o, int n) {
  extern __shared__ float lds[];  // p[max_steps], q[64]
  float* p = lds;
  float* qs = lds + S.max_steps;
  const int row = blockIdx.x / S.n_heads, h = blockIdx.x % S.n_heads, lane = threadIdx.x;
  if (row >= n) return;
  const int tr = S.ids[row];
  const int t = S.lens[tr];
  if (t >= S.max_steps) {  // the host bounds step counts; keep the cache in bounds regardless
    if (lane == 0) atomicOr(S.err, 1);
    return;
  }
  const int d = S.d_model;
  const float* src = qkv + (size_t)row * 3 * d + h * 64;
  const float q = src[lane], k = src[d + lane], v = src[2 * d + lane];
  const int i = lane & 31;
  const float theta = exp2f(-(float)i * (13.287712379549449f / 32.f));  // 10000^(-i/32)
  float sn, cs;
  sincosf((float)t * theta, &sn, &cs);
  const float qp = __shfl_xor(q, 32, 64), kp = __shfl_xor(k, 32, 64);
  const float qr = lane < 32 ? q * cs - qp * sn : qp * sn + q * cs;
  const float kr = lane < 32 ? k * cs - kp * sn : kp * sn + k * cs;
  float* kt = S.cache + (((size_t)tr * S.n_layers + layer) * S.n_heads + h) * (size_t)(2 * 64 * S.max_steps);
  float* vc = kt + (size_t)64 * S.max_steps;
  kt[(size_t)lane * S.max_steps + t] = kr;
  vc[(size_t)t * 64 + lane] = v;
  qs[lane] = qr;
  __syncthreads();
  const float scale = 0.125f;  // 1 / sqrt(64)
  float mx = wave_sum(qr * kr) * scale;
  const float st = mx;
  for (int j = lane; j < t; j += 64) {
    float s = 0.f;
#pragma unroll 8
    for (int e = 0; e < 64; ++e) s = fmaf(qs[e], kt[(size_t)e * S.max_steps + j], s);
    s *= scale;
    p[j] = s;
    mx = fmaxf(mx, s);
  }
  mx = wave_max(mx);
  float sum = 0.f;
  for (int j = lane; j < t; j += 64) {
    const float e = expf(p[j] - mx);
    p[j] = e;
    sum += e;
  }
  const float pt = expf(st - mx);
  sum = wave_sum(sum) + pt;
  __syncthreads();
  float acc = pt * v;
  for (int j = 0; j < t; ++j) acc = fmaf(p[j], vc[(size_t)j * 64 + lane], acc);
  o[(size_t)row * d + h * 64 + lane] = acc / sum;
}

// y = sigmoid(w_out . LN_out(x_row)); the trace's step count advances.
__global__ __launch_bounds__(256) void seq_head_kernel(SeqDev S, const float* x, float* scores, int n) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (row >= n) return;
  const int d = S.d_model;
  const float* xr = x + (size_t)row * d;
  float s = 0.f;
  for (int i = lane; i < d; i += 64) s += xr[i];
  const float mean = wave_sum(s) / d;
  float v = 0.f;
  for (int i = lane; i < d; i += 64) v += (xr[i] - mean) * (xr[i] - mean);
  const float rstd = 1.f / sqrtf(wave_sum(v) / d + kSeqLnEps);
  float z = 0.f;
  for (int i = lane; i < d; i += 64) z += ((xr[i] - mean) * rstd * S.ln_out_g[i] + S.ln_out_b[i]) * S.w_out[i];
  z = wave_sum(z);
  if (lane == 0) {
    scores[row] = 1.f / (1.f + expf(-z));
    S.lens[S.ids[row]] += 1;
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

hipError_t seq_ln_rows(const void* in, bool in_bf16, float* out, int dim, const float* g, const float* b, int n,
                       hipStream_t s) {
  hipLaunchKernelGGL(ln_rows_kernel, dim3((n + 3) / 4), dim3(256), 0, s, in, (int)in_bf16, out, dim, g, b, n);
  return hipGetLastError();
}

hipError_t seq_gemm(const float* A, const float* W, float* C, int M, int N, int K, int splits, int epi,
                    const float* R, float* part, hipStream_t s) {
  const int ks = K / splits;
  hipLaunchKernelGGL(gemm_kernel, dim3(N / kBN, (M + kBM - 1) / kBM, splits), dim3(256), 0, s, A, W, C, M, N, K,
                     ks, epi, R, part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const size_t MN = (size_t)M * N;
  hipLaunchKernelGGL(seq_reduce_kernel, dim3((unsigned)((MN + 255) / 256)), dim3(256), 0, s, part, splits, C, MN,
                     epi, R);
  return hipGetLastError();
}

hipError_t seq_swiglu(const float* a, float* g, int n, int f, hipStream_t s) {
  const size_t total = (size_t)n * f;
  hipLaunchKernelGGL(swiglu_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, a, g, n, f);
  return hipGetLastError();
}

hipError_t seq_attention(const SeqDev& S, int layer, const float* qkv, float* o, int n, hipStream_t s) {
  const size_t lds = sizeof(float) * ((size_t)S.max_steps + 64);
  hipLaunchKernelGGL(seq_attn_kernel, dim3(n * S.n_heads), dim3(64), lds, s, S, layer, qkv, o, n);
  return hipGetLastError();
}

hipError_t seq_head(const SeqDev& S, const float* x, float* scores, int n, hipStream_t s) {
  hipLaunchKernelGGL(seq_head_kernel, dim3((n + 3) / 4), dim3(256), 0, s, S, x, scores, n);
  return hipGetLastError();
}

hipError_t seq_fork(const SeqDev& S, const int32_t* pairs, int n, hipStream_t s) {
  const size_t region_f4 = (size_t)S.n_layers * S.n_heads * 2 * 64 * S.max_steps / 4;
  const unsigned slices = (unsigned)std::max<size_t>(1, std::min<size_t>(64, (region_f4 + 255) / 256));
  hipLaunchKernelGGL(seq_fork_kernel, dim3(slices, n), dim3(256), 0, s, S, pairs, region_f4);
  return hipGetLastError();
}

hipError_t seq_set_len(const SeqDev& S, const int32_t* ids, int n, int value, hipStream_t s) {
  hipLaunchKernelGGL(seq_set_len_kernel, dim3((n + 255) / 256), dim3(256), 0, s, S, ids, n, value);
  return hipGetLastError();
}

}  // namespace gambit
