// Device side of the sequence scorer: its view of the caller's memory and
// the kernel launchers (seqscorer.hip).
#pragma once
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "kernels.h"

namespace gambit {

constexpr float kSeqLnEps = 1e-5f;
// Row stride of a head's cached keys and values: max_steps rounded up to a
// multiple of 4 (16-byte loads of four consecutive steps).
__host__ __device__ constexpr int seq_kstride(int max_steps) { return (max_steps + 3) & ~3; }
// Floats of one (trace, layer, head) cache region: keys and values, plus 64
// floats of padding so that regions do not start at the same offset modulo
// a large power of two (every region's first lines would fall on the same
// memory channels).
__host__ __device__ constexpr size_t seq_region_floats(int max_steps) {
  return (size_t)2 * 64 * seq_kstride(max_steps) + 64;
}
enum : int { kEpiNone = 0, kEpiSwiGLU = 1 };

struct SeqDev {
  const int32_t* ids;     // [n] listed trace slots, this boundary
  int32_t* lens;          // [max_traces] steps held per slot
  int32_t* err;           // device error word
  float* cache;           // [max_traces][n_layers][n_heads] regions of seq_region_floats: keys [ks / 4][64][4],
                          // values [ks][64], ks = seq_kstride
  const float* ln_out_g;
  const float* ln_out_b;
  const float* w_out;
  int32_t d_model, n_heads, n_layers, max_steps;
};

// C = A W^T (fp32); N a multiple of 64, K / splits a multiple of 16.
// part != NULL: the raw sums of the splits go to part[splits][M][N] (for
// seq_reduce_ln); else one split, written to C as it is (kEpiNone) or
// through the SwiGLU gate (kEpiSwiGLU).
hipError_t seq_gemm(const float* A, const float* W, float* C, int M, int N, int K, int splits, int epi, float* part,
                    hipStream_t s);
// The input projection's bf16 planes [3][dm][dim] of W_in scaled by the
// input LayerNorm's gain (hi + mid + lo equal it exactly), their row sums c
// and dv = W_in b (one launch, at creation).
hipError_t seq_prep_input(const float* w_in, const float* ln_g, const float* ln_b, int dim, int dm, uint16_t* planes,
                          float* c, float* dv, hipStream_t s);
// x = GELU(LN_in(h) W_in^T) from the split partial sums of h against the
// planes (part [splits][n][3 d]), then as seq_reduce_ln.
hipError_t seq_reduce_in(const uint16_t* h, int dim, const float* part, int splits, const float* c, const float* dv,
                         float* x, int d, const float* g, const float* b, float* u, bool head, const SeqDev& S,
                         float* scores, int n, hipStream_t s);
// x = R + the sum of the splits of part (R, the residual, may be x itself),
// then u = LN(x; g, b), or with head the output head's scores and the step
// counts' advance.
hipError_t seq_reduce_ln(const float* part, int splits, const float* R, float* x, int d, const float* g,
                         const float* b, float* u, bool head, const SeqDev& S, float* scores, int n, hipStream_t s);
// parts[s][t][u] = the sum over split s's k range of h[t][k] w[u][k], bf16
// operands and fp32 sums, for s < splits: the MLP scorer's split-k GEMM
// without its epilogue (mlp_scorer.hip).  dim a multiple of 128, units a
// multiple of 4, 1 <= splits <= dim / 128; bf16_partial_splits gives the
// MLP scorer's count (at most kMlpSplitBytes of sums when above one).
inline int bf16_partial_splits(int32_t n, int32_t dim, int32_t units) {
  const int s = mlp_splits(n, units);
  return s < dim / 128 ? s : dim / 128;
}
hipError_t bf16_gemm_partials(const uint16_t* h, const uint16_t* w, int32_t n, int32_t dim, int32_t units,
                              int32_t splits, float* parts, hipStream_t s);
hipError_t seq_attention(const SeqDev& S, int layer, const float* qkv, float* o, int n, hipStream_t s);
hipError_t seq_fork(const SeqDev& S, const int32_t* pairs, int n, hipStream_t s);
hipError_t seq_set_len(const SeqDev& S, const int32_t* ids, int n, int value, hipStream_t s);

}  // namespace gambit
