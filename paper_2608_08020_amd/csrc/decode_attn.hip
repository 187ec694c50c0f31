// Shared-prefix split-K paged GQA decode attention for gfx950.
//
// Traces that branched from a common parent share the parent's KV blocks
// (Alg. 1 notation, Branch; Sec. 4.1 Case 2; Sec. 5.3: children inherit the
// parent's physical KV-cache).  The host plan cuts every trace's context
// into runs of blocks that the same set of traces reference; one work unit
// is (run chunk, KV head, tile of up to 128 rows), where a row is one
// (member trace, query head of the GQA group).  A workgroup stages each
// 64-token slice of the chunk's K and V through LDS once and applies it to
// all its rows, so a block shared by m traces is read from HBM once per
// step instead of m times.  Each unit leaves an unnormalised partial
// (running max, running sum, accumulator) per row; the merge kernel
// combines a row's partials by log-sum-exp.
//
// The two contractions run on the bf16 matrix cores
// (v_mfma_f32_16x16x32_bf16):
//   S^T[token][row] = K[token][:] . Q[row][:]          (A = K, B = Q^T)
//   O^T[d][row]    += V^T[d][token] . P^T[token][row]   (A = V^T, B = P^T)
// Computing S transposed leaves each lane holding, for one row, four
// consecutive tokens of each 16-token half, which is exactly the B-operand
// layout of the second product, so P never moves between lanes.  P is split
// into bf16 hi + lo parts (two MFMAs) so the P.V product keeps ~16 bits of
// P's precision.  fp8 E4M3 KV is widened to bf16 (exact) while it is staged
// into LDS; the per-block K scale multiplies the scores of its 16 tokens and
// the V scale multiplies P before the P.V product.
#include <cmath>

#include "kernels.h"

namespace gambit {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kStageTok = 64;            // tokens staged per pipeline step (4 blocks)
constexpr int kRowBytes = kHeadDim * 2;  // one bf16 token row of one head in LDS
constexpr int kRBW = kRowsPerWG / 64;    // 16-row blocks per wave (4 waves)

__device__ inline int lds_off(int row, int chunk) {
  // 16 chunks of 16 B per row, XOR-swizzled by the row so that reads of one
  // chunk index across 16 rows, and of 16 chunks of one row, hit distinct banks
  return row * kRowBytes + ((chunk ^ (row & 15)) << 4);
}

__device__ inline uint32_t pack_bf16x2(float a, float b) {
  const __bf16 x = (__bf16)a, y = (__bf16)b;
  return (uint32_t)__builtin_bit_cast(uint16_t, x) | ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
}

// 16 fp8 E4M3 codes -> 16 bf16 (two 16-byte chunks).  The widening is exact.
__device__ inline void fp8x16_to_bf16(const uint4 in, uint4& lo, uint4& hi) {
  const uint32_t w[4] = {in.x, in.y, in.z, in.w};
  uint32_t o[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const f32x2 a = __builtin_amdgcn_cvt_pk_f32_fp8(w[i], false);
    const f32x2 b = __builtin_amdgcn_cvt_pk_f32_fp8(w[i], true);
    o[2 * i] = pack_bf16x2(a[0], a[1]);
    o[2 * i + 1] = pack_bf16x2(b[0], b[1]);
  }
  lo = make_uint4(o[0], o[1], o[2], o[3]);
  hi = make_uint4(o[4], o[5], o[6], o[7]);
}

// A table entry outside the pool is never dereferenced: the token reads as
// zeros and the device error word records it (a -1 marks "no token here").
__device__ inline bool valid_block(const DevPool& P, int b) {
  if ((unsigned)b < (unsigned)P.num_blocks) return true;
  if (b != -1) atomicOr(P.err, kErrBadBlock);
  return false;
}

struct Regs {
  uint4 k[4], v[4];
};

template <bool FP8>
__device__ inline void load_stage(const DevPool& P, const int32_t* brow, int kvh, int ntok, int s,
                                  Regs& r) {
  const int t = threadIdx.x;
  if constexpr (!FP8) {
    // 4 blocks x 16 tokens x 16 chunks = 1024 chunks of K (and of V)
    const int tok = t >> 4, c = t & 15;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int ti = s * kStageTok + n * kBlock + tok;
      const int b = ti < ntok ? brow[s * 4 + n] : -1;
      if (valid_block(P, b)) {
        const size_t off = (((size_t)b * P.Hkv + kvh) * kBlock + tok) * kRowBytes + c * 16;
        r.k[n] = *reinterpret_cast<const uint4*>(P.k_cache + off);
        r.v[n] = *reinterpret_cast<const uint4*>(P.v_cache + off);
      } else {
        r.k[n] = make_uint4(0, 0, 0, 0);
        r.v[n] = make_uint4(0, 0, 0, 0);
      }
    }
  } else {
    // 4 blocks x 16 tokens x 8 chunks = 512 chunks of fp8 K (and of V)
    const int c8 = t & 7, tok = (t >> 3) & 15, half = t >> 7;
#pragma unroll
    for (int n = 0; n < 2; ++n) {
      const int blk = 2 * n + half;
      const int ti = s * kStageTok + blk * kBlock + tok;
      const int b = ti < ntok ? brow[s * 4 + blk] : -1;
      if (valid_block(P, b)) {
        const size_t off = (((size_t)b * P.Hkv + kvh) * kBlock + tok) * kHeadDim + c8 * 16;
        r.k[n] = *reinterpret_cast<const uint4*>(P.k_cache + off);
        r.v[n] = *reinterpret_cast<const uint4*>(P.v_cache + off);
      } else {
        r.k[n] = make_uint4(0, 0, 0, 0);
        r.v[n] = make_uint4(0, 0, 0, 0);
      }
    }
  }
}

template <bool FP8>
__device__ inline void store_stage(uint8_t* kl, uint8_t* vl, const Regs& r) {
  const int t = threadIdx.x;
  if constexpr (!FP8) {
    const int tok = t >> 4, c = t & 15;
#pragma unroll
    for (int n = 0; n < 4; ++n) {
      const int row = n * kBlock + tok;
      *reinterpret_cast<uint4*>(kl + lds_off(row, c)) = r.k[n];
      *reinterpret_cast<uint4*>(vl + lds_off(row, c)) = r.v[n];
    }
  } else {
    const int c8 = t & 7, tok = (t >> 3) & 15, half = t >> 7;
#pragma unroll
    for (int n = 0; n < 2; ++n) {
      const int row = (2 * n + half) * kBlock + tok;
      uint4 lo, hi;
      fp8x16_to_bf16(r.k[n], lo, hi);
      *reinterpret_cast<uint4*>(kl + lds_off(row, 2 * c8)) = lo;
      *reinterpret_cast<uint4*>(kl + lds_off(row, 2 * c8 + 1)) = hi;
      fp8x16_to_bf16(r.v[n], lo, hi);
      *reinterpret_cast<uint4*>(vl + lds_off(row, 2 * c8)) = lo;
      *reinterpret_cast<uint4*>(vl + lds_off(row, 2 * c8 + 1)) = hi;
    }
  }
}

__device__ inline float wave_max_over_groups(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  x = fmaxf(x, __shfl_xor(x, 32));
  return x;
}

__device__ inline float wave_sum_over_groups(float x) {
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}

template <bool FP8>
__global__ __launch_bounds__(kThreads, 2) void attn_units_kernel(DevPool P, AttnLaunch A) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[2][2][kStageTok * kRowBytes];

  // Workgroups are dispatched round-robin over the 8 XCDs, so workgroup bid
  // runs on XCD bid % 8.  The plan assigns each unit to an XCD (row tiles
  // that re-read the same chunk go to the same XCD and share its L2) and
  // lists every XCD's units contiguously.
  const int x = blockIdx.x & 7, slot = blockIdx.x >> 3;
  if (slot >= A.xcd_off[x + 1] - A.xcd_off[x]) return;
  const AttnUnit U = A.units[A.xcd_off[x] + slot];
  if (U.mem_cnt == 0) return;

  const int32_t* brow = P.table + (size_t)U.owner * P.max_blocks + U.jb0;
  const int ntok = U.nblk >= 0 ? U.nblk * kBlock : P.seq_len[U.owner] - U.jb0 * kBlock;
  if (ntok <= 0) return;
  const int nstage = (ntok + kStageTok - 1) / kStageTok;
  const int g = P.g;
  const int R = U.mem_cnt * g;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int lq = lane >> 4, lr = lane & 15;

  // Q^T operands of this wave's row blocks: lane (lq, lr) holds row lr,
  // d = 32 kb + 8 lq .. +7 for kb = 0..3.
  bf16x8 qf[kRBW][4];
  bool active[kRBW];
#pragma unroll
  for (int i = 0; i < kRBW; ++i) {
    const int rb = wave + 4 * i;
    active[i] = rb * 16 < R;
    const int r = rb * 16 + lr;
    if (r < R) {
      const int pos = A.members[U.mem_off + r / g];
      const int h = U.kvh * g + r % g;
      const bf16x8* qp = reinterpret_cast<const bf16x8*>(A.q + ((size_t)pos * P.Hq + h) * kHeadDim + lq * 8);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) qf[i][kb] = qp[kb * 4];
    } else {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) qf[i][kb] = bf16x8{};
    }
  }

  float m_run[kRBW], l_run[kRBW];
  f32x4 acc[kRBW][8];
#pragma unroll
  for (int i = 0; i < kRBW; ++i) {
    m_run[i] = -INFINITY;
    l_run[i] = 0.f;
#pragma unroll
    for (int r = 0; r < 8; ++r) acc[i][r] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  Regs regs;
  load_stage<FP8>(P, brow, U.kvh, ntok, 0, regs);
  store_stage<FP8>(lds[0][0], lds[0][1], regs);
  __syncthreads();

  for (int s = 0; s < nstage; ++s) {
    const int buf = s & 1;
    if (s + 1 < nstage) load_stage<FP8>(P, brow, U.kvh, ntok, s + 1, regs);

    const uint8_t* kl = lds[buf][0];
    const uint8_t* vl = lds[buf][1];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int t0 = s * kStageTok + st * 32;  // first token of the 32-token sub-tile
      if (t0 >= ntok) break;
      bool any = false;
#pragma unroll
      for (int i = 0; i < kRBW; ++i) any |= active[i];
      if (!any) break;

      float ks0 = 1.f, ks1 = 1.f, vs0 = 1.f, vs1 = 1.f;
      if constexpr (FP8) {
        const int b0 = brow[t0 / kBlock];
        if ((unsigned)b0 < (unsigned)P.num_blocks) {
          ks0 = P.kv_scale[2 * b0];
          vs0 = P.kv_scale[2 * b0 + 1];
        }
        if (t0 + kBlock < ntok) {
          const int b1 = brow[t0 / kBlock + 1];
          if ((unsigned)b1 < (unsigned)P.num_blocks) {
            ks1 = P.kv_scale[2 * b1];
            vs1 = P.kv_scale[2 * b1 + 1];
          }
        }
      }

      // K operands: token row 32 st + 16 half + lr, chunk 4 kb + lq.
      bf16x8 kf[2][4];
#pragma unroll
      for (int hf = 0; hf < 2; ++hf)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
          kf[hf][kb] = *reinterpret_cast<const bf16x8*>(kl + lds_off(st * 32 + hf * 16 + lr, kb * 4 + lq));

      // V operands: lane (lq, lr) reads d-chunk lr of its 8 tokens
      // tok(e) = 4 lq + e (e < 4) and 16 + 4 lq + e - 4 (e >= 4), then
      // transposes so that operand r holds d = 8 lr + r of those 8 tokens.
      bf16x8 vf[8];
      {
        bf16x8 vraw[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int tok = st * 32 + (e < 4 ? 4 * lq + e : 16 + 4 * lq + e - 4);
          vraw[e] = *reinterpret_cast<const bf16x8*>(vl + lds_off(tok, lr));
        }
#pragma unroll
        for (int r = 0; r < 8; ++r)
#pragma unroll
          for (int e = 0; e < 8; ++e) vf[r][e] = vraw[e][r];
      }

#pragma unroll
      for (int i = 0; i < kRBW; ++i) {
        if (!active[i]) continue;
        f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[0][kb], qf[i][kb], s0, 0, 0, 0);
          s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[1][kb], qf[i][kb], s1, 0, 0, 0);
        }
        // lane (lq, lr): s0[e] is token t0 + 4 lq + e, s1[e] token t0 + 16 + 4 lq + e, row lr
        float sv[8];
        const float c0 = A.scale_log2 * ks0, c1 = A.scale_log2 * ks1;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          sv[e] = (t0 + 4 * lq + e < ntok) ? s0[e] * c0 : -INFINITY;
          sv[4 + e] = (t0 + 16 + 4 * lq + e < ntok) ? s1[e] * c1 : -INFINITY;
        }
        float mx = sv[0];
#pragma unroll
        for (int e = 1; e < 8; ++e) mx = fmaxf(mx, sv[e]);
        mx = wave_max_over_groups(mx);
        const float m_new = fmaxf(m_run[i], mx);
        const float alpha = exp2f(m_run[i] - m_new);
        float p[8], psum = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          p[e] = exp2f(sv[e] - m_new);
          psum += p[e];
        }
        l_run[i] = l_run[i] * alpha + psum;
        m_run[i] = m_new;
#pragma unroll
        for (int r = 0; r < 8; ++r) acc[i][r] *= alpha;
        bf16x8 ph, pl;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float pv = FP8 ? p[e] * (e < 4 ? vs0 : vs1) : p[e];
          const __bf16 hb = (__bf16)pv;
          ph[e] = hb;
          pl[e] = (__bf16)(pv - (float)hb);
        }
#pragma unroll
        for (int r = 0; r < 8; ++r) {
          acc[i][r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[r], ph, acc[i][r], 0, 0, 0);
          acc[i][r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[r], pl, acc[i][r], 0, 0, 0);
        }
      }
    }

    if (s + 1 < nstage) store_stage<FP8>(lds[buf ^ 1][0], lds[buf ^ 1][1], regs);
    __syncthreads();
  }

  // Partials: lane (lq, lr) holds O[row lr][32 lq .. 32 lq + 31] with
  // acc[i][r][e] at d = 32 lq + 8 e + r.
#pragma unroll
  for (int i = 0; i < kRBW; ++i) {
    if (!active[i]) continue;
    const float l = wave_sum_over_groups(l_run[i]);
    const int r = (wave + 4 * i) * 16 + lr;
    if (r >= R) continue;
    const int pos = A.members[U.mem_off + r / g];
    const int h = U.kvh * g + r % g;
    const size_t idx = ((size_t)pos * P.Hq + h) * A.kmax + U.kidx;
    f32x4* dst = reinterpret_cast<f32x4*>(A.part_acc + idx * kHeadDim + 32 * lq);
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const int e = k >> 1, rb = 4 * (k & 1);
      dst[k] = f32x4{acc[i][rb][e], acc[i][rb + 1][e], acc[i][rb + 2][e], acc[i][rb + 3][e]};
    }
    if (lq == 0) A.part_ml[idx] = float2{m_run[i], l};
  }
}

// Log-sum-exp merge of a row's partials, in partial-slot order.  One wave
// per (list position, query head); lane l owns d = 2 l, 2 l + 1.
__global__ __launch_bounds__(256) void merge_kernel(DevPool P, AttnLaunch A) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= A.n * P.Hq) return;
  const int lane = threadIdx.x & 63;
  const int pos = row / P.Hq;
  const int nk = A.nk[pos];
  const float2* ml = A.part_ml + (size_t)row * A.kmax;
  const float* pa = A.part_acc + (size_t)row * A.kmax * kHeadDim;
  float M = -INFINITY;
  for (int k = 0; k < nk; ++k) M = fmaxf(M, ml[k].x);
  float L = 0.f, o0 = 0.f, o1 = 0.f;
  for (int k = 0; k < nk; ++k) {
    const float w = exp2f(ml[k].x - M);
    L += w * ml[k].y;
    const float2 a = *reinterpret_cast<const float2*>(pa + (size_t)k * kHeadDim + 2 * lane);
    o0 += w * a.x;
    o1 += w * a.y;
  }
  const float inv = 1.f / L;
  o0 *= inv;
  o1 *= inv;
  if (A.out_f32) {
    reinterpret_cast<float2*>(A.out)[(size_t)row * (kHeadDim / 2) + lane] = float2{o0, o1};
  } else {
    reinterpret_cast<uint32_t*>(A.out)[(size_t)row * (kHeadDim / 2) + lane] = pack_bf16x2(o0, o1);
  }
}

}  // namespace

hipError_t launch_attention_units(const DevPool& P, const AttnLaunch& A, hipStream_t s) {
  if (A.n <= 0 || A.grid <= 0) return hipSuccess;
  if (P.esize == 1)
    hipLaunchKernelGGL(attn_units_kernel<true>, dim3(A.grid), dim3(kThreads), 0, s, P, A);
  else
    hipLaunchKernelGGL(attn_units_kernel<false>, dim3(A.grid), dim3(kThreads), 0, s, P, A);
  return hipGetLastError();
}

hipError_t launch_attention_merge(const DevPool& P, const AttnLaunch& A, hipStream_t s) {
  if (A.n <= 0) return hipSuccess;
  const int rows = A.n * P.Hq;
  hipLaunchKernelGGL(merge_kernel, dim3((rows + 3) / 4), dim3(256), 0, s, P, A);
  return hipGetLastError();
}

}  // namespace gambit
