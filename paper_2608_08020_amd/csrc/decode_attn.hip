// Shared-prefix split-K paged GQA decode attention for gfx950.
//
// Traces that branched from a common parent share the parent's KV blocks
// (Alg. 1 notation, Branch; Sec. 4.1 Case 2; Sec. 5.3: children inherit the
// parent's physical KV-cache).  The host plan cuts every trace's context
// into runs of blocks that the same set of traces reference and cuts each
// run into chunks.  The rows of a chunk are (member trace, query head of
// the GQA group) pairs, in blocks of 16.  Each chunk's K/V is read from HBM
// once per step for all its rows; its result per row is an unnormalised
// partial (reference max, sum, accumulator) that the merge kernel combines
// by log-sum-exp.
//
// Two kinds of workgroup share one launch, interleaved on every XCD:
//  * narrow: four independent one-row-block units, one per wave.  A wave
//    streams its chunk 32 tokens at a time straight from HBM into matrix-core
//    operand layouts, double-buffered in registers, with no LDS and no
//    barrier (this is where most of the bytes are: chunks that 1-4 traces
//    share).
//  * cooperative: one chunk with 2-4 row blocks (more rows become several
//    workgroups).  The workgroup stages each 32-token tile into LDS once
//    (double-buffered) and each wave applies it to its row block, so a chunk
//    is read from L2/HBM once per four row blocks instead of once per row
//    block; many row blocks re-reading one chunk through L2 otherwise
//    contend for the same L2 channels.
//
// The contractions run on the bf16 matrix cores (v_mfma_f32_16x16x32_bf16):
//   S^T[token][row] = K[token][:] . Q[row][:]          (A = K, B = Q^T)
//   O^T[d][row]    += V^T[d][token] . P^T[token][row]   (A = V^T, B = P^T)
// Computing S transposed leaves each lane holding, for one row, four
// consecutive tokens of each 16-token half, which is exactly the B-operand
// layout of the second product, so P never moves between lanes.  V is read
// as 16 bytes of d for each of a lane's 8 tokens and transposed in
// registers.  P is split into bf16 hi + lo parts (two MFMAs) so the P.V
// product keeps ~16 bits of P.  fp8 E4M3 K/V are widened to bf16 (exact);
// a block's K scale multiplies its 16 scores and the V scale multiplies P.
#include <cmath>

#include "kernels.h"

namespace gambit {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;          // four waves
constexpr int kLdsRow = 2 * kHeadDim;  // bytes of one bf16 token row of one head

__device__ inline uint32_t pack_bf16x2(float a, float b) {
  const __bf16 x = (__bf16)a, y = (__bf16)b;
  return (uint32_t)__builtin_bit_cast(uint16_t, x) | ((uint32_t)__builtin_bit_cast(uint16_t, y) << 16);
}

// 8 fp8 E4M3 codes (two dwords) -> 8 bf16.  The widening is exact.
__device__ inline bf16x8 fp8x8_to_bf16(uint32_t w0, uint32_t w1) {
  const f32x2 a = __builtin_amdgcn_cvt_pk_f32_fp8(w0, false);
  const f32x2 b = __builtin_amdgcn_cvt_pk_f32_fp8(w0, true);
  const f32x2 c = __builtin_amdgcn_cvt_pk_f32_fp8(w1, false);
  const f32x2 d = __builtin_amdgcn_cvt_pk_f32_fp8(w1, true);
  const uint4 u = make_uint4(pack_bf16x2(a[0], a[1]), pack_bf16x2(b[0], b[1]), pack_bf16x2(c[0], c[1]),
                             pack_bf16x2(d[0], d[1]));
  return __builtin_bit_cast(bf16x8, u);
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

// Token of the 32-token tile that B-operand element e of lane group q holds:
// 4 q + e for e < 4 (first 16-token half), 16 + 4 q + e - 4 otherwise.
__device__ inline int tile_token(int q, int e) { return e < 4 ? 4 * q + e : 12 + 4 * q + e; }

// d layout of the A/B operands of S^T (the same for K and Q):
//   natural:  operand kb, lane group q, element e  ->  d = 32 kb + 8 q + e
//   fp8 HBM:  operand kb, lane group q, element e  ->  d = 64 (kb/2) + 16 q + 8 (kb%2) + e
// (one 16-byte fp8 load feeds two operands when K comes straight from HBM).
__device__ inline int q_offset(bool fp8_direct, int kb, int q) {
  return fp8_direct ? 64 * (kb >> 1) + 16 * q + 8 * (kb & 1) : 32 * kb + 8 * q;
}

// 16 chunks of 16 B per LDS token row, XOR-swizzled by the row so that the
// K reads (one chunk index over 16 rows) and V reads (16 chunks of one row)
// hit distinct banks.
__device__ inline int lds_off(int row, int chunk) { return row * kLdsRow + ((chunk ^ (row & 15)) << 4); }

template <bool FP8>
__device__ inline size_t head_off(int b, int Hkv, int kvh) {
  constexpr size_t kTileHead = (size_t)kBlock * (FP8 ? kHeadDim : 2 * kHeadDim);
  return ((size_t)b * Hkv + kvh) * kTileHead;
}

struct RowState {
  float m, l;  // reference max (log2 units) and per-lane running sum of exp2(s - m)
  f32x4 acc[8];
};

__device__ inline void row_init(RowState& st) {
  st.m = -INFINITY;
  st.l = 0.f;
#pragma unroll
  for (int r = 0; r < 8; ++r) st.acc[r] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// A row's reference max moves only when a score exceeds it by more than
// 2^kLazy; until then P stays <= 2^kLazy and the accumulators need no
// rescaling.  The result is the same softmax; only the reference differs.
constexpr float kLazy = 8.f;

__device__ inline void qk_mfma(const bf16x8 (&kf)[2][4], const bf16x8 (&qf)[4], f32x4& s0, f32x4& s1) {
  s0 = f32x4{0.f, 0.f, 0.f, 0.f};
  s1 = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kb = 0; kb < 4; ++kb) {
    s0 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[0][kb], qf[kb], s0, 0, 0, 0);
    s1 = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[1][kb], qf[kb], s1, 0, 0, 0);
  }
}

// Softmax update for one tile; returns P (scaled by the V scales) as bf16
// hi + lo.  lane (lq, lr): s0[e] is token t0 + 4 lq + e, s1[e] token
// t0 + 16 + 4 lq + e, of row lr.
__device__ inline void softmax_p(f32x4 s0, f32x4 s1, int t0, int ntok, int lq, float c0, float c1, float vs0,
                                 float vs1, RowState& st, bf16x8& ph, bf16x8& pl) {
  float sv[8];
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    sv[e] = s0[e] * c0;
    sv[4 + e] = s1[e] * c1;
  }
  if (t0 + 32 > ntok) {
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (t0 + tile_token(lq, e) >= ntok) sv[e] = -INFINITY;
  }
  float mx = sv[0];
#pragma unroll
  for (int e = 1; e < 8; ++e) mx = fmaxf(mx, sv[e]);
  // Move a row's reference only when one of its scores outgrows it by more
  // than 2^kLazy (always on the first tile, whose reference is -inf).  The
  // lane-local test needs no cross-lane traffic; only when some lane fails
  // it are the row maxima reduced over the row's four lanes.
  if (__builtin_amdgcn_ballot_w64(mx > st.m + kLazy)) {
    mx = wave_max_over_groups(mx);
    const bool move = mx > st.m + kLazy;
    const float m_new = move ? mx : st.m;
    const float alpha = exp2f(st.m - m_new);
    st.l *= alpha;
#pragma unroll
    for (int r = 0; r < 8; ++r) st.acc[r] *= alpha;
    st.m = m_new;
  }
  float psum = 0.f, hi[8], lo[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float p = exp2f(sv[e] - st.m);
    psum += p;
    const float pv = p * (e < 4 ? vs0 : vs1);
    hi[e] = (float)(__bf16)pv;  // exact in fp32
    lo[e] = pv - hi[e];
  }
  st.l += psum;
  ph = __builtin_bit_cast(bf16x8, make_uint4(pack_bf16x2(hi[0], hi[1]), pack_bf16x2(hi[2], hi[3]),
                                             pack_bf16x2(hi[4], hi[5]), pack_bf16x2(hi[6], hi[7])));
  pl = __builtin_bit_cast(bf16x8, make_uint4(pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]),
                                             pack_bf16x2(lo[4], lo[5]), pack_bf16x2(lo[6], lo[7])));
}

// V^T operands from the lane's 8 token rows (d-chunk lr of each): operand r
// holds d = 8 lr + r of the 8 tokens.  An 8 x 8 transpose of 16-bit values
// in 32 byte-selects: dword j of operand r pairs element r of rows 2 j and
// 2 j + 1 (low halves for even r, high halves for odd r).
__device__ inline void transpose_v(const uint4 (&vraw)[8], bf16x8 (&vf)[8]) {
  uint32_t w[8][4];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    w[e][0] = vraw[e].x;
    w[e][1] = vraw[e].y;
    w[e][2] = vraw[e].z;
    w[e][3] = vraw[e].w;
  }
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const uint32_t sel = (r & 1) ? 0x07060302u : 0x05040100u;
    uint32_t o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = __builtin_amdgcn_perm(w[2 * j + 1][r >> 1], w[2 * j][r >> 1], sel);
    vf[r] = __builtin_bit_cast(bf16x8, make_uint4(o[0], o[1], o[2], o[3]));
  }
}

__device__ inline void pv_mfma(const bf16x8 (&vf)[8], const bf16x8& ph, const bf16x8& pl, RowState& st) {
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    st.acc[r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[r], ph, st.acc[r], 0, 0, 0);
    st.acc[r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[r], pl, st.acc[r], 0, 0, 0);
  }
}

// Partials: lane (lq, lr) holds O[row lr][32 lq .. 32 lq + 31] with
// acc[r][e] at d = 32 lq + 8 e + r.
__device__ inline void write_partial(const DevPool& P, const AttnLaunch& A, const AttnUnit& U, int row0, int R,
                                     int lq, int lr, const RowState& st) {
  const float l = wave_sum_over_groups(st.l);
  const int r = row0 + lr;
  if (r >= R) return;
  const int g = P.g;
  const int pos = A.members[U.mem_off + r / g];
  const int h = U.kvh * g + r % g;
  const size_t idx = ((size_t)pos * P.Hq + h) * A.kmax + U.kidx;
  f32x4* dst = reinterpret_cast<f32x4*>(A.part_acc + idx * kHeadDim + 32 * lq);
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int e = k >> 1, rb = 4 * (k & 1);
    dst[k] = f32x4{st.acc[rb][e], st.acc[rb + 1][e], st.acc[rb + 2][e], st.acc[rb + 3][e]};
  }
  if (lq == 0) A.part_ml[idx] = float2{st.m, l};
}

// Q^T operand of the row block starting at row0: lane (lq, lr) holds row
// row0 + lr in the given d layout (zeros past the unit's rows).
__device__ inline void load_q(const DevPool& P, const AttnLaunch& A, const AttnUnit& U, int row0, int R, bool fp8_direct,
                              int lq, int lr, bf16x8 (&qf)[4]) {
  const int r = row0 + lr;
  if (r < R) {
    const int pos = A.members[U.mem_off + r / P.g];
    const int h = U.kvh * P.g + r % P.g;
    const uint16_t* qrow = A.q + ((size_t)pos * P.Hq + h) * kHeadDim;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) qf[kb] = *reinterpret_cast<const bf16x8*>(qrow + q_offset(fp8_direct, kb, lq));
  } else {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) qf[kb] = bf16x8{};
  }
}

// The unit's block ids (and fp8 scales) 64 at a time, one per lane, read
// back with readlane, so no tile waits on a table load.  Entries outside
// the pool are never dereferenced: they become block 0 and the device error
// word records them.
template <bool FP8>
struct BlockIds {
  const DevPool& P;
  const int32_t* brow;
  int nblk, lane, win;
  int cur_id, nxt_id;
  float cur_ks, cur_vs, nxt_ks, nxt_vs;

  __device__ BlockIds(const DevPool& P_, const int32_t* brow_, int nblk_, int lane_)
      : P(P_), brow(brow_), nblk(nblk_), lane(lane_), win(0) {
    fetch(0, cur_id, cur_ks, cur_vs);
    fetch(1, nxt_id, nxt_ks, nxt_vs);
  }
  __device__ void fetch(int w, int& id, float& ks, float& vs) {
    id = 0;
    ks = vs = 1.f;
    const int j = 64 * w + lane;
    if (j < nblk) {
      id = brow[j];
      if ((unsigned)id >= (unsigned)P.num_blocks) {
        atomicOr(P.err, kErrBadBlock);
        id = 0;
      }
      if constexpr (FP8) {
        ks = P.kv_scale[2 * id];
        vs = P.kv_scale[2 * id + 1];
      }
    }
  }
  // ids and scales of tile i (logical blocks 2 i and 2 i + 1; a missing
  // second block aliases the first, its tokens are masked).  Tiles are
  // visited in increasing order.
  __device__ void tile(int i, int& b0, int& b1, float& ks0, float& ks1, float& vs0, float& vs1) {
    const int j0 = 2 * i, j1 = 2 * i + 1 < nblk ? 2 * i + 1 : 2 * i;
    if ((j1 >> 6) > win + 1) {
      cur_id = nxt_id;
      cur_ks = nxt_ks;
      cur_vs = nxt_vs;
      ++win;
      fetch(win + 1, nxt_id, nxt_ks, nxt_vs);
    }
    const bool c0 = (j0 >> 6) == win, c1 = (j1 >> 6) == win;
    b0 = __builtin_amdgcn_readlane(c0 ? cur_id : nxt_id, j0 & 63);
    b1 = __builtin_amdgcn_readlane(c1 ? cur_id : nxt_id, j1 & 63);
    ks0 = ks1 = vs0 = vs1 = 1.f;
    if constexpr (FP8) {
      ks0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, c0 ? cur_ks : nxt_ks), j0 & 63));
      vs0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, c0 ? cur_vs : nxt_vs), j0 & 63));
      ks1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, c1 ? cur_ks : nxt_ks), j1 & 63));
      vs1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, c1 ? cur_vs : nxt_vs), j1 & 63));
    }
  }
};

struct TileMeta {
  int b0, b1;
  float ks0, ks1, vs0, vs1;
};

// ---------------------------------------------------------------- narrow --
// Raw operands of one 32-token tile, loaded straight from HBM.  bf16: K 2
// halves x 4 d-groups of 16 bytes, V 8 tokens x 16 bytes.  fp8: half the
// bytes (K in k[.][0..1], V in the low 8 bytes of each v[e]).
struct Tile {
  uint4 k[2][4];
  uint4 v[8];
};

template <bool FP8>
__device__ inline void load_k(const uint8_t* base0, const uint8_t* base1, int lq, int lr, Tile& t) {
  constexpr int RB = FP8 ? kHeadDim : 2 * kHeadDim;  // bytes of one token row of one head
#pragma unroll
  for (int hf = 0; hf < 2; ++hf) {  // lane (lq, lr) reads token lr of each half
    const uint8_t* row = (hf ? base1 : base0) + lr * RB;
    if constexpr (!FP8) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) t.k[hf][kb] = *reinterpret_cast<const uint4*>(row + 64 * kb + 16 * lq);
    } else {
#pragma unroll
      for (int i = 0; i < 2; ++i) t.k[hf][i] = *reinterpret_cast<const uint4*>(row + 64 * i + 16 * lq);
    }
  }
}

template <bool FP8>
__device__ inline void load_v(const uint8_t* base0, const uint8_t* base1, int lq, int lr, Tile& t) {
  constexpr int RB = FP8 ? kHeadDim : 2 * kHeadDim;
#pragma unroll
  for (int e = 0; e < 8; ++e) {  // lane (lq, lr) reads d-chunk lr of its 8 tokens
    const int tok = tile_token(lq, e);
    const uint8_t* row = (tok < 16 ? base0 : base1) + (tok & 15) * RB;
    if constexpr (!FP8) {
      t.v[e] = *reinterpret_cast<const uint4*>(row + 16 * lr);
    } else {
      const uint2 x = *reinterpret_cast<const uint2*>(row + 8 * lr);
      t.v[e] = make_uint4(x.x, x.y, 0, 0);
    }
  }
}

template <bool FP8>
__device__ inline void qk_direct(const Tile& t, const bf16x8 (&qf)[4], f32x4& s0, f32x4& s1) {
  bf16x8 kf[2][4];
#pragma unroll
  for (int hf = 0; hf < 2; ++hf) {
    if constexpr (!FP8) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) kf[hf][kb] = __builtin_bit_cast(bf16x8, t.k[hf][kb]);
    } else {
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        kf[hf][2 * i] = fp8x8_to_bf16(t.k[hf][i].x, t.k[hf][i].y);
        kf[hf][2 * i + 1] = fp8x8_to_bf16(t.k[hf][i].z, t.k[hf][i].w);
      }
    }
  }
  qk_mfma(kf, qf, s0, s1);
}

template <bool FP8>
__device__ inline void pv_direct(Tile& t, f32x4 s0, f32x4 s1, int t0, int ntok, int lq, const TileMeta& m,
                                 float sl, RowState& st) {
  bf16x8 ph, pl;
  softmax_p(s0, s1, t0, ntok, lq, sl * m.ks0, sl * m.ks1, m.vs0, m.vs1, st, ph, pl);
  // a token past the end reads as zero (its P is zero, but the slot may
  // hold stale bits)
  if (t0 + 32 > ntok) {
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (t0 + tile_token(lq, e) >= ntok) t.v[e] = make_uint4(0, 0, 0, 0);
  }
  uint4 vraw[8];
  bf16x8 vf[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    if constexpr (!FP8)
      vraw[e] = t.v[e];
    else
      vraw[e] = __builtin_bit_cast(uint4, fp8x8_to_bf16(t.v[e].x, t.v[e].y));
  }
  transpose_v(vraw, vf);
  pv_mfma(vf, ph, pl, st);
}

// One wave, one 16-row unit.  Tile j lives in register buffer j % 2.  Step
// i issues the QK product of tile i + 1 before the softmax and P.V of tile
// i, so the matrix cores and the vector ALUs overlap; a buffer's K half is
// refilled with tile j + 2 right after QK(j) and its V half right after
// P.V(j), so two tiles are always in flight.
template <bool FP8>
__device__ void narrow_unit(const DevPool& P, const AttnLaunch& A, const AttnUnit& U, int lane) {
  const int32_t* brow = P.table + (size_t)U.owner * P.max_blocks + U.jb0;
  const int ntok = U.nblk >= 0 ? U.nblk * kBlock : P.seq_len[U.owner] - U.jb0 * kBlock;
  if (ntok <= 0) return;
  const int R = U.mem_cnt * P.g;  // <= 16
  const int lq = lane >> 4, lr = lane & 15;
  const int nblk = (ntok + kBlock - 1) / kBlock;
  const int ntile = (ntok + 31) / 32;
  BlockIds<FP8> ids(P, brow, nblk, lane);
  bf16x8 qf[4];
  load_q(P, A, U, 0, R, FP8, lq, lr, qf);
  RowState st;
  row_init(st);
  const float sl = A.scale_log2;

  auto fetch_k = [&](const TileMeta& m, Tile& t) {
    load_k<FP8>(P.k_cache + head_off<FP8>(m.b0, P.Hkv, U.kvh), P.k_cache + head_off<FP8>(m.b1, P.Hkv, U.kvh), lq,
                lr, t);
  };
  auto fetch_v = [&](const TileMeta& m, Tile& t) {
    load_v<FP8>(P.v_cache + head_off<FP8>(m.b0, P.Hkv, U.kvh), P.v_cache + head_off<FP8>(m.b1, P.Hkv, U.kvh), lq,
                lr, t);
  };
  auto meta = [&](int i, TileMeta& m) { ids.tile(i, m.b0, m.b1, m.ks0, m.ks1, m.vs0, m.vs1); };
  Tile ta, tb;
  TileMeta ma{}, mb{}, na{}, nb{};  // current and next (tile + 2) metadata of buffers A and B
  meta(0, ma);
  fetch_k(ma, ta);
  fetch_v(ma, ta);
  if (ntile > 1) {
    meta(1, mb);
    fetch_k(mb, tb);
    fetch_v(mb, tb);
  }
  f32x4 s0, s1;
  qk_direct<FP8>(ta, qf, s0, s1);
  if (ntile > 2) {
    meta(2, na);
    fetch_k(na, ta);
  }
  auto step = [&](int i, Tile& t, TileMeta& m, TileMeta& n, Tile& to, TileMeta& no) {
    const f32x4 r0 = s0, r1 = s1;
    if (i + 1 < ntile) {
      qk_direct<FP8>(to, qf, s0, s1);
      if (i + 3 < ntile) {
        meta(i + 3, no);
        fetch_k(no, to);
      }
    }
    pv_direct<FP8>(t, r0, r1, 32 * i, ntok, lq, m, sl, st);
    if (i + 2 < ntile) {
      fetch_v(n, t);
      m = n;
    }
  };
  for (int i = 0; i < ntile; i += 2) {
    step(i, ta, ma, na, tb, nb);
    if (i + 1 < ntile) step(i + 1, tb, mb, nb, ta, na);
  }
  write_partial(P, A, U, 0, R, lq, lr, st);
}

// ----------------------------------------------------------- cooperative --
// Staging registers of one 32-token tile: each of the 256 threads moves two
// 16-byte chunks of K and two of V (bf16), or one of each (fp8).
struct Stage {
  uint4 k[2], v[2];
};

template <bool FP8>
__device__ inline void stage_load(const DevPool& P, int kvh, const TileMeta& m, int t0, int ntok, Stage& s) {
  const int t = threadIdx.x;
  if constexpr (!FP8) {
    // thread t moves chunk t & 15 of token t >> 4 of each 16-token half
    const int tok = t >> 4, ch = t & 15;
    const size_t in_blk = (size_t)tok * kLdsRow + ch * 16;
    const size_t o0 = head_off<false>(m.b0, P.Hkv, kvh) + in_blk;
    const size_t o1 = head_off<false>(m.b1, P.Hkv, kvh) + in_blk;
    const bool v0 = t0 + tok < ntok, v1 = t0 + 16 + tok < ntok;
    s.k[0] = v0 ? *reinterpret_cast<const uint4*>(P.k_cache + o0) : make_uint4(0, 0, 0, 0);
    s.v[0] = v0 ? *reinterpret_cast<const uint4*>(P.v_cache + o0) : make_uint4(0, 0, 0, 0);
    s.k[1] = v1 ? *reinterpret_cast<const uint4*>(P.k_cache + o1) : make_uint4(0, 0, 0, 0);
    s.v[1] = v1 ? *reinterpret_cast<const uint4*>(P.v_cache + o1) : make_uint4(0, 0, 0, 0);
  } else {
    const int tok = t >> 3, ch8 = t & 7;  // 32 tokens x 8 chunks of 16 fp8 codes
    if (t0 + tok < ntok) {
      const size_t off = head_off<true>(tok < 16 ? m.b0 : m.b1, P.Hkv, kvh) + (tok & 15) * kHeadDim + ch8 * 16;
      s.k[0] = *reinterpret_cast<const uint4*>(P.k_cache + off);
      s.v[0] = *reinterpret_cast<const uint4*>(P.v_cache + off);
    } else {
      s.k[0] = s.v[0] = make_uint4(0, 0, 0, 0);
    }
  }
}

template <bool FP8>
__device__ inline void stage_store(uint8_t* kl, uint8_t* vl, const Stage& s) {
  const int t = threadIdx.x;
  if constexpr (!FP8) {
    const int tok = t >> 4, ch = t & 15;
    *reinterpret_cast<uint4*>(kl + lds_off(tok, ch)) = s.k[0];
    *reinterpret_cast<uint4*>(vl + lds_off(tok, ch)) = s.v[0];
    *reinterpret_cast<uint4*>(kl + lds_off(16 + tok, ch)) = s.k[1];
    *reinterpret_cast<uint4*>(vl + lds_off(16 + tok, ch)) = s.v[1];
  } else {
    const int tok = t >> 3, ch8 = t & 7;
    const uint4 k0 = s.k[0], v0 = s.v[0];
    *reinterpret_cast<bf16x8*>(kl + lds_off(tok, 2 * ch8)) = fp8x8_to_bf16(k0.x, k0.y);
    *reinterpret_cast<bf16x8*>(kl + lds_off(tok, 2 * ch8 + 1)) = fp8x8_to_bf16(k0.z, k0.w);
    *reinterpret_cast<bf16x8*>(vl + lds_off(tok, 2 * ch8)) = fp8x8_to_bf16(v0.x, v0.y);
    *reinterpret_cast<bf16x8*>(vl + lds_off(tok, 2 * ch8 + 1)) = fp8x8_to_bf16(v0.z, v0.w);
  }
}

// One workgroup, one chunk, up to 4 row blocks: wave w owns row block w.
// Every wave takes part in every barrier.
template <bool FP8>
__device__ void coop_unit(const DevPool& P, const AttnLaunch& A, const AttnUnit& U, int wave, int lane,
                          uint8_t (&lds)[2][2][32 * kLdsRow]) {
  const int32_t* brow = P.table + (size_t)U.owner * P.max_blocks + U.jb0;
  const int ntok = U.nblk >= 0 ? U.nblk * kBlock : P.seq_len[U.owner] - U.jb0 * kBlock;
  if (ntok <= 0) return;  // uniform over the workgroup
  const int R = U.mem_cnt * P.g;  // <= 64
  const int lq = lane >> 4, lr = lane & 15;
  const int nblk = (ntok + kBlock - 1) / kBlock;
  const int ntile = (ntok + 31) / 32;
  const int row0 = 16 * wave;
  const bool active = row0 < R;
  BlockIds<FP8> ids(P, brow, nblk, lane);
  bf16x8 qf[4];
  load_q(P, A, U, row0, R, false, lq, lr, qf);
  RowState st;
  row_init(st);
  const float sl = A.scale_log2;

  TileMeta m{}, mn{};
  ids.tile(0, m.b0, m.b1, m.ks0, m.ks1, m.vs0, m.vs1);
  Stage stg;
  stage_load<FP8>(P, U.kvh, m, 0, ntok, stg);
  stage_store<FP8>(lds[0][0], lds[0][1], stg);
  __syncthreads();
  for (int i = 0; i < ntile; ++i) {
    const int buf = i & 1;
    const bool more = i + 1 < ntile;
    if (more) {
      ids.tile(i + 1, mn.b0, mn.b1, mn.ks0, mn.ks1, mn.vs0, mn.vs1);
      stage_load<FP8>(P, U.kvh, mn, 32 * (i + 1), ntok, stg);
    }
    if (active) {
      const uint8_t* kl = lds[buf][0];
      const uint8_t* vl = lds[buf][1];
      f32x4 s0, s1;
      {
        bf16x8 kf[2][4];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
            kf[hf][kb] = *reinterpret_cast<const bf16x8*>(kl + lds_off(16 * hf + lr, 4 * kb + lq));
        qk_mfma(kf, qf, s0, s1);
      }
      bf16x8 ph, pl;
      softmax_p(s0, s1, 32 * i, ntok, lq, sl * m.ks0, sl * m.ks1, m.vs0, m.vs1, st, ph, pl);
      uint4 vraw[8];
      bf16x8 vf[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) vraw[e] = *reinterpret_cast<const uint4*>(vl + lds_off(tile_token(lq, e), lr));
      transpose_v(vraw, vf);
      pv_mfma(vf, ph, pl, st);
    }
    if (more) {
      stage_store<FP8>(lds[buf ^ 1][0], lds[buf ^ 1][1], stg);
      m = mn;
    }
    __syncthreads();
  }
  if (active) write_partial(P, A, U, row0, R, lq, lr, st);
}

// Workgroups are dispatched round-robin over the 8 XCDs, so workgroup bid
// runs on XCD bid % 8.  The plan lists every XCD's workgroup slots
// contiguously, four entries per slot: a cooperative item (flagged in its
// first entry) or four narrow units.  Cooperative (compute-bound) and
// narrow (HBM-bound) slots are interleaved so both kinds share every CU.
template <bool FP8>
__global__ __launch_bounds__(kThreads, 2) void attn_units_kernel(DevPool P, AttnLaunch A) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[2][2][32 * kLdsRow];
  const int x = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int base = A.xcd_off[x] + 4 * slot, end = A.xcd_off[x + 1];
  if (base >= end) return;  // uniform over the workgroup
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const AttnUnit U0 = A.units[base];
  if (U0.flags & kUnitCoop) {
    if (U0.mem_cnt > 0) coop_unit<FP8>(P, A, U0, wave, lane, lds);
    return;
  }
  if (base + wave >= end) return;  // no barrier on the narrow path
  const AttnUnit U = A.units[base + wave];
  if (U.mem_cnt > 0) narrow_unit<FP8>(P, A, U, lane);
}

// Log-sum-exp merge of a row's partials.  One wave per (list position,
// query head): lane k < nk reads partial k's (max, sum), the wave reduces the
// maximum and the weighted sum, then every lane accumulates its two d values
// over the partials with the weights broadcast from their lanes.
__global__ __launch_bounds__(256) void merge_kernel(DevPool P, AttnLaunch A) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= A.n * P.Hq) return;
  const int lane = threadIdx.x & 63;
  const int pos = row / P.Hq;
  const int nk = A.nk[pos];  // <= kmax <= 64
  const float2* ml = A.part_ml + (size_t)row * A.kmax;
  const float* pa = A.part_acc + (size_t)row * A.kmax * kHeadDim;
  const float2 mine = lane < nk ? ml[lane] : float2{-INFINITY, 0.f};
  float M = mine.x;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));
  const float w = lane < nk ? exp2f(mine.x - M) : 0.f;
  float L = w * mine.y;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) L += __shfl_xor(L, off);
  float o0 = 0.f, o1 = 0.f;
  int k = 0;
  for (; k + 4 <= nk; k += 4) {
    float2 a[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) a[j] = *reinterpret_cast<const float2*>(pa + (size_t)(k + j) * kHeadDim + 2 * lane);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float wk = __shfl(w, k + j);
      o0 += wk * a[j].x;
      o1 += wk * a[j].y;
    }
  }
  for (; k < nk; ++k) {
    const float2 a = *reinterpret_cast<const float2*>(pa + (size_t)k * kHeadDim + 2 * lane);
    const float wk = __shfl(w, k);
    o0 += wk * a.x;
    o1 += wk * a.y;
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
