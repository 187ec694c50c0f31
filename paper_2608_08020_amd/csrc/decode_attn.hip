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
//  * narrow: four independent units, one per wave, of one row block (fp8:
//    up to two).  A wave streams its chunk 32 tokens at a time straight from
//    HBM into matrix-core operand registers, double-buffered, with no LDS
//    and no barrier (this is where most of the bytes are: chunks that 1-4
//    traces share).
//  * cooperative: one chunk with 2-8 row blocks (more rows become several
//    workgroups, placed on one XCD so their re-reads hit its L2).  The
//    workgroup streams 32-token tiles into a 4-stage LDS ring by direct
//    global-to-LDS loads, three tiles ahead, and each wave applies a tile to
//    its one or two row blocks, so a chunk is read once per up to eight row
//    blocks instead of once per row block.
//
// The launch also performs the decode step's append: the unit that covers
// a trace's last block writes the new token's K and V there (quantising
// bf16 input to E4M3FN for fp8 pools when asked), and enters a block the
// token opens - chosen by the host by the allocation rule and passed in the
// launch arguments - into the block table, refcounts and free set.  The
// merge kernel then advances the lengths.
//
// The contractions run on the bf16 matrix cores (v_mfma_f32_16x16x32_bf16):
//   S^T[token][row] = K[token][:] . Q[row][:]          (A = K, B = Q^T)
//   O^T[d][row]    += V^T[d][token] . P^T[token][row]   (A = V^T, B = P^T)
// Of a 32-token tile (blocks b0, b1), the first S^T product takes tokens
// 8 j + {0..3} and the second 8 j + {4..7} (j = 0..3) as its 16 A rows, so
// lane group q ends up holding, for its row, the scores of tokens 8 q .. 8 q
// + 7: exactly the B operand of the second product, and V^T's A operand is
// then 8 consecutive tokens of one d.  The cache tile layout (K in 16-byte
// d-chunks with token rows in k_phys order, V transposed) makes each
// operand one 16-byte load per lane and each load instruction a few whole
// 128-byte lines.  P is split into bf16 hi + lo parts (two MFMAs) so the P.V
// product keeps ~16 bits of P.  fp8 E4M3 K/V are widened to bf16 (exact); a
// block's K scale multiplies its scores and its V scale multiplies P.
#include <cmath>

#include "kernels.h"
#include "lds_dma.h"

namespace gambit {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;                      // four waves
constexpr int kTileBytes = kBlock * kHeadDim * 2;  // one bf16 (block, head) tile
// LDS stage of one 32-token tile, always bf16: K of the two blocks (the
// second shifted by 128 bytes, so the two 128-byte halves of a K read fall
// in different banks), then V^T of the two blocks stored as [token half
// (8 tokens)][d][16 bytes], so the lanes of a V read, which take 16
// consecutive d of one half, read contiguous bytes (no bank conflicts).
constexpr int kLdsK1 = kTileBytes + 128;
constexpr int kLdsV = kLdsK1 + kTileBytes;
constexpr int kStage = kLdsV + 2 * kTileBytes;

typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two floats -> two bf16 (round to nearest even) in one dword, a in the low half.
__device__ inline uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, bf16x2));
}

// fp8 E4M3 codes -> bf16 (exact: unit scale).  Code k of a dword becomes
// element k of the result.
__device__ inline uint2 fp8x4_to_bf16(uint32_t w) {
  const bf16x2 a = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.f, false);
  const bf16x2 b = __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.f, true);
  return make_uint2(__builtin_bit_cast(uint32_t, a), __builtin_bit_cast(uint32_t, b));
}

__device__ inline uint4 fp8x8_to_bf16(uint32_t w0, uint32_t w1) {
  const uint2 a = fp8x4_to_bf16(w0), b = fp8x4_to_bf16(w1);
  return make_uint4(a.x, a.y, b.x, b.y);
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

// d layout of the A/B operands of S^T (the same for K and Q):
//   natural:  operand kb, lane group q, element e  ->  d = 32 kb + 8 q + e
//   fp8 HBM:  operand kb, lane group q, element e  ->  d = 64 (kb/2) + 16 q + 8 (kb%2) + e
// (one 16-byte fp8 load feeds two operands when K comes straight from HBM).
__device__ inline int q_offset(bool fp8_direct, int kb, int q) {
  return fp8_direct ? 64 * (kb >> 1) + 16 * q + 8 * (kb & 1) : 32 * kb + 8 * q;
}

template <bool FP8>
__device__ inline size_t head_off(int b, int Hkv, int kvh) {
  constexpr size_t kTileHead = (size_t)kBlock * (FP8 ? kHeadDim : 2 * kHeadDim);
  return ((size_t)b * Hkv + kvh) * kTileHead;
}

// Keep the first nv of 8 bf16 values (two per dword).
__device__ inline uint4 keep_first(uint4 x, int nv) {
  x.x &= nv >= 2 ? 0xffffffffu : (nv == 1 ? 0xffffu : 0u);
  x.y &= nv >= 4 ? 0xffffffffu : (nv == 3 ? 0xffffu : 0u);
  x.z &= nv >= 6 ? 0xffffffffu : (nv == 5 ? 0xffffu : 0u);
  x.w &= nv >= 8 ? 0xffffffffu : (nv == 7 ? 0xffffu : 0u);
  return x;
}

// Keep the first n of the four fp8 codes of a dword.
__device__ inline uint32_t keep_bytes(uint32_t w, int n) {
  return n >= 4 ? w : (n <= 0 ? 0u : w & ((1u << (8 * n)) - 1u));
}

// The narrow path's KV reads are streaming: each byte is read once per
// launch by one wave and the working set is far larger than L2 and the
// memory-side cache, so they carry the non-temporal hint (on gfx950 a plain
// read stream sustains ~6.4 TB/s without it and ~7.2 TB/s with it).  The
// cooperative path keeps the default policy: items that split one chunk's
// rows re-read it and should find it in L2 (measured: the hint there costs
// more than it saves, even for chunks no other item reads).
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

__device__ inline uint4 ld_stream16(const uint8_t* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ inline uint2 ld_stream8(const uint8_t* p) {
  const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
  return make_uint2(v.x, v.y);
}

// A zero the compiler cannot see through (keeps loads that use it where
// they are written).
__device__ inline int opaque_zero() {
  int z;
  asm volatile("v_mov_b32 %0, 0" : "=v"(z));
  return z;
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

// Softmax update for one tile.  Lane (q, row): s0[e] and s1[e] are the raw
// scores of tokens 8 q + e and 8 q + 4 + e; c = softmax scale x log2(e) x the
// block's K scale; the first nv of the lane's 8 tokens exist when `partial`.
// Returns P (times the block's V scale for fp8) as bf16 hi + lo.
template <bool FP8>
__device__ inline void softmax_p(const f32x4& s0, const f32x4& s1, bool partial, int nv, float c, float vsc,
                                 RowState& st, bf16x8& ph, bf16x8& pl) {
  float sv[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
  if (partial) {
    // Only a chunk's last tile is partial; the empty asm keeps this a branch
    // (if-converted, the selects would run on every tile).
    asm volatile("");
#pragma unroll
    for (int e = 0; e < 8; ++e) sv[e] = e < nv ? sv[e] : -INFINITY;
  }
  float mx = fmaxf(fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3])), fmaxf(fmaxf(sv[4], sv[5]), fmaxf(sv[6], sv[7])));
  mx *= c;  // c > 0
  // Move a row's reference only when one of its scores outgrows it by more
  // than 2^kLazy (always on the first tile, whose reference is -inf).  The
  // lane-local test needs no cross-lane traffic; only when some lane fails
  // it are the row maxima reduced over the row's four lanes.
  if (__builtin_amdgcn_ballot_w64(mx > st.m + kLazy)) {
    mx = wave_max_over_groups(mx);
    const float m_new = mx > st.m + kLazy ? mx : st.m;
    const float alpha = __builtin_amdgcn_exp2f(st.m - m_new);
    st.l *= alpha;
#pragma unroll
    for (int r = 0; r < 8; ++r) st.acc[r] *= alpha;
    st.m = m_new;
  }
  const float nm = -st.m;
  float p[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) p[e] = __builtin_amdgcn_exp2f(fmaf(sv[e], c, nm));
  st.l += ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7]));
  uint32_t hw[4], lw[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    float a = p[2 * j], b = p[2 * j + 1];
    if constexpr (FP8) {
      a *= vsc;
      b *= vsc;
    }
    hw[j] = pack_bf16x2(a, b);
    const float ah = __builtin_bit_cast(float, hw[j] << 16);
    const float bh = __builtin_bit_cast(float, hw[j] & 0xffff0000u);
    lw[j] = pack_bf16x2(a - ah, b - bh);  // both differences are exact in fp32
  }
  ph = __builtin_bit_cast(bf16x8, make_uint4(hw[0], hw[1], hw[2], hw[3]));
  pl = __builtin_bit_cast(bf16x8, make_uint4(lw[0], lw[1], lw[2], lw[3]));
}

__device__ inline void pv_mfma(const bf16x8 (&vf)[8], const bf16x8& ph, const bf16x8& pl, RowState& st) {
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    st.acc[r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[r], ph, st.acc[r], 0, 0, 0);
    st.acc[r] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf[r], pl, st.acc[r], 0, 0, 0);
  }
}

// Partials: lane (q, lr) holds O[row lr][16 r + 4 q + e] in acc[r][e].
__device__ inline void write_partial(const DevPool& P, const AttnLaunch& A, const AttnUnit& U, int row0, int R,
                                     int q, int lr, const RowState& st) {
  const float l = wave_sum_over_groups(st.l);
  const int r = row0 + lr;
  if (r >= R) return;
  const int g = P.g;
  const int pos = A.members[U.mem_off + r / g];
  const int h = U.kvh * g + r % g;
  const size_t idx = ((size_t)pos * P.Hq + h) * A.kmax + U.kidx;
  f32x4* dst = reinterpret_cast<f32x4*>(A.part_acc + idx * kHeadDim + 4 * q);
#pragma unroll
  for (int k = 0; k < 8; ++k) __builtin_nontemporal_store(st.acc[k], dst + 4 * k);  // read once, by the merge
  if (q == 0) A.part_ml[idx] = float2{st.m, l};
}

// Q^T operand of the row block starting at row0: lane (q, lr) holds row
// row0 + lr in the given d layout (zeros past the unit's rows).
__device__ inline void load_q(const DevPool& P, const AttnLaunch& A, const AttnUnit& U, int row0, int R, bool fp8_direct,
                              int q, int lr, bf16x8 (&qf)[4]) {
  const int r = row0 + lr;
  if (r < R) {
    const int pos = A.members[U.mem_off + r / P.g];
    const int h = U.kvh * P.g + r % P.g;
    const uint16_t* qrow = A.q + ((size_t)pos * P.Hq + h) * kHeadDim;
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) qf[kb] = *reinterpret_cast<const bf16x8*>(qrow + q_offset(fp8_direct, kb, q));
  } else {
#pragma unroll
    for (int kb = 0; kb < 4; ++kb) qf[kb] = bf16x8{};
  }
}

// The unit's block ids (and fp8 scales) 64 at a time, one per lane, read
// back with readlane.  Window w + 1 is fetched when the tiles enter window
// w, so a tile never waits on a table load.  Entries outside the pool are
// never dereferenced: they become block 0 and the device error word records
// them (bf16 checks the id when a tile takes it; fp8 when the window is
// fetched, before its scales are read).
template <bool FP8>
struct BlockIds {
  const DevPool& P;
  const int32_t* brow;
  int nblk, lane, win;
  int fresh_j, fresh_id;  // a block this launch opened (its table entry is not read back)
  float fresh_scale;
  int cur_id, nxt_id;
  float cur_ks, cur_vs, nxt_ks, nxt_vs;

  __device__ BlockIds(const DevPool& P_, const int32_t* brow_, int nblk_, int lane_, int fresh_j_ = -1,
                      int fresh_id_ = 0, float fresh_scale_ = 1.f)
      : P(P_), brow(brow_), nblk(nblk_), lane(lane_), win(0), fresh_j(fresh_j_), fresh_id(fresh_id_),
        fresh_scale(fresh_scale_) {
    fetch(0, cur_id, cur_ks, cur_vs);
    fetch(1, nxt_id, nxt_ks, nxt_vs);
  }
  // Lanes past the unit's last block re-read its last entry (never used);
  // the unconditional load lets the id land in place without a copy.
  __device__ void fetch(int w, int& id, float& ks, float& vs) {
    const int j = min(64 * w + lane, nblk - 1);
    id = brow[j];
    ks = vs = 1.f;
    if (j == fresh_j) {
      id = fresh_id;
      ks = vs = fresh_scale;
      return;
    }
    if constexpr (FP8) {
      if ((unsigned)id >= (unsigned)P.num_blocks) {
        atomicOr(P.err, kErrBadBlock);
        id = 0;
      }
      ks = P.kv_scale[2 * id];
      vs = P.kv_scale[2 * id + 1];
    }
  }
  __device__ int checked(int b) {
    if constexpr (!FP8) {
      if ((unsigned)b >= (unsigned)P.num_blocks) {
        if (lane == 0) atomicOr(P.err, kErrBadBlock);
        b = 0;
      }
    }
    return b;
  }
  // ids and scales of tile i (logical blocks 2 i and 2 i + 1, both in one
  // window; a missing second block aliases the first, its tokens are
  // masked).  Tiles are visited in increasing order.
  __device__ void tile(int i, int& b0, int& b1, float& ks0, float& ks1, float& vs0, float& vs1) {
    const int j0 = 2 * i, j1 = 2 * i + 1 < nblk ? 2 * i + 1 : 2 * i;
    if ((j0 >> 6) > win) {
      cur_id = nxt_id;
      cur_ks = nxt_ks;
      cur_vs = nxt_vs;
      ++win;
      fetch(win + 1, nxt_id, nxt_ks, nxt_vs);
    }
    b0 = checked(__builtin_amdgcn_readlane(cur_id, j0 & 63));
    b1 = checked(__builtin_amdgcn_readlane(cur_id, j1 & 63));
    ks0 = ks1 = vs0 = vs1 = 1.f;
    if constexpr (FP8) {
      ks0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, cur_ks), j0 & 63));
      vs0 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, cur_vs), j0 & 63));
      ks1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, cur_ks), j1 & 63));
      vs1 = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, cur_vs), j1 & 63));
    }
  }
};

struct TileMeta {
  int b0, b1;
  float ks0, ks1, vs0, vs1;
};

// Per-lane constants of one 32-token tile.  Lane (q, i): K operands read A
// row i (block i / 8, token row k_phys order 8 h + i % 8 of half h), d-chunk
// 4 kb + q; V^T operands read d = 16 r + lr, tokens 8 q .. 8 q + 7 (block
// q / 2).
struct LaneGeom {
  int q, lr;
  bool kb1, vb1;  // K / V operands of this lane come from the tile's second block
};

__device__ inline LaneGeom lane_geom(int lane) {
  LaneGeom g;
  g.q = lane >> 4;
  g.lr = lane & 15;
  g.kb1 = (lane & 8) != 0;
  g.vb1 = (g.q & 2) != 0;
  return g;
}

// Scale of the scores / of P for the lane's 8 tokens (all in one block).
__device__ inline void lane_scales(const LaneGeom& g, const TileMeta& m, float sl, float& c, float& vsc) {
  c = sl * (g.vb1 ? m.ks1 : m.ks0);
  vsc = g.vb1 ? m.vs1 : m.vs0;
}

// ---------------------------------------------------------------- narrow --
// Raw operands of one 32-token tile, loaded straight from HBM.  bf16: K 2
// halves x 4 d-groups of 16 bytes, V^T 8 operands of 16 bytes.  fp8: half
// the bytes (a 16-byte K load feeds two operands).
template <bool FP8>
struct Tile;
template <>
struct Tile<false> {
  uint4 k[2][4];
  uint4 v[8];
};
template <>
struct Tile<true> {
  uint4 k[2][2];
  uint2 v[8];
};

template <bool FP8>
__device__ inline void load_k(const uint8_t* kc0, const uint8_t* kc1, const LaneGeom& g, int lane, Tile<FP8>& t) {
  const uint8_t* base = (g.kb1 ? kc1 : kc0) + g.q * 256 + (lane & 7) * 16;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
#pragma unroll
    for (int j = 0; j < (FP8 ? 2 : 4); ++j) t.k[h][j] = ld_stream16(base + j * 1024 + h * 128);
  }
}

template <bool FP8>
__device__ inline void load_v(const uint8_t* vc0, const uint8_t* vc1, const LaneGeom& g, Tile<FP8>& t) {
  if constexpr (!FP8) {
    const uint8_t* base = (g.vb1 ? vc1 : vc0) + g.lr * 32 + (g.q & 1) * 16;
#pragma unroll
    for (int r = 0; r < 8; ++r) t.v[r] = ld_stream16(base + r * 512);
  } else {
    const uint8_t* base = (g.vb1 ? vc1 : vc0) + g.lr * 16 + (g.q & 1) * 8;
#pragma unroll
    for (int r = 0; r < 8; ++r) t.v[r] = ld_stream8(base + r * 256);
  }
}

// Scores of one tile for RB row blocks: every K operand feeds all of them.
// fp8 operands are widened two at a time right before their products (the
// products accumulate in the same order as qk_mfma's), which keeps few
// widened operands live.
template <bool FP8, int RB>
__device__ inline void qk_direct(const Tile<FP8>& t, const bf16x8 (&qf)[RB][4], f32x4 (&s0)[RB], f32x4 (&s1)[RB]) {
  if constexpr (!FP8) {
    bf16x8 kf[2][4];
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) kf[h][kb] = __builtin_bit_cast(bf16x8, t.k[h][kb]);
#pragma unroll
    for (int r = 0; r < RB; ++r) qk_mfma(kf, qf[r], s0[r], s1[r]);
  } else {
#pragma unroll
    for (int r = 0; r < RB; ++r) s0[r] = s1[r] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const bf16x8 a = __builtin_bit_cast(bf16x8, fp8x8_to_bf16(t.k[h][j].x, t.k[h][j].y));
        const bf16x8 b = __builtin_bit_cast(bf16x8, fp8x8_to_bf16(t.k[h][j].z, t.k[h][j].w));
#pragma unroll
        for (int r = 0; r < RB; ++r) {
          f32x4& acc = h ? s1[r] : s0[r];
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qf[r][2 * j], acc, 0, 0, 0);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b, qf[r][2 * j + 1], acc, 0, 0, 0);
        }
      }
    }
  }
}

template <bool FP8, int RB>
__device__ inline void pv_direct(Tile<FP8>& t, const f32x4 (&s0)[RB], const f32x4 (&s1)[RB], int t0, int ntok,
                                 const LaneGeom& g, const TileMeta& m, float sl, RowState (&st)[RB]) {
  const bool partial = t0 + 32 > ntok;
  const int nv = min(max(ntok - t0 - 8 * g.q, 0), 8);
  float c, vsc;
  lane_scales(g, m, sl, c, vsc);
  bf16x8 ph[RB], pl[RB];
#pragma unroll
  for (int r = 0; r < RB; ++r) softmax_p<FP8>(s0[r], s1[r], partial, nv, c, vsc, st[r], ph[r], pl[r]);
  // A token past the end reads as zero (its P is zero, but the slot may
  // hold stale bits).  Masked in place, so the common path copies nothing.
  if (partial) {
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      if constexpr (!FP8)
        t.v[r] = keep_first(t.v[r], nv);
      else
        t.v[r] = make_uint2(keep_bytes(t.v[r].x, nv), keep_bytes(t.v[r].y, nv - 4));
    }
  }
  // each V operand (widened from fp8 right before use) feeds every row block
#pragma unroll
  for (int d = 0; d < 8; ++d) {
    bf16x8 vf;
    if constexpr (!FP8)
      vf = __builtin_bit_cast(bf16x8, t.v[d]);
    else
      vf = __builtin_bit_cast(bf16x8, fp8x8_to_bf16(t.v[d].x, t.v[d].y));
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      st[r].acc[d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, ph[r], st[r].acc[d], 0, 0, 0);
      st[r].acc[d] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pl[r], st[r].acc[d], 0, 0, 0);
    }
  }
}

// The decode step's append, for one KV head: the unit whose end is read at
// run time covers its trace's last block, so it writes the new token there;
// the unit waits for the stores before its first tile load.  Only this wave
// touches this (block, head) tile in the launch.  len is the trace's length
// including the new token.  When the token opens a block, the block comes
// from the launch's list (the host took it by the allocation rule); the KV
// head 0 unit enters it in the table, refcount, free set (and fp8 scales),
// and every head's unit uses the id directly.  Returns that block, or -1.
// OCP E4M3FN code of a finite fp32 value: the nearest of the format's values
// (ties to an even mantissa), magnitudes from 448 up saturating to 448.
// Normal results: round the fp32 significand to 3 bits at bit 20 (round to
// nearest even), then move the exponent bias from 127 to 7; a carry out of
// the mantissa steps the exponent, which is the correct next value.  Below
// 2^-6 the codes are the multiples of 2^-9, so the code is |y| * 512 rounded
// to the nearest even integer (8 becomes the smallest normal, code 8).
__device__ inline uint32_t e4m3fn_code(float y) {
  const uint32_t u = __float_as_uint(y);
  const uint32_t sign = (u >> 24) & 0x80u;
  const float a = fabsf(y);
  uint32_t c;
  if (a >= 448.f) {
    c = 0x7Eu;
  } else if (a < 0.015625f) {
    c = (uint32_t)__builtin_rintf(a * 512.f);
  } else {
    const uint32_t m = u & 0x7FFFFFFFu;
    c = ((m + 0x7FFFFu + ((m >> 20) & 1u)) >> 20) - ((127u - 7u) << 3);
  }
  return sign | c;
}

__device__ inline int fresh_block(const AttnLaunch& A, int pos) {
  int lo = 0, hi = A.n_new;  // new_pos is ascending
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (A.new_pos[mid] < pos)
      lo = mid + 1;
    else
      hi = mid;
  }
  return lo < A.n_new && A.new_pos[lo] == pos ? A.new_blk[lo] : -1;
}

template <bool FP8>
__device__ inline int append_token(const DevPool& P, const AttnLaunch& A, const AttnUnit& U, int lane, int len) {
  constexpr int es = FP8 ? 1 : 2;
  const int tpos = len - 1;
  const int pos = A.members[U.mem_off];
  int b, fresh = -1;
  if (A.len_bias && (tpos & 15) == 0) {
    b = fresh = fresh_block(A, pos);
    if ((unsigned)b < (unsigned)P.num_blocks && U.kvh == 0 && lane == 0) {
      if (A.claim) {
        P.table[(size_t)U.owner * P.max_blocks + (tpos >> 4)] = b;
        P.refcount[b] = 1;
        atomicAnd(&P.freebits[b >> 5], ~(1u << (b & 31)));
      }
      if (P.kv_scale) {
        P.kv_scale[2 * b] = A.new_scale;
        P.kv_scale[2 * b + 1] = A.new_scale;
      }
    }
  } else {
    b = P.table[(size_t)U.owner * P.max_blocks + (tpos >> 4)];
  }
  if ((unsigned)b >= (unsigned)P.num_blocks) {
    if (lane == 0) atomicOr(P.err, kErrBadBlock);
    return -1;
  }
  const int row = tpos & 15;
  const size_t tile = head_off<FP8>(b, P.Hkv, U.kvh);
  if constexpr (FP8) {
    if (A.new_bf16) {  // quantise on append with the landing block's scales
      const float sk = fresh >= 0 ? A.new_scale : P.kv_scale[2 * b];
      const float sv = fresh >= 0 ? A.new_scale : P.kv_scale[2 * b + 1];
      const size_t src = ((size_t)pos * P.Hkv + U.kvh) * kHeadDim + 2 * lane;  // bf16 elements
      const uint32_t kk = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint16_t*>(A.k_new) + src);
      const uint32_t vv = *reinterpret_cast<const uint32_t*>(reinterpret_cast<const uint16_t*>(A.v_new) + src);
      const uint32_t k0 = e4m3fn_code(__uint_as_float(kk << 16) / sk);
      const uint32_t k1 = e4m3fn_code(__uint_as_float(kk & 0xFFFF0000u) / sk);
      const uint32_t v0 = e4m3fn_code(__uint_as_float(vv << 16) / sv);
      const uint32_t v1 = e4m3fn_code(__uint_as_float(vv & 0xFFFF0000u) / sv);
      const int d = 2 * lane;  // elements d, d + 1 of one 16-byte K chunk
      *reinterpret_cast<uint16_t*>(P.k_cache + tile + ((size_t)(d >> 4) * kBlock + k_phys(row)) * 16 + (d & 15)) =
          (uint16_t)(k0 | (k1 << 8));
      P.v_cache[tile + (size_t)d * kBlock + row] = (uint8_t)v0;
      P.v_cache[tile + (size_t)(d + 1) * kBlock + row] = (uint8_t)v1;
      return fresh;
    }
  }
  const size_t src = ((size_t)pos * P.Hkv + U.kvh) * kHeadDim * es;
  if (lane < kHeadDim * es / 16)  // K: 16-byte d-chunks at token row k_phys(row)
    *reinterpret_cast<uint4*>(P.k_cache + tile + ((size_t)lane * kBlock + k_phys(row)) * 16) =
        *reinterpret_cast<const uint4*>(A.k_new + src + lane * 16);
#pragma unroll
  for (int e = 0; e < 2; ++e) {  // V transposed: element d at d * 16 + row
    const int d = 2 * lane + e;
    if constexpr (FP8)
      P.v_cache[tile + (size_t)d * kBlock + row] = A.v_new[src + d];
    else
      *reinterpret_cast<uint16_t*>(P.v_cache + tile + ((size_t)d * kBlock + row) * 2) =
          reinterpret_cast<const uint16_t*>(A.v_new + src)[d];
  }
  return fresh;
}

// One wave, one unit of up to 16 RB rows (RB row blocks; each K and V
// operand loaded from HBM feeds all of them).  Tile j lives in register
// buffer j % 2.  Step i issues the QK product of tile i + 1 before the
// softmax and P.V of tile i, so the matrix cores and the vector ALUs
// overlap; a buffer's K half is refilled with tile j + 2 right after QK(j)
// and its V half right after P.V(j), so two tiles are always in flight.
template <bool FP8, int RB>
__device__ void narrow_unit(const DevPool& P, const AttnLaunch& A, const AttnUnit& U, int lane, uint8_t* qlds) {
  const int32_t* brow = P.table + (size_t)U.owner * P.max_blocks + U.jb0;
  const int len = U.nblk >= 0 ? 0 : P.seq_len[U.owner] + A.len_bias;
  const int ntok = U.nblk >= 0 ? U.nblk * kBlock : len - U.jb0 * kBlock;
  if (ntok <= 0) return;
  const int fresh = U.nblk < 0 ? append_token<FP8>(P, A, U, lane, len) : -1;
  const int R = U.mem_cnt * P.g;  // <= 16 RB
  const LaneGeom g = lane_geom(lane);
  const int nblk = (ntok + kBlock - 1) / kBlock;
  const int ntile = (ntok + 31) / 32;
  BlockIds<FP8> ids(P, brow, nblk, lane, fresh >= 0 ? nblk - 1 : -1, fresh, A.new_scale);
  // One row block keeps its Q operands in registers; two keep them in this
  // wave's LDS region (a narrow workgroup uses no other LDS) and read them
  // back for every tile, which leaves the registers to the two running
  // states and the tiles in flight.
  bf16x8 qf[1][4];
  RowState st[RB];
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    load_q(P, A, U, 16 * r, R, FP8, g.q, g.lr, qf[0]);
    if constexpr (RB > 1) {
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
        *reinterpret_cast<bf16x8*>(qlds + (4 * r + kb) * 1024 + lane * 16) = qf[0][kb];
    }
    row_init(st[r]);
  }
  auto scores = [&](const Tile<FP8>& t, f32x4 (&s0)[RB], f32x4 (&s1)[RB]) {
    if constexpr (RB == 1) {
      qk_direct<FP8, 1>(t, qf, s0, s1);
    } else {
      // the offset is an opaque zero, so the reads stay in the loop
      const uint8_t* qb = qlds + lane * 16 + opaque_zero();
      bf16x8 qq[RB][4];
#pragma unroll
      for (int r = 0; r < RB; ++r)
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) qq[r][kb] = *reinterpret_cast<const bf16x8*>(qb + (4 * r + kb) * 1024);
      qk_direct<FP8, RB>(t, qq, s0, s1);
    }
  };
  const float sl = A.scale_log2;

  auto fetch_k = [&](const TileMeta& m, Tile<FP8>& t) {
    load_k<FP8>(P.k_cache + head_off<FP8>(m.b0, P.Hkv, U.kvh), P.k_cache + head_off<FP8>(m.b1, P.Hkv, U.kvh), g,
                lane, t);
  };
  auto fetch_v = [&](const TileMeta& m, Tile<FP8>& t) {
    load_v<FP8>(P.v_cache + head_off<FP8>(m.b0, P.Hkv, U.kvh), P.v_cache + head_off<FP8>(m.b1, P.Hkv, U.kvh), g, t);
  };
  auto meta = [&](int i, TileMeta& m) { ids.tile(i, m.b0, m.b1, m.ks0, m.ks1, m.vs0, m.vs1); };
  Tile<FP8> ta, tb;
  TileMeta ma{}, mb{}, na{}, nb{};  // current and next (tile + 2) metadata of buffers A and B
  if (U.nblk < 0) __builtin_amdgcn_s_waitcnt(0);  // the appended token is in the cache
  meta(0, ma);
  fetch_k(ma, ta);
  fetch_v(ma, ta);
  if (ntile > 1) {
    meta(1, mb);
    fetch_k(mb, tb);
    fetch_v(mb, tb);
  }
  f32x4 s0[RB], s1[RB];
  scores(ta, s0, s1);
  if (ntile > 2) {
    meta(2, na);
    fetch_k(na, ta);
  }
  auto step = [&](int i, Tile<FP8>& t, TileMeta& m, TileMeta& n, Tile<FP8>& to, TileMeta& no) {
    f32x4 r0[RB], r1[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) {
      r0[r] = s0[r];
      r1[r] = s1[r];
    }
    if (i + 1 < ntile) {
      scores(to, s0, s1);
      if (i + 3 < ntile) {
        meta(i + 3, no);
        fetch_k(no, to);
      }
    }
    pv_direct<FP8, RB>(t, r0, r1, 32 * i, ntok, g, m, sl, st);
    if (i + 2 < ntile) {
      fetch_v(n, t);
      m = n;
    }
  };
  for (int i = 0; i < ntile; i += 2) {
    step(i, ta, ma, na, tb, nb);
    if (i + 1 < ntile) step(i + 1, tb, mb, nb, ta, na);
  }
#pragma unroll
  for (int r = 0; r < RB; ++r) write_partial(P, A, U, 16 * r, R, g.q, g.lr, st[r]);
}

// ----------------------------------------------------------- cooperative --
__device__ inline int lds_v(int blk, int d, int half) { return kLdsV + blk * kTileBytes + half * 2048 + d * 16; }

// bf16 tiles reach LDS by direct global->LDS loads (no registers): a ring of
// kRing stages with kAhead tiles in flight, so a workgroup waits for a
// tile's L2/HBM round trip only once per kAhead tiles.
constexpr int kRing = 4;
constexpr int kAhead = 3;
constexpr int kDmaPerTile = 4;  // 16-byte loads per thread per tile

// Direct global->LDS loads (dma16, dma4) come from lds_dma.h; completion is
// waited for explicitly (wait_tiles).
constexpr int kIdsBytes = 2 * 64 * 4;  // two windows of 64 block ids

// fp8 stage: the raw tiles (K of both blocks, then V^T of both, 2 KiB each,
// in the cache's own layout) and the tile's block scales (K0, V0, K1, V1,
// repeated over 256 bytes).  The second block's K starts 128 bytes later, so
// the two 128-byte halves of a K read (one per block) fall in different
// banks.  Half the bytes of a bf16 tile, so the ring is deeper for the same
// bytes in flight.
constexpr int kK1_8 = 2048 + 128;       // second block's K
constexpr int kV8 = kK1_8 + 2048;       // V^T of both blocks
constexpr int kMeta8 = kV8 + 2 * 2048;  // block scales
constexpr int kStage8 = kMeta8 + 256;
constexpr int kRing8 = 7;
constexpr int kAhead8 = 6;
static_assert(kAhead8 < kRing8 && kAhead8 <= 6, "ring depth and the waits' range");

// Waits until at most `later` tiles' direct loads of this wave are still in
// flight (loads retire in issue order).
__device__ inline void wait_tiles(int later) {
  // s_waitcnt immediate: vmcnt in bits 3:0, expcnt 6:4 and lgkmcnt 11:8 at
  // their maxima (no wait).
  if (later >= 2)
    __builtin_amdgcn_s_waitcnt(0x0F70 | (2 * kDmaPerTile));
  else if (later == 1)
    __builtin_amdgcn_s_waitcnt(0x0F70 | kDmaPerTile);
  else
    __builtin_amdgcn_s_waitcnt(0x0F70);
}

// The same for PER direct loads per tile and up to 5 later tiles.
template <int PER>
__device__ inline void wait_tiles_per(int later) {
  static_assert(5 * PER <= 15, "vmcnt immediate");
  switch (later) {
    case 0: __builtin_amdgcn_s_waitcnt(0x0F70); break;
    case 1: __builtin_amdgcn_s_waitcnt(0x0F70 | PER); break;
    case 2: __builtin_amdgcn_s_waitcnt(0x0F70 | (2 * PER)); break;
    case 3: __builtin_amdgcn_s_waitcnt(0x0F70 | (3 * PER)); break;
    case 4: __builtin_amdgcn_s_waitcnt(0x0F70 | (4 * PER)); break;
    default: __builtin_amdgcn_s_waitcnt(0x0F70 | (5 * PER)); break;
  }
}

// One workgroup, one chunk, up to 4 x RB row blocks: wave w owns row
// blocks RB w .. RB w + RB - 1, so each K/V operand a wave reads from LDS
// feeds RB row blocks (and RB independent chains of products overlap in
// the wave).  Every wave takes part in every barrier.
//
// Tiles reach LDS by direct global-to-LDS loads in a ring of `ring` stages
// with `ahead` tiles in flight.  bf16 stages hold the layout above; fp8
// stages hold the raw tiles in the cache's layout, and every wave widens
// the operands it reads (as the narrow path does from HBM), so an fp8 tile
// moves half the bytes and the ring is deeper.
template <bool FP8, int RB>
__device__ void coop_unit(const DevPool& P, const AttnLaunch& A, const AttnUnit& U, int wave, int lane,
                          uint8_t* lds) {
  constexpr int ring = FP8 ? kRing8 : kRing, ahead = FP8 ? kAhead8 : kAhead;
  constexpr int stage = FP8 ? kStage8 : kStage;
  const int32_t* brow = P.table + (size_t)U.owner * P.max_blocks + U.jb0;
  // a cooperative item is a shared run: its end is in the plan
  const int ntok = U.nblk >= 0 ? U.nblk * kBlock : P.seq_len[U.owner] + A.len_bias - U.jb0 * kBlock;
  if (ntok <= 0) return;  // uniform over the workgroup
  const int R = U.mem_cnt * P.g;  // <= 64 RB
  const LaneGeom g = lane_geom(lane);
  const int nblk = (ntok + kBlock - 1) / kBlock;
  const int ntile = (ntok + 31) / 32;
  const int row0 = 16 * RB * wave;
  const bool active = row0 < R;
  bf16x8 qf[RB][4];
  RowState st[RB];
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    load_q(P, A, U, row0 + 16 * r, R, FP8, g.q, g.lr, qf[r]);
    row_init(st[r]);
  }
  const float sl = A.scale_log2;
  // lane's operand offsets in a stage
  const int koff = FP8 ? (g.kb1 ? kK1_8 : 0) + g.q * 256 + (lane & 7) * 16
                       : (g.kb1 ? kLdsK1 : 0) + g.q * 256 + (lane & 7) * 16;
  const int voff = FP8 ? kV8 + (g.vb1 ? 2048 : 0) + g.lr * 16 + (g.q & 1) * 8 : lds_v(g.vb1 ? 1 : 0, g.lr, g.q & 1);

  // Scores of one tile for every row block (K from the stage holding it).
  auto qk = [&](const uint8_t* stg, f32x4 (&s0)[RB], f32x4 (&s1)[RB]) {
    bf16x8 kf[2][4];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      if constexpr (!FP8) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
          kf[h][kb] = *reinterpret_cast<const bf16x8*>(stg + koff + kb * 1024 + h * 128);
      } else {
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          const uint4 w = *reinterpret_cast<const uint4*>(stg + koff + j * 1024 + h * 128);
          kf[h][2 * j] = __builtin_bit_cast(bf16x8, fp8x8_to_bf16(w.x, w.y));
          kf[h][2 * j + 1] = __builtin_bit_cast(bf16x8, fp8x8_to_bf16(w.z, w.w));
        }
      }
    }
#pragma unroll
    for (int r = 0; r < RB; ++r) qk_mfma(kf, qf[r], s0[r], s1[r]);
  };
  // Softmax and P.V of tile i from its scores.  V of tokens past the end is
  // zeroed (a missing second block aliases the first; its P is zero, but
  // the bits need not be finite).
  auto pv = [&](const uint8_t* stg, int i, const f32x4 (&s0)[RB], const f32x4 (&s1)[RB]) {
    const int t0 = 32 * i;
    const bool partial = t0 + 32 > ntok;
    const int nv = min(max(ntok - t0 - 8 * g.q, 0), 8);
    TileMeta m{0, 0, 1.f, 1.f, 1.f, 1.f};
    bf16x8 vf[8];
    if constexpr (FP8) {
      const float4 sc = *reinterpret_cast<const float4*>(stg + kMeta8);  // K0, V0, K1, V1
      m = TileMeta{0, 0, sc.x, sc.z, sc.y, sc.w};
    }
    float c, vsc;
    lane_scales(g, m, sl, c, vsc);
    bf16x8 ph[RB], pl[RB];
#pragma unroll
    for (int r = 0; r < RB; ++r) softmax_p<FP8>(s0[r], s1[r], partial, nv, c, vsc, st[r], ph[r], pl[r]);
    if constexpr (!FP8) {
      uint4 vr[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) vr[r] = *reinterpret_cast<const uint4*>(stg + voff + r * 256);
      if (partial) {
#pragma unroll
        for (int r = 0; r < 8; ++r) vr[r] = keep_first(vr[r], nv);
      }
#pragma unroll
      for (int r = 0; r < 8; ++r) vf[r] = __builtin_bit_cast(bf16x8, vr[r]);
    } else {
      uint2 vr[8];
#pragma unroll
      for (int r = 0; r < 8; ++r) vr[r] = *reinterpret_cast<const uint2*>(stg + voff + r * 256);
      if (partial) {
#pragma unroll
        for (int r = 0; r < 8; ++r) vr[r] = make_uint2(keep_bytes(vr[r].x, nv), keep_bytes(vr[r].y, nv - 4));
      }
#pragma unroll
      for (int r = 0; r < 8; ++r) vf[r] = __builtin_bit_cast(bf16x8, fp8x8_to_bf16(vr[r].x, vr[r].y));
    }
#pragma unroll
    for (int r = 0; r < RB; ++r) pv_mfma(vf, ph[r], pl[r], st[r]);
  };

  const int t = threadIdx.x;
  // Block ids live in LDS, two windows of 64: wave 0 loads window w + 1
  // when the tiles it issues enter window w.  Its completion is covered by
  // the per-tile waits (it retires before the tile loads issued after it),
  // and the tiles of window w - 1, whose slot it reuses, were issued before
  // the barrier.
  int32_t* idw = reinterpret_cast<int32_t*>(lds + ring * stage);
  auto fetch_ids = [&](int w) {
    if (wave == 0) dma4(brow + min(64 * w + lane, nblk - 1), idw + 64 * (w & 1));
  };
  auto issue = [&](int i) {
    const int j0 = 2 * i;
    if ((j0 & 63) == 0 && j0 > 0) fetch_ids((j0 >> 6) + 1);
    const int2 pr = *reinterpret_cast<const int2*>(idw + 64 * ((j0 >> 6) & 1) + (j0 & 63));
    int b0 = __builtin_amdgcn_readfirstlane(pr.x);
    int b1 = j0 + 1 < nblk ? __builtin_amdgcn_readfirstlane(pr.y) : b0;
    if ((unsigned)b0 >= (unsigned)P.num_blocks || (unsigned)b1 >= (unsigned)P.num_blocks) {
      if (t == 0) atomicOr(P.err, kErrBadBlock);
      b0 = (unsigned)b0 < (unsigned)P.num_blocks ? b0 : 0;
      b1 = (unsigned)b1 < (unsigned)P.num_blocks ? b1 : 0;
    }
    uint8_t* stg = lds + (i % ring) * stage;
    if constexpr (!FP8) {
      // Lane t of wave w loads a 16-byte chunk of each 4 KB region of a
      // tile into LDS slot t: K chunk t, and the V^T chunk (d = t % 128,
      // token half t / 128) that the LDS layout puts in slot t.
      const int kofs = t * 16;
      const int vofs = (t & 127) * 32 + 16 * (t >> 7);
      uint8_t* dst = stg + wave * 1024;
      const size_t o0 = head_off<false>(b0, P.Hkv, U.kvh), o1 = head_off<false>(b1, P.Hkv, U.kvh);
      dma16(P.k_cache + o0 + kofs, dst);
      dma16(P.k_cache + o1 + kofs, dst + kLdsK1);
      dma16(P.v_cache + o0 + vofs, dst + kLdsV);
      dma16(P.v_cache + o1 + vofs, dst + kLdsV + kTileBytes);
    } else {
      // Waves 0-1 move block b0's K and V^T tiles, waves 2-3 block b1's
      // (lane t to byte 16 (t % 128) of its block's K and V^T); wave 0 also
      // moves the scales, lane l the l % 4-th of (K0, V0, K1, V1).
      if (wave == 0) dma4(P.kv_scale + 2 * ((lane & 2) ? b1 : b0) + (lane & 1), stg + kMeta8);
      const size_t o = head_off<true>(wave < 2 ? b0 : b1, P.Hkv, U.kvh) + (t & 127) * 16;
      dma16(P.k_cache + o, stg + wave * 1024 + (wave < 2 ? 0 : kK1_8 - 2048));
      dma16(P.v_cache + o, stg + kV8 + wave * 1024);
    }
  };
  // Waits until this wave's loads of the tiles before the `later` last
  // issued ones are in LDS (wave 0 issues one more load per fp8 tile).
  auto wait = [&](int later) {
    if constexpr (!FP8)
      wait_tiles(later);
    else if (wave == 0)
      wait_tiles_per<3>(later);
    else
      wait_tiles_per<2>(later);
  };
  fetch_ids(0);
  if (nblk > 64) fetch_ids(1);
  __builtin_amdgcn_s_waitcnt(0x0F70);  // Q operands and the first id windows are in
  barrier_no_fence();
  for (int i = 0; i < ahead && i < ntile; ++i) issue(i);
  wait(min(ahead, ntile) - 1);  // tile 0 is in LDS
  barrier_no_fence();
  f32x4 s0[RB], s1[RB];
  if (active) qk(lds, s0, s1);
  // Iteration i issues the scores of tile i + 1 before the softmax and P.V
  // of tile i, so the matrix cores work while the vector ALUs do the
  // softmax.  Tile i + 1 must be in LDS first; stage (i - 1) % ring, read
  // for the last time in iteration i - 1, takes tile i + ahead.
  for (int i = 0; i < ntile; ++i) {
    const bool more = i + 1 < ntile;
    wait(max(min(ahead - 2, ntile - 2 - i), 0));  // this wave's loads of tile i + 1 are in LDS
    barrier_no_fence();                            // ... and every wave's
    if (i + ahead < ntile) issue(i + ahead);
    if (active) {
      f32x4 n0[RB], n1[RB];
      if (more) qk(lds + ((i + 1) % ring) * stage, n0, n1);
      pv(lds + (i % ring) * stage, i, s0, s1);
#pragma unroll
      for (int r = 0; r < RB; ++r) {
        s0[r] = n0[r];
        s1[r] = n1[r];
      }
    }
  }
  if (active) {
#pragma unroll
    for (int r = 0; r < RB; ++r) write_partial(P, A, U, row0 + 16 * r, R, g.q, g.lr, st[r]);
  }
}

// Workgroups are dispatched round-robin over the 8 XCDs, so workgroup bid
// runs on XCD bid % 8.  The plan lists every XCD's workgroup slots
// contiguously, four entries per slot: a cooperative item (flagged in its
// first entry) or four narrow units, in the order they should start
// (longest first).  Cooperative (compute-bound) and narrow (HBM-bound)
// slots are interleaved so both kinds share every CU.  Workgroup j of an
// XCD runs slot j, except in the XCD's last kTailSlots slots: those are
// claimed at run time, from the front by the XCD's own workgroups and from
// the back (the shortest slots) by workgroups of XCDs that have no work
// left, so the XCDs finish together.  One atomic word per XCD holds both
// claim counts (front in the low half), so front and back claims never
// meet; there are at least as many workgroups as slots.

__device__ inline int tail_start(const AttnLaunch& A, int x) {
  return max((A.xcd_off[x + 1] - A.xcd_off[x]) / kUnitsPerWG - kTailSlots, 0);
}

template <bool FP8>
__global__ __launch_bounds__(kThreads, 2) void attn_units_kernel(DevPool P, AttnLaunch A) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[(FP8 ? kRing8 * kStage8 : kRing * kStage) + kIdsBytes];
  static_assert(!FP8 || 4 * 8192 <= kRing8 * kStage8, "narrow waves' Q regions (two row blocks)");
  __shared__ int claimed;
  if (threadIdx.x == 0) {
    const int x = blockIdx.x & 7, j = blockIdx.x >> 3;
    int b = -1;
    if (j < tail_start(A, x)) {
      b = A.xcd_off[x] + kUnitsPerWG * j;
    } else {
      for (int k = 0; k < 8 && b < 0; ++k) {
        const int y = (x + k) & 7;
        const int s0 = tail_start(A, y);
        const int m = (A.xcd_off[y + 1] - A.xcd_off[y]) / kUnitsPerWG - s0;
        if (m <= 0) continue;
        const unsigned old = atomicAdd(reinterpret_cast<unsigned*>(A.queues) + y, k == 0 ? 1u : 0x10000u);
        const int f = (int)(old & 0xffffu), bk = (int)(old >> 16);
        if (f + bk < m) b = A.xcd_off[y] + kUnitsPerWG * (s0 + (k == 0 ? f : m - 1 - bk));
      }
    }
    claimed = b;
  }
  __syncthreads();
  const int base = claimed;
  if (base < 0) return;  // uniform over the workgroup
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const AttnUnit U0 = A.units[base];
  if (U0.flags & kUnitCoop) {
    // up to 64 rows: one row block per wave; more: two
    if (U0.mem_cnt * P.g > 4 * kRowsPerUnit)
      coop_unit<FP8, 2>(P, A, U0, wave, lane, lds);
    else if (U0.mem_cnt > 0)
      coop_unit<FP8, 1>(P, A, U0, wave, lane, lds);
    return;
  }
  const AttnUnit U = A.units[base + wave];  // a narrow slot always has four entries
  // no barrier on the narrow path; fp8 units of 17-32 rows take two row
  // blocks in one wave
  if constexpr (FP8) {
    if (U.mem_cnt * P.g > kRowsPerUnit)
      narrow_unit<FP8, 2>(P, A, U, lane, lds + wave * 8192);
    else if (U.mem_cnt > 0)
      narrow_unit<FP8, 1>(P, A, U, lane, nullptr);
  } else if (U.mem_cnt > 0) {
    narrow_unit<FP8, 1>(P, A, U, lane, nullptr);
  }
}

// Log-sum-exp merge of a row's partials.  One wave per (list position,
// query head): lane k < nk reads partial k's (max, sum), the wave reduces the
// maximum and the weighted sum, then every lane accumulates its two d values
// over the partials with the weights broadcast from their lanes.
__global__ __launch_bounds__(256) void merge_kernel(DevPool P, AttnLaunch A) {
  if (blockIdx.x == 0 && threadIdx.x < 8) A.queues[threadIdx.x] = 0;  // for the next attention launch
  if (A.len_bias && A.advance) {  // the step's token is in: advance the lengths (and GenLen, Alg. 1)
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < A.n) {
      const int t = A.list[i];
      P.seq_len[t] += 1;
      P.gen[t] += 1;
    }
  }
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
  // Partials are read once: eight loads in flight, streaming; added in
  // partial order.
  float o0 = 0.f, o1 = 0.f;
  int k = 0;
  for (; k + 8 <= nk; k += 8) {
    f32x2 a[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
      a[j] = __builtin_nontemporal_load(reinterpret_cast<const f32x2*>(pa + (size_t)(k + j) * kHeadDim + 2 * lane));
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float wk = __shfl(w, k + j);
      o0 += wk * a[j].x;
      o1 += wk * a[j].y;
    }
  }
  for (; k < nk; ++k) {
    const f32x2 a = __builtin_nontemporal_load(reinterpret_cast<const f32x2*>(pa + (size_t)k * kHeadDim + 2 * lane));
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
