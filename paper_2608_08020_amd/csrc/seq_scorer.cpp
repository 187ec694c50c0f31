// Host side of the sequence scorer (App. A.1, Eqs. 4-6): validation, the
// per-slot step counts (host mirror), workspace carving and the launch
// sequence of one boundary.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "gambit.h"
#include "seq_kernels.h"

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct SeqLayout {
  size_t ids, pairs, lens, err, cache, planes, cvec, dvec, part, x, u, qkv, o, g, total;
  int out_splits;  // of the d_model-wide projections (W_o, W_2) over their K
};

bool seq_layout(const gambit_scorer_desc* d, SeqLayout* L) {
  if (!d || d->input_dim <= 0 || d->d_model <= 0 || d->n_heads <= 0 || d->n_layers < 0 || d->d_ff <= 0 ||
      d->max_steps <= 0 || d->max_traces <= 0)
    return false;
  if (d->d_model != 64 * d->n_heads) return false;              // head_dim 64
  if (d->input_dim % 128 || d->d_ff % 64) return false;         // GEMM tiles
  if (d->max_steps > 8192) return false;                        // LDS of the attention step
  const size_t T = d->max_traces, D = d->input_dim, dm = d->d_model, f = d->d_ff;
  // W_o (K = d_model) and W_2 (K = d_ff) have d_model / 64 column tiles:
  // split their K four ways (while the parts stay >= 64 deep) to fill the GPU
  L->out_splits = 4;
  while (L->out_splits > 1 && (dm % (64 * (size_t)L->out_splits) || f % (64 * (size_t)L->out_splits)))
    --L->out_splits;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes);
    return at;
  };
  L->ids = take(4 * T);
  L->pairs = take(8 * T);
  L->lens = take(4 * T);
  L->err = take(64);
  L->cache = take(4 * T * d->n_layers * d->n_heads * gambit::seq_region_floats(d->max_steps));
  L->planes = take(2 * 3 * dm * D);
  L->cvec = take(4 * dm);
  L->dvec = take(4 * dm);
  // split partial sums: the input projection's (splits x n x 3 d_model, the
  // largest over every n <= max_traces) or W_o's and W_2's
  size_t part = (size_t)L->out_splits * T * dm;
  for (size_t n = 1; n <= T; ++n)
    part = std::max(part, (size_t)gambit::bf16_partial_splits((int)n, (int)D, (int)(3 * dm)) * n * 3 * dm);
  L->part = take(4 * part);
  L->x = take(4 * T * dm);
  L->u = take(4 * T * dm);
  L->qkv = take(4 * T * 3 * dm);
  L->o = take(4 * T * dm);
  L->g = take(4 * T * f);
  L->total = o;
  return true;
}

}  // namespace

struct gambit_scorer {
  gambit_scorer_desc d{};
  SeqLayout L{};
  uint8_t* ws = nullptr;
  gambit::SeqDev dev{};
  std::vector<int32_t> lens;  // host mirror of the step counts
  int32_t* stage = nullptr;   // pinned staging for id uploads
  hipEvent_t stage_ev = nullptr;
  std::string last_error;
};

namespace {

gambit_status sfail(gambit_scorer* q, gambit_status s, const char* fmt, ...) {
  if (q) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    q->last_error = buf;
  }
  return s;
}

#define SEQ_TRY(q, expr, where)                                                                   \
  do {                                                                                            \
    const hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess) return sfail(q, GAMBIT_ERR_DEVICE, "%s: %s", where, hipGetErrorString(e_)); \
  } while (0)

template <class T>
T* wsp(gambit_scorer* q, size_t off) {
  return reinterpret_cast<T*>(q->ws + off);
}

gambit_status upload(gambit_scorer* q, int32_t* dst, const int32_t* src, size_t n, hipStream_t s) {
  if (n == 0) return GAMBIT_OK;
  SEQ_TRY(q, hipEventSynchronize(q->stage_ev), "staging fence");
  std::memcpy(q->stage, src, n * 4);
  SEQ_TRY(q, hipMemcpyAsync(dst, q->stage, n * 4, hipMemcpyHostToDevice, s), "upload");
  SEQ_TRY(q, hipEventRecord(q->stage_ev, s), "staging fence");
  return GAMBIT_OK;
}

gambit_status check_slots(gambit_scorer* q, int32_t n, const int32_t* ids, const char* what,
                          std::vector<char>* seen_out = nullptr) {
  if (n < 0 || n > q->d.max_traces) return sfail(q, GAMBIT_ERR_INVALID, "%s count %d out of range", what, n);
  if (n > 0 && !ids) return sfail(q, GAMBIT_ERR_INVALID, "%s list is NULL", what);
  std::vector<char> seen(q->d.max_traces, 0);
  for (int i = 0; i < n; ++i) {
    const int t = ids[i];
    if (t < 0 || t >= q->d.max_traces) return sfail(q, GAMBIT_ERR_INVALID, "%s id %d out of range", what, t);
    if (seen[t]) return sfail(q, GAMBIT_ERR_INVALID, "duplicate %s id %d", what, t);
    seen[t] = 1;
  }
  if (seen_out) seen_out->swap(seen);
  return GAMBIT_OK;
}

inline hipStream_t S(void* s) { return static_cast<hipStream_t>(s); }

}  // namespace

extern "C" {

size_t gambit_scorer_workspace_size(const gambit_scorer_desc* desc) {
  SeqLayout L;
  return seq_layout(desc, &L) ? L.total : 0;
}

gambit_status gambit_scorer_create(const gambit_scorer_desc* desc, void* stream, gambit_scorer** out) {
  if (!out) return GAMBIT_ERR_INVALID;
  *out = nullptr;
  SeqLayout L;
  if (!seq_layout(desc, &L)) return GAMBIT_ERR_INVALID;
  if (!desc->ln_in_g || !desc->ln_in_b || !desc->w_in || !desc->ln_out_g || !desc->ln_out_b || !desc->w_out ||
      !desc->workspace)
    return GAMBIT_ERR_INVALID;
  if (desc->n_layers > 0 && (!desc->ln1_g || !desc->ln1_b || !desc->w_qkv || !desc->w_o || !desc->ln2_g ||
                             !desc->ln2_b || !desc->w_13 || !desc->w_2))
    return GAMBIT_ERR_INVALID;
  if (desc->workspace_bytes < L.total) return GAMBIT_ERR_WORKSPACE;
  if (reinterpret_cast<uintptr_t>(desc->workspace) % kAlign) return GAMBIT_ERR_INVALID;
  auto* q = new gambit_scorer;
  q->d = *desc;
  q->L = L;
  q->ws = static_cast<uint8_t*>(desc->workspace);
  q->lens.assign(desc->max_traces, 0);
  gambit::SeqDev& D = q->dev;
  D.ids = wsp<int32_t>(q, L.ids);
  D.lens = wsp<int32_t>(q, L.lens);
  D.err = wsp<int32_t>(q, L.err);
  D.cache = wsp<float>(q, L.cache);
  D.ln_out_g = desc->ln_out_g;
  D.ln_out_b = desc->ln_out_b;
  D.w_out = desc->w_out;
  D.d_model = desc->d_model;
  D.n_heads = desc->n_heads;
  D.n_layers = desc->n_layers;
  D.max_steps = desc->max_steps;
  hipError_t e = hipHostMalloc(reinterpret_cast<void**>(&q->stage), 8 * (size_t)desc->max_traces,
                               hipHostMallocDefault);
  if (e == hipSuccess) e = hipEventCreateWithFlags(&q->stage_ev, hipEventDisableTiming);
  if (e == hipSuccess) e = hipEventRecord(q->stage_ev, S(stream));
  // the input projection's planes, row sums and bias term (w_in, ln_in_g and
  // ln_in_b are not read again)
  if (e == hipSuccess)
    e = gambit::seq_prep_input(desc->w_in, desc->ln_in_g, desc->ln_in_b, desc->input_dim, desc->d_model,
                               wsp<uint16_t>(q, L.planes), wsp<float>(q, L.cvec), wsp<float>(q, L.dvec), S(stream));
  // every slot starts with no steps; the error word starts clear
  std::vector<int32_t> all(desc->max_traces);
  for (int i = 0; i < desc->max_traces; ++i) all[i] = i;
  if (e == hipSuccess && upload(q, wsp<int32_t>(q, L.pairs), all.data(), all.size(), S(stream)) == GAMBIT_OK) {
    e = gambit::seq_set_len(D, wsp<int32_t>(q, L.pairs), desc->max_traces, 0, S(stream));
    if (e == hipSuccess) e = hipMemsetAsync(D.err, 0, 64, S(stream));
  } else if (e == hipSuccess) {
    e = hipErrorUnknown;
  }
  // the set-up is complete before create returns, so steps on any stream
  // see the planes, the step counts and the error word
  if (e == hipSuccess) e = hipStreamSynchronize(S(stream));
  if (e != hipSuccess) {
    gambit_scorer_destroy(q);
    return GAMBIT_ERR_DEVICE;
  }
  *out = q;
  return GAMBIT_OK;
}

gambit_status gambit_scorer_destroy(gambit_scorer* q) {
  if (!q) return GAMBIT_ERR_INVALID;
  if (q->stage_ev) {
    (void)hipEventSynchronize(q->stage_ev);
    (void)hipEventDestroy(q->stage_ev);
  }
  if (q->stage) (void)hipHostFree(q->stage);
  delete q;
  return GAMBIT_OK;
}

gambit_status gambit_scorer_step(gambit_scorer* q, int32_t n, const int32_t* ids, const void* h, float* scores_out,
                              void* stream) {
  if (!q) return GAMBIT_ERR_INVALID;
  gambit_status st = check_slots(q, n, ids, "trace");
  if (st) return st;
  if (n == 0) return GAMBIT_OK;
  if (!h || !scores_out) return sfail(q, GAMBIT_ERR_INVALID, "NULL buffer");
  for (int i = 0; i < n; ++i)
    if (q->lens[ids[i]] >= q->d.max_steps)
      return sfail(q, GAMBIT_ERR_INVALID, "trace %d already holds %d steps", ids[i], q->d.max_steps);
  hipStream_t s = S(stream);
  st = upload(q, wsp<int32_t>(q, q->L.ids), ids, n, s);
  if (st) return st;
  const gambit_scorer_desc& d = q->d;
  const int D = d.input_dim, dm = d.d_model, f = d.d_ff;
  float* part = wsp<float>(q, q->L.part);
  float* x = wsp<float>(q, q->L.x);
  float* u = wsp<float>(q, q->L.u);
  float* qkv = wsp<float>(q, q->L.qkv);
  float* o = wsp<float>(q, q->L.o);
  float* g = wsp<float>(q, q->L.g);
  using namespace gambit;
  const uint16_t* hb = static_cast<const uint16_t*>(h);
  const int in_splits = bf16_partial_splits(n, D, 3 * dm);
  SEQ_TRY(q, bf16_gemm_partials(hb, wsp<uint16_t>(q, q->L.planes), n, D, 3 * dm, in_splits, part, s),
          "input projection");
  // each K-split projection's reduce also takes the LayerNorm after it: LN1
  // of the next layer, LN2, or LN_out with the head after the last layer
  {
    const bool head = d.n_layers == 0;
    SEQ_TRY(q, seq_reduce_in(hb, D, part, in_splits, wsp<float>(q, q->L.cvec), wsp<float>(q, q->L.dvec), x, dm,
                             head ? nullptr : d.ln1_g, head ? nullptr : d.ln1_b, u, head, q->dev, scores_out, n, s),
            "input projection reduce");
  }
  auto reduce_ln = [&](int splits, const float* R, int next_ln1, const char* where) -> gambit_status {
    const bool head = next_ln1 >= d.n_layers;
    const float* g = head ? nullptr : d.ln1_g + (size_t)next_ln1 * dm;
    const float* b = head ? nullptr : d.ln1_b + (size_t)next_ln1 * dm;
    SEQ_TRY(q, seq_reduce_ln(part, splits, R, x, dm, g, b, u, head, q->dev, scores_out, n, s), where);
    return GAMBIT_OK;
  };
  for (int l = 0; l < d.n_layers; ++l) {
    const size_t dd = (size_t)dm * dm;
    SEQ_TRY(q, seq_gemm(u, d.w_qkv + 3 * dd * l, qkv, n, 3 * dm, dm, 1, kEpiNone, nullptr, s),
            "QKV");
    SEQ_TRY(q, seq_attention(q->dev, l, qkv, o, n, s), "attention step");
    SEQ_TRY(q, seq_gemm(o, d.w_o + dd * l, x, n, dm, dm, q->L.out_splits, kEpiNone, part, s),
            "output projection");
    SEQ_TRY(q, seq_reduce_ln(part, q->L.out_splits, x, x, dm, d.ln2_g + (size_t)l * dm,
                             d.ln2_b + (size_t)l * dm, u, false, q->dev, scores_out, n, s),
            "output projection reduce, LN2");
    SEQ_TRY(q, seq_gemm(u, d.w_13 + 2 * (size_t)f * dm * l, g, n, 2 * f, dm, 1, kEpiSwiGLU, nullptr, s),
            "SwiGLU");
    SEQ_TRY(q, seq_gemm(g, d.w_2 + (size_t)f * dm * l, x, n, dm, f, q->L.out_splits, kEpiNone, part, s),
            "SwiGLU out");
    st = reduce_ln(q->L.out_splits, x, l + 1, "SwiGLU out reduce, next LayerNorm");
    if (st) return st;
  }
  for (int i = 0; i < n; ++i) ++q->lens[ids[i]];
  return GAMBIT_OK;
}

gambit_status gambit_scorer_fork(gambit_scorer* q, int32_t n, const int32_t* parents, const int32_t* children,
                              void* stream) {
  if (!q) return GAMBIT_ERR_INVALID;
  std::vector<char> is_child;
  gambit_status st = check_slots(q, n, children, "child", &is_child);
  if (st) return st;
  if (n > 0 && !parents) return sfail(q, GAMBIT_ERR_INVALID, "parent list is NULL");
  for (int i = 0; i < n; ++i) {
    const int p = parents[i];
    if (p < 0 || p >= q->d.max_traces) return sfail(q, GAMBIT_ERR_INVALID, "parent id %d out of range", p);
    if (is_child[p]) return sfail(q, GAMBIT_ERR_INVALID, "trace %d is both parent and child", p);
  }
  if (n == 0) return GAMBIT_OK;
  std::vector<int32_t> pairs(2 * (size_t)n);
  for (int i = 0; i < n; ++i) {
    pairs[2 * i] = children[i];
    pairs[2 * i + 1] = parents[i];
  }
  int32_t* dp = wsp<int32_t>(q, q->L.pairs);
  st = upload(q, dp, pairs.data(), pairs.size(), S(stream));
  if (st) return st;
  SEQ_TRY(q, gambit::seq_fork(q->dev, dp, n, S(stream)), "fork");
  for (int i = 0; i < n; ++i) q->lens[children[i]] = q->lens[parents[i]];
  return GAMBIT_OK;
}

gambit_status gambit_scorer_free(gambit_scorer* q, int32_t n, const int32_t* ids, void* stream) {
  if (!q) return GAMBIT_ERR_INVALID;
  gambit_status st = check_slots(q, n, ids, "trace");
  if (st) return st;
  if (n == 0) return GAMBIT_OK;
  int32_t* di = wsp<int32_t>(q, q->L.pairs);
  st = upload(q, di, ids, n, S(stream));
  if (st) return st;
  SEQ_TRY(q, gambit::seq_set_len(q->dev, di, n, 0, S(stream)), "free");
  for (int i = 0; i < n; ++i) q->lens[ids[i]] = 0;
  return GAMBIT_OK;
}

int32_t gambit_scorer_steps(const gambit_scorer* q, int32_t id) {
  if (!q || id < 0 || id >= q->d.max_traces) return -1;
  return q->lens[id];
}

gambit_status gambit_scorer_check(gambit_scorer* q, void* stream) {
  if (!q) return GAMBIT_ERR_INVALID;
  std::vector<int32_t> lens(q->d.max_traces);
  int32_t err = 0;
  SEQ_TRY(q, hipMemcpyAsync(lens.data(), q->dev.lens, 4 * lens.size(), hipMemcpyDeviceToHost, S(stream)),
          "read step counts");
  SEQ_TRY(q, hipMemcpyAsync(&err, q->dev.err, 4, hipMemcpyDeviceToHost, S(stream)), "read error word");
  SEQ_TRY(q, hipStreamSynchronize(S(stream)), "sync");
  if (err) return sfail(q, GAMBIT_ERR_DEVICE, "device error word %d", err);
  for (int t = 0; t < q->d.max_traces; ++t)
    if (lens[t] != q->lens[t])
      return sfail(q, GAMBIT_ERR_DEVICE, "slot %d: device holds %d steps, host %d", t, lens[t], q->lens[t]);
  return GAMBIT_OK;
}

const char* gambit_scorer_last_error(const gambit_scorer* q) { return q ? q->last_error.c_str() : ""; }

}  // extern "C"
