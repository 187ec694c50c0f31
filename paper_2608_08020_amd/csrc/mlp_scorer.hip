// Host entry points of the 2-layer MLP scorer (the paper's main-evaluation
// probe on the thought-boundary hidden state, Sec. 4.1 and Sec. 5.1):
// argument validation and the launch of the fused kernels in
// probe_topk.hip.  Two entry points share those kernels: gambit_mlp_score
// takes its scratch (the tiles' partial logits) from a caller workspace;
// gambit_mlp_score_static takes it from a buffer the library holds in
// device memory for the life of the process, so that callers that cannot
// allocate device memory at all (code under HIP graph capture, serving
// loops that forbid allocation) can score.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/gambit.h"
#include "kernels.h"

namespace {

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
  if (!mlp || !h || !scores_out || n <= 0 || n > gambit::kMaxRank) return GAMBIT_ERR_INVALID;
  if (mlp->dim <= 0 || mlp->dim % 128 || mlp->hidden <= 0 || mlp->hidden % 64 ||
      (mlp->activation != GAMBIT_ACT_RELU && mlp->activation != GAMBIT_ACT_GELU) || !mlp->w1 || !mlp->b1 || !mlp->w2)
    return GAMBIT_ERR_INVALID;
  if (keep < 0 || keep > n || (keep > 0 && (!trace_ids || !keep_out))) return GAMBIT_ERR_INVALID;
  return GAMBIT_OK;
}

gambit_status launch(int32_t n, const void* h, const gambit_mlp* mlp, float* scores_out, const int32_t* trace_ids,
                     int32_t keep, int32_t* keep_out, float* parts, void* stream) {
  gambit::MlpLaunch L{};
  L.n = n;
  L.dim = mlp->dim;
  L.hidden = mlp->hidden;
  L.act = mlp->activation;
  L.h = static_cast<const uint16_t*>(h);
  L.w1 = static_cast<const uint16_t*>(mlp->w1);
  L.b1 = mlp->b1;
  L.w2 = mlp->w2;
  L.b2 = mlp->b2;
  L.parts = parts;
  L.scores_out = scores_out;
  L.ids = trace_ids;
  L.keep = keep;
  L.keep_out = keep_out;
  return gambit::launch_mlp_score(L, static_cast<hipStream_t>(stream)) == hipSuccess ? GAMBIT_OK
                                                                                      : GAMBIT_ERR_DEVICE;
}

}  // namespace

extern "C" {

size_t gambit_mlp_workspace_size(int32_t n, int32_t hidden) {
  if (n <= 0 || hidden <= 0 || hidden % 64) return 0;  // the documented unit multiple
  return 4 * (size_t)n * (hidden / gambit::kMlpTileH);
}

gambit_status gambit_mlp_score(int32_t n, const void* h, const gambit_mlp* mlp, float* scores_out,
                               const int32_t* trace_ids, int32_t keep, int32_t* keep_out, void* workspace,
                               size_t workspace_bytes, void* stream) {
  const gambit_status st = check_mlp(n, h, mlp, scores_out, trace_ids, keep, keep_out);
  if (st != GAMBIT_OK) return st;
  if (!workspace || workspace_bytes < gambit_mlp_workspace_size(n, mlp->hidden)) return GAMBIT_ERR_WORKSPACE;
  return launch(n, h, mlp, scores_out, trace_ids, keep, keep_out, static_cast<float*>(workspace), stream);
}

gambit_status gambit_mlp_score_static(int32_t n, const void* h, const gambit_mlp* mlp, float* scores_out,
                                      const int32_t* trace_ids, int32_t keep, int32_t* keep_out, void* stream) {
  const gambit_status st = check_mlp(n, h, mlp, scores_out, trace_ids, keep, keep_out);
  if (st != GAMBIT_OK) return st;
  if (gambit_mlp_workspace_size(n, mlp->hidden) > kStaticScratchBytes) return GAMBIT_ERR_WORKSPACE;
  void* parts = nullptr;
  if (device_scratch(&parts) != hipSuccess) return GAMBIT_ERR_DEVICE;
  return launch(n, h, mlp, scores_out, trace_ids, keep, keep_out, static_cast<float*>(parts), stream);
}

}  // extern "C"
