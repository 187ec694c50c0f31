// Streaming-read ceiling of the device memory, for reporting the attention
// kernel's achieved bandwidth against what plain reads of the same chip
// reach (the published HBM peak is the roofline; this is the practical one).
//
// The buffer is cut into 64 KiB chunks; workgroup w reads a contiguous run
// of chunks (the runs differ in length by at most one chunk).  Per chunk
// each of the four waves issues 16 loads of 16 bytes per lane, waves
// interleaved by 1 KiB, so a workgroup has 64 KiB in flight.  Every dword
// is read exactly once and folded by XOR into the workgroup's sink word, so
// the XOR of all sink words equals the XOR of the buffer's dwords (what the
// correctness test checks), and the loads cannot be dropped.
#include <hip/hip_runtime.h>

#include "gambit.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
constexpr size_t kChunk = 65536;

template <bool NT>
__global__ __launch_bounds__(256) void stream_read_kernel(const uint8_t* buf, size_t nchunks, uint32_t* sink) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const size_t q = nchunks / gridDim.x, r = nchunks % gridDim.x, w = blockIdx.x;
  const size_t c0 = w * q + (w < r ? w : r), c1 = c0 + q + (w < r ? 1 : 0);
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (size_t c = c0; c < c1; ++c) {
    const uint8_t* base = buf + c * kChunk + (size_t)wave * 1024 + (size_t)lane * 16;
    u32x4 v[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const u32x4* p = reinterpret_cast<const u32x4*>(base + (size_t)k * 4096);
      if constexpr (NT)
        v[k] = __builtin_nontemporal_load(p);
      else
        v[k] = *p;
    }
#pragma unroll
    for (int k = 0; k < 16; ++k) acc ^= v[k];
  }
  atomicXor(sink + blockIdx.x, acc.x ^ acc.y ^ acc.z ^ acc.w);
}

}  // namespace

extern "C" gambit_status gambit_stream_read(const void* buf, size_t bytes, int32_t nontemporal, int32_t grid,
                                            uint32_t* sink, void* stream) {
  if (!buf || !sink || bytes == 0 || bytes % kChunk != 0 || grid < 1 || grid > 65535 ||
      (size_t)grid > bytes / kChunk || (reinterpret_cast<uintptr_t>(buf) & 15) != 0 ||
      (nontemporal != 0 && nontemporal != 1))
    return GAMBIT_ERR_INVALID;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const uint8_t* b = static_cast<const uint8_t*>(buf);
  if (nontemporal)
    stream_read_kernel<true><<<grid, 256, 0, s>>>(b, bytes / kChunk, sink);
  else
    stream_read_kernel<false><<<grid, 256, 0, s>>>(b, bytes / kChunk, sink);
  return hipGetLastError() == hipSuccess ? GAMBIT_OK : GAMBIT_ERR_DEVICE;
}
