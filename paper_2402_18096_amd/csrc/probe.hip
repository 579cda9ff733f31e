// Streaming-read probe: the HBM read bandwidth a plain kernel reaches on this
// device, the practical ceiling next to the data-sheet peak in the roofline
// figures.  Each thread keeps four 16-byte loads in flight and walks the
// buffer with a grid stride (front to back, or back to front); the loaded
// words are folded and stored only if the fold hits a sentinel, which keeps
// the loads without a store per load.
#include <algorithm>

#include "mikv_internal.h"

namespace mikv {

namespace {

constexpr int kProbeThreads = 256, kProbeInFlight = 4, kProbeMaxBlocks = 8192;
constexpr uint32_t kProbeSentinel = 0x9e3779b9u;

__global__ __launch_bounds__(kProbeThreads) void stream_read_kernel(const uint4 *__restrict__ p, size_t n16,
                                                                    int backwards, uint32_t *sink) {
  const size_t tid = (size_t)blockIdx.x * kProbeThreads + threadIdx.x;
  const size_t nth = (size_t)gridDim.x * kProbeThreads;
  uint32_t fold = 0u;
  for (size_t i = tid; i < n16; i += nth * kProbeInFlight) {
    uint4 v[kProbeInFlight];
#pragma unroll
    for (int u = 0; u < kProbeInFlight; ++u) {
      const size_t j = i + (size_t)u * nth;
      v[u] = j < n16 ? p[backwards ? n16 - 1 - j : j] : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < kProbeInFlight; ++u) fold ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (fold == kProbeSentinel) sink[0] = fold;
}

}  // namespace

}  // namespace mikv

using namespace mikv;

extern "C" int mikv_stream_read_probe(const void *buf, size_t bytes, int32_t backwards, uint32_t *sink,
                                      void *stream) {
  if (!buf || !sink) return set_error(MIKV_ERR_INVALID_ARG, "mikv_stream_read_probe: NULL pointer");
  if (bytes == 0 || bytes % 16 != 0 || (uintptr_t)buf % 16 != 0)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_stream_read_probe: buf must be 16-byte aligned, bytes a positive multiple of 16");
  const size_t n16 = bytes / 16;
  const size_t per_block = (size_t)kProbeThreads * kProbeInFlight;
  const int blocks = (int)std::min<size_t>(kProbeMaxBlocks, (n16 + per_block - 1) / per_block);
  hipLaunchKernelGGL(stream_read_kernel, dim3(blocks), dim3(kProbeThreads), 0, (hipStream_t)stream,
                     reinterpret_cast<const uint4 *>(buf), n16, backwards ? 1 : 0, sink);
  return check_launch("mikv_stream_read_probe");
}
