// Streaming-read probe: the HBM read bandwidth a plain kernel reaches on this
// device, the practical ceiling next to the data-sheet peak in the roofline
// figures.  Each block reads one contiguous chunk of the buffer, 256 threads
// with four 16-byte loads in flight each; chunks in the leading
// `resident_bytes` are read with plain loads, the others with non-temporal
// loads, the split the attention kernel makes between the rows the
// last-level cache keeps across steps and those it streams.  The loaded
// words are folded and stored only if the fold hits a sentinel, which keeps
// the loads without a store per load.
#include <algorithm>

#include "mikv_internal.h"

namespace mikv {

namespace {

constexpr int kProbeThreads = 256, kProbeInFlight = 4, kProbeMaxBlocks = 8192;
constexpr size_t kProbeGrain = (size_t)kProbeThreads * kProbeInFlight;  // 16-byte words per block iteration
constexpr uint32_t kProbeSentinel = 0x9e3779b9u;

typedef uint32_t v4u __attribute__((ext_vector_type(4)));

template <bool NT>
__device__ inline uint32_t read_chunk(const v4u *__restrict__ p, size_t start, size_t end) {
  uint32_t fold = 0u;
  for (size_t i = start + threadIdx.x; i < end; i += kProbeGrain) {
    v4u v[kProbeInFlight];
#pragma unroll
    for (int u = 0; u < kProbeInFlight; ++u) {
      const size_t j = i + (size_t)u * kProbeThreads;
      if (j < end)
        v[u] = NT ? __builtin_nontemporal_load(&p[j]) : p[j];
      else
        v[u] = v4u{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kProbeInFlight; ++u) fold ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  return fold;
}

// Block b reads chunk b (chunk gridDim.x - 1 - b backwards, so the chunks are
// dispatched in the opposite order) of `chunk16` 16-byte words.
__global__ __launch_bounds__(kProbeThreads) void stream_read_kernel(const v4u *__restrict__ p, size_t n16,
                                                                    size_t chunk16, size_t res16, int backwards,
                                                                    uint32_t *sink) {
  const size_t b = backwards ? gridDim.x - 1 - blockIdx.x : blockIdx.x;
  const size_t start = b * chunk16, end = std::min(start + chunk16, n16);
  const uint32_t fold = start < res16 ? read_chunk<false>(p, start, end) : read_chunk<true>(p, start, end);
  if (fold == kProbeSentinel) sink[0] = fold;
}

}  // namespace

}  // namespace mikv

using namespace mikv;

extern "C" int mikv_stream_read_probe(const void *buf, size_t bytes, size_t resident_bytes, int32_t backwards,
                                      uint32_t *sink, void *stream) {
  if (!buf || !sink) return set_error(MIKV_ERR_INVALID_ARG, "mikv_stream_read_probe: NULL pointer");
  if (bytes == 0 || bytes % 16 != 0 || (uintptr_t)buf % 16 != 0)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_stream_read_probe: buf must be 16-byte aligned, bytes a positive multiple of 16");
  const size_t n16 = bytes / 16;
  // whole block iterations per chunk, at most kProbeMaxBlocks chunks
  const size_t per_block = (n16 + kProbeMaxBlocks - 1) / kProbeMaxBlocks;
  const size_t chunk16 = (per_block + kProbeGrain - 1) / kProbeGrain * kProbeGrain;
  const int blocks = (int)((n16 + chunk16 - 1) / chunk16);
  hipLaunchKernelGGL(stream_read_kernel, dim3(blocks), dim3(kProbeThreads), 0, (hipStream_t)stream,
                     reinterpret_cast<const v4u *>(buf), n16, chunk16, std::min(resident_bytes / 16, n16),
                     backwards ? 1 : 0, sink);
  return check_launch("mikv_stream_read_probe");
}

