// Query/key channel balancer, Section 3.2, Eq. 2:
//   b[b, h, c] = sqrt( max_{t, i in group(h)} |q| / max_t |k| ),  1 if a max is 0.
// Pass 1: one block per (token chunk, head) reduces |q| and |k| per channel
// over its chunk and writes the chunk maxima; pass 2 reduces the chunk
// maxima per head and applies the correctly rounded fp32 divide and square
// root.  Maxima are exact and the reduction order does not matter, so the
// result is deterministic.
#include "mikv_internal.h"

namespace mikv {

namespace {

constexpr int kBalChunk = 512;  // tokens per block in pass 1

typedef uint16_t u16x2_t __attribute__((ext_vector_type(2)));

// Running max of |x| over 8 fp16 channels held as 4 packed dwords: with the
// sign bit cleared, fp16 bit patterns order as unsigned integers, so a
// packed 16-bit unsigned max is the exact |x| max.
__device__ inline void absmax8(uint32_t m[4], uint4 v) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const u16x2_t a = __builtin_bit_cast(u16x2_t, m[j]), b = __builtin_bit_cast(u16x2_t, w[j] & 0x7fff7fffu);
    m[j] = __builtin_bit_cast(uint32_t, __builtin_elementwise_max(a, b));
  }
}

// Thread -> (token row r of 16, channels [8 l, 8 l + 8)): a wave reads four
// whole 256-byte rows per load, 16 bytes per lane; four rows in flight per
// thread and pass.
__global__ __launch_bounds__(256) void balance_partial_kernel(const uint16_t *q, const uint16_t *k, int q_heads,
                                                              int kv_heads, int T, int nchunks, float *ws) {
  const int h = blockIdx.y, chunk = blockIdx.x;
  const int b = h / kv_heads, kvh = h % kv_heads;
  const int G = q_heads / kv_heads;
  const int l = threadIdx.x & 15, r = threadIdx.x >> 4;
  const int t0 = chunk * kBalChunk, t1 = min(t0 + kBalChunk, T);
  uint32_t km[4] = {0u, 0u, 0u, 0u}, qm[4] = {0u, 0u, 0u, 0u};
  auto scan = [&](const uint16_t *base, uint32_t m[4]) {
    const uint4 *rows = reinterpret_cast<const uint4 *>(base);
    for (int t = t0 + r; t < t1; t += 64) {
      uint4 v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = t + 16 * u < t1 ? rows[(int64_t)(t + 16 * u) * (kHeadDim / 8) + l] : uint4{0, 0, 0, 0};
#pragma unroll
      for (int u = 0; u < 4; ++u) absmax8(m, v[u]);
    }
  };
  scan(k + (int64_t)h * T * kHeadDim, km);
  for (int i = 0; i < G; ++i) scan(q + ((int64_t)b * q_heads + kvh * G + i) * T * kHeadDim, qm);
  __shared__ uint4 s_q[16][16], s_k[16][16];
  s_q[r][l] = make_uint4(qm[0], qm[1], qm[2], qm[3]);
  s_k[r][l] = make_uint4(km[0], km[1], km[2], km[3]);
  __syncthreads();
  if (threadIdx.x < kHeadDim) {  // channel c: max over the 16 rows
    const int c = threadIdx.x, lc = c / 8, j = (c % 8) / 2, hi = c % 2;
    uint32_t qb = 0u, kb = 0u;
#pragma unroll
    for (int rr = 0; rr < 16; ++rr) {
      const uint4 a = s_q[rr][lc], bk = s_k[rr][lc];
      const uint32_t aw[4] = {a.x, a.y, a.z, a.w}, bw[4] = {bk.x, bk.y, bk.z, bk.w};
      qb = max(qb, (aw[j] >> (16 * hi)) & 0xffffu);
      kb = max(kb, (bw[j] >> (16 * hi)) & 0xffffu);
    }
    float *dst = ws + ((int64_t)h * nchunks + chunk) * 2 * kHeadDim;
    dst[c] = f16_to_f32((uint16_t)qb);
    dst[kHeadDim + c] = f16_to_f32((uint16_t)kb);
  }
}

__global__ __launch_bounds__(kHeadDim) void balance_final_kernel(const float *ws, int nchunks, float *balance) {
  const int h = blockIdx.x, c = threadIdx.x;
  float qm = 0.0f, km = 0.0f;
  for (int i = 0; i < nchunks; ++i) {
    const float *src = ws + ((int64_t)h * nchunks + i) * 2 * kHeadDim;
    qm = fmaxf(qm, src[c]);
    km = fmaxf(km, src[kHeadDim + c]);
  }
  balance[(int64_t)h * kHeadDim + c] = (qm == 0.0f || km == 0.0f) ? 1.0f : sqrtf(qm / km);
}

}  // namespace

}  // namespace mikv

using namespace mikv;

extern "C" size_t mikv_balance_workspace_size(int32_t batch, int32_t kv_heads, int32_t tokens) {
  if (batch < 1 || kv_heads < 1 || tokens < 1) return 0;
  const int64_t nchunks = (tokens + kBalChunk - 1) / kBalChunk;
  return (size_t)((int64_t)batch * kv_heads * nchunks * 2 * kHeadDim * 4);
}

extern "C" int mikv_balance_channels(const uint16_t *q_prefill, const uint16_t *k_prefill, int32_t batch,
                                     int32_t q_heads, int32_t kv_heads, int32_t tokens, int32_t head_dim,
                                     float *balance, void *ws, size_t ws_bytes, void *stream) {
  if (!q_prefill || !k_prefill || !balance)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_balance_channels: NULL pointer");
  if (batch < 1 || q_heads < 1 || kv_heads < 1 || tokens < 1 || q_heads % kv_heads != 0)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_balance_channels: bad sizes");
  if (head_dim != kHeadDim) return set_error(MIKV_ERR_UNSUPPORTED, "mikv_balance_channels: head_dim must be 128");
  if (((uintptr_t)q_prefill | (uintptr_t)k_prefill) % 16 != 0)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_balance_channels: q_prefill and k_prefill must be 16-byte aligned");
  if (!ws || ws_bytes < mikv_balance_workspace_size(batch, kv_heads, tokens))
    return set_error(MIKV_ERR_CAPACITY, "mikv_balance_channels: workspace too small");
  const int nchunks = (tokens + kBalChunk - 1) / kBalChunk;
  const int NH = batch * kv_heads;
  hipStream_t st = (hipStream_t)stream;
  hipLaunchKernelGGL(balance_partial_kernel, dim3(nchunks, NH), dim3(256), 0, st, q_prefill, k_prefill, q_heads,
                     kv_heads, tokens, nchunks, (float *)ws);
  hipLaunchKernelGGL(balance_final_kernel, dim3(NH), dim3(kHeadDim), 0, st, (const float *)ws, nchunks, balance);
  return check_launch("mikv_balance_channels");
}
