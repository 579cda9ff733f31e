// Query/key channel balancer, Section 3.2, Eq. 2:
//   b[b, h, c] = sqrt( max_{t, i in group(h)} |q| / max_t |k| ),  1 if a max is 0.
// Pass 1: one block per (token chunk, head) reduces |q| and |k| per channel
// over its chunk (thread = channel, coalesced 256-byte rows) and writes the
// chunk maxima; pass 2 reduces the chunk maxima per head and applies the
// correctly rounded fp32 divide and square root.  Maxima are exact and the
// reduction order does not matter, so the result is deterministic.
#include "mikv_internal.h"

namespace mikv {

namespace {

constexpr int kBalChunk = 512;  // tokens per block in pass 1

__global__ __launch_bounds__(256) void balance_partial_kernel(const uint16_t *q, const uint16_t *k, int q_heads,
                                                              int kv_heads, int T, int nchunks, float *ws) {
  const int h = blockIdx.y, chunk = blockIdx.x;
  const int b = h / kv_heads, kvh = h % kv_heads;
  const int G = q_heads / kv_heads;
  const int c = threadIdx.x & (kHeadDim - 1), half = threadIdx.x >> 7;
  const int t0 = chunk * kBalChunk, t1 = min(t0 + kBalChunk, T);
  float qm = 0.0f, km = 0.0f;
  const uint16_t *kp = k + (int64_t)h * T * kHeadDim;
  for (int t = t0 + half; t < t1; t += 2) km = fmaxf(km, fabsf(f16_to_f32(kp[(int64_t)t * kHeadDim + c])));
  for (int i = 0; i < G; ++i) {
    const uint16_t *qp = q + ((int64_t)b * q_heads + kvh * G + i) * T * kHeadDim;
    for (int t = t0 + half; t < t1; t += 2) qm = fmaxf(qm, fabsf(f16_to_f32(qp[(int64_t)t * kHeadDim + c])));
  }
  __shared__ float s_q[kHeadDim], s_k[kHeadDim];
  if (half == 1) {
    s_q[c] = qm;
    s_k[c] = km;
  }
  __syncthreads();
  if (half == 0) {
    float *dst = ws + ((int64_t)h * nchunks + chunk) * 2 * kHeadDim;
    dst[c] = fmaxf(qm, s_q[c]);
    dst[kHeadDim + c] = fmaxf(km, s_k[c]);
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
