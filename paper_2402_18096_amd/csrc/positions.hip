// Position-indexed forms of the step's probabilities and scores.  The
// attention writes each pool's probabilities in slot order (the order the
// pools hold their tokens); mikv_probs_by_position scatters them into
// [B, Hq, length] position order through the pools' position maps, the
// layout in which the step's probabilities are stated (softmax over the token
// positions, Section 3.4 / Fig. 3).  mikv_importance_update_positions is the
// H2O accumulation (Sections 3.1, 4.1) over such position-indexed rows.
#include <algorithm>

#include "mikv_internal.h"

namespace mikv {

namespace {

constexpr int kPosBlock = 256;

__global__ __launch_bounds__(kPosBlock) void zero_rows_kernel(float *probs, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * kPosBlock + threadIdx.x; i < n; i += (int64_t)gridDim.x * kPosBlock)
    probs[i] = 0.0f;
}

// Block (x, h, pool): slots [x * kPosBlock, ...) of KV head h's pool; every
// query head of the group gets the slot's probability at the slot's position.
__global__ __launch_bounds__(kPosBlock) void scatter_positions_kernel(const float *probs_hi, const float *probs_lo,
                                                                     const int32_t *hi_pos, const int32_t *lo_pos,
                                                                     const int32_t *n_hi, const int32_t *n_lo, int cap_hi,
                                                                     int cap_lo, int q_heads, int kv_heads, int length,
                                                                     float *probs) {
  const int h = blockIdx.y, is_lo = blockIdx.z;
  const int cap = is_lo ? cap_lo : cap_hi;
  const int n = min(is_lo ? n_lo[h] : n_hi[h], cap);
  const int s = blockIdx.x * kPosBlock + threadIdx.x;
  if (s >= n) return;
  const int pos = (is_lo ? lo_pos : hi_pos)[(int64_t)h * cap + s];
  if (pos < 0 || pos >= length) return;
  const float *src = is_lo ? probs_lo : probs_hi;
  const int G = q_heads / kv_heads, b = h / kv_heads, kvh = h % kv_heads;
  for (int i = 0; i < G; ++i) {
    const int64_t qh = (int64_t)b * q_heads + kvh * G + i;
    probs[qh * length + pos] = src[qh * cap + s];
  }
}

// Block (x, h): positions [x * kPosBlock, ...) of KV head h = b * Hkv + k.
// The group's probabilities are summed left to right in query-head order,
// then added to the score once (fp32 throughout).
__global__ __launch_bounds__(kPosBlock) void importance_positions_kernel(float *acc, const float *probs, int q_heads,
                                                                        int kv_heads, int length, int64_t max_len) {
  const int h = blockIdx.y;
  const int j = blockIdx.x * kPosBlock + threadIdx.x;
  if (j >= length) return;
  const int G = q_heads / kv_heads, b = h / kv_heads, kvh = h % kv_heads;
  const float *p = probs + ((int64_t)b * q_heads + (int64_t)kvh * G) * max_len + j;
  float sum = p[0];
  for (int i = 1; i < G; ++i) sum = sum + p[(int64_t)i * max_len];
  acc[(int64_t)h * max_len + j] += sum;
}

}  // namespace

}  // namespace mikv

using namespace mikv;

extern "C" int mikv_probs_by_position(const mikv_cache *c, int32_t length, const float *probs_hi,
                                      const float *probs_lo, float *probs, void *stream) {
  if (int e = validate_cache(c)) return e;
  if (!probs_hi || !probs || (!evicting(c) && !probs_lo))
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_probs_by_position: NULL pointer");
  if (length < 1) return set_error(MIKV_ERR_INVALID_ARG, "mikv_probs_by_position: length must be >= 1");
  if (length > c->max_len)
    return set_error(MIKV_ERR_CAPACITY, "mikv_probs_by_position: length %d exceeds max_len %d", length, c->max_len);
  hipStream_t st = (hipStream_t)stream;
  const int64_t total = (int64_t)c->batch * c->q_heads * length;
  const int zblocks = (int)std::min<int64_t>(4096, (total + kPosBlock - 1) / kPosBlock);
  hipLaunchKernelGGL(zero_rows_kernel, dim3(zblocks), dim3(kPosBlock), 0, st, probs, total);
  const int cap = std::max(c->cap_hi, evicting(c) ? 0 : c->cap_lo);
  dim3 grid((cap + kPosBlock - 1) / kPosBlock, n_heads_of(c), evicting(c) ? 1 : 2);
  hipLaunchKernelGGL(scatter_positions_kernel, grid, dim3(kPosBlock), 0, st, probs_hi, probs_lo, c->hi_pos,
                     c->lo_pos, c->n_hi, c->n_lo, c->cap_hi, evicting(c) ? 0 : c->cap_lo, c->q_heads, c->kv_heads,
                     length, probs);
  return check_launch("mikv_probs_by_position");
}

extern "C" int mikv_importance_update_positions(float *acc, const float *probs, int32_t batch, int32_t q_heads,
                                                int32_t kv_heads, int32_t length, int32_t max_len, void *stream) {
  if (!acc || !probs) return set_error(MIKV_ERR_INVALID_ARG, "mikv_importance_update_positions: NULL pointer");
  if (batch < 1 || q_heads < 1 || kv_heads < 1 || max_len < 1)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_importance_update_positions: batch, q_heads, kv_heads and max_len "
                                           "must be >= 1");
  if (q_heads % kv_heads != 0)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_importance_update_positions: q_heads (%d) not a multiple of "
                                           "kv_heads (%d)", q_heads, kv_heads);
  if (length < 0) return set_error(MIKV_ERR_INVALID_ARG, "mikv_importance_update_positions: length must be >= 0");
  if (length > max_len)
    return set_error(MIKV_ERR_CAPACITY, "mikv_importance_update_positions: length %d exceeds max_len %d", length,
                     max_len);
  if (length == 0) return MIKV_OK;
  dim3 grid((length + kPosBlock - 1) / kPosBlock, batch * kv_heads);
  hipLaunchKernelGGL(importance_positions_kernel, grid, dim3(kPosBlock), 0, (hipStream_t)stream, acc, probs, q_heads,
                     kv_heads, length, (int64_t)max_len);
  return check_launch("mikv_importance_update_positions");
}
