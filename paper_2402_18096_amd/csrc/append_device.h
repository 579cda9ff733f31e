// Device side of the Eq. 1 quantizer for single rows and of the append of
// one decoded token to the importance pool (Sections 3.1, 3.2), shared by
// the quantize kernels and the decode-step attention kernel, which folds the
// append of the new token into its own launch.
#ifndef MIKV_APPEND_DEVICE_H
#define MIKV_APPEND_DEVICE_H

#include "mikv_internal.h"

namespace mikv {

namespace {

// Load 32 fp16 channels starting at `src` (16-byte aligned) into fp32,
// multiplied by the balancer when one is given (Eq. 3; one fp32 product).
__device__ inline void load_row_segment(const uint16_t *src, const float *bal, float x[32]) {
  const uint4 *s4 = reinterpret_cast<const uint4 *>(src);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint4 w = s4[i];
    uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[i * 8 + 2 * j] = f16_to_f32((uint16_t)(ws[j] & 0xffffu));
      x[i * 8 + 2 * j + 1] = f16_to_f32((uint16_t)(ws[j] >> 16));
    }
  }
  if (bal) {
#pragma unroll
    for (int c = 0; c < 32; ++c) x[c] = x[c] * bal[c];
  }
}

// Eq. 1 codes of one 32-channel segment at BITS: group min/max (a group of
// g channels spans g/32 adjacent lanes, combined with shuffles), the group's
// fp16 (alpha, beta) and the packed little-endian words w[BITS].
template <int BITS>
__device__ inline GroupParams quantize_words(const float x[32], int group, uint32_t w[BITS]) {
  float mn = x[0], mx = x[0];
#pragma unroll
  for (int c = 1; c < 32; ++c) {
    mn = fminf(mn, x[c]);
    mx = fmaxf(mx, x[c]);
  }
  // combine across the lanes of one group (group/32 lanes, aligned)
  for (int o = 1; o < group / 32; o <<= 1) {
    mn = fminf(mn, __shfl_xor(mn, o, 64));
    mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  }
  GroupParams p = group_params(mn, mx, BITS);
  encode32<BITS>(x, p, w);
  return p;
}

// Quantize one 32-channel segment (lane part `lane4` of its row) at BITS:
// writes the packed codes (32*BITS/8 bytes at `codes`) and, from the first
// lane of each group, the (alpha, beta) pair at `param`.
template <int BITS>
__device__ inline void quantize_segment(const float x[32], int group, int lane4, uint8_t *codes,
                                        uint32_t *param, bool store) {
  uint32_t w[BITS];
  GroupParams p = quantize_words<BITS>(x, group, w);
  if (!store) return;
  uint32_t *dst = reinterpret_cast<uint32_t *>(codes);
#pragma unroll
  for (int i = 0; i < BITS; ++i) dst[i] = w[i];
  if ((lane4 % (group / 32)) == 0) *param = (uint32_t)p.a16 | ((uint32_t)p.b16 << 16);
}

// Where one new token goes: the importance pool (rows, group parameters,
// positions, scores), the position map and the status word, and the token's
// key and value rows ([B * Hkv, 128] fp16) with the key balancer.
struct AppendArgs {
  uint8_t *hi_k, *hi_v;     // fp16 rows or INT8 codes
  uint32_t *hi_kp, *hi_vp;  // (alpha, beta) pairs of INT8 rows
  int32_t *hi_pos;
  float *hi_acc;
  uint8_t *map;             // nullable
  int32_t *status;
  const uint16_t *k, *v;    // the new token's rows
  const float *balance;     // nullable (Eq. 3)
  const float *score_init;  // nullable: initial score 0
  int cap_hi, max_len, group, pos;
};

// Writes the new token of head h into importance-pool slot `slot` (an index
// below cap_hi): 8 lanes, 0-3 the key row's 32-channel segments, 4-7 the
// value row's; lane 0 also records the position, the initial score and the
// map entry.  The pool count is the caller's.
template <int HI_BITS>
__device__ inline void append_row(const AppendArgs &P, int h, int slot, int lane8) {
  const int is_v = lane8 >> 2, lane4 = lane8 & 3;
  const float *bal = (!is_v && P.balance) ? P.balance + (int64_t)h * kHeadDim + lane4 * 32 : nullptr;
  float x[32];
  load_row_segment(lane_pick(is_v, P.v, P.k) + (int64_t)h * kHeadDim + lane4 * 32, bal, x);
  const int64_t row = (int64_t)h * P.cap_hi + slot;
  if constexpr (HI_BITS == 16) {
    uint32_t w[16];
#pragma unroll
    for (int c = 0; c < 16; ++c) w[c] = pack_f16x2(x[2 * c], x[2 * c + 1]);
    uint4 *d4 = reinterpret_cast<uint4 *>(lane_pick(is_v, P.hi_v, P.hi_k) + (row * kHeadDim + lane4 * 32) * 2);
#pragma unroll
    for (int i = 0; i < 4; ++i) d4[i] = make_uint4(w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]);
  } else {
    const int ng = kHeadDim / P.group;
    uint8_t *dst = lane_pick(is_v, P.hi_v, P.hi_k) + row * (kHeadDim * HI_BITS / 8) + lane4 * (32 * HI_BITS / 8);
    uint32_t *par = lane_pick(is_v, P.hi_vp, P.hi_kp) + row * ng + (lane4 * 32) / P.group;
    quantize_segment<HI_BITS>(x, P.group, lane4, dst, par, true);
  }
  if (lane8 == 0) {
    P.hi_pos[row] = P.pos;
    P.hi_acc[row] = P.score_init ? P.score_init[h] : 0.0f;
    if (P.map) P.map[(int64_t)h * P.max_len + P.pos] = 1;
  }
}

}  // namespace

}  // namespace mikv

#endif  // MIKV_APPEND_DEVICE_H
