// Importance scores of the prompt tokens (the H2O accumulated attention at
// the end of prefill, Section 3.1 / Section 4.1): every prompt query i
// attends causally to keys 0..i, and token j's score is the sum of its
// softmax probabilities over all queries i >= j and over the query heads
// that share its KV head,
//   score[b, h, j] = sum_{g in group(h)} sum_{i >= j} softmax_i(q_i . k / sqrt(d))_j.
// The logits are a dense contraction (Q K^T per head), so both passes run
// on the matrix cores (v_mfma_f32_16x16x32_f16, fp16 operands as given,
// fp32 accumulation):
//   pass 1  one wave per 64 queries of one query head: online row maximum
//           (raised lazily) and normaliser over the causal keys, in log2 units;
//   pass 2  one wave per 64 keys of one KV head: recomputes the same 16x16
//           logit tiles (bit-identical: same operands, same tile origin),
//           turns them into probabilities with the pass-1 statistics and
//           sums them down the columns, over every query head of the group.
// Tiles entirely below the causal diagonal and inside the prompt (nearly
// all of them) skip the mask.
// Lane l = 16 a + n of a wave: A operand = rows n of the query tile, B
// operand = rows n of the key tile, each lane taking channels
// [32 c + 8 a, 32 c + 8 a + 8) of MFMA c (the same split on both sides, so
// the four MFMAs cover all 128 channels); the result holds logit rows
// 4 a .. 4 a + 3 of column n.
#include "mikv_internal.h"

namespace mikv {

namespace {

constexpr int kTileBlocks = 4;  // 16-row tiles per wave in each pass (64 rows)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLazy = 8.0f;   // raise a row's running maximum only past this (log2 units)

typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));

__device__ inline h8_t as_h8(uint4 v) { return __builtin_bit_cast(h8_t, v); }

// Operand of MFMA c for row `row` of a [T, 128] fp16 matrix (zero past T).
__device__ inline void load_rows(const uint16_t *base, int row, int T, int a, uint4 op[4]) {
#pragma unroll
  for (int c = 0; c < 4; ++c)
    op[c] = row < T ? *reinterpret_cast<const uint4 *>(base + (int64_t)row * kHeadDim + 32 * c + 8 * a)
                    : make_uint4(0u, 0u, 0u, 0u);
}

__device__ inline f4_t logits(const uint4 aq[4], const uint4 bk[4]) {
  f4_t d = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
  for (int c = 0; c < 4; ++c) d = __builtin_amdgcn_mfma_f32_16x16x32_f16(as_h8(aq[c]), as_h8(bk[c]), d, 0, 0, 0);
  return d;
}

// Reductions over the 16 lanes of one row of the wave (one logit row).
__device__ inline float max16(float v) {
  v = fmaxf(v, dpp_mov<0xB1>(v));
  v = fmaxf(v, dpp_mov<0x4E>(v));
  v = fmaxf(v, dpp_mov<0x141>(v));
  return fmaxf(v, dpp_mov<0x140>(v));
}
__device__ inline float sum16(float v) {
  v += dpp_mov<0xB1>(v);
  v += dpp_mov<0x4E>(v);
  v += dpp_mov<0x141>(v);
  return v + dpp_mov<0x140>(v);
}

// Pass 1: (max, normaliser) of every query row, log2 units.
__global__ __launch_bounds__(64) void prefill_rowstats_kernel(const uint16_t *q, const uint16_t *k, int q_heads,
                                                              int kv_heads, int T, float s2scale, float2 *stats) {
  const int lane = threadIdx.x, n = lane & 15, a = lane >> 4;
  const int qh = blockIdx.y, b = qh / q_heads, hq = qh % q_heads;
  const int hk = b * kv_heads + hq / (q_heads / kv_heads);
  const int i_base = blockIdx.x * 16 * kTileBlocks;
  const uint16_t *qb = q + (int64_t)qh * T * kHeadDim, *kb = k + (int64_t)hk * T * kHeadDim;
  uint4 aq[kTileBlocks][4];
#pragma unroll
  for (int rb = 0; rb < kTileBlocks; ++rb) load_rows(qb, i_base + 16 * rb + n, T, a, aq[rb]);
  // Lazy row maximum (log2 units, the same in the 16 lanes of a row): raised
  // only when a logit exceeds it by more than kLazy, decided for the whole
  // wave with one ballot, so the common tile needs no cross-lane reduction;
  // each lane sums its own exp2 terms, reduced once at the end.
  float m[kTileBlocks][4], l[kTileBlocks][4];
#pragma unroll
  for (int rb = 0; rb < kTileBlocks; ++rb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      m[rb][r] = -__builtin_huge_valf();
      l[rb][r] = 0.0f;
    }
  const int j_end = min(T, i_base + 16 * kTileBlocks);  // keys past the last query are masked
  for (int j0 = 0; j0 < j_end; j0 += 16) {
    uint4 bk[4];
    load_rows(kb, j0 + n, T, a, bk);
    const int kj = j0 + n;
#pragma unroll
    for (int rb = 0; rb < kTileBlocks; ++rb) {
      if (j0 > i_base + 16 * rb + 15) continue;  // tile above the diagonal (wave-uniform)
      const f4_t d = logits(aq[rb], bk);
      // a tile below the diagonal and inside the prompt needs no mask
      const bool full = j0 + 15 <= i_base + 16 * rb && i_base + 16 * rb + 15 < T;  // wave-uniform
      float s[4];
      bool raise = false;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int qi = i_base + 16 * rb + 4 * a + r;
        s[r] = full || (kj <= qi && qi < T) ? d[r] * s2scale : -__builtin_huge_valf();
        raise = raise || s[r] > m[rb][r] + kLazy;
      }
      if (__ballot(raise)) {  // wave-uniform
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float mn = fmaxf(m[rb][r], max16(s[r]));
          if (mn != m[rb][r]) {  // row-uniform; mn is finite here
            l[rb][r] *= m[rb][r] == -__builtin_huge_valf() ? 0.0f : __builtin_amdgcn_exp2f(m[rb][r] - mn);
            m[rb][r] = mn;
          }
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) l[rb][r] += s[r] == -__builtin_huge_valf() ? 0.0f : __builtin_amdgcn_exp2f(s[r] - m[rb][r]);
    }
  }
#pragma unroll
  for (int rb = 0; rb < kTileBlocks; ++rb)
#pragma unroll
    for (int r = 0; r < 4; ++r) l[rb][r] = sum16(l[rb][r]);
  if (n == 0) {
#pragma unroll
    for (int rb = 0; rb < kTileBlocks; ++rb)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int qi = i_base + 16 * rb + 4 * a + r;
        if (qi < T) stats[(int64_t)qh * T + qi] = make_float2(m[rb][r], 1.0f / l[rb][r]);
      }
  }
}

// Pass 2: column sums of the probabilities, over the causal queries of every
// query head of the KV head's group.  Grid x runs over key blocks from the
// first (the longest column) on.
__global__ __launch_bounds__(64) void prefill_colsum_kernel(const uint16_t *q, const uint16_t *k, int q_heads,
                                                            int kv_heads, int T, float s2scale, const float2 *stats,
                                                            float *scores) {
  const int lane = threadIdx.x, n = lane & 15, a = lane >> 4;
  const int hk = blockIdx.y, b = hk / kv_heads, kvh = hk % kv_heads;
  const int G = q_heads / kv_heads;
  const int j_base = blockIdx.x * 16 * kTileBlocks;
  const uint16_t *kb = k + (int64_t)hk * T * kHeadDim;
  uint4 bk[kTileBlocks][4];
#pragma unroll
  for (int cb = 0; cb < kTileBlocks; ++cb) load_rows(kb, j_base + 16 * cb + n, T, a, bk[cb]);
  float cs[kTileBlocks];
#pragma unroll
  for (int cb = 0; cb < kTileBlocks; ++cb) cs[cb] = 0.0f;
  for (int g = 0; g < G; ++g) {
    const int qh = b * q_heads + kvh * G + g;
    const uint16_t *qb = q + (int64_t)qh * T * kHeadDim;
    const float2 *st = stats + (int64_t)qh * T;
    for (int i0 = j_base; i0 < T; i0 += 16) {
      uint4 aq[4];
      load_rows(qb, i0 + n, T, a, aq);
      float2 ml[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int qi = i0 + 4 * a + r;
        ml[r] = qi < T ? st[qi] : make_float2(0.0f, 0.0f);
      }
#pragma unroll
      for (int cb = 0; cb < kTileBlocks; ++cb) {
        if (j_base + 16 * cb > i0 + 15) continue;  // tile above the diagonal (wave-uniform)
        const f4_t d = logits(aq, bk[cb]);
        const int kj = j_base + 16 * cb + n;
        // a tile below the diagonal and inside the prompt needs no mask;
        // the exponent is one fused multiply-add (within an ulp of pass 1's)
        const bool full = j_base + 16 * cb + 15 <= i0 && i0 + 15 < T;  // wave-uniform
        if (full) {
#pragma unroll
          for (int r = 0; r < 4; ++r)
            cs[cb] = fmaf(__builtin_amdgcn_exp2f(fmaf(d[r], s2scale, -ml[r].x)), ml[r].y, cs[cb]);
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int qi = i0 + 4 * a + r;
            const bool valid = kj <= qi && qi < T;
            const float p = __builtin_amdgcn_exp2f(fmaf(d[r], s2scale, -ml[r].x)) * ml[r].y;
            cs[cb] += valid ? p : 0.0f;
          }
        }
      }
    }
  }
#pragma unroll
  for (int cb = 0; cb < kTileBlocks; ++cb) {
    float v = cs[cb] + __shfl_xor(cs[cb], 16, 64);
    v += __shfl_xor(v, 32, 64);
    const int kj = j_base + 16 * cb + n;
    if (a == 0 && kj < T) scores[(int64_t)hk * T + kj] = v;
  }
}

}  // namespace

}  // namespace mikv

using namespace mikv;

extern "C" size_t mikv_prefill_importance_workspace_size(int32_t batch, int32_t q_heads, int32_t tokens) {
  if (batch < 1 || q_heads < 1 || tokens < 1) return 0;
  return (size_t)((int64_t)batch * q_heads * tokens * 8);
}

extern "C" int mikv_prefill_importance(const uint16_t *q_prefill, const uint16_t *k_prefill, int32_t batch,
                                       int32_t q_heads, int32_t kv_heads, int32_t tokens, int32_t head_dim,
                                       float scale, float *scores, void *ws, size_t ws_bytes, void *stream) {
  if (!q_prefill || !k_prefill || !scores)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_prefill_importance: NULL pointer");
  if (batch < 1 || q_heads < 1 || kv_heads < 1 || tokens < 1 || q_heads % kv_heads != 0)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_prefill_importance: bad sizes");
  const int G = q_heads / kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return set_error(MIKV_ERR_UNSUPPORTED, "mikv_prefill_importance: query heads per KV head must be 1, 2, 4 or 8");
  if (head_dim != kHeadDim) return set_error(MIKV_ERR_UNSUPPORTED, "mikv_prefill_importance: head_dim must be 128");
  if (!(scale > 0.0f)) return set_error(MIKV_ERR_INVALID_ARG, "mikv_prefill_importance: scale must be > 0");
  if (((uintptr_t)q_prefill | (uintptr_t)k_prefill) % 16 != 0)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_prefill_importance: q_prefill and k_prefill must be 16-byte aligned");
  if (!ws || ws_bytes < mikv_prefill_importance_workspace_size(batch, q_heads, tokens))
    return set_error(MIKV_ERR_CAPACITY, "mikv_prefill_importance: workspace too small");
  const int blocks = (tokens + 16 * kTileBlocks - 1) / (16 * kTileBlocks);
  const float s2scale = scale * kLog2e;
  hipStream_t st = (hipStream_t)stream;
  float2 *stats = (float2 *)ws;
  hipLaunchKernelGGL(prefill_rowstats_kernel, dim3(blocks, batch * q_heads), dim3(64), 0, st, q_prefill, k_prefill,
                     q_heads, kv_heads, tokens, s2scale, stats);
  hipLaunchKernelGGL(prefill_colsum_kernel, dim3(blocks, batch * kv_heads), dim3(64), 0, st, q_prefill, k_prefill,
                     q_heads, kv_heads, tokens, s2scale, (const float2 *)stats, scores);
  return check_launch("mikv_prefill_importance");
}
