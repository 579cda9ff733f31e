// Internal helpers of libmikv: device math shared by the kernels, and host
// validation/error plumbing shared by the entry points.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <cstdarg>
#include <cstdio>

#include "../../include/mikv.h"

namespace mikv {

constexpr int kHeadDim = 128;
constexpr int kKeyBlock = 64;  // positions per block of per-channel key parameters

// Default bytes of a cache the attention reads with plain loads each step
// (the rest it streams with non-temporal loads): what the 256 MB last-level
// cache keeps from one step to the next next to the step's other traffic
// (measured on long_context: 160 MB 98.9, 192 MB 98.2, 224 MB 95.5 us per
// attention launch).  mikv_set_resident_bytes changes it at run time.
#ifndef MIKV_RESIDENT_MB
#define MIKV_RESIDENT_MB 224
#endif
constexpr int64_t kResidentBytes = (int64_t)MIKV_RESIDENT_MB << 20;

// ---------------------------------------------------------------------------
// Host: error reporting.
// ---------------------------------------------------------------------------
int set_error(int code, const char *fmt, ...);
int check_launch(const char *what);

// Validate a cache descriptor (host side, before any launch).
int validate_cache(const mikv_cache *c);

// Internal launches of the decode step (attention.hip): the attention's
// partial phase, which with k_new/v_new non-NULL also appends the new token
// (position length - 1) to the importance pool, leaving n_hi to the
// finalize; and the finalize with the importance update and the re-rank
// fused (block 0 of each head updates the head's scores, then runs its
// select), which with `appended` set counts that token into n_hi.
int decode_partial(const mikv_cache *c, int32_t length, const uint16_t *q, const float *balance, float scale,
                   float *out, float *probs_hi, float *probs_lo, int32_t flags, void *ws, size_t ws_bytes,
                   const uint16_t *k_new, const uint16_t *v_new, hipStream_t st);
int decode_finalize_select(const mikv_cache *c, int32_t length, const uint16_t *q, const float *balance, float scale,
                           float *out, float *probs_hi, float *probs_lo, void *ws, size_t ws_bytes, int32_t k_heavy,
                           int32_t window, void *sel_ws, bool appended, hipStream_t st);
// The separate finalize and re-rank launches of the decode step (caches with
// many heads), with the same meaning of `appended` (attention.hip,
// select.hip).
int decode_finalize(const mikv_cache *c, int32_t length, const uint16_t *q, const float *balance, float scale,
                    float *out, float *probs_hi, float *probs_lo, int32_t flags, void *ws, size_t ws_bytes,
                    bool appended, hipStream_t st);
int select_topk(const mikv_cache *c, int32_t length, int32_t k_heavy, int32_t window, void *ws, size_t ws_bytes,
                bool appended, hipStream_t st);

inline int group_size_of(const mikv_cache *c) { return c->q_heads / c->kv_heads; }
// lo_bits == 0: no retained pool; tokens that leave the importance pool are
// evicted (the 0-bit retained cache, i.e. H2O eviction).
inline bool evicting(const mikv_cache *c) { return c->lo_bits == 0; }
// Key of the kernel instantiation for the cache's formats.  An evicting
// cache runs the 2-bit instantiation with its retained pool empty.
inline int format_key(const mikv_cache *c) { return c->hi_bits * 100 + (evicting(c) ? 2 : c->lo_bits); }
inline int n_heads_of(const mikv_cache *c) { return c->batch * c->kv_heads; }
// Blocks of per-channel key parameters per head (key_block 64).
inline int key_blocks_of(const mikv_cache *c) { return c->max_len / kKeyBlock; }

// Per-channel key parameters of key block `blk` from the keys of its 64
// positions in the importance pool (quantize.hip): the block completed
// during decoding.  key_block caches only.
int close_key_block_from_pool(const mikv_cache *c, int32_t blk, hipStream_t st);

// Bytes of one token (key + value, codes + fp16 params) in a pool of `bits`.
inline int64_t token_bytes(int bits, int group) {
  if (bits == 16) return 2 * kHeadDim * 2;
  return 2 * (kHeadDim * bits / 8 + 4 * (kHeadDim / group));
}

// ---------------------------------------------------------------------------
// Device: exact arithmetic helpers.
// ---------------------------------------------------------------------------

// fp32 -> fp16, round to nearest even, from the IEEE 754 binary16 definition
// in integer arithmetic (exact also for fp16 subnormal results, independent
// of the hardware conversion's denormal mode).
__host__ __device__ inline uint16_t f32_to_f16_rne(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  uint32_t sign = (u >> 16) & 0x8000u;
  uint32_t a = u & 0x7fffffffu;
  if (a >= 0x7f800000u) return (uint16_t)(sign | 0x7c00u | (a > 0x7f800000u ? 0x200u : 0u));
  if (a >= 0x477ff000u) return (uint16_t)(sign | 0x7c00u);  // rounds to infinity
  if (a < 0x38800000u) {                                      // fp16 subnormal or zero
    uint32_t e = a >> 23;
    if (e < 102u) return (uint16_t)sign;                      // below half the smallest subnormal
    uint32_t m = (a & 0x7fffffu) | 0x800000u;
    uint32_t s = 126u - e;                                    // 14 .. 24
    uint32_t r = m >> s;
    uint32_t rem = m & ((1u << s) - 1u);
    uint32_t half = 1u << (s - 1u);
    if (rem > half || (rem == half && (r & 1u))) ++r;
    return (uint16_t)(sign | r);
  }
  uint32_t r = ((a >> 23) - 112u) << 10 | ((a >> 13) & 0x3ffu);
  uint32_t rem = a & 0x1fffu;
  if (rem > 0x1000u || (rem == 0x1000u && (r & 1u))) ++r;
  return (uint16_t)(sign | r);
}

// Two fp32 values to an fp16 pair (low half first) with the hardware
// conversion: IEEE round to nearest even, fp16 subnormals kept (the default
// floating-point mode these kernels run in).  Used for stored fp16 rows; the
// per-group scale and zero use f32_to_f16_rne above.
__device__ inline uint32_t pack_f16x2(float lo, float hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)lo) |
         ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)hi) << 16);
}

__device__ inline float f16_to_f32(uint16_t h) {
  return (float)__builtin_bit_cast(_Float16, h);
}

// Order-preserving map of an fp32 score to uint32 (-0 treated as +0).
__device__ inline uint32_t ordered_bits(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  if (u == 0x80000000u) u = 0u;
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Eq. 1 parameters of one group from its min and max (fp32), exactly as the
// stored format defines them.  The library is compiled with
// -ffp-contract=off, so every operator below is one correctly rounded fp32
// operation (division included: hipcc's default is the correctly rounded
// fp32 divide and square root); fused multiply-adds are only those written
// explicitly with fmaf.
struct GroupParams {
  uint16_t a16, b16;
  float a, b;
};

__device__ inline GroupParams group_params(float mn, float mx, int bits) {
  GroupParams p;
  float top = (float)((1 << bits) - 1);
  float alpha32 = (mx - mn) / top;
  p.a16 = f32_to_f16_rne(alpha32);
  p.b16 = f32_to_f16_rne(mn);
  p.a = f16_to_f32(p.a16);
  p.b = f16_to_f32(p.b16);
  return p;
}

__device__ inline uint32_t encode(float x, const GroupParams &p, int bits) {
  if (p.a == 0.0f) return 0u;
  float t = rintf((x - p.b) / p.a);
  float top = (float)((1 << bits) - 1);
  t = fminf(fmaxf(t, 0.0f), top);
  return (uint32_t)t;
}

// Put code `v` of channel c (of a lane's 32) into the packed little-endian
// words w[BITS], least significant bits first; a 3-bit code can straddle two
// words.
template <int BITS>
__device__ inline void put_code(uint32_t w[BITS], int c, uint32_t v) {
  const int bit = c * BITS, wi = bit / 32, sh = bit % 32;
  w[wi] |= v << sh;
  if (sh + BITS > 32) w[wi + 1] |= v >> (32 - sh);
}

// encode() of the 32 values of one lane's segment, packed LSB-first into
// w[BITS], without a divide per value: the quotient (x - beta) / alpha is
// estimated as (x - beta) * fl(1 / alpha), within 1.5 ulp of the correctly
// rounded quotient.  The rounded code can only differ where a half-integer
// lies between the two, so where an estimate is within 2^-20 (relative) of
// a half-integer the wave recomputes its quotients with the true divide;
// the codes are then those of encode() bit for bit.
template <int BITS>
__device__ inline void encode32(const float x[32], const GroupParams &p, uint32_t w[BITS]) {
  const float top = (float)((1 << BITS) - 1);
  const bool zero = p.a == 0.0f;
  const float ra = zero ? 0.0f : 1.0f / p.a;
  float q[32];
  bool near = false;
#pragma unroll
  for (int c = 0; c < 32; ++c) {
    q[c] = (x[c] - p.b) * ra;
    const float f = q[c] - floorf(q[c]);
    near = near || fabsf(f - 0.5f) <= fmaxf(fabsf(q[c]), 1.0f) * 0x1p-20f;
  }
  if (__ballot(near)) {
#pragma unroll
    for (int c = 0; c < 32; ++c) q[c] = zero ? 0.0f : (x[c] - p.b) / p.a;
  }
#pragma unroll
  for (int i = 0; i < BITS; ++i) w[i] = 0u;
#pragma unroll
  for (int c = 0; c < 32; ++c) put_code<BITS>(w, c, (uint32_t)fminf(fmaxf(rintf(q[c]), 0.0f), top));
}

// Eq. 1 codes of the 32 channels [32 * lane4, 32 * lane4 + 32) of a key with
// its block's per-channel parameters, packed LSB-first into w[BITS].
template <int BITS>
__device__ inline void encode_key_channels(const float x[32], const uint32_t *blk_par, int lane4, uint32_t w[BITS]) {
#pragma unroll
  for (int i = 0; i < BITS; ++i) w[i] = 0u;
  const uint4 *p4 = reinterpret_cast<const uint4 *>(blk_par + lane4 * 32);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint4 pw = p4[j];
    const uint32_t ws[4] = {pw.x, pw.y, pw.z, pw.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      GroupParams gp;
      gp.a16 = (uint16_t)(ws[e] & 0xffffu);
      gp.b16 = (uint16_t)(ws[e] >> 16);
      gp.a = f16_to_f32(gp.a16);
      gp.b = f16_to_f32(gp.b16);
      put_code<BITS>(w, 4 * j + e, encode(x[4 * j + e], gp, BITS));
    }
  }
}

// c ? a : b for wave-uniform pointers (argument fields) and a per-lane
// condition, selected as values: a select between two fields of an argument
// struct can otherwise become a per-lane indexed load from the struct, which
// the compiler serves by copying the whole struct to scratch memory.
template <class T>
__device__ inline T *lane_pick(bool c, T *a, T *b) {
  const uint64_t ua = (uint64_t)a, ub = (uint64_t)b;
  const uint64_t fa = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(ua >> 32)) << 32) |
                      (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)ua);
  const uint64_t fb = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(ub >> 32)) << 32) |
                      (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)ub);
  return reinterpret_cast<T *>(c ? fa : fb);
}

// ---------------------------------------------------------------------------
// Retained-pool 2-bit value codes for GQA: tiles of 32 slots.
// Byte q (0..31) of a slot interleaves the four 32-channel segments: it
// holds channels q, q + 32, q + 64 and q + 96 at bits 0-1, 2-3, 4-5 and 6-7.
// In a tile (1024 bytes) byte q of slot s sits at
//   16 * (16 * (s % 32 / 8) + q % 16) + 8 * (q / 16) + s % 8:
// the 16 bytes at 16 l are bytes l % 16 and l % 16 + 16 of the 8 slots
// 8 (l / 16) .. 8 (l / 16) + 7, which is what lane l of the decode
// attention's value product uses (every field of every byte: one matrix-core
// column block per segment, tokens along the reduction).
// ---------------------------------------------------------------------------
// The tiled value layout is used where the matrix cores read it: 2-bit
// retained pools shared by two or more query heads (GQA).  With one query
// head per KV head the values stay token-major (the vector path reads a
// token's row per lane).
__host__ __device__ inline bool int2_values_tiled(int lo_bits, int q_heads, int kv_heads) {
  return lo_bits == 2 && q_heads >= 2 * kv_heads;
}

__host__ __device__ inline int64_t int2_v_byte(int64_t slot, int q) {
  return (slot >> 5) * 1024 + 16 * (16 * ((slot & 31) >> 3) + (q & 15)) + 8 * (q >> 4) + (slot & 7);
}

// Store a slot's 2-bit value row into the tiled layout.  Called by the four
// lanes of the row together (lanes 4k .. 4k+3 of the wave, segment `part` =
// lane % 4, each with the 64 codes of its segment, channel 32 part + c at
// bit 2c of w[0] | w[1] << 32): lane `part` gathers the 16-bit chunk `part`
// of every segment's codes and writes bytes 8 part .. 8 part + 7.
__device__ inline void store_int2_v(uint8_t *head_base, int64_t slot, int part, const uint32_t w[2]) {
  uint32_t lo = 0u, hi = 0u;  // the lane's bytes 0-3 and 4-7
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    // round r: this lane sends chunk part ^ r of its own segment and
    // receives chunk `part` of segment part ^ r
    const int want = part ^ r;
    const uint32_t mine = (((want & 2) ? w[1] : w[0]) >> (16 * (want & 1))) & 0xffffu;
    const uint32_t c = r == 0 ? mine : (uint32_t)__shfl_xor((int)mine, r, 64);
    const int sh = 2 * (part ^ r);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t f = ((c >> (2 * e)) & 3u) << sh;
      if (e < 4)
        lo |= f << (8 * e);
      else
        hi |= f << (8 * (e - 4));
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e)
    head_base[int2_v_byte(slot, 8 * part + e)] = (uint8_t)(((e < 4 ? lo : hi) >> (8 * (e & 3))) & 0xffu);
}

// ---------------------------------------------------------------------------
// Device: wave-level reductions (wave64).
// ---------------------------------------------------------------------------
template <int WIDTH>
__device__ inline float sum_lanes(float v) {
#pragma unroll
  for (int o = WIDTH / 2; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Whole-wave reductions (every lane active): four DPP steps inside each row
// of 16 lanes (quad swaps, half-row and row mirrors), then the four row
// results read out as scalars.  The result is wave-uniform.
template <int CTRL>
__device__ inline float dpp_mov(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), CTRL, 0xF, 0xF, true));
}

__device__ inline float lane_value(float v, int lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}

__device__ inline float wave_max(float v) {
  v = fmaxf(v, dpp_mov<0xB1>(v));
  v = fmaxf(v, dpp_mov<0x4E>(v));
  v = fmaxf(v, dpp_mov<0x141>(v));
  v = fmaxf(v, dpp_mov<0x140>(v));
  return fmaxf(fmaxf(lane_value(v, 0), lane_value(v, 16)), fmaxf(lane_value(v, 32), lane_value(v, 48)));
}

__device__ inline float wave_sum(float v) {
  v += dpp_mov<0xB1>(v);
  v += dpp_mov<0x4E>(v);
  v += dpp_mov<0x141>(v);
  v += dpp_mov<0x140>(v);
  return (lane_value(v, 0) + lane_value(v, 16)) + (lane_value(v, 32) + lane_value(v, 48));
}

}  // namespace mikv
