// Decode-step attention over the mixed-precision cache (Section 3.4, Fig. 3
// left) and the importance update (the H2O accumulated-attention score).
//
// Split-K over the sequence: every block takes one contiguous chunk of one
// pool of one (sequence, KV head) -- chunks are homogeneous in precision
// (the pools are grouped by precision, which permutation invariance allows)
// and sized by bytes, so fp16/INT8 and INT2/INT4 chunks cost about the same.
// A block serves all G query heads of the KV group, so GQA loads K/V once.
//
// One wave per chunk (many small work units keep every CU streaming).
// Lanes: LPT = 128/CPL lanes per token, each owning CPL channels (CPL = 32;
// 16 from four query heads per KV head and for fp16 importance rows, whose
// lanes hold two spread 16-byte pieces so a token's lanes read whole
// 128-byte lines; 8 at eight query heads per KV head); a wave covers
// 64/LPT tokens per tile and UNROLL tiles per iteration.  Rows are read
// through buffer descriptors spanning the head's occupied slots (reads past
// them return zero and are masked), contiguous across the lanes of a tile:
// plainly for the cache's resident share (kept in the last-level cache from
// one step to the next), non-temporally for the rest.
//
// Inner loop, with every code c in [0, 2^N) of a group with scale alpha and
// zero beta (Eq. 1, decoded value alpha*c + beta):
//   score:  q . k = alpha * sum_c q_c code_c + beta * sum_c q_c
//   value:  e * v = (e*alpha) * code + e*beta, the e*beta part summed apart.
// Codes are turned into fp16 operands with one AND per two codes: a code c
// placed in the mantissa bits of a zero-exponent half is the fp16 subnormal
// c * 2^(s-24), s the code's bit offset inside the half (codes never reach
// the exponent bits; offsets 10..15 are shifted down first).  Products with
// such halves are exact in fp32, the 2^(s-24) factors are folded into the
// query (key side, v_dot2_f32_f16) and into the final sums (value side,
// fp32 fma with an fp16 operand).  fp16 rows are used as stored.
//
// Softmax: the running maximum is wave-uniform and only raised when a score
// exceeds it by more than 2^8 in the exponential (checked with a ballot), so
// the common tile needs no cross-lane max.  Scores are kept in log2 units.
// The partial phase writes per-chunk (max, sum, value-sum) records and the
// scores; the finalize phase merges the records exactly, turns scores into
// probabilities and optionally adds them to the importance scores.
#include <algorithm>
#include <atomic>
#include <type_traits>

#include "append_device.h"
#include "mikv_internal.h"
#include "select_device.h"

namespace mikv {

namespace {

constexpr int kBlock = 256;        // finalize / importance kernels
constexpr int kWaves = 1;          // the partial kernel runs one wave per chunk
// Chunk record per query head and chunk: max, sum, the pool's token count
// as the partial phase saw it (int32 bits), a pad word, value sum[128]
// (kept 16-byte aligned for vector loads).
constexpr int kRecN = 2;
constexpr int kRecO = 4;
constexpr int kRec = kRecO + kHeadDim;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLog2e = 1.4426950408889634f;
// The scores (written by the partial kernel into the probability arrays)
// and the probabilities that replace them are each touched once per step:
// they are written and read with non-temporal hints, so that this traffic
// does not push the cache rows out of the last-level cache, from which the
// next step reads part of them again (measured at the Mistral shape: 75 ->
// 70 us per attention launch, 97 -> 92 us per step).
constexpr float kLazy = 8.0f;       // raise the running max only past this (log2 units)
constexpr int kMaxChunk = 1024;     // tokens per chunk at most (the chunk's scores are held in LDS)
// Tokens per chunk at most for G query heads per KV head: the chunk's
// scores (G x chunk fp32) stay within 8 KiB of LDS, so LDS does not bound
// the waves per CU below what the registers allow.
__host__ __device__ constexpr int max_chunk(int G) { return G <= 2 ? kMaxChunk : 2048 / G; }

typedef _Float16 half2_t __attribute__((ext_vector_type(2)));

struct AttnArgs {
  const uint8_t *hi_k, *hi_v;
  const uint32_t *hi_kp, *hi_vp;
  const int32_t *n_hi;
  const uint8_t *lo_k, *lo_v;
  const uint32_t *lo_kp, *lo_vp;
  const int32_t *n_lo;
  const uint16_t *q;
  const float *balance;
  float scale;
  float *scores_hi, *scores_lo;  // [B*Hq, cap] scores in log2 units (nullable)
  float *partials;               // [B*Hq, nc_hi + nc_lo, kRec]
  float *probs_hi, *probs_lo;    // outputs (nullable)
  float *acc;                    // hi_acc when accumulating (nullable)
  float *out;                    // [B*Hq, 128]
  int cap_hi, cap_lo, group, q_heads, kv_heads;
  int chunk_hi, chunk_lo, nc_hi, nc_lo, nc_first;
  // Decode step: the new token is appended by the partial phase (app.k
  // non-NULL) and n_hi does not count it until the re-rank writes it.
  AppendArgs app;
  int hi_pending;
  int pool_major;  // dispatch every importance-pool chunk first (fp16 importance pools under GQA)
  int res_hi, res_lo;  // heads [0, res) of each pool are read plainly, the others streamed
  int order;       // 0: the grid order below; 1: heads reversed; 2: the whole grid reversed
  // per-channel retained keys (key_block 64): (alpha, beta) words
  // [NH, n_kblk, 128] per key block, found through the token's position
  const uint32_t *lo_kb;
  const int32_t *lo_pos;
  int n_kblk;
};

// Importance-pool tokens of head h, the pending new token included.
__device__ inline int hi_count(const AttnArgs &A, int h) {
  const int n = A.n_hi[h];
  return n + (A.hi_pending && n < A.cap_hi ? 1 : 0);
}

// ---------------------------------------------------------------------------
// Packed-row formats.  A lane's CPL channels are held as NP = CPL/2 fp16
// pairs; pair p holds lane-local channels lo(p) and hi(p), scaled by
// 2^(cls(p) - 24) for codes (exact fp16 subnormals), or the stored fp16
// values for BITS == 16.
// ---------------------------------------------------------------------------
template <int BITS>
struct Fmt {
  static constexpr bool kQuant = BITS != 16;
  __host__ __device__ static constexpr int lo(int p) {
    return BITS == 16 || BITS == 3 ? 2 * p
         : BITS == 8  ? 4 * (p / 2) + p % 2
         : BITS == 4  ? 8 * (p / 4) + p % 4
                      : 16 * (p / 8) + p % 8;
  }
  __host__ __device__ static constexpr int hi(int p) {
    return BITS == 16 || BITS == 3 ? 2 * p + 1 : lo(p) + (BITS == 8 ? 2 : BITS == 4 ? 4 : 8);
  }
  __host__ __device__ static constexpr int cls(int p) {
    return BITS == 4 ? 4 * (p % 2) : BITS == 2 ? 2 * (p % 4) : 0;
  }
  template <int CPL>
  __device__ static inline void unpack(const uint32_t *raw, uint32_t *out) {
    if constexpr (BITS == 16) {
#pragma unroll
      for (int j = 0; j < CPL / 2; ++j) out[j] = raw[j];
    } else if constexpr (BITS == 3) {
      // 3-bit codes straddle bytes and words: each pair (channels 2j,
      // 2j+1, bits 6j .. 6j+5 of the lane's 3 CPL bits, which start at bit
      // 0 of raw[0]) is extracted from the 64-bit window that holds it into
      // the low bits of the two halves
      constexpr int KW = CPL == 32 ? 3 : 2;
#pragma unroll
      for (int j = 0; j < CPL / 2; ++j) {
        const int bit = 6 * j, wi = bit / 32, sh = bit % 32;
        const uint64_t win = ((uint64_t)(wi + 1 < KW ? raw[wi + 1] : 0u) << 32) | raw[wi];
        const uint32_t x = (uint32_t)(win >> sh);
        out[j] = (x & 7u) | (((x >> 3) & 7u) << 16);
      }
    } else if constexpr (BITS == 8) {
#pragma unroll
      for (int j = 0; j < CPL / 4; ++j) {
        out[2 * j] = raw[j] & 0x00ff00ffu;
        out[2 * j + 1] = (raw[j] >> 8) & 0x00ff00ffu;
      }
    } else if constexpr (BITS == 4) {
#pragma unroll
      for (int j = 0; j < CPL / 8; ++j) {
        const uint32_t x = raw[j], y = x >> 8;
        out[4 * j] = x & 0x000f000fu;
        out[4 * j + 1] = x & 0x00f000f0u;
        out[4 * j + 2] = y & 0x000f000fu;
        out[4 * j + 3] = y & 0x00f000f0u;
      }
    } else {
#pragma unroll
      for (int j = 0; j < CPL / 16; ++j) {
        const uint32_t x = raw[j], y = x >> 8;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          out[8 * j + k] = x & (0x00030003u << (2 * k));
          out[8 * j + 4 + k] = y & (0x00030003u << (2 * k));
        }
      }
    }
  }
};

__device__ inline half2_t as_h2(uint32_t u) { return __builtin_bit_cast(half2_t, u); }

// Codes enter the dot products as fp16 subnormals code * 2^(cls - 24), so
// the query channel paired with a code of class cls is scaled by 2^-cls.
// Scaled down, a small query channel would itself become an fp16 subnormal
// and lose bits (and the matrix cores handle subnormal operands at reduced
// precision), so the query is instead scaled by 2^(shift - cls) with shift
// = the format's largest cls: never below 1, exact in fp16.  A wave whose
// largest |q_hat| would overflow fp16 that way keeps shift 0.  The shift is
// undone in the score scale (wave-uniform).
template <int MAXCLS>
__device__ inline int query_shift(float qmax_lane) {
  if constexpr (MAXCLS == 0) {
    return 0;
  } else {
    const float m = wave_max(qmax_lane);
    return m * (float)(1 << MAXCLS) < 60000.0f ? MAXCLS : 0;
  }
}

// Sum over the LPT consecutive lanes of a token (LPT = 4, 8 or 16).
template <int LPT>
__device__ inline float token_sum(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0xB1, 0xF, 0xF, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x4E, 0xF, 0xF, true));
  if constexpr (LPT >= 8)  // other quad of the half-row
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x141, 0xF, 0xF, true));
  if constexpr (LPT == 16)  // other half of the row
    v += __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, v), 0x140, 0xF, 0xF, true));
  return v;
}

// Sum over the 64/LPT lanes that hold the same `part` (same channels,
// different tokens): rotations inside each 16-lane row, shuffles across rows.
template <int LPT>
__device__ inline float sum_token_lanes(float v) {
  if constexpr (LPT == 4) {
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x124, 0xF, 0xF, false));
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x128, 0xF, 0xF, false));
  } else if constexpr (LPT == 8) {
    v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x128, 0xF, 0xF, false));
  }  // LPT 16: one token per row
  v += __shfl_xor(v, 16, 64);
  v += __shfl_xor(v, 32, 64);
  return v;
}

// A 3-bit lane segment of 16 (8) channels is 48 (24) bits: two dwords are
// loaded from the dword that holds its first bit and shifted (seg_shift) so
// that the segment starts at bit 0.
template <int BITS, int CPL>
struct Rows {
  static constexpr int KW = BITS == 16 ? CPL / 2 : BITS == 3 && CPL <= 16 ? 2 : CPL * BITS / 32;  // raw dwords per segment
  uint32_t k[KW], v[KW];
  uint32_t kp, vp;
};

typedef __amdgpu_buffer_rsrc_t rsrc_t;
// Cache-policy bits of the cache-row loads: streamed rows are read
// non-temporally (the nt bit), the rest plainly; see attn_partial_kernel.
constexpr int kStreamPolicy = 2;
constexpr int kRsrcFlags = 0x00020000;  // raw (untyped) buffer, gfx9 descriptor word 3

// A buffer resource over `bytes` bytes at `base`: loads at offsets past the
// end return zero (so reading past the occupied slots of a pool is safe).
__device__ inline rsrc_t make_rsrc(const void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kRsrcFlags);
}

// Load one token's row segments (this lane's channels) and group params at
// byte offsets `orow` (rows) and `opar` (params) of the head's pools.
// WHICH: 1 the key segment and its group parameters, 2 the value's, 3 both.
// PIECE: bytes between the lane's 16-byte pieces of a row; CPOL: the
// loads' cache-policy bits.
template <int BITS, int CPL, int WHICH = 3, int PIECE = 16, int CPOL = 0>
__device__ inline void load_seg_rows(Rows<BITS, CPL> &r, rsrc_t rk, rsrc_t rv, rsrc_t rkp, rsrc_t rvp, uint32_t orow,
                                     uint32_t opar, uint32_t okp) {
  constexpr int KW = Rows<BITS, CPL>::KW;
  constexpr bool LK = (WHICH & 1) != 0, LV = (WHICH & 2) != 0;
  if constexpr (KW >= 4) {
#pragma unroll
    for (int i = 0; i < KW / 4; ++i) {
      if constexpr (LK) {
        auto a = __builtin_amdgcn_raw_buffer_load_b128(rk, orow + PIECE * i, 0, CPOL);
#pragma unroll
        for (int j = 0; j < 4; ++j) r.k[4 * i + j] = a[j];
      }
      if constexpr (LV) {
        auto b = __builtin_amdgcn_raw_buffer_load_b128(rv, orow + PIECE * i, 0, CPOL);
#pragma unroll
        for (int j = 0; j < 4; ++j) r.v[4 * i + j] = b[j];
      }
    }
  } else if constexpr (KW == 3) {
    if constexpr (LK) {
      auto a = __builtin_amdgcn_raw_buffer_load_b96(rk, orow, 0, CPOL);
      r.k[0] = a[0]; r.k[1] = a[1]; r.k[2] = a[2];
    }
    if constexpr (LV) {
      auto b = __builtin_amdgcn_raw_buffer_load_b96(rv, orow, 0, CPOL);
      r.v[0] = b[0]; r.v[1] = b[1]; r.v[2] = b[2];
    }
  } else if constexpr (KW == 2) {
    if constexpr (LK) {
      auto a = __builtin_amdgcn_raw_buffer_load_b64(rk, orow, 0, CPOL);
      r.k[0] = a[0]; r.k[1] = a[1];
    }
    if constexpr (LV) {
      auto b = __builtin_amdgcn_raw_buffer_load_b64(rv, orow, 0, CPOL);
      r.v[0] = b[0]; r.v[1] = b[1];
    }
  } else {
    if constexpr (LK) r.k[0] = __builtin_amdgcn_raw_buffer_load_b32(rk, orow, 0, CPOL);
    if constexpr (LV) r.v[0] = __builtin_amdgcn_raw_buffer_load_b32(rv, orow, 0, CPOL);
  }
  if constexpr (BITS != 16) {
    if constexpr (LK) r.kp = __builtin_amdgcn_raw_buffer_load_b32(rkp, okp, 0, CPOL);
    if constexpr (LV) r.vp = __builtin_amdgcn_raw_buffer_load_b32(rvp, opar, 0, CPOL);
  }
}

// KPC: retained keys quantized per channel over 64-position blocks
// (Appendix C).  The key's "parameter" word is then its position; a lane
// keeps q_c * alpha_c (times the code class factor) and sum_c q_c beta_c for
// the block of its current token and refreshes them when the block changes.
template <int BITS, int G, int CPL, bool SPLITQ, int UNROLL, int PREFETCH, bool KPC = false, bool STREAM = false>
__device__ void attn_chunk(const AttnArgs &A, int h, int chunk, int rec_chunk, bool is_hi, float *s_lds) {
  using F = Fmt<BITS>;
  constexpr int LPT = kHeadDim / CPL, TPW = 64 / LPT, NP = CPL / 2;
  constexpr bool Q = F::kQuant;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int part = lane % LPT, tsub = lane / LPT;
  const int b = h / A.kv_heads, kvh = h % A.kv_heads;
  const int qh0 = b * A.q_heads + kvh * G;

  const int cap = is_hi ? A.cap_hi : A.cap_lo;
  const int chunk_len = is_hi ? A.chunk_hi : A.chunk_lo;
  // The pool count comes through a vector load; make it provably
  // wave-uniform, so the buffer descriptors built from it live in scalar
  // registers (a value the compiler thinks divergent would wrap every load in
  // a per-lane loop).
  const int n_pool = __builtin_amdgcn_readfirstlane(is_hi ? hi_count(A, h) : A.n_lo[h]);
  const int start = chunk * chunk_len;
  const int end = min(start + chunk_len, n_pool);
  constexpr int64_t kRow = BITS == 16 ? kHeadDim * 2 : kHeadDim * BITS / 8;
  const int ng = kHeadDim / A.group;
  const uint8_t *kb = (is_hi ? A.hi_k : A.lo_k) + (int64_t)h * cap * kRow;
  const uint8_t *vb = (is_hi ? A.hi_v : A.lo_v) + (int64_t)h * cap * kRow;
  const uint32_t *kpb = Q ? (is_hi ? A.hi_kp : A.lo_kp) + (int64_t)h * cap * ng : nullptr;
  const uint32_t *vpb = Q ? (is_hi ? A.hi_vp : A.lo_vp) + (int64_t)h * cap * ng : nullptr;
  float *scores = is_hi ? A.scores_hi : A.scores_lo;
  const float s2scale = A.scale * kLog2e;

  // Query (Eq. 4: q / balance), as fp16 pairs matching the format's pairing,
  // each pair scaled by 2^(qshift - cls) (query_shift); with SPLITQ a second
  // fp16 pair carries the rounding remainder.  qsum24 = 2^(qshift - 24) * the
  // sum of the lane's query channels (fp32).
  float m2[G], l[G], bsum[G], o[G][CPL];
#pragma unroll
  for (int i = 0; i < G; ++i) {
    m2[i] = kNegInf;
    l[i] = 0.0f;
    bsum[i] = 0.0f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) o[i][c] = 0.0f;
  }

  constexpr int kPerIter = kWaves * TPW * UNROLL;
  // chunks are whole multiples of 128 tokens, at most max_chunk(G): an
  // iteration never runs past the LDS score buffer
  static_assert(128 % kPerIter == 0 && max_chunk(G) % 128 == 0, "iteration must divide 128 tokens");
  constexpr int kSeg = Rows<BITS, CPL>::KW * 4;  // bytes loaded per lane's row segment
  // byte offset of the lane's segment in a row, and the bit shift that
  // aligns it (non-zero only for 3-bit segments of 48 or 24 bits, which
  // start inside a dword)
  constexpr bool kSeg3 = BITS == 3 && CPL <= 16;
  constexpr int kSeg3Bytes = 3 * CPL / 8;
  // fp16 rows are read spread: piece j of the lane (8 channels, 16 bytes)
  // holds channels 8 (part + LPT j) .. + 7, so each load of the LPT lanes of
  // a token covers whole 128-byte lines of its row, which streaming
  // (non-temporal) loads need to fetch every line once.  Other formats hold
  // CPL consecutive channels per lane.
  constexpr bool kSpread = BITS == 16;
  constexpr int kPiece = kSpread ? 16 * LPT : 16;
  auto chan8 = [&](int j) { return kSpread ? 8 * (part + LPT * j) : part * CPL + 8 * j; };  // first channel of piece j
  const uint32_t seg_off =
      kSeg3 ? 4u * (uint32_t)((kSeg3Bytes * part) / 4) : kSpread ? 16u * (uint32_t)part : (uint32_t)(part * kSeg);
  const int seg_shift = kSeg3 ? 8 * ((kSeg3Bytes * part) % 4) : 0;
  auto seg_words = [&](const uint32_t *raw, uint32_t *out) {
    if constexpr (kSeg3) {
      out[0] = __builtin_amdgcn_alignbit(raw[1], raw[0], seg_shift);
      out[1] = raw[1] >> seg_shift;
    } else {
#pragma unroll
      for (int i = 0; i < Rows<BITS, CPL>::KW; ++i) out[i] = raw[i];
    }
  };
  const int n_iter = end > start ? (end - start + kPerIter - 1) / kPerIter : 0;
  const int first = start + wave * TPW * UNROLL + tsub;  // this lane's token in iteration 0, u = 0
  const int g_lane = (part * CPL) / A.group;
  // Buffer resources over this head's occupied slots; a lane's offset is
  // fixed per iteration and the unroll steps are immediate offsets.
  const rsrc_t rk = make_rsrc(kb, (uint32_t)n_pool * (uint32_t)kRow);
  const rsrc_t rv = make_rsrc(vb, (uint32_t)n_pool * (uint32_t)kRow);
  const rsrc_t rkp = KPC ? make_rsrc(A.lo_pos + (int64_t)h * cap, (uint32_t)n_pool * 4u)
                         : make_rsrc(Q ? (const void *)kpb : (const void *)kb, Q ? (uint32_t)n_pool * ng * 4u : 0u);
  const rsrc_t rvp = make_rsrc(Q ? (const void *)vpb : (const void *)vb, Q ? (uint32_t)n_pool * ng * 4u : 0u);
  const uint32_t lane_tok = (uint32_t)(start + wave * TPW * UNROLL + tsub);
  const uint32_t off_row0 = lane_tok * (uint32_t)kRow + seg_off;
  const uint32_t off_par0 = (lane_tok * (uint32_t)ng + (uint32_t)g_lane) * 4u;
  const uint32_t off_kp0 = KPC ? lane_tok * 4u : off_par0;

  // With `live` false the loads go through empty descriptors: they return
  // zero without a memory access, so a load needs no branch around it.
  const rsrc_t r_none = make_rsrc(kb, 0u);
  auto load_part = [&](auto which, Rows<BITS, CPL>(&r)[UNROLL], int it, bool live = true) {
    const uint32_t orow = off_row0 + (uint32_t)(it * kPerIter) * (uint32_t)kRow;
    const uint32_t opar = off_par0 + (uint32_t)(it * kPerIter) * (uint32_t)ng * 4u;
    const uint32_t okp = KPC ? off_kp0 + (uint32_t)(it * kPerIter) * 4u : opar;
    const rsrc_t ak = live ? rk : r_none, av = live ? rv : r_none;
    const rsrc_t akp = live ? rkp : r_none, avp = live ? rvp : r_none;
#pragma unroll
    for (int u = 0; u < UNROLL; ++u)
      load_seg_rows<BITS, CPL, decltype(which)::value, kPiece, STREAM ? kStreamPolicy : 0>(r[u], ak, av, akp, avp, orow + (uint32_t)(u * TPW * kRow),
                                                       opar + (uint32_t)(u * TPW) * (uint32_t)ng * 4u,
                                                       KPC ? okp + (uint32_t)(u * TPW) * 4u
                                                           : opar + (uint32_t)(u * TPW) * (uint32_t)ng * 4u);
  };
  auto load_it = [&](Rows<BITS, CPL>(&r)[UNROLL], int it) { load_part(std::integral_constant<int, 3>{}, r, it); };

  // The first iterations' rows do not depend on the query: issue them first.
  Rows<BITS, CPL> cur[UNROLL], n1[PREFETCH >= 1 ? UNROLL : 1], n2[PREFETCH >= 2 ? UNROLL : 1];
  if (n_iter > 0) load_it(cur, 0);
  if constexpr (PREFETCH >= 1) {
    if (n_iter > 1) load_it(n1, 1);
  }
  if constexpr (PREFETCH >= 2) {
    if (n_iter > 2) load_it(n2, 2);
  }

  // Every query (and balancer) word this lane needs is loaded with 16-byte
  // loads issued together, before any of them is used: the chunk's K/V
  // stream starts one memory round trip after the wave does.
  half2_t qh[G][NP], ql[G][SPLITQ ? NP : 1];
  float qsum24[G];  // 2^-24 * sum of the lane's query channels
  float qkeep[KPC ? G : 1][KPC ? CPL : 1];  // KPC: the lane's query channels (fp32)
  uint4 qraw[G][CPL / 8];
#pragma unroll
  for (int i = 0; i < G; ++i) {
    const uint16_t *qrow = A.q + (int64_t)(qh0 + i) * kHeadDim;
#pragma unroll
    for (int j = 0; j < CPL / 8; ++j) qraw[i][j] = *reinterpret_cast<const uint4 *>(qrow + chan8(j));
  }
  float bal[SPLITQ ? CPL : 1];
  if constexpr (SPLITQ) {
    const float *brow = A.balance + (int64_t)h * kHeadDim;
#pragma unroll
    for (int j = 0; j < CPL / 4; ++j) {
      const float4 v = *reinterpret_cast<const float4 *>(brow + chan8(j >> 1) + 4 * (j & 1));
      bal[4 * j] = v.x;
      bal[4 * j + 1] = v.y;
      bal[4 * j + 2] = v.z;
      bal[4 * j + 3] = v.w;
    }
  }
  constexpr int kMaxCls = BITS == 2 ? 6 : BITS == 4 ? 4 : 0;
  int qshift = 0;
  if constexpr (kMaxCls > 0 && !KPC) {
    // bound on |q_hat| over the wave: max |q| / min b
    uint32_t mb = 0;
#pragma unroll
    for (int i = 0; i < G; ++i)
#pragma unroll
      for (int j = 0; j < CPL / 8; ++j) {
        const uint32_t w[4] = {qraw[i][j].x, qraw[i][j].y, qraw[i][j].z, qraw[i][j].w};
#pragma unroll
        for (int k = 0; k < 4; ++k) mb = max(mb, max(w[k] & 0x7fffu, (w[k] >> 16) & 0x7fffu));
      }
    float bound = f16_to_f32((uint16_t)mb);
    if constexpr (SPLITQ) {
      float bmin = bal[0];
#pragma unroll
      for (int c = 1; c < CPL; ++c) bmin = fminf(bmin, bal[c]);
      bound = bound / bmin;
    }
    qshift = query_shift<kMaxCls>(bound);
  }
  const float s2scale_q = Q ? __builtin_ldexpf(s2scale, 24 - qshift) : s2scale;
#pragma unroll
  for (int i = 0; i < G; ++i) {
    float qf[CPL];
#pragma unroll
    for (int j = 0; j < CPL / 8; ++j) {
      const uint32_t w[4] = {qraw[i][j].x, qraw[i][j].y, qraw[i][j].z, qraw[i][j].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        qf[8 * j + 2 * k] = f16_to_f32((uint16_t)(w[k] & 0xffffu));
        qf[8 * j + 2 * k + 1] = f16_to_f32((uint16_t)(w[k] >> 16));
      }
    }
    if constexpr (SPLITQ) {
#pragma unroll
      for (int c = 0; c < CPL; ++c) qf[c] = qf[c] / bal[c];
    }
    auto qhat = [&](int c) { return qf[c]; };
    if constexpr (KPC) {
#pragma unroll
      for (int c = 0; c < CPL; ++c) qkeep[i][c] = qf[c];
    }
    float s = 0.0f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) s += qhat(c);
    qsum24[i] = __builtin_ldexpf(s, qshift - 24);
#pragma unroll
    for (int p = 0; p < NP; ++p) {
      const float sc = __builtin_ldexpf(1.0f, qshift - F::cls(p));
      const float a = qhat(F::lo(p)) * sc, bb = qhat(F::hi(p)) * sc;
      const _Float16 ah = (_Float16)a, bh = (_Float16)bb;
      qh[i][p] = half2_t{ah, bh};
      if constexpr (SPLITQ) ql[i][p] = half2_t{(_Float16)(a - (float)ah), (_Float16)(bb - (float)bh)};
    }
  }

  // The chunk's scores stay in LDS (written by the lanes that hold them)
  // and go out in one burst after the loop: no global store is issued
  // between the loads of the stream (stores and loads share one completion
  // counter, so stores in the loop delay every later load wait).
  float *score_row[G];
#pragma unroll
  for (int i = 0; i < G; ++i) score_row[i] = scores ? scores + (int64_t)(qh0 + i) * cap : nullptr;

  // KPC: q_c * alpha_c * 2^-cls (qa) and 2^-24 sum_c q_c beta_c (b24) of
  // the lane's channels for key block kblk
  float qa[KPC ? G : 1][KPC ? CPL : 1], b24[KPC ? G : 1];
  int kblk = -1;
  const rsrc_t rkb = KPC ? make_rsrc(A.lo_kb + ((int64_t)h * A.n_kblk) * kHeadDim, (uint32_t)A.n_kblk * kHeadDim * 4u)
                         : r_none;
  auto kpc_refresh = [&](int blk) {
    if constexpr (KPC) {
      uint32_t pw[CPL];
#pragma unroll
      for (int j = 0; j < CPL / 4; ++j) {
        auto w = __builtin_amdgcn_raw_buffer_load_b128(rkb, ((uint32_t)blk * kHeadDim + part * CPL + 4 * j) * 4u, 0, 0);
#pragma unroll
        for (int e = 0; e < 4; ++e) pw[4 * j + e] = w[e];
      }
#pragma unroll
      for (int i = 0; i < G; ++i) {
        float bs = 0.0f;
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          const float sc = __builtin_ldexpf(1.0f, -F::cls(p));
#pragma unroll
          for (int side = 0; side < 2; ++side) {
            const int c = side ? F::hi(p) : F::lo(p);
            const float a = f16_to_f32((uint16_t)(pw[c] & 0xffffu)), b = f16_to_f32((uint16_t)(pw[c] >> 16));
            qa[i][c] = (qkeep[i][c] * a) * sc;
            bs = fmaf(qkeep[i][c], b, bs);
          }
        }
        b24[i] = __builtin_ldexpf(bs, -24);
      }
      kblk = blk;
    }
  };

  float s2[UNROLL][G];
  // Scores of one iteration (and the lazy running-max update).
  auto proc_k = [&](Rows<BITS, CPL>(&cur)[UNROLL], int it) {
    bool valid[UNROLL];
    uint64_t raise = 0;  // lanes whose score passes the lazy threshold (a ballot per token)
    const int rem = end - it * kPerIter;  // wave-uniform: a token is valid when first + u * TPW < rem
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      valid[u] = first < rem - u * TPW;
      uint32_t kx[NP], kraw[Rows<BITS, CPL>::KW];
      seg_words(cur[u].k, kraw);
      F::template unpack<CPL>(kraw, kx);
      const half2_t kab = as_h2(cur[u].kp);  // (alpha, beta) of the key group
      if constexpr (KPC) {
        // the token's key block (the parameter word is its position); tokens
        // past the pool read position 0 and are masked below
        const int blk = min(max((int)cur[u].kp / kKeyBlock, 0), max(A.n_kblk - 1, 0));
        if (blk != kblk) kpc_refresh(blk);
      }
#pragma unroll
      for (int i = 0; i < G; ++i) {
        float d = 0.0f;
        if constexpr (KPC) {
          // 2^-24 sum_c q_c alpha_c code_c: each masked code is an exact
          // fp16 subnormal (code * 2^(cls - 24)) in a mixed-precision FMA
#pragma unroll
          for (int p = 0; p < NP; ++p) {
            const half2_t hk = as_h2(kx[p]);
            d = fmaf(qa[i][F::lo(p)], (float)hk.x, d);
            d = fmaf(qa[i][F::hi(p)], (float)hk.y, d);
          }
        } else {
#pragma unroll
          for (int p = 0; p < NP; ++p) d = __builtin_amdgcn_fdot2(as_h2(kx[p]), qh[i][p], d, false);
          if constexpr (SPLITQ) {
#pragma unroll
            for (int p = 0; p < NP; ++p) d = __builtin_amdgcn_fdot2(as_h2(kx[p]), ql[i][p], d, false);
          }
        }
        // 2^-24 (alpha * 2^24 * d + beta * qsum): the fp16 scale and zero
        // enter mixed-precision FMAs as stored; the power of two goes into
        // the final scale, so the result is the same bits
        float s = KPC ? d + b24[i] : Q ? fmaf((float)kab.x, d, fmaf((float)kab.y, qsum24[i], 0.0f)) : d;
        s = token_sum<LPT>(s) * s2scale_q;
        s = valid[u] ? s : kNegInf;
        s2[u][i] = s;
        // every lane of the token holds s: all of them store it (same
        // value, same address), which keeps the loop free of exec-mask
        // branches around the store
        s_lds[i * max_chunk(G) + it * kPerIter + u * TPW + tsub] = s;
        raise |= __ballot(s > m2[i] + kLazy);
      }
    }
    if (raise) {
#pragma unroll
      for (int i = 0; i < G; ++i) {
        float mx = s2[0][i];
#pragma unroll
        for (int u = 1; u < UNROLL; ++u) mx = fmaxf(mx, s2[u][i]);
        mx = wave_max(mx);
        if (mx > m2[i]) {
          const float f = m2[i] == kNegInf ? 0.0f : __builtin_amdgcn_exp2f(m2[i] - mx);
          l[i] *= f;
          bsum[i] *= f;
#pragma unroll
          for (int c = 0; c < CPL; ++c) o[i][c] *= f;
          m2[i] = mx;
        }
      }
    }
  };
  // Value sums of one iteration.
  auto proc_v = [&](Rows<BITS, CPL>(&cur)[UNROLL]) {
#pragma unroll
    for (int u = 0; u < UNROLL; ++u) {
      uint32_t vx[NP], vraw[Rows<BITS, CPL>::KW];
      seg_words(cur[u].v, vraw);
      F::template unpack<CPL>(vraw, vx);
      const half2_t vab = as_h2(cur[u].vp);  // (alpha, beta) of the value group
#pragma unroll
      for (int i = 0; i < G; ++i) {
        // past the pool s2 = -inf, and m2 is finite from the first iteration
        // on (its first token is valid and raises the max), so e = 0
        const float e = __builtin_amdgcn_exp2f(s2[u][i] - m2[i]);
        l[i] += e;
        const float w = Q ? fmaf(e, (float)vab.x, 0.0f) : e;
        if constexpr (Q) bsum[i] = fmaf(e, (float)vab.y, bsum[i]);
#pragma unroll
        for (int p = 0; p < NP; ++p) {
          const half2_t hv = as_h2(vx[p]);
          o[i][F::lo(p)] = fmaf(w, (float)hv.x, o[i][F::lo(p)]);
          o[i][F::hi(p)] = fmaf(w, (float)hv.y, o[i][F::hi(p)]);
        }
      }
    }
  };
  auto proc = [&](Rows<BITS, CPL>(&cur)[UNROLL], int it) {
    proc_k(cur, it);
    proc_v(cur);
  };

  // Software pipeline: the rows of the next PREFETCH iterations are loaded
  // while the current one is computed.  PREFETCH < 0: half steps in the
  // same registers -- the next iteration's keys are loaded as soon as the
  // scores are done, its values as soon as the value sums are, so one half
  // of the rows is always in flight without extra registers.
  if constexpr (PREFETCH < 0) {
    // (no branch around the loads, and scheduling barriers: a load issued
    // early would need registers of its own)
    for (int it = 0; it < n_iter; ++it) {
      const bool live = it + 1 < n_iter;
      proc_k(cur, it);
      __builtin_amdgcn_sched_barrier(0);
      load_part(std::integral_constant<int, 1>{}, cur, it + 1, live);
      __builtin_amdgcn_sched_barrier(0);
      proc_v(cur);
      __builtin_amdgcn_sched_barrier(0);
      load_part(std::integral_constant<int, 2>{}, cur, it + 1, live);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else if constexpr (PREFETCH == 0) {
    for (int it = 0; it < n_iter; ++it) {
      if (it > 0) load_it(cur, it);
      proc(cur, it);
    }
  } else if constexpr (PREFETCH == 1) {
    for (int it = 0; it < n_iter; ++it) {
      proc(cur, it);
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) cur[u] = n1[u];
      if (it + 2 < n_iter) load_it(n1, it + 2);
    }
  } else {
    for (int it = 0; it < n_iter; ++it) {
      proc(cur, it);
#pragma unroll
      for (int u = 0; u < UNROLL; ++u) {
        cur[u] = n1[u];
        n1[u] = n2[u];
      }
      if (it + 3 < n_iter) load_it(n2, it + 3);
    }
  }
  if (scores) {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int i = 0; i < G; ++i)
      for (int j = lane; j < end - start; j += 64)
        __builtin_nontemporal_store(s_lds[i * max_chunk(G) + j], &score_row[i][start + j]);
  }

  // Undo the code scaling, add the beta part, merge the lanes of equal
  // `part` (same channels), and write this chunk's record.
#pragma unroll
  for (int i = 0; i < G; ++i) {
    if constexpr (Q) {
#pragma unroll
      for (int p = 0; p < NP; ++p) {
        const float sc = __builtin_ldexpf(1.0f, 24 - F::cls(p));
        o[i][F::lo(p)] = fmaf(o[i][F::lo(p)], sc, bsum[i]);
        o[i][F::hi(p)] = fmaf(o[i][F::hi(p)], sc, bsum[i]);
      }
    }
    l[i] = wave_sum(l[i]) * (1.0f / LPT);  // every lane of a token added its e
#pragma unroll
    for (int c = 0; c < CPL; ++c) o[i][c] = sum_token_lanes<LPT>(o[i][c]);
  }
  const int nc = A.nc_hi + A.nc_lo;
#pragma unroll
  for (int i = 0; i < G; ++i) {
    float *rec = A.partials + ((int64_t)(qh0 + i) * nc + rec_chunk) * kRec;
    if (lane == 0) {
      rec[0] = m2[i];
      rec[1] = l[i];
      rec[kRecN] = __builtin_bit_cast(float, n_pool);
    }
    if (tsub == 0) {
#pragma unroll
      for (int c = 0; c < CPL / 4; ++c)
        *reinterpret_cast<float4 *>(rec + kRecO + chan8(c >> 1) + 4 * (c & 1)) =
            make_float4(o[i][4 * c], o[i][4 * c + 1], o[i][4 * c + 2], o[i][4 * c + 3]);
    }
  }
}

// ---------------------------------------------------------------------------
// The 2-bit retained pool on the matrix cores (16x16x32 fp16 MFMA).
//
// Lane l = 16 a + n.  Scores of a 16-token tile: B holds the tile's key
// codes as exact fp16 subnormals: the 2-bit field of class k (its position
// in the byte) is shifted to mantissa bits 6-7 (k even: code * 2^-18) or
// 8-9 (k odd: code * 2^-16) of its 16-bit half.  The matrix cores multiply
// the deepest fp16 subnormals (code * 2^-24, 2^-22) at reduced precision,
// about 5e-6 relative, but subnormals from 2^-18 up exactly (measured).
// Lane (n, a) holds the 32 codes of channels [32a, 32a + 32) of token n, so
// the token-major key rows are read as they are stored.  A
// holds the query: row 4 s + gamma carries q_hat (times 2^qshift, and 4 more
// for even classes, so every product is q * code * 2^(qshift - 16)) of query
// slot s on the channels of quantization group gamma and 0 elsewhere, so
// lane (n, a) receives, for query slot a, one partial dot product per group
// and applies token n's per-group scale and zero (folded Eq. 1).
//
// Value sums: the pool's value codes are stored in 32-slot tiles
// (int2_v_byte): lane (n, g) reads, in one 16-byte load, bytes n and n + 16
// of slots 8g..8g+7, whose fields are channels n + 32j and n + 16 + 32j.
// For n-block nb (channels 16nb..16nb+15) it takes field nb/2 of byte
// n + 16(nb%2), moved to bits 8-9 of its half: B = codes * 2^-16 (tokens x
// channels, the scale undone on the output); A = the softmax weights
// e * alpha of the column's group,
// split in an fp16 high and low part (rows 2i and 2i+1 for query i) and
// staged through LDS into the operand layout.
// ---------------------------------------------------------------------------
typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u4_t __attribute__((ext_vector_type(4)));

__device__ inline h8_t pack_h8(uint32_t x, uint32_t y, uint32_t z, uint32_t w) {
  const u4_t u = {x, y, z, w};
  return __builtin_bit_cast(h8_t, u);
}

__device__ inline f4_t mfma32(h8_t a, h8_t b, f4_t c) { return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0); }

// Reductions over the 16 lanes of each row (lane group); result in all 16.
__device__ inline float row_max16(float v) {
  v = fmaxf(v, dpp_mov<0xB1>(v));
  v = fmaxf(v, dpp_mov<0x4E>(v));
  v = fmaxf(v, dpp_mov<0x141>(v));
  return fmaxf(v, dpp_mov<0x140>(v));
}
__device__ inline float row_sum16(float v) {
  v += dpp_mov<0xB1>(v);
  v += dpp_mov<0x4E>(v);
  v += dpp_mov<0x141>(v);
  return v + dpp_mov<0x140>(v);
}

#ifndef MIKV_INT2_KEY_TILES
#define MIKV_INT2_KEY_TILES 2
#endif
constexpr int kKT = MIKV_INT2_KEY_TILES;  // 16-token key tiles per iteration (2 or 4)
constexpr int kVT = kKT / 2;              // 32-token value tiles per iteration
constexpr int kItTok = 16 * kKT;          // tokens per iteration
// Operand element -> slot inside a lane group's 8 (and back): bits 0 and 1
// swapped, the order the masked code pairs come out in.
__host__ __device__ constexpr int tau8(int e) { return (e & 4) | ((e & 1) << 1) | ((e >> 1) & 1); }

// LDS weight staging: [group][value tile][row 0..15][lane group][element]
// halves; rows past 2G stay zero, so every lane reads its operand.
__device__ inline int w_index(int gamma, int vt, int row, int g, int e) {
  return (((gamma * kVT + vt) * 16 + row) * 4 + g) * 8 + e;
}
constexpr int kWLds = 4 * kVT * 16 * 4 * 8;  // halves (4 KiB per value tile)

template <int G, bool SPLITQ, int NG, bool STREAM>
__device__ void attn_chunk_int2(const AttnArgs &A, int h, int chunk, int rec_chunk, float *s_lds, _Float16 *w_lds) {
  constexpr int QS = G < 4 ? G : 4;    // distinct query slots in one row block
  constexpr int NSET = G > 4 ? 2 : 1;  // query sets (G = 8: queries 0-3 and 4-7)
  constexpr int R = 4 / QS;            // lane groups holding the same query slot
  constexpr int NGL = (NG + R - 1) / R;  // value groups each lane weights
  constexpr int NP = SPLITQ ? 2 : 1;   // fp16 parts of the query
  constexpr int GROUP = kHeadDim / NG;
  constexpr int kCpol = STREAM ? kStreamPolicy : 0;
  const int lane = threadIdx.x & 63, n = lane & 15, a = lane >> 4;
  const int qs = a % QS, rho = a / QS;
  const int b = h / A.kv_heads, kvh = h % A.kv_heads;
  const int qh0 = b * A.q_heads + kvh * G;
  const int cap = A.cap_lo;
  const int n_pool = __builtin_amdgcn_readfirstlane(A.n_lo[h]);
  const int start = chunk * A.chunk_lo;
  const int end = min(start + A.chunk_lo, n_pool);
  const int n_iter = end > start ? (end - start + kItTok - 1) / kItTok : 0;
  float *scores = A.scores_lo;

  const rsrc_t rk = make_rsrc(A.lo_k + (int64_t)h * cap * 32, (uint32_t)n_pool * 32u);
  const rsrc_t rv = make_rsrc(A.lo_v + (int64_t)h * cap * 32, (uint32_t)((n_pool + 31) / 32) * 1024u);
  const rsrc_t rkp = make_rsrc(A.lo_kp + (int64_t)h * cap * NG, (uint32_t)n_pool * NG * 4u);
  const rsrc_t rvp = make_rsrc(A.lo_vp + (int64_t)h * cap * NG, (uint32_t)n_pool * NG * 4u);

  // One iteration's loads: key codes and parameter rows of the four key
  // tiles (the lane's value groups only), value codes of the two tiles.
  struct Ld {
    uint32_t kc[kKT][2];
    uint32_t kp[kKT][NG];
    uint32_t vp[kKT][NGL];
    uint32_t vc[kVT][4];
  };
  // KEYS: the key codes and parameters; VALS: the value codes and
  // parameters.  With `live` false every load goes through an empty
  // descriptor (zero, no memory access), so no branch is needed around it.
  const rsrc_t r_none = make_rsrc(A.lo_k, 0u);
  auto load = [&](Ld &d, int it, bool keys, bool vals, bool live) {
    const uint32_t t0 = (uint32_t)(start + it * kItTok);
    const rsrc_t ak = live ? rk : r_none, av = live ? rv : r_none;
    const rsrc_t akp = live ? rkp : r_none, avp = live ? rvp : r_none;
#pragma unroll
    for (int q = 0; q < kKT; ++q) {
      const uint32_t slot = t0 + 16 * q + n;
      if (keys) {
        auto kc = __builtin_amdgcn_raw_buffer_load_b64(ak, slot * 32u + 8u * a, 0, kCpol);
        d.kc[q][0] = kc[0];
        d.kc[q][1] = kc[1];
        if constexpr (NG == 4) {
          auto kp = __builtin_amdgcn_raw_buffer_load_b128(akp, slot * 16u, 0, kCpol);
#pragma unroll
          for (int j = 0; j < 4; ++j) d.kp[q][j] = kp[j];
        } else if constexpr (NG == 2) {
          auto kp = __builtin_amdgcn_raw_buffer_load_b64(akp, slot * 8u, 0, kCpol);
          d.kp[q][0] = kp[0];
          d.kp[q][1] = kp[1];
        } else {
          d.kp[q][0] = __builtin_amdgcn_raw_buffer_load_b32(akp, slot * 4u, 0, kCpol);
        }
      }
      if (vals) {
        if constexpr (R == 1 && NG == 4) {  // every group: the whole row, one load
          auto vp = __builtin_amdgcn_raw_buffer_load_b128(avp, slot * 16u, 0, kCpol);
#pragma unroll
          for (int j = 0; j < 4; ++j) d.vp[q][j] = vp[j];
        } else if constexpr (R == 1 && NG == 2) {
          auto vp = __builtin_amdgcn_raw_buffer_load_b64(avp, slot * 8u, 0, kCpol);
          d.vp[q][0] = vp[0];
          d.vp[q][1] = vp[1];
        } else {
#pragma unroll
          for (int j = 0; j < NGL; ++j)
            d.vp[q][j] = __builtin_amdgcn_raw_buffer_load_b32(avp, (slot * NG + (uint32_t)((rho + R * j) % NG)) * 4u, 0, kCpol);
        }
      }
    }
    if (vals) {
#pragma unroll
      for (int vt = 0; vt < kVT; ++vt) {
        const uint32_t tile = (t0 >> 5) + vt;
        auto vc = __builtin_amdgcn_raw_buffer_load_b128(av, tile * 1024u + 16u * (uint32_t)lane, 0, kCpol);
#pragma unroll
        for (int j = 0; j < 4; ++j) d.vc[vt][j] = vc[j];
      }
    }
  };
  Ld cur;
  load(cur, 0, true, true, n_iter > 0);

  // zero the weight rows (rows past 2G are never written)
  {
    uint4 *w4 = reinterpret_cast<uint4 *>(w_lds);
#pragma unroll
    for (int j = 0; j < kWLds / 8 / 64; ++j) w4[j * 64 + lane] = make_uint4(0u, 0u, 0u, 0u);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  // Query operands.  As an A row, lane l is row m = n: query slot m/4 (mod
  // QS) of set st, group m%4, over K block a (channels [32a, 32a + 32)).
  h8_t AK[NSET][NP][4];
  float qpart[NSET];
  // the query scaled by 2^(qshift - 2 k) for class k (query_shift)
  float qfs[NSET][32];
  float qmax = 0.0f;
#pragma unroll
  for (int st = 0; st < NSET; ++st) {
    const int iq = (n / 4) % QS + 4 * st;
    const uint4 *q4 = reinterpret_cast<const uint4 *>(A.q + (int64_t)(qh0 + iq) * kHeadDim + 32 * a);
    uint4 qr[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) qr[j] = q4[j];
    float *qf = qfs[st];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t w[4] = {qr[j].x, qr[j].y, qr[j].z, qr[j].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        qf[8 * j + 2 * k] = f16_to_f32((uint16_t)(w[k] & 0xffffu));
        qf[8 * j + 2 * k + 1] = f16_to_f32((uint16_t)(w[k] >> 16));
      }
    }
    if constexpr (SPLITQ) {
      const float4 *b4 = reinterpret_cast<const float4 *>(A.balance + (int64_t)h * kHeadDim + 32 * a);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float4 v = b4[j];
        qf[4 * j] = qf[4 * j] / v.x;
        qf[4 * j + 1] = qf[4 * j + 1] / v.y;
        qf[4 * j + 2] = qf[4 * j + 2] / v.z;
        qf[4 * j + 3] = qf[4 * j + 3] / v.w;
      }
    }
#pragma unroll
    for (int j = 0; j < 32; ++j) qmax = fmaxf(qmax, fabsf(qf[j]));
  }
  // the even-class query operand carries 2^(qshift + 2): largest qshift in
  // {6, 4, 2, 0} that keeps it within fp16 (wave-uniform)
  const float qm = wave_max(qmax);
  const int qshift = qm * 256.0f < 60000.0f ? 6 : qm * 64.0f < 60000.0f ? 4 : qm * 16.0f < 60000.0f ? 2 : 0;
  const float s2scale_q = __builtin_ldexpf(A.scale * kLog2e, 16 - qshift);
#pragma unroll
  for (int st = 0; st < NSET; ++st) {
    const float *qf = qfs[st];
    float ps = 0.0f;
#pragma unroll
    for (int j = 0; j < 32; ++j) ps += qf[j];
    qpart[st] = ps;
    const float keep = (32 * a) / GROUP == n % 4 ? 1.0f : 0.0f;  // the lane's channels lie in one group
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t hw[4], lw[4];
#pragma unroll
      for (int d = 0; d < 4; ++d) {
        float vv[2];
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int e = 2 * d + hf;
          const int j = 16 * (i >> 1) + 4 * (i & 1) + (e >> 1) + 8 * (e & 1);
          vv[hf] = qf[j] * (keep * __builtin_ldexpf(1.0f, qshift + ((e >> 1) & 1 ? 0 : 2)));
        }
        const _Float16 h0 = (_Float16)vv[0], h1 = (_Float16)vv[1];
        hw[d] = (uint32_t)__builtin_bit_cast(uint16_t, h0) | ((uint32_t)__builtin_bit_cast(uint16_t, h1) << 16);
        if constexpr (SPLITQ) {
          const _Float16 l0 = (_Float16)(vv[0] - (float)h0), l1 = (_Float16)(vv[1] - (float)h1);
          lw[d] = (uint32_t)__builtin_bit_cast(uint16_t, l0) | ((uint32_t)__builtin_bit_cast(uint16_t, l1) << 16);
        }
      }
      AK[st][0][i] = pack_h8(hw[0], hw[1], hw[2], hw[3]);
      if constexpr (SPLITQ) AK[st][NP - 1][i] = pack_h8(lw[0], lw[1], lw[2], lw[3]);
    }
  }
  // Sum of q_hat over each group for the lane's own query slot (the zero
  // term of the folded dequantization), from the rows 4 s of lane groups a'.
  float qsl[NSET][NG];
#pragma unroll
  for (int st = 0; st < NSET; ++st) {
    float all[QS][NG];
#pragma unroll
    for (int s3 = 0; s3 < QS; ++s3) {
#pragma unroll
      for (int gm = 0; gm < NG; ++gm) all[s3][gm] = 0.0f;
#pragma unroll
      for (int ap = 0; ap < 4; ++ap) all[s3][(32 * ap) / GROUP] += lane_value(qpart[st], 16 * ap + 4 * s3);
    }
#pragma unroll
    for (int gm = 0; gm < NG; ++gm) {
      float v = all[0][gm];
#pragma unroll
      for (int s3 = 1; s3 < QS; ++s3) v = qs == s3 ? all[s3][gm] : v;
      qsl[st][gm] = __builtin_ldexpf(v, qshift - 16);  // 2^(qshift - 16): the scale of the scores below
    }
  }

  float m2q[G];       // running max per query (wave-uniform, log2 units)
  float m_own[NSET];  // the max of the lane's own query
#pragma unroll
  for (int i = 0; i < G; ++i) m2q[i] = kNegInf;
#pragma unroll
  for (int st = 0; st < NSET; ++st) m_own[st] = kNegInf;
  float l_l[NSET], bs_l[NSET][NGL];
#pragma unroll
  for (int st = 0; st < NSET; ++st) {
    l_l[st] = 0.0f;
#pragma unroll
    for (int j = 0; j < NGL; ++j) bs_l[st][j] = 0.0f;
  }
  // a lane's duplicate value group (fewer groups than replicas) adds nothing
  float dup[NGL];
#pragma unroll
  for (int j = 0; j < NGL; ++j) dup[j] = rho + R * j < NG ? 1.0f : 0.0f;
  f4_t CV[8];
#pragma unroll
  for (int nb = 0; nb < 8; ++nb) CV[nb] = f4_t{0.0f, 0.0f, 0.0f, 0.0f};
  // value fields go to bits 8-9 of each half (code * 2^-16)
  constexpr uint32_t mk = 0x03000300u;

  // Half-step pipeline (as in attn_chunk): the next iteration's keys are
  // loaded once the scores are done, its values once the value MFMAs are.
  for (int it = 0; it < n_iter; ++it) {
    const bool live = it + 1 < n_iter;
    const int t0 = start + it * kItTok;
    // --- scores of the four key tiles
    float s2[kKT][NSET];
    uint64_t raise = 0;
#pragma unroll
    for (int q = 0; q < kKT; ++q) {
      // code pairs of bytes 0, 2 (fields k at bits 2k) and bytes 1, 3
      // (bits 8 + 2k), each field moved to bits 6-7 (k even) or 8-9 (k odd)
      // of its half: code * 2^-18 or code * 2^-16
      uint32_t P[16];
#pragma unroll
      for (int w = 0; w < 2; ++w) {
        const uint32_t x = cur.kc[q][w];
        const uint32_t l6 = x << 6, l2 = x << 2, r2 = x >> 2, r6 = x >> 6;
        P[(2 * w) * 4 + 0] = l6 & 0x00c000c0u;
        P[(2 * w) * 4 + 1] = l6 & 0x03000300u;
        P[(2 * w) * 4 + 2] = l2 & 0x00c000c0u;
        P[(2 * w) * 4 + 3] = l2 & 0x03000300u;
        P[(2 * w + 1) * 4 + 0] = r2 & 0x00c000c0u;
        P[(2 * w + 1) * 4 + 1] = r2 & 0x03000300u;
        P[(2 * w + 1) * 4 + 2] = r6 & 0x00c000c0u;
        P[(2 * w + 1) * 4 + 3] = r6 & 0x03000300u;
      }
      const bool valid = t0 + 16 * q + n < end;
#pragma unroll
      for (int st = 0; st < NSET; ++st) {
        f4_t C = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int pt = 0; pt < NP; ++pt)
#pragma unroll
          for (int i = 0; i < 4; ++i)
            C = mfma32(AK[st][pt][i], pack_h8(P[4 * i], P[4 * i + 1], P[4 * i + 2], P[4 * i + 3]), C);
        // 2^(qshift - 16) times the folded score (the fp16 scale and zero enter
        // mixed-precision FMAs as stored; the power of two is in the scale)
        // (two independent chains: no dependent mixed FMAs back to back)
        float sp[2] = {0.0f, 0.0f};
#pragma unroll
        for (int gm = 0; gm < NG; ++gm) {
          const half2_t kab = as_h2(cur.kp[q][gm]);
          sp[gm & 1] = fmaf((float)kab.x, C[gm], fmaf((float)kab.y, qsl[st][gm], sp[gm & 1]));
        }
        // -inf for a token past the chunk, as a select (no branch)
        const float v2 = fmaf(sp[0] + sp[1], s2scale_q, valid ? 0.0f : kNegInf);
        s2[q][st] = v2;
        if (scores) s_lds[(qs + 4 * st) * max_chunk(G) + (t0 - start) + 16 * q + n] = v2;  // replicas agree
        raise |= __ballot(v2 > m_own[st] + kLazy);
      }
    }
    // --- lazy running max (per query; rare after the first tokens)
    if (raise) {
      float f[G];
#pragma unroll
      for (int i = 0; i < G; ++i) f[i] = 1.0f;
#pragma unroll
      for (int st = 0; st < NSET; ++st) {
        float mx = s2[0][st];
#pragma unroll
        for (int q = 1; q < kKT; ++q) mx = fmaxf(mx, s2[q][st]);
        mx = row_max16(mx);
        float ra[4];
#pragma unroll
        for (int ap = 0; ap < 4; ++ap) ra[ap] = lane_value(mx, 16 * ap);
#pragma unroll
        for (int s3 = 0; s3 < QS; ++s3) {
          float qm = kNegInf;
#pragma unroll
          for (int ap = 0; ap < 4; ++ap)
            if (ap % QS == s3) qm = fmaxf(qm, ra[ap]);
          const int iq = s3 + 4 * st;
          if (qm > m2q[iq]) {
            f[iq] = m2q[iq] == kNegInf ? 0.0f : __builtin_amdgcn_exp2f(m2q[iq] - qm);
            m2q[iq] = qm;
          }
        }
      }
#pragma unroll
      for (int st = 0; st < NSET; ++st) {
        float fo = f[4 * st], mo = m2q[4 * st];
#pragma unroll
        for (int s3 = 1; s3 < QS; ++s3) {
          fo = qs == s3 ? f[s3 + 4 * st] : fo;
          mo = qs == s3 ? m2q[s3 + 4 * st] : mo;
        }
        m_own[st] = mo;
        l_l[st] *= fo;
#pragma unroll
        for (int j = 0; j < NGL; ++j) bs_l[st][j] *= fo;
      }
      // value accumulators: register r of lane group a is row 4a + r, query (4a + r) / 2
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float fr = 1.0f;
#pragma unroll
        for (int i = 0; i < G; ++i) fr = (4 * a + r) / 2 == i ? f[i] : fr;
#pragma unroll
        for (int nb = 0; nb < 8; ++nb) CV[nb][r] *= fr;
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    load(cur, it + 1, true, false, live);
    __builtin_amdgcn_sched_barrier(0);
    // --- weights e * alpha into LDS (the A layout of the value MFMAs)
#pragma unroll
    for (int q = 0; q < kKT; ++q) {
      const int p = 16 * q + n, vt = p >> 5, u = p & 31;
      const int gv = u >> 3, ei = tau8(u & 7);
#pragma unroll
      for (int st = 0; st < NSET; ++st) {
        const int iq = qs + 4 * st;
        const float e = __builtin_amdgcn_exp2f(s2[q][st] - m_own[st]);  // 0 for -inf scores
        l_l[st] += e;
#pragma unroll
        for (int j = 0; j < NGL; ++j) {
          const int gm = (rho + R * j) % NG;
          const half2_t vab = as_h2(cur.vp[q][j]);  // (alpha, beta) of the value group
          bs_l[st][j] = fmaf(e * dup[j], (float)vab.y, bs_l[st][j]);
          // e * alpha as fp16 high and low parts, each one mixed FMA: the low
          // part rounds the exact residual e * alpha - high
          const _Float16 wh = (_Float16)fmaf(e, (float)vab.x, 0.0f);
          const _Float16 wl = (_Float16)fmaf(e, (float)vab.x, -(float)wh);
          w_lds[w_index(gm, vt, 2 * iq, gv, ei)] = wh;
          w_lds[w_index(gm, vt, 2 * iq + 1, gv, ei)] = wl;
        }
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // --- value MFMAs
#pragma unroll
    for (int vt = 0; vt < kVT; ++vt) {
      h8_t AV[NG];
#pragma unroll
      for (int gm = 0; gm < NG; ++gm) AV[gm] = *reinterpret_cast<const h8_t *>(w_lds + w_index(gm, vt, n, a, 0));
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) {
        // channels 16 nb + n: segment j = nb / 2 (field j of every byte),
        // bytes n + 16 (nb % 2) of the lane's 8 slots
        const int j = nb >> 1;
        const uint32_t d0 = cur.vc[vt][2 * (nb & 1)], d1 = cur.vc[vt][2 * (nb & 1) + 1];
        CV[nb] = mfma32(AV[(16 * nb) / GROUP],
                        pack_h8((d0 << (8 - 2 * j)) & mk, (d0 >> (2 * j)) & mk, (d1 << (8 - 2 * j)) & mk,
                                (d1 >> (2 * j)) & mk),
                        CV[nb]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    load(cur, it + 1, false, true, live);
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }

  // Scores of the chunk: one burst from LDS.
  const int nc = A.nc_hi + A.nc_lo;
  if (scores) {
#pragma unroll
    for (int i = 0; i < G; ++i) {
      float *row = scores + (int64_t)(qh0 + i) * cap;
      for (int j = lane; j < end - start; j += 64) __builtin_nontemporal_store(s_lds[i * max_chunk(G) + j], &row[start + j]);
    }
  }
  // Normalisers and zero terms per (query, group), wave-uniform.
  float lq[G], bq[G][NG];
#pragma unroll
  for (int st = 0; st < NSET; ++st) {
    const float lr = row_sum16(l_l[st]);
    float br[NGL];
#pragma unroll
    for (int j = 0; j < NGL; ++j) br[j] = row_sum16(bs_l[st][j]);
#pragma unroll
    for (int s3 = 0; s3 < QS; ++s3) {
      const int iq = s3 + 4 * st;
      lq[iq] = lane_value(lr, 16 * s3);  // replica 0 of the slot
#pragma unroll
      for (int gm = 0; gm < NG; ++gm) bq[iq][gm] = lane_value(br[gm / R], 16 * (s3 + QS * (gm % R)));
    }
  }
  // Record per query: max, normaliser, value sums (lane group i/2 holds
  // query i in registers 2(i%2), 2(i%2)+1).
  constexpr float colscale = 65536.0f;  // undoes the value encoding (code * 2^-16)
#pragma unroll
  for (int i = 0; i < G; ++i) {
    float *rec = A.partials + ((int64_t)(qh0 + i) * nc + rec_chunk) * kRec;
    if (lane == 0) {
      rec[0] = m2q[i];
      rec[1] = lq[i];
      rec[kRecN] = __builtin_bit_cast(float, n_pool);
    }
    if (a == i / 2) {
      const int r0 = 2 * (i % 2);
#pragma unroll
      for (int nb = 0; nb < 8; ++nb) rec[kRecO + 16 * nb + n] = fmaf(CV[nb][r0] + CV[nb][r0 + 1], colscale, bq[i][(16 * nb) / GROUP]);
    }
  }
}

// Tuning: token tiles per lane per iteration and prefetch depth (-1: the
// half-step pipeline of attn_chunk), for low-bit (INT2/INT4) and high-bit
// (fp16/INT8) rows.
#ifndef MIKV_UNROLL_LOWBIT
#define MIKV_UNROLL_LOWBIT 8
#endif
#ifndef MIKV_UNROLL_HIGHBIT
#define MIKV_UNROLL_HIGHBIT 2
#endif
#ifndef MIKV_PREFETCH_LOWBIT
#define MIKV_PREFETCH_LOWBIT -1
#endif
#ifndef MIKV_PREFETCH_HIGHBIT
#define MIKV_PREFETCH_HIGHBIT -1
#endif
// INT4 rows are twice the INT2 ones: half the tiles per iteration keep the
// same bytes in flight and the registers of one more wave per SIMD.
#ifndef MIKV_UNROLL_INT4
#define MIKV_UNROLL_INT4 4
#endif
// A balanced 2-bit pool (the query in two fp16 parts) takes half the tiles:
// with eight it needs 171 registers and two waves per SIMD, with four 136 and
// three (llama2_13b: 266.6-272.1 -> 261.4-264.4 us per launch, step 303.7-307.4
// -> 299.2-299.8 us; long_context, unbalanced, keeps eight: four measured
// even).
#ifndef MIKV_UNROLL_LOWBIT_SPLIT
#define MIKV_UNROLL_LOWBIT_SPLIT 4
#endif
template <int BITS, bool SPLITQ = false>
constexpr int unroll_for() {
  return BITS == 4 || BITS == 3 ? MIKV_UNROLL_INT4
       : BITS <= 4              ? (SPLITQ ? MIKV_UNROLL_LOWBIT_SPLIT : MIKV_UNROLL_LOWBIT)
                                : MIKV_UNROLL_HIGHBIT;
}
// An fp16 importance pool with one query head per KV head (the least work
// per byte) keeps four tiles in flight (long_context 106.5-107.0 -> 105.0-
// 105.5 us per step); under GQA and for INT8 pools four were slower
// (mistral_7b 87.0 -> 92.8, llama2_7b 44.4 -> 46.0).
#ifndef MIKV_UNROLL_F16_MHA
#define MIKV_UNROLL_F16_MHA 4
#endif
template <int HI, int G>
constexpr int unroll_hi() { return HI == 16 && G == 1 ? MIKV_UNROLL_F16_MHA : unroll_for<HI>(); }
template <int BITS>
constexpr int prefetch_for() { return BITS <= 4 ? MIKV_PREFETCH_LOWBIT : MIKV_PREFETCH_HIGHBIT; }

// Query heads per KV head from which a lane holds 16 channels instead of 32
// (fewer accumulators per lane at larger GQA groups).
#ifndef MIKV_NARROW_FROM_G
#define MIKV_NARROW_FROM_G 4
#endif
#ifndef MIKV_WAVES_PER_EU
#define MIKV_WAVES_PER_EU 1
#endif
#ifndef MIKV_CHUNK_KB
#define MIKV_CHUNK_KB 96  // under GQA
#endif
#ifndef MIKV_CHUNK_KB_MHA
#define MIKV_CHUNK_KB_MHA 64  // one query head per KV head (measured: 13B shape -2.5 %, long_context even)
#endif
#ifndef MIKV_CHUNK_HI_SCALE
#define MIKV_CHUNK_HI_SCALE 2  // MHA importance-pool chunks hold this many times the bytes
#endif
#ifndef MIKV_CHUNK_HI_SCALE_F16
#define MIKV_CHUNK_HI_SCALE_F16 4  // the same for an fp16 importance pool
#endif

// The decode step's new token: written into importance-pool slot n_hi by
// the wave whose chunk holds that slot, before the wave reads its chunk (no
// other wave reads the slot, and chunks are whole iterations, so no other
// wave's loads reach it).  A full pool sets the status bit instead (wave
// of chunk 0).
template <int HI>
__device__ inline void append_in_chunk(const AttnArgs &A, int h, int chunk) {
  const int n0 = __builtin_amdgcn_readfirstlane(A.n_hi[h]);
  const int lane = threadIdx.x & 63;
  if (n0 >= A.cap_hi) {
    if (chunk == 0 && lane == 0) atomicOr(A.app.status, MIKV_DEVERR_HI_FULL);
    return;
  }
  if (chunk != n0 / A.chunk_hi) return;
  if (lane < 8) append_row<HI>(A.app, h, n0, lane);
  // the lanes that read the slot see the stored row (one wave per block)
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

template <int HI, int LO, int G, bool SPLITQ, bool KPC = false>
__global__ __launch_bounds__(64) __attribute__((amdgpu_waves_per_eu(MIKV_WAVES_PER_EU)))
void attn_partial_kernel(AttnArgs A) {
  constexpr int CPL = G >= MIKV_NARROW_FROM_G ? 16 : 32;  // channels per lane
  // 3-, 4- and 8-bit retained pools at eight query heads per KV head: 8
  // channels per lane (a 3-, 4- or 8-byte segment), so the lane's G x CPL
  // value sums fit the registers of two waves per SIMD instead of spilling
  constexpr int CPL_LO = (LO == 3 || LO == 4 || LO == 8) && G >= 8 ? 8 : CPL;
  // fp16 importance pool: 16 channels per lane in two spread pieces, so the
  // lanes of a token read whole 128-byte lines with each load (which
  // non-temporal loads need to fetch a line once, and which read the
  // resident rows faster too: long_context with an evicting cache 38.9 ->
  // 36.2 us per launch); with eight query heads per KV head 8 channels, which
  // halves the value sums a lane holds (G x CPL registers), and so do INT8
  // and INT4 importance pools at eight.  INT8 below eight: streamed rows 16
  // channels per lane (one piece per line), resident rows the wider lanes,
  // which cost fewer cross-lane sums per token.
  constexpr int CPL_HI = G >= 8 ? 8 : HI == 16 ? 16 : CPL;
  constexpr int CPL_HI_S = G >= 8 ? 8 : HI == 16 || HI == 8 ? 16 : CPL;
  // Block -> (head, chunk): first every head's importance-pool chunks and
  // the retained-pool chunks that cannot be empty (nc_first per head; with
  // pool_major all importance-pool chunks, the longest-running waves of an
  // fp16 pool, before any retained-pool chunk), then
  // the retained-pool chunks that may be (a wave that finds its chunk empty
  // costs little at the end of the grid, but holds up the dispatch of the
  // work behind it anywhere else).
  // Every other step runs the order backwards (A.order, set from the
  // cache length): the last-level cache still holds the end of the previous
  // step's stream, which is then read first.
  const int n_heads = gridDim.x / (A.nc_hi + A.nc_lo);
  const int n_first = n_heads * A.nc_first;  // blocks of the first part
  const int bid = A.order == 2 ? (int)gridDim.x - 1 - (int)blockIdx.x : (int)blockIdx.x;
  int h, c;
  if (A.pool_major && bid < n_heads * A.nc_hi) {
    h = bid / A.nc_hi;
    c = bid % A.nc_hi;
  } else if (A.pool_major && bid < n_first) {
    const int e = bid - n_heads * A.nc_hi, per = A.nc_first - A.nc_hi;
    h = e / per;
    c = A.nc_hi + e % per;
  } else if (bid < n_first) {
    h = bid / A.nc_first;
    c = bid % A.nc_first;
  } else {
    const int rest = A.nc_hi + A.nc_lo - A.nc_first, e = bid - n_first;
    h = e / rest;
    c = A.nc_first + e % rest;
  }
  if (A.order == 1) h = n_heads - 1 - h;
  __shared__ float s_lds[G * max_chunk(G)];  // the chunk's scores, [G][max_chunk(G)]
  // The rows of the first res_hi / res_lo heads of each pool (as much as the
  // last-level cache keeps from one step to the next) are read with plain
  // loads, which that cache allocates; all other rows are streamed with
  // non-temporal loads, which do not push the resident rows out.
  if (c < A.nc_hi) {
    if (A.hi_pending) append_in_chunk<HI>(A, h, c);
    if (h < A.res_hi)
      attn_chunk<HI, G, CPL_HI, SPLITQ, unroll_hi<HI, G>(), prefetch_for<HI>()>(A, h, c, c, true, s_lds);
    else
      attn_chunk<HI, G, CPL_HI_S, SPLITQ, unroll_hi<HI, G>(), prefetch_for<HI>(), false, true>(A, h, c, c, true, s_lds);
  } else if constexpr (KPC) {
    attn_chunk<LO, G, CPL, SPLITQ, unroll_for<LO>(), prefetch_for<LO>(), true>(A, h, c - A.nc_hi, c, false, s_lds);
  } else if constexpr (LO == 2 && G >= 2) {
    __shared__ __align__(16) _Float16 w_lds[kWLds];  // value-MFMA weights, see w_index
    const bool res = h < A.res_lo;
    if (A.group == 32) {
      if (res) attn_chunk_int2<G, SPLITQ, 4, false>(A, h, c - A.nc_hi, c, s_lds, w_lds);
      else attn_chunk_int2<G, SPLITQ, 4, true>(A, h, c - A.nc_hi, c, s_lds, w_lds);
    } else if (A.group == 64) {
      if (res) attn_chunk_int2<G, SPLITQ, 2, false>(A, h, c - A.nc_hi, c, s_lds, w_lds);
      else attn_chunk_int2<G, SPLITQ, 2, true>(A, h, c - A.nc_hi, c, s_lds, w_lds);
    } else {
      if (res) attn_chunk_int2<G, SPLITQ, 1, false>(A, h, c - A.nc_hi, c, s_lds, w_lds);
      else attn_chunk_int2<G, SPLITQ, 1, true>(A, h, c - A.nc_hi, c, s_lds, w_lds);
    }
  } else {
    if (h < A.res_lo)
      attn_chunk<LO, G, CPL_LO, SPLITQ, unroll_for<LO, SPLITQ>(), prefetch_for<LO>()>(A, h, c - A.nc_hi, c, false, s_lds);
    else
      attn_chunk<LO, G, CPL_LO, SPLITQ, unroll_for<LO, SPLITQ>(), prefetch_for<LO>(), false, true>(A, h, c - A.nc_hi, c, false, s_lds);
  }
}

// Softmax over the whole sequence from the chunk records (Section 2.1): a
// query head's max M is the largest chunk max, its normaliser L the chunk
// sums rescaled by exp2(m_r - M); the output is the rescaled value sums / L.
// Each block of the finalize kernel derives (M, 1/L) of the G query heads of
// KV head h from the (m, l) pairs, then turns one tile of scores into
// probabilities (and adds their GQA sum to the importance scores when
// asked); block 0 also merges the value sums into the output.
constexpr int kProbTile = 8 * kBlock;  // scores per block and query head

// (M, 1/L) of query heads qh0 .. qh0+G-1, computed by every wave on its own
// (no LDS, no barrier): lane r merges the (m, l) pairs of records r, r+64, ...
template <int G>
__device__ inline void head_stats(const AttnArgs &A, int qh0, int nc, float M[G], float inv[G]) {
  const int lane = threadIdx.x & 63;
  float m[G], l[G];
#pragma unroll
  for (int i = 0; i < G; ++i) {
    m[i] = kNegInf;
    l[i] = 0.0f;
  }
  for (int r = lane; r < nc; r += 64) {
    float2 ml[G];
#pragma unroll
    for (int i = 0; i < G; ++i)
      ml[i] = *reinterpret_cast<const float2 *>(A.partials + ((int64_t)(qh0 + i) * nc + r) * kRec);
#pragma unroll
    for (int i = 0; i < G; ++i) {
      if (ml[i].x > m[i]) {
        l[i] = fmaf(l[i], __builtin_amdgcn_exp2f(m[i] - ml[i].x), ml[i].y);
        m[i] = ml[i].x;
      } else if (ml[i].x != kNegInf) {
        l[i] = fmaf(ml[i].y, __builtin_amdgcn_exp2f(ml[i].x - m[i]), l[i]);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < G; ++i) {
    M[i] = wave_max(m[i]);
    inv[i] = 1.0f / wave_sum(m[i] == kNegInf ? 0.0f : l[i] * __builtin_amdgcn_exp2f(m[i] - M[i]));
  }
}

// One probability tile (kProbTile scores of every query head of KV head h):
// loaded first, so that the latency overlaps the statistics, then stored.
template <int G>
struct ProbTile {
  static constexpr int kPer = kProbTile / kBlock;
  float sv[kPer][G], a[kPer];
  int t[kPer];
  int n_pool;
};

// n_pool: the pool's token count (< 0: read the live counter).
template <int G>
__device__ inline ProbTile<G> prob_tile_load(const AttnArgs &A, int h, int qh0, bool is_hi, int tile, bool has_tile,
                                             bool accumulate, int n_pool = -1) {
  ProbTile<G> T;
  const int cap = is_hi ? A.cap_hi : A.cap_lo;
  const float *scores = is_hi ? A.scores_hi : A.scores_lo;
  const float *acc = is_hi && accumulate ? A.acc : nullptr;
#pragma unroll
  for (int u = 0; u < ProbTile<G>::kPer; ++u) {
    T.t[u] = tile * kProbTile + u * kBlock + threadIdx.x;
    const bool ok = has_tile && T.t[u] < cap;
#pragma unroll
    for (int i = 0; i < G; ++i)
      T.sv[u][i] = ok ? __builtin_nontemporal_load(&scores[(int64_t)(qh0 + i) * cap + T.t[u]]) : 0.0f;
    T.a[u] = ok && acc ? acc[(int64_t)h * A.cap_hi + T.t[u]] : 0.0f;
  }
  T.n_pool = !has_tile ? 0 : n_pool >= 0 ? n_pool : is_hi ? hi_count(A, h) : A.n_lo[h];
  return T;
}

// Probabilities of one tile, stored; with the importance update, the new
// score of every slot also goes to a_new[u] (the old one past the pool).
template <int G>
__device__ inline void prob_tile_store(const AttnArgs &A, int h, int qh0, bool is_hi, bool accumulate,
                                       const ProbTile<G> &T, const float M[G], const float inv[G],
                                       float *a_new = nullptr) {
  const int cap = is_hi ? A.cap_hi : A.cap_lo;
  float *probs = is_hi ? A.probs_hi : A.probs_lo;
  float *acc = is_hi && accumulate ? A.acc : nullptr;
#pragma unroll
  for (int u = 0; u < ProbTile<G>::kPer; ++u) {
    if (T.t[u] >= T.n_pool) {
      if (a_new) a_new[u] = T.a[u];
      continue;
    }
    float sum = 0.0f;
#pragma unroll
    for (int i = 0; i < G; ++i) {
      const float p = __builtin_amdgcn_exp2f(T.sv[u][i] - M[i]) * inv[i];
      if (probs) __builtin_nontemporal_store(p, &probs[(int64_t)(qh0 + i) * cap + T.t[u]]);
      sum = i == 0 ? p : sum + p;
    }
    const float an = T.a[u] + sum;
    if (acc) acc[(int64_t)h * A.cap_hi + T.t[u]] = an;
    if (a_new) a_new[u] = an;
  }
}

// Output merge of the G query heads (whole block): thread -> (record split
// s, query head i, 4 channels q4), partial sums reduced in LDS.
template <int G>
__device__ inline void merge_output(const AttnArgs &A, int qh0, int nc, const float M[G], const float inv[G]) {
  constexpr int S = 8 / G;
  // Up to four query heads, a wave works on one head (i wave-uniform, so
  // picking its statistics is a scalar select, not a per-lane indexed array);
  // eight heads take two per wave.
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int q4 = lane & 31;
  const int i = G <= 4 ? __builtin_amdgcn_readfirstlane(wave % G) : (threadIdx.x / 32) % G;
  const int s = G <= 4 ? (wave / G) * 2 + (lane >> 5) : threadIdx.x / (32 * G);
  const float *rec = A.partials + (int64_t)(qh0 + i) * nc * kRec;
  float Mi = M[0], invi = inv[0];
#pragma unroll
  for (int j = 1; j < G; ++j)
    if (i == j) {
      Mi = M[j];
      invi = inv[j];
    }
  float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  // RB records per thread and batch, all loaded before any is used (a
  // missing record reads record 0 and gets weight 0): one memory round trip
  // per batch (a plain loop waits for every record in turn)
  constexpr int RB = 8;
  for (int r0 = s; r0 < nc; r0 += RB * S) {
    float mr[RB];
    float4 o[RB];
#pragma unroll
    for (int k = 0; k < RB; ++k) {
      const int r = r0 + k * S;
      const float *rr = rec + (int64_t)(r < nc ? r : 0) * kRec;
      mr[k] = r < nc ? rr[0] : kNegInf;
      o[k] = reinterpret_cast<const float4 *>(rr + kRecO)[q4];
    }
#pragma unroll
    for (int k = 0; k < RB; ++k) {
      const float w = mr[k] == kNegInf ? 0.0f : __builtin_amdgcn_exp2f(mr[k] - Mi);
      v.x = fmaf(o[k].x, w, v.x);
      v.y = fmaf(o[k].y, w, v.y);
      v.z = fmaf(o[k].z, w, v.z);
      v.w = fmaf(o[k].w, w, v.w);
    }
  }
  __shared__ float4 s_o[kBlock];
  const int slot = (s * G + i) * 32 + q4;  // LDS by (split, head, channels)
  s_o[slot] = v;
  __syncthreads();
  if (s == 0) {
    for (int s2 = 1; s2 < S; ++s2) {
      const float4 u = s_o[slot + s2 * 32 * G];
      v.x += u.x;
      v.y += u.y;
      v.z += u.z;
      v.w += u.w;
    }
    reinterpret_cast<float4 *>(A.out + (int64_t)(qh0 + i) * kHeadDim)[q4] =
        make_float4(v.x * invi, v.y * invi, v.z * invi, v.w * invi);
  }
}

// Block (h, 0) merges the output of head h; blocks (h, 1..) turn one
// probability tile each into probabilities (importance-pool tiles first).
// Heads run along x, so the longest blocks, the merges, are dispatched first.
// (Register budget: 8 blocks per CU for one query head per KV head, 6 for
// two; the grids of many-head caches hold several blocks per CU.)
template <int G>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(G == 1 ? 8 : G == 2 ? 6 : 1)))
void attn_finalize_kernel(AttnArgs A, int accumulate, int tiles_hi, int tiles_lo) {
  const int h = blockIdx.x, c = blockIdx.y;  // heads fastest: every head's block 0 is dispatched first
  const int b = h / A.kv_heads, kvh = h % A.kv_heads;
  const int qh0 = b * A.q_heads + kvh * G;
  const int nc = A.nc_hi + A.nc_lo;
  float M[G], inv[G];
  if (c == 0) {  // the merge holds no tile
    head_stats<G>(A, qh0, nc, M, inv);
    merge_output<G>(A, qh0, nc, M, inv);
    return;
  }
  const int tile = c - 1;
  const bool is_hi = tile < tiles_hi;
  const bool has_tile = is_hi || tile - tiles_hi < tiles_lo;
  const ProbTile<G> T = prob_tile_load<G>(A, h, qh0, is_hi, is_hi ? tile : tile - tiles_hi, has_tile, accumulate);
  head_stats<G>(A, qh0, nc, M, inv);
  if (has_tile) prob_tile_store<G>(A, h, qh0, is_hi, accumulate, T, M, inv);
}

// Finalize with the importance update and the re-rank fused (the decode
// step).  Block (h, 0) of head h turns every importance-pool tile into
// probabilities and new scores and, its own writes being the only scores
// the re-rank reads, runs the head's top-k and demotion on the scores it
// still holds in registers (the positions and the last slot are loaded
// with the tiles, so the re-rank adds one memory round trip: the demoted
// row).  Block (h, 1) merges the output; blocks (h, 2..) handle the
// retained-pool tiles.  Heads run along x, so every head's re-rank block is
// dispatched before any tile block.  No block waits on another.
#ifndef MIKV_LO_TILES
#define MIKV_LO_TILES 8
#endif
// Retained-pool probability tiles per finalize block (a tile per query head
// of the group costs the same registers as G tiles of one head):
// MIKV_LO_TILES / G, except 4 at G = 4, where the fewer, longer blocks (216
// registers, two waves per SIMD) finish the step sooner than 2 or 1 tiles
// per block (8 is slower again).
#ifndef MIKV_LO_TILES_G4
#define MIKV_LO_TILES_G4 4
#endif
__host__ __device__ constexpr int lo_tiles_per_block(int G) {
  return G == 4 ? MIKV_LO_TILES_G4 : MIKV_LO_TILES / G > 1 ? MIKV_LO_TILES / G : 1;
}

template <int G, int HI, int LO>
__global__ __launch_bounds__(kBlock) void finalize_select_kernel(AttnArgs A, int tiles_hi, int tiles_lo, SelArgs S) {
  static_assert(kSel == kBlock && kSelItems * kBlock == 2 * kProbTile, "select items = two probability tiles");
  const int h = blockIdx.x, c = blockIdx.y;  // heads fastest: every head's block 0 is dispatched first
  const int b = h / A.kv_heads, kvh = h % A.kv_heads;
  const int qh0 = b * A.q_heads + kvh * G;
  const int nc = A.nc_hi + A.nc_lo;
  if (c == 1) {  // the merge holds no tile
    float M[G], inv[G];
    head_stats<G>(A, qh0, nc, M, inv);
    merge_output<G>(A, qh0, nc, M, inv);
    return;
  }
  if (c > 1) {
    // kLoTiles retained-pool tiles per block, all loaded before the
    // statistics: fewer, longer blocks (one round of blocks per step).
    // Block (h, 0) raises n_lo when it demotes, concurrently with this
    // block, so the retained pool's size at attention time comes from the
    // record of the head's first retained-pool chunk, written by the
    // partial phase.
    constexpr int KT = lo_tiles_per_block(G);
    const int t0 = (c - 2) * KT;
    const int n_lo_att = __builtin_bit_cast(
        int, A.partials[((int64_t)qh0 * nc + A.nc_hi) * kRec + kRecN]);
    ProbTile<G> T[KT];
#pragma unroll
    for (int k = 0; k < KT; ++k)
      T[k] = prob_tile_load<G>(A, h, qh0, false, t0 + k, t0 + k < tiles_lo, false, n_lo_att);
    float M[G], inv[G];
    head_stats<G>(A, qh0, nc, M, inv);
#pragma unroll
    for (int k = 0; k < KT; ++k)
      if (t0 + k < tiles_lo) prob_tile_store<G>(A, h, qh0, false, false, T[k], M, inv);
    return;
  }
  // Everything the re-rank reads besides the new scores is loaded together
  // with the first two tiles and the chunk statistics.
  const int n = __builtin_amdgcn_readfirstlane(hi_count(A, h));
  const int n_lo0 = __builtin_amdgcn_readfirstlane(S.n_lo[h]);
  const int thr = S.length - S.window;  // positions >= thr are in the window
  // two tiles in flight for one or two query heads per KV head; with more,
  // the second waits for the statistics (the block's register budget also
  // bounds the occupancy of the retained-pool tile blocks)
  constexpr bool kTwoAhead = G <= 2;
  const ProbTile<G> T0 = prob_tile_load<G>(A, h, qh0, true, 0, tiles_hi > 0, true);
  ProbTile<G> T1;
  if constexpr (kTwoAhead) T1 = prob_tile_load<G>(A, h, qh0, true, 1, tiles_hi > 1, true);
  int pv[kSelItems];
  const int32_t *pos = S.hi_pos + (int64_t)h * S.cap_hi;
#pragma unroll
  for (int u = 0; u < kSelItems; ++u) {
    const int i = u * kSel + threadIdx.x;
    pv[u] = i < S.cap_hi ? pos[i] : thr;
  }
  SlotData<HI> last = n > 0 ? load_slot<HI>(S, h, n - 1) : SlotData<HI>{};
  float M[G], inv[G];
  head_stats<G>(A, qh0, nc, M, inv);
  float an[kSelItems];
  prob_tile_store<G>(A, h, qh0, true, true, T0, M, inv, an);
  if constexpr (!kTwoAhead) T1 = prob_tile_load<G>(A, h, qh0, true, 1, tiles_hi > 1, true);
  prob_tile_store<G>(A, h, qh0, true, true, T1, M, inv, an + ProbTile<G>::kPer);
  for (int tile = 2; tile < tiles_hi; ++tile) {
    const ProbTile<G> T = prob_tile_load<G>(A, h, qh0, true, tile, true, true);
    prob_tile_store<G>(A, h, qh0, true, true, T, M, inv);
  }
  // slot u * kSel + t of thread t is item u of the two first tiles
  SelScan sc;
  __shared__ float s_last;
#pragma unroll
  for (int u = 0; u < kSelItems; ++u) {
    const int i = u * kSel + threadIdx.x;
    if (i < n && pv[u] < thr) sc.add(i, pv[u], an[u]);
    if (i == n - 1) s_last = an[u];
  }
  // slots past the first two tiles: from memory, written above by this same thread
  if (S.cap_hi > kSel * kSelItems) select_scan(S, h, kSel * kSelItems, n, thr, sc);
  __syncthreads();  // the block's score updates (and s_last) are complete before the re-rank uses them
  if (threadIdx.x == 0 && n > 0)
    last.acc = n - 1 < kSel * kSelItems ? s_last : S.hi_acc[(int64_t)h * S.cap_hi + n - 1];
  select_finish<HI, LO>(S, h, n, n_lo0, sc, last, A.hi_pending != 0);
}

template <int G>
__global__ __launch_bounds__(kBlock) void importance_kernel(float *acc, const float *probs, const int32_t *n_hi,
                                                            int cap_hi, int q_heads, int kv_heads) {
  const int h = blockIdx.y;
  const int t = blockIdx.x * kBlock + threadIdx.x;
  if (t >= n_hi[h]) return;
  const int b = h / kv_heads, kvh = h % kv_heads;
  const int qh0 = b * q_heads + kvh * G;
  float sum = probs[(int64_t)qh0 * cap_hi + t];
#pragma unroll
  for (int i = 1; i < G; ++i) sum = sum + probs[(int64_t)(qh0 + i) * cap_hi + t];
  acc[(int64_t)h * cap_hi + t] += sum;
}

// ---------------------------------------------------------------------------
// Host side.
// ---------------------------------------------------------------------------
struct Plan {
  int chunk_hi, chunk_lo, nc_hi, nc_lo;
  int nc_first;  // nc_hi + the retained-pool chunks that hold tokens whatever the split
  int64_t head_bytes_hi, head_bytes_lo;  // packed bytes of one head's occupied span per pool (upper bound)
};

int round_up(int64_t x, int m) { return (int)(((x + m - 1) / m) * m); }

// The resident share (mikv_set_resident_bytes): bytes of a cache read with
// plain loads.
std::atomic<int64_t> g_resident_bytes{kResidentBytes};
int64_t resident_budget() { return g_resident_bytes.load(std::memory_order_relaxed); }

// size_bound: the plan with the most chunks the resident share can give
// (workspaces are sized from it, so a workspace stays large enough when the
// share changes).
Plan make_plan(const mikv_cache *c, int length, bool size_bound = false) {
  Plan p;
  const int64_t NH = n_heads_of(c);
  // an evicting cache has no retained pool: no chunks for it
  const int span_hi = std::min(length, c->cap_hi), span_lo = evicting(c) ? 0 : std::min(length, c->cap_lo);
  const int64_t bh = token_bytes(c->hi_bits, c->group), bl = token_bytes(evicting(c) ? 2 : c->lo_bits, c->group);
  const int64_t total = NH * (span_hi * bh + span_lo * bl);
  p.head_bytes_hi = span_hi * bh;
  p.head_bytes_lo = span_lo * bl;
  // One wave per chunk; up to 64 KiB (MHA) or 96 KiB (GQA) of packed K/V per
  // chunk (many small work units balance the CUs best), at least 16 KiB so
  // the per-chunk merge stays cheap.  Chunks are whole wave iterations (128
  // tokens).
  const int64_t chunk_kb = group_size_of(c) == 1 ? MIKV_CHUNK_KB_MHA : MIKV_CHUNK_KB;
  int64_t target = std::max<int64_t>(std::min<int64_t>(total / 4096, chunk_kb << 10), 16 << 10);
  const int cmax = max_chunk(group_size_of(c));
  // MHA importance-pool rows cost the least work per byte: more bytes per
  // chunk there cut the per-wave overhead (twice: 4 % of the long_context
  // step).  Four times pays only for an fp16 pool read from the last-level
  // cache (the whole pool within the resident share: long_context warm
  // 1.3 % faster); streamed from HBM those longer waves were slower (cold
  // step 130 -> 134 us), and an INT8 pool lost 2.6 % at the 13B shape.
  // GQA rows carry G queries' work and keep one share.
  const bool hi_resident = !size_bound && NH * p.head_bytes_hi <= resident_budget();
  const int64_t hi_scale = c->hi_bits == 16 && hi_resident ? MIKV_CHUNK_HI_SCALE_F16 : MIKV_CHUNK_HI_SCALE;
  const int64_t target_hi = group_size_of(c) == 1 ? target * hi_scale : target;
  p.chunk_hi = std::min(cmax, std::max(128, round_up(target_hi / bh, 128)));
  p.chunk_lo = std::min(cmax, std::max(128, round_up(target / bl, 128)));
  p.nc_hi = std::max(1, (span_hi + p.chunk_hi - 1) / p.chunk_hi);
  p.nc_lo = evicting(c) ? 0 : std::max(1, (span_lo + p.chunk_lo - 1) / p.chunk_lo);
  // every token is in one of the pools, so at least length - cap_hi are in
  // the retained one (only the dispatch order depends on this)
  const int lo_min = std::max(0, std::min(span_lo, length - c->cap_hi));
  p.nc_first = p.nc_hi + std::min(p.nc_lo, (lo_min + p.chunk_lo - 1) / p.chunk_lo);
  return p;
}

size_t workspace_bytes_for(const mikv_cache *c, const Plan &p) {
  const int64_t BQ = (int64_t)c->batch * c->q_heads;
  return (size_t)(BQ * (p.nc_hi + p.nc_lo) * kRec * 4 + BQ * c->cap_hi * 4);
}

AttnArgs make_args(const mikv_cache *c, const Plan &p, const uint16_t *q, const float *balance, float scale,
                   float *out, float *probs_hi, float *probs_lo, int flags, void *ws) {
  AttnArgs A;
  A.hi_k = (const uint8_t *)c->hi_k;
  A.hi_v = (const uint8_t *)c->hi_v;
  A.hi_kp = (const uint32_t *)c->hi_kp;
  A.hi_vp = (const uint32_t *)c->hi_vp;
  A.n_hi = c->n_hi;
  A.lo_k = c->lo_k;
  A.lo_v = c->lo_v;
  A.lo_kp = (const uint32_t *)c->lo_kp;
  A.lo_vp = (const uint32_t *)c->lo_vp;
  A.n_lo = c->n_lo;
  A.q = q;
  A.balance = balance;
  A.scale = scale;
  const int64_t BQ = (int64_t)c->batch * c->q_heads;
  A.partials = (float *)ws;
  float *ws_scores = A.partials + BQ * (p.nc_hi + p.nc_lo) * kRec;
  const bool acc = (flags & MIKV_ATTN_ACCUMULATE) != 0;
  A.scores_hi = probs_hi ? probs_hi : (acc ? ws_scores : nullptr);
  A.scores_lo = probs_lo;
  A.probs_hi = probs_hi;
  A.probs_lo = probs_lo;
  A.acc = acc ? c->hi_acc : nullptr;
  A.out = out;
  A.cap_hi = c->cap_hi;
  A.cap_lo = c->cap_lo;
  A.group = c->group;
  A.q_heads = c->q_heads;
  A.kv_heads = c->kv_heads;
  A.chunk_hi = p.chunk_hi;
  A.chunk_lo = p.chunk_lo;
  A.nc_hi = p.nc_hi;
  A.nc_lo = p.nc_lo;
  A.nc_first = p.nc_first;
  A.app = AppendArgs{};
  A.hi_pending = 0;
  // fp16 importance-pool chunks under GQA run longest: dispatched first, the
  // tail of the grid is shorter (measured: mistral_7b 66.0 -> 64.7 us per
  // launch).  With one query head per KV head the resident importance-pool
  // rows (last-level cache) and the streamed retained-pool rows (HBM) are
  // best read side by side, head by head (long_context 98.2 -> 95.0 us).
  A.pool_major = c->hi_bits == 16 && group_size_of(c) > 1 ? 1 : 0;
  A.order = 0;
  // Rows read plainly: up to resident_budget() bytes of the cache,
  // importance pool first (it is read by every step whatever the re-rank
  // does), then retained-pool heads.
  {
    const int64_t NH = n_heads_of(c);
    int64_t budget = resident_budget();
    const int64_t hb = std::max<int64_t>(p.head_bytes_hi, 1), lb = std::max<int64_t>(p.head_bytes_lo, 1);
    A.res_hi = (int)std::min<int64_t>(NH, budget / hb);
    budget -= (int64_t)A.res_hi * p.head_bytes_hi;
    A.res_lo = A.res_hi == NH ? (int)std::min<int64_t>(NH, budget / lb) : 0;
  }
  A.lo_kb = c->key_block ? (const uint32_t *)c->lo_kb : nullptr;
  A.lo_pos = c->lo_pos;
  A.n_kblk = c->key_block ? key_blocks_of(c) : 0;
  return A;
}

// The fold of the decode step's append into the attention (position
// length - 1).
void set_append(AttnArgs &A, const mikv_cache *c, int32_t length, const uint16_t *k_new, const uint16_t *v_new,
                const float *balance) {
  AppendArgs &a = A.app;
  a.hi_k = (uint8_t *)c->hi_k;
  a.hi_v = (uint8_t *)c->hi_v;
  a.hi_kp = (uint32_t *)c->hi_kp;
  a.hi_vp = (uint32_t *)c->hi_vp;
  a.hi_pos = c->hi_pos;
  a.hi_acc = c->hi_acc;
  a.map = c->map;
  a.status = c->status;
  a.k = k_new;
  a.v = v_new;
  a.balance = balance;
  a.score_init = nullptr;
  a.cap_hi = c->cap_hi;
  a.max_len = c->max_len;
  a.group = c->group;
  a.pos = length - 1;
  A.hi_pending = 1;
}

template <int HI, int LO, bool SPLITQ>
void launch_partial_q(const AttnArgs &A, int G, dim3 grid, hipStream_t st) {
  switch (G) {
    case 1: hipLaunchKernelGGL((attn_partial_kernel<HI, LO, 1, SPLITQ>), grid, dim3(64), 0, st, A); break;
    case 2: hipLaunchKernelGGL((attn_partial_kernel<HI, LO, 2, SPLITQ>), grid, dim3(64), 0, st, A); break;
    case 4: hipLaunchKernelGGL((attn_partial_kernel<HI, LO, 4, SPLITQ>), grid, dim3(64), 0, st, A); break;
    default: hipLaunchKernelGGL((attn_partial_kernel<HI, LO, 8, SPLITQ>), grid, dim3(64), 0, st, A); break;
  }
}

// A balanced query (q / b) is not an fp16 value in general: carry it as two
// fp16 parts.  An unbalanced query is fp16 already.
template <int HI, int LO>
void launch_partial_g(const AttnArgs &A, int G, dim3 grid, hipStream_t st) {
  if (A.balance)
    launch_partial_q<HI, LO, true>(A, G, grid, st);
  else
    launch_partial_q<HI, LO, false>(A, G, grid, st);
}

int check_attention_args(const mikv_cache *c, int32_t length, const uint16_t *q, const float *balance, float *out,
                         void *ws, size_t ws_bytes, const char *who) {
  int rc = validate_cache(c);
  if (rc) return rc;
  if (!q || !out) return set_error(MIKV_ERR_INVALID_ARG, "%s: q/out is NULL", who);
  if (((uintptr_t)q | (uintptr_t)balance) % 16 != 0)
    return set_error(MIKV_ERR_INVALID_ARG, "%s: q and balance must be 16-byte aligned", who);
  if (length < 1) return set_error(MIKV_ERR_INVALID_ARG, "%s: length must be >= 1", who);
  if (length > c->max_len) return set_error(MIKV_ERR_CAPACITY, "%s: length %d > max_len %d", who, length, c->max_len);
  size_t need = workspace_bytes_for(c, make_plan(c, length, true));
  if (!ws || ws_bytes < need) return set_error(MIKV_ERR_CAPACITY, "%s: workspace too small (%zu < %zu)", who, ws_bytes, need);
  return MIKV_OK;
}

}  // namespace

}  // namespace mikv

using namespace mikv;

extern "C" size_t mikv_decode_workspace_size(const mikv_cache *c, int32_t length) {
  if (!c || length < 1 || validate_cache(c)) return 0;
  return workspace_bytes_for(c, make_plan(c, length, true));
}

namespace mikv {

int decode_partial(const mikv_cache *c, int32_t length, const uint16_t *q, const float *balance, float scale,
                   float *out, float *probs_hi, float *probs_lo, int32_t flags, void *ws, size_t ws_bytes,
                   const uint16_t *k_new, const uint16_t *v_new, hipStream_t st) {
  int rc = check_attention_args(c, length, q, balance, out, ws, ws_bytes, "mikv_decode_attention_partial");
  if (rc) return rc;
  Plan p = make_plan(c, length);
  AttnArgs A = make_args(c, p, q, balance, scale, out, probs_hi, probs_lo, flags, ws);
  if (k_new) set_append(A, c, length, k_new, v_new, balance);
  // Odd lengths run the grid backwards, so consecutive decode steps read the
  // cache in opposite orders and each starts on what the 256 MB last-level
  // cache kept from the one before.  Wholly backwards with an fp16 importance
  // pool and one query head per KV head; under GQA or with an INT8 pool only
  // the head order flips, which keeps the longest waves at the front
  // (measured per step: long_context 136.4 -> 123.7 us wholly, 132.2 heads
  // only; mistral_7b 89.5 -> 87.0 heads only, 88.3 wholly; llama2_13b 335.7
  // -> 329.2 heads only; llama2_7b, whose cache fits that cache, unchanged).
  if (length & 1) A.order = c->hi_bits == 16 && group_size_of(c) == 1 ? 2 : 1;
  dim3 grid((p.nc_hi + p.nc_lo) * n_heads_of(c));
  const int G = group_size_of(c);
  if (c->key_block) {
    // per-channel retained keys: fp16 importance pool, one query head per
    // KV head, no balancer (validated)
    if (balance) return set_error(MIKV_ERR_INVALID_ARG, "mikv_decode_attention: per-channel keys take no balancer");
    switch (c->lo_bits) {
      case 2: hipLaunchKernelGGL((attn_partial_kernel<16, 2, 1, false, true>), grid, dim3(64), 0, st, A); break;
      case 3: hipLaunchKernelGGL((attn_partial_kernel<16, 3, 1, false, true>), grid, dim3(64), 0, st, A); break;
      default: hipLaunchKernelGGL((attn_partial_kernel<16, 4, 1, false, true>), grid, dim3(64), 0, st, A); break;
    }
    return check_launch("mikv_decode_attention_partial");
  }
  switch (format_key(c)) {
    case 1602: launch_partial_g<16, 2>(A, G, grid, st); break;
    case 1604: launch_partial_g<16, 4>(A, G, grid, st); break;
    case 1608: launch_partial_g<16, 8>(A, G, grid, st); break;
    case 802: launch_partial_g<8, 2>(A, G, grid, st); break;
    case 1603: launch_partial_g<16, 3>(A, G, grid, st); break;
    case 803: launch_partial_g<8, 3>(A, G, grid, st); break;
    case 402: launch_partial_g<4, 2>(A, G, grid, st); break;
    case 804: launch_partial_g<8, 4>(A, G, grid, st); break;
    default: launch_partial_g<8, 8>(A, G, grid, st); break;
  }
  return check_launch("mikv_decode_attention_partial");
}

template <int HI, int LO>
void launch_finalize_select(const AttnArgs &A, const SelArgs &S, int G, dim3 grid, int tiles_hi, int tiles_lo,
                            hipStream_t st) {
  switch (G) {
    case 1: hipLaunchKernelGGL((finalize_select_kernel<1, HI, LO>), grid, dim3(kBlock), 0, st, A, tiles_hi, tiles_lo, S); break;
    case 2: hipLaunchKernelGGL((finalize_select_kernel<2, HI, LO>), grid, dim3(kBlock), 0, st, A, tiles_hi, tiles_lo, S); break;
    case 4: hipLaunchKernelGGL((finalize_select_kernel<4, HI, LO>), grid, dim3(kBlock), 0, st, A, tiles_hi, tiles_lo, S); break;
    default: hipLaunchKernelGGL((finalize_select_kernel<8, HI, LO>), grid, dim3(kBlock), 0, st, A, tiles_hi, tiles_lo, S); break;
  }
}

int decode_finalize_select(const mikv_cache *c, int32_t length, const uint16_t *q, const float *balance, float scale,
                           float *out, float *probs_hi, float *probs_lo, void *ws, size_t ws_bytes, int32_t k_heavy,
                           int32_t window, void *sel_ws, bool appended, hipStream_t st) {
  int rc = check_attention_args(c, length, q, balance, out, ws, ws_bytes, "mikv_decode_step");
  if (rc) return rc;
  Plan p = make_plan(c, length);
  AttnArgs A = make_args(c, p, q, balance, scale, out, probs_hi, probs_lo, MIKV_ATTN_ACCUMULATE, ws);
  A.hi_pending = appended ? 1 : 0;
  const SelArgs S = make_sel_args(c, length, k_heavy, window, sel_ws);
  const int span_hi = std::min(length, c->cap_hi), span_lo = std::min(length, c->cap_lo);
  const int tiles_hi = (span_hi + kProbTile - 1) / kProbTile;  // probabilities accumulated
  const int tiles_lo = A.probs_lo && !evicting(c) ? (span_lo + kProbTile - 1) / kProbTile : 0;
  const int kt = lo_tiles_per_block(group_size_of(c));
  dim3 grid(n_heads_of(c), 2 + (tiles_lo + kt - 1) / kt);  // y = 0: importance pool and re-rank, 1: output
  const int G = group_size_of(c);
  switch (format_key(c)) {
    case 1602: launch_finalize_select<16, 2>(A, S, G, grid, tiles_hi, tiles_lo, st); break;
    case 1604: launch_finalize_select<16, 4>(A, S, G, grid, tiles_hi, tiles_lo, st); break;
    case 1608: launch_finalize_select<16, 8>(A, S, G, grid, tiles_hi, tiles_lo, st); break;
    case 802: launch_finalize_select<8, 2>(A, S, G, grid, tiles_hi, tiles_lo, st); break;
    case 1603: launch_finalize_select<16, 3>(A, S, G, grid, tiles_hi, tiles_lo, st); break;
    case 803: launch_finalize_select<8, 3>(A, S, G, grid, tiles_hi, tiles_lo, st); break;
    case 402: launch_finalize_select<4, 2>(A, S, G, grid, tiles_hi, tiles_lo, st); break;
    case 804: launch_finalize_select<8, 4>(A, S, G, grid, tiles_hi, tiles_lo, st); break;
    default: launch_finalize_select<8, 8>(A, S, G, grid, tiles_hi, tiles_lo, st); break;
  }
  return check_launch("mikv_decode_step (finalize and select)");
}

}  // namespace mikv

extern "C" int mikv_decode_attention_partial(const mikv_cache *c, int32_t length, const uint16_t *q,
                                             const float *balance, float scale, float *out, float *probs_hi,
                                             float *probs_lo, int32_t flags, void *ws, size_t ws_bytes,
                                             void *stream) {
  return decode_partial(c, length, q, balance, scale, out, probs_hi, probs_lo, flags, ws, ws_bytes, nullptr, nullptr,
                        (hipStream_t)stream);
}

namespace mikv {

int decode_finalize(const mikv_cache *c, int32_t length, const uint16_t *q, const float *balance, float scale,
                    float *out, float *probs_hi, float *probs_lo, int32_t flags, void *ws, size_t ws_bytes,
                    bool appended, hipStream_t st) {
  int rc = check_attention_args(c, length, q, balance, out, ws, ws_bytes, "mikv_decode_attention_finalize");
  if (rc) return rc;
  Plan p = make_plan(c, length);
  AttnArgs A = make_args(c, p, q, balance, scale, out, probs_hi, probs_lo, flags, ws);
  A.hi_pending = appended ? 1 : 0;
  const int acc = (flags & MIKV_ATTN_ACCUMULATE) ? 1 : 0;
  // probability tiles: importance pool when its probabilities are emitted or
  // accumulated, retained pool when its probabilities are emitted
  const int span_hi = std::min(length, c->cap_hi), span_lo = std::min(length, c->cap_lo);
  const int tiles_hi = (A.scores_hi && (A.probs_hi || A.acc)) ? (span_hi + kProbTile - 1) / kProbTile : 0;
  const int tiles_lo = A.probs_lo && !evicting(c) ? (span_lo + kProbTile - 1) / kProbTile : 0;
  dim3 grid(n_heads_of(c), 1 + tiles_hi + tiles_lo);  // y = 0: output
  switch (group_size_of(c)) {
    case 1: hipLaunchKernelGGL(attn_finalize_kernel<1>, grid, dim3(kBlock), 0, st, A, acc, tiles_hi, tiles_lo); break;
    case 2: hipLaunchKernelGGL(attn_finalize_kernel<2>, grid, dim3(kBlock), 0, st, A, acc, tiles_hi, tiles_lo); break;
    case 4: hipLaunchKernelGGL(attn_finalize_kernel<4>, grid, dim3(kBlock), 0, st, A, acc, tiles_hi, tiles_lo); break;
    default: hipLaunchKernelGGL(attn_finalize_kernel<8>, grid, dim3(kBlock), 0, st, A, acc, tiles_hi, tiles_lo); break;
  }
  return check_launch("mikv_decode_attention_finalize");
}

}  // namespace mikv

extern "C" int mikv_decode_attention_finalize(const mikv_cache *c, int32_t length, const uint16_t *q,
                                              const float *balance, float scale, float *out, float *probs_hi,
                                              float *probs_lo, int32_t flags, void *ws, size_t ws_bytes,
                                              void *stream) {
  return decode_finalize(c, length, q, balance, scale, out, probs_hi, probs_lo, flags, ws, ws_bytes, false,
                         (hipStream_t)stream);
}

extern "C" int mikv_decode_attention(const mikv_cache *c, int32_t length, const uint16_t *q, const float *balance,
                                     float scale, float *out, float *probs_hi, float *probs_lo, int32_t flags,
                                     void *ws, size_t ws_bytes, void *stream) {
  int rc = mikv_decode_attention_partial(c, length, q, balance, scale, out, probs_hi, probs_lo, flags, ws,
                                         ws_bytes, stream);
  if (rc) return rc;
  return mikv_decode_attention_finalize(c, length, q, balance, scale, out, probs_hi, probs_lo, flags, ws,
                                        ws_bytes, stream);
}

extern "C" int mikv_importance_update(const mikv_cache *c, int32_t length, const float *probs_hi, void *stream) {
  int rc = validate_cache(c);
  if (rc) return rc;
  if (!probs_hi) return set_error(MIKV_ERR_INVALID_ARG, "mikv_importance_update: probs_hi is NULL");
  if (length < 1 || length > c->max_len)
    return set_error(length < 1 ? MIKV_ERR_INVALID_ARG : MIKV_ERR_CAPACITY,
                     "mikv_importance_update: length %d outside [1, max_len]", length);
  const int span = std::min(length, c->cap_hi);
  dim3 grid((span + kBlock - 1) / kBlock, n_heads_of(c));
  hipStream_t st = (hipStream_t)stream;
  switch (group_size_of(c)) {
    case 1:
      hipLaunchKernelGGL(importance_kernel<1>, grid, dim3(kBlock), 0, st, c->hi_acc, probs_hi, c->n_hi, c->cap_hi,
                         c->q_heads, c->kv_heads);
      break;
    case 2:
      hipLaunchKernelGGL(importance_kernel<2>, grid, dim3(kBlock), 0, st, c->hi_acc, probs_hi, c->n_hi, c->cap_hi,
                         c->q_heads, c->kv_heads);
      break;
    case 4:
      hipLaunchKernelGGL(importance_kernel<4>, grid, dim3(kBlock), 0, st, c->hi_acc, probs_hi, c->n_hi, c->cap_hi,
                         c->q_heads, c->kv_heads);
      break;
    default:
      hipLaunchKernelGGL(importance_kernel<8>, grid, dim3(kBlock), 0, st, c->hi_acc, probs_hi, c->n_hi, c->cap_hi,
                         c->q_heads, c->kv_heads);
  }
  return check_launch("mikv_importance_update");
}

extern "C" size_t mikv_resident_bytes(void) { return (size_t)mikv::resident_budget(); }

extern "C" int mikv_set_resident_bytes(size_t bytes) {
  if (bytes > ((size_t)1 << 62)) return mikv::set_error(MIKV_ERR_INVALID_ARG, "mikv_set_resident_bytes: %zu bytes is out of range", bytes);
  mikv::g_resident_bytes.store((int64_t)bytes, std::memory_order_relaxed);
  return MIKV_OK;
}
