// Decode-step attention over the mixed-precision cache (Section 3.4, Fig. 3
// left) and the importance update (the H2O accumulated-attention score).
//
// Split-K over the sequence: every block takes one contiguous chunk of one
// pool of one (sequence, KV head) -- chunks are homogeneous in precision
// (the pools are grouped by precision, which permutation invariance allows)
// and sized by bytes, so the fp16/INT8 and INT2/INT4 chunks cost about the
// same.  A block serves all G query heads of the KV group, so GQA loads K/V
// once.  Lanes: LPT lanes per token, each owning CPL = 128/LPT contiguous
// channels; a wave covers 64/LPT tokens per iteration with fully coalesced
// loads of the packed rows.  Each lane keeps its own value sums, the running
// maximum is wave-uniform (tile maxima via lane shuffles), and the lanes and
// waves are merged once per chunk.  The partial phase writes per-chunk
// (max, sum, value-sum) records and the raw scores; the finalize phase merges
// the records exactly, turns scores into probabilities and, optionally, adds
// them to the importance scores.
#include "mikv_internal.h"

namespace mikv {

namespace {

constexpr int kBlock = 256;
constexpr int kWaves = kBlock / 64;
constexpr int kRec = 2 + kHeadDim;  // (max, sum, value-sum[128]) per query head and chunk
constexpr float kNegInf = -__builtin_huge_valf();

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
  float *scores_hi, *scores_lo;  // [B*Hq, cap] raw scores (nullable)
  float *partials;               // [B*Hq, nc_hi + nc_lo, kRec]
  float *probs_hi, *probs_lo;    // outputs (nullable)
  float *acc;                    // hi_acc when accumulating (nullable)
  float *out;                    // [B*Hq, 128]
  int cap_hi, cap_lo, group, q_heads, kv_heads;
  int chunk_hi, chunk_lo, nc_hi, nc_lo;
};

// Channels per lane for a GQA group of G query heads (keeps q and the value
// sums of all G heads in registers: G * CPL <= 32).
template <int G>
struct LaneShape {
  static constexpr int CPL = G == 1 ? 32 : (G == 2 ? 16 : (G == 4 ? 8 : 4));
  static constexpr int LPT = kHeadDim / CPL;
  static constexpr int TPW = 64 / LPT;  // tokens per wave iteration
};

// Raw storage of CPL channels of one token at BITS (16 = fp16).
template <int BITS, int CPL>
struct Seg {
  static constexpr int kBytes = BITS == 16 ? CPL * 2 : CPL * BITS / 8;
  static constexpr int kWords = kBytes >= 4 ? kBytes / 4 : 1;
  uint32_t w[kWords];
  uint32_t param;
};

template <int BITS, int CPL>
__device__ inline void load_seg(Seg<BITS, CPL> &s, const uint8_t *rowbase, const uint32_t *parbase,
                                int part, int group) {
  constexpr int B = Seg<BITS, CPL>::kBytes;
  const uint8_t *p = rowbase + part * B;
  if constexpr (B >= 16) {
#pragma unroll
    for (int i = 0; i < B / 16; ++i) {
      uint4 v = reinterpret_cast<const uint4 *>(p)[i];
      s.w[4 * i] = v.x;
      s.w[4 * i + 1] = v.y;
      s.w[4 * i + 2] = v.z;
      s.w[4 * i + 3] = v.w;
    }
  } else if constexpr (B == 8) {
    uint2 v = *reinterpret_cast<const uint2 *>(p);
    s.w[0] = v.x;
    s.w[1] = v.y;
  } else if constexpr (B == 4) {
    s.w[0] = *reinterpret_cast<const uint32_t *>(p);
  } else if constexpr (B == 2) {
    s.w[0] = *reinterpret_cast<const uint16_t *>(p);
  } else {
    s.w[0] = *p;
  }
  if constexpr (BITS != 16) s.param = parbase[(part * CPL) / group];
}

// Decoded fp32 value of channel c of the segment: the fp16 value, or
// alpha * code + beta (the product is exact, so fmaf rounds exactly once,
// like the separate multiply and add of Eq. 1).
template <int BITS, int CPL>
__device__ inline float seg_value(const Seg<BITS, CPL> &s, int c, float a, float b) {
  if constexpr (BITS == 16) {
    return f16_to_f32((uint16_t)(s.w[c >> 1] >> (16 * (c & 1))));
  } else {
    uint32_t code = (s.w[(c * BITS) / 32] >> ((c * BITS) % 32)) & ((1u << BITS) - 1u);
    return fmaf(a, (float)code, b);
  }
}

template <int BITS>
__device__ inline void seg_params(uint32_t param, float &a, float &b) {
  if constexpr (BITS == 16) {
    a = 1.0f;
    b = 0.0f;
  } else {
    a = f16_to_f32((uint16_t)(param & 0xffffu));
    b = f16_to_f32((uint16_t)(param >> 16));
  }
}

template <int BITS, int G>
__device__ void attn_chunk(const AttnArgs &A, int h, int chunk, int rec_chunk, bool is_hi) {
  using S = LaneShape<G>;
  constexpr int CPL = S::CPL, LPT = S::LPT, TPW = S::TPW;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int part = lane % LPT, tsub = lane / LPT;
  const int b = h / A.kv_heads, kvh = h % A.kv_heads;
  const int qh0 = b * A.q_heads + kvh * G;  // first query head of the group

  const int cap = is_hi ? A.cap_hi : A.cap_lo;
  const int chunk_len = is_hi ? A.chunk_hi : A.chunk_lo;
  const int n_pool = is_hi ? A.n_hi[h] : A.n_lo[h];
  const int start = chunk * chunk_len;
  const int end = min(start + chunk_len, n_pool);
  const int64_t row_bytes = BITS == 16 ? kHeadDim * 2 : kHeadDim * BITS / 8;
  const int ng = kHeadDim / A.group;
  const uint8_t *kbase = (is_hi ? A.hi_k : A.lo_k) + (int64_t)h * cap * row_bytes;
  const uint8_t *vbase = (is_hi ? A.hi_v : A.lo_v) + (int64_t)h * cap * row_bytes;
  const uint32_t *kpbase = (is_hi ? A.hi_kp : A.lo_kp) + (int64_t)h * cap * ng;
  const uint32_t *vpbase = (is_hi ? A.hi_vp : A.lo_vp) + (int64_t)h * cap * ng;
  float *scores = is_hi ? A.scores_hi : A.scores_lo;

  // q_hat = q / balance (Eq. 4), this lane's channels, all G heads.
  float qr[G][CPL];
#pragma unroll
  for (int i = 0; i < G; ++i) {
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      int ch = part * CPL + c;
      float qv = f16_to_f32(A.q[(int64_t)(qh0 + i) * kHeadDim + ch]);
      if (A.balance) qv = qv / A.balance[(int64_t)h * kHeadDim + ch];
      qr[i][c] = qv;
    }
  }

  float m[G], l[G], o[G][CPL];
#pragma unroll
  for (int i = 0; i < G; ++i) {
    m[i] = kNegInf;
    l[i] = 0.0f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) o[i][c] = 0.0f;
  }

  for (int base = start; base < end; base += kWaves * TPW) {
    const int tok = base + wave * TPW + tsub;
    const bool valid = tok < end;
    const int slot = valid ? tok : start;  // invalid lanes re-read a valid row
    Seg<BITS, CPL> ks, vs;
    load_seg<BITS, CPL>(ks, kbase + (int64_t)slot * row_bytes, kpbase + (int64_t)slot * ng, part, A.group);
    load_seg<BITS, CPL>(vs, vbase + (int64_t)slot * row_bytes, vpbase + (int64_t)slot * ng, part, A.group);
    float ka, kb, va, vb;
    seg_params<BITS>(ks.param, ka, kb);
    seg_params<BITS>(vs.param, va, vb);

    float s[G];
#pragma unroll
    for (int i = 0; i < G; ++i) s[i] = 0.0f;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      float kv = seg_value<BITS, CPL>(ks, c, ka, kb);
#pragma unroll
      for (int i = 0; i < G; ++i) s[i] = fmaf(qr[i][c], kv, s[i]);
    }
#pragma unroll
    for (int i = 0; i < G; ++i) {
      s[i] = sum_lanes<LPT>(s[i]) * A.scale;
      if (!valid) s[i] = kNegInf;
      if (scores && valid && part == 0) scores[(int64_t)(qh0 + i) * cap + tok] = s[i];
      float tmax = wave_max(s[i]);
      if (tmax > m[i]) {
        float f = m[i] == kNegInf ? 0.0f : __expf(m[i] - tmax);
        l[i] *= f;
#pragma unroll
        for (int c = 0; c < CPL; ++c) o[i][c] *= f;
        m[i] = tmax;
      }
      s[i] = valid ? __expf(s[i] - m[i]) : 0.0f;
      if (part == 0) l[i] += s[i];
    }
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
      float vv = seg_value<BITS, CPL>(vs, c, va, vb);
#pragma unroll
      for (int i = 0; i < G; ++i) o[i][c] = fmaf(s[i], vv, o[i][c]);
    }
  }

  // merge lanes of equal `part` (same channels), then waves through LDS
#pragma unroll
  for (int i = 0; i < G; ++i) {
    l[i] = wave_sum(l[i]);
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
#pragma unroll
      for (int off = LPT; off < 64; off <<= 1) o[i][c] += __shfl_xor(o[i][c], off, 64);
    }
  }
  __shared__ float s_m[kWaves][G], s_l[kWaves][G];
  __shared__ float s_o[kWaves][G][kHeadDim];
  if (lane == 0) {
#pragma unroll
    for (int i = 0; i < G; ++i) {
      s_m[wave][i] = m[i];
      s_l[wave][i] = l[i];
    }
  }
  if (tsub == 0) {
#pragma unroll
    for (int i = 0; i < G; ++i)
#pragma unroll
      for (int c = 0; c < CPL; ++c) s_o[wave][i][part * CPL + c] = o[i][c];
  }
  __syncthreads();
  const int nc = A.nc_hi + A.nc_lo;
  for (int idx = threadIdx.x; idx < G * kRec; idx += kBlock) {
    const int i = idx / kRec, e = idx % kRec;
    float M = kNegInf;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, s_m[w][i]);
    float val = 0.0f;
    if (e == 0) {
      val = M;
    } else {
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        float f = s_m[w][i] == kNegInf ? 0.0f : __expf(s_m[w][i] - M);
        val += f * (e == 1 ? s_l[w][i] : s_o[w][i][e - 2]);
      }
    }
    A.partials[((int64_t)(qh0 + i) * nc + rec_chunk) * kRec + e] = val;
  }
}

template <int HI, int LO, int G>
__global__ __launch_bounds__(kBlock) void attn_partial_kernel(AttnArgs A) {
  const int h = blockIdx.y, c = blockIdx.x;
  if (c < A.nc_hi)
    attn_chunk<HI, G>(A, h, c, c, true);
  else
    attn_chunk<LO, G>(A, h, c - A.nc_hi, c, false);
}

// Merge the chunk records of every query head of KV head h; turn this
// block's chunk of raw scores into probabilities (and optionally add them to
// the importance scores); block 0 of each head also writes the output.
template <int G>
__global__ __launch_bounds__(kBlock) void attn_finalize_kernel(AttnArgs A, int accumulate) {
  const int h = blockIdx.y, c = blockIdx.x;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int b = h / A.kv_heads, kvh = h % A.kv_heads;
  const int qh0 = b * A.q_heads + kvh * G;
  const int nc = A.nc_hi + A.nc_lo;
  __shared__ float s_M[G], s_L[G];
  for (int i = wave; i < G; i += kWaves) {
    const float *rec = A.partials + (int64_t)(qh0 + i) * nc * kRec;
    float M = kNegInf;
    for (int r = lane; r < nc; r += 64) M = fmaxf(M, rec[(int64_t)r * kRec]);
    M = wave_max(M);
    float L = 0.0f;
    for (int r = lane; r < nc; r += 64) {
      float mr = rec[(int64_t)r * kRec];
      if (mr != kNegInf) L += rec[(int64_t)r * kRec + 1] * __expf(mr - M);
    }
    L = wave_sum(L);
    if (lane == 0) {
      s_M[i] = M;
      s_L[i] = L;
    }
  }
  __syncthreads();

  const bool is_hi = c < A.nc_hi;
  const int chunk = is_hi ? c : c - A.nc_hi;
  const int chunk_len = is_hi ? A.chunk_hi : A.chunk_lo;
  const int n_pool = is_hi ? A.n_hi[h] : A.n_lo[h];
  const int cap = is_hi ? A.cap_hi : A.cap_lo;
  const float *scores = is_hi ? A.scores_hi : A.scores_lo;
  float *probs = is_hi ? A.probs_hi : A.probs_lo;
  const bool acc = is_hi && accumulate && A.acc;
  if (scores && (probs || acc)) {
    const int start = chunk * chunk_len, end = min(start + chunk_len, n_pool);
    for (int t = start + threadIdx.x; t < end; t += kBlock) {
      float sum = 0.0f;
#pragma unroll
      for (int i = 0; i < G; ++i) {
        float p = __expf(scores[(int64_t)(qh0 + i) * cap + t] - s_M[i]) / s_L[i];
        if (probs) probs[(int64_t)(qh0 + i) * cap + t] = p;
        sum = i == 0 ? p : sum + p;
      }
      if (acc) A.acc[(int64_t)h * A.cap_hi + t] += sum;
    }
  }
  if (c == 0) {
    for (int idx = threadIdx.x; idx < G * kHeadDim; idx += kBlock) {
      const int i = idx / kHeadDim, d = idx % kHeadDim;
      const float *rec = A.partials + (int64_t)(qh0 + i) * nc * kRec;
      float v = 0.0f;
      for (int r = 0; r < nc; ++r) {
        float mr = rec[(int64_t)r * kRec];
        if (mr != kNegInf) v += rec[(int64_t)r * kRec + 2 + d] * __expf(mr - s_M[i]);
      }
      A.out[(int64_t)(qh0 + i) * kHeadDim + d] = v / s_L[i];
    }
  }
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
};

int round_up(int64_t x, int m) { return (int)(((x + m - 1) / m) * m); }

Plan make_plan(const mikv_cache *c, int length) {
  Plan p;
  const int64_t NH = n_heads_of(c);
  const int span_hi = std::min(length, c->cap_hi), span_lo = std::min(length, c->cap_lo);
  const int64_t bh = token_bytes(c->hi_bits, c->group), bl = token_bytes(c->lo_bits, c->group);
  const int64_t total = NH * (span_hi * bh + span_lo * bl);
  // Aim for ~8 blocks per CU over 256 CUs, at least 32 KiB and at most
  // 512 KiB of packed K/V per block.
  int64_t target = std::min<int64_t>(std::max<int64_t>(total / 2048, 32 << 10), 512 << 10);
  p.chunk_hi = std::max(64, round_up(target / bh, 64));
  p.chunk_lo = std::max(64, round_up(target / bl, 64));
  p.nc_hi = std::max(1, (span_hi + p.chunk_hi - 1) / p.chunk_hi);
  p.nc_lo = std::max(1, (span_lo + p.chunk_lo - 1) / p.chunk_lo);
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
  return A;
}

template <int HI, int LO>
void launch_partial_g(const AttnArgs &A, int G, dim3 grid, hipStream_t st) {
  switch (G) {
    case 1: hipLaunchKernelGGL((attn_partial_kernel<HI, LO, 1>), grid, dim3(kBlock), 0, st, A); break;
    case 2: hipLaunchKernelGGL((attn_partial_kernel<HI, LO, 2>), grid, dim3(kBlock), 0, st, A); break;
    case 4: hipLaunchKernelGGL((attn_partial_kernel<HI, LO, 4>), grid, dim3(kBlock), 0, st, A); break;
    default: hipLaunchKernelGGL((attn_partial_kernel<HI, LO, 8>), grid, dim3(kBlock), 0, st, A); break;
  }
}

int check_attention_args(const mikv_cache *c, int32_t length, const uint16_t *q, float *out, void *ws,
                         size_t ws_bytes, const char *who) {
  int rc = validate_cache(c);
  if (rc) return rc;
  if (!q || !out) return set_error(MIKV_ERR_INVALID_ARG, "%s: q/out is NULL", who);
  if (length < 1) return set_error(MIKV_ERR_INVALID_ARG, "%s: length must be >= 1", who);
  if (length > c->max_len) return set_error(MIKV_ERR_CAPACITY, "%s: length %d > max_len %d", who, length, c->max_len);
  Plan p = make_plan(c, length);
  size_t need = workspace_bytes_for(c, p);
  if (!ws || ws_bytes < need) return set_error(MIKV_ERR_CAPACITY, "%s: workspace too small (%zu < %zu)", who, ws_bytes, need);
  return MIKV_OK;
}

}  // namespace

}  // namespace mikv

using namespace mikv;

extern "C" size_t mikv_decode_workspace_size(const mikv_cache *c, int32_t length) {
  if (!c || length < 1 || validate_cache(c)) return 0;
  return workspace_bytes_for(c, make_plan(c, length));
}

extern "C" int mikv_decode_attention_partial(const mikv_cache *c, int32_t length, const uint16_t *q,
                                             const float *balance, float scale, float *out, float *probs_hi,
                                             float *probs_lo, int32_t flags, void *ws, size_t ws_bytes,
                                             void *stream) {
  int rc = check_attention_args(c, length, q, out, ws, ws_bytes, "mikv_decode_attention_partial");
  if (rc) return rc;
  Plan p = make_plan(c, length);
  AttnArgs A = make_args(c, p, q, balance, scale, out, probs_hi, probs_lo, flags, ws);
  dim3 grid(p.nc_hi + p.nc_lo, n_heads_of(c));
  hipStream_t st = (hipStream_t)stream;
  const int G = group_size_of(c);
  switch (c->hi_bits * 100 + c->lo_bits) {
    case 1602: launch_partial_g<16, 2>(A, G, grid, st); break;
    case 1604: launch_partial_g<16, 4>(A, G, grid, st); break;
    case 1608: launch_partial_g<16, 8>(A, G, grid, st); break;
    case 802: launch_partial_g<8, 2>(A, G, grid, st); break;
    case 804: launch_partial_g<8, 4>(A, G, grid, st); break;
    default: launch_partial_g<8, 8>(A, G, grid, st); break;
  }
  return check_launch("mikv_decode_attention_partial");
}

extern "C" int mikv_decode_attention_finalize(const mikv_cache *c, int32_t length, const uint16_t *q,
                                              const float *balance, float scale, float *out, float *probs_hi,
                                              float *probs_lo, int32_t flags, void *ws, size_t ws_bytes,
                                              void *stream) {
  int rc = check_attention_args(c, length, q, out, ws, ws_bytes, "mikv_decode_attention_finalize");
  if (rc) return rc;
  Plan p = make_plan(c, length);
  AttnArgs A = make_args(c, p, q, balance, scale, out, probs_hi, probs_lo, flags, ws);
  dim3 grid(p.nc_hi + p.nc_lo, n_heads_of(c));
  hipStream_t st = (hipStream_t)stream;
  const int acc = (flags & MIKV_ATTN_ACCUMULATE) ? 1 : 0;
  switch (group_size_of(c)) {
    case 1: hipLaunchKernelGGL(attn_finalize_kernel<1>, grid, dim3(kBlock), 0, st, A, acc); break;
    case 2: hipLaunchKernelGGL(attn_finalize_kernel<2>, grid, dim3(kBlock), 0, st, A, acc); break;
    case 4: hipLaunchKernelGGL(attn_finalize_kernel<4>, grid, dim3(kBlock), 0, st, A, acc); break;
    default: hipLaunchKernelGGL(attn_finalize_kernel<8>, grid, dim3(kBlock), 0, st, A, acc); break;
  }
  return check_launch("mikv_decode_attention_finalize");
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
