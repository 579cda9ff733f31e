// Eq. 1 quantizer (Section 3.1) with the Eq. 3 key balancer (Section 3.2):
// raw row quantization and placement of new tokens into the two pools.
//
// Work layout: every lane owns 32 contiguous channels of one row (a key or
// value vector of one token), i.e. 4 lanes per row and 16 rows per wave.  A
// quantization group of g channels spans g/32 adjacent lanes, which combine
// their min/max with lane shuffles.  Loads are 4 x 16 B per lane, contiguous
// across the lanes of a row (coalesced); codes are written as whole dwords.
#include "append_device.h"
#include "mikv_internal.h"

namespace mikv {

namespace {

constexpr int kChunk = 256;  // tokens per block in the placement kernels

template <int BITS>
__global__ __launch_bounds__(256) void quantize_rows_kernel(const uint16_t *x, int64_t rows,
                                                            const float *balance, int rows_per_balance,
                                                            int group, uint8_t *codes, uint16_t *params) {
  int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  int64_t row = t >> 2;
  int lane4 = (int)(t & 3);
  bool live = row < rows;
  int64_t r = live ? row : rows - 1;  // dead lanes shadow the last row (no stores)
  float xs[32];
  const float *bal = balance ? balance + (r / rows_per_balance) * kHeadDim + lane4 * 32 : nullptr;
  load_row_segment(x + r * kHeadDim + lane4 * 32, bal, xs);
  int ng = kHeadDim / group;
  uint32_t *prow = reinterpret_cast<uint32_t *>(params) + r * ng + (lane4 * 32) / group;
  quantize_segment<BITS>(xs, group, lane4, codes + r * (kHeadDim * BITS / 8) + lane4 * (32 * BITS / 8),
                         prow, live);
}

// Device view of the cache for the placement kernels.
struct Pools {
  uint8_t *hi_k, *hi_v;      // fp16 rows, or INT8/INT4 codes
  uint32_t *hi_kp, *hi_vp;   // (alpha, beta) pairs
  int32_t *hi_pos;
  float *hi_acc;
  int32_t *n_hi;
  uint8_t *lo_k, *lo_v;
  uint32_t *lo_kp, *lo_vp;
  int32_t *lo_pos, *n_lo;
  uint8_t *map;
  int32_t *status;
  int cap_hi, cap_lo, max_len, group;
  int v_tiled;  // 2-bit values in the tiled layout (int2_values_tiled)
  int evict;    // no retained pool: tokens not placed in the importance pool are dropped
  // per-channel keys: (alpha, beta) words [NH, n_kblk, 128] per key block
  const uint32_t *lo_kb;
  int n_kblk;
};

Pools make_pools(const mikv_cache *c) {
  Pools p;
  p.hi_k = (uint8_t *)c->hi_k;
  p.hi_v = (uint8_t *)c->hi_v;
  p.hi_kp = (uint32_t *)c->hi_kp;
  p.hi_vp = (uint32_t *)c->hi_vp;
  p.hi_pos = c->hi_pos;
  p.hi_acc = c->hi_acc;
  p.n_hi = c->n_hi;
  p.lo_k = c->lo_k;
  p.lo_v = c->lo_v;
  p.lo_kp = (uint32_t *)c->lo_kp;
  p.lo_vp = (uint32_t *)c->lo_vp;
  p.lo_pos = c->lo_pos;
  p.n_lo = c->n_lo;
  p.map = c->map;
  p.status = c->status;
  p.cap_hi = c->cap_hi;
  p.cap_lo = c->cap_lo;
  p.max_len = c->max_len;
  p.group = c->group;
  p.v_tiled = int2_values_tiled(c->lo_bits, c->q_heads, c->kv_heads) ? 1 : 0;
  p.evict = evicting(c) ? 1 : 0;
  p.lo_kb = c->key_block ? (const uint32_t *)c->lo_kb : nullptr;
  p.n_kblk = c->key_block ? key_blocks_of(c) : 0;
  return p;
}

// Per-channel key quantization (Appendix C): Eq. 1 over the 64 keys of a
// block, channel by channel.  Thread t takes channel t % 128 of half the
// block's rows (t / 128); the halves combine in LDS.  `row_of(i)` gives the
// fp16 row of the block's i-th position, or NULL when that key is missing
// (then nothing is written and the status bit is set).
template <class RowOf>
__device__ inline void block_params(RowOf row_of, uint32_t *dst, int bits, int32_t *status) {
  __shared__ float s_mn[kHeadDim], s_mx[kHeadDim];
  __shared__ int s_missing;
  const int c = threadIdx.x & (kHeadDim - 1), half = threadIdx.x >> 7;
  if (threadIdx.x == 0) s_missing = 0;
  __syncthreads();
  float mn = __builtin_huge_valf(), mx = -__builtin_huge_valf();
  for (int i = half * (kKeyBlock / 2); i < (half + 1) * (kKeyBlock / 2); ++i) {
    const uint16_t *r = row_of(i);
    if (!r) {
      s_missing = 1;
      continue;
    }
    const float x = f16_to_f32(r[c]);
    mn = fminf(mn, x);
    mx = fmaxf(mx, x);
  }
  if (half == 1) {
    s_mn[c] = mn;
    s_mx[c] = mx;
  }
  __syncthreads();
  if (half == 0) {
    if (s_missing) {
      if (c == 0) atomicOr(status, MIKV_DEVERR_KEY_BLOCK);
      return;
    }
    const GroupParams p = group_params(fminf(mn, s_mn[c]), fmaxf(mx, s_mx[c]), bits);
    dst[c] = (uint32_t)p.a16 | ((uint32_t)p.b16 << 16);
  }
}

// Blocks whose 64 positions all lie in the rows being placed: block
// blockIdx.x of the range, head blockIdx.y; k is fp16 [NH, n, 128] for
// positions pos0 .. pos0 + n - 1.
__global__ __launch_bounds__(256) void key_block_rows_kernel(Pools P, const uint16_t *k, int pos0, int n, int blk0,
                                                             int bits) {
  const int h = blockIdx.y, blk = blk0 + blockIdx.x;
  const int64_t first = (int64_t)blk * kKeyBlock - pos0;  // row of the block's first position
  auto row_of = [&](int i) -> const uint16_t * { return k + ((int64_t)h * n + first + i) * kHeadDim; };
  block_params(row_of, const_cast<uint32_t *>(P.lo_kb) + ((int64_t)h * P.n_kblk + blk) * kHeadDim, bits, P.status);
}

// A block completed during decoding: its keys are in the importance pool
// (every position of it is in the recent window), found by position.
__global__ __launch_bounds__(256) void key_block_pool_kernel(Pools P, int blk, int bits) {
  const int h = blockIdx.x;
  __shared__ int s_slot[kKeyBlock];
  if (threadIdx.x < kKeyBlock) s_slot[threadIdx.x] = -1;
  __syncthreads();
  const int n = min(P.n_hi[h], P.cap_hi);
  const int p0 = blk * kKeyBlock;
  const int32_t *pos = P.hi_pos + (int64_t)h * P.cap_hi;
  for (int i = threadIdx.x; i < n; i += 256) {
    const int p = pos[i];
    if (p >= p0 && p < p0 + kKeyBlock) s_slot[p - p0] = i;
  }
  __syncthreads();
  const uint16_t *hk = reinterpret_cast<const uint16_t *>(P.hi_k) + (int64_t)h * P.cap_hi * kHeadDim;
  auto row_of = [&](int i) -> const uint16_t * {
    const int sl = s_slot[i];
    return sl < 0 ? nullptr : hk + (int64_t)sl * kHeadDim;
  };
  block_params(row_of, const_cast<uint32_t *>(P.lo_kb) + ((int64_t)h * P.n_kblk + blk) * kHeadDim, bits, P.status);
}


__host__ __device__ inline AppendArgs append_args(const Pools &P, const uint16_t *k, const uint16_t *v,
                                                  const float *balance, int pos, const float *score_init) {
  AppendArgs a;
  a.hi_k = P.hi_k;
  a.hi_v = P.hi_v;
  a.hi_kp = P.hi_kp;
  a.hi_vp = P.hi_vp;
  a.hi_pos = P.hi_pos;
  a.hi_acc = P.hi_acc;
  a.map = P.map;
  a.status = P.status;
  a.k = k;
  a.v = v;
  a.balance = balance;
  a.score_init = score_init;
  a.cap_hi = P.cap_hi;
  a.max_len = P.max_len;
  a.group = P.group;
  a.pos = pos;
  return a;
}

// Count importance tokens per chunk of kChunk tokens: counts[h, chunk].
__global__ __launch_bounds__(kChunk) void count_hi_kernel(const uint8_t *hi_mask, int n, int nchunks,
                                                          int32_t *counts) {
  int h = blockIdx.y, chunk = blockIdx.x;
  int j = chunk * kChunk + threadIdx.x;
  int v = (j < n && hi_mask[(int64_t)h * n + j]) ? 1 : 0;
  __shared__ int s[kChunk / 64];
  int w = __popcll(__ballot(v));
  if ((threadIdx.x & 63) == 0) s[threadIdx.x >> 6] = w;
  __syncthreads();
  if (threadIdx.x == 0) {
    int t = 0;
    for (int i = 0; i < kChunk / 64; ++i) t += s[i];
    counts[h * nchunks + chunk] = t;
  }
}

// Place tokens [chunk*kChunk, ...) of head blockIdx.y.  With `counts`
// (mask given) slots come from the per-chunk counts and an in-block scan;
// without, every token goes to the importance pool in order.  When `commit`
// is set (a single chunk per head), the block also advances n_hi/n_lo.
template <int HI_BITS, int LO_BITS>
__global__ __launch_bounds__(256) void place_kernel(Pools P, const uint16_t *k, const uint16_t *v,
                                                    const float *balance, int pos0, int n,
                                                    const uint8_t *hi_mask, const float *score_init,
                                                    const int32_t *counts, int nchunks, int commit) {
  const int h = blockIdx.y, chunk = blockIdx.x, tid = threadIdx.x;
  __shared__ int s_slot[kChunk];
  __shared__ uint8_t s_hi[kChunk];
  __shared__ int s_wave[kChunk / 64][2];
  __shared__ int s_base[2];
  __shared__ int s_total[2];
  const int j0 = chunk * kChunk;
  const int cnt = min(kChunk, n - j0);
  const int n_hi0 = P.n_hi[h], n_lo0 = P.n_lo[h];

  // --- slot assignment -------------------------------------------------
  int j = j0 + tid;
  int is_hi = 1;
  if (hi_mask) is_hi = (tid < cnt && hi_mask[(int64_t)h * n + j]) ? 1 : 0;
  int live = tid < cnt;
  unsigned long long bh = __ballot(live && is_hi);
  unsigned long long bl = __ballot(live && !is_hi);
  unsigned long long below = (1ull << (tid & 63)) - 1ull;
  int r_hi = __popcll(bh & below), r_lo = __popcll(bl & below);
  if ((tid & 63) == 0) {
    s_wave[tid >> 6][0] = __popcll(bh);
    s_wave[tid >> 6][1] = __popcll(bl);
  }
  if (tid == 0) {
    int bhi = 0, blo = 0;
    if (counts) {
      for (int c = 0; c < chunk; ++c) {
        int ch = counts[h * nchunks + c];
        bhi += ch;
        blo += kChunk - ch;
      }
    } else {
      bhi = j0;
    }
    s_base[0] = n_hi0 + bhi;
    s_base[1] = n_lo0 + blo;
  }
  __syncthreads();
  if (tid == 0) {
    int th = 0, tl = 0;
    for (int w = 0; w < kChunk / 64; ++w) {
      th += s_wave[w][0];
      tl += s_wave[w][1];
    }
    s_total[0] = th;
    s_total[1] = tl;
  }
  for (int w = 0; w < (tid >> 6); ++w) {
    r_hi += s_wave[w][0];
    r_lo += s_wave[w][1];
  }
  if (live) {
    int slot = is_hi ? s_base[0] + r_hi : s_base[1] + r_lo;
    int cap = is_hi ? P.cap_hi : P.cap_lo;
    if (!is_hi && P.evict) {
      slot = -1;  // evicted: stored nowhere (the map says "not in the importance pool")
    } else if (!is_hi && P.lo_kb &&
               ((pos0 + j) / kKeyBlock * kKeyBlock < pos0 || (pos0 + j) / kKeyBlock * kKeyBlock + kKeyBlock > pos0 + n)) {
      // a retained key needs its block's parameters: the block must lie
      // within the placed positions
      atomicOr(P.status, MIKV_DEVERR_KEY_BLOCK);
      slot = -1;
    } else if (slot >= cap) {
      atomicOr(P.status, is_hi ? MIKV_DEVERR_HI_FULL : MIKV_DEVERR_LO_FULL);
      slot = -1;
    }
    s_slot[tid] = slot;
    s_hi[tid] = (uint8_t)is_hi;
    int pos = pos0 + j;
    if (slot >= 0) {
      if (is_hi) {
        P.hi_pos[(int64_t)h * P.cap_hi + slot] = pos;
        P.hi_acc[(int64_t)h * P.cap_hi + slot] = score_init ? score_init[(int64_t)h * n + j] : 0.0f;
      } else {
        P.lo_pos[(int64_t)h * P.cap_lo + slot] = pos;
      }
      if (P.map) P.map[(int64_t)h * P.max_len + pos] = (uint8_t)is_hi;
    } else if (!is_hi && P.evict && P.map) {
      P.map[(int64_t)h * P.max_len + pos] = 0;
    }
  }
  __syncthreads();

  // --- quantize / store rows: 4 lanes per row, rows = (token, K|V) ------
  const int lane4 = tid & 3;
  const int ng = kHeadDim / P.group;
  for (int r = tid >> 2; r < 2 * cnt; r += 256 / 4) {
    const int t = r >> 1, is_v = r & 1;
    const int slot = s_slot[t];
    const int hi = s_hi[t];
    const int64_t src_row = (int64_t)h * n + j0 + t;
    const uint16_t *src = (is_v ? v : k) + src_row * kHeadDim + lane4 * 32;
    const float *bal = (!is_v && balance) ? balance + (int64_t)h * kHeadDim + lane4 * 32 : nullptr;
    float x[32];
    load_row_segment(src, bal, x);
    // every lane of a group must take part in the shuffles: no early exit
    const bool store = slot >= 0;
    const int sl = store ? slot : 0;
    if (hi) {
      if (HI_BITS == 16) {
        if (store) {
          uint8_t *dst = (is_v ? P.hi_v : P.hi_k) + (((int64_t)h * P.cap_hi + sl) * kHeadDim + lane4 * 32) * 2;
          uint32_t w[16];
#pragma unroll
          for (int c = 0; c < 16; ++c)
            w[c] = pack_f16x2(x[2 * c], x[2 * c + 1]);
          uint4 *d4 = reinterpret_cast<uint4 *>(dst);
#pragma unroll
          for (int i = 0; i < 4; ++i) d4[i] = make_uint4(w[4 * i], w[4 * i + 1], w[4 * i + 2], w[4 * i + 3]);
        }
      } else {
        uint8_t *dst = (is_v ? P.hi_v : P.hi_k) + ((int64_t)h * P.cap_hi + sl) * (kHeadDim * HI_BITS / 8) +
                       lane4 * (32 * HI_BITS / 8);
        uint32_t *par = (is_v ? P.hi_vp : P.hi_kp) + ((int64_t)h * P.cap_hi + sl) * ng + (lane4 * 32) / P.group;
        quantize_segment<HI_BITS>(x, P.group, lane4, dst, par, store);
      }
    } else if (P.evict) {
      // evicted token (no retained pool): nothing to store; the four lanes
      // of the row take this branch together
    } else if (LO_BITS == 2 && is_v && P.v_tiled) {
      // 2-bit values of a GQA cache go to the tiled layout, byte by byte
      uint32_t w[2];
      GroupParams gp = quantize_words<2>(x, P.group, w);
      if (store) {
        store_int2_v(P.lo_v + (int64_t)h * P.cap_lo * (kHeadDim / 4), sl, lane4, w);
        if ((lane4 % (P.group / 32)) == 0)
          P.lo_vp[((int64_t)h * P.cap_lo + sl) * ng + (lane4 * 32) / P.group] =
              (uint32_t)gp.a16 | ((uint32_t)gp.b16 << 16);
      }
    } else if (!is_v && P.lo_kb) {
      // per-channel key: codes with its block's parameters (the block is
      // complete: the placement below refused tokens of incomplete blocks)
      if (store) {
        uint32_t w[LO_BITS];
        const int blk = (pos0 + j0 + t) / kKeyBlock;
        encode_key_channels<LO_BITS>(x, P.lo_kb + ((int64_t)h * P.n_kblk + blk) * kHeadDim, lane4, w);
        uint32_t *dst = reinterpret_cast<uint32_t *>(P.lo_k + ((int64_t)h * P.cap_lo + sl) * (kHeadDim * LO_BITS / 8) +
                                                     lane4 * (32 * LO_BITS / 8));
#pragma unroll
        for (int i = 0; i < LO_BITS; ++i) dst[i] = w[i];
      }
    } else {
      uint8_t *dst = (is_v ? P.lo_v : P.lo_k) + ((int64_t)h * P.cap_lo + sl) * (kHeadDim * LO_BITS / 8) +
                     lane4 * (32 * LO_BITS / 8);
      uint32_t *par = (is_v ? P.lo_vp : P.lo_kp) + ((int64_t)h * P.cap_lo + sl) * ng + (lane4 * 32) / P.group;
      quantize_segment<LO_BITS>(x, P.group, lane4, dst, par, store);
    }
  }
  if (commit) {
    __syncthreads();
    if (tid == 0) {
      P.n_hi[h] = min(n_hi0 + s_total[0], P.cap_hi);
      if (!P.evict) P.n_lo[h] = min(n_lo0 + s_total[1], P.cap_lo);
    }
  }
}

// One new token per head into the importance pool (the decoding step):
// 8 lanes per head, lanes 0-3 the key row, 4-7 the value row; lane 0 of the
// head then advances n_hi (or flags a full pool).
template <int HI_BITS>
__global__ __launch_bounds__(64) void append_one_kernel(Pools P, const uint16_t *k, const uint16_t *v,
                                                        const float *balance, int pos, const float *score_init,
                                                        int n_heads) {
  const int t = blockIdx.x * 64 + threadIdx.x;
  const int h = t >> 3;
  if (h >= n_heads) return;  // all 8 lanes of a head leave together
  const int n0 = P.n_hi[h];
  if (n0 < P.cap_hi) {  // the same for the 8 lanes of the head
    const AppendArgs app = append_args(P, k, v, balance, pos, score_init);
    append_row<HI_BITS>(app, h, n0, t & 7);
    if ((t & 7) == 0) P.n_hi[h] = n0 + 1;
  } else if ((t & 7) == 0) {
    atomicOr(P.status, MIKV_DEVERR_HI_FULL);
  }
}

// Advance n_hi/n_lo after a multi-chunk placement.
__global__ void commit_counts_kernel(Pools P, int n_heads, int n, const int32_t *counts, int nchunks) {
  int h = blockIdx.x * blockDim.x + threadIdx.x;
  if (h >= n_heads) return;
  int th = n;
  int tl = 0;
  if (counts) {
    th = 0;
    for (int c = 0; c < nchunks; ++c) th += counts[h * nchunks + c];
    tl = n - th;
  }
  P.n_hi[h] = min(P.n_hi[h] + th, P.cap_hi);
  if (!P.evict) P.n_lo[h] = min(P.n_lo[h] + tl, P.cap_lo);
}

template <int HI_BITS, int LO_BITS>
void launch_place(const mikv_cache *c, const uint16_t *k, const uint16_t *v, const float *balance, int pos0,
                  int n, const uint8_t *hi_mask, const float *score_init, int32_t *counts, hipStream_t st) {
  Pools P = make_pools(c);
  int NH = n_heads_of(c);
  if (n == 1 && !hi_mask) {
    hipLaunchKernelGGL((append_one_kernel<HI_BITS>), dim3((NH * 8 + 63) / 64), dim3(64), 0, st, P, k, v, balance,
                       pos0, score_init, NH);
    return;
  }
  int nchunks = (n + kChunk - 1) / kChunk;
  if (P.lo_kb) {
    // parameters of the key blocks that lie within the placed positions,
    // before the retained keys are encoded with them
    const int b0 = (pos0 + kKeyBlock - 1) / kKeyBlock, b1 = (pos0 + n) / kKeyBlock;
    if (b1 > b0)
      hipLaunchKernelGGL(key_block_rows_kernel, dim3(b1 - b0, NH), dim3(256), 0, st, P, k, pos0, n, b0, LO_BITS);
  }
  if (hi_mask) {
    hipLaunchKernelGGL(count_hi_kernel, dim3(nchunks, NH), dim3(kChunk), 0, st, hi_mask, n, nchunks, counts);
  }
  int commit = nchunks == 1 ? 1 : 0;
  hipLaunchKernelGGL((place_kernel<HI_BITS, LO_BITS>), dim3(nchunks, NH), dim3(256), 0, st, P, k, v, balance,
                     pos0, n, hi_mask, score_init, hi_mask ? counts : nullptr, nchunks, commit);
  if (!commit) {
    hipLaunchKernelGGL(commit_counts_kernel, dim3((NH + 255) / 256), dim3(256), 0, st, P, NH, n,
                       hi_mask ? counts : nullptr, nchunks);
  }
}

}  // namespace

int close_key_block_from_pool(const mikv_cache *c, int32_t blk, hipStream_t st) {
  if (!c->key_block || blk < 0 || blk >= key_blocks_of(c)) return MIKV_OK;
  hipLaunchKernelGGL(key_block_pool_kernel, dim3(n_heads_of(c)), dim3(256), 0, st, make_pools(c), (int)blk,
                     (int)c->lo_bits);
  return check_launch("key block parameters");
}

}  // namespace mikv

using namespace mikv;

extern "C" int mikv_quantize_rows(const uint16_t *x, int64_t rows, int32_t head_dim, const float *balance,
                                  int32_t rows_per_balance, int32_t bits, int32_t group, uint8_t *codes,
                                  uint16_t *params, void *stream) {
  if (rows < 0) return set_error(MIKV_ERR_INVALID_ARG, "mikv_quantize_rows: rows < 0");
  if (rows == 0) return MIKV_OK;  // nothing to do; pointers may be NULL
  if (!x || !codes || !params) return set_error(MIKV_ERR_INVALID_ARG, "mikv_quantize_rows: NULL pointer");
  if (head_dim != kHeadDim) return set_error(MIKV_ERR_UNSUPPORTED, "mikv_quantize_rows: head_dim must be 128");
  if (bits != 2 && bits != 3 && bits != 4 && bits != 8)
    return set_error(MIKV_ERR_UNSUPPORTED, "mikv_quantize_rows: bits must be 2, 3, 4 or 8");
  if (group != 32 && group != 64 && group != 128)
    return set_error(MIKV_ERR_UNSUPPORTED, "mikv_quantize_rows: group must be 32, 64 or 128");
  if (balance && rows_per_balance < 1)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_quantize_rows: rows_per_balance must be >= 1");
  hipStream_t st = (hipStream_t)stream;
  int64_t threads = rows * 4;
  dim3 grid((unsigned)((threads + 255) / 256));
  switch (bits) {
    case 2:
      hipLaunchKernelGGL(quantize_rows_kernel<2>, grid, dim3(256), 0, st, x, rows, balance, rows_per_balance,
                         group, codes, params);
      break;
    case 3:
      hipLaunchKernelGGL(quantize_rows_kernel<3>, grid, dim3(256), 0, st, x, rows, balance, rows_per_balance,
                         group, codes, params);
      break;
    case 4:
      hipLaunchKernelGGL(quantize_rows_kernel<4>, grid, dim3(256), 0, st, x, rows, balance, rows_per_balance,
                         group, codes, params);
      break;
    default:
      hipLaunchKernelGGL(quantize_rows_kernel<8>, grid, dim3(256), 0, st, x, rows, balance, rows_per_balance,
                         group, codes, params);
  }
  return check_launch("mikv_quantize_rows");
}

extern "C" size_t mikv_quantize_workspace_size(const mikv_cache *c, int32_t n) {
  if (!c || n < 1) return 0;
  int64_t nchunks = (n + kChunk - 1) / kChunk;
  return (size_t)(nchunks * (int64_t)c->batch * c->kv_heads * 4);
}

extern "C" int mikv_quantize_kv(const mikv_cache *c, const uint16_t *k, const uint16_t *v, const float *balance,
                                int32_t pos0, int32_t n, const uint8_t *hi_mask, const float *score_init,
                                void *workspace, size_t workspace_bytes, void *stream) {
  int rc = validate_cache(c);
  if (rc) return rc;
  if (!k || !v) return set_error(MIKV_ERR_INVALID_ARG, "mikv_quantize_kv: k/v is NULL");
  if (n < 1 || pos0 < 0) return set_error(MIKV_ERR_INVALID_ARG, "mikv_quantize_kv: need n >= 1, pos0 >= 0");
  if ((int64_t)pos0 + n > c->max_len)
    return set_error(MIKV_ERR_CAPACITY, "mikv_quantize_kv: positions up to %lld exceed max_len %d",
                     (long long)pos0 + n, c->max_len);
  if (hi_mask) {
    if (!workspace || workspace_bytes < mikv_quantize_workspace_size(c, n))
      return set_error(MIKV_ERR_CAPACITY, "mikv_quantize_kv: workspace too small (%zu < %zu)", workspace_bytes,
                       mikv_quantize_workspace_size(c, n));
  }
  if (c->key_block && balance)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_quantize_kv: per-channel keys take no balancer");
  hipStream_t st = (hipStream_t)stream;
  int32_t *counts = (int32_t *)workspace;
  switch (format_key(c)) {
    case 1602: launch_place<16, 2>(c, k, v, balance, pos0, n, hi_mask, score_init, counts, st); break;
    case 1604: launch_place<16, 4>(c, k, v, balance, pos0, n, hi_mask, score_init, counts, st); break;
    case 1608: launch_place<16, 8>(c, k, v, balance, pos0, n, hi_mask, score_init, counts, st); break;
    case 802: launch_place<8, 2>(c, k, v, balance, pos0, n, hi_mask, score_init, counts, st); break;
    case 1603: launch_place<16, 3>(c, k, v, balance, pos0, n, hi_mask, score_init, counts, st); break;
    case 803: launch_place<8, 3>(c, k, v, balance, pos0, n, hi_mask, score_init, counts, st); break;
    case 402: launch_place<4, 2>(c, k, v, balance, pos0, n, hi_mask, score_init, counts, st); break;
    case 804: launch_place<8, 4>(c, k, v, balance, pos0, n, hi_mask, score_init, counts, st); break;
    default: launch_place<8, 8>(c, k, v, balance, pos0, n, hi_mask, score_init, counts, st); break;
  }
  rc = check_launch("mikv_quantize_kv");
  if (rc || !c->key_block) return rc;
  // a key block that started before pos0 and is complete now: its
  // parameters from the importance pool, where its keys are
  const int b = pos0 / kKeyBlock;
  if (pos0 % kKeyBlock != 0 && (b + 1) * kKeyBlock <= pos0 + n) return close_key_block_from_pool(c, b, st);
  return MIKV_OK;
}
