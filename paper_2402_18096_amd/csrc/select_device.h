// Device side of the top-k re-rank with a recent window and the demotion of
// tokens that leave the importance cache (Fig. 3 right; Sections 2.1, 3.1),
// shared by the select kernels and the fused finalize-and-select kernel of
// the decode step.
//
// One block per (sequence, KV head).  Ranking uses the unique 64-bit key
// (order-preserving score bits << 32 | position): a larger key is more
// important, and an exact score tie goes to the newer token.  The cut is
// found by an 8-pass, 8-bit MSB-first radix select over the eligible keys
// (LDS histogram per pass), or by a single min-reduction when exactly one
// token must go -- the steady state of decoding, where each step adds one
// token and the budget grows by at most one.
#ifndef MIKV_SELECT_DEVICE_H
#define MIKV_SELECT_DEVICE_H

#include "mikv_internal.h"

namespace mikv {

namespace {

constexpr int kSel = 256;

__device__ inline uint64_t rank_key(float score, int pos) {
  return ((uint64_t)ordered_bits(score) << 32) | (uint32_t)pos;
}

__device__ inline uint64_t block_min_u64(uint64_t v, uint64_t *s_tmp) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    uint64_t w = __shfl_xor(v, o, 64);
    v = w < v ? w : v;
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) s_tmp[wave] = v;
  __syncthreads();
  uint64_t r = s_tmp[0];
  for (int w = 1; w < kSel / 64; ++w) r = s_tmp[w] < r ? s_tmp[w] : r;
  __syncthreads();
  return r;
}

__device__ inline int block_sum_int(int v, int *s_tmp) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) s_tmp[wave] = v;
  __syncthreads();
  int r = 0;
  for (int w = 0; w < kSel / 64; ++w) r += s_tmp[w];
  __syncthreads();
  return r;
}

// Key of ascending rank `rank` (1-based) among the n candidates with
// elig(i); keys are unique so the result identifies exactly one candidate.
template <class Elig, class Key>
__device__ uint64_t radix_select(int n, int rank, Elig elig, Key key) {
  __shared__ uint32_t hist[256];
  __shared__ uint64_t s_prefix;
  __shared__ int s_rank;
  uint64_t prefix = 0, mask = 0;
  for (int pass = 0; pass < 8; ++pass) {
    const int shift = 56 - 8 * pass;
    hist[threadIdx.x] = 0;
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += kSel) {
      if (!elig(i)) continue;
      uint64_t k = key(i);
      if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 0xff], 1u);
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int cum = 0, d = 0;
      for (; d < 255; ++d) {
        if (cum + (int)hist[d] >= rank) break;
        cum += hist[d];
      }
      s_prefix = prefix | ((uint64_t)d << shift);
      s_rank = rank - cum;
    }
    __syncthreads();
    prefix = s_prefix;
    rank = s_rank;
    mask |= (uint64_t)0xff << shift;
    __syncthreads();
  }
  return prefix;
}

// Ordered compaction: writes, in ascending i, every i in [lo, hi) with
// flag(i) to out[0..), returns the count.  Whole block takes part.
template <class Flag>
__device__ int compact(int lo, int hi, Flag flag, int32_t *out) {
  __shared__ int s_w[kSel / 64];
  __shared__ int s_base;
  __syncthreads();
  if (threadIdx.x == 0) s_base = 0;
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int t0 = lo; t0 < hi; t0 += kSel) {
    const int i = t0 + threadIdx.x;
    const bool f = i < hi && flag(i);
    unsigned long long bal = __ballot(f);
    if (lane == 0) s_w[wave] = __popcll(bal);
    __syncthreads();
    int off = s_base;
    for (int w = 0; w < wave; ++w) off += s_w[w];
    if (f) out[off + __popcll(bal & ((1ull << lane) - 1ull))] = i;
    __syncthreads();
    if (threadIdx.x == 0) {
      int t = 0;
      for (int w = 0; w < kSel / 64; ++w) t += s_w[w];
      s_base += t;
    }
    __syncthreads();
  }
  const int total = s_base;
  __syncthreads();
  return total;
}

struct SelArgs {
  uint8_t *hi_k, *hi_v;
  uint32_t *hi_kp, *hi_vp;
  int32_t *hi_pos;
  float *hi_acc;
  int32_t *n_hi;
  uint8_t *lo_k, *lo_v;
  uint32_t *lo_kp, *lo_vp;
  int32_t *lo_pos, *n_lo;
  uint8_t *map;
  int32_t *status;
  int32_t *ws;
  int cap_hi, cap_lo, max_len, group;
  int length, k_heavy, window;
  int v_tiled;  // 2-bit values in the tiled layout (int2_values_tiled)
  int pending;  // n_hi does not yet count the step's appended token (slot n_hi holds it)
  int evict;    // no retained pool: a token that leaves the importance pool is dropped
  // per-channel keys: (alpha, beta) words [NH, n_kblk, 128] per key block
  const uint32_t *lo_kb;
  int n_kblk;
};

// Decode the 32 channels [part*32, part*32+32) of an importance-pool row.
template <int HI_BITS>
__device__ inline void load_hi_segment(const SelArgs &A, const uint8_t *rows, const uint32_t *pars, int64_t slot,
                                       int part, float x[32]) {
  if constexpr (HI_BITS == 16) {
    const uint4 *s4 = reinterpret_cast<const uint4 *>(rows + (slot * kHeadDim + part * 32) * 2);
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
  } else if constexpr (HI_BITS == 8) {
    const uint4 *s4 = reinterpret_cast<const uint4 *>(rows + slot * kHeadDim + part * 32);
    const uint32_t par = pars[slot * (kHeadDim / A.group) + (part * 32) / A.group];
    const float a = f16_to_f32((uint16_t)(par & 0xffffu)), b = f16_to_f32((uint16_t)(par >> 16));
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      uint4 w = s4[i];
      uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int j = 0; j < 16; ++j) x[i * 16 + j] = fmaf(a, (float)((ws[j >> 2] >> (8 * (j & 3))) & 0xffu), b);
    }
  } else {  // INT4: 32 codes in 16 bytes, channel c at bits 4c
    const uint4 w = *reinterpret_cast<const uint4 *>(rows + slot * (kHeadDim / 2) + part * 16);
    const uint32_t par = pars[slot * (kHeadDim / A.group) + (part * 32) / A.group];
    const float a = f16_to_f32((uint16_t)(par & 0xffffu)), b = f16_to_f32((uint16_t)(par >> 16));
    const uint32_t ws[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int j = 0; j < 32; ++j) x[j] = fmaf(a, (float)((ws[j >> 3] >> (4 * (j & 7))) & 0xfu), b);
  }
}

// Eq. 1 codes at LO_BITS of 32 decoded channels (a group spans group/32
// lanes): the packed little-endian words and the group parameters.
template <int LO_BITS>
__device__ inline GroupParams lo_words(const SelArgs &A, const float x[32], uint32_t w[LO_BITS]) {
  float mn = x[0], mx = x[0];
#pragma unroll
  for (int c = 1; c < 32; ++c) {
    mn = fminf(mn, x[c]);
    mx = fmaxf(mx, x[c]);
  }
  for (int o = 1; o < A.group / 32; o <<= 1) {
    mn = fminf(mn, __shfl_xor(mn, o, 64));
    mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  }
  GroupParams p = group_params(mn, mx, LO_BITS);
#pragma unroll
  for (int i = 0; i < LO_BITS; ++i) w[i] = 0u;
#pragma unroll
  for (int c = 0; c < 32; ++c) put_code<LO_BITS>(w, c, encode(x[c], p, LO_BITS));
  return p;
}

// Eq. 1 at LO_BITS of 32 decoded channels into retained-pool slot lslot:
// codes token-major, except 2-bit values of a GQA cache (tiled layout).
template <int LO_BITS>
__device__ inline void store_lo_segment(const SelArgs &A, int h, int64_t lslot, bool is_v, int part,
                                        const float x[32], int pos) {
  const int ng = kHeadDim / A.group;
  uint32_t w[LO_BITS];
  if (!is_v && A.lo_kb) {
    // per-channel key: its block's parameters (the block is complete: the
    // token has left a window of at least one block)
    encode_key_channels<LO_BITS>(x, A.lo_kb + ((int64_t)h * A.n_kblk + pos / kKeyBlock) * kHeadDim, part, w);
    uint32_t *codes = reinterpret_cast<uint32_t *>(A.lo_k + lslot * (kHeadDim * LO_BITS / 8) + part * (32 * LO_BITS / 8));
#pragma unroll
    for (int i = 0; i < LO_BITS; ++i) codes[i] = w[i];
    return;
  }
  GroupParams p = lo_words<LO_BITS>(A, x, w);
  if (LO_BITS == 2 && is_v && A.v_tiled) {
    store_int2_v(A.lo_v + (int64_t)h * A.cap_lo * (kHeadDim / 4), lslot - (int64_t)h * A.cap_lo, part, w);
  } else {
    uint32_t *codes = reinterpret_cast<uint32_t *>(lane_pick(is_v, A.lo_v, A.lo_k) + lslot * (kHeadDim * LO_BITS / 8) +
                                                   part * (32 * LO_BITS / 8));
#pragma unroll
    for (int i = 0; i < LO_BITS; ++i) codes[i] = w[i];
  }
  if ((part % (A.group / 32)) == 0)
    lane_pick(is_v, A.lo_vp, A.lo_kp)[lslot * ng + (part * 32) / A.group] = (uint32_t)p.a16 | ((uint32_t)p.b16 << 16);
}

template <int HI_BITS, int LO_BITS>
__device__ inline void demote_row(const SelArgs &A, int h, int slot, int64_t lslot, int p) {
  if (threadIdx.x >= 8) return;
  const int ng = kHeadDim / A.group;
  const int64_t hrow = HI_BITS == 16 ? 2 * kHeadDim : kHeadDim * HI_BITS / 8;
  const int is_v = threadIdx.x >> 2, part = threadIdx.x & 3;
  const uint8_t *rows = lane_pick(is_v, A.hi_v, A.hi_k) + (int64_t)h * A.cap_hi * hrow;
  const uint32_t *pars = HI_BITS == 16 ? nullptr : lane_pick(is_v, A.hi_vp, A.hi_kp) + (int64_t)h * A.cap_hi * ng;
  float x[32];
  load_hi_segment<HI_BITS>(A, rows, pars, slot, part, x);
  store_lo_segment<LO_BITS>(A, h, lslot, is_v, part, x, p);
  if (threadIdx.x == 0) {
    A.lo_pos[lslot] = p;
    if (A.map) A.map[(int64_t)h * A.max_len + p] = 0;
  }
}

// One importance-pool slot's data (rows, position, score and, for INT8
// rows, the scale/zero words), spread over the block: threads below
// 2 * row/16 hold a 16-byte piece of the K or V row, threads 64.. a scale
// word, thread 0 the position and score.  Loaded early, stored late.
template <int HI_BITS>
struct SlotData {
  uint4 piece;
  uint32_t par;
  int pos;
  float acc;
};

template <int HI_BITS>
__device__ inline SlotData<HI_BITS> load_slot(const SelArgs &A, int h, int src) {
  constexpr int64_t hrow = HI_BITS == 16 ? 2 * kHeadDim : kHeadDim * HI_BITS / 8;
  constexpr int chunks = hrow / 16;
  const int ng = kHeadDim / A.group;
  SlotData<HI_BITS> d{};
  if (threadIdx.x < 2 * chunks) {
    const uint8_t *base = lane_pick(threadIdx.x < chunks, A.hi_k, A.hi_v) + (int64_t)h * A.cap_hi * hrow;
    d.piece = reinterpret_cast<const uint4 *>(base + (int64_t)src * hrow)[threadIdx.x % chunks];
  }
  if (HI_BITS != 16 && threadIdx.x >= 64 && threadIdx.x < 64 + 2 * ng) {
    const uint32_t *pp = lane_pick(threadIdx.x - 64 < (unsigned)ng, A.hi_kp, A.hi_vp);
    d.par = pp[((int64_t)h * A.cap_hi + src) * ng + (threadIdx.x - 64) % ng];
  }
  if (threadIdx.x == 0) {
    d.pos = A.hi_pos[(int64_t)h * A.cap_hi + src];
    d.acc = A.hi_acc[(int64_t)h * A.cap_hi + src];
  }
  return d;
}

template <int HI_BITS>
__device__ inline void store_slot(const SelArgs &A, int h, int dst, const SlotData<HI_BITS> &d) {
  constexpr int64_t hrow = HI_BITS == 16 ? 2 * kHeadDim : kHeadDim * HI_BITS / 8;
  constexpr int chunks = hrow / 16;
  const int ng = kHeadDim / A.group;
  if (threadIdx.x < 2 * chunks) {
    uint8_t *base = lane_pick(threadIdx.x < chunks, A.hi_k, A.hi_v) + (int64_t)h * A.cap_hi * hrow;
    reinterpret_cast<uint4 *>(base + (int64_t)dst * hrow)[threadIdx.x % chunks] = d.piece;
  }
  if (HI_BITS != 16 && threadIdx.x >= 64 && threadIdx.x < 64 + 2 * ng) {
    uint32_t *pp = lane_pick(threadIdx.x - 64 < (unsigned)ng, A.hi_kp, A.hi_vp);
    pp[((int64_t)h * A.cap_hi + dst) * ng + (threadIdx.x - 64) % ng] = d.par;
  }
  if (threadIdx.x == 0) {
    A.hi_pos[(int64_t)h * A.cap_hi + dst] = d.pos;
    A.hi_acc[(int64_t)h * A.cap_hi + dst] = d.acc;
  }
}

constexpr int kSelItems = 16;  // importance-pool slots per thread held in registers

// The running candidate state of one thread: eligible slots seen and the
// least important of them (key and slot).
struct SelScan {
  int cnt = 0, arg = -1;
  uint64_t mn = ~0ull;
  __device__ inline void add(int slot, int p, float score) {
    ++cnt;
    const uint64_t k = rank_key(score, p);
    if (k < mn) {
      mn = k;
      arg = slot;
    }
  }
};

// Scan slots [from, cap_hi) of head h from memory, kSel * kSelItems slots
// per round trip; thread t reads slots t, t + kSel, ...  The loads run to
// the capacity, so they need not wait for the pool count.
__device__ inline void select_scan(const SelArgs &A, int h, int from, int n, int thr, SelScan &sc) {
  const int32_t *pos = A.hi_pos + (int64_t)h * A.cap_hi;
  const float *acc = A.hi_acc + (int64_t)h * A.cap_hi;
  for (int base = from; base < A.cap_hi; base += kSel * kSelItems) {
    int pv[kSelItems];
    float av[kSelItems];
#pragma unroll
    for (int u = 0; u < kSelItems; ++u) {
      const int i = base + u * kSel + threadIdx.x;
      pv[u] = i < A.cap_hi ? pos[i] : thr;
      av[u] = i < A.cap_hi ? acc[i] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < kSelItems; ++u) {
      const int i = base + u * kSel + threadIdx.x;
      if (i < n && pv[u] < thr) sc.add(i, pv[u], av[u]);
    }
  }
}

// Second half of the re-rank of head h, once every thread has scanned its
// slots: count, find the cut, demote and refill.  `n` and `n_lo0` are the
// pool counts before the re-rank, `last` the prefetched last slot.  With
// `set_n` (n_hi in memory does not yet count an appended token) n_hi is
// written even when no token leaves.
template <int HI_BITS, int LO_BITS>
__device__ __attribute__((always_inline)) void select_finish(const SelArgs &A, int h, int n, int n_lo0, const SelScan &sc,
                              const SlotData<HI_BITS> &last, bool set_n = false) {
  __shared__ int s_tmp_i[kSel / 64];
  __shared__ uint64_t s_tmp_u[kSel / 64];
  __shared__ int s_arg[3];
  const int thr = A.length - A.window;  // positions >= thr are in the window
  const int32_t *pos = A.hi_pos + (int64_t)h * A.cap_hi;
  const float *acc = A.hi_acc + (int64_t)h * A.cap_hi;
  auto elig = [&](int i) { return pos[i] < thr; };
  auto key = [&](int i) { return rank_key(acc[i], pos[i]); };

  const int n_elig = block_sum_int(sc.cnt, s_tmp_i);
  const int n_dem = n_elig - A.k_heavy;
  if (n_dem <= 0 || (!A.evict && n_lo0 + n_dem > A.cap_lo)) {
    if (threadIdx.x == 0) {
      if (n_dem > 0) atomicOr(A.status, MIKV_DEVERR_LO_FULL);
      if (set_n) A.n_hi[h] = n;
    }
    return;
  }

  if (n_dem == 1) {
    // Steady state of decoding: the least important eligible token leaves;
    // the last slot fills its hole.
    const uint64_t cut = block_min_u64(sc.mn, s_tmp_u);
    if (sc.arg >= 0 && sc.mn == cut) s_arg[0] = sc.arg;
    __syncthreads();
    const int slot = s_arg[0];
    // the key's low word is the position
    if (!A.evict)
      demote_row<HI_BITS, LO_BITS>(A, h, slot, (int64_t)h * A.cap_lo + n_lo0, (int)(uint32_t)cut);
    else if (threadIdx.x == 0 && A.map)
      A.map[(int64_t)h * A.max_len + (int)(uint32_t)cut] = 0;
    __syncthreads();
    if (slot != n - 1) store_slot<HI_BITS>(A, h, slot, last);
    if (threadIdx.x == 0) {
      A.n_hi[h] = n - 1;
      if (!A.evict) A.n_lo[h] = n_lo0 + 1;
    }
    return;
  }

  // General case (several tokens leave): radix select of the cut, then
  // ordered compaction of the holes and of the survivors that fill them.
  const uint64_t cut = radix_select(n, n_dem, elig, key);
  auto demoted = [&](int i) { return elig(i) && key(i) <= cut; };

  int32_t *dem_list = A.ws + (int64_t)h * 2 * A.cap_hi;
  int32_t *fill_list = dem_list + A.cap_hi;
  const int n_new = n - n_dem;
  compact(0, n, demoted, dem_list);
  const int n_fill = compact(n_new, n, [&](int i) { return !demoted(i); }, fill_list);

  // re-quantize the demoted tokens into the retained pool (4 lanes per row)
  const int ng = kHeadDim / A.group;
  const int64_t hrow = HI_BITS == 16 ? 2 * kHeadDim : kHeadDim * HI_BITS / 8;
  for (int r = threadIdx.x >> 2; r < (A.evict ? 0 : 2 * n_dem); r += kSel / 4) {
    const int d = r >> 1, is_v = r & 1, part = threadIdx.x & 3;
    const int slot = dem_list[d];
    const uint8_t *rows = lane_pick(is_v, A.hi_v, A.hi_k) + (int64_t)h * A.cap_hi * hrow;
    const uint32_t *pars = HI_BITS == 16 ? nullptr : lane_pick(is_v, A.hi_vp, A.hi_kp) + (int64_t)h * A.cap_hi * ng;
    float x[32];
    load_hi_segment<HI_BITS>(A, rows, pars, slot, part, x);
    const int64_t lslot = (int64_t)h * A.cap_lo + n_lo0 + d;
    store_lo_segment<LO_BITS>(A, h, lslot, is_v, part, x, pos[slot]);
    if (part == 0 && !is_v) {
      const int p = pos[slot];
      A.lo_pos[lslot] = p;
      if (A.map) A.map[(int64_t)h * A.max_len + p] = 0;
    }
  }
  if (A.evict && A.map) {
    for (int d = threadIdx.x; d < n_dem; d += kSel) A.map[(int64_t)h * A.max_len + pos[dem_list[d]]] = 0;
  }
  __syncthreads();

  // refill the holes below n_new with the survivors above it (16 B moves)
  const int64_t hbytes = hrow;  // bytes per K (or V) row
  const int chunks = (int)(hbytes / 16);
  uint8_t *hk = A.hi_k + (int64_t)h * A.cap_hi * hrow;
  uint8_t *hv = A.hi_v + (int64_t)h * A.cap_hi * hrow;
  for (int idx = threadIdx.x; idx < n_fill * 2 * chunks; idx += kSel) {
    const int f = idx / (2 * chunks), rem = idx % (2 * chunks);
    const int src = fill_list[f], dst = dem_list[f];
    uint8_t *base = rem < chunks ? hk : hv;
    const int ck = rem % chunks;
    reinterpret_cast<uint4 *>(base + (int64_t)dst * hrow)[ck] = reinterpret_cast<const uint4 *>(base + (int64_t)src * hrow)[ck];
  }
  for (int f = threadIdx.x; f < n_fill; f += kSel) {
    const int src = fill_list[f], dst = dem_list[f];
    A.hi_pos[(int64_t)h * A.cap_hi + dst] = pos[src];
    A.hi_acc[(int64_t)h * A.cap_hi + dst] = acc[src];
    if (HI_BITS != 16) {
      for (int g = 0; g < ng; ++g) {
        A.hi_kp[((int64_t)h * A.cap_hi + dst) * ng + g] = A.hi_kp[((int64_t)h * A.cap_hi + src) * ng + g];
        A.hi_vp[((int64_t)h * A.cap_hi + dst) * ng + g] = A.hi_vp[((int64_t)h * A.cap_hi + src) * ng + g];
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    A.n_hi[h] = n_new;
    if (!A.evict) A.n_lo[h] = n_lo0 + n_dem;
  }
}

// Re-rank and demote for head h; the whole block (kSel threads) takes part.
template <int HI_BITS, int LO_BITS>
__device__ __attribute__((always_inline)) void select_head(const SelArgs &A, int h) {
  const int n_mem = __builtin_amdgcn_readfirstlane(A.n_hi[h]);
  const int n = n_mem + (A.pending && n_mem < A.cap_hi ? 1 : 0);
  const int n_lo0 = __builtin_amdgcn_readfirstlane(A.n_lo[h]);
  SelScan sc;
  select_scan(A, h, 0, n, A.length - A.window, sc);
  // The last slot fills the hole of a demoted token: fetch it now, its
  // latency then hides behind the reductions.
  const SlotData<HI_BITS> last = n > 0 ? load_slot<HI_BITS>(A, h, n - 1) : SlotData<HI_BITS>{};
  select_finish<HI_BITS, LO_BITS>(A, h, n, n_lo0, sc, last, A.pending != 0);
}

// Arguments of a select for the cache `c` (host side).
inline SelArgs make_sel_args(const mikv_cache *c, int length, int k_heavy, int window, void *ws) {
  SelArgs A;
  A.hi_k = (uint8_t *)c->hi_k;
  A.hi_v = (uint8_t *)c->hi_v;
  A.hi_kp = (uint32_t *)c->hi_kp;
  A.hi_vp = (uint32_t *)c->hi_vp;
  A.hi_pos = c->hi_pos;
  A.hi_acc = c->hi_acc;
  A.n_hi = c->n_hi;
  A.lo_k = c->lo_k;
  A.lo_v = c->lo_v;
  A.lo_kp = (uint32_t *)c->lo_kp;
  A.lo_vp = (uint32_t *)c->lo_vp;
  A.lo_pos = c->lo_pos;
  A.n_lo = c->n_lo;
  A.map = c->map;
  A.status = c->status;
  A.ws = (int32_t *)ws;
  A.cap_hi = c->cap_hi;
  A.cap_lo = c->cap_lo;
  A.max_len = c->max_len;
  A.group = c->group;
  A.length = length;
  A.k_heavy = k_heavy;
  A.window = window;
  A.v_tiled = int2_values_tiled(c->lo_bits, c->q_heads, c->kv_heads) ? 1 : 0;
  A.pending = 0;
  A.evict = evicting(c) ? 1 : 0;
  A.lo_kb = c->key_block ? (const uint32_t *)c->lo_kb : nullptr;
  A.n_kblk = c->key_block ? key_blocks_of(c) : 0;
  return A;
}

}  // namespace

}  // namespace mikv

#endif  // MIKV_SELECT_DEVICE_H
