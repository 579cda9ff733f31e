// Top-k re-ranking with a recent window, demotion of tokens that fall out of
// the importance cache to the retained cache (re-quantized with Eq. 1), and
// the first selection after prefill (Fig. 3 right; Sections 2.1, 3.1).  The
// per-head device code is in select_device.h.
#include <algorithm>

#include "select_device.h"

namespace mikv {

namespace {

// (Register budget: five blocks per CU, so 1280 heads take one round.)
template <int HI_BITS, int LO_BITS>
__global__ __launch_bounds__(kSel) __attribute__((amdgpu_waves_per_eu(5))) void select_kernel(SelArgs A) {
  select_head<HI_BITS, LO_BITS>(A, blockIdx.x);
}

__global__ __launch_bounds__(kSel) void select_prefill_kernel(const float *scores, int length, int k_heavy, int window,
                                                              uint8_t *hi_mask) {
  const int h = blockIdx.x;
  const float *sc = scores + (int64_t)h * length;
  uint8_t *mask = hi_mask + (int64_t)h * length;
  const int thr = length - window > 0 ? length - window : 0;
  const int n_dem = thr - k_heavy;
  uint64_t cut = 0;
  bool any = n_dem > 0;
  if (any) {
    auto elig = [&](int i) { return i < thr; };
    auto key = [&](int i) { return rank_key(sc[i], i); };
    cut = radix_select(thr, n_dem, elig, key);
  }
  for (int j = threadIdx.x; j < length; j += kSel) {
    uint8_t hi = 1;
    if (any && j < thr && rank_key(sc[j], j) <= cut) hi = 0;
    mask[j] = hi;
  }
}

// The sorted heavy-token list (Fig. 3 right: the tokens the re-rank kept
// for their accumulated attention): per head, the importance-pool tokens
// outside the window, most important first by the rank key (score
// descending, an exact tie to the newer token).  One block per head sorts
// the pool's keys in LDS with a bitonic network (window tokens and empty
// slots get key 0, below every real key, so they sort last).
constexpr int kHeavyMaxSlots = 8192;  // importance-pool slots a head may hold for the list (64 KiB of keys)

__global__ __launch_bounds__(kSel) void heavy_list_kernel(const int32_t *n_hi, const int32_t *hi_pos,
                                                          const float *hi_acc, int cap_hi, int P, int thr, int k_heavy,
                                                          int32_t *heavy_idx) {
  extern __shared__ uint64_t s_key[];  // [P], P a power of two >= cap_hi
  const int h = blockIdx.x;
  const int n = min(n_hi[h], cap_hi);
  const int32_t *pos = hi_pos + (int64_t)h * cap_hi;
  const float *acc = hi_acc + (int64_t)h * cap_hi;
  for (int i = threadIdx.x; i < P; i += kSel) {
    uint64_t k = 0;
    if (i < n) {
      const int p = pos[i];
      if (p < thr) k = rank_key(acc[i], p);
    }
    s_key[i] = k;
  }
  __syncthreads();
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = threadIdx.x; i < P; i += kSel) {
        const int l = i ^ j;
        if (l > i) {
          const uint64_t a = s_key[i], b = s_key[l];
          // descending overall: runs with (i & k) == 0 descend, the others ascend
          const bool swap = (i & k) == 0 ? a < b : a > b;
          if (swap) {
            s_key[i] = b;
            s_key[l] = a;
          }
        }
      }
      __syncthreads();
    }
  }
  int32_t *out = heavy_idx + (int64_t)h * k_heavy;
  for (int r = threadIdx.x; r < k_heavy; r += kSel) {
    const uint64_t k = r < P ? s_key[r] : 0;
    out[r] = k != 0 ? (int32_t)(uint32_t)(k & 0xffffffffu) : -1;
  }
}

template <int HI, int LO>
void launch_select(const SelArgs &A, int NH, hipStream_t st) {
  hipLaunchKernelGGL((select_kernel<HI, LO>), dim3(NH), dim3(kSel), 0, st, A);
}

}  // namespace

}  // namespace mikv

using namespace mikv;

extern "C" size_t mikv_select_workspace_size(const mikv_cache *c) {
  if (!c) return 0;
  return (size_t)2 * 4 * (size_t)c->batch * c->kv_heads * (size_t)std::max(c->cap_hi, 1);
}

namespace mikv {

int select_topk(const mikv_cache *c, int32_t length, int32_t k_heavy, int32_t window, void *ws, size_t ws_bytes,
                bool appended, hipStream_t st) {
  int rc = validate_cache(c);
  if (rc) return rc;
  if (k_heavy < 0 || window < 0) return set_error(MIKV_ERR_INVALID_ARG, "mikv_select_topk: negative k_heavy/window");
  if (length < 1 || length > c->max_len)
    return set_error(length < 1 ? MIKV_ERR_INVALID_ARG : MIKV_ERR_CAPACITY,
                     "mikv_select_topk: length %d outside [1, max_len]", length);
  if (!ws || ws_bytes < mikv_select_workspace_size(c))
    return set_error(MIKV_ERR_CAPACITY, "mikv_select_topk: workspace too small");
  if (c->key_block && window < kKeyBlock)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_select_topk: per-channel keys need a window >= %d (got %d)",
                     kKeyBlock, window);
  SelArgs A = make_sel_args(c, length, k_heavy, window, ws);
  A.pending = appended ? 1 : 0;
  const int NH = n_heads_of(c);
  switch (format_key(c)) {
    case 1602: launch_select<16, 2>(A, NH, st); break;
    case 1604: launch_select<16, 4>(A, NH, st); break;
    case 1608: launch_select<16, 8>(A, NH, st); break;
    case 802: launch_select<8, 2>(A, NH, st); break;
    case 1603: launch_select<16, 3>(A, NH, st); break;
    case 803: launch_select<8, 3>(A, NH, st); break;
    case 402: launch_select<4, 2>(A, NH, st); break;
    case 804: launch_select<8, 4>(A, NH, st); break;
    default: launch_select<8, 8>(A, NH, st); break;
  }
  return check_launch("mikv_select_topk");
}

}  // namespace mikv

extern "C" int mikv_select_topk(const mikv_cache *c, int32_t length, int32_t k_heavy, int32_t window,
                                int32_t *heavy_idx, void *ws, size_t ws_bytes, void *stream) {
  if (heavy_idx && c && c->cap_hi > kHeavyMaxSlots)
    return set_error(MIKV_ERR_UNSUPPORTED, "mikv_select_topk: the heavy list needs cap_hi <= %d (got %d)",
                     kHeavyMaxSlots, c->cap_hi);
  int rc = select_topk(c, length, k_heavy, window, ws, ws_bytes, false, (hipStream_t)stream);
  if (rc || !heavy_idx || k_heavy == 0) return rc;
  int P = 1;
  while (P < c->cap_hi) P <<= 1;
  const int thr = std::max(0, length - window);
  hipLaunchKernelGGL(heavy_list_kernel, dim3(n_heads_of(c)), dim3(kSel), (size_t)P * sizeof(uint64_t),
                     (hipStream_t)stream, c->n_hi, c->hi_pos, c->hi_acc, c->cap_hi, P, thr, k_heavy, heavy_idx);
  return check_launch("mikv_select_topk (heavy list)");
}

extern "C" int32_t mikv_heavy_budget(int32_t length, int32_t ratio_num, int32_t ratio_den, int32_t window,
                                     int32_t window_in_ratio) {
  if (length < 0 || ratio_num < 0 || ratio_den < 1 || window < 0) return -1;
  int64_t k = (int64_t)ratio_num * length / ratio_den;
  if (window_in_ratio) k -= window;
  return (int32_t)std::max<int64_t>(0, k);
}

extern "C" int mikv_select_prefill(const float *scores, int32_t n_heads, int32_t length, int32_t k_heavy,
                                   int32_t window, uint8_t *hi_mask, void *stream) {
  if (!scores || !hi_mask) return set_error(MIKV_ERR_INVALID_ARG, "mikv_select_prefill: NULL pointer");
  if (n_heads < 1 || length < 1 || k_heavy < 0 || window < 0)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_select_prefill: bad sizes");
  hipLaunchKernelGGL(select_prefill_kernel, dim3(n_heads), dim3(kSel), 0, (hipStream_t)stream, scores, length,
                     k_heavy, window, hi_mask);
  return check_launch("mikv_select_prefill");
}
