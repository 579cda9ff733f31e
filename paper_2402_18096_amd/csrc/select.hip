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

extern "C" int mikv_select_topk(const mikv_cache *c, int32_t length, int32_t k_heavy, int32_t window, void *ws,
                                size_t ws_bytes, void *stream) {
  return select_topk(c, length, k_heavy, window, ws, ws_bytes, false, (hipStream_t)stream);
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
