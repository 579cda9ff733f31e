// One whole decode step of the method in one call (Fig. 3): append the new
// token, attention over both pools, importance update, re-rank and demote.
// A single host call keeps the step from being bound by per-call host
// overhead; optional events mark the phase boundaries for profiling.
#include <algorithm>
#include <mutex>

#include "mikv_internal.h"

using namespace mikv;

// Run the re-rank inside the finalize launch when the importance update is
// fused and the cache has at most this many (sequence, KV head) pairs.
// Fusing saves a launch but gives the finalize the select's larger resource
// footprint (lower occupancy): measured on MI355X it helps 128 heads (GQA),
// is neutral at 128-256 and costs 3 % at 1280.  0 turns fusing off.
#ifndef MIKV_STEP_FUSE_SELECT_MAX_HEADS
#define MIKV_STEP_FUSE_SELECT_MAX_HEADS 512
#endif

// Workspace of a step: the attention's, then the select's (256-byte aligned).
static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

extern "C" size_t mikv_decode_step_workspace_size(const mikv_cache *c, int32_t length) {
  size_t a = mikv_decode_workspace_size(c, length);
  if (!a) return 0;
  return align256(a) + mikv_select_workspace_size(c);
}

extern "C" int mikv_decode_step(const mikv_cache *c, int32_t length, const uint16_t *q, const uint16_t *k_new,
                                const uint16_t *v_new, const float *balance, float scale, float *out, float *probs_hi,
                                float *probs_lo, int32_t k_heavy, int32_t window, int32_t flags, void *workspace,
                                size_t workspace_bytes, void *const *phase_events, void *stream) {
  int rc = validate_cache(c);
  if (rc) return rc;
  if (!q || !k_new || !v_new || !out) return set_error(MIKV_ERR_INVALID_ARG, "mikv_decode_step: NULL input/output");
  if (length < 1 || length > c->max_len)
    return set_error(length < 1 ? MIKV_ERR_INVALID_ARG : MIKV_ERR_CAPACITY,
                     "mikv_decode_step: length %d outside [1, max_len]", length);
  if (k_heavy < 0 || window < 0) return set_error(MIKV_ERR_INVALID_ARG, "mikv_decode_step: negative k_heavy/window");
  const bool fused = (flags & MIKV_ATTN_ACCUMULATE) != 0;
  if (!fused && !probs_hi)
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_decode_step: probs_hi is required unless MIKV_ATTN_ACCUMULATE");
  if (c->key_block && (balance || window < kKeyBlock))
    return set_error(MIKV_ERR_INVALID_ARG, "mikv_decode_step: per-channel keys need no balancer and a window >= %d",
                     kKeyBlock);
  // the new token (position length - 1) completes a key block: its
  // per-channel parameters are taken at the end of the step, from the
  // importance pool (the fused paths append inside the attention)
  const int close_blk = c->key_block && fused && length % kKeyBlock == 0 ? length / kKeyBlock - 1 : -1;
  const size_t need = mikv_decode_step_workspace_size(c, length);
  if (!workspace || workspace_bytes < need)
    return set_error(MIKV_ERR_CAPACITY, "mikv_decode_step: workspace too small (%zu < %zu)", workspace_bytes, need);
  const size_t attn_ws = align256(mikv_decode_workspace_size(c, length));
  uint8_t *ws = (uint8_t *)workspace;
  hipStream_t st = (hipStream_t)stream;
  auto mark = [&](int i) {
    if (phase_events && phase_events[i]) hipEventRecord((hipEvent_t)phase_events[i], st);
  };
  mark(0);
  if (fused && n_heads_of(c) <= MIKV_STEP_FUSE_SELECT_MAX_HEADS) {
    // Two launches: the attention's partial phase, which also appends the
    // new token; then finalize, importance update and re-rank.
    mark(1);
    rc = decode_partial(c, length, q, balance, scale, out, probs_hi, probs_lo, flags, ws, attn_ws, k_new, v_new, st);
    if (rc) return rc;
    mark(2);
    rc = decode_finalize_select(c, length, q, balance, scale, out, probs_hi, probs_lo, ws, attn_ws, k_heavy, window,
                                ws + attn_ws, true, st);
    if (rc) return rc;
    if (close_blk >= 0 && (rc = close_key_block_from_pool(c, close_blk, st))) return rc;
    mark(3);
    mark(4);
    mark(5);
    return MIKV_OK;
  }
  if (fused) {
    // Three launches: partial phase with the append, finalize with the
    // importance update, re-rank (which counts the new token into n_hi).
    mark(1);
    rc = decode_partial(c, length, q, balance, scale, out, probs_hi, probs_lo, flags, ws, attn_ws, k_new, v_new, st);
    if (rc) return rc;
    mark(2);
    rc = decode_finalize(c, length, q, balance, scale, out, probs_hi, probs_lo, flags, ws, attn_ws, true, st);
    if (rc) return rc;
    mark(3);
    mark(4);
    rc = select_topk(c, length, k_heavy, window, ws + attn_ws, workspace_bytes - attn_ws, true, st);
    if (rc) return rc;
    if (close_blk >= 0 && (rc = close_key_block_from_pool(c, close_blk, st))) return rc;
    mark(5);
    return MIKV_OK;
  }
  rc = mikv_quantize_kv(c, k_new, v_new, balance, length - 1, 1, nullptr, nullptr, nullptr, 0, stream);
  if (rc) return rc;
  mark(1);
  rc = decode_partial(c, length, q, balance, scale, out, probs_hi, probs_lo, flags, ws, attn_ws, nullptr, nullptr,
                      st);
  if (rc) return rc;
  mark(2);
  rc = mikv_decode_attention_finalize(c, length, q, balance, scale, out, probs_hi, probs_lo, flags, ws, attn_ws,
                                      stream);
  if (rc) return rc;
  mark(3);
  rc = mikv_importance_update(c, length, probs_hi, stream);
  if (rc) return rc;
  mark(4);
  rc = mikv_select_topk(c, length, k_heavy, window, nullptr, ws + attn_ws, workspace_bytes - attn_ws, stream);
  if (rc) return rc;
  mark(5);
  return MIKV_OK;
}

// ---------------------------------------------------------------------------
// The decode step without a caller workspace, for callers that cannot
// allocate device memory.  Its workspace is a file-scope device array; each
// GPU the library runs on holds its own copy until the process ends.  In
// host code the array's name is not a device address: its address on the
// current device comes from hipGetSymbolAddress, once per device, and only
// that pointer is handed to kernels.
// ---------------------------------------------------------------------------
namespace {

constexpr size_t kScratchBytes = MIKV_DECODE_STEP_NOALLOC_MAX_WORKSPACE;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices];

// Device address of the scratch array on the current device.
int scratch_on_current_device(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return set_error(MIKV_ERR_HIP, "mikv_decode_step_noalloc: hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return set_error(MIKV_ERR_UNSUPPORTED, "mikv_decode_step_noalloc: device %d beyond the %d supported", dev,
                     kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return set_error(MIKV_ERR_HIP, "mikv_decode_step_noalloc: hipGetSymbolAddress: %s", hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MIKV_OK;
}

}  // namespace

extern "C" int mikv_decode_step_noalloc(const mikv_cache *c, int32_t length, const uint16_t *q,
                                        const uint16_t *k_new, const uint16_t *v_new, const float *balance,
                                        float scale, float *out, float *probs_hi, float *probs_lo, int32_t k_heavy,
                                        int32_t window, int32_t flags, void *const *phase_events, void *stream) {
  int rc = validate_cache(c);
  if (rc) return rc;
  if (length < 1 || length > c->max_len)
    return set_error(length < 1 ? MIKV_ERR_INVALID_ARG : MIKV_ERR_CAPACITY,
                     "mikv_decode_step_noalloc: length %d outside [1, max_len]", length);
  const size_t need = mikv_decode_step_workspace_size(c, length);
  if (need > kScratchBytes)
    return set_error(MIKV_ERR_CAPACITY,
                     "mikv_decode_step_noalloc: the step needs %zu bytes of workspace, more than the %zu of the "
                     "library's scratch array (use mikv_decode_step with a workspace)",
                     need, kScratchBytes);
  void *ws = nullptr;
  rc = scratch_on_current_device(&ws);
  if (rc) return rc;
  return mikv_decode_step(c, length, q, k_new, v_new, balance, scale, out, probs_hi, probs_lo, k_heavy, window, flags,
                          ws, kScratchBytes, phase_events, stream);
}
