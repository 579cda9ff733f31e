// Host-side plumbing of the C ABI: thread-local error messages, launch
// checks and validation of the cache descriptor.
#include <string>

#include "mikv_internal.h"

namespace mikv {

static thread_local std::string g_last_error;

int set_error(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

int check_launch(const char *what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return set_error(MIKV_ERR_HIP, "%s: launch failed: %s", what, hipGetErrorString(e));
  return MIKV_OK;
}

int validate_cache(const mikv_cache *c) {
  if (!c) return set_error(MIKV_ERR_INVALID_ARG, "cache descriptor is NULL");
  if (c->batch < 1 || c->q_heads < 1 || c->kv_heads < 1)
    return set_error(MIKV_ERR_INVALID_ARG, "batch/q_heads/kv_heads must be >= 1");
  if (c->q_heads % c->kv_heads != 0)
    return set_error(MIKV_ERR_INVALID_ARG, "q_heads (%d) not a multiple of kv_heads (%d)", c->q_heads,
                     c->kv_heads);
  int G = c->q_heads / c->kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8)
    return set_error(MIKV_ERR_UNSUPPORTED, "query heads per KV head must be 1, 2, 4 or 8 (got %d)", G);
  if (c->head_dim != kHeadDim)
    return set_error(MIKV_ERR_UNSUPPORTED, "head_dim must be 128 (got %d)", c->head_dim);
  if (c->group != 32 && c->group != 64 && c->group != 128)
    return set_error(MIKV_ERR_UNSUPPORTED, "group must be 32, 64 or 128 (got %d)", c->group);
  if (c->hi_bits != 16 && c->hi_bits != 8 && c->hi_bits != 4)
    return set_error(MIKV_ERR_UNSUPPORTED, "hi_bits must be 16, 8 or 4 (got %d)", c->hi_bits);
  if (c->hi_bits == 4 && c->lo_bits != 2 && c->lo_bits != 0)
    return set_error(MIKV_ERR_UNSUPPORTED, "an INT4 importance pool needs lo_bits 2 or 0 (got %d)", c->lo_bits);
  if (c->lo_bits != 0 && c->lo_bits != 2 && c->lo_bits != 3 && c->lo_bits != 4 && c->lo_bits != 8)
    return set_error(MIKV_ERR_UNSUPPORTED, "lo_bits must be 0, 2, 3, 4 or 8 (got %d)", c->lo_bits);
  if (c->cap_hi < 1 || (!evicting(c) && c->cap_lo < 1) || c->max_len < 1)
    return set_error(MIKV_ERR_INVALID_ARG, "cap_hi, cap_lo (unless lo_bits is 0) and max_len must be >= 1");
  if (int2_values_tiled(c->lo_bits, c->q_heads, c->kv_heads) && c->cap_lo % 32 != 0)
    return set_error(MIKV_ERR_INVALID_ARG,
                     "cap_lo must be a multiple of 32 for a 2-bit retained pool shared by query heads (got %d)",
                     c->cap_lo);
  if (c->key_block != 0 && c->key_block != kKeyBlock)
    return set_error(MIKV_ERR_UNSUPPORTED, "key_block must be 0 or %d (got %d)", kKeyBlock, c->key_block);
  if (c->key_block) {
    if (c->hi_bits != 16 || (c->lo_bits != 2 && c->lo_bits != 3 && c->lo_bits != 4) || G != 1)
      return set_error(MIKV_ERR_UNSUPPORTED,
                       "per-channel keys need hi_bits 16, lo_bits 2, 3 or 4 and one query head per KV head");
    if (!c->lo_kb) return set_error(MIKV_ERR_INVALID_ARG, "key_block %d needs lo_kb", c->key_block);
  }
  if (!c->hi_k || !c->hi_v || !c->hi_pos || !c->hi_acc || !c->n_hi || !c->n_lo || !c->status ||
      (!evicting(c) && (!c->lo_k || !c->lo_v || (!c->lo_kp && !c->key_block) || !c->lo_vp || !c->lo_pos)))
    return set_error(MIKV_ERR_INVALID_ARG, "a required cache pointer is NULL");
  if (c->hi_bits != 16 && (!c->hi_kp || !c->hi_vp))
    return set_error(MIKV_ERR_INVALID_ARG, "hi_kp/hi_vp are required for an INT8 or INT4 importance pool");
  return MIKV_OK;
}

}  // namespace mikv

extern "C" const char *mikv_last_error(void) { return mikv::g_last_error.c_str(); }
