"""The C ABI on the CPU: libmikv.so loads, exports every symbol include/mikv.h
declares, and rejects bad arguments on the host before launching anything
(no GPU is needed for any of these calls)."""
import ctypes
import os
import re

import pytest
import torch  # noqa: F401  (loads the HIP runtime libmikv.so links against)

from paper_2402_18096_amd import mikv

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "mikv.h")

pytestmark = pytest.mark.skipif(not os.path.exists(mikv.LIB_PATH), reason="libmikv.so not built")


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(mikv_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    L = mikv.lib()
    names = declared_symbols()
    assert len(names) == 25
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(mikv.EXPORTS)


def _desc(**kw):
    d = dict(batch=1, q_heads=4, kv_heads=4, head_dim=128, group=32, hi_bits=16, lo_bits=2, cap_hi=8, cap_lo=32,
             max_len=16)
    d.update(kw)
    c = mikv.CacheDesc()
    for k, v in d.items():
        setattr(c, k, v)
    for f in ("hi_k", "hi_v", "hi_pos", "hi_acc", "n_hi", "lo_k", "lo_v", "lo_kp", "lo_vp", "lo_pos", "n_lo",
              "status"):
        setattr(c, f, 0x1000)  # never dereferenced: validation fails or nothing launches
    return c


def _call_attention(c, length=4, ws_bytes=1 << 30):
    L = mikv.lib()
    return L.mikv_decode_attention(ctypes.byref(c), length, ctypes.c_void_p(0x1000), None, 0.1,
                                   ctypes.c_void_p(0x1000), None, None, 0, ctypes.c_void_p(0x1000), ws_bytes, None)


@pytest.mark.parametrize("field,value,code", [
    ("head_dim", 64, 2), ("group", 48, 2), ("hi_bits", 2, 2), ("lo_bits", 5, 2),
    ("q_heads", 6, 1), ("kv_heads", 0, 1), ("cap_hi", 0, 1), ("batch", 0, 1),
])
def test_cache_validation_errors(field, value, code):
    c = _desc(**{field: value})
    assert _call_attention(c) == code
    assert mikv.lib().mikv_last_error()


def test_per_channel_keys_supported_formats():
    """Per-channel key blocks (Appendix C): 64 positions, fp16 importance pool,
    2/3/4-bit retained codes, one query head per KV head, block parameters
    given; anything else is refused before a launch."""
    assert _call_attention(_desc(key_block=32, lo_kb=0x1000)) == 2
    assert _call_attention(_desc(key_block=64, lo_kb=0x1000, q_heads=4, kv_heads=2)) == 2
    assert _call_attention(_desc(key_block=64, lo_kb=0x1000, hi_bits=8, hi_kp=0x1000, hi_vp=0x1000)) == 2
    assert _call_attention(_desc(key_block=64, lo_kb=0x1000, lo_bits=8)) == 2
    assert _call_attention(_desc(key_block=64)) == 1                     # lo_kb missing
    L = mikv.lib()
    p = ctypes.c_void_p(0x1000)
    c = _desc(key_block=64, lo_kb=0x1000, max_len=256, cap_lo=256)
    # the re-rank and the decode step need a window of at least one key block
    assert L.mikv_select_topk(ctypes.byref(c), 4, 1, 32, None, p, 1 << 20, None) == 1
    assert L.mikv_decode_step(ctypes.byref(c), 4, p, p, p, None, 0.1, p, p, None, 1, 32, 0, p, 1 << 30, None,
                              None) == 1


def test_int4_importance_pool_needs_two_bit_or_evicting_retained_pool():
    assert _call_attention(_desc(hi_bits=4, lo_bits=4)) == 2
    assert _call_attention(_desc(hi_bits=4, lo_bits=8)) == 2


def test_two_bit_gqa_pool_capacity_multiple_of_32():
    """2-bit retained pools shared by query heads store values in 32-slot
    tiles (validation only: every call in this file fails before any
    launch); with one query head per KV head any capacity is accepted by
    validation (the call then fails on the workspace)."""
    assert _call_attention(_desc(q_heads=8, kv_heads=4, cap_lo=48)) == 1
    assert "multiple of 32" in mikv.lib().mikv_last_error().decode()
    assert _call_attention(_desc(cap_lo=48), ws_bytes=16) == 3


def test_gqa_group_must_be_power_of_two_up_to_8():
    assert _call_attention(_desc(q_heads=12, kv_heads=4)) == 2   # G = 3
    assert _call_attention(_desc(q_heads=64, kv_heads=4)) == 2   # G = 16


def test_null_pointers_and_capacity():
    L = mikv.lib()
    c = _desc()
    c.n_hi = 0
    assert _call_attention(c) == 1
    c = _desc()
    assert _call_attention(c, length=17) == 3        # length > max_len
    assert _call_attention(c, ws_bytes=16) == 3      # workspace too small
    assert L.mikv_quantize_rows(None, 4, 128, None, 1, 2, 32, None, None, None) == 1
    assert L.mikv_quantize_rows(ctypes.c_void_p(1), 4, 128, None, 1, 5, 32, ctypes.c_void_p(1),
                                ctypes.c_void_p(1), None) == 2
    assert L.mikv_select_topk(ctypes.byref(_desc()), 4, -1, 0, None, ctypes.c_void_p(1), 1 << 20, None) == 1
    # the heavy list is limited to 8192 importance-pool slots per head
    assert L.mikv_select_topk(ctypes.byref(_desc(cap_hi=9000, max_len=9000)), 4, 1, 0, ctypes.c_void_p(1),
                              ctypes.c_void_p(1), 1 << 30, None) == 2
    assert L.mikv_select_prefill(None, 1, 4, 1, 1, None, None) == 1
    assert L.mikv_balance_channels(ctypes.c_void_p(1), ctypes.c_void_p(1), 1, 4, 4, 8, 64, ctypes.c_void_p(1),
                                   ctypes.c_void_p(1), 1 << 20, None) == 2
    # 16-byte alignment of the prefill rows (checked on the host, nothing launched)
    assert L.mikv_balance_channels(ctypes.c_void_p(0x1002), ctypes.c_void_p(0x1000), 1, 4, 4, 8, 128,
                                   ctypes.c_void_p(0x1000), ctypes.c_void_p(0x1000), 1 << 20, None) == 1
    # prefill importance: host-side validation, nothing launched
    assert L.mikv_prefill_importance(None, None, 1, 2, 2, 8, 128, ctypes.c_float(0.1), None, None, 0, None) == 1
    assert L.mikv_prefill_importance(qk_ := ctypes.c_void_p(0x1000), qk_, 1, 2, 2, 8, 64, ctypes.c_float(0.1),
                                     qk_, qk_, 1 << 20, None) == 2
    assert L.mikv_prefill_importance(qk_, qk_, 1, 6, 2, 8, 128, ctypes.c_float(0.1), qk_, qk_, 1 << 20, None) == 2
    assert L.mikv_prefill_importance(ctypes.c_void_p(0x1008), qk_, 1, 2, 2, 8, 128, ctypes.c_float(0.1), qk_, qk_,
                                     1 << 20, None) == 1
    assert L.mikv_prefill_importance(qk_, qk_, 1, 2, 2, 8, 128, ctypes.c_float(0.1), qk_, qk_, 8, None) == 3
    assert L.mikv_prefill_importance_workspace_size(1, 2, 8) == 2 * 8 * 8
    assert L.mikv_importance_update(ctypes.byref(_desc()), 4, None, None) == 1
    qk = ctypes.c_void_p(0x1000)
    assert L.mikv_quantize_kv(ctypes.byref(_desc()), qk, qk, None, 10, 8, None, None, None, 0, None) == 3


def test_workspace_sizes_are_consistent():
    L = mikv.lib()
    c = _desc(cap_hi=100, cap_lo=1024, max_len=1000)
    a = L.mikv_decode_workspace_size(ctypes.byref(c), 500)
    assert a >= 4 * 4 * 100   # at least the scores scratch of the importance pool
    assert L.mikv_select_workspace_size(ctypes.byref(c)) == 2 * 4 * 1 * 4 * 100
    assert L.mikv_balance_workspace_size(1, 4, 1000) > 0


def test_noalloc_step_rejects_a_workspace_beyond_its_scratch_array():
    """mikv_decode_step_noalloc refuses, on the host and before touching the
    device, a step whose workspace exceeds the library's scratch array."""
    c = _desc(batch=96, q_heads=40, kv_heads=40, hi_bits=8, cap_hi=1764, cap_lo=8504, max_len=8504)
    c.hi_kp = c.hi_vp = 0x1000
    L = mikv.lib()
    assert L.mikv_decode_step_workspace_size(ctypes.byref(c), 8400) > (64 << 20)
    p = ctypes.c_void_p(0x1000)
    rc = L.mikv_decode_step_noalloc(ctypes.byref(c), 8400, p, p, p, None, 0.1, p, None, None, 10, 64,
                                    mikv.ATTN_ACCUMULATE, None, None)
    assert rc == 3
    assert b"scratch" in L.mikv_last_error()


def test_heavy_budget():
    """The re-rank's budget: floor(ratio * length), less the window when it
    counts towards the ratio, never negative; invalid arguments give -1."""
    L = mikv.lib()
    assert L.mikv_heavy_budget(513, 1, 5, 32, 0) == 102          # top 20 % plus the last 32
    assert L.mikv_heavy_budget(4097, 1, 4, 64, 1) == 960
    assert L.mikv_heavy_budget(32769, 1, 10, 128, 1) == 3148
    assert L.mikv_heavy_budget(100, 1, 10, 128, 1) == 0
    assert L.mikv_heavy_budget(2 ** 31 - 1, 3, 4, 0, 0) == (2 ** 31 - 1) * 3 // 4   # no 32-bit overflow
    assert L.mikv_heavy_budget(10, 1, 0, 0, 0) == -1
    assert L.mikv_heavy_budget(-1, 1, 2, 0, 0) == -1


def test_stream_read_probe_validates_on_the_host():
    """The read-bandwidth probe refuses a NULL, misaligned or ragged buffer
    before launching anything."""
    L = mikv.lib()
    p = ctypes.c_void_p(0x1000)
    assert L.mikv_stream_read_probe(None, 1024, 0, 0, p, None) == 1
    assert L.mikv_stream_read_probe(ctypes.c_void_p(0x1008), 1024, 0, 0, p, None) == 1
    assert L.mikv_stream_read_probe(p, 1000, 0, 1, p, None) == 1
    assert L.mikv_stream_read_probe(p, 0, 0, 0, p, None) == 1
    assert b"16-byte" in L.mikv_last_error()


def test_probs_by_position_validates_on_the_host():
    """The position scatter refuses NULL buffers (a retained pool needs its
    probabilities), a non-positive length and one beyond max_len before
    launching anything."""
    L = mikv.lib()
    c = _desc()
    p = ctypes.c_void_p(0x1000)
    assert L.mikv_probs_by_position(ctypes.byref(c), 4, None, p, p, None) == 1
    assert L.mikv_probs_by_position(ctypes.byref(c), 4, p, None, p, None) == 1
    assert L.mikv_probs_by_position(ctypes.byref(c), 4, p, p, None, None) == 1
    assert L.mikv_probs_by_position(ctypes.byref(c), 0, p, p, p, None) == 1
    assert L.mikv_probs_by_position(ctypes.byref(c), c.max_len + 1, p, p, p, None) == 3


def test_importance_update_positions_validates_on_the_host():
    """The position-indexed importance update refuses NULL buffers, empty
    or ungrouped head counts, a negative length and one beyond max_len before
    launching anything; length 0 is a no-op that touches no memory."""
    L = mikv.lib()
    p = ctypes.c_void_p(0x1000)
    assert L.mikv_importance_update_positions(None, p, 1, 4, 4, 8, 16, None) == 1
    assert L.mikv_importance_update_positions(p, None, 1, 4, 4, 8, 16, None) == 1
    assert L.mikv_importance_update_positions(p, p, 0, 4, 4, 8, 16, None) == 1
    assert L.mikv_importance_update_positions(p, p, 1, 6, 4, 8, 16, None) == 1
    assert L.mikv_importance_update_positions(p, p, 1, 4, 4, -1, 16, None) == 1
    assert L.mikv_importance_update_positions(p, p, 1, 4, 4, 17, 16, None) == 3
    assert L.mikv_importance_update_positions(p, p, 1, 4, 4, 0, 16, None) == 0


@pytest.mark.parametrize("shape", [
    dict(batch=4, q_heads=32, kv_heads=32, cap_hi=3400, cap_lo=29760, max_len=33024),  # long_context
    dict(batch=16, q_heads=32, kv_heads=8, cap_hi=1700, cap_lo=14848, max_len=16512),  # mistral_7b
    dict(),
])
def test_workspace_size_does_not_depend_on_the_resident_share(shape):
    """The chunk split of an fp16 importance pool depends on whether the pool
    lies inside the resident share, but workspaces are sized from the split
    with the most chunks: a workspace sized under one share is large enough
    under any other (the size is the same)."""
    L = mikv.lib()
    c = _desc(**shape)
    length = c.max_len
    default = mikv.mikv_resident_bytes()
    try:
        sizes = []
        for share in (0, default, 1 << 40):
            mikv.mikv_set_resident_bytes(share)
            sizes.append((L.mikv_decode_workspace_size(ctypes.byref(c), length),
                          L.mikv_decode_step_workspace_size(ctypes.byref(c), length)))
    finally:
        mikv.mikv_set_resident_bytes(default)
    assert sizes[0][0] > 0 and sizes[0][1] > 0
    assert sizes[0] == sizes[1] == sizes[2]


def test_resident_budget_fits_the_last_level_cache():
    """The attention's plainly-read share of a cache defaults to a positive
    size below the 256 MB last-level cache it is meant to stay in, and can be
    set and restored; an out-of-range size is refused."""
    default = mikv.mikv_resident_bytes()
    assert 0 < default < 256 << 20
    try:
        mikv.mikv_set_resident_bytes(0)
        assert mikv.mikv_resident_bytes() == 0
        mikv.mikv_set_resident_bytes(1 << 40)
        assert mikv.mikv_resident_bytes() == 1 << 40
        assert mikv.lib().mikv_set_resident_bytes((1 << 62) + 1) == 1
        assert mikv.mikv_resident_bytes() == 1 << 40
    finally:
        mikv.mikv_set_resident_bytes(default)
    assert mikv.mikv_resident_bytes() == default
