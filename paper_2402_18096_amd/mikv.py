"""ctypes binding of libmikv.so (C ABI in include/mikv.h).

Argument marshalling only: every function below forwards torch tensors'
device pointers to the C entry point of the same name, on torch's current
HIP stream, and raises :class:`MikvError` on a non-zero status.  All compute
happens in the HIP kernels.  There is no fallback: if the library has not
been built the first call raises.

:class:`MikvCache` allocates the caller-owned buffers of one cache (torch
tensors, so torch's allocator provides the device memory) and
:class:`MikvDecoder` strings the calls into the prefill and decode-step
sequence of the method.
"""
from __future__ import annotations

import ctypes
import math
import os
from ctypes import c_float, c_int32, c_int64, c_size_t, c_void_p
from typing import Optional

import torch

# MIKV_LIB selects another build of the library (e.g. to compare builds).
LIB_PATH = os.environ.get("MIKV_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmikv.so")
HEAD_DIM = 128
ATTN_ACCUMULATE = 1
DEVERR_HI_FULL = 1
DEVERR_LO_FULL = 2
DEVERR_KEY_BLOCK = 4


class MikvError(RuntimeError):
    pass


class CacheDesc(ctypes.Structure):
    """Mirror of ``struct mikv_cache``."""
    _fields_ = [(n, c_int32) for n in ("batch", "q_heads", "kv_heads", "head_dim", "group", "hi_bits",
                                       "lo_bits", "cap_hi", "cap_lo", "max_len")] + \
               [(n, c_void_p) for n in ("hi_k", "hi_v", "hi_kp", "hi_vp", "hi_pos", "hi_acc", "n_hi",
                                        "lo_k", "lo_v", "lo_kp", "lo_vp", "lo_pos", "n_lo", "map", "status")] + \
               [("key_block", c_int32), ("lo_kb", c_void_p)]


_LIB = None
_PC = ctypes.POINTER(CacheDesc)

_SIGS = {
    "mikv_last_error": (ctypes.c_char_p, []),
    "mikv_balance_workspace_size": (c_size_t, [c_int32, c_int32, c_int32]),
    "mikv_balance_channels": (c_int32, [c_void_p, c_void_p, c_int32, c_int32, c_int32, c_int32, c_int32,
                                        c_void_p, c_void_p, c_size_t, c_void_p]),
    "mikv_prefill_importance_workspace_size": (c_size_t, [c_int32, c_int32, c_int32]),
    "mikv_prefill_importance": (c_int32, [c_void_p, c_void_p, c_int32, c_int32, c_int32, c_int32, c_int32, c_float,
                                          c_void_p, c_void_p, c_size_t, c_void_p]),
    "mikv_quantize_rows": (c_int32, [c_void_p, c_int64, c_int32, c_void_p, c_int32, c_int32, c_int32,
                                     c_void_p, c_void_p, c_void_p]),
    "mikv_quantize_workspace_size": (c_size_t, [_PC, c_int32]),
    "mikv_quantize_kv": (c_int32, [_PC, c_void_p, c_void_p, c_void_p, c_int32, c_int32, c_void_p, c_void_p,
                                   c_void_p, c_size_t, c_void_p]),
    "mikv_decode_workspace_size": (c_size_t, [_PC, c_int32]),
    "mikv_importance_update": (c_int32, [_PC, c_int32, c_void_p, c_void_p]),
    "mikv_select_workspace_size": (c_size_t, [_PC]),
    "mikv_select_topk": (c_int32, [_PC, c_int32, c_int32, c_int32, c_void_p, c_void_p, c_size_t, c_void_p]),
    "mikv_heavy_budget": (c_int32, [c_int32, c_int32, c_int32, c_int32, c_int32]),
    "mikv_select_prefill": (c_int32, [c_void_p, c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p]),
}
for _n in ("mikv_decode_attention", "mikv_decode_attention_partial", "mikv_decode_attention_finalize"):
    _SIGS[_n] = (c_int32, [_PC, c_int32, c_void_p, c_void_p, c_float, c_void_p, c_void_p, c_void_p, c_int32,
                           c_void_p, c_size_t, c_void_p])

_SIGS["mikv_decode_step_workspace_size"] = (c_size_t, [_PC, c_int32])
_SIGS["mikv_decode_step"] = (c_int32, [_PC, c_int32, c_void_p, c_void_p, c_void_p, c_void_p, c_float, c_void_p,
                                       c_void_p, c_void_p, c_int32, c_int32, c_int32, c_void_p, c_size_t, c_void_p,
                                       c_void_p])

_SIGS["mikv_decode_step_noalloc"] = (c_int32, [_PC, c_int32, c_void_p, c_void_p, c_void_p, c_void_p, c_float,
                                               c_void_p, c_void_p, c_void_p, c_int32, c_int32, c_int32, c_void_p,
                                               c_void_p])

_SIGS["mikv_stream_read_probe"] = (c_int32, [c_void_p, c_size_t, c_size_t, c_int32, c_void_p, c_void_p])
_SIGS["mikv_resident_bytes"] = (c_size_t, [])
_SIGS["mikv_probs_by_position"] = (c_int32, [c_void_p, c_int32, c_void_p, c_void_p, c_void_p, c_void_p])
_SIGS["mikv_importance_update_positions"] = (c_int32, [c_void_p, c_void_p, c_int32, c_int32, c_int32, c_int32,
                                                       c_int32, c_void_p])
_SIGS["mikv_set_resident_bytes"] = (c_int32, [c_size_t])

EXPORTS = tuple(_SIGS)


def lib():
    """Load libmikv.so (after torch, so both share torch's HIP runtime)."""
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise MikvError(f"{LIB_PATH} is missing: build it with `python -m paper_2402_18096_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype, f.argtypes = res, args
        _LIB = L
    return _LIB


def _check(rc: int, name: str):
    if rc != 0:
        raise MikvError(f"{name} failed with status {rc}: {lib().mikv_last_error().decode()}")


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise MikvError("tensors passed to libmikv must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _require(t: torch.Tensor, dtype, shape=None, name="tensor"):
    if t.dtype != dtype:
        raise MikvError(f"{name}: expected {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise MikvError(f"{name}: must be a device tensor")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise MikvError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")


def _workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 16), dtype=torch.uint8, device=device)


# -- cache ------------------------------------------------------------------------

class MikvCache:
    """Device buffers of one mixed-precision cache (see ``struct mikv_cache``).

    A 2-bit retained pool shared by several query heads keeps its value codes
    in tiles of 32 slots, so its capacity is rounded up to a multiple of 32.
    ``lo_bits=0`` is the eviction baseline: no retained pool is allocated
    (capacity 0) and tokens that leave the importance pool are dropped."""

    def __init__(self, batch: int, q_heads: int, kv_heads: int, group: int, hi_bits: int, lo_bits: int,
                 cap_hi: int, cap_lo: int, max_len: int, device="cuda", with_map: bool = True, key_block: int = 0):
        self.values_tiled = lo_bits == 2 and q_heads >= 2 * kv_heads
        if lo_bits == 0:
            cap_lo = 0
        if self.values_tiled:
            cap_lo = (cap_lo + 31) // 32 * 32
        self.batch, self.q_heads, self.kv_heads = batch, q_heads, kv_heads
        self.group, self.hi_bits, self.lo_bits = group, hi_bits, lo_bits
        self.cap_hi, self.cap_lo, self.max_len = cap_hi, cap_lo, max_len
        self.device = torch.device(device)
        NH, D, ng = batch * kv_heads, HEAD_DIM, HEAD_DIM // group
        z = lambda *s, dt: torch.zeros(*s, dtype=dt, device=self.device)
        if hi_bits == 16:
            self.hi_k, self.hi_v = z(NH, cap_hi, D, dt=torch.float16), z(NH, cap_hi, D, dt=torch.float16)
            self.hi_kp = self.hi_vp = None
        else:
            hrow = D * hi_bits // 8  # INT8 or INT4 codes, packed
            self.hi_k, self.hi_v = z(NH, cap_hi, hrow, dt=torch.uint8), z(NH, cap_hi, hrow, dt=torch.uint8)
            self.hi_kp, self.hi_vp = z(NH, cap_hi, ng, 2, dt=torch.int16), z(NH, cap_hi, ng, 2, dt=torch.int16)
        self.hi_pos = z(NH, cap_hi, dt=torch.int32)
        self.hi_acc = z(NH, cap_hi, dt=torch.float32)
        self.n_hi = z(NH, dt=torch.int32)
        row = D * lo_bits // 8
        self.lo_k, self.lo_v = z(NH, cap_lo, row, dt=torch.uint8), z(NH, cap_lo, row, dt=torch.uint8)
        # per-token key parameters, or (key_block 64) per-block, per-channel ones
        self.key_block = key_block
        self.lo_kp = None if key_block else z(NH, cap_lo, ng, 2, dt=torch.int16)
        self.lo_vp = z(NH, cap_lo, ng, 2, dt=torch.int16)
        self.lo_kb = z(NH, max(1, max_len // key_block), D, 2, dt=torch.int16) if key_block else None
        self.lo_pos = z(NH, cap_lo, dt=torch.int32)
        self.n_lo = z(NH, dt=torch.int32)
        self.map = z(NH, max_len, dt=torch.uint8) if with_map else None
        self.status = z(1, dt=torch.int32)
        p = lambda t: None if t is None else t.data_ptr()
        self.desc = CacheDesc(batch, q_heads, kv_heads, D, group, hi_bits, lo_bits, cap_hi, cap_lo, max_len,
                              p(self.hi_k), p(self.hi_v), p(self.hi_kp), p(self.hi_vp), p(self.hi_pos),
                              p(self.hi_acc), p(self.n_hi), p(self.lo_k), p(self.lo_v), p(self.lo_kp),
                              p(self.lo_vp), p(self.lo_pos), p(self.n_lo), p(self.map), p(self.status),
                              key_block, p(self.lo_kb))

    @property
    def n_heads(self) -> int:
        return self.batch * self.kv_heads

    def ref(self):
        return ctypes.byref(self.desc)

    def packed_bytes(self, length: int, n_hi: int) -> int:
        """Packed K/V bytes of the cache (codes + fp16 alpha/beta + fp16 values)
        when every head holds `length` tokens, `n_hi` of them high precision."""
        def tb(bits):
            if bits == 0:  # evicted tokens are not stored
                return 0
            if bits == 16:
                return 4 * HEAD_DIM
            codes = HEAD_DIM * bits // 8
            if self.key_block:  # key: codes + its share of the block's per-channel (alpha, beta)
                return codes + 4 * HEAD_DIM // self.key_block + codes + 4 * (HEAD_DIM // self.group)
            return 2 * (codes + 4 * (HEAD_DIM // self.group))
        return self.n_heads * (n_hi * tb(self.hi_bits) + (length - n_hi) * tb(self.lo_bits))


# -- entry points -----------------------------------------------------------------

def mikv_balance_channels(q_prefill: torch.Tensor, k_prefill: torch.Tensor, balance: torch.Tensor,
                          workspace: Optional[torch.Tensor] = None):
    B, Hq, T, D = q_prefill.shape
    Hkv = k_prefill.shape[1]
    _require(q_prefill, torch.float16, name="q_prefill")
    _require(k_prefill, torch.float16, (B, Hkv, T, D), "k_prefill")
    _require(balance, torch.float32, (B, Hkv, D), "balance")
    L = lib()
    nbytes = L.mikv_balance_workspace_size(B, Hkv, T)
    ws = workspace if workspace is not None else _workspace(nbytes, q_prefill.device)
    _check(L.mikv_balance_channels(_ptr(q_prefill), _ptr(k_prefill), B, Hq, Hkv, T, D, _ptr(balance), _ptr(ws),
                                   ws.numel(), _stream()), "mikv_balance_channels")


def mikv_prefill_importance(q_prefill: torch.Tensor, k_prefill: torch.Tensor, scores: torch.Tensor,
                            scale: Optional[float] = None, workspace: Optional[torch.Tensor] = None):
    """H2O importance of the prompt tokens: column sums of causal softmax
    attention over the prompt, summed over each KV head's query heads.
    q_prefill fp16 [B, Hq, T, 128], k_prefill fp16 [B, Hkv, T, 128] -> scores fp32 [B, Hkv, T]."""
    B, Hq, T, D = q_prefill.shape
    Hkv = k_prefill.shape[1]
    _require(q_prefill, torch.float16, name="q_prefill")
    _require(k_prefill, torch.float16, (B, Hkv, T, D), "k_prefill")
    _require(scores, torch.float32, (B, Hkv, T), "scores")
    L = lib()
    nbytes = L.mikv_prefill_importance_workspace_size(B, Hq, T)
    ws = workspace if workspace is not None else _workspace(nbytes, q_prefill.device)
    scale = 1.0 / math.sqrt(D) if scale is None else scale
    _check(L.mikv_prefill_importance(_ptr(q_prefill), _ptr(k_prefill), B, Hq, Hkv, T, D, scale, _ptr(scores),
                                     _ptr(ws), ws.numel(), _stream()), "mikv_prefill_importance")


def mikv_quantize_rows(x: torch.Tensor, bits: int, group: int, codes: torch.Tensor, params: torch.Tensor,
                       balance: Optional[torch.Tensor] = None, rows_per_balance: int = 1):
    rows = x.numel() // HEAD_DIM
    _require(x, torch.float16, name="x")
    _require(codes, torch.uint8, name="codes")
    if codes.numel() != rows * HEAD_DIM * bits // 8 or params.numel() != rows * (HEAD_DIM // group) * 2:
        raise MikvError("mikv_quantize_rows: codes/params size mismatch")
    _check(lib().mikv_quantize_rows(_ptr(x), rows, HEAD_DIM, _ptr(balance), rows_per_balance, bits, group,
                                    _ptr(codes), _ptr(params), _stream()), "mikv_quantize_rows")


def mikv_quantize_kv(cache: MikvCache, k: torch.Tensor, v: torch.Tensor, pos0: int,
                     balance: Optional[torch.Tensor] = None, hi_mask: Optional[torch.Tensor] = None,
                     score_init: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None):
    n = k.shape[2]
    shp = (cache.batch, cache.kv_heads, n, HEAD_DIM)
    _require(k, torch.float16, shp, "k")
    _require(v, torch.float16, shp, "v")
    if hi_mask is not None:
        _require(hi_mask, torch.uint8, shp[:3], "hi_mask")
    if score_init is not None:
        _require(score_init, torch.float32, shp[:3], "score_init")
    L = lib()
    ws = workspace
    if ws is None and hi_mask is not None:
        ws = _workspace(L.mikv_quantize_workspace_size(cache.ref(), n), k.device)
    _check(L.mikv_quantize_kv(cache.ref(), _ptr(k), _ptr(v), _ptr(balance), pos0, n, _ptr(hi_mask),
                              _ptr(score_init), _ptr(ws), 0 if ws is None else ws.numel(), _stream()),
           "mikv_quantize_kv")


def _attention(name, cache, length, q, out, probs_hi, probs_lo, balance, scale, flags, workspace):
    _require(q, torch.float16, (cache.batch, cache.q_heads, HEAD_DIM), "q")
    _require(out, torch.float32, (cache.batch, cache.q_heads, HEAD_DIM), "out")
    if probs_hi is not None:
        _require(probs_hi, torch.float32, (cache.batch, cache.q_heads, cache.cap_hi), "probs_hi")
    if probs_lo is not None:
        _require(probs_lo, torch.float32, (cache.batch, cache.q_heads, cache.cap_lo), "probs_lo")
    L = lib()
    ws = workspace if workspace is not None else _workspace(L.mikv_decode_workspace_size(cache.ref(), length),
                                                            q.device)
    scale = 1.0 / math.sqrt(HEAD_DIM) if scale is None else scale
    _check(getattr(L, name)(cache.ref(), length, _ptr(q), _ptr(balance), scale, _ptr(out), _ptr(probs_hi),
                            _ptr(probs_lo), flags, _ptr(ws), ws.numel(), _stream()), name)


def mikv_decode_attention(cache, length, q, out, probs_hi=None, probs_lo=None, balance=None, scale=None,
                          flags=0, workspace=None):
    _attention("mikv_decode_attention", cache, length, q, out, probs_hi, probs_lo, balance, scale, flags, workspace)


def mikv_decode_attention_partial(cache, length, q, out, probs_hi=None, probs_lo=None, balance=None, scale=None,
                                  flags=0, workspace=None):
    _attention("mikv_decode_attention_partial", cache, length, q, out, probs_hi, probs_lo, balance, scale, flags,
               workspace)


def mikv_decode_attention_finalize(cache, length, q, out, probs_hi=None, probs_lo=None, balance=None, scale=None,
                                   flags=0, workspace=None):
    _attention("mikv_decode_attention_finalize", cache, length, q, out, probs_hi, probs_lo, balance, scale, flags,
               workspace)


def mikv_decode_workspace_size(cache: MikvCache, length: int) -> int:
    return int(lib().mikv_decode_workspace_size(cache.ref(), length))


def mikv_importance_update(cache: MikvCache, length: int, probs_hi: torch.Tensor):
    _require(probs_hi, torch.float32, (cache.batch, cache.q_heads, cache.cap_hi), "probs_hi")
    _check(lib().mikv_importance_update(cache.ref(), length, _ptr(probs_hi), _stream()), "mikv_importance_update")


def mikv_select_topk(cache: MikvCache, length: int, k_heavy: int, window: int,
                     workspace: Optional[torch.Tensor] = None, heavy_idx: Optional[torch.Tensor] = None):
    L = lib()
    if heavy_idx is not None:
        _require(heavy_idx, torch.int32, (cache.batch, cache.kv_heads, k_heavy), "heavy_idx")
    ws = workspace if workspace is not None else _workspace(L.mikv_select_workspace_size(cache.ref()),
                                                            cache.device)
    _check(L.mikv_select_topk(cache.ref(), length, k_heavy, window, _ptr(heavy_idx), _ptr(ws), ws.numel(),
                              _stream()), "mikv_select_topk")


def mikv_select_prefill(scores: torch.Tensor, k_heavy: int, window: int, hi_mask: torch.Tensor):
    H, T = scores.shape[0], scores.shape[-1]
    _require(scores, torch.float32, name="scores")
    _require(hi_mask, torch.uint8, tuple(scores.shape), "hi_mask")
    _check(lib().mikv_select_prefill(_ptr(scores), scores.numel() // T, T, k_heavy, window, _ptr(hi_mask),
                                     _stream()), "mikv_select_prefill")


def mikv_stream_read_probe(buf: torch.Tensor, sink: torch.Tensor, resident_bytes: int = 0, backwards: bool = False):
    """Stream the bytes of `buf` (contiguous, 16-byte aligned device tensor)
    through the library's read-bandwidth probe, the leading `resident_bytes`
    with plain loads and the rest non-temporally, front to back or back to
    front; `sink` is one int32."""
    if not buf.is_contiguous():
        raise MikvError("mikv_stream_read_probe: buf must be contiguous")
    if resident_bytes < 0:
        raise MikvError("mikv_stream_read_probe: resident_bytes must be >= 0")
    _require(sink, torch.int32, name="sink")
    _check(lib().mikv_stream_read_probe(_ptr(buf), buf.numel() * buf.element_size(), int(resident_bytes),
                                        int(bool(backwards)), _ptr(sink), _stream()), "mikv_stream_read_probe")


def mikv_probs_by_position(cache: MikvCache, length: int, probs_hi: torch.Tensor, probs_lo, probs: torch.Tensor):
    """Scatter the slot-ordered probabilities of both pools into ``probs``
    fp32 [B, Hq, length] by token position (0 for dropped tokens)."""
    _require(probs_hi, torch.float32, name="probs_hi")
    _require(probs, torch.float32, name="probs")
    if probs_lo is not None:
        _require(probs_lo, torch.float32, name="probs_lo")
    if probs.numel() != cache.batch * cache.q_heads * length:
        raise MikvError("mikv_probs_by_position: probs must hold B * Hq * length floats")
    _check(lib().mikv_probs_by_position(cache.ref(), length, _ptr(probs_hi), _ptr(probs_lo), _ptr(probs),
                                        _stream()), "mikv_probs_by_position")


def mikv_importance_update_positions(acc: torch.Tensor, probs: torch.Tensor, length: int):
    """H2O accumulation over position-indexed rows: acc fp32 [B, Hkv, Lmax]
    += the group sums of probs fp32 [B, Hq, Lmax] at positions < length."""
    _require(acc, torch.float32, name="acc")
    _require(probs, torch.float32, name="probs")
    if acc.dim() != 3 or probs.dim() != 3 or acc.shape[0] != probs.shape[0] or acc.shape[2] != probs.shape[2]:
        raise MikvError("mikv_importance_update_positions: acc [B, Hkv, Lmax] and probs [B, Hq, Lmax] expected")
    B, Hkv, Lmax = acc.shape
    _check(lib().mikv_importance_update_positions(_ptr(acc), _ptr(probs), B, probs.shape[1], Hkv, length, Lmax,
                                                  _stream()), "mikv_importance_update_positions")


def mikv_resident_bytes() -> int:
    """Bytes of a cache the attention reads with plain loads each step (the
    rest it streams non-temporally)."""
    return int(lib().mikv_resident_bytes())


def mikv_set_resident_bytes(nbytes: int) -> None:
    """Set that share (process-wide, from the next launch on)."""
    if nbytes < 0:
        raise MikvError("mikv_set_resident_bytes: bytes must be >= 0")
    _check(lib().mikv_set_resident_bytes(int(nbytes)), "mikv_set_resident_bytes")


def mikv_decode_step(cache: MikvCache, length: int, q, k_new, v_new, out, k_heavy: int, window: int,
                     probs_hi=None, probs_lo=None, balance=None, scale=None, flags=0, workspace=None,
                     phase_events=None):
    """Whole decode step in one native call; ``phase_events`` is an optional
    sequence of 6 ``torch.cuda.Event`` (already recorded once, so they exist)."""
    _require(q, torch.float16, (cache.batch, cache.q_heads, HEAD_DIM), "q")
    _require(k_new, torch.float16, (cache.batch, cache.kv_heads, HEAD_DIM), "k_new")
    _require(v_new, torch.float16, (cache.batch, cache.kv_heads, HEAD_DIM), "v_new")
    _require(out, torch.float32, (cache.batch, cache.q_heads, HEAD_DIM), "out")
    L = lib()
    ws = workspace if workspace is not None else _workspace(L.mikv_decode_step_workspace_size(cache.ref(), length),
                                                            q.device)
    ev = None
    if phase_events is not None:
        ev = (c_void_p * 6)(*[e.cuda_event if e is not None else None for e in phase_events])
    scale = 1.0 / math.sqrt(HEAD_DIM) if scale is None else scale
    _check(L.mikv_decode_step(cache.ref(), length, _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(balance), scale,
                              _ptr(out), _ptr(probs_hi), _ptr(probs_lo), k_heavy, window, flags, _ptr(ws),
                              ws.numel(), ev, _stream()), "mikv_decode_step")


def mikv_decode_step_noalloc(cache: MikvCache, length: int, q, k_new, v_new, out, k_heavy: int, window: int,
                             probs_hi=None, probs_lo=None, balance=None, scale=None, flags=0, phase_events=None):
    """mikv_decode_step with the library's own device scratch array as its
    workspace: nothing is allocated, here or in the library."""
    _require(q, torch.float16, (cache.batch, cache.q_heads, HEAD_DIM), "q")
    _require(k_new, torch.float16, (cache.batch, cache.kv_heads, HEAD_DIM), "k_new")
    _require(v_new, torch.float16, (cache.batch, cache.kv_heads, HEAD_DIM), "v_new")
    _require(out, torch.float32, (cache.batch, cache.q_heads, HEAD_DIM), "out")
    ev = None
    if phase_events is not None:
        ev = (c_void_p * 6)(*[e.cuda_event if e is not None else None for e in phase_events])
    scale = 1.0 / math.sqrt(HEAD_DIM) if scale is None else scale
    _check(lib().mikv_decode_step_noalloc(cache.ref(), length, _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(balance),
                                          scale, _ptr(out), _ptr(probs_hi), _ptr(probs_lo), k_heavy, window, flags,
                                          ev, _stream()), "mikv_decode_step_noalloc")


# -- the method's step sequence ---------------------------------------------------

def heavy_budget(length: int, ratio_num: int, ratio_den: int, window: int, window_in_ratio: bool) -> int:
    """High-precision tokens outside the window for a cache of `length`
    (mikv_heavy_budget: floor(ratio * length), less the window when it counts
    towards the ratio)."""
    k = lib().mikv_heavy_budget(length, ratio_num, ratio_den, window, int(bool(window_in_ratio)))
    if k < 0:
        raise MikvError(f"mikv_heavy_budget: invalid arguments ({length}, {ratio_num}/{ratio_den}, {window})")
    return int(k)


class MikvDecoder:
    """Prefill and decode steps of one workload on one GPU.

    A decode step is: append the new token (mikv_quantize_kv), attention
    (mikv_decode_attention, probabilities of both pools emitted), importance
    update (mikv_importance_update, or fused into attention with
    ``fused=True``) and re-rank/demote (mikv_select_topk).
    """

    def __init__(self, wl, max_len: Optional[int] = None, device="cuda", fused: bool = False,
                 cap_slack: int = 64):
        self.wl, self.device, self.fused = wl, torch.device(device), fused
        self.max_len = max_len or (wl.context + wl.steps)
        cap_hi = min(self.max_len, heavy_budget(self.max_len, wl.ratio_num, wl.ratio_den, wl.window,
                                                wl.window_in_ratio) + wl.window + cap_slack)
        self.cache = MikvCache(wl.batch, wl.q_heads, wl.kv_heads, wl.group, wl.hi_bits, wl.lo_bits, cap_hi,
                               self.max_len, self.max_len, device, key_block=wl.key_block)
        c = self.cache
        self.length = 0
        self.balance = None
        self.heavy_idx = None
        B, Hq = wl.batch, wl.q_heads
        self.out = torch.zeros(B, Hq, HEAD_DIM, dtype=torch.float32, device=self.device)
        self.probs_hi = torch.zeros(B, Hq, c.cap_hi, dtype=torch.float32, device=self.device)
        self.probs_lo = torch.zeros(B, Hq, c.cap_lo, dtype=torch.float32, device=self.device)
        L = lib()
        ws = max(L.mikv_decode_workspace_size(c.ref(), n) for n in range(1, self.max_len + 1))
        self.attn_ws = _workspace(ws, self.device)
        self.sel_ws = _workspace(L.mikv_select_workspace_size(c.ref()), self.device)
        sws = max(L.mikv_decode_step_workspace_size(c.ref(), n) for n in range(1, self.max_len + 1))
        self.step_ws = _workspace(sws, self.device)

    def k_heavy(self, length: int) -> int:
        wl = self.wl
        return heavy_budget(length, wl.ratio_num, wl.ratio_den, wl.window, wl.window_in_ratio)

    def prefill(self, k: torch.Tensor, v: torch.Tensor, scores: Optional[torch.Tensor],
                q_prefill: Optional[torch.Tensor] = None):
        """k, v fp16 [B, Hkv, T, D]; scores fp32 [B, Hkv, T], or None to use the
        prompt's own H2O importance (mikv_prefill_importance, which needs
        q_prefill); q_prefill fp16 [B, Hq, T, D] (also when the workload
        balances keys and queries)."""
        wl, T = self.wl, k.shape[2]
        if scores is None:
            if q_prefill is None:
                raise MikvError("prefill: the prompt's importance needs q_prefill")
            scores = torch.empty(wl.batch, wl.kv_heads, T, dtype=torch.float32, device=self.device)
            mikv_prefill_importance(q_prefill, k, scores)
        if wl.balanced:
            self.balance = torch.empty(wl.batch, wl.kv_heads, HEAD_DIM, dtype=torch.float32, device=self.device)
            mikv_balance_channels(q_prefill, k, self.balance)
        mask = torch.empty(wl.batch, wl.kv_heads, T, dtype=torch.uint8, device=self.device)
        mikv_select_prefill(scores, self.k_heavy(T), wl.window, mask)
        mikv_quantize_kv(self.cache, k, v, 0, self.balance, mask, scores)
        self.length = T

    def step(self, q: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor, emit_lo: bool = True,
             after_attention=None, emit_heavy: bool = False):
        """One decode step; q fp16 [B, Hq, D], k_new/v_new fp16 [B, Hkv, D].
        ``after_attention`` (optional) is called between attention and the
        importance update, e.g. to snapshot the slot-ordered probabilities;
        with ``emit_heavy`` the re-rank also writes the sorted heavy-token
        list to ``self.heavy_idx`` [B, Hkv, k_heavy]."""
        c = self.cache
        mikv_quantize_kv(c, k_new.unsqueeze(2), v_new.unsqueeze(2), self.length, self.balance)
        self.length += 1
        L = self.length
        flags = ATTN_ACCUMULATE if self.fused else 0
        mikv_decode_attention(c, L, q, self.out, self.probs_hi, self.probs_lo if emit_lo else None,
                              self.balance, None, flags, self.attn_ws)
        if after_attention is not None:
            after_attention()
        if not self.fused:
            mikv_importance_update(c, L, self.probs_hi)
        kh = self.k_heavy(L)
        heavy = None
        if emit_heavy:
            heavy = torch.empty(c.batch, c.kv_heads, kh, dtype=torch.int32, device=self.device)
        mikv_select_topk(c, L, kh, self.wl.window, self.sel_ws, heavy)
        self.heavy_idx = heavy
        return self.out

    def step_native(self, q: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor, emit_lo: bool = True,
                    phase_events=None):
        """The same decode step as :meth:`step`, launched by one native call."""
        self.length += 1
        L = self.length
        mikv_decode_step(self.cache, L, q, k_new, v_new, self.out, self.k_heavy(L), self.wl.window, self.probs_hi,
                         self.probs_lo if emit_lo else None, self.balance, None,
                         ATTN_ACCUMULATE if self.fused else 0, self.step_ws, phase_events)
        return self.out
