"""Seeded synthetic workloads for the MiKV decode path.

This module only *draws inputs*: shapes, value distributions and the seeded
importance scores.  It holds none of the method's arithmetic (no quantizer,
no attention, no budget rule), so the CPU oracle and the HIP path can both
take their inputs from here without sharing any computation.

The paper's experiments ran real Llama-2 / Mistral checkpoints on public
benchmarks (Section 4.1); neither is available, so the inputs below stand in
for them.  They take the per-layer attention shapes of those models (head
dimension 128; Llama-2-7b 32 heads, 13b 40 heads, Mistral-7b 32 query heads
over 8 KV heads) and the outlier structure Section 3.2 describes: a few fixed
outlier channels in keys and queries, duplicated by RoPE, i.e. appearing as
channel pairs (c, c + 64).

All tensors are generated with ``torch.Generator`` on the requested device so
that the large workloads can be drawn directly in GPU memory; small cases are
drawn on the CPU.  The same seed on the same device kind gives the same
values.  fp16 tensors are produced by drawing fp32 and rounding to fp16.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import torch

HEAD_DIM = 128


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic workload (a single attention layer's shape, whole batch).

    ``ratio_num / ratio_den`` is the importance ratio (fraction of tokens kept
    at high precision), ``window`` the recent window, and ``window_in_ratio``
    says whether the window is counted inside that ratio (the workload text
    "25 % of tokens (top-k plus a 64-token window)") or added on top of it
    ("the top 20 % plus the last 32 tokens").
    """

    name: str
    batch: int
    q_heads: int
    kv_heads: int
    context: int          # tokens in the cache before the first decode step
    steps: int            # decode steps the workload runs
    hi_bits: int          # 16 = fp16 importance cache, 8 = INT8
    lo_bits: int          # retained-cache precision (2 or 4; 0 = evict, the H2O baseline)
    group: int            # quantization group size (channels)
    ratio_num: int
    ratio_den: int
    window: int
    window_in_ratio: bool
    balanced: bool        # apply the key/query channel balancer
    k_dist: str           # "normal" or "student_t4"
    kv_outlier_channels: int
    kv_outlier_scale: float
    q_outlier_channels: int
    q_outlier_scale: float
    seed: int
    head_dim: int = HEAD_DIM
    key_block: int = 0    # 0: per-token keys; 64: retained keys per channel over 64-position blocks

    @property
    def group_size(self) -> int:
        return self.q_heads // self.kv_heads

    @property
    def n_heads(self) -> int:
        """Independent (batch, KV head) pairs."""
        return self.batch * self.kv_heads

    def with_(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# The five workloads.  Windows marked "reading" are not fixed by the workload
# text and are chosen as stated in the design notes.
WORKLOADS = {
    # 1 sequence, 4 heads, 512-token context, one decode step; fp16 + INT2 g32;
    # top 20 % by seeded score plus the last 32 tokens kept fp16.
    "tiny": Workload("tiny", 1, 4, 4, 512, 1, 16, 2, 32, 1, 5, 32, False, False,
                     "normal", 4, 10.0, 0, 1.0, 20240228 + 1),
    # Llama-2-7B layer: 8 x 32 heads, 4096 context, INT8 + INT4 g64, 25 %
    # (window of 64 inside the ratio), 64 decode steps.
    "llama2_7b": Workload("llama2_7b", 8, 32, 32, 4096, 64, 8, 4, 64, 1, 4, 64, True, False,
                          "normal", 4, 10.0, 0, 1.0, 20240228 + 2),
    # Llama-2-13B layer: 32 x 40 heads, 8192 context, INT8 + INT2 g32, 20 %,
    # balanced keys/queries, Student-t(4) keys, 32 decode steps (window: reading).
    "llama2_13b": Workload("llama2_13b", 32, 40, 40, 8192, 32, 8, 2, 32, 1, 5, 64, True, True,
                           "student_t4", 0, 1.0, 4, 10.0, 20240228 + 3),
    # Mistral-7B GQA layer: 16 sequences, 32 query heads over 8 KV heads, 16384
    # context, fp16 + INT2 g32, 10 %, 8 outlier channels x20, 128 decode steps
    # (window: reading).
    "mistral_7b": Workload("mistral_7b", 16, 32, 8, 16384, 128, 16, 2, 32, 1, 10, 128, True, False,
                           "normal", 8, 20.0, 0, 1.0, 20240228 + 4),
    # Long context: 4 x 32 heads, 32768-token prefill, fp16 + INT2 g32, 10 %
    # with a 128-token window inside the ratio, 256 decode steps.
    "long_context": Workload("long_context", 4, 32, 32, 32768, 256, 16, 2, 32, 1, 10, 128, True, False,
                             "normal", 4, 10.0, 0, 1.0, 20240228 + 5),
}

WORKLOAD_ORDER = ["tiny", "llama2_7b", "llama2_13b", "mistral_7b", "long_context"]

# Sub-stream identifiers: each kind of input gets its own generator so that,
# e.g., drawing more decode steps never changes the prefill cache.
_STREAM_OUTLIER, _STREAM_K, _STREAM_V, _STREAM_QP, _STREAM_SCORE, _STREAM_Q, _STREAM_KNEW, _STREAM_VNEW = range(8)


def _gen(wl: Workload, stream: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(wl.seed * 16 + stream)
    return g


def outlier_channels(wl: Workload, n_channels: int) -> torch.Tensor:
    """Per KV head, ``n_channels`` fixed outlier channels as RoPE pairs (c, c+64).

    Returns a bool mask [kv_heads, head_dim] (CPU).  The same channels are used
    for every sequence and token, as Section 3.2 observes.
    """
    mask = torch.zeros(wl.kv_heads, wl.head_dim, dtype=torch.bool)
    if n_channels == 0:
        return mask
    assert n_channels % 2 == 0
    g = _gen(wl, _STREAM_OUTLIER, "cpu")
    half = wl.head_dim // 2
    for h in range(wl.kv_heads):
        base = torch.randperm(half, generator=g)[: n_channels // 2]
        mask[h, base] = True
        mask[h, base + half] = True
    return mask


def _draw(shape, dist: str, g: torch.Generator, device) -> torch.Tensor:
    if dist == "normal":
        return torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if dist == "student_t4":
        # t(4) = z / sqrt(chi2_4 / 4), chi2_4 the sum of four squared normals.
        z = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
        chi = torch.zeros(shape, device=device, dtype=torch.float32)
        for _ in range(4):
            e = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
            chi.addcmul_(e, e)
        return z / torch.sqrt(chi / 4.0)
    raise ValueError(dist)


def _scale_channels(x: torch.Tensor, mask: torch.Tensor, scale: float) -> torch.Tensor:
    """x: [..., H, T, D] fp32; mask [H, D]."""
    if not bool(mask.any()):
        return x
    f = torch.where(mask, torch.tensor(scale), torch.tensor(1.0)).to(x.device)
    return x * f[:, None, :]


def prefill_kv(wl: Workload, device="cpu", batches: Optional[range] = None):
    """Prefill keys and values, fp16 [B, Hkv, context, D].

    Drawn batch element by batch element (one generator per stream, consumed in
    order), so ``batches`` can restrict the output to a sub-range without
    changing the values of the elements that are returned.
    """
    batches = range(wl.batch) if batches is None else batches
    gk, gv = _gen(wl, _STREAM_K, device), _gen(wl, _STREAM_V, device)
    mask = outlier_channels(wl, wl.kv_outlier_channels)
    shape = (wl.kv_heads, wl.context, wl.head_dim)
    ks, vs = [], []
    for b in range(max(batches) + 1):
        k = _draw(shape, wl.k_dist, gk, device)
        v = _draw(shape, "normal", gv, device)
        if b in batches:
            ks.append(_scale_channels(k, mask, wl.kv_outlier_scale).half())
            vs.append(_scale_channels(v, mask, wl.kv_outlier_scale).half())
    return torch.stack(ks), torch.stack(vs)


def prefill_queries(wl: Workload, device="cpu", batches: Optional[range] = None):
    """Prefill-prompt queries fp16 [B, Hq, context, D] (used by the balancer)."""
    batches = range(wl.batch) if batches is None else batches
    g = _gen(wl, _STREAM_QP, device)
    kvmask = outlier_channels(wl.with_(seed=wl.seed + 7), wl.q_outlier_channels)
    qmask = kvmask.repeat_interleave(wl.group_size, dim=0)
    out = []
    for b in range(max(batches) + 1):
        q = torch.randn((wl.q_heads, wl.context, wl.head_dim), generator=g, device=device)
        if b in batches:
            out.append(_scale_channels(q, qmask, wl.q_outlier_scale).half())
    return torch.stack(out)


def initial_scores(wl: Workload, device="cpu") -> torch.Tensor:
    """Seeded importance scores for the prefill tokens, fp32 [B, Hkv, context].

    Zipf(1.1) over token positions: score_j proportional to (pi(j)+1)^-1.1 for
    a seeded permutation pi per (sequence, KV head), normalised so each head's
    scores sum to the context length (as if every prompt query had given one
    unit of attention).
    """
    g = _gen(wl, _STREAM_SCORE, "cpu")
    n = wl.context
    ranks = torch.arange(1, n + 1, dtype=torch.float64)
    base = ranks.pow(-1.1)
    base = base * (n / base.sum())
    out = torch.empty(wl.batch, wl.kv_heads, n, dtype=torch.float32)
    for b in range(wl.batch):
        for h in range(wl.kv_heads):
            perm = torch.randperm(n, generator=g)
            out[b, h] = base[perm].float()
    return out.to(device)


def decode_inputs(wl: Workload, n_steps: int, device="cpu"):
    """Per-step decode inputs, all steps at once.

    Returns (q [S, B, Hq, D], k_new [S, B, Hkv, D], v_new [S, B, Hkv, D]),
    fp16.  New keys/values follow the cache's own distribution; queries are
    N(0,1) with the workload's query outlier channels.
    """
    gq, gk, gv = (_gen(wl, s, device) for s in (_STREAM_Q, _STREAM_KNEW, _STREAM_VNEW))
    kvmask = outlier_channels(wl, wl.kv_outlier_channels)
    qmask = outlier_channels(wl.with_(seed=wl.seed + 7), wl.q_outlier_channels).repeat_interleave(
        wl.group_size, dim=0)
    shape_q = (n_steps * wl.batch, wl.q_heads, 1, wl.head_dim)
    shape_kv = (n_steps * wl.batch, wl.kv_heads, 1, wl.head_dim)
    q = _scale_channels(torch.randn(shape_q, generator=gq, device=device), qmask, wl.q_outlier_scale)
    k = _scale_channels(_draw(shape_kv, wl.k_dist, gk, device), kvmask, wl.kv_outlier_scale)
    v = _scale_channels(_draw(shape_kv, "normal", gv, device), kvmask, wl.kv_outlier_scale)
    r = lambda x, h: x.reshape(n_steps, wl.batch, h, wl.head_dim).half()
    return r(q, wl.q_heads), r(k, wl.kv_heads), r(v, wl.kv_heads)


def small_workload(name: str, **overrides) -> Workload:
    """A workload with the named configuration's precisions and distributions
    but smaller shapes (for parity tests the oracle finishes in seconds)."""
    return WORKLOADS[name].with_(**overrides)
