"""Parity of the HIP path with the oracle on the GPU.

Every call goes through the C ABI (the ctypes binding).  Bit-exact: codes,
fp16 scale/zero, fp16 values, balancer, precision maps, importance scores.
Tolerance: attention output (2e-3 abs / 1e-3 rel) and probabilities.
Workloads are the five configurations at reduced sizes (several chunks per
pool with ragged tails), plus edge cases.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2402_18096_amd import mikv, workloads
from tests.parity import SCALE, Lockstep, SampledLockstep, compare_state, np16
from tests.parity import inputs as parity_inputs
from tests.quant_inputs import tie_rows

pytestmark = pytest.mark.gpu


def _dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda:0")


# -- raw quantizer ----------------------------------------------------------------

def _adversarial_rows(rng, rows, bits, group):
    x = rng.standard_normal((rows, 128)).astype(np.float32) * 2
    x[0::7] += 1000.3                          # offset-dominated groups (clamp)
    x[1::7] *= 1e-6                            # fp16-subnormal alpha and beta
    x[2::7] = np.round(x[2::7] * 2) / 2        # many exact ties
    x[3::7, :64] = 0.7                         # degenerate groups
    x[4::7] *= 500                             # large magnitudes
    x[5::7] = rng.integers(0, 256, (len(x[5::7]), 128))  # integer-valued
    x[6::7] = tie_rows(rng, len(x[6::7]), bits, group)   # exact quotient ties
    return x.astype(np.float16)


@pytest.mark.parametrize("bits", [2, 3, 4, 8])
@pytest.mark.parametrize("group", [32, 64, 128])
@pytest.mark.parametrize("balanced", [False, True])
def test_quantize_rows_bit_exact(bits, group, balanced):
    dev = _dev()
    rng = np.random.default_rng(bits * 1000 + group + balanced)
    rows = 4099
    x = _adversarial_rows(rng, rows, bits, group)
    bal = None
    rpb = 64
    if balanced:
        bal = (2.0 ** rng.uniform(-3, 3, ((rows + rpb - 1) // rpb, 128))).astype(np.float32)
    codes = torch.empty(rows, 128 * bits // 8, dtype=torch.uint8, device=dev)
    params = torch.empty(rows, 128 // group, 2, dtype=torch.int16, device=dev)
    mikv.mikv_quantize_rows(torch.from_numpy(x.view(np.int16)).to(dev).view(torch.float16), bits, group, codes,
                            params, None if bal is None else torch.from_numpy(bal).to(dev), rpb)
    torch.cuda.synchronize()
    xf = x.astype(np.float32)
    if bal is not None:
        xf = xf * np.repeat(bal, rpb, axis=0)[:rows]
    c_ref, a_ref, b_ref = oracle.quantize(xf, bits, group)
    np.testing.assert_array_equal(codes.cpu().numpy(), oracle.pack(c_ref, bits))
    p = params.cpu().numpy().view(np.uint16)
    np.testing.assert_array_equal(p[..., 0], a_ref)
    np.testing.assert_array_equal(p[..., 1], b_ref)


def test_quantize_rows_empty_is_noop():
    dev = _dev()
    codes = torch.zeros(1, 32, dtype=torch.uint8, device=dev)
    params = torch.zeros(1, 4, 2, dtype=torch.int16, device=dev)
    x = torch.zeros(0, 128, dtype=torch.float16, device=dev)
    mikv.lib()
    rc = mikv.lib().mikv_quantize_rows(mikv._ptr(x), 0, 128, None, 1, 2, 32, mikv._ptr(codes), mikv._ptr(params),
                                       mikv._stream())
    assert rc == 0


# -- balancer -------------------------------------------------------------------------

@pytest.mark.parametrize("G", [1, 4])
def test_balancer_bit_exact(G):
    dev = _dev()
    rng = np.random.default_rng(G)
    B, Hkv, T = 2, 3, 1500
    q = (rng.standard_normal((B, Hkv * G, T, 128)) * np.where(np.arange(128) % 17 == 0, 25, 1)).astype(np.float16)
    k = rng.standard_t(4, (B, Hkv, T, 128)).astype(np.float16)
    q[0, :G, :, 5] = 0      # zero query channel -> b = 1
    k[1, 2, :, 9] = 0       # zero key channel -> b = 1
    out = torch.empty(B, Hkv, 128, dtype=torch.float32, device=dev)
    tq = torch.from_numpy(q.view(np.int16)).to(dev).view(torch.float16)
    tk = torch.from_numpy(k.view(np.int16)).to(dev).view(torch.float16)
    mikv.mikv_balance_channels(tq, tk, out)
    torch.cuda.synchronize()
    ref = oracle.balancer(q.reshape(B, Hkv, G, T, 128), k)
    np.testing.assert_array_equal(out.cpu().numpy().view(np.uint32), ref.view(np.uint32))


# -- selection -------------------------------------------------------------------------

@pytest.mark.parametrize("L,k,W", [(1000, 150, 32), (5000, 900, 128), (300, 0, 10), (300, 500, 10), (64, 10, 100),
                                   (33000, 3000, 128)])
def test_select_prefill_matches_oracle(L, k, W):
    dev = _dev()
    rng = np.random.default_rng(L + k)
    H = 5
    sc = (rng.integers(0, 50, (H, L)) / 64).astype(np.float32)   # many exact ties
    sc[0] = rng.random(L).astype(np.float32)
    sc[1, ::3] = -0.0
    mask = torch.empty(H, L, dtype=torch.uint8, device=dev)
    mikv.mikv_select_prefill(torch.from_numpy(sc).to(dev), k, W, mask)
    torch.cuda.synchronize()
    got = mask.cpu().numpy().astype(bool)
    for h in range(H):
        np.testing.assert_array_equal(got[h], oracle.select(sc[h], None, L, k, W, initial=True))


# -- lock-step decode ------------------------------------------------------------------

SMALL = {
    "tiny": dict(),
    "llama2_7b": dict(batch=2, q_heads=3, kv_heads=3, context=1500),
    "llama2_13b": dict(batch=2, q_heads=3, kv_heads=3, context=1700),
    "mistral_7b": dict(batch=2, q_heads=8, kv_heads=2, context=2300),
    "long_context": dict(batch=1, q_heads=3, kv_heads=3, context=4100),
}


@pytest.mark.parametrize("name", workloads.WORKLOAD_ORDER)
@pytest.mark.parametrize("fused", [False, True])
def test_lockstep_decode(name, fused):
    _dev()
    wl = workloads.small_workload(name, **SMALL[name])
    steps = 6
    run = Lockstep(wl, steps, fused=fused)
    run.prefill()
    for t in range(steps):
        run.step(t)


def _pool_head_bytes(wl, cache, length):
    """Packed bytes of one head's importance and retained pools as the
    attention sizes its resident share (occupied span at most the capacity)."""
    def token_bytes(bits):
        return 2 * 128 * 2 if bits == 16 else 2 * (128 * bits // 8 + 4 * (128 // wl.group))
    lo_bits = wl.lo_bits or 2
    return (min(length, cache.cap_hi) * token_bytes(wl.hi_bits),
            (min(length, cache.cap_lo) * token_bytes(lo_bits)) if wl.lo_bits else 0)


@pytest.mark.gpu
@pytest.mark.parametrize("name,evict", [("long_context", False), ("mistral_7b", False), ("long_context", True)])
def test_probs_by_position_full_size(name, evict):
    """mikv_probs_by_position at a full benchmark shape (the largest grids,
    a ragged last block): every head's row equals the slot-ordered
    probabilities gathered by position on the host, bit for bit, and each
    query head's probabilities sum to 1 over the positions (Section 3.4)."""
    wl = workloads.WORKLOADS[name].with_(lo_bits=0) if evict else workloads.WORKLOADS[name]
    dev = _dev()
    dec = mikv.MikvDecoder(wl, max_len=wl.context + 2, device=dev, fused=False)
    k, v = workloads.prefill_kv(wl, dev)
    sc = workloads.initial_scores(wl, dev)
    qp = workloads.prefill_queries(wl, dev) if wl.balanced else None
    dec.prefill(k, v, sc, qp)
    del k, v, qp
    q, kn, vn = workloads.decode_inputs(wl, 2, dev)
    c = dec.cache
    G, NH = wl.group_size, wl.n_heads
    for t in range(2):
        snap = {}

        def after_attention():
            L = dec.length
            pos = torch.empty(c.batch * c.q_heads * L, dtype=torch.float32, device=dev)
            mikv.mikv_probs_by_position(c, L, dec.probs_hi, dec.probs_lo if c.lo_bits else None, pos)
            torch.cuda.synchronize()
            snap["pos"] = pos.cpu().numpy().reshape(NH, G, L)
            snap["ph"] = dec.probs_hi.cpu().numpy().reshape(NH, G, c.cap_hi)
            snap["pl"] = dec.probs_lo.cpu().numpy().reshape(NH, G, c.cap_lo)
            snap["maps"] = [x.cpu().numpy() for x in (c.n_hi, c.n_lo, c.hi_pos, c.lo_pos)]

        dec.step(q[t], kn[t], vn[t], after_attention=after_attention)
        torch.cuda.synchronize()
        L = dec.length
        n_hi, n_lo, hi_pos, lo_pos = snap["maps"]
        want = np.zeros((NH, G, L), np.float32)
        for h in range(NH):
            want[h][:, hi_pos[h, :n_hi[h]]] = snap["ph"][h, :, :n_hi[h]]
            if c.lo_bits:
                want[h][:, lo_pos[h, :n_lo[h]]] = snap["pl"][h, :, :n_lo[h]]
        if c.lo_bits:
            assert (n_hi + n_lo == L).all(), f"step {t}: the pools do not hold every position"
        np.testing.assert_array_equal(snap["pos"], want, err_msg=f"{name} step {t}: mikv_probs_by_position")
        sums = snap["pos"].astype(np.float64).sum(axis=2)
        np.testing.assert_allclose(sums, 1.0, atol=1e-4, err_msg=f"{name} step {t}: probabilities do not sum to 1")


@pytest.mark.gpu
@pytest.mark.parametrize("B,Hq,Hkv,L,Lmax", [(1, 1, 1, 1, 1), (2, 4, 4, 300, 333), (1, 8, 2, 257, 257),
                                             (3, 16, 2, 1000, 1500), (4, 32, 32, 32769, 32769),
                                             (16, 32, 8, 16385, 16386)])
def test_importance_update_positions_matches_oracle(B, Hq, Hkv, L, Lmax):
    """mikv_importance_update_positions against the oracle's H2O accumulation
    (Sections 3.1, 4.1), bit for bit, at tiny, ragged and full benchmark
    shapes (long_context, mistral_7b); positions at or past L keep their
    score."""
    _dev()
    G = Hq // Hkv
    g = torch.Generator().manual_seed(B * 1000003 + Hq * 1009 + L)
    probs = torch.rand(B, Hq, Lmax, generator=g) * 2e-3
    acc = torch.rand(B, Hkv, Lmax, generator=g) * 50.0
    acc_gpu = acc.cuda()
    mikv.mikv_importance_update_positions(acc_gpu, probs.cuda(), L)
    torch.cuda.synchronize()
    got = acc_gpu.cpu().numpy()
    a, p = acc.numpy(), probs.numpy()
    want = a.copy()
    for b in range(B):
        for k in range(Hkv):
            want[b, k, :L] = oracle.accumulate(a[b, k, :L], p[b, k * G:(k + 1) * G, :L])
    np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32))


@pytest.mark.gpu
@pytest.mark.parametrize("name,lo_bits", [("tiny", None), ("mistral_7b", None), ("llama2_13b", None),
                                          ("long_context", 0)])
def test_position_indexed_update_matches_the_cache_step(name, lo_bits):
    """The position-indexed calls compose to the cache's own update: scores
    scattered to positions, plus mikv_importance_update_positions over
    mikv_probs_by_position's output, give every importance-pool token the
    score the slot-ordered update and re-rank leave in its slot (bit for
    bit, over several steps; GQA, balanced and evicting caches)."""
    _dev()
    kw = dict(SMALL[name], **({} if lo_bits is None else {"lo_bits": lo_bits}))
    wl = workloads.small_workload(name, **kw)
    steps = 5
    k, v, sc, qp, q, kn, vn = parity_inputs(wl, steps)
    dec = mikv.MikvDecoder(wl, max_len=wl.context + steps, device="cuda", fused=False)
    dec.prefill(k.cuda(), v.cuda(), sc.cuda(), qp.cuda() if qp is not None else None)
    c = dec.cache
    B, Hq, Hkv, NH = wl.batch, wl.q_heads, wl.kv_heads, wl.n_heads
    for t in range(steps):
        snap = {}

        def after_attention():
            L = dec.length
            n_hi, hi_pos, acc = c.n_hi.cpu().numpy(), c.hi_pos.cpu().numpy(), c.hi_acc.cpu().numpy()
            acc_pos = np.zeros((NH, L), np.float32)
            for h in range(NH):
                acc_pos[h, hi_pos[h, :n_hi[h]]] = acc[h, :n_hi[h]]
            acc_t = torch.from_numpy(acc_pos).reshape(B, Hkv, L).cuda()
            probs = torch.empty(B, Hq, L, dtype=torch.float32, device="cuda")
            mikv.mikv_probs_by_position(c, L, dec.probs_hi, dec.probs_lo if c.lo_bits else None, probs)
            mikv.mikv_importance_update_positions(acc_t, probs, L)
            snap["acc_pos"] = acc_t.cpu().numpy().reshape(NH, L)

        dec.step(q[t].cuda(), kn[t].cuda(), vn[t].cuda(), after_attention=after_attention)
        torch.cuda.synchronize()
        n_hi, hi_pos, acc = c.n_hi.cpu().numpy(), c.hi_pos.cpu().numpy(), c.hi_acc.cpu().numpy()
        for h in range(NH):
            got = acc[h, :n_hi[h]]
            want = snap["acc_pos"][h, hi_pos[h, :n_hi[h]]]
            np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32),
                                          err_msg=f"{name} step {t} head {h}: scores")


@pytest.mark.parametrize("name", workloads.WORKLOAD_ORDER)
@pytest.mark.parametrize("share", ["none", "half_hi", "half_lo"])
def test_lockstep_streamed_rows(name, share):
    """The attention reads a resident share of the cache with plain loads and
    streams the rest with non-temporal loads (streamed fp16 and INT8
    importance rows 16 channels per lane, fp16 in spread pieces).  With
    nothing resident, with half the heads' importance pools resident, and
    with every importance pool and half the retained pools resident, the
    decode step matches the oracle as it does with the default share."""
    _dev()
    wl = workloads.small_workload(name, **SMALL[name])
    steps = 4
    default = mikv.mikv_resident_bytes()
    run = Lockstep(wl, steps, fused=True)
    try:
        hb, lb = _pool_head_bytes(wl, run.dec.cache, wl.context + steps)
        nh = wl.n_heads
        budget = {"none": 0, "half_hi": (nh // 2) * hb, "half_lo": nh * hb + (nh // 2) * lb}[share]
        mikv.mikv_set_resident_bytes(budget)
        run.prefill()
        for t in range(steps):
            run.step(t)
    finally:
        mikv.mikv_set_resident_bytes(default)


@pytest.mark.parametrize("name", workloads.WORKLOAD_ORDER)
def test_full_size_sampled_heads(name):
    """Every workload at its full size, in the benchmark's launch configuration
    (one native call per step, importance fused, probabilities of both pools
    emitted), with the oracle following the first, a middle and the last
    head: bit-exact state, attention and probabilities within tolerance."""
    _dev()
    wl = workloads.WORKLOADS[name]
    NH = wl.n_heads
    steps = min(wl.steps, 3)
    print(f"[full-size] {name}: {NH} heads, context {wl.context}, {steps} steps", flush=True)
    run = SampledLockstep(wl, steps, heads=[0, NH // 2 + 1 if NH > 2 else 0, NH - 1])
    run.prefill()
    for t in range(steps):
        run.step(t)
    del run
    torch.cuda.empty_cache()


def test_full_size_gqa8_sampled_heads():
    """Eight query heads per KV head (Llama-2-70b's grouping) at the Mistral
    cache size (16 x 32 query heads over 4 KV heads, 16384 tokens), in the
    benchmark's launch configuration, the oracle following three heads over
    four steps (both grid orders)."""
    _dev()
    wl = workloads.WORKLOADS["mistral_7b"].with_(kv_heads=4)
    NH = wl.n_heads
    print(f"[full-size] G=8: {NH} heads, context {wl.context}, 4 steps", flush=True)
    run = SampledLockstep(wl, 4, heads=[0, NH // 2 + 1, NH - 1])
    run.prefill()
    for t in range(4):
        run.step(t)
    del run
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["mistral_7b", "long_context"])
def test_full_size_whole_trajectory(name):
    """The GQA and long-context workloads at full size through their whole
    step count (128 and 256 decode steps) in the benchmark's launch
    configuration: attention output and probabilities of three sampled heads
    checked every step, the bit-exact state every 16th step and at the end."""
    _dev()
    wl = workloads.WORKLOADS[name]
    NH = wl.n_heads
    print(f"[trajectory] {name}: {NH} heads, context {wl.context}, {wl.steps} steps", flush=True)
    run = SampledLockstep(wl, wl.steps, heads=[0, NH // 2 + 1, NH - 1])
    run.prefill()
    worst = 0.0
    for t in range(wl.steps):
        worst = max(worst, run.step(t, check_state=t % 16 == 15 or t == wl.steps - 1))
    print(f"[trajectory] {name}: max |o - o_ref| over {wl.steps} steps {worst:.3e}", flush=True)
    del run
    torch.cuda.empty_cache()


def test_free_running_trajectory_report():
    """The oracle free-running beside the GPU (each ranks with its own
    probabilities) on the long_context workload for 32 steps: a report of
    precision-map differences and near-ties at the cut (not a gate), and,
    while the maps still agree, attention outputs within tolerance."""
    _dev()
    import json

    from tests.parity import O_ATOL
    from tests.trajectory import run_report
    wl = workloads.WORKLOADS["long_context"]
    rep = run_report(wl, 32, [0, wl.n_heads // 2 + 1, wl.n_heads - 1])
    summary = {k: v for k, v in rep.items() if k != "per_step"}
    print("[trajectory report] " + json.dumps(summary), flush=True)
    assert len(rep["per_step"]) == 32
    assert rep["max_abs_o_diff_before_divergence"] is None or rep["max_abs_o_diff_before_divergence"] < 2 * O_ATOL
    torch.cuda.empty_cache()


@pytest.mark.parametrize("scale", [20.0, 40.0])
def test_lockstep_gqa_outlier_margin(scale):
    """The Mistral shape with its 8 outlier channels at x20 and x40: the
    attention output must stay within a quarter of the allowed error (the
    matrix-core loop multiplies no code below 2^-18, where the matrix cores
    lose precision), every step bit-exact otherwise."""
    _dev()
    wl = workloads.small_workload("mistral_7b", batch=1, q_heads=8, kv_heads=2, context=16384, kv_outlier_scale=scale)
    run = Lockstep(wl, 6, fused=True)
    run.prefill()
    worst = 0.0
    for t in range(6):
        run.step(t)
        worst = max(worst, run.last_margin)
    print(f"[outlier x{scale:g}] largest share of the output allowance used: {worst:.3f}", flush=True)
    assert worst < 0.25


def test_lockstep_gqa8():
    """Eight query heads per KV head (Llama-2-70b's grouping)."""
    _dev()
    wl = workloads.small_workload("mistral_7b", batch=1, q_heads=16, kv_heads=2, context=900)
    run = Lockstep(wl, 4)
    run.prefill()
    for t in range(4):
        run.step(t)


def test_lockstep_window_outside_ratio_many_demotions():
    """Budget shrinking faster than one token per step (window counted on top
    of a ratio that the workload then lowers) exercises the radix-select path
    of the re-rank with several demotions per head."""
    _dev()
    wl = workloads.small_workload("long_context", batch=1, q_heads=2, kv_heads=2, context=2000, ratio_num=1,
                                  ratio_den=4)
    run = Lockstep(wl, 3)
    run.prefill()
    run.step(0)
    run.wl = wl.with_(ratio_den=6)            # budget drops from ~25 % to ~17 %
    run.dec.wl = run.wl
    run.step(1)
    run.step(2)


@pytest.mark.parametrize("ratio", [(0, 1), (1, 1)])
def test_lockstep_single_pool(ratio):
    """Ratio 0 and window 0 (every token retained at low precision: uniform
    RTN) and ratio 1 (every token at high precision)."""
    _dev()
    wl = workloads.small_workload("tiny", context=700, ratio_num=ratio[0], ratio_den=ratio[1],
                                  window=0 if ratio[0] == 0 else 32)
    run = Lockstep(wl, 3)
    run.prefill()
    for t in range(3):
        run.step(t)


@pytest.mark.parametrize("name", ["long_context", "llama2_13b", "mistral_7b"])
@pytest.mark.parametrize("fused", [False, True])
def test_lockstep_eviction(name, fused):
    """The eviction baseline (lo_bits 0, H2O): no retained pool, attention
    over the importance pool only, demoted tokens dropped -- fp16 and
    balanced INT8 importance pools, MHA and GQA."""
    _dev()
    wl = workloads.small_workload(name, **SMALL[name], lo_bits=0)
    run = Lockstep(wl, 4, fused=fused)
    run.prefill()
    for t in range(4):
        run.step(t)


def test_lockstep_eviction_with_int4_importance_cache():
    """Eviction with an INT4 importance cache (hi_bits 4, lo_bits 0), GQA."""
    _dev()
    wl = workloads.small_workload("mistral_7b", **SMALL["mistral_7b"], hi_bits=4, lo_bits=0)
    run = Lockstep(wl, 3, fused=True)
    run.prefill()
    for t in range(3):
        run.step(t)


def test_lockstep_eviction_many_demotions():
    """Several evictions per head and step (the radix-select path)."""
    _dev()
    wl = workloads.small_workload("long_context", batch=1, q_heads=2, kv_heads=2, context=2000, ratio_num=1,
                                  ratio_den=4, lo_bits=0)
    run = Lockstep(wl, 2)
    run.prefill()
    run.step(0)
    run.wl = wl.with_(ratio_den=6)
    run.dec.wl = run.wl
    run.step(1)


def test_full_size_eviction_sampled_heads():
    """The eviction baseline at the long_context size in the benchmark's
    launch configuration, the oracle following three heads."""
    _dev()
    wl = workloads.WORKLOADS["long_context"].with_(lo_bits=0)
    NH = wl.n_heads
    print(f"[full-size eviction] long_context: {NH} heads, context {wl.context}, 2 steps", flush=True)
    run = SampledLockstep(wl, 2, heads=[0, NH // 2 + 1, NH - 1])
    run.prefill()
    for t in range(2):
        run.step(t)
    del run
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name,shape", [
    ("tiny", dict(batch=1, q_heads=2, kv_heads=2, context=300)),          # ragged: not a multiple of 64
    ("mistral_7b", dict(batch=2, q_heads=8, kv_heads=2, context=200)),    # GQA 4, outliers x20
    ("llama2_13b", dict(batch=1, q_heads=2, kv_heads=2, context=1000)),   # Student-t keys
    ("long_context", dict(batch=1, q_heads=2, kv_heads=1, context=17)),   # GQA 2, one partial tile
    ("tiny", dict(batch=1, q_heads=1, kv_heads=1, context=1)),            # a single token
])
def test_prefill_importance_matches_oracle(name, shape):
    """H2O importance of the prompt (column sums of causal softmax attention,
    summed over the query heads of each KV head) against the fp64 oracle;
    fp32 sums in another order, so within 1e-4 relative, and the total mass
    G * T of every head.  The prefill selection over these scores then
    matches the oracle's selection over the same scores bit for bit."""
    dev = _dev()
    wl = workloads.small_workload(name, **shape)
    k, _ = workloads.prefill_kv(wl, dev)
    q = workloads.prefill_queries(wl, dev)
    got = torch.empty(wl.batch, wl.kv_heads, wl.context, dtype=torch.float32, device=dev)
    mikv.mikv_prefill_importance(q, k, got, SCALE)
    torch.cuda.synchronize()
    got = got.cpu().numpy().reshape(wl.n_heads, wl.context)
    G, T = wl.group_size, wl.context
    qn = np16(q).reshape(wl.n_heads, G, T, 128)
    kn = np16(k).reshape(wl.n_heads, T, 128)
    for h in range(wl.n_heads):
        ref = oracle.prefill_importance(qn[h], kn[h], SCALE)
        np.testing.assert_allclose(got[h], ref, rtol=1e-4, atol=1e-6, err_msg=f"{name} head {h}")
        assert abs(float(got[h].sum(dtype=np.float64)) - G * T) < 1e-4 * G * T
    if T > 40:
        kh, W = T // 5, 16
        mask = torch.empty(wl.batch, wl.kv_heads, T, dtype=torch.uint8, device=dev)
        mikv.mikv_select_prefill(torch.from_numpy(got).reshape(wl.batch, wl.kv_heads, T).to(dev), kh, W, mask)
        torch.cuda.synchronize()
        m = mask.cpu().numpy().reshape(wl.n_heads, T).astype(bool)
        for h in range(wl.n_heads):
            np.testing.assert_array_equal(m[h], oracle.select(got[h], None, T, kh, W, initial=True))


def test_lockstep_with_prompt_importance():
    """A decode run whose first selection uses the prompt's own H2O scores
    (mikv_prefill_importance) instead of seeded ones: the oracle takes the
    GPU's scores (the lockstep protocol) and every later step stays exact."""
    _dev()
    wl = workloads.small_workload("long_context", batch=1, q_heads=2, kv_heads=2, context=1500)
    run = Lockstep(wl, 3)
    q = workloads.prefill_queries(wl, "cuda")
    sc = torch.empty(wl.batch, wl.kv_heads, wl.context, dtype=torch.float32, device="cuda")
    mikv.mikv_prefill_importance(q, run.k.cuda(), sc, SCALE)
    torch.cuda.synchronize()
    ref = oracle.prefill_importance(np16(q).reshape(2, 1, wl.context, 128)[0], np16(run.k).reshape(2, wl.context, 128)[0],
                                    SCALE)
    np.testing.assert_allclose(sc.cpu().numpy().reshape(2, -1)[0], ref, rtol=1e-4, atol=1e-6)
    run.sc = sc.cpu()
    run.prefill()
    for t in range(3):
        run.step(t)


@pytest.mark.parametrize("name", ["long_context", "llama2_7b", "llama2_13b", "mistral_7b"])
@pytest.mark.parametrize("fused", [False, True])
def test_lockstep_int4_importance_cache(name, fused):
    """Table 3's INT4 importance cache over the 2-bit retained cache: MHA,
    balanced (13B shape) and GQA, demotions re-quantizing decoded INT4 rows."""
    _dev()
    wl = workloads.small_workload(name, **SMALL[name], hi_bits=4, lo_bits=2)
    run = Lockstep(wl, 4, fused=fused)
    run.prefill()
    for t in range(4):
        run.step(t)


def test_full_size_int4_importance_sampled_heads():
    """The INT4 importance cache at the long_context size in the benchmark's
    launch configuration, the oracle following three heads."""
    _dev()
    wl = workloads.WORKLOADS["long_context"].with_(hi_bits=4)
    NH = wl.n_heads
    print(f"[full-size int4 importance] long_context: {NH} heads, 2 steps", flush=True)
    run = SampledLockstep(wl, 2, heads=[0, NH // 2 + 1, NH - 1])
    run.prefill()
    for t in range(2):
        run.step(t)
    del run
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name,extra", [
    ("long_context", {}),
    ("llama2_7b", {}),                                    # INT8 importance pool, group 64
    ("llama2_13b", {}),                                   # balanced INT8 importance pool
    ("mistral_7b", dict(q_heads=4, kv_heads=2)),          # two query heads per KV head
    ("mistral_7b", {}),                                   # four (16-channel lanes, 48-bit code segments)
    ("mistral_7b", dict(batch=1, q_heads=16, kv_heads=2, context=900)),  # eight
])
@pytest.mark.parametrize("fused", [False, True])
def test_lockstep_int3_retained_cache(name, extra, fused):
    """The INT3 retained cache of Tables 1 and 2 (codes straddling bytes):
    prefill, attention, demotion and re-quantization, bit-exact state."""
    _dev()
    wl = workloads.small_workload(name, **{**SMALL[name], **extra}, lo_bits=3)
    run = Lockstep(wl, 4, fused=fused)
    run.prefill()
    for t in range(4):
        run.step(t)


@pytest.mark.parametrize("lo_bits,extra", [
    (4, dict(q_heads=4, kv_heads=2)),                         # two query heads per KV head
    (4, {}),                                                  # four (16-channel lanes)
    (4, dict(batch=1, q_heads=16, kv_heads=2, context=900)),  # eight (8-channel lanes)
    (8, dict(q_heads=2, kv_heads=2)),                         # one
    (8, {}),                                                  # four
    (8, dict(batch=1, q_heads=16, kv_heads=2, context=900)),  # eight (8-channel lanes)
])
@pytest.mark.parametrize("fused", [False, True])
def test_lockstep_int4_int8_retained_cache(lo_bits, extra, fused):
    """4- and 8-bit retained caches (the wider low precisions of Tables 1-3)
    at the Mistral shape with one to eight query heads per KV head: prefill,
    attention, demotion and re-quantization, bit-exact state every step."""
    _dev()
    wl = workloads.small_workload("mistral_7b", **{**SMALL["mistral_7b"], **extra}, lo_bits=lo_bits)
    run = Lockstep(wl, 4, fused=fused)
    run.prefill()
    for t in range(4):
        run.step(t)


@pytest.mark.parametrize("name", ["long_context", "mistral_7b"])
def test_full_size_int3_retained_sampled_heads(name):
    """The INT3 retained cache at the long_context and Mistral (GQA, four
    query heads per KV head) sizes in the benchmark's launch configuration,
    the oracle following three heads."""
    _dev()
    wl = workloads.WORKLOADS[name].with_(lo_bits=3)
    NH = wl.n_heads
    print(f"[full-size int3 retained] {name}: {NH} heads, 2 steps", flush=True)
    run = SampledLockstep(wl, 2, heads=[0, NH // 2 + 1, NH - 1])
    run.prefill()
    for t in range(2):
        run.step(t)
    del run
    torch.cuda.empty_cache()


# -- per-channel key quantization (Appendix C) -------------------------------------

def _channel_keys(name, **kw):
    """A workload with the retained keys quantized per channel over 64-position
    blocks: fp16 importance cache, no balancer (the per-channel quantizer
    replaces it, Table 6)."""
    return workloads.small_workload(name, **kw).with_(hi_bits=16, balanced=False, key_block=64)


@pytest.mark.parametrize("name,shape", [
    ("long_context", dict(batch=1, q_heads=3, kv_heads=3, context=4090)),     # a block completes at step 5
    ("llama2_13b", dict(batch=2, q_heads=3, kv_heads=3, context=1725)),       # Student-t keys, INT2 g32, W 64
    ("long_context", dict(batch=1, q_heads=2, kv_heads=2, context=2000, lo_bits=3)),
    ("llama2_7b", dict(batch=1, q_heads=2, kv_heads=2, context=1500, lo_bits=4)),
])
@pytest.mark.parametrize("fused", [False, True])
def test_lockstep_per_channel_keys(name, shape, fused):
    """Per-channel key blocks through prefill (parameters from the prompt),
    decode steps (a block completing from the importance pool), attention
    over per-channel retained keys and per-token demotion codes: bit-exact
    state including every block's parameters, o and p within tolerance."""
    _dev()
    wl = _channel_keys(name, **shape)
    run = Lockstep(wl, 8, fused=fused)
    run.prefill()
    for t in range(8):
        run.step(t)


def test_lockstep_per_channel_keys_demote_from_decoded_blocks():
    """Long enough (W = 64, 100 steps) that blocks completed during decoding
    lose tokens to the retained pool, whose keys then take those blocks'
    parameters; the many-demotion path runs on the last steps."""
    _dev()
    wl = _channel_keys("long_context", batch=1, q_heads=2, kv_heads=2, context=700, window=64)
    run = Lockstep(wl, 100, fused=True)
    run.prefill()
    for t in range(100):
        if t == 96:
            run.wl = wl.with_(ratio_den=14)        # budget drops: several demotions per head
            run.dec.wl = run.wl
        run.step(t, check_state=t % 8 == 7 or t >= 96)
    nb = run.orc.kb_done.sum(1)
    assert (nb == (700 + 100) // 64).all()


@pytest.mark.parametrize("name", ["long_context", "llama2_13b"])
def test_full_size_per_channel_keys_sampled_heads(name):
    """Per-channel keys at the full long_context and 13B shapes in the
    benchmark's launch configuration, the oracle following three heads."""
    _dev()
    wl = workloads.WORKLOADS[name].with_(hi_bits=16, balanced=False, key_block=64)
    NH = wl.n_heads
    print(f"[full-size per-channel keys] {name}: {NH} heads, 2 steps", flush=True)
    run = SampledLockstep(wl, 2, heads=[0, NH // 2 + 1, NH - 1])
    run.prefill()
    for t in range(2):
        run.step(t)
    del run
    torch.cuda.empty_cache()


def test_capacity_overflow_sets_status_without_writing_out_of_bounds():
    dev = _dev()
    c = mikv.MikvCache(1, 2, 2, 32, 16, 2, cap_hi=4, cap_lo=32, max_len=64, device=dev)
    k = torch.randn(1, 2, 6, 128, device=dev).half()
    mikv.mikv_quantize_kv(c, k, k.clone(), 0)    # six tokens into a 4-slot importance pool
    torch.cuda.synchronize()
    assert int(c.status.item()) & mikv.DEVERR_HI_FULL
    assert c.n_hi.cpu().tolist() == [4, 4]


@pytest.mark.parametrize("name", ["llama2_13b", "mistral_7b"])
@pytest.mark.parametrize("fused", [False, True])
def test_native_step_matches_call_sequence(name, fused):
    """mikv_decode_step (one native call) leaves exactly the state that the
    four separate calls leave, and the same outputs: the attention output and
    both probability buffers compared slot for slot over their whole
    capacity, so a slot that only one of them writes (e.g. a retained-pool
    slot filled by this step's demotion) shows up."""
    _dev()
    wl = workloads.small_workload(name, **SMALL[name])
    steps = 5
    run = Lockstep(wl, steps, fused=fused)
    run.prefill()
    other = mikv.MikvDecoder(wl, max_len=wl.context + steps, device="cuda", fused=fused)
    other.prefill(run.k.cuda(), run.v.cuda(), run.sc.cuda(), run.qp.cuda() if run.qp is not None else None)
    # stale contents that a stray write would overwrite
    for d in (run.dec, other):
        d.probs_hi.fill_(-1.0)
        d.probs_lo.fill_(-1.0)
    for t in range(steps):
        n_lo0 = other.cache.n_lo.clone()
        run.step(t)
        other.step_native(run.q[t].cuda(), run.kn[t].cuda(), run.vn[t].cuda())
        torch.cuda.synchronize()
        compare_state(other.cache, run.orc, tag=f"native step {t}")
        np.testing.assert_array_equal(other.out.cpu().numpy(), run.dec.out.cpu().numpy())
        np.testing.assert_array_equal(other.probs_hi.cpu().numpy().view(np.uint32),
                                      run.dec.probs_hi.cpu().numpy().view(np.uint32), err_msg=f"step {t}: probs_hi")
        np.testing.assert_array_equal(other.probs_lo.cpu().numpy().view(np.uint32),
                                      run.dec.probs_lo.cpu().numpy().view(np.uint32), err_msg=f"step {t}: probs_lo")
        # the slots this step's demotions filled were not attended: untouched
        n_lo1 = other.cache.n_lo.cpu().numpy()
        pl = other.probs_lo.cpu().numpy().reshape(wl.n_heads, wl.group_size, -1)
        for h, (a, b) in enumerate(zip(n_lo0.cpu().numpy(), n_lo1)):
            assert (pl[h, :, a:b] == -1.0).all(), f"step {t} head {h}: retained slots {a}..{b} written"



def test_fp16_pool_rounding_edge_cases():
    """fp16 importance-pool rows are f16(f32(k) * b) with round to nearest
    even (Eq. 3): balance factors chosen so that every product is an exact
    tie (1 + 2^-11), lands in the fp16 subnormal range (2^-16), overflows
    (2^12) or rounds generically; both the many-token placement and the
    one-token append store bit-for-bit what the oracle stores."""
    dev = _dev()
    B, H, n, n1 = 1, 2, 40, 8
    c = mikv.MikvCache(B, H, H, 32, 16, 2, cap_hi=64, cap_lo=64, max_len=64, device=dev)
    rng = np.random.default_rng(5)
    k = (rng.standard_normal((B, H, n + n1, 128)) * 8).astype(np.float16)
    # m * 2^-24 (m < 2048: fp16 subnormals and the smallest normals) halved:
    # an exact tie whenever m is odd, rounding to the even neighbour
    m = rng.integers(1, 2048, (B, H, n + n1, 16)) * rng.choice([-1, 1], (B, H, n + n1, 16))
    k[..., :16] = (m * 2.0 ** -24).astype(np.float16)
    k[..., 16:24] = rng.choice([-1.0, 1.0], (B, H, n + n1, 8)).astype(np.float16)  # 1 + 2^-11: a tie
    b = np.empty((B, H, 128), np.float32)
    b[..., :16] = np.float32(0.5)
    b[..., 16:32] = np.float32(1 + 2.0 ** -11)
    b[..., 32:64] = np.float32(2.0 ** -16)
    b[..., 64:96] = rng.uniform(0.3, 3.7, (B, H, 32)).astype(np.float32)
    b[..., 96:] = np.float32(2.0 ** 12)
    kt = torch.from_numpy(k.view(np.int16)).view(torch.float16).to(dev)
    bt = torch.from_numpy(b).to(dev)
    mikv.mikv_quantize_kv(c, kt[:, :, :n].contiguous(), kt[:, :, :n].contiguous(), 0, balance=bt)
    for j in range(n1):
        kj = kt[:, :, n + j:n + j + 1].contiguous()
        mikv.mikv_quantize_kv(c, kj, kj.clone(), n + j, balance=bt)
    torch.cuda.synchronize()
    assert int(c.status.item()) == 0
    got = c.hi_k.cpu().numpy().view(np.uint16)[:, : n + n1]
    want = oracle.f16_bits(oracle.balance_keys(k.reshape(H, n + n1, 128), b.reshape(H, 1, 128)))
    assert np.isinf(want.view(np.float16)).any() and ((want & 0x7c00) == 0).any()
    exact = k.reshape(H, n + n1, 128)[..., :16].astype(np.float64) * 0.5
    assert (exact != want[..., :16].view(np.float16).astype(np.float64)).any()   # ties were rounded
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("backwards", [False, True])
def test_stream_read_probe_reads_every_chunk(backwards):
    """The read probe (a measurement utility) folds every 16-byte word it
    reads per thread and writes the sink only when a thread's fold hits its
    sentinel: a buffer of zeros with the sentinel planted at one word makes
    the sink appear exactly when that word was read.  Planted at the first,
    a middle and the last word, in the plainly read (resident) part and in
    the streamed part, over a ragged size, in both chunk orders."""
    dev = _dev()
    sentinel = 0x9E3779B9
    n16 = 3 * 8192 * 1024 // 16 + 37  # about 1500 chunks, the last one ragged
    for resident in (0, n16 * 8):
        for word in (0, n16 // 2 + 5, n16 - 1):
            buf = torch.zeros(n16 * 4, dtype=torch.int32, device=dev)
            buf[4 * word + 1] = int(np.uint32(sentinel).view(np.int32))
            sink = torch.zeros(1, dtype=torch.int32, device=dev)
            mikv.mikv_stream_read_probe(buf, sink, resident, backwards)
            torch.cuda.synchronize()
            assert int(sink.item()) & 0xFFFFFFFF == sentinel, (resident, word)
