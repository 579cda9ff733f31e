"""mikv_decode_step_noalloc: the decode step with the library's own device
scratch array as its workspace, against mikv_decode_step with a caller
workspace, through the C ABI.  Both run the same kernels, so the results
must be identical bit for bit (codes, scales, positions, map, scores,
attention output and probabilities).  Two calls in a row share the scratch
array; the second runs a smaller cache, so anything it read from the first
call's leftovers would show."""
import numpy as np
import pytest
import torch

from paper_2402_18096_amd import mikv, workloads
from tests.parity import gather_gpu_state

pytestmark = pytest.mark.gpu


def _pair(wl, steps):
    k, v = workloads.prefill_kv(wl, "cuda")
    sc = workloads.initial_scores(wl, "cuda")
    qp = workloads.prefill_queries(wl, "cuda") if wl.balanced else None
    q, kn, vn = workloads.decode_inputs(wl, steps, "cuda")
    decs = []
    for _ in range(2):
        d = mikv.MikvDecoder(wl, max_len=wl.context + steps, device="cuda", fused=True)
        d.prefill(k, v, sc, qp)
        d.probs_hi.fill_(-1.0)
        d.probs_lo.fill_(-1.0)
        decs.append(d)
    return decs, (q, kn, vn)


def _same(a: mikv.MikvDecoder, b: mikv.MikvDecoder, tag):
    sa, sb = gather_gpu_state(a.cache), gather_gpu_state(b.cache)
    for key in sa:
        if sa[key] is None:
            assert sb[key] is None
            continue
        np.testing.assert_array_equal(sa[key], sb[key], err_msg=f"{tag}: {key}")
    for name in ("out", "probs_hi", "probs_lo"):
        x, y = getattr(a, name).cpu().numpy(), getattr(b, name).cpu().numpy()
        np.testing.assert_array_equal(x.view(np.uint32), y.view(np.uint32), err_msg=f"{tag}: {name}")
    assert int(a.cache.status.item()) == int(b.cache.status.item()) == 0


def _run(wl, steps, tag):
    (ref, na), (q, kn, vn) = _pair(wl, steps)
    for t in range(steps):
        ref.step_native(q[t], kn[t], vn[t])
        na.length += 1
        L = na.length
        mikv.mikv_decode_step_noalloc(na.cache, L, q[t], kn[t], vn[t], na.out, na.k_heavy(L), wl.window, na.probs_hi,
                                      na.probs_lo, na.balance, None, mikv.ATTN_ACCUMULATE)
        torch.cuda.synchronize()
        _same(ref, na, f"{tag} step {t}")


def test_noalloc_step_matches_workspace_step_twice_second_smaller():
    # first call: a long-context shape (many chunks, both pools, one demotion a step)
    wl1 = workloads.small_workload("long_context", batch=2, q_heads=4, kv_heads=4, context=6000)
    print(f"[noalloc] first: {wl1.n_heads} heads, context {wl1.context}", flush=True)
    _run(wl1, 3, "first")
    # second call, smaller: GQA, INT2 values tiled, a fraction of the first's workspace
    wl2 = workloads.small_workload("mistral_7b", batch=1, q_heads=8, kv_heads=2, context=700)
    print(f"[noalloc] second: {wl2.n_heads} heads, context {wl2.context}", flush=True)
    _run(wl2, 3, "second")

