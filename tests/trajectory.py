"""Free-running trajectory report: the GPU decoder and the oracle run the same
decode steps side by side, each ranking tokens with its own probabilities
(unlike the lock-step protocol, where the oracle takes the GPU's).  The two
importance scores then differ by floating-point rounding only, so the
precision maps agree until a near-tie at the top-k cut falls the other way;
the report counts where and when that happens.

Per step and sampled head it records: map entries that differ, the score gap
at the oracle's cut (last kept minus first demoted eligible token) and the
eligible tokens within 1e-6 of the cut score, and the largest |o_gpu - o_oracle|.

    python -m tests.trajectory --workload long_context --steps 64

prints one JSON report (GPU and oracle run in this process).
"""
from __future__ import annotations

import argparse
import json
import math

import numpy as np
import torch

import oracle
from paper_2402_18096_amd import mikv, workloads
from tests.parity import np16

SCALE = 1.0 / math.sqrt(128.0)


def cut_stats(orc: oracle.OracleCache, h: int, k_heavy: int, window: int):
    """Score gap at the cut and near-ties, from the oracle's scores before its selection."""
    L = orc.length
    pos = np.arange(L)
    elig = orc.is_hi[h, :L] & (pos < L - window)
    acc = np.sort(orc.acc[h, :L][elig].astype(np.float64))[::-1]
    if k_heavy <= 0 or k_heavy >= len(acc):
        return None, 0
    cut = acc[k_heavy - 1]
    return float(acc[k_heavy - 1] - acc[k_heavy]), int((np.abs(acc - cut) < 1e-6).sum())


def run_report(wl, steps: int, heads) -> dict:
    heads = sorted(set(int(h) for h in heads))
    NH, G, T = wl.n_heads, wl.group_size, wl.context
    dev = "cuda"
    dec = mikv.MikvDecoder(wl, max_len=T + steps, device=dev, fused=True)
    k, v = workloads.prefill_kv(wl, dev)
    sc = workloads.initial_scores(wl, dev)
    q, kn, vn = workloads.decode_inputs(wl, steps, dev)
    sel = torch.tensor(heads, device=dev)
    ks = np16(k.reshape(NH, T, 128).index_select(0, sel))
    vs = np16(v.reshape(NH, T, 128).index_select(0, sel))
    scs = sc.reshape(NH, T).index_select(0, sel).cpu().numpy()
    assert not wl.balanced, "the report covers unbalanced workloads"
    dec.prefill(k, v, sc)
    del k, v
    orc = oracle.OracleCache(len(heads), G, dec.max_len, wl.hi_bits, wl.lo_bits, wl.group, key_block=wl.key_block)
    orc.prefill(ks, vs, scs, dec.k_heavy(T), wl.window)
    rows = []
    for t in range(steps):
        dec.step_native(q[t], kn[t], vn[t])
        torch.cuda.synchronize()
        L = dec.length
        sub = lambda x, per: x.reshape(NH, per, *x.shape[2:]).index_select(0, sel)
        orc.append(np16(sub(kn[t], 1)[:, 0]), np16(sub(vn[t], 1)[:, 0]))
        o_ref, p_ref = orc.attend(np16(sub(q[t], G)), SCALE)
        orc.accumulate(p_ref)                                  # the oracle's own probabilities
        kh = dec.k_heavy(L)
        stats = [cut_stats(orc, i, kh, wl.window) for i in range(len(heads))]
        orc.select(kh, wl.window)
        gmap = dec.cache.map.index_select(0, sel)[:, :L].cpu().numpy().astype(bool)
        diff = (gmap != orc.is_hi[:, :L]).sum(1)
        o_gpu = sub(dec.out, G).cpu().numpy()
        rows.append({"step": t, "map_diff": diff.tolist(), "cut_gap": [s[0] for s in stats],
                     "near_ties": [s[1] for s in stats], "max_abs_o_diff": float(np.abs(o_gpu - o_ref).max())})
    first = next((r["step"] for r in rows if any(r["map_diff"])), None)
    gaps = [g for r in rows for g in r["cut_gap"] if g is not None]
    return {"workload": wl.name, "heads": heads, "steps": steps, "first_map_divergence": first,
            "map_diff_last": rows[-1]["map_diff"], "min_cut_gap": min(gaps) if gaps else None,
            "near_tie_steps": sum(1 for r in rows if any(n > 1 for n in r["near_ties"])),
            "max_abs_o_diff": max(r["max_abs_o_diff"] for r in rows),
            "max_abs_o_diff_before_divergence": max((r["max_abs_o_diff"] for r in rows
                                                     if first is None or r["step"] < first), default=None),
            "per_step": rows}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="long_context")
    ap.add_argument("--steps", type=int, default=64)
    args = ap.parse_args()
    wl = workloads.WORKLOADS[args.workload]
    rep = run_report(wl, args.steps, [0, wl.n_heads // 2 + 1, wl.n_heads - 1])
    print(json.dumps(rep))


if __name__ == "__main__":
    main()
