"""Helpers shared by the GPU parity tests: run the HIP path and the oracle on
the same seeded inputs and compare.

The GPU keeps each head's tokens in two pools in slot order, with a position
array per pool; the oracle keeps them by position.  Slot order is not part
of the method (attention is permutation invariant), so the comparison maps
every GPU slot to its position and then compares, bit for bit, the set of
high-precision positions, every stored code, fp16 value and fp16
scale/zero, and the importance scores of the high-precision tokens (the only
scores the method reads again).  Attention outputs and probabilities are
compared within tolerance.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle
from paper_2402_18096_amd import mikv, workloads

SCALE = 1.0 / math.sqrt(128.0)
# Attention output tolerance (stated for the method's decode attention).
O_ATOL, O_RTOL = 2e-3, 1e-3
# Probabilities: fp32 scores and exponentials; derived bound, see the design notes.
P_ATOL, P_RTOL = 1e-9, 1e-3


def inputs(wl, steps, device="cpu"):
    k, v = workloads.prefill_kv(wl, device)
    sc = workloads.initial_scores(wl, device)
    qp = workloads.prefill_queries(wl, device) if wl.balanced else None
    q, kn, vn = workloads.decode_inputs(wl, steps, device)
    return k, v, sc, qp, q, kn, vn


def np16(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().numpy().view(np.float16)


def int2_values_token_major(v: np.ndarray, cap: int) -> np.ndarray:
    """Retained-pool 2-bit value codes [NH, cap * 32] in the tiled layout back
    to LSB-first token-major rows [NH, cap, 32].  Tiled: byte q of slot s (at
    s//32 * 1024 + 16 * (16 * (s%32 // 8) + q % 16) + 8 * (q // 16) + s % 8)
    holds channels q + 32 j at bits 2 j; token-major: channel c at bit 2 (c % 4)
    of byte c // 4."""
    slot = np.arange(cap)[:, None]
    ch = np.arange(128)[None, :]
    q, j = ch % 32, ch // 32
    idx = (slot // 32) * 1024 + 16 * (16 * ((slot % 32) // 8) + q % 16) + 8 * (q // 16) + slot % 8
    tiled = v.reshape(v.shape[0], -1)
    codes = (tiled[:, idx] >> (2 * j)[None]) & 3                      # [NH, cap, 128]
    c4 = codes.reshape(v.shape[0], cap, 32, 4).astype(np.uint8)
    return (c4[..., 0] | (c4[..., 1] << 2) | (c4[..., 2] << 4) | (c4[..., 3] << 6)).astype(np.uint8)


def gather_gpu_state(c: mikv.MikvCache, heads=None):
    """Position-indexed copy of the GPU cache: dict of numpy arrays [NH, L...]
    (with ``heads``, only those heads, in that order, selected on the device)."""
    sel = None if heads is None else torch.tensor(list(heads), device=c.n_hi.device)
    get = lambda t: None if t is None else (t if sel is None else t.index_select(0, sel)).cpu().numpy()
    n_hi = get(c.n_hi)
    n_lo = get(c.n_lo)
    hi_pos = get(c.hi_pos)
    lo_pos = get(c.lo_pos)
    hk = get(c.hi_k).view(np.uint16 if c.hi_bits == 16 else np.uint8)
    hv = get(c.hi_v).view(np.uint16 if c.hi_bits == 16 else np.uint8)
    acc = get(c.hi_acc)
    lk, lv = get(c.lo_k), get(c.lo_v)
    if c.values_tiled:
        lv = int2_values_token_major(lv, c.cap_lo)
    lkp = get(c.lo_kp)
    lvp = get(c.lo_vp).view(np.uint16)
    lkb = get(c.lo_kb)
    hkp, hvp = get(c.hi_kp), get(c.hi_vp)
    v16 = lambda x: None if x is None else x.view(np.uint16)
    return dict(n_hi=n_hi, n_lo=n_lo, hi_pos=hi_pos, lo_pos=lo_pos, hk=hk, hv=hv, acc=acc, lk=lk, lv=lv, lkp=v16(lkp),
                lvp=lvp, hkp=v16(hkp), hvp=v16(hvp), lkb=v16(lkb), map=get(c.map))


def compare_state(c: mikv.MikvCache, orc: oracle.OracleCache, heads=None, tag=""):
    """Bit-exact comparison of the GPU cache with the oracle's, by position
    (oracle head i against GPU head heads[i])."""
    s = gather_gpu_state(c, heads)
    L = orc.length
    names = list(range(orc.n_heads)) if heads is None else list(heads)
    for oh in range(orc.n_heads):
        gh, hid = oh, names[oh]  # row of the gathered state, GPU head index (for messages)
        nh, nl = int(s["n_hi"][gh]), int(s["n_lo"][gh])
        hp = s["hi_pos"][gh, :nh]
        lp = s["lo_pos"][gh, :nl]
        pos_hi = np.zeros(L, bool)
        pos_hi[hp] = True
        if orc.lo_bits:
            assert nh + nl == L, f"{tag} head {hid}: {nh}+{nl} tokens, expected {L}"
            assert len(set(hp.tolist()) | set(lp.tolist())) == L, f"{tag} head {hid}: positions not a partition"
        else:  # eviction: nothing is retained, every importance-pool position distinct
            assert nl == 0, f"{tag} head {hid}: {nl} retained tokens in an evicting cache"
            assert len(set(hp.tolist())) == nh, f"{tag} head {hid}: repeated positions"
        np.testing.assert_array_equal(pos_hi, orc.is_hi[oh, :L], err_msg=f"{tag} head {hid}: precision map")
        if s["map"] is not None:
            np.testing.assert_array_equal(s["map"][gh, :L].astype(bool), pos_hi, err_msg=f"{tag} head {hid}: map")
        # importance pool contents and scores
        hpk = (lambda x: x) if orc.hi_bits in (16, 8) else (lambda x: oracle.pack(x, orc.hi_bits))
        np.testing.assert_array_equal(s["hk"][gh, :nh], hpk(orc.hk[oh, hp]), err_msg=f"{tag} head {hid}: hi K")
        np.testing.assert_array_equal(s["hv"][gh, :nh], hpk(orc.hv[oh, hp]), err_msg=f"{tag} head {hid}: hi V")
        if orc.hi_bits != 16:
            np.testing.assert_array_equal(s["hkp"][gh, :nh, :, 0], orc.hk_a[oh, hp], err_msg=f"{tag} hi K alpha")
            np.testing.assert_array_equal(s["hkp"][gh, :nh, :, 1], orc.hk_b[oh, hp], err_msg=f"{tag} hi K beta")
            np.testing.assert_array_equal(s["hvp"][gh, :nh, :, 0], orc.hv_a[oh, hp], err_msg=f"{tag} hi V alpha")
            np.testing.assert_array_equal(s["hvp"][gh, :nh, :, 1], orc.hv_b[oh, hp], err_msg=f"{tag} hi V beta")
        np.testing.assert_array_equal(s["acc"][gh, :nh].view(np.uint32), orc.acc[oh, hp].view(np.uint32),
                                      err_msg=f"{tag} head {hid}: importance scores")
        # retained pool: packed codes and fp16 scale/zero
        bits = orc.lo_bits
        if bits == 0:
            continue
        np.testing.assert_array_equal(s["lk"][gh, :nl], oracle.pack(orc.lk[oh, lp], bits), err_msg=f"{tag} lo K codes")
        np.testing.assert_array_equal(s["lv"][gh, :nl], oracle.pack(orc.lv[oh, lp], bits), err_msg=f"{tag} lo V codes")
        if orc.key_block:
            # per-channel key parameters of every complete block
            nb = int(orc.kb_done[oh].sum())
            assert orc.kb_done[oh, :nb].all()
            np.testing.assert_array_equal(s["lkb"][gh, :nb, :, 0], orc.kb_a[oh, :nb], err_msg=f"{tag} key block alpha")
            np.testing.assert_array_equal(s["lkb"][gh, :nb, :, 1], orc.kb_b[oh, :nb], err_msg=f"{tag} key block beta")
        else:
            np.testing.assert_array_equal(s["lkp"][gh, :nl, :, 0], orc.lk_a[oh, lp], err_msg=f"{tag} lo K alpha")
            np.testing.assert_array_equal(s["lkp"][gh, :nl, :, 1], orc.lk_b[oh, lp], err_msg=f"{tag} lo K beta")
        np.testing.assert_array_equal(s["lvp"][gh, :nl, :, 0], orc.lv_a[oh, lp], err_msg=f"{tag} lo V alpha")
        np.testing.assert_array_equal(s["lvp"][gh, :nl, :, 1], orc.lv_b[oh, lp], err_msg=f"{tag} lo V beta")


def probs_by_position(c: mikv.MikvCache, probs_hi, probs_lo, n_hi, n_lo, hi_pos, lo_pos, L):
    """GPU probabilities (slot order) -> [NH, G, L] position order."""
    G = c.q_heads // c.kv_heads
    ph = probs_hi.cpu().numpy().reshape(c.n_heads, G, c.cap_hi)
    pl = probs_lo.cpu().numpy().reshape(c.n_heads, G, c.cap_lo)
    # an evicting cache gives evicted positions probability 0
    out = np.full((c.n_heads, G, L), np.nan if c.lo_bits else 0.0, np.float32)
    for h in range(c.n_heads):
        out[h][:, hi_pos[h, :n_hi[h]]] = ph[h, :, :n_hi[h]]
        out[h][:, lo_pos[h, :n_lo[h]]] = pl[h, :, :n_lo[h]]
    return out


class Lockstep:
    """GPU decoder and oracle side by side on one workload."""

    def __init__(self, wl, steps, fused=False, max_len=None):
        self.wl, self.steps = wl, steps
        self.k, self.v, self.sc, self.qp, self.q, self.kn, self.vn = inputs(wl, steps)
        self.dec = mikv.MikvDecoder(wl, max_len=max_len or wl.context + steps, device="cuda", fused=fused)
        NH, G = wl.n_heads, wl.group_size
        self.orc = oracle.OracleCache(NH, G, self.dec.max_len, wl.hi_bits, wl.lo_bits, wl.group,
                                      key_block=wl.key_block)
        self.bal = None

    def prefill(self):
        wl, NH, T = self.wl, self.wl.n_heads, self.wl.context
        self.dec.prefill(self.k.cuda(), self.v.cuda(), self.sc.cuda(),
                         self.qp.cuda() if self.qp is not None else None)
        if wl.balanced:
            qp = np16(self.qp).reshape(wl.batch, wl.kv_heads, wl.group_size, T, 128).reshape(NH, wl.group_size, T, 128)
            self.bal = oracle.balancer(qp, np16(self.k).reshape(NH, T, 128))
            got = self.dec.balance.cpu().numpy().reshape(NH, 128)
            np.testing.assert_array_equal(got.view(np.uint32), self.bal.view(np.uint32), err_msg="balancer")
        kh = oracle.heavy_budget(T, wl.ratio_num, wl.ratio_den, wl.window, wl.window_in_ratio)
        self.orc.prefill(np16(self.k).reshape(NH, T, 128), np16(self.v).reshape(NH, T, 128),
                         self.sc.numpy().reshape(NH, T), kh, wl.window, self.bal)
        torch.cuda.synchronize()
        compare_state(self.dec.cache, self.orc, tag="prefill")

    def step(self, t, check_state=True):
        wl, NH, G = self.wl, self.wl.n_heads, self.wl.group_size
        snap = {}

        def after_attention():
            c = self.dec.cache
            snap["n_hi"] = c.n_hi.cpu().numpy()
            snap["n_lo"] = c.n_lo.cpu().numpy()
            snap["hi_pos"] = c.hi_pos.cpu().numpy()
            snap["lo_pos"] = c.lo_pos.cpu().numpy()
            snap["p_hi"] = self.dec.probs_hi.clone()
            snap["p_lo"] = self.dec.probs_lo.clone()
            snap["out"] = self.dec.out.cpu().numpy()
            # the library's own scatter by position, compared below
            pos = torch.empty(c.batch * c.q_heads * self.dec.length, dtype=torch.float32, device="cuda")
            mikv.mikv_probs_by_position(c, self.dec.length, self.dec.probs_hi,
                                        self.dec.probs_lo if c.lo_bits else None, pos)
            snap["p_pos"] = pos.cpu().numpy()

        self.dec.step(self.q[t].cuda(), self.kn[t].cuda(), self.vn[t].cuda(), after_attention=after_attention,
                      emit_heavy=self.dec.cache.cap_hi <= 8192)
        torch.cuda.synchronize()
        L = self.dec.length
        self.orc.append(np16(self.kn[t]).reshape(NH, 128), np16(self.vn[t]).reshape(NH, 128), self.bal)
        o_ref, p_ref = self.orc.attend(np16(self.q[t]).reshape(NH, G, 128), SCALE, self.bal)
        o_gpu = snap["out"].reshape(NH, G, 128)
        np.testing.assert_allclose(o_gpu, o_ref, atol=O_ATOL, rtol=O_RTOL, err_msg=f"step {t}: attention output")
        p_gpu = probs_by_position(self.dec.cache, snap["p_hi"], snap["p_lo"], snap["n_hi"], snap["n_lo"],
                                  snap["hi_pos"], snap["lo_pos"], L)
        assert not np.isnan(p_gpu).any(), f"step {t}: a position got no probability"
        # the scatter moves the same floats: bit-exact
        np.testing.assert_array_equal(snap["p_pos"].reshape(NH, G, L), p_gpu,
                                      err_msg=f"step {t}: mikv_probs_by_position")
        np.testing.assert_allclose(p_gpu, p_ref, atol=P_ATOL, rtol=P_RTOL, err_msg=f"step {t}: probabilities")
        # importance update and selection fed with the GPU's probabilities
        self.orc.accumulate(p_gpu)
        kh = oracle.heavy_budget(L, wl.ratio_num, wl.ratio_den, wl.window, wl.window_in_ratio)
        self.orc.select(kh, wl.window)
        if check_state:
            compare_state(self.dec.cache, self.orc, tag=f"step {t}")
        if self.dec.heavy_idx is not None:
            # the sorted heavy-token list of the re-rank, bit for bit
            got = self.dec.heavy_idx.cpu().numpy().reshape(NH, kh)
            for h in range(NH):
                want = np.full(kh, -1, np.int64)
                hl = oracle.heavy_list(self.orc.acc[h], self.orc.is_hi[h], L, wl.window)[:kh]
                want[:len(hl)] = hl
                np.testing.assert_array_equal(got[h], want, err_msg=f"step {t} head {h}: heavy list")
        err_o = float(np.max(np.abs(o_gpu - o_ref)))
        err_p = float(np.max(np.abs(p_gpu - p_ref) / np.maximum(np.abs(p_ref), 1e-30)))
        # the largest share of the allowed output error used by any element
        self.last_margin = float(np.max(np.abs(o_gpu - o_ref) / (O_ATOL + O_RTOL * np.abs(o_ref))))
        return err_o, err_p


class SampledLockstep:
    """The benchmark's launch configuration at full size -- every head on the
    GPU, one mikv_decode_step per token with the importance update fused --
    checked on a sample of heads that the oracle follows.

    Inside one native step the top-k re-rank runs after attention and moves
    slots, so the slot -> position map at attention time is rebuilt from the
    state before the step plus the appended token (slot n_hi, position L-1).
    """

    def __init__(self, wl, steps, heads):
        self.wl, self.steps = wl, steps
        self.heads = sorted(set(int(h) for h in heads))
        NH, G, T = wl.n_heads, wl.group_size, wl.context
        dev = "cuda"
        self.dec = mikv.MikvDecoder(wl, max_len=T + steps, device=dev, fused=True)
        k, v = workloads.prefill_kv(wl, dev)
        sc = workloads.initial_scores(wl, dev)
        qp = workloads.prefill_queries(wl, dev) if wl.balanced else None
        self.q, self.kn, self.vn = workloads.decode_inputs(wl, steps, dev)
        sel = torch.tensor(self.heads, device=dev)
        self.sel = sel
        self.k_s = np16(k.reshape(NH, T, 128).index_select(0, sel))
        self.v_s = np16(v.reshape(NH, T, 128).index_select(0, sel))
        self.sc_s = sc.reshape(NH, T).index_select(0, sel).cpu().numpy()
        self.qp_s = np16(qp.reshape(NH, G, T, 128).index_select(0, sel)) if qp is not None else None
        self.dec.prefill(k, v, sc, qp)
        del k, v, qp
        self.orc = oracle.OracleCache(len(self.heads), G, self.dec.max_len, wl.hi_bits, wl.lo_bits, wl.group,
                                      key_block=wl.key_block)
        self.bal = None

    def prefill(self):
        wl, T = self.wl, self.wl.context
        if wl.balanced:
            self.bal = oracle.balancer(self.qp_s, self.k_s)
            got = self.dec.balance.reshape(wl.n_heads, 128).index_select(0, self.sel).cpu().numpy()
            np.testing.assert_array_equal(got.view(np.uint32), self.bal.view(np.uint32), err_msg="balancer")
        kh = oracle.heavy_budget(T, wl.ratio_num, wl.ratio_den, wl.window, wl.window_in_ratio)
        self.orc.prefill(self.k_s, self.v_s, self.sc_s, kh, wl.window, self.bal)
        torch.cuda.synchronize()
        compare_state(self.dec.cache, self.orc, heads=self.heads, tag="prefill")

    def _rows(self, t: torch.Tensor, per_head: int):
        """Rows of the sampled heads of a [B, H*, ...] tensor, as [S, per_head, ...] numpy."""
        NH = self.wl.n_heads
        x = t.reshape(NH, per_head, *t.shape[2:]).index_select(0, self.sel)
        return x.cpu().numpy()

    def step(self, t, check_state=True):
        wl, G = self.wl, self.wl.group_size
        c = self.dec.cache
        S = len(self.heads)
        n_hi0 = c.n_hi.index_select(0, self.sel).cpu().numpy()
        n_lo0 = c.n_lo.index_select(0, self.sel).cpu().numpy()
        hi_pos0 = c.hi_pos.index_select(0, self.sel).cpu().numpy()
        lo_pos0 = c.lo_pos.index_select(0, self.sel).cpu().numpy()
        self.dec.step_native(self.q[t], self.kn[t], self.vn[t])
        torch.cuda.synchronize()
        L = self.dec.length
        assert int(c.status.item()) == 0, f"step {t}: device status {int(c.status.item())}"
        # slot -> position map as it was during attention
        n_hi_att = n_hi0 + 1
        hi_pos_att = hi_pos0.copy()
        for i in range(S):
            hi_pos_att[i, n_hi0[i]] = L - 1
        ph = self._rows(self.dec.probs_hi, G)
        pl = self._rows(self.dec.probs_lo, G)
        p_gpu = np.full((S, G, L), np.nan if wl.lo_bits else 0.0, np.float32)
        for i in range(S):
            p_gpu[i][:, hi_pos_att[i, :n_hi_att[i]]] = ph[i, :, :n_hi_att[i]]
            p_gpu[i][:, lo_pos0[i, :n_lo0[i]]] = pl[i, :, :n_lo0[i]]
        o_gpu = self._rows(self.dec.out, G)
        kn = np16(self.kn[t].reshape(wl.n_heads, 128).index_select(0, self.sel))
        vn = np16(self.vn[t].reshape(wl.n_heads, 128).index_select(0, self.sel))
        self.orc.append(kn, vn, self.bal)
        q = np16(self.q[t].reshape(wl.n_heads, G, 128).index_select(0, self.sel))
        o_ref, p_ref = self.orc.attend(q, SCALE, self.bal)
        np.testing.assert_allclose(o_gpu, o_ref, atol=O_ATOL, rtol=O_RTOL, err_msg=f"step {t}: attention output")
        assert not np.isnan(p_gpu).any(), f"step {t}: a position got no probability"
        np.testing.assert_allclose(p_gpu, p_ref, atol=P_ATOL, rtol=P_RTOL, err_msg=f"step {t}: probabilities")
        self.orc.accumulate(p_gpu)
        kh = oracle.heavy_budget(L, wl.ratio_num, wl.ratio_den, wl.window, wl.window_in_ratio)
        self.orc.select(kh, wl.window)
        if check_state:
            compare_state(c, self.orc, heads=self.heads, tag=f"step {t}")
        return float(np.max(np.abs(o_gpu - o_ref)))
