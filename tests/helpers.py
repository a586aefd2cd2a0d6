"""Helpers shared by the GPU parity tests: build seeded workloads, run the HIP
path through the C ABI and the CPU oracle on the same input bits, compare."""
from __future__ import annotations

import numpy as np
import torch

from paper_2609_33135_amd import workloads as W

TOL_MAX_ABS = 1e-2      # bf16 vs bf16, element-wise
TOL_MEAN_REL = 1e-3     # sum |a - b| / sum |b|


def bf16_f64(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


gen_qkv = W.gen_qkv
make_pages = W.make_pages
slots_for = W.slots_for
bits = W.bits


def bf16_ulp(x: np.ndarray) -> np.ndarray:
    """Spacing of BF16 values at |x| (8 significant bits)."""
    ax = np.maximum(np.abs(x), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(ax)) - 7)


# Running totals over every comparison of the session (printed by conftest at
# the end of the run): how many elements were compared, how many passed only
# through the one-ulp clause (|a - b| > 1e-2 but within one BF16 ulp, |x| >= 2),
# and the largest |a - b| among elements whose magnitudes are below 2.
TALLY = {"elements": 0, "ulp_clause_only": 0, "max_abs_below_2": 0.0}


def compare_bf16(got_bits, ref_bits, what=""):
    """Element-wise bar: |a - b| <= 1e-2, or at most one BF16 unit in the last
    place of the larger magnitude (outputs above 2 have a BF16 spacing of
    2^-6 > 1e-2, so one rounding step is the finest difference the format can
    express there).  Elements below 2 in magnitude are held to 1e-2 exactly.
    Returns (max |a - b| over elements, mean relative error, number of
    elements failing the bar); the session tally counts the elements that
    pass only through the ulp clause."""
    a = bf16_f64(got_bits)
    b = bf16_f64(ref_bits)
    diff = np.abs(a - b)
    max_abs = float(diff.max()) if diff.size else 0.0
    mean_rel = float(diff.sum() / max(np.abs(b).sum(), 1e-30))
    mag = np.maximum(np.abs(a), np.abs(b))
    allow = np.maximum(TOL_MAX_ABS, bf16_ulp(mag))
    bad = diff > allow
    small = mag < 2.0
    bad |= small & (diff > TOL_MAX_ABS)
    n_bad = int(bad.sum())
    TALLY["elements"] += int(diff.size)
    TALLY["ulp_clause_only"] += int(((diff > TOL_MAX_ABS) & ~bad).sum())
    if small.any():
        TALLY["max_abs_below_2"] = max(TALLY["max_abs_below_2"], float(diff[small].max()))
    return max_abs, mean_rel, n_bad


class Run:
    """One quantize (+ optional prefill) through the HIP path and the oracle."""

    def __init__(self, orc, mp, seed, seqlens, h_q, h_kv, outliers=True, smooth=True,
                 tscale_unit=False, shuffle=True, device="cuda", mxfp4=False, pv=None,
                 qkv=None, stale_fill=False, spare_pages=0):
        """pv: None, "bf16" or "nvfp4" (precision assignment of the PV product).
        qkv: explicit (q, k, v) bf16 device tensors instead of the seeded recipe.
        stale_fill: fill every cache plane with 0xFF bytes (E4M3 NaN codes, BF16
        NaN compensation) before the quantization pass, as a recycled page would
        hold; spare_pages: extra cache pages no sequence maps."""
        self.orc, self.mp = orc, mp
        self.mxfp4 = mxfp4
        self.pv = pv
        self.pv_flag = {None: 0, "bf16": mp.PV_BF16, "nvfp4": mp.PV_NVFP4}[pv]
        self.pv_orc = {None: 0, "bf16": orc.PV_BF16, "nvfp4": orc.PV_NVFP4}[pv]
        self.seqlens = list(seqlens)
        self.h_q, self.h_kv = h_q, h_kv
        self.smooth = smooth
        B = len(seqlens)
        self.B = B
        q, k, v = gen_qkv(seed, seqlens, h_q, h_kv, outliers, device) if qkv is None else qkv
        self.q, self.k, self.v = q, k, v
        cu = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32)
        self.cu = cu
        self.pt, self.n_pages = make_pages(seed, seqlens, shuffle)
        slots = np.concatenate([slots_for(self.pt, b, np.arange(n)) for b, n in enumerate(seqlens)]) \
            if cu[-1] > 0 else np.zeros(0, np.int64)
        self.slots = slots
        flags = (mp.SMOOTH if smooth else 0) | mp.COMPUTE_STATS | (mp.TSCALE_UNIT if tscale_unit else 0) \
            | (mp.MXFP4 if mxfp4 else 0) | self.pv_flag
        self.flags = flags
        # HIP path
        T = int(cu[-1])
        self.cache = mp.PagedCache(max(self.n_pages, 1) + spare_pages, h_q, h_kv, device, smooth=True,
                                   pv=self.pv_flag)
        if stale_fill:
            for plane in (self.cache.k_codes, self.cache.k_scales, self.cache.v_codes):
                plane.fill_(0xFF)
            self.cache.ds.view(torch.int16).fill_(-1)
        self.stats = mp.SeqStats(B, h_q, h_kv, device)
        self.qq = mp.QuantQ(T, B, h_q, device)
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)
        self.cu_d = dev(cu)
        self.slots_d = dev(slots)
        mp.quantize_qk(q, k, v, self.cu_d, self.slots_d, self.cache, self.stats, self.qq, flags,
                       max(seqlens) if seqlens else 0)
        torch.cuda.synchronize()
        # oracle on the same bits
        self.ref = orc.quantize_qk(bits(q), bits(k), bits(v), cu, slots, max(self.n_pages, 1) + spare_pages,
                                   (orc.SMOOTH if smooth else 0) | orc.COMPUTE_STATS |
                                   (orc.TSCALE_UNIT if tscale_unit else 0) |
                                   (orc.MXFP4 if mxfp4 else 0) | self.pv_orc)

    def gpu_quant(self):
        c = self.cache
        out = dict(q_codes=self.qq.codes, q_scales=self.qq.scales, q_tscale=self.qq.tscale,
                   q_mean=self.stats.q_mean, k_mean=self.stats.k_mean,
                   k_tscale=self.stats.k_tscale, k_codes=c.k_codes, k_scales=c.k_scales,
                   v_codes=c.v_codes, ds=c.ds)
        res = {}
        for k_, t in out.items():
            if t.dtype == torch.bfloat16:
                res[k_] = bits(t)
            else:
                res[k_] = t.detach().cpu().numpy()
        return res

    def prefill_gpu(self, q_start=None, kv_len=None, extra_flags=0):
        mp = self.mp
        B = self.B
        q_start = np.zeros(B, np.int32) if q_start is None else np.asarray(q_start, np.int32)
        kv_len = np.asarray(self.seqlens if kv_len is None else kv_len, np.int32)
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
        T = int(self.cu[-1])
        out = torch.full((T, self.h_q, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
        mp.prefill(self.qq, self.cache, self.stats, self.cu_d, dev(q_start), dev(kv_len),
                   dev(self.pt), out, max(self.seqlens),
                   (mp.SMOOTH if self.smooth else 0) | (mp.MXFP4 if self.mxfp4 else 0) | self.pv_flag
                   | extra_flags)
        torch.cuda.synchronize()
        return bits(out)

    def prefill_oracle(self, items, q_start=None, kv_len=None):
        B = self.B
        q_start = np.zeros(B, np.int32) if q_start is None else np.asarray(q_start, np.int32)
        kv_len = np.asarray(self.seqlens if kv_len is None else kv_len, np.int32)
        r = self.ref
        o16, o64 = self.orc.prefill(r["cache"], self.pt, kv_len, r["k_tscale"], r["q_codes"],
                                    r["q_scales"], r["q_tscale"], self.cu, q_start, items,
                                    smooth=self.smooth, mxfp4=self.mxfp4, pv=self.pv_orc)
        return o16, o64

    def decode_last_gpu(self, partition, kv_len=None, extra_flags=0):
        """Decode with each sequence's last query token over its whole cache (the
        query's own key included); returns bf16 bits [B][H_q][128]."""
        mp = self.mp
        B = self.B
        last = self.cu[1:] - 1
        qq = mp.QuantQ(B, B, self.h_q, "cuda")
        idx = torch.from_numpy(last.astype(np.int64)).cuda()
        qq.codes.copy_(self.qq.codes.index_select(0, idx))
        qq.scales.copy_(self.qq.scales.index_select(0, idx))
        qq.tscale.copy_(self.qq.tscale)
        kv = np.asarray(self.seqlens if kv_len is None else kv_len, np.int32)
        maxp = int(max((kv + partition - 1) // partition))
        ws = torch.empty(mp.decode_workspace_size(B, self.h_q, maxp) // 4, dtype=torch.float32,
                         device="cuda")
        out = torch.full((B, self.h_q, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
        mp.decode_paged(qq, self.cache, self.stats, dev(kv), dev(self.pt), out, partition, maxp, ws,
                        (mp.SMOOTH if self.smooth else 0) | (mp.MXFP4 if self.mxfp4 else 0)
                        | extra_flags)
        torch.cuda.synchronize()
        return bits(out)

    def decode_last_oracle(self, partition, kv_len=None):
        r = self.ref
        last = self.cu[1:] - 1
        kv = np.asarray(self.seqlens if kv_len is None else kv_len, np.int32)
        items = np.array([(b, h) for b in range(self.B) for h in range(self.h_q)], np.int32)
        o16, _ = self.orc.decode(r["cache"], self.pt, kv, r["k_tscale"], r["q_codes"][last],
                                 r["q_scales"][last], r["q_tscale"], partition, items,
                                 smooth=self.smooth, mxfp4=self.mxfp4)
        return o16.reshape(self.B, self.h_q, 128)

