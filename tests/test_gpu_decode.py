"""GPU parity of split-KV paged decode against the oracle (Sec. 5.3, Sec. 6).

Flow per test, mirrored on both sides: prefill-time cache write of the
context (statistics computed and frozen), decode-time append of the new token
(centered against the frozen means, its K/V/Delta_S written to the cache
first), then one decode query per sequence over all kv_len keys.
"""
import numpy as np
import pytest
import torch

from tests import helpers as H

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def mp():
    import paper_2609_33135_amd as mp
    assert torch.cuda.is_available()
    mp.lib()
    return mp


class DecodeRun:
    def __init__(self, orc, mp, seed, kv_lens, h_q, h_kv, smooth=True, outliers=True, mxfp4=False):
        self.orc, self.mp = orc, mp
        self.kv = np.asarray(kv_lens, np.int32)
        B = len(kv_lens)
        self.B, self.h_q, self.h_kv, self.smooth = B, h_q, h_kv, smooth
        self.mxfp4 = mxfp4
        ctx = [int(n) - 1 for n in kv_lens]
        self.pt, n_pages = H.make_pages(seed, kv_lens)
        self.n_pages = max(n_pages, 1)
        flags_s = (mp.SMOOTH if smooth else 0) | (mp.MXFP4 if mxfp4 else 0)
        oflags_s = (orc.SMOOTH if smooth else 0) | (orc.MXFP4 if mxfp4 else 0)
        # 1) context cache write with statistics
        q, k, v = H.gen_qkv(seed, ctx, h_q, h_kv, outliers, "cuda")
        cu = np.concatenate([[0], np.cumsum(ctx)]).astype(np.int32)
        slots = np.concatenate([H.slots_for(self.pt, b, np.arange(n)) for b, n in enumerate(ctx)]) \
            .astype(np.int64)
        self.cache = mp.PagedCache(self.n_pages, h_q, h_kv, "cuda")
        self.stats = mp.SeqStats(B, h_q, h_kv, "cuda")
        qq0 = mp.QuantQ(int(cu[-1]), B, h_q, "cuda")
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()
        mp.quantize_qk(q, k, v, dev(cu), dev(slots), self.cache, self.stats, qq0,
                       flags_s | mp.COMPUTE_STATS, max(max(ctx), 0))
        ref0 = orc.quantize_qk(H.bits(q), H.bits(k), H.bits(v), cu, slots, self.n_pages,
                               oflags_s | orc.COMPUTE_STATS)
        del q, k, v, qq0
        # 2) append the new token of every sequence (its own counter position)
        qn, kn, vn = H.gen_qkv(seed, [1] * B, h_q, h_kv, outliers, "cuda", tok_offsets=ctx)
        cu1 = np.arange(B + 1, dtype=np.int32)
        slots1 = np.array([H.slots_for(self.pt, b, [ctx[b]])[0] for b in range(B)], np.int64)
        self.qq = mp.QuantQ(B, B, h_q, "cuda")
        mp.quantize_qk(qn, kn, vn, dev(cu1), dev(slots1), self.cache, self.stats, self.qq,
                       flags_s, 1)
        torch.cuda.synchronize()
        self.ref = orc.quantize_qk(H.bits(qn), H.bits(kn), H.bits(vn), cu1, slots1, self.n_pages,
                                   oflags_s, q_mean=ref0["q_mean"], k_mean=ref0["k_mean"],
                                   k_tscale=ref0["k_tscale"], cache=ref0["cache"])
        self.dev = dev

    def gpu(self, partition):
        mp = self.mp
        maxp = int(max((self.kv + partition - 1) // partition))
        # the contents on entry do not matter: start from random bits
        n_ws = mp.decode_workspace_size(self.B, self.h_q, maxp) // 4
        ws = torch.randint(-2**31, 2**31 - 1, (n_ws,), dtype=torch.int32, device="cuda").view(torch.float32)
        res = []
        for _ in range(2):   # the second call finds the first call's states in the workspace
            out = torch.full((self.B, self.h_q, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
            mp.decode_paged(self.qq, self.cache, self.stats, self.dev(self.kv), self.dev(self.pt), out,
                            partition, maxp, ws,
                            (mp.SMOOTH if self.smooth else 0) | (mp.MXFP4 if self.mxfp4 else 0))
            torch.cuda.synchronize()
            res.append(H.bits(out))
        assert np.array_equal(res[0], res[1]), "second call on the same workspace differs"
        return res[0]

    def oracle(self, partition, items=None):
        r = self.ref
        if items is None:
            items = np.array([(b, h) for b in range(self.B) for h in range(self.h_q)], np.int32)
        o16, _ = self.orc.decode(r["cache"], self.pt, self.kv, r["k_tscale"], r["q_codes"],
                                 r["q_scales"], r["q_tscale"], partition, items, smooth=self.smooth,
                                 mxfp4=self.mxfp4)
        return items, o16


def _cmp(run, partition, label):
    got = run.gpu(partition)
    items, ref = run.oracle(partition)
    g = got[items[:, 0], items[:, 1]]
    assert not np.isnan(H.bf16_f64(g)).any()
    max_abs, mean_rel, n_bad = H.compare_bf16(g, ref)
    print(f"{label} P={partition}: max|d| {max_abs:.3e} mean rel {mean_rel:.3e}", flush=True)
    assert mean_rel <= H.TOL_MEAN_REL and n_bad == 0, (n_bad, max_abs)


@pytest.mark.parametrize("partition", [128, 256, 1024])
def test_decode_small_llama_gqa(orc, mp, partition):
    print(f"case: decode small 32q/8kv P={partition}", flush=True)
    run = DecodeRun(orc, mp, 41, [1, 2, 127, 129, 700, 1500], 32, 8)
    _cmp(run, partition, "small llama")


def test_decode_qwen_gqa5(orc, mp):
    print("case: decode qwen 40q/8kv", flush=True)
    run = DecodeRun(orc, mp, 43, [300, 2049, 4000], 40, 8)
    _cmp(run, 512, "qwen")


def test_decode_direct(orc, mp):
    print("case: decode direct", flush=True)
    run = DecodeRun(orc, mp, 47, [999, 64], 8, 2, smooth=False)
    _cmp(run, 256, "direct")


def test_decode_medium_contexts(orc, mp):
    print("case: decode medium contexts", flush=True)
    rng = np.random.default_rng(3)
    lens = rng.integers(4000, 24000, 8)
    run = DecodeRun(orc, mp, 53, lens, 32, 8)
    part = mp.decode_choose_partition(lens, 8, 256)
    _cmp(run, part, "medium")


@pytest.mark.parametrize("h_q,h_kv", [(24, 12), (4, 1)])
def test_decode_many_sequences(orc, mp, h_q, h_kv):
    """70 sequences (the device-side pair numbering scans 64 sequences at a
    time), lengths from 1 to 700 with several one-partition sequences, and KV
    head counts that are not a multiple of 8."""
    print(f"case: decode 70 sequences {h_q}q/{h_kv}kv", flush=True)
    rng = np.random.default_rng(79)
    lens = rng.integers(1, 700, 70)
    lens[[0, 5, 63, 64, 69]] = [1, 128, 129, 700, 2]
    run = DecodeRun(orc, mp, 79, lens, h_q, h_kv)
    _cmp(run, 128, f"70 seqs {h_q}/{h_kv}")


def test_decode_large_batch_grid(orc, mp):
    """600 sequences: above 512 the kernel switches from the packed block map
    to the three-dimensional grid; both must reach every partition once."""
    print("case: decode 600 sequences 8q/2kv", flush=True)
    rng = np.random.default_rng(83)
    lens = rng.integers(1, 400, 600)
    lens[[0, 511, 512, 599]] = [1, 399, 129, 257]
    run = DecodeRun(orc, mp, 83, lens, 8, 2)
    _cmp(run, 128, "600 seqs 8/2")


def test_decode_matches_prefill_last_row(orc, mp):
    """With one partition covering the context, decode of the last token equals
    the last row of prefill over the same cache (same tiles, same order)."""
    print("case: decode vs prefill last row", flush=True)
    n = 777
    run = H.Run(orc, mp, 61, [n], 8, 2)
    pre = run.prefill_gpu()
    qq = mp.QuantQ(1, 1, 8, "cuda")
    qq.codes.copy_(run.qq.codes[n - 1:n])
    qq.scales.copy_(run.qq.scales[n - 1:n])
    qq.tscale.copy_(run.qq.tscale)
    ws = torch.empty(mp.decode_workspace_size(1, 8, 1) // 4, dtype=torch.float32, device="cuda")
    out = torch.empty((1, 8, 128), dtype=torch.bfloat16, device="cuda")
    mp.decode_paged(qq, run.cache, run.stats, torch.tensor([n], dtype=torch.int32, device="cuda"),
                    torch.from_numpy(run.pt).cuda(), out, 1024, 1, ws, mp.SMOOTH)
    torch.cuda.synchronize()
    a = H.bf16_f64(H.bits(out)[0])
    b = H.bf16_f64(pre[n - 1])
    assert np.max(np.abs(a - b)) <= 2 ** -7 * np.max(np.abs(b))


@pytest.mark.parametrize("smooth", [True, False])
def test_decode_mxfp4(orc, mp, smooth):
    """MXFP4 variant: QK on the scaled FP4 MFMA against the oracle's MXFP4 mode."""
    print(f"case: decode mxfp4 smooth={smooth}", flush=True)
    run = DecodeRun(orc, mp, 71, [1, 130, 777, 2500], 32, 8, smooth=smooth, mxfp4=True)
    _cmp(run, 256, f"mxfp4 smooth={smooth}")
