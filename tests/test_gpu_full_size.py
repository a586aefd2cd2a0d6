"""GPU parity at the full workload sizes, in the launch configuration the
benchmark times (its own setup functions build the inputs and launch the
kernels).  The oracle quantizes the same input bits itself and evaluates
sampled outputs one by one:

  * Qwen3-14B-shaped causal prefill, 131072 tokens, 40 q / 8 kv heads: every
    quantizer output compared bit for bit, sampled rows of several heads;
  * Llama-3.1-8B-shaped paged decode, batch 32, contexts U[16384, 131072]:
    every query head of the shortest, the longest and one middle sequence;
  * the same decode with all 32 contexts at 131072 keys (partition 4096), over
    an MXFP4 K cache, and over an unsmoothed cache;
  * the MXFP4 variant, the BF16 / NVFP4 PV precision assignments, the other
    compensation placements and the unsmoothed variant of the 131072-token
    prefill;
  * the mixed serving step (Qwen shapes): a 32768-token chunk at position
    65536 over its paged prefix, plus 64 decode sequences, one launch sequence
    on one stream; sampled chunk rows and sampled decode sequences.
"""
import math
import os
import sys

import numpy as np
import pytest
import torch

from tests import helpers as H

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


@pytest.fixture(scope="module")
def mp():
    import paper_2609_33135_amd as mp
    assert torch.cuda.is_available()
    mp.lib()
    return mp


@pytest.fixture(scope="module")
def bench():
    import bench as B
    return B


@pytest.fixture(scope="module")
def W():
    from paper_2609_33135_amd import workloads
    return workloads


def _report(label, got, ref):
    max_abs, mean_rel, n_bad = H.compare_bf16(got, ref)
    print(f"{label}: {got.size} values, max|d| {max_abs:.3e} mean rel {mean_rel:.3e} "
          f"bad {n_bad}", flush=True)
    assert not np.isnan(H.bf16_f64(got)).any()
    assert mean_rel <= H.TOL_MEAN_REL and n_bad == 0, (label, n_bad, max_abs, mean_rel)


def _oracle_sequence_cache(orc, W, seed, b, ctx, h_q, h_kv, outliers, device="cuda", mx=False, smooth=True):
    """Oracle cache of one sequence's context (its own contiguous pages; the result
    does not depend on the physical page order), statistics computed on it."""
    q, k, v = W.gen_qkv(seed, [ctx], h_q, h_kv, outliers, device, seq_ids=[b])
    npg = max(1, (ctx + 1 + 63) // 64)
    pt = np.arange(npg, dtype=np.int32).reshape(1, npg)
    slots = np.arange(ctx, dtype=np.int64)
    ref = orc.quantize_qk(H.bits(q), H.bits(k), H.bits(v), np.array([0, ctx], np.int32), slots, npg,
                          (orc.SMOOTH if smooth else 0) | orc.COMPUTE_STATS | (orc.MXFP4 if mx else 0))
    del q, k, v
    return ref, pt


def _oracle_decode_one(orc, W, seed, b, kv, h_q, h_kv, outliers, partition, mx=False, smooth=True):
    ctx = kv - 1
    ref0, pt = _oracle_sequence_cache(orc, W, seed, b, ctx, h_q, h_kv, outliers, mx=mx, smooth=smooth)
    qn, kn, vn = W.gen_qkv(seed, [1], h_q, h_kv, outliers, "cuda", tok_offsets=[ctx], seq_ids=[b])
    ref = orc.quantize_qk(H.bits(qn), H.bits(kn), H.bits(vn), np.array([0, 1], np.int32),
                          np.array([ctx], np.int64), pt.shape[1],
                          (orc.SMOOTH if smooth else 0) | (orc.MXFP4 if mx else 0),
                          q_mean=ref0["q_mean"], k_mean=ref0["k_mean"], k_tscale=ref0["k_tscale"],
                          cache=ref0["cache"])
    items = np.array([(0, h) for h in range(h_q)], np.int32)
    o16, _ = orc.decode(ref["cache"], pt, np.array([kv], np.int32), ref["k_tscale"],
                        ref["q_codes"], ref["q_scales"], ref["q_tscale"], partition, items,
                        smooth=smooth, mxfp4=mx)
    return o16


def test_qwen_prefill_131072(orc, mp, bench, W):
    seq = 131072
    print(f"case: qwen prefill {seq} full-size (bench launch)", flush=True)
    st = bench.setup_prefill(torch, np, mp, W, seq, smooth=True)
    bench.run_quant(mp, st)
    bench.run_prefill(mp, st)
    torch.cuda.synchronize()
    out = H.bits(st["out"])
    wl = st["wl"]
    ref = orc.quantize_qk(H.bits(st["q"]), H.bits(st["k"]), H.bits(st["v"]),
                          np.array([0, seq], np.int32), W.slots_for(st["pt"], 0, range(seq)),
                          st["n_pages"], orc.SMOOTH | orc.COMPUTE_STATS)
    print("oracle quantization done", flush=True)
    # a2-a4 at full size: every code, scale, statistic and compensation value
    c = st["cache"]
    pairs = [("q_codes", st["qq"].codes), ("q_scales", st["qq"].scales),
             ("q_tscale", st["qq"].tscale), ("k_tscale", st["stats"].k_tscale)]
    for name, t in pairs:
        assert np.array_equal(t.cpu().numpy(), ref[name]), name
    assert np.array_equal(H.bits(st["stats"].q_mean), ref["q_mean"])
    assert np.array_equal(H.bits(st["stats"].k_mean), ref["k_mean"])
    rc = ref["cache"]
    for name in ("k_codes", "k_scales", "v_codes"):
        assert np.array_equal(getattr(c, name).cpu().numpy(), rc[name]), name
    assert np.array_equal(H.bits(c.ds), rc["ds"])
    # sampled output rows: the first tiles, the last tile, spread rows
    rng = np.random.default_rng(3)
    rows = np.unique(np.concatenate([np.arange(0, 130, 7), rng.integers(0, seq, 24),
                                     np.arange(seq - 130, seq, 9), [seq - 1]]))
    heads = [0, 7, 21, 39]
    items = np.array([(0, int(r), h) for r in rows for h in heads], np.int32)
    o16, _ = orc.prefill(rc, st["pt"], [seq], ref["k_tscale"], ref["q_codes"], ref["q_scales"],
                         ref["q_tscale"], [0, seq], [0], items)
    got = out[items[:, 1], items[:, 2]]
    _report(f"qwen prefill {seq}", got, o16)


def test_llama_decode_batch32(orc, mp, bench, W):
    print("case: llama decode batch 32 full-size (bench launch)", flush=True)
    sd = bench.setup_decode(torch, np, mp, W, 32)
    bench.run_decode(mp, sd)
    torch.cuda.synchronize()
    out = H.bits(sd["out"])
    wl = sd["wl"]
    lens = np.asarray(sd["lens"])
    order = np.argsort(lens)
    picks = [int(order[0]), int(order[len(order) // 2]), int(order[-1])]
    for b in picks:
        o16 = _oracle_decode_one(orc, W, wl.seed, b, int(lens[b]), wl.h_q, wl.h_kv, wl.outliers,
                                 sd["part"])
        _report(f"llama decode seq {b} kv {lens[b]} partition {sd['part']}", out[b], o16)


def test_llama_decode_128k_partition4096(orc, mp, bench, W):
    """The decode_128k point of the benchmark: 32 contexts of 131072 keys, the
    partition the benchmark's policy picks (4096 tokens); the first, a middle
    and the last sequence, every query head."""
    print("case: llama decode 32 x 131072 (bench launch)", flush=True)
    sd = bench.setup_decode(torch, np, mp, W, 32, ctx_range=(131072, 131072))
    assert sd["part"] == 4096, sd["part"]
    bench.run_decode(mp, sd)
    torch.cuda.synchronize()
    out = H.bits(sd["out"])
    wl = sd["wl"]
    lens = np.asarray(sd["lens"])
    for b in (0, 15, 31):
        o16 = _oracle_decode_one(orc, W, wl.seed, b, int(lens[b]), wl.h_q, wl.h_kv, wl.outliers,
                                 sd["part"])
        _report(f"llama decode 128k seq {b} partition {sd['part']}", out[b], o16)


@pytest.mark.parametrize("mx,smooth", [(True, True), (False, False)])
def test_llama_decode_batch32_variants(orc, mp, bench, W, mx, smooth):
    """The decode_mxfp4 and direct (unsmoothed cache) points of the benchmark, on
    the batch-32 Llama decode: the shortest, a middle and the longest sequence."""
    print(f"case: llama decode batch 32 mx={mx} smooth={smooth} full-size (bench launch)", flush=True)
    sd = bench.setup_decode(torch, np, mp, W, 32, mx=mx, smooth=smooth)
    bench.run_decode(mp, sd)
    torch.cuda.synchronize()
    out = H.bits(sd["out"])
    wl = sd["wl"]
    lens = np.asarray(sd["lens"])
    order = np.argsort(lens)
    for b in (int(order[0]), int(order[len(order) // 2]), int(order[-1])):
        o16 = _oracle_decode_one(orc, W, wl.seed, b, int(lens[b]), wl.h_q, wl.h_kv, wl.outliers,
                                 sd["part"], mx=mx, smooth=smooth)
        _report(f"llama decode mx={mx} smooth={smooth} seq {b} kv {lens[b]}", out[b], o16)


def test_qwen_prefill_131072_mxfp4(orc, mp, bench, W):
    """The MXFP4 variant at the full Qwen size in the benchmark's launch: every
    code and E8M0 scale bit for bit, sampled rows of four heads."""
    seq = 131072
    print(f"case: qwen prefill {seq} mxfp4 full-size (bench launch)", flush=True)
    st = bench.setup_prefill(torch, np, mp, W, seq, smooth=True, mx=True)
    bench.run_quant(mp, st)
    bench.run_prefill(mp, st)
    torch.cuda.synchronize()
    out = H.bits(st["out"])
    ref = orc.quantize_qk(H.bits(st["q"]), H.bits(st["k"]), H.bits(st["v"]),
                          np.array([0, seq], np.int32), W.slots_for(st["pt"], 0, range(seq)),
                          st["n_pages"], orc.SMOOTH | orc.COMPUTE_STATS | orc.MXFP4)
    print("oracle quantization done", flush=True)
    assert np.array_equal(st["qq"].codes.cpu().numpy(), ref["q_codes"])
    assert np.array_equal(st["qq"].scales.cpu().numpy(), ref["q_scales"])
    rc = ref["cache"]
    for name in ("k_codes", "k_scales", "v_codes"):
        assert np.array_equal(getattr(st["cache"], name).cpu().numpy(), rc[name]), name
    assert np.array_equal(H.bits(st["cache"].ds), rc["ds"])
    rng = np.random.default_rng(4)
    rows = np.unique(np.concatenate([np.arange(0, 130, 9), rng.integers(0, seq, 20),
                                     np.arange(seq - 130, seq, 13), [seq - 1]]))
    heads = [0, 9, 26, 39]
    items = np.array([(0, int(r), h) for r in rows for h in heads], np.int32)
    o16, _ = orc.prefill(rc, st["pt"], [seq], ref["k_tscale"], ref["q_codes"], ref["q_scales"],
                         ref["q_tscale"], [0, seq], [0], items, mxfp4=True)
    _report(f"qwen prefill {seq} mxfp4", out[items[:, 1], items[:, 2]], o16)


def test_qwen_prefill_131072_placements_and_direct(orc, mp, bench, W):
    """The other launches the benchmark times at the full Qwen size: the rank-one
    BF16 MFMA seed gives the default kernel's bytes; the element-wise placement
    (scores rounded in another FP32 order, so a P code near an FP8 rounding
    boundary may fall the other way) matches the oracle on sampled rows; the
    direct (unsmoothed) variant matches the oracle without compensation on
    sampled rows."""
    seq = 131072
    print(f"case: qwen prefill {seq} placements + direct (bench launches)", flush=True)
    st = bench.setup_prefill(torch, np, mp, W, seq, smooth=True)
    bench.run_quant(mp, st)
    bench.run_prefill(mp, st)
    torch.cuda.synchronize()
    base = H.bits(st["out"]).copy()
    st["flags"] = mp.SMOOTH | mp.SEED_MFMA
    bench.run_prefill(mp, st)
    torch.cuda.synchronize()
    assert np.array_equal(H.bits(st["out"]), base), "rank-one MFMA seed"
    st["flags"] = mp.SMOOTH | mp.SEED_ELEMWISE
    bench.run_prefill(mp, st)
    torch.cuda.synchronize()
    ew = H.bits(st["out"]).copy()
    rng = np.random.default_rng(6)
    rows = np.unique(np.concatenate([np.arange(0, 130, 13), rng.integers(0, seq, 12),
                                     np.arange(seq - 130, seq, 19), [seq - 1]]))
    heads = [3, 17, 38]
    items = np.array([(0, int(r), h) for r in rows for h in heads], np.int32)
    ref = orc.quantize_qk(H.bits(st["q"]), H.bits(st["k"]), H.bits(st["v"]),
                          np.array([0, seq], np.int32), W.slots_for(st["pt"], 0, range(seq)),
                          st["n_pages"], orc.SMOOTH | orc.COMPUTE_STATS)
    o16, _ = orc.prefill(ref["cache"], st["pt"], [seq], ref["k_tscale"], ref["q_codes"], ref["q_scales"],
                         ref["q_tscale"], [0, seq], [0], items)
    _report(f"qwen prefill {seq} element-wise", ew[items[:, 1], items[:, 2]], o16)
    del ref
    # direct: quantization and attention without the smoothing
    sd = bench.setup_prefill(torch, np, mp, W, seq, smooth=False)
    bench.run_quant(mp, sd)
    bench.run_prefill(mp, sd)
    torch.cuda.synchronize()
    ref = orc.quantize_qk(H.bits(sd["q"]), H.bits(sd["k"]), H.bits(sd["v"]),
                          np.array([0, seq], np.int32), W.slots_for(sd["pt"], 0, range(seq)),
                          sd["n_pages"], orc.COMPUTE_STATS)
    o16, _ = orc.prefill(ref["cache"], sd["pt"], [seq], ref["k_tscale"], ref["q_codes"], ref["q_scales"],
                         ref["q_tscale"], [0, seq], [0], items, smooth=False)
    _report(f"qwen prefill {seq} direct", H.bits(sd["out"])[items[:, 1], items[:, 2]], o16)


@pytest.mark.parametrize("pv", ["bf16", "nvfp4"])
def test_qwen_prefill_131072_pv_precisions(orc, mp, bench, W, pv):
    """The two other PV precision assignments (Sec. 3.1) at the full Qwen size in
    the benchmark's launch (precision_assignments): the V copy they read bit for
    bit, sampled rows of four heads."""
    seq = 131072
    print(f"case: qwen prefill {seq} pv={pv} full-size (bench launch)", flush=True)
    flag = mp.PV_BF16 if pv == "bf16" else mp.PV_NVFP4
    st = bench.setup_prefill(torch, np, mp, W, seq, smooth=True, pv=flag)
    bench.run_quant(mp, st)
    bench.run_prefill(mp, st)
    torch.cuda.synchronize()
    out = H.bits(st["out"])
    oflag = orc.PV_BF16 if pv == "bf16" else orc.PV_NVFP4
    ref = orc.quantize_qk(H.bits(st["q"]), H.bits(st["k"]), H.bits(st["v"]),
                          np.array([0, seq], np.int32), W.slots_for(st["pt"], 0, range(seq)),
                          st["n_pages"], orc.SMOOTH | orc.COMPUTE_STATS | oflag)
    print("oracle quantization done", flush=True)
    rc = ref["cache"]
    got_aux = H.bits(st["cache"].v_aux) if pv == "bf16" else st["cache"].v_aux.cpu().numpy()
    assert np.array_equal(got_aux.reshape(-1), np.asarray(rc["v_aux"]).reshape(-1))
    rng = np.random.default_rng(5)
    rows = np.unique(np.concatenate([np.arange(0, 130, 11), rng.integers(0, seq, 16),
                                     np.arange(seq - 130, seq, 17), [seq - 1]]))
    heads = [0, 13, 27, 39]
    items = np.array([(0, int(r), h) for r in rows for h in heads], np.int32)
    o16, _ = orc.prefill(rc, st["pt"], [seq], ref["k_tscale"], ref["q_codes"], ref["q_scales"],
                         ref["q_tscale"], [0, seq], [0], items, pv=oflag)
    _report(f"qwen prefill {seq} pv {pv}", out[items[:, 1], items[:, 2]], o16)


def test_mixed_step_qwen(orc, mp, W):
    """Chunked prefill of 32768 tokens at position 65536 over a 65536-token paged
    prefix, plus 64 decode sequences, all on one stream in one launch sequence."""
    print("case: mixed step (qwen shapes)", flush=True)
    pre, dec = W.mixed_step()
    dev = "cuda"
    d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    h_q, h_kv = pre.h_q, pre.h_kv
    prefix, chunk = pre.q_start[0], pre.seqlens[0]
    total = prefix + chunk
    # one cache for the whole step: the prefill request's pages, then the decode batch's
    pt_pre, np_pre = W.make_pages(pre.seed, [total])
    pt_dec, np_dec = W.make_pages(dec.seed, dec.kv_len)
    pt_dec = pt_dec + np_pre
    cache = mp.PagedCache(np_pre + np_dec, h_q, h_kv, dev)
    # --- before the step: the prefix of the request and the decode contexts are cached
    qp, kp, vp = W.gen_qkv(pre.seed, [prefix], h_q, h_kv, True, dev)
    st_pre = mp.SeqStats(1, h_q, h_kv, dev)
    mp.quantize_qk(qp, kp, vp, d(np.array([0, prefix], np.int32)),
                   d(W.slots_for(pt_pre, 0, range(prefix))), cache, st_pre,
                   mp.QuantQ(prefix, 1, h_q, dev), mp.SMOOTH | mp.COMPUTE_STATS, prefix)
    del qp, kp, vp
    st_dec = mp.SeqStats(dec.batch, h_q, h_kv, dev)
    for b, n in enumerate(dec.kv_len):
        ctx = n - 1
        q, k, v = W.gen_qkv(dec.seed, [ctx], h_q, h_kv, True, dev, seq_ids=[b])
        sb = mp.SeqStats(1, h_q, h_kv, dev)
        mp.quantize_qk(q, k, v, d(np.array([0, ctx], np.int32)), d(W.slots_for(pt_dec, b, range(ctx))),
                       cache, sb, mp.QuantQ(ctx, 1, h_q, dev), mp.SMOOTH | mp.COMPUTE_STATS, ctx)
        st_dec.q_mean[b].copy_(sb.q_mean[0])
        st_dec.k_mean[b].copy_(sb.k_mean[0])
        st_dec.k_tscale[b].copy_(sb.k_tscale[0])
        del q, k, v
    torch.cuda.synchronize()
    print("mixed step: caches written", flush=True)
    # --- the step: quantize the chunk and the decode tokens, then prefill and decode
    qc, kc, vc = W.gen_qkv(pre.seed, [chunk], h_q, h_kv, True, dev, tok_offsets=[prefix])
    qq_pre = mp.QuantQ(chunk, 1, h_q, dev)
    mp.quantize_qk(qc, kc, vc, d(np.array([0, chunk], np.int32)),
                   d(W.slots_for(pt_pre, 0, range(prefix, total))), cache, st_pre, qq_pre,
                   mp.SMOOTH, chunk)
    lens = np.asarray(dec.kv_len)
    qn, kn, vn = W.gen_qkv(dec.seed, [1] * dec.batch, h_q, h_kv, True, dev,
                           tok_offsets=[int(n) - 1 for n in lens])
    qq_dec = mp.QuantQ(dec.batch, dec.batch, h_q, dev)
    slots1 = np.array([W.slots_for(pt_dec, b, [int(lens[b]) - 1])[0] for b in range(dec.batch)],
                      np.int64)
    mp.quantize_qk(qn, kn, vn, d(np.arange(dec.batch + 1, dtype=np.int32)), d(slots1), cache,
                   st_dec, qq_dec, mp.SMOOTH, 1)
    out_pre = torch.empty((chunk, h_q, 128), dtype=torch.bfloat16, device=dev)
    mp.prefill(qq_pre, cache, st_pre, d(np.array([0, chunk], np.int32)),
               d(np.array([prefix], np.int32)), d(np.array([total], np.int32)), d(pt_pre), out_pre,
               chunk, mp.SMOOTH)
    part = mp.decode_choose_partition(lens, h_kv, torch.cuda.get_device_properties(0).multi_processor_count)
    maxp = max(math.ceil(n / part) for n in lens)
    ws = torch.empty(mp.decode_workspace_size(dec.batch, h_q, maxp) // 4, dtype=torch.float32,
                     device=dev)
    out_dec = torch.empty((dec.batch, h_q, 128), dtype=torch.bfloat16, device=dev)
    mp.decode_paged(qq_dec, cache, st_dec, d(lens.astype(np.int32)), d(pt_dec), out_dec, part, maxp,
                    ws, mp.SMOOTH)
    torch.cuda.synchronize()
    print("mixed step: launched", flush=True)
    got_pre = H.bits(out_pre)
    got_dec = H.bits(out_dec)
    # --- the same step as one fused launch: identical bytes, twice (counters reset)
    wsm = torch.zeros(mp.mixed_workspace_size(dec.batch, h_q, h_kv, maxp) // 4, dtype=torch.float32,
                      device=dev)
    for rep in range(2):
        fo_pre = torch.full_like(out_pre, float("nan"))
        fo_dec = torch.full_like(out_dec, float("nan"))
        mp.mixed_step(dict(qq=qq_pre, cache=cache, stats=st_pre, cu_seqlens_q=d(np.array([0, chunk], np.int32)),
                           q_start=d(np.array([prefix], np.int32)), kv_len=d(np.array([total], np.int32)),
                           page_table=d(pt_pre), out=fo_pre, max_seqlen_q=chunk),
                      dict(qq=qq_dec, cache=cache, stats=st_dec, kv_len=d(lens.astype(np.int32)),
                           page_table=d(pt_dec), out=fo_dec, partition_tokens=part, max_partitions=maxp),
                      wsm, mp.SMOOTH)
        torch.cuda.synchronize()
        assert np.array_equal(H.bits(fo_pre), got_pre), f"fused prefill differs (call {rep})"
        assert np.array_equal(H.bits(fo_dec), got_dec), f"fused decode differs (call {rep})"
    print("mixed step: fused launch identical", flush=True)
    # --- oracle: the request (prefix statistics frozen, chunk appended), sampled rows
    qp, kp, vp = W.gen_qkv(pre.seed, [prefix], h_q, h_kv, True, dev)
    npg = (total + 63) // 64
    pt_o = np.arange(npg, dtype=np.int32).reshape(1, npg)
    ref0 = orc.quantize_qk(H.bits(qp), H.bits(kp), H.bits(vp), np.array([0, prefix], np.int32),
                           np.arange(prefix, dtype=np.int64), npg, orc.SMOOTH | orc.COMPUTE_STATS)
    del qp, kp, vp
    ref = orc.quantize_qk(H.bits(qc), H.bits(kc), H.bits(vc), np.array([0, chunk], np.int32),
                          np.arange(prefix, total, dtype=np.int64), npg, orc.SMOOTH,
                          q_mean=ref0["q_mean"], k_mean=ref0["k_mean"], k_tscale=ref0["k_tscale"],
                          cache=ref0["cache"])
    assert np.array_equal(qq_pre.codes.cpu().numpy(), ref["q_codes"])
    assert np.array_equal(qq_pre.scales.cpu().numpy(), ref["q_scales"])
    rng = np.random.default_rng(5)
    rows = np.unique(np.concatenate([np.arange(0, 40, 3), rng.integers(0, chunk, 16), [chunk - 1]]))
    heads = [0, 19, 39]
    items = np.array([(0, int(r), h) for r in rows for h in heads], np.int32)
    o16, _ = orc.prefill(ref["cache"], pt_o, [total], ref["k_tscale"], ref["q_codes"],
                         ref["q_scales"], ref["q_tscale"], [0, chunk], [prefix], items)
    _report("mixed step chunked prefill", got_pre[items[:, 1], items[:, 2]], o16)
    # --- oracle: two decode sequences (shortest and longest)
    order = np.argsort(lens)
    for b in (int(order[0]), int(order[-1])):
        o16 = _oracle_decode_one(orc, W, dec.seed, b, int(lens[b]), h_q, h_kv, True, part)
        _report(f"mixed step decode seq {b} kv {lens[b]}", got_dec[b], o16)
