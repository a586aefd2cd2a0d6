"""GPU parity at the edges of the input contract.

* Extreme magnitudes (Sec. 2.1 Eq. 1 with the power-of-two second-level
  scale): query and key heads near 1e-17, where both tensor scales sit at the
  bottom of their range, and tiny queries against huge keys, where they sit at
  opposite ends.  The scales' product and its inverse enter the kernels as the
  softmax factor and the compensation scale.
* Recycled cache pages (Sec. 6, paged KV cache): every cache plane filled
  with 0xFF bytes before the quantization pass (E4M3 NaN codes, BF16 NaN
  compensation values), sequence lengths that end inside a page and inside a
  128-key tile, spare pages no sequence maps, several decode partitions, and
  the one-launch mixed step.  The kernels must read only the slots a sequence
  owns, or mask what they read past its end before it can reach the output.
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


def _check(label, got, ref):
    max_abs, mean_rel, n_bad = H.compare_bf16(got, ref)
    print(f"{label}: {got.size} values, max|d| {max_abs:.3e} mean rel {mean_rel:.3e} bad {n_bad}",
          flush=True)
    assert not np.isnan(H.bf16_f64(got)).any(), label
    assert n_bad == 0 and mean_rel <= H.TOL_MEAN_REL, (label, n_bad, max_abs, mean_rel)


def _all_items(run):
    return np.array([(b, i, h) for b, n in enumerate(run.seqlens) for i in range(n)
                     for h in range(run.h_q)], np.int32)


def _prefill_vs_oracle(run, label):
    got = run.prefill_gpu()
    items = _all_items(run)
    ref, _ = run.prefill_oracle(items)
    rows = run.cu[items[:, 0]] + items[:, 1]
    _check(label, got[rows, items[:, 2]], ref)
    return got


def _scaled_qkv(seed, seqlens, h_q, h_kv, q_scale, k_scale):
    q, k, v = H.gen_qkv(seed, seqlens, h_q, h_kv, True, "cuda")
    # powers of two: exact in BF16 in this range
    return (q.float() * q_scale).to(torch.bfloat16), (k.float() * k_scale).to(torch.bfloat16), v


@pytest.mark.parametrize("mxfp4", [False, True])
def test_tiny_heads(orc, mp, mxfp4):
    """Q and K near 1e-17 (x 2^-60): NVFP4 tensor scales both at 2^-63, so
    tQ * tK = 2^-126; every row attends uniformly."""
    print(f"case: tiny heads mxfp4={mxfp4}", flush=True)
    seqlens = [300, 77]
    qkv = _scaled_qkv(91, seqlens, 8, 2, 2.0 ** -60, 2.0 ** -60)
    run = H.Run(orc, mp, 91, seqlens, 8, 2, qkv=qkv, mxfp4=mxfp4)
    if not mxfp4:
        g = run.gpu_quant()
        assert np.all(g["q_tscale"] == np.float32(2.0 ** -63))
        assert np.all(g["k_tscale"] == np.float32(2.0 ** -63))
        assert np.array_equal(g["q_codes"], run.ref["q_codes"])
        assert np.array_equal(g["ds"][:run.n_pages], run.ref["cache"]["ds"][:run.n_pages])
    _prefill_vs_oracle(run, f"tiny heads prefill mxfp4={mxfp4}")
    for part in (128, 256):
        _check(f"tiny heads decode P={part}", run.decode_last_gpu(part), run.decode_last_oracle(part))


def test_tiny_queries_huge_keys(orc, mp):
    """Q x 2^-72 and K x 2^72 (about 2e-22 and 5e21): the query tensor scale is
    clamped at 2^-63 (its group scales drop into the E4M3 subnormals), the key
    tensor scale at 2^63 (its largest group scales saturate at 448), while the
    true scores stay of order one."""
    print("case: tiny queries, huge keys", flush=True)
    seqlens = [260, 129]
    qkv = _scaled_qkv(93, seqlens, 8, 2, 2.0 ** -72, 2.0 ** 72)
    run = H.Run(orc, mp, 93, seqlens, 8, 2, qkv=qkv)
    g = run.gpu_quant()
    assert np.all(g["q_tscale"] == np.float32(2.0 ** -63))
    assert np.all(g["k_tscale"] == np.float32(2.0 ** 63))
    for name in ("q_codes", "q_scales"):
        assert np.array_equal(g[name], run.ref[name]), name
    for name in ("k_codes", "k_scales", "v_codes", "ds"):
        assert np.array_equal(g[name][:run.n_pages], run.ref["cache"][name][:run.n_pages]), name
    _prefill_vs_oracle(run, "tiny q / huge k prefill")
    _check("tiny q / huge k decode", run.decode_last_gpu(128), run.decode_last_oracle(128))


@pytest.mark.parametrize("mxfp4", [False, True])
@pytest.mark.parametrize("smooth", [True, False])
def test_stale_cache_prefill_and_decode(orc, mp, mxfp4, smooth):
    """Cache planes start as 0xFF (NaN codes) plus two spare pages; lengths end
    inside pages and tiles.  Prefill and decode (several partitions) match the
    oracle, whose cache never holds such bytes."""
    print(f"case: stale cache mxfp4={mxfp4} smooth={smooth}", flush=True)
    seqlens = [1, 63, 65, 200, 333]
    run = H.Run(orc, mp, 95, seqlens, 8, 2, smooth=smooth, mxfp4=mxfp4, stale_fill=True,
                spare_pages=2)
    _prefill_vs_oracle(run, f"stale prefill mx={mxfp4} smooth={smooth}")
    for part in (128, 256, 384):
        _check(f"stale decode P={part}", run.decode_last_gpu(part), run.decode_last_oracle(part))
    # a shorter visible context than what was written: the tail keys hold valid
    # codes that must be masked like stale ones
    kv = [max(1, n - 5) for n in seqlens]
    _check("stale decode, kv_len below the written length", run.decode_last_gpu(256, kv_len=kv),
           run.decode_last_oracle(256, kv_len=kv))


def test_stale_cache_mixed_step(orc, mp):
    """The one-launch mixed step over a 0xFF-filled cache: prefill of every row
    plus decode of every sequence's last token, equal to the separate launches
    and to the oracle."""
    print("case: stale cache mixed step", flush=True)
    seqlens = [70, 129, 250]
    run = H.Run(orc, mp, 97, seqlens, 8, 2, stale_fill=True, spare_pages=1)
    sep_pre = _prefill_vs_oracle(run, "stale mixed: separate prefill")
    part = 128
    sep_dec = run.decode_last_gpu(part)
    _check("stale mixed: separate decode", sep_dec, run.decode_last_oracle(part))
    B = run.B
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
    last = run.cu[1:] - 1
    qd = mp.QuantQ(B, B, run.h_q, "cuda")
    idx = torch.from_numpy(last.astype(np.int64)).cuda()
    qd.codes.copy_(run.qq.codes.index_select(0, idx))
    qd.scales.copy_(run.qq.scales.index_select(0, idx))
    qd.tscale.copy_(run.qq.tscale)
    kv = np.asarray(seqlens, np.int32)
    maxp = int(max((kv + part - 1) // part))
    wsm = torch.zeros(mp.mixed_workspace_size(B, run.h_q, run.h_kv, maxp) // 4, dtype=torch.float32,
                      device="cuda")
    T = int(run.cu[-1])
    for rep in range(2):
        out_pre = torch.full((T, run.h_q, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
        out_dec = torch.full((B, run.h_q, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
        mp.mixed_step(dict(qq=run.qq, cache=run.cache, stats=run.stats, cu_seqlens_q=run.cu_d,
                           q_start=dev(np.zeros(B, np.int32)), kv_len=dev(kv), page_table=dev(run.pt),
                           out=out_pre, max_seqlen_q=max(seqlens)),
                      dict(qq=qd, cache=run.cache, stats=run.stats, kv_len=dev(kv),
                           page_table=dev(run.pt), out=out_dec, partition_tokens=part,
                           max_partitions=maxp),
                      wsm, mp.SMOOTH)
        torch.cuda.synchronize()
        assert np.array_equal(H.bits(out_pre), sep_pre), f"mixed prefill differs (call {rep})"
        assert np.array_equal(H.bits(out_dec), sep_dec), f"mixed decode differs (call {rep})"
