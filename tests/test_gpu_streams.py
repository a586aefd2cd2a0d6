"""Calls on caller-provided streams.

Every entry point enqueues its work on the stream it is given.  Prefill and
decode issued on two different (default-priority) streams over the same
read-only cache, with separate outputs and workspaces, must reproduce the
bytes of the same calls made one after the other; a quantization call on a
side stream must produce the same codes as on the default stream."""
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


def test_two_streams_match_serial(orc, mp):
    print("case: prefill and decode on two streams", flush=True)
    seqlens = [700, 260, 129]
    h_q, h_kv, part = 8, 2, 256
    run = H.Run(orc, mp, 107, seqlens, h_q, h_kv)
    B = run.B
    T = int(run.cu[-1])
    want_pre = run.prefill_gpu()
    want_dec = run.decode_last_gpu(part)

    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to("cuda")
    kv = dev(np.asarray(seqlens, np.int32))
    q_start = dev(np.zeros(B, np.int32))
    pt = dev(run.pt)
    last = torch.from_numpy((run.cu[1:] - 1).astype(np.int64)).cuda()
    qd = mp.QuantQ(B, B, h_q, "cuda")
    qd.codes.copy_(run.qq.codes.index_select(0, last))
    qd.scales.copy_(run.qq.scales.index_select(0, last))
    qd.tscale.copy_(run.qq.tscale)
    maxp = int(max((np.asarray(seqlens) + part - 1) // part))
    ws = torch.zeros(mp.decode_workspace_size(B, h_q, maxp) // 4, dtype=torch.float32, device="cuda")
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    for rep in range(3):
        pre = torch.full((T, h_q, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
        dec = torch.full((B, h_q, 128), float("nan"), dtype=torch.bfloat16, device="cuda")
        torch.cuda.synchronize()
        with torch.cuda.stream(s1):
            mp.prefill(run.qq, run.cache, run.stats, run.cu_d, q_start, kv, pt, pre, max(seqlens), mp.SMOOTH,
                       stream=s1)
        with torch.cuda.stream(s2):
            mp.decode_paged(qd, run.cache, run.stats, kv, pt, dec, part, maxp, ws, mp.SMOOTH, stream=s2)
        s1.synchronize()
        s2.synchronize()
        assert np.array_equal(H.bits(pre), want_pre), f"round {rep}: prefill on a side stream"
        assert np.array_equal(H.bits(dec), want_dec), f"round {rep}: decode on a side stream"


def test_quantize_on_side_stream(orc, mp):
    print("case: quantize on a side stream", flush=True)
    seqlens = [333, 64]
    run = H.Run(orc, mp, 109, seqlens, 8, 2)
    want = run.gpu_quant()
    cache = mp.PagedCache(run.cache.num_pages, 8, 2, "cuda", smooth=True)
    stats = mp.SeqStats(run.B, 8, 2, "cuda")
    qq = mp.QuantQ(int(run.cu[-1]), run.B, 8, "cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        mp.quantize_qk(run.q, run.k, run.v, run.cu_d, run.slots_d, cache, stats, qq, run.flags, max(seqlens),
                       stream=s)
    s.synchronize()
    got = dict(q_codes=qq.codes, q_scales=qq.scales, k_codes=cache.k_codes, k_scales=cache.k_scales,
               v_codes=cache.v_codes, ds=cache.ds, q_mean=stats.q_mean, k_mean=stats.k_mean,
               k_tscale=stats.k_tscale, q_tscale=qq.tscale)
    for k_, t in got.items():
        a = H.bits(t) if t.dtype == torch.bfloat16 else t.detach().cpu().numpy()
        assert np.array_equal(a, want[k_]), k_
